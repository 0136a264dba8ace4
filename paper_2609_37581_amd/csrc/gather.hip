// Row gather / sequence compaction (Sec. 4.1: the kept visual rows go to the
// LLM; Sec. 4.2: the K_2 kept visual rows and every prefix and text row go to
// the remaining layers).  Output row r of sample b reads input row
//   r                        for r < P,
//   P + idx[b, r - P]        for P <= r < P + n_kept,
//   r - n_kept + K_in        after that,
// as raw 16-byte vectors, so every tensor is copied bit for bit.  One launch
// covers up to four row tensors (grid z) plus the int64 position planes.
#include "common.hpp"
#include "kernels.hpp"

namespace trevs {

__device__ __forceinline__ int src_row(const GatherArgs& a, int b, int r) {
  if (r < a.P) return r;
  if (r < a.P + a.n_kept) {
    const int i = a.idx[(size_t)b * a.n_kept + (r - a.P)];
    return a.P + min(max(i, 0), a.K_in - 1);  // indices come from the selection, always in range
  }
  return r - a.n_kept + a.K_in;
}

__global__ __launch_bounds__(kGatherThreads) void gather_kernel(GatherArgs a) {
  const int tid = threadIdx.x;
  const int b = blockIdx.y, z = blockIdx.z;
  const int r0 = blockIdx.x * kGatherRowsPerBlock;
  if (z < a.n_tensors) {
    const GatherTensor t = a.t[z];
    const int tpr = 1 << t.tpr_log2;
    const int sub = tid >> t.tpr_log2, v0 = tid & (tpr - 1);
    const int vpr = t.row_bytes >> 4;
    const int rows_par = kGatherThreads >> t.tpr_log2;
    for (int rr = sub; rr < kGatherRowsPerBlock; rr += rows_par) {
      const int ro = r0 + rr;
      if (ro >= a.rows_out) break;
      const int ri = src_row(a, b, ro);
      const uint8_t* src = t.src + (size_t)b * t.src_bstride + (size_t)ri * t.row_bytes;
      uint8_t* dst = t.dst + (size_t)b * t.dst_bstride + (size_t)ro * t.row_bytes;
      for (int v = v0; v < vpr; v += 4 * tpr) {
        u32x4 x[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int vv = v + u * tpr;
          x[u] = vv < vpr ? ldg16(src + (size_t)vv * 16) : zero4();
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int vv = v + u * tpr;
          if (vv < vpr) stg16_stream(dst + (size_t)vv * 16, x[u]);
        }
      }
    }
    return;
  }
  // position-id planes
  for (int e = tid; e < a.n_pos * kGatherRowsPerBlock; e += kGatherThreads) {
    const int p = e / kGatherRowsPerBlock, rr = e - p * kGatherRowsPerBlock;
    const int ro = r0 + rr;
    if (ro >= a.rows_out) continue;
    const size_t plane = (size_t)p * a.B + b;
    a.pos_out[plane * a.rows_out + ro] = a.pos[plane * a.S + src_row(a, b, ro)];
  }
}

hipError_t launch_gather(const GatherArgs& a, hipStream_t s) {
  const int zdim = a.n_tensors + (a.pos ? 1 : 0);
  const dim3 grid((a.rows_out + kGatherRowsPerBlock - 1) / kGatherRowsPerBlock, a.B, zdim);
  hipLaunchKernelGGL(gather_kernel, grid, dim3(kGatherThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace trevs
