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

// The kept-index entry output row r would read (clamped to a valid entry, so
// it can be loaded unconditionally), and the source row given that entry.
__device__ __forceinline__ const int32_t* idx_entry(const GatherArgs& a, int b, int r) {
  return a.idx + (size_t)b * a.n_kept + min(max(r - a.P, 0), a.n_kept - 1);
}
__device__ __forceinline__ int src_row_of(const GatherArgs& a, int r, int i) {
  if (r < a.P) return r;
  if (r < a.P + a.n_kept) return a.P + min(max(i, 0), a.K_in - 1);  // indices come from the selection
  return r - a.n_kept + a.K_in;
}
__device__ __forceinline__ int src_row(const GatherArgs& a, int b, int r) {
  return src_row_of(a, r, *idx_entry(a, b, r));
}

// Buffer resource over one row: accesses at or past `bytes` read zero and
// write nothing, which masks the tail of a row without any branch.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t row_rsrc(const void* p, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), 0, bytes, kBufferRsrcWord3);
}

// A wave copies one output row of more than 1 KB, kGatherBatch 1 KB segments
// at a time, or kGatherShortRows rows of at most 1 KB (the K and V rows of a
// few heads), one per load.  All loads of a batch are issued before the
// first store, and each row's buffer bounds drop the bytes past its end (so
// rows up to 8 KB take one batch; the small batch keeps occupancy high).
__global__ __launch_bounds__(kGatherThreads) void gather_kernel(GatherArgs a) {
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int b = blockIdx.y, z = blockIdx.z;
  const int r0 = blockIdx.x * kGatherRowsPerBlock;
  if (z < a.n_tensors) {
    static_assert(kGatherRowsPerBlock == kGatherThreads / 64, "one long row per wave");
    const GatherTensor t = a.t[z];
    const size_t sb = (size_t)b * t.src_bstride, db = (size_t)b * t.dst_bstride;
    if (t.row_bytes <= 1024) {
      // short rows: blocks beyond rows_out / (waves * kGatherShortRows) are idle
      const int rb0 = (blockIdx.x * (kGatherThreads / 64) + wave) * kGatherShortRows;
      if (rb0 >= a.rows_out) return;
      // every source row is looked up before the first data load, so the
      // lookups do not wait behind the data
      int ient[kGatherShortRows];
#pragma unroll
      for (int k = 0; k < kGatherShortRows; ++k) ient[k] = *idx_entry(a, b, min(rb0 + k, a.rows_out - 1));
      int srow[kGatherShortRows];
#pragma unroll
      for (int k = 0; k < kGatherShortRows; ++k) srow[k] = src_row_of(a, min(rb0 + k, a.rows_out - 1), ient[k]);
      u32x4 x[kGatherShortRows];
#pragma unroll
      for (int k = 0; k < kGatherShortRows; ++k) {
        const __amdgpu_buffer_rsrc_t src = row_rsrc(t.src + sb + (size_t)srow[k] * t.row_bytes, t.row_bytes);
        x[k] = __builtin_amdgcn_raw_buffer_load_b128(src, lane * 16, 0, kCachePolicyStream);
      }
#pragma unroll
      for (int k = 0; k < kGatherShortRows; ++k) {
        // rows past the end were loaded again from the last row; store nothing
        const __amdgpu_buffer_rsrc_t dst = row_rsrc(t.dst + db + (size_t)(rb0 + k) * t.row_bytes,
                                                    rb0 + k < a.rows_out ? t.row_bytes : 0);
        __builtin_amdgcn_raw_buffer_store_b128(x[k], dst, lane * 16, 0, 0);
      }
      return;
    }
    const int row = r0 + wave;
    if (row >= a.rows_out) return;
    const __amdgpu_buffer_rsrc_t src =
        row_rsrc(t.src + sb + (size_t)src_row(a, b, row) * t.row_bytes, t.row_bytes);
    const __amdgpu_buffer_rsrc_t dst = row_rsrc(t.dst + db + (size_t)row * t.row_bytes, t.row_bytes);
    // (the whole offset goes in the bounds-checked vector operand)
    for (int o = lane * 16; o < t.row_bytes; o += kGatherBatch * 1024) {
      u32x4 x[kGatherBatch];
#pragma unroll
      for (int k = 0; k < kGatherBatch; ++k)
        x[k] = __builtin_amdgcn_raw_buffer_load_b128(src, o + k * 1024, 0, kCachePolicyStream);
#pragma unroll
      for (int k = 0; k < kGatherBatch; ++k) __builtin_amdgcn_raw_buffer_store_b128(x[k], dst, o + k * 1024, 0, 0);
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
