// Stage 2 (in-LLM) kernels: text->vision attention statistics, head variance
// and high-variance head set, and the token score (Sec. 4.2, Eq. (8)-(9)).
#include "common.hpp"
#include "kernels.hpp"

namespace trevs {

// ---------------------------------------------------------------------------
// Statistics pass.  For every (query head h, text row q) the row of logits
// x_i = scale * Q[q,h] . K[i, h/G] over the visual keys is reduced online to
// (max, sum e, sum e^2) with e = exp(x - max), in log2 units.  The grid is
// (split of the visual keys) x (group of 32-row column blocks) along x, KV
// head along y, sample along z.  Within a KV head the rows r = (h - g*G) *
// T_max + q of all G query heads share every key tile, which each lane feeds
// to the matrix cores as operand A (visual rows) against its own resident Q
// row as operand B, so a lane's 16 accumulators are 16 visual columns of its
// own text row: the softmax statistics stay in-lane.
// ---------------------------------------------------------------------------
template <class In, int DH, int NW>
__global__ __launch_bounds__(64 * NW) void t2v_stats_kernel(StatsArgs a) {
  constexpr int ROWB = DH * In::kBytes;
  constexpr int HALFB = ROWB / 2;
  constexpr int NF = HALFB / 64;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, col = lane & 31;
  const int split = blockIdx.x % a.n_split, rg = blockIdx.x / a.n_split;
  const int g = blockIdx.y, b = blockIdx.z;
  const int R = a.G * a.T_max;
  const int rblock = rg * NW + wave;
  if (rblock * 32 >= R) return;  // whole wave idle (no workgroup barrier in this kernel)
  const int r = rblock * 32 + col;
  const bool rvalid = r < R;
  const int hl = rvalid ? r / a.T_max : 0, q = rvalid ? r - hl * a.T_max : 0;
  const int h = g * a.G + hl;

  u32x4 qf[NF][4];
  {
    const uint8_t* qp = reinterpret_cast<const uint8_t*>(a.q) +
                        (((size_t)b * a.S + a.P + a.K_in + q) * a.H_q + h) * ROWB + half * HALFB;
#pragma unroll
    for (int f = 0; f < NF; ++f)
#pragma unroll
      for (int j = 0; j < 4; ++j) qf[f][j] = rvalid ? ldg16(qp + f * 64 + j * 16) : zero4();
  }
  const int i_begin = split * a.split_len;
  const int i_end = min(a.K_in, i_begin + a.split_len);
  const uint8_t* kbase = reinterpret_cast<const uint8_t*>(a.k) +
                         ((size_t)b * a.S + a.P) * a.H_kv * ROWB + (size_t)g * ROWB + half * HALFB;
  const size_t kstride = (size_t)a.H_kv * ROWB;

  float m = -INFINITY, l = 0.f, l2 = 0.f;
  for (int ib = i_begin; ib < i_end; ib += 32) {
    const int i = ib + col;
    const uint8_t* kp = kbase + (size_t)(i < i_end ? i : i_begin) * kstride;
    f32x16 acc;
#pragma unroll
    for (int rr = 0; rr < 16; ++rr) acc[rr] = 0.f;
#pragma unroll
    for (int f = 0; f < NF; ++f) {
      u32x4 kf[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) kf[j] = ldg16(kp + f * 64 + j * 16);
      acc = mfma_frag(kf, qf[f], acc, In{});
    }
    float y[16];
    float mb = -INFINITY;
#pragma unroll
    for (int rr = 0; rr < 16; ++rr) {
      y[rr] = (ib + mfma_row(rr, half) < i_end) ? acc[rr] * a.scale_log2e : -INFINITY;
      mb = fmaxf(mb, y[rr]);
    }
    if (mb > -INFINITY) {
      const float mn = fmaxf(m, mb);
      const float c = exp2f(m - mn);
      float s1 = 0.f, s2 = 0.f;
#pragma unroll
      for (int rr = 0; rr < 16; ++rr) {
        const float e = exp2f(y[rr] - mn);
        s1 += e;
        s2 = fmaf(e, e, s2);
      }
      l = fmaf(l, c, s1);
      l2 = fmaf(l2, c * c, s2);
      m = mn;
    }
  }
  const float mo = __shfl_xor(m, 32, 64), lo = __shfl_xor(l, 32, 64), l2o = __shfl_xor(l2, 32, 64);
  const float M = fmaxf(m, mo);
  float L = 0.f, L2 = 0.f;
  if (M > -INFINITY) {
    const float c1 = exp2f(m - M), c2 = exp2f(mo - M);
    L = l * c1 + lo * c2;
    L2 = l2 * c1 * c1 + l2o * c2 * c2;
  }
  if (half == 0 && rvalid)
    a.part[(((size_t)b * a.H_q + h) * a.T_max + q) * a.n_split + split] = make_float4(M, L, L2, 0.f);
}

// ---------------------------------------------------------------------------
// Head pass, one workgroup per sample.  Merges the split statistics of every
// (h, q) row into its log-sum-exp (optionally joined with the row's
// non-visual log-sum-exp), the population variance of the row's visual
// attention, the head variance u_h averaged over the valid text rows
// (Eq. (8)), and the n_keep heads first under (u desc, h asc).
// ---------------------------------------------------------------------------
constexpr int kMaxHeads = 256;

__global__ __launch_bounds__(256) void t2v_heads_kernel(HeadArgs a) {
  __shared__ float u_lds[kMaxHeads];
  __shared__ int sel_lds[kMaxHeads];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int b = blockIdx.x;
  const int Tb = a.text_len ? a.text_len[b] : a.T_max;
  const float invK = 1.f / (float)a.K_in;
  for (int h = wave; h < a.H_q; h += 4) {
    float vs = 0.f;
    for (int q = lane; q < a.T_max; q += 64) {
      const size_t row = ((size_t)b * a.H_q + h) * a.T_max + q;
      const float4* pp = a.part + row * a.n_split;
      float m = -INFINITY, l = 0.f, l2 = 0.f;
      for (int s = 0; s < a.n_split; ++s) {
        const float4 p = pp[s];
        if (p.x == -INFINITY) continue;
        const float mn = fmaxf(m, p.x);
        const float c1 = exp2f(m - mn), c2 = exp2f(p.x - mn);
        l = l * c1 + p.y * c2;
        l2 = l2 * c1 * c1 + p.z * c2 * c2;
        m = mn;
      }
      float lse2 = m + log2f(l);
      if (a.lse_rest) {
        const float r2 = a.lse_rest[row] * kLog2e;
        const float mx = fmaxf(lse2, r2);
        lse2 = mx + log2f(exp2f(lse2 - mx) + exp2f(r2 - mx));
      }
      a.lse2[row] = lse2;
      if (q < Tb) {
        const float f = exp2f(m - lse2);
        vs += f * f * (l2 - l * l * invK) * invK;
      }
    }
    vs = wave_sum(vs);
    if (lane == 0) u_lds[h] = vs / (float)Tb;
  }
  __syncthreads();
  for (int h = tid; h < a.H_q; h += 256) {
    const float u = u_lds[h];
    int rank = 0;
    for (int h2 = 0; h2 < a.H_q; ++h2) {
      const float u2 = u_lds[h2];
      rank += (u2 > u || (u2 == u && h2 < h)) ? 1 : 0;
    }
    sel_lds[h] = rank < a.n_keep;
    a.head_var[(size_t)b * a.H_q + h] = u;
  }
  __syncthreads();
  for (int h = tid; h < a.H_q; h += 256) {
    if (!sel_lds[h]) continue;
    int pos = 0;
    for (int h2 = 0; h2 < h; ++h2) pos += sel_lds[h2];
    if (pos < a.n_keep) a.head_sel[(size_t)b * a.n_keep + pos] = h;  // ranks are distinct for finite u
  }
}

// ---------------------------------------------------------------------------
// Token score.  A workgroup owns 32 visual tokens of one sample; wave w takes
// the 32-row text blocks w, w+QW, ...  For each selected head (ascending) the
// wave recomputes the logits on the matrix cores (operand A = its text rows,
// operand B = the 32 key rows of the head's KV group), turns them into
// attention with the row log-sum-exp of the head pass, and adds them up over
// heads in-lane; then max over valid text rows, across waves via LDS, and
// divide by |H*| (Eq. (9)).
// ---------------------------------------------------------------------------
template <class In, int DH, int QW>
__global__ __launch_bounds__(64 * QW) void t2v_score_kernel(ScoreArgs a) {
  constexpr int ROWB = DH * In::kBytes;
  constexpr int HALFB = ROWB / 2;
  constexpr int NF = HALFB / 64;
  __shared__ float pmax[QW][32];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, col = lane & 31;
  const int ib = blockIdx.x * 32, b = blockIdx.y;
  const int Tb = a.text_len ? a.text_len[b] : a.T_max;
  const int i = ib + col;
  const int i_ld = i < a.K_in ? i : a.K_in - 1;
  const size_t seq0 = (size_t)b * a.S;
  const uint8_t* kbase = reinterpret_cast<const uint8_t*>(a.k) +
                         ((seq0 + a.P + i_ld) * a.H_kv) * ROWB + half * HALFB;
  float pm = 0.f;
  for (int qb = wave; qb * 32 < Tb; qb += QW) {
    const int qrow = qb * 32 + col;
    const bool qvalid = qrow < a.T_max;
    const uint8_t* qbase = reinterpret_cast<const uint8_t*>(a.q) +
                           ((seq0 + a.P + a.K_in + (qvalid ? qrow : 0)) * a.H_q) * ROWB + half * HALFB;
    float accs[16];
#pragma unroll
    for (int rr = 0; rr < 16; ++rr) accs[rr] = 0.f;
    int gprev = -1;
    u32x4 kf[NF][4];
    for (int hi = 0; hi < a.n_keep; ++hi) {
      const int h = min(max(a.head_sel[(size_t)b * a.n_keep + hi], 0), a.H_q - 1);
      const int g = h / a.G;
      if (g != gprev) {
#pragma unroll
        for (int f = 0; f < NF; ++f)
#pragma unroll
          for (int j = 0; j < 4; ++j) kf[f][j] = ldg16(kbase + (size_t)g * ROWB + f * 64 + j * 16);
        gprev = g;
      }
      f32x16 acc;
#pragma unroll
      for (int rr = 0; rr < 16; ++rr) acc[rr] = 0.f;
#pragma unroll
      for (int f = 0; f < NF; ++f) {
        u32x4 qf[4];
#pragma unroll
        for (int j = 0; j < 4; ++j)
          qf[j] = qvalid ? ldg16(qbase + (size_t)h * ROWB + f * 64 + j * 16) : zero4();
        acc = mfma_frag(qf, kf[f], acc, In{});
      }
      const float* lrow = a.lse2 + ((size_t)b * a.H_q + h) * a.T_max;
#pragma unroll
      for (int rr = 0; rr < 16; ++rr) {
        const int qq = qb * 32 + mfma_row(rr, half);
        const float lse = qq < a.T_max ? lrow[qq] : 0.f;
        accs[rr] += exp2f(fmaf(acc[rr], a.scale_log2e, -lse));
      }
    }
#pragma unroll
    for (int rr = 0; rr < 16; ++rr)
      if (qb * 32 + mfma_row(rr, half) < Tb) pm = fmaxf(pm, accs[rr]);
  }
  pm = fmaxf(pm, __shfl_xor(pm, 32, 64));
  if (half == 0) pmax[wave][col] = pm;
  __syncthreads();
  if (tid < 32 && ib + tid < a.K_in) {
    float v = pmax[0][tid];
#pragma unroll
    for (int w = 1; w < QW; ++w) v = fmaxf(v, pmax[w][tid]);
    a.p[(size_t)b * a.K_in + ib + tid] = v / (float)a.n_keep;
  }
}

// ---------------------------------------------------------------- launchers
template <class In, int DH>
static void launch_stats_t(const StatsArgs& a, hipStream_t s) {
  const int nrb = (a.G * a.T_max + 31) / 32;
  const dim3 grid(a.n_split * a.n_rgroups, a.H_kv, a.B);
  if (nrb >= 4)
    hipLaunchKernelGGL((t2v_stats_kernel<In, DH, 4>), grid, dim3(256), 0, s, a);
  else if (nrb >= 2)
    hipLaunchKernelGGL((t2v_stats_kernel<In, DH, 2>), grid, dim3(128), 0, s, a);
  else
    hipLaunchKernelGGL((t2v_stats_kernel<In, DH, 1>), grid, dim3(64), 0, s, a);
}

template <class In>
static void launch_stats_d(const StatsArgs& a, int dh, hipStream_t s) {
  if (dh == 64)
    launch_stats_t<In, 64>(a, s);
  else if (dh == 128)
    launch_stats_t<In, 128>(a, s);
  else
    launch_stats_t<In, 256>(a, s);
}

hipError_t launch_stats(const StatsArgs& a, int dtype, int dh, hipStream_t s) {
  if (dtype == 1)
    launch_stats_d<BF16>(a, dh, s);
  else
    launch_stats_d<F32>(a, dh, s);
  return hipGetLastError();
}

hipError_t launch_heads(const HeadArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(t2v_heads_kernel, dim3(a.B), dim3(256), 0, s, a);
  return hipGetLastError();
}

int score_qblocks(int T_max) {
  const int qb = (T_max + 31) / 32;
  return qb >= 4 ? 4 : (qb >= 2 ? 2 : 1);
}

template <class In, int DH>
static void launch_score_t(const ScoreArgs& a, hipStream_t s) {
  const dim3 grid((a.K_in + 31) / 32, a.B);
  switch (score_qblocks(a.T_max)) {
    case 4: hipLaunchKernelGGL((t2v_score_kernel<In, DH, 4>), grid, dim3(256), 0, s, a); break;
    case 2: hipLaunchKernelGGL((t2v_score_kernel<In, DH, 2>), grid, dim3(128), 0, s, a); break;
    default: hipLaunchKernelGGL((t2v_score_kernel<In, DH, 1>), grid, dim3(64), 0, s, a); break;
  }
}

template <class In>
static void launch_score_d(const ScoreArgs& a, int dh, hipStream_t s) {
  if (dh == 64)
    launch_score_t<In, 64>(a, s);
  else if (dh == 128)
    launch_score_t<In, 128>(a, s);
  else
    launch_score_t<In, 256>(a, s);
}

hipError_t launch_score(const ScoreArgs& a, int dtype, int dh, hipStream_t s) {
  if (dtype == 1)
    launch_score_d<BF16>(a, dh, s);
  else
    launch_score_d<F32>(a, dh, s);
  return hipGetLastError();
}

}  // namespace trevs
