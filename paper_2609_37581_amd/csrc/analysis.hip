// Diagnostics of the preliminary analysis (Sec. 3): the visual attention
// profile of every head and its text sensitivity between two questions
// (Eq. (1)), and the Spearman rank correlation of visual saliency and textual
// relevance within the top-K saliency set.
#include "common.hpp"
#include "kernels.hpp"

namespace trevs {

// ---------------------------------------------------------------------------
// Visual profile of one head: profile[i] = (1/T_b) sum_{q<T_b} A[h,q,i] with
// A the text->vision attention of the statistics pass (its row log-sum-exps
// come in through lse2).  A workgroup owns V visual tokens of one (sample,
// query head); workgroups of one (sample, KV head) are numbered
// consecutively and mapped onto one XCD, so the key tile they share stays in
// that L2.  The key tile sits in LDS; wave w takes the 32-row text blocks
// w, w+QW, ..., recomputes the logits on the matrix cores (operand A = text
// rows, operand B = key rows), turns them into attention and sums them
// in-lane over its text rows.  The two half-waves and the waves are then
// summed through LDS.
// ---------------------------------------------------------------------------
template <class In, int DH, int QW>
__global__ __launch_bounds__(64 * QW) void t2v_profile_kernel(ProfileArgs a) {
  constexpr int ROWB = DH * In::kBytes;
  constexpr int HALFB = ROWB / 2;
  constexpr int NF = HALFB / 64;
  constexpr int NT = 64 * QW;
  constexpr int VB = ROWB <= 256 ? 2 : 1;  // 32-token blocks per workgroup
  constexpr int V = 32 * VB;
  constexpr int LROW = ROWB + 16;
  constexpr int CPR = ROWB / 16;
  constexpr int TV = V * CPR;
  constexpr int TVT = (TV + NT - 1) / NT;
  __shared__ __attribute__((aligned(16))) uint8_t klds[V * LROW];
  __shared__ float red[QW][V];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, col = lane & 31;
  const int lin = xcd_remap(blockIdx.x, gridDim.x);
  const int hl = lin % a.G;
  const int tile = (lin / a.G) % a.n_vtiles;
  const int bg = lin / (a.G * a.n_vtiles);
  const int g = bg % a.H_kv, b = bg / a.H_kv;
  const int h = g * a.G + hl, i0 = tile * V;
  const size_t seq0 = (size_t)b * a.S;

  // key rows i0..i0+V-1 of KV head g (rows past K_in re-read the last row)
  {
    const uint8_t* kbase = reinterpret_cast<const uint8_t*>(a.k) + (seq0 + a.P) * a.H_kv * ROWB +
                           (size_t)g * ROWB;
    const size_t kstride = (size_t)a.H_kv * ROWB;
    u32x4 kv[TVT];
#pragma unroll
    for (int k = 0; k < TVT; ++k) {
      const int v = min(tid + k * NT, TV - 1), row = v / CPR, c = v - row * CPR;
      kv[k] = ldg16(kbase + (size_t)min(i0 + row, a.K_in - 1) * kstride + c * 16);
    }
#pragma unroll
    for (int k = 0; k < TVT; ++k) {
      const int v = tid + k * NT;
      if (v < TV) {
        const int row = v / CPR, c = v - row * CPR;
        *reinterpret_cast<u32x4*>(&klds[row * LROW + c * 16]) = kv[k];
      }
    }
  }
  __syncthreads();

  const int Tb = a.text_len ? a.text_len[b] : a.T_max;
  const int n_qblk = (Tb + 31) / 32;
  float tot[VB];
#pragma unroll
  for (int vb = 0; vb < VB; ++vb) tot[vb] = 0.f;
  for (int qb = wave; qb < n_qblk; qb += QW) {
    const int qrow = min(qb * 32 + col, a.T_max - 1);
    const uint8_t* qp = reinterpret_cast<const uint8_t*>(a.q) +
                        ((seq0 + a.P + a.K_in + qrow) * a.H_q + h) * ROWB + half * HALFB;
    u32x4 qf[NF][4];
#pragma unroll
    for (int f = 0; f < NF; ++f)
#pragma unroll
      for (int j = 0; j < 4; ++j) qf[f][j] = ldg16(qp + f * 64 + j * 16);
    // rows of lse2 are padded to a multiple of 32: the block's reads stay in
    // the row; entries past T_b are masked below
    const float* lrow = a.lse2 + ((size_t)b * a.H_q + h) * a.T_pad + qb * 32 + 4 * half;
    float4 lse[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) lse[j] = *reinterpret_cast<const float4*>(lrow + 8 * j);
#pragma unroll
    for (int vb = 0; vb < VB; ++vb) {
      const uint8_t* p = &klds[(vb * 32 + col) * LROW + half * HALFB];
      f32x16 acc;
#pragma unroll
      for (int rr = 0; rr < 16; ++rr) acc[rr] = 0.f;
#pragma unroll
      for (int f = 0; f < NF; ++f) {
        u32x4 kf[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) kf[j] = *reinterpret_cast<const u32x4*>(p + f * 64 + j * 16);
        acc = mfma_frag(qf[f], kf, acc, In{});
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float l4[4] = {lse[j].x, lse[j].y, lse[j].z, lse[j].w};
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          const float e = __builtin_amdgcn_exp2f(fmaf(acc[4 * j + c], a.scale_log2e, -l4[c]));
          tot[vb] += (qb * 32 + mfma_row(4 * j + c, half) < Tb) ? e : 0.f;
        }
      }
    }
  }
  // a lane's registers are text rows of visual column vb*32 + col; the two
  // half-waves hold different rows of the same column
#pragma unroll
  for (int vb = 0; vb < VB; ++vb) {
    const float t = tot[vb] + __shfl_xor(tot[vb], 32, 64);
    if (half == 0) red[wave][vb * 32 + col] = t;
  }
  __syncthreads();
  const float inv_t = 1.f / (float)Tb;
  for (int t = tid; t < V; t += NT) {
    if (i0 + t < a.K_in) {
      float v = red[0][t];
#pragma unroll
      for (int w = 1; w < QW; ++w) v += red[w][t];
      a.profile[((size_t)b * a.H_q + h) * a.K_in + i0 + t] = v * inv_t;
    }
  }
}

// ---------------------------------------------------------------------------
// Text sensitivity, one workgroup per (head, sample): Eq. (1) between the
// two questions' profiles, with the dot product and squared norms summed in
// double (a sensitivity near 0 is a small difference of O(1) terms).
// ---------------------------------------------------------------------------
constexpr int kSensThreads = 256;

__device__ __forceinline__ double wave_sum_f64(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__global__ __launch_bounds__(kSensThreads) void sensitivity_kernel(SensitivityArgs a) {
  __shared__ double red[3][kSensThreads / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int h = blockIdx.x, b = blockIdx.y;
  const size_t base = ((size_t)b * a.H_q + h) * a.K_in;
  double d = 0.0, n0 = 0.0, n1 = 0.0;
  for (int i = tid; i < a.K_in; i += kSensThreads) {
    const double x = a.profile[0][base + i], y = a.profile[1][base + i];
    d = fma(x, y, d);
    n0 = fma(x, x, n0);
    n1 = fma(y, y, n1);
  }
  d = wave_sum_f64(d);
  n0 = wave_sum_f64(n0);
  n1 = wave_sum_f64(n1);
  if (lane == 0) {
    red[0][wave] = d;
    red[1][wave] = n0;
    red[2][wave] = n1;
  }
  __syncthreads();
  if (tid == 0) {
    double D = 0.0, N0 = 0.0, N1 = 0.0;
    for (int w = 0; w < kSensThreads / 64; ++w) {
      D += red[0][w];
      N0 += red[1][w];
      N1 += red[2][w];
    }
    a.ts[(size_t)b * a.H_q + h] = (float)(1.0 - D / sqrt(N0 * N1));
  }
}

// ---------------------------------------------------------------------------
// Spearman correlation within the top-K saliency set.  The average rank of
// token i in a K-vector x is r_i = #{x_j < x_i} + (#{x_j == x_i} + 1) / 2
// (1-based, ties sharing the mean of the ranks they span), so
// c_i = 2 r_i - (K + 1) is an integer in [1-K, K-1] that sums to zero: the
// centred rank, doubled.  The correlation of the ranks is
// sum c^v c^t / sqrt(sum (c^v)^2 sum (c^t)^2), and all three sums are exact
// in 64-bit integers.  A workgroup ranks kRankTile tokens (one per lane of
// every wave) against the whole set: the set's (s^v, s^t) pairs are staged
// through LDS in chunks, each wave counts over every 16th entry of a chunk
// (the same entry for all lanes, an LDS broadcast), and the counts of the
// waves are added through LDS.  A second kernel adds the workgroups'
// integer sums per sample and forms the ratio in double.
// ---------------------------------------------------------------------------
constexpr int kRankWaves = 16;
constexpr int kRankChunk = 1024;

__global__ __launch_bounds__(64 * kRankWaves) void spearman_rank_kernel(SpearmanArgs a) {
  __shared__ float2 vals[kRankChunk];
  __shared__ int cnt[4][kRankWaves][64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int tile = blockIdx.x, b = blockIdx.y;
  const int K = a.K;
  const int32_t* idx = a.idx + (size_t)b * K;
  const float* sv = a.sv + (size_t)b * a.N;
  const float* st = a.st + (size_t)b * a.N;
  const int i = tile * kRankTile + lane;
  const int ii = min(max(idx[min(i, K - 1)], 0), a.N - 1);
  const float vi = sv[ii], ti = st[ii];
  int lv = 0, ev = 0, lt = 0, et = 0;
  for (int c0 = 0; c0 < K; c0 += kRankChunk) {
    const int n = min(kRankChunk, K - c0);
    for (int j = tid; j < n; j += 64 * kRankWaves) {
      const int jj = min(max(idx[c0 + j], 0), a.N - 1);
      vals[j] = make_float2(sv[jj], st[jj]);
    }
    __syncthreads();
    for (int j = wave; j < n; j += kRankWaves) {
      const float2 p = vals[j];
      lv += p.x < vi ? 1 : 0;
      ev += p.x == vi ? 1 : 0;
      lt += p.y < ti ? 1 : 0;
      et += p.y == ti ? 1 : 0;
    }
    __syncthreads();
  }
  cnt[0][wave][lane] = lv;
  cnt[1][wave][lane] = ev;
  cnt[2][wave][lane] = lt;
  cnt[3][wave][lane] = et;
  __syncthreads();
  if (wave == 0) {
    int LV = 0, EV = 0, LT = 0, ET = 0;
#pragma unroll
    for (int w = 0; w < kRankWaves; ++w) {
      LV += cnt[0][w][lane];
      EV += cnt[1][w][lane];
      LT += cnt[2][w][lane];
      ET += cnt[3][w][lane];
    }
    long long cv = 0, ct = 0;
    if (i < K) {
      cv = 2LL * LV + EV + 1 - ((long long)K + 1);
      ct = 2LL * LT + ET + 1 - ((long long)K + 1);
    }
    long long s_vt = cv * ct, s_vv = cv * cv, s_tt = ct * ct;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      s_vt += __shfl_xor(s_vt, o, 64);
      s_vv += __shfl_xor(s_vv, o, 64);
      s_tt += __shfl_xor(s_tt, o, 64);
    }
    if (lane == 0) {
      long long* out = a.part + ((size_t)b * a.n_tiles + tile) * 4;
      out[0] = s_vt;
      out[1] = s_vv;
      out[2] = s_tt;
      out[3] = 0;
    }
  }
}

__global__ __launch_bounds__(64) void spearman_final_kernel(SpearmanArgs a, int B) {
  const int b = blockIdx.x * 64 + threadIdx.x;
  if (b >= B) return;
  long long s_vt = 0, s_vv = 0, s_tt = 0;
  const long long* p = a.part + (size_t)b * a.n_tiles * 4;
  for (int t = 0; t < a.n_tiles; ++t) {
    s_vt += p[4 * t];
    s_vv += p[4 * t + 1];
    s_tt += p[4 * t + 2];
  }
  a.rho[b] = (s_vv == 0 || s_tt == 0) ? __builtin_nan("")
                                      : (double)s_vt / sqrt((double)s_vv * (double)s_tt);
}

// ---------------------------------------------------------------- launchers
static int profile_waves(int T_max) {
  const int qb = (T_max + 31) / 32;
  return qb >= 4 ? 4 : (qb >= 2 ? 2 : 1);
}

template <class In, int DH>
static void launch_profile_t(const ProfileArgs& a, hipStream_t s) {
  const dim3 grid(a.B * a.H_q * a.n_vtiles);
  switch (profile_waves(a.T_max)) {
    case 4: hipLaunchKernelGGL((t2v_profile_kernel<In, DH, 4>), grid, dim3(256), 0, s, a); break;
    case 2: hipLaunchKernelGGL((t2v_profile_kernel<In, DH, 2>), grid, dim3(128), 0, s, a); break;
    default: hipLaunchKernelGGL((t2v_profile_kernel<In, DH, 1>), grid, dim3(64), 0, s, a); break;
  }
}

template <class In>
static void launch_profile_d(const ProfileArgs& a, int dh, hipStream_t s) {
  if (dh == 64)
    launch_profile_t<In, 64>(a, s);
  else if (dh == 128)
    launch_profile_t<In, 128>(a, s);
  else
    launch_profile_t<In, 256>(a, s);
}

hipError_t launch_profile(const ProfileArgs& a, int dtype, int dh, hipStream_t s) {
  if (dtype == 1)
    launch_profile_d<BF16>(a, dh, s);
  else
    launch_profile_d<F32>(a, dh, s);
  return hipGetLastError();
}

hipError_t launch_sensitivity(const SensitivityArgs& a, int B, hipStream_t s) {
  hipLaunchKernelGGL(sensitivity_kernel, dim3(a.H_q, B), dim3(kSensThreads), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_spearman(const SpearmanArgs& a, int B, hipStream_t s) {
  hipLaunchKernelGGL(spearman_rank_kernel, dim3(a.n_tiles, B), dim3(64 * kRankWaves), 0, s, a);
  hipLaunchKernelGGL(spearman_final_kernel, dim3((B + 63) / 64), dim3(64), 0, s, a, B);
  return hipGetLastError();
}

}  // namespace trevs
