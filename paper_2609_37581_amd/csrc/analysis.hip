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
// come in through lse2).  A workgroup owns one (sample, query head) and one
// split of the visual keys; workgroups of one (sample, KV head) are numbered
// consecutively and mapped onto one XCD, so the keys the group's query heads
// share stay in that L2.  Wave w keeps the Q rows of text block w (of the
// current pass) resident as MFMA operand A; the 32-key tiles of the split
// stream through a ring of register stages into two alternating LDS buffers
// and are read by every wave as operand B, so a lane's 16 accumulators are
// 16 text rows of one visual column.  Each wave turns them into attention,
// sums its rows in-lane and across the half-waves, and parks the column sums
// in LDS; after the tile's barrier the first 32 threads add the waves' sums
// in a fixed order into the split's running column sums (deterministic).
// ---------------------------------------------------------------------------
// Key tiles in flight: about TREVS_PROFILE_RING_VECS 16-byte vectors per
// thread in registers.  A shallow ring keeps the kernel at 111 VGPRs, four
// waves per SIMD, which hides the loads better than a deep ring at two
// waves per SIMD (30.6 us against 38.3 us at the 16,384-token workload).
#ifndef TREVS_PROFILE_RING_VECS
#define TREVS_PROFILE_RING_VECS 2
#endif
constexpr int profile_ring(int vectors_per_tile) {
  return vectors_per_tile >= TREVS_PROFILE_RING_VECS ? 1
                                                     : TREVS_PROFILE_RING_VECS / vectors_per_tile;
}

template <class In, int DH, int QW>
__global__ __launch_bounds__(64 * QW) void t2v_profile_kernel(ProfileArgs a) {
  constexpr int ROWB = DH * In::kBytes;
  constexpr int HALFB = ROWB / 2;
  constexpr int NF = HALFB / 64;
  constexpr int NT = 64 * QW;
  constexpr int LROW = ROWB + 16;
  constexpr int CPR = ROWB / 16;
  constexpr int TV = 32 * CPR;  // 16-byte vectors of one key tile
  constexpr int TVT = (TV + NT - 1) / NT;
  constexpr int RING = profile_ring(TVT);
  __shared__ __attribute__((aligned(16))) uint8_t klds[2][32 * LROW];
  __shared__ float red[2][QW][32];
  __shared__ float colsum[kProfileSplitMax];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, col = lane & 31;
  const int lin = xcd_remap(blockIdx.x, gridDim.x);
  const int split = lin % a.n_split;
  const int hl = (lin / a.n_split) % a.G;
  const int bg = lin / (a.n_split * a.G);
  const int g = bg % a.H_kv, b = bg / a.H_kv;
  const int h = g * a.G + hl;
  const size_t seq0 = (size_t)b * a.S;
  const int i_begin = split * a.split_len;
  const int i_end = min(a.K_in, i_begin + a.split_len);
  const int n_tiles = (i_end - i_begin + 31) / 32;
  for (int t = tid; t < n_tiles * 32; t += NT) colsum[t] = 0.f;

  const uint8_t* kbase = reinterpret_cast<const uint8_t*>(a.k) + (seq0 + a.P) * a.H_kv * ROWB +
                         (size_t)g * ROWB;
  const size_t kstride = (size_t)a.H_kv * ROWB;
  // one key tile (rows ib..ib+31) into registers; rows past the split re-read
  // row i_begin (valid, cached)
  auto load_tile = [&](int ib, u32x4 (&dst)[TVT]) {
#pragma unroll
    for (int k = 0; k < TVT; ++k) {
      const int v = min(tid + k * NT, TV - 1), row = v / CPR, c = v - row * CPR;
      const int i = ib + row;
      dst[k] = ldg16(kbase + (size_t)(i < i_end ? i : i_begin) * kstride + c * 16);
    }
  };
  auto store_tile = [&](int buf, const u32x4 (&src)[TVT]) {
#pragma unroll
    for (int k = 0; k < TVT; ++k) {
      const int v = tid + k * NT;
      if (v < TV) {
        const int row = v / CPR, c = v - row * CPR;
        *reinterpret_cast<u32x4*>(&klds[buf][row * LROW + c * 16]) = src[k];
      }
    }
  };

  const int Tb = text_rows(a.text_len, b, a.T_max);
  const int n_qblk = (Tb + 31) / 32;
  const int n_pass = (n_qblk + QW - 1) / QW;  // uniform over the workgroup (barriers below)
  const int n_iter = (n_tiles + RING - 1) / RING;
  for (int pass = 0; pass < n_pass; ++pass) {
    // text block of this wave; a wave past the last block reads a valid block
    // and masks every row
    const int qb = pass * QW + wave;
    const int qbc = min(qb, n_qblk - 1);
    const int qrow = min(qbc * 32 + col, a.T_max - 1);
    const uint8_t* qp = reinterpret_cast<const uint8_t*>(a.q) +
                        ((seq0 + a.P + a.K_in + qrow) * a.H_q + h) * ROWB + half * HALFB;
    u32x4 qf[NF][4];
#pragma unroll
    for (int f = 0; f < NF; ++f)
#pragma unroll
      for (int j = 0; j < 4; ++j) qf[f][j] = ldg16(qp + f * 64 + j * 16);
    // rows of lse2 are padded to a multiple of 32: the block's reads stay in
    // the row; entries past T_b are masked below
    const float* lrow = a.lse2 + ((size_t)b * a.H_q + h) * a.T_pad + qbc * 32 + 4 * half;
    float nl[16];  // minus the row log-sum-exp, or -inf for a masked row
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float4 l = *reinterpret_cast<const float4*>(lrow + 8 * j);
      const float l4[4] = {l.x, l.y, l.z, l.w};
#pragma unroll
      for (int c = 0; c < 4; ++c)
        nl[4 * j + c] = (qb * 32 + mfma_row(4 * j + c, half) < Tb) ? -l4[c] : -INFINITY;
    }

    u32x4 ring[RING][TVT];
#pragma unroll
    for (int c = 0; c < RING; ++c) load_tile(i_begin + 32 * c, ring[c]);
    for (int it = 0; it < n_iter; ++it) {
#pragma unroll
      for (int c = 0; c < RING; ++c) {
        const int t = it * RING + c;
        // LDS buffer (t % 2) was last read at tile t - 2, before every wave
        // passed the barrier of tile t - 1
        store_tile(t & 1, ring[c]);
        load_tile(i_begin + 32 * (t + RING), ring[c]);
        __syncthreads();
        if (t < n_tiles) {
          const uint8_t* p = &klds[t & 1][col * LROW + half * HALFB];
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
          float sum = 0.f;
#pragma unroll
          for (int rr = 0; rr < 16; ++rr) sum += __builtin_amdgcn_exp2f(fmaf(acc[rr], a.scale_log2e, nl[rr]));
          sum += __shfl_xor(sum, 32, 64);
          if (half == 0) red[t & 1][wave][col] = sum;
        }
        // the sums parked at this tile are read after the next barrier, and
        // red[t & 1] is written again only after the one after it
        if (t >= 1 && t - 1 < n_tiles && tid < 32) {
          float v = 0.f;
#pragma unroll
          for (int w = 0; w < QW; ++w) v += red[(t - 1) & 1][w][tid];
          colsum[(t - 1) * 32 + tid] += v;
        }
      }
    }
    __syncthreads();
    // the last tile's sums (every earlier one was added inside the loop)
    const int tl = n_iter * RING - 1;
    if (tl < n_tiles && tid < 32) {
      float v = 0.f;
#pragma unroll
      for (int w = 0; w < QW; ++w) v += red[tl & 1][w][tid];
      colsum[tl * 32 + tid] += v;
    }
    __syncthreads();
  }
  const float inv_t = 1.f / (float)Tb;
  float* out = a.profile + ((size_t)b * a.H_q + h) * a.K_in;
  for (int t = tid; t < i_end - i_begin; t += NT) out[i_begin + t] = colsum[t] * inv_t;
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
  for (int i0 = tid; i0 < a.K_in; i0 += 8 * kSensThreads) {  // 16 loads in flight
    float x[8], y[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int i = min(i0 + k * kSensThreads, a.K_in - 1);
      x[k] = a.profile[0][base + i];
      y[k] = a.profile[1][base + i];
    }
#pragma unroll
    for (int k = 0; k < 8; ++k)
      if (i0 + k * kSensThreads < a.K_in) {
        d = fma((double)x[k], (double)y[k], d);
        n0 = fma((double)x[k], (double)x[k], n0);
        n1 = fma((double)y[k], (double)y[k], n1);
      }
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
constexpr int kRankThreads = 64 * kRankWaves;
constexpr int kRankChunk = 4096;                  // (s^v, s^t) pairs staged in LDS per step
constexpr int kRankPer = kRankChunk / kRankThreads;  // pairs each thread stages

__global__ __launch_bounds__(kRankThreads) void spearman_rank_kernel(SpearmanArgs a) {
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
    // every index load of the chunk first, then every value load
    int jj[kRankPer];
#pragma unroll
    for (int e = 0; e < kRankPer; ++e) {
      const int j = tid + e * kRankThreads;
      jj[e] = j < n ? min(max(idx[c0 + j], 0), a.N - 1) : 0;
    }
    float2 v[kRankPer];
#pragma unroll
    for (int e = 0; e < kRankPer; ++e) v[e] = make_float2(sv[jj[e]], st[jj[e]]);
#pragma unroll
    for (int e = 0; e < kRankPer; ++e) {
      const int j = tid + e * kRankThreads;
      if (j < n) vals[j] = v[e];
    }
    __syncthreads();
#pragma unroll 4
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

// One wave per sample: the workgroups' integer sums, then the ratio.
__global__ __launch_bounds__(64) void spearman_final_kernel(SpearmanArgs a) {
  const int b = blockIdx.x, lane = threadIdx.x;
  long long s_vt = 0, s_vv = 0, s_tt = 0;
  const long long* p = a.part + (size_t)b * a.n_tiles * 4;
  for (int t = lane; t < a.n_tiles; t += 64) {
    s_vt += p[4 * t];
    s_vv += p[4 * t + 1];
    s_tt += p[4 * t + 2];
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    s_vt += __shfl_xor(s_vt, o, 64);
    s_vv += __shfl_xor(s_vv, o, 64);
    s_tt += __shfl_xor(s_tt, o, 64);
  }
  if (lane == 0)
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
  const dim3 grid(a.B * a.H_q * a.n_split);
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
  hipLaunchKernelGGL(spearman_rank_kernel, dim3(a.n_tiles, B), dim3(kRankThreads), 0, s, a);
  hipLaunchKernelGGL(spearman_final_kernel, dim3(B), dim3(64), 0, s, a);
  return hipGetLastError();
}

}  // namespace trevs
