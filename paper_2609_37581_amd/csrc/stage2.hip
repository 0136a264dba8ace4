// Stage 2 (in-LLM) kernels: text->vision attention statistics, head variance
// and high-variance head set, and the token score (Sec. 4.2, Eq. (8)-(9)).
#include <algorithm>
#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"

namespace trevs {

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Key tiles in flight per statistics workgroup: 8 vectors of 16 bytes per
// thread in registers (even, at least 2).
constexpr int stats_ring(int vectors_per_tile) { return vectors_per_tile >= 4 ? 2 : 8 / vectors_per_tile; }

// ---------------------------------------------------------------------------
// Statistics pass.  For every (query head h, text row q) the row of logits
// x_i = scale * Q[q,h] . K[i, h/G] over the visual keys is reduced online to
// (max, sum e, sum e^2) with e = exp(x - max), in log2 units.  Within a KV
// head the rows r = (h - g*G) * T_max + q of all G query heads share every
// key tile.  A workgroup of NW waves owns NW column blocks of 32 rows (each
// wave keeps its 32 Q rows resident as MFMA operand B) and one split of the
// visual keys; each 32-key tile is loaded once into LDS (two buffers
// alternate) and read by every wave as operand A, so a lane's 16 accumulators
// are 16 visual columns of its own text row and the softmax statistics stay
// in-lane.  Workgroups of one (sample, KV head) are numbered consecutively
// and mapped onto one XCD, so their keys and queries stay in that L2.
//
// For the causal softmax domain each workgroup also reduces, into separate
// (max, sum e), a share of every text row's non-visual causal keys: key index
// j < P is prefix row j, and j >= P is text row j - P (sequence row
// j + K_in), valid for text row q while j - P <= q.  Split s takes keys
// [s*rest_len, (s+1)*rest_len) after its visual keys, in the same tile
// stream, so the extra work is spread evenly over the grid.  Every row sees
// at least its own key, so the merged non-visual log-sum-exp is finite.
// ---------------------------------------------------------------------------
// (two-wave workgroups over rows of at most 256 bytes are held to four waves
// per SIMD: at 2048 of them, LLaVA-1.5 batch 64, all are resident at once,
// 45.5 -> 43.3 us; wider rows hold too many Q registers for four)
template <class In, int DH>
constexpr int stats_min_waves(int NW) { return NW == 2 && DH * In::kBytes <= 256 ? 4 : 1; }
template <class In, int DH, int NW, bool CAUSAL>
__global__ __launch_bounds__(64 * NW, (stats_min_waves<In, DH>(NW))) void t2v_stats_kernel(StatsArgs a) {
  constexpr int ROWB = DH * In::kBytes;
  constexpr int HALFB = ROWB / 2;
  constexpr int NF = HALFB / 64;
  constexpr int NT = 64 * NW;
  constexpr int LROW = ROWB + 16;
  constexpr int TV = 32 * ROWB / 16;           // 16-byte vectors of one key tile
  constexpr int TVT = (TV + NT - 1) / NT;
  __shared__ __attribute__((aligned(16))) uint8_t klds[2][32 * LROW];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, col = lane & 31;
  const int lin = xcd_remap(blockIdx.x, gridDim.x);
  const int split = lin % a.n_split;
  const int rg = (lin / a.n_split) % a.n_rgroups;
  const int bg = lin / (a.n_split * a.n_rgroups);
  const int g = bg % a.H_kv, b = bg / a.H_kv;
  const int R = a.G * a.T_max;
  const int r = (rg * NW + wave) * 32 + col;
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
      for (int j = 0; j < 4; ++j) qf[f][j] = ldg16(qp + f * 64 + j * 16);
  }
  // visual keys [i_begin, i_end) in nv tiles, then the non-visual causal keys
  // [j_begin, j_end) in nr tiles
  const int i_begin = split * a.split_len;
  const int i_end = min(a.K_in, i_begin + a.split_len);
  const int nv = (i_end - i_begin + 31) / 32;
  const int j_begin = CAUSAL ? min(split * a.rest_len, a.P + a.T_max) : 0;
  const int j_end = CAUSAL ? min(a.P + a.T_max, j_begin + a.rest_len) : 0;
  const int n_tiles = nv + (j_end - j_begin + 31) / 32;
  const int climit = a.P + q;  // last non-visual key index this lane's row attends
  const uint8_t* kbase = reinterpret_cast<const uint8_t*>(a.k) +
                         (size_t)b * a.S * a.H_kv * ROWB + (size_t)g * ROWB;
  const size_t kstride = (size_t)a.H_kv * ROWB;
  // tile t into registers: rows past a range (and tiles past the last) re-read
  // a valid row of the range (cached)
  auto load_tile = [&](int t, u32x4 (&dst)[TVT]) {
    const bool vis = !CAUSAL || t < nv || t >= n_tiles;  // uniform
    const int kb = t < nv ? i_begin + 32 * t : (t < n_tiles ? j_begin + 32 * (t - nv) : i_begin);
#pragma unroll
    for (int k = 0; k < TVT; ++k) {
      const int v = min(tid + k * NT, TV - 1), row = v / (ROWB / 16), c = v - row * (ROWB / 16);
      const int i = kb + row;
      int srow;
      if (vis) {
        srow = a.P + (i < i_end ? i : i_begin);
      } else {
        const int j = i < j_end ? i : j_begin;
        srow = j < a.P ? j : j + a.K_in;
      }
      dst[k] = ldg16(kbase + (size_t)srow * kstride + c * 16);
    }
  };
  auto store_tile = [&](int buf, const u32x4 (&src)[TVT]) {
#pragma unroll
    for (int k = 0; k < TVT; ++k) {
      const int v = tid + k * NT;
      if (v < TV) {
        const int row = v / (ROWB / 16), c = v - row * (ROWB / 16);
        *reinterpret_cast<u32x4*>(&klds[buf][row * LROW + c * 16]) = src[k];
      }
    }
  };

  // Online (max, sum e, sum e^2) in log2 units.  The logit scale is positive,
  // so the tile maximum is taken on the raw dot products and scaled once, and
  // each term is exp2(fma(dot, scale, -max)): about four vector operations
  // and one exp per logit.  Only a split's last visual tile can hold keys
  // past its end; it alone takes the masked path (so do the non-visual tiles,
  // whose causal limit differs per row).
  float m = -INFINITY, l = 0.f, l2 = 0.f;     // visual keys
  float mr = -INFINITY, lr = 0.f, l2r = 0.f;  // non-visual causal keys
  auto process = [&](int buf, int kb, int kend, int lim, auto full, float& m_, float& l_, float& l2_) {
    f32x16 acc;
#pragma unroll
    for (int rr = 0; rr < 16; ++rr) acc[rr] = 0.f;
    const uint8_t* p = &klds[buf][col * LROW + half * HALFB];
#pragma unroll
    for (int f = 0; f < NF; ++f) {
      u32x4 kf[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) kf[j] = *reinterpret_cast<const u32x4*>(p + f * 64 + j * 16);
      acc = mfma_frag(kf, qf[f], acc, In{});
    }
    if constexpr (!decltype(full)::value) {
#pragma unroll
      for (int rr = 0; rr < 16; ++rr) {
        const int i = kb + mfma_row(rr, half);
        if (i >= kend || i > lim) acc[rr] = -INFINITY;
      }
    }
    float mx = acc[0];
#pragma unroll
    for (int rr = 1; rr < 16; ++rr) mx = fmaxf(mx, acc[rr]);
    const float mn = fmaxf(m_, mx * a.scale_log2e);
    if (decltype(full)::value || mn > -INFINITY) {
      const float c = fast_exp2(m_ - mn);
      float s1 = 0.f, s2 = 0.f;
#pragma unroll
      for (int rr = 0; rr < 16; ++rr) {
        const float e = fast_exp2(fmaf(acc[rr], a.scale_log2e, -mn));
        s1 += e;
        s2 = fmaf(e, e, s2);
      }
      l_ = fmaf(l_, c, s1);
      l2_ = fmaf(l2_, c * c, s2);
      m_ = mn;
    }
  };
  // key tiles stream through a ring of RING register buffers (that many
  // tiles in flight from memory) into two alternating LDS buffers; the tiles
  // past the last are loaded (a valid row again) but never reduced
  constexpr int RING = stats_ring(TVT);
  const int n_iter = (n_tiles + RING - 1) / RING;
  u32x4 ring[RING][TVT];
#pragma unroll
  for (int c = 0; c < RING; ++c) load_tile(c, ring[c]);
  for (int it = 0; it < n_iter; ++it) {
#pragma unroll
    for (int c = 0; c < RING; ++c) {
      const int t = it * RING + c;
      // LDS buffer (t % 2) was last read at tile t - 2, before every wave
      // passed the barrier of tile t - 1
      store_tile(c % 2, ring[c]);
      load_tile(t + RING, ring[c]);
      __syncthreads();
      if (t < nv) {
        const int ib = i_begin + 32 * t;
        if (ib + 32 <= i_end)
          process(c % 2, ib, i_end, INT_MAX, std::true_type{}, m, l, l2);
        else
          process(c % 2, ib, i_end, INT_MAX, std::false_type{}, m, l, l2);
      } else if (CAUSAL && t < n_tiles) {
        process(c % 2, j_begin + 32 * (t - nv), j_end, climit, std::false_type{}, mr, lr, l2r);
      }
    }
  }
  // merge the two half-waves' (max, sum e, sum e^2)
  auto merge_halves = [&](float m_, float l_, float l2_) {
    const float mo = __shfl_xor(m_, 32, 64), lo = __shfl_xor(l_, 32, 64), l2o = __shfl_xor(l2_, 32, 64);
    const float M = fmaxf(m_, mo);
    float L = 0.f, L2 = 0.f;
    if (M > -INFINITY) {
      const float c1 = fast_exp2(m_ - M), c2 = fast_exp2(mo - M);
      L = l_ * c1 + lo * c2;
      L2 = l2_ * c1 * c1 + l2o * c2 * c2;
    }
    return make_float4(M, L, L2, 0.f);
  };
  const size_t slot = (((size_t)b * a.H_q + h) * a.T_max + q) * a.n_split + split;
  const float4 vs = merge_halves(m, l, l2);
  if (half == 0 && rvalid) a.part[slot] = vs;
  if constexpr (CAUSAL) {
    const float4 rs = merge_halves(mr, lr, l2r);
    if (half == 0 && rvalid) a.part_rest[slot] = rs;
  }
}

// ---------------------------------------------------------------------------
// Head pass, one workgroup per (head, sample).  Merges the split statistics
// of every text row into its log-sum-exp (optionally joined with the row's
// non-visual log-sum-exp, given by the caller or merged from the causal rest
// statistics) and the population variance of the row's visual attention,
// then averages over the valid text rows: u_h of Eq. (8).
// ---------------------------------------------------------------------------
constexpr int kHeadThreads = 128;

__global__ __launch_bounds__(kHeadThreads) void t2v_heads_kernel(HeadArgs a) {
  __shared__ float red[kHeadThreads / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int h = blockIdx.x, b = blockIdx.y;
  const int Tb = text_rows(a.text_len, b, a.T_max);
  const float invK = 1.f / (float)a.K_in;
  float vs = 0.f;
  for (int q = tid; q < a.T_max; q += kHeadThreads) {
    const size_t row = ((size_t)b * a.H_q + h) * a.T_max + q;
    const float4* pp = a.part + row * a.n_split;
    const size_t lrow = ((size_t)b * a.H_q + h) * a.T_pad + q;
    // the splits' partials 8 at a time, every load issued before the merge
    float m = -INFINITY, l = 0.f, l2 = 0.f;
    for (int s0 = 0; s0 < a.n_split; s0 += 8) {
      float4 pv[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) pv[k] = pp[min(s0 + k, a.n_split - 1)];
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const float4 p = pv[k];
        const float mn = fmaxf(m, p.x);
        if (s0 + k < a.n_split && mn > -INFINITY) {
          const float c1 = fast_exp2(m - mn), c2 = fast_exp2(p.x - mn);
          l = l * c1 + p.y * c2;
          l2 = l2 * c1 * c1 + p.z * c2 * c2;
          m = mn;
        }
      }
    }
    float lse2 = m + log2f(l);
    if (a.lse_rest || a.part_rest) {
      float r2;
      if (a.part_rest) {
        const float4* pr = a.part_rest + row * a.n_split;
        float mr = -INFINITY, lr = 0.f;
        for (int s0 = 0; s0 < a.n_split; s0 += 8) {
          float4 pv[8];
#pragma unroll
          for (int k = 0; k < 8; ++k) pv[k] = pr[min(s0 + k, a.n_split - 1)];
#pragma unroll
          for (int k = 0; k < 8; ++k) {
            const float4 p = pv[k];
            const float mn = fmaxf(mr, p.x);
            if (s0 + k < a.n_split && mn > -INFINITY) {
              lr = lr * fast_exp2(mr - mn) + p.y * fast_exp2(p.x - mn);
              mr = mn;
            }
          }
        }
        r2 = mr + log2f(lr);
      } else {
        r2 = a.lse_rest[row] * kLog2e;
      }
      const float mx = fmaxf(lse2, r2);
      lse2 = mx + log2f(fast_exp2(lse2 - mx) + fast_exp2(r2 - mx));
    }
    a.lse2[lrow] = lse2;
    if (q < Tb) {
      const float f = fast_exp2(m - lse2);
      vs += f * f * (l2 - l * l * invK) * invK;
    }
  }
  vs = wave_sum(vs);
  if (lane == 0) red[wave] = vs;
  __syncthreads();
  if (tid == 0) {
    float t = 0.f;
    for (int w = 0; w < kHeadThreads / 64; ++w) t += red[w];
    a.head_var[(size_t)b * a.H_q + h] = t / (float)Tb;
  }
}

// ---------------------------------------------------------------------------
// Head pass from given row statistics, one workgroup per (head, sample): each
// text row's log-sum-exp is taken from the caller (the layer's own attention
// pass), converted to log2 units, and u_h of Eq. (8) is the mean over the
// valid rows of S2/K - (S1/K)^2, with S1 and S2 the row's sum and sum of
// squares of its attention over the visual columns.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kHeadThreads) void heads_given_kernel(const float* row_stats, HeadArgs a) {
  __shared__ float red[kHeadThreads / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int h = blockIdx.x, b = blockIdx.y;
  const int Tb = text_rows(a.text_len, b, a.T_max);
  const float invK = 1.f / (float)a.K_in;
  float vs = 0.f;
  for (int q = tid; q < a.T_max; q += kHeadThreads) {
    const size_t row = ((size_t)b * a.H_q + h) * a.T_max + q;
    const float lse = row_stats[3 * row], s1 = row_stats[3 * row + 1], s2 = row_stats[3 * row + 2];
    a.lse2[((size_t)b * a.H_q + h) * a.T_pad + q] = lse * kLog2e;
    if (q < Tb) {
      const float mean = s1 * invK;
      vs += s2 * invK - mean * mean;
    }
  }
  vs = wave_sum(vs);
  if (lane == 0) red[wave] = vs;
  __syncthreads();
  if (tid == 0) {
    float t = 0.f;
    for (int w = 0; w < kHeadThreads / 64; ++w) t += red[w];
    a.head_var[(size_t)b * a.H_q + h] = t / (float)Tb;
  }
}

// ---------------------------------------------------------------------------
// Token score.  A workgroup owns V = 32*VB visual tokens of one sample (tiles
// of one sample are numbered consecutively and mapped onto one XCD, so the
// sample's queries and keys stay in that L2).  It first ranks the heads of
// its sample by (u desc, h asc) and keeps the first n_keep: the
// high-variance set H*, ascending (the sample's first tile also stores it).
// Wave w owns the 32 text rows of block pass*QW + (w % QW) and the keys of
// 32-token block w / QW (or all V keys with one wave per text block).  For each
// selected head the pass's Q rows (QW*32 of them) and their row log-sum-exps
// are staged in LDS with coalesced 16-byte loads (a 32-row MFMA operand read
// straight from memory would touch 32 rows per instruction), one head ahead.
// H* is ascending, so its heads of one KV group are consecutive: the key tile
// of a group is staged in LDS once and serves every selected head of the
// group (the next group's tile waits in registers).  The logits are
// recomputed on the matrix cores (operand A = text rows, operand B = key
// rows), turned into attention and summed over heads in-lane.  Then max over
// the valid text rows, across waves via LDS, and divide by |H*| (Eq. (9)).
// With a head split (small grids) workgroup (tile, split) sums only its hps
// selected heads and writes the sums per (valid text row, token);
// t2v_score_merge_kernel finishes Eq. (9).
// ---------------------------------------------------------------------------
constexpr int kMaxHeads = 256;

// Waves per 32-row text block: with 64-token tiles two waves split the keys
// (32 each) and share the staged Q rows, two waves per SIMD (23 us against
// 26 us with one wave per text block at the 16,384-token workload).
#ifndef TREVS_SCORE_WPB
#define TREVS_SCORE_WPB 2
#endif
template <int ROWB>
struct ScoreTile {
  static constexpr int VB = ROWB <= 256 ? 2 : 1;  // 32-token blocks per workgroup
  static constexpr int V = 32 * VB;
  static constexpr int WPB = VB == 2 ? TREVS_SCORE_WPB : 1;  // waves per 32-row text block
};

template <class In, int DH, int QW>
__global__ __launch_bounds__(64 * QW * ScoreTile<DH * In::kBytes>::WPB) void t2v_score_kernel(ScoreArgs a) {
  constexpr int ROWB = DH * In::kBytes;
  constexpr int HALFB = ROWB / 2;
  constexpr int NF = HALFB / 64;
  constexpr int WPB = ScoreTile<ROWB>::WPB;
  constexpr int VB = ScoreTile<ROWB>::VB / WPB;  // 32-token blocks per wave
  constexpr int V = ScoreTile<ROWB>::V;
  constexpr int NT = 64 * QW * WPB;
  constexpr int LROW = ROWB + 16;
  constexpr int CPR = ROWB / 16;
  constexpr int QR = 32 * QW;                  // text rows of a pass
  constexpr int KVT = V * CPR / NT;            // 16-byte vectors per thread: key tile
  constexpr int QVT = QR * CPR / NT;           // ... and Q rows
  static_assert(KVT * NT == V * CPR && QVT * NT == QR * CPR, "stage split");
  __shared__ __attribute__((aligned(16))) uint8_t klds[2][V * LROW];
  __shared__ __attribute__((aligned(16))) uint8_t qlds[2][QR * LROW];
  __shared__ __attribute__((aligned(16))) float llds[2][QR];
  __shared__ float pmax[QW][V];
  __shared__ float u_lds[kMaxHeads];
  __shared__ int sel_lds[kMaxHeads];
  __shared__ int heads[kMaxHeads];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int wave = wv % QW, vw = wv / QW;  // text block of the pass, key blocks vw*VB..
  const int half = lane >> 5, col = lane & 31;
  // the head splits of one tile are consecutive workgroups (one XCD)
  const int lin0 = xcd_remap(blockIdx.x, gridDim.x);
  const int lin = lin0 / a.n_hsplit, hs = lin0 - lin * a.n_hsplit;
  const int b = lin / a.n_vtiles, i0 = (lin - b * a.n_vtiles) * V;
  const int Hq = a.H_q, nk = a.n_keep;
  const int h_lo = hs * a.hps, h_hi = min(nk, h_lo + a.hps);  // selected-head indices of this split

  // ---- high-variance head set H*: the rank of head h under (u desc, h asc)
  // counts the heads before it, 64 comparisons per ballot (wave w ranks heads
  // w, w + QW, ...); wave 0 then writes the selected heads in ascending order
  for (int h = tid; h < Hq; h += NT) {
    u_lds[h] = a.head_var[(size_t)b * Hq + h];
    heads[h] = 0;
  }
  __syncthreads();
  for (int h = wv; h < Hq; h += QW * WPB) {
    const float u = u_lds[h];
    int rank = 0;
    for (int c0 = 0; c0 < Hq; c0 += 64) {
      const int h2 = c0 + lane;
      const float u2 = h2 < Hq ? u_lds[h2] : 0.f;
      rank += (int)__popcll(__ballot(h2 < Hq && (u2 > u || (u2 == u && h2 < h))));
    }
    if (lane == 0) sel_lds[h] = rank < nk;
  }
  __syncthreads();
  if (wv == 0) {
    int base = 0;
    for (int c0 = 0; c0 < Hq; c0 += 64) {
      const int h = c0 + lane;
      const bool sel = h < Hq && sel_lds[h];
      const unsigned long long bal = __ballot(sel);
      const int pos = base + (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(bal >> 32),
                                                            __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0u));
      if (sel && pos < nk) {  // ranks are distinct for finite u
        heads[pos] = h;
        if (i0 == 0 && hs == 0 && a.head_sel) a.head_sel[(size_t)b * nk + pos] = h;
      }
      base += (int)__popcll(bal);
    }
  }
  __syncthreads();
  auto head_at = [&](int hi) { return min(max(heads[min(hi, nk - 1)], 0), Hq - 1); };

  const int Tb = text_rows(a.text_len, b, a.T_max);
  const size_t seq0 = (size_t)b * a.S;
  const uint8_t* kbase = reinterpret_cast<const uint8_t*>(a.k) + (seq0 + a.P) * a.H_kv * ROWB;
  const size_t kstride = (size_t)a.H_kv * ROWB;
  const uint8_t* qtext = reinterpret_cast<const uint8_t*>(a.q) + (seq0 + a.P + a.K_in) * a.H_q * ROWB;
  const size_t qstride = (size_t)a.H_q * ROWB;
  // first head index after hi that belongs to another KV group
  auto next_group = [&](int hi) {
    const int g = head_at(hi) / a.G;
    int j = hi + 1;
    while (j < nk && head_at(j) / a.G == g) ++j;
    return j;
  };
  // key rows i0..i0+V-1 of KV group g (rows past K_in re-read the last row)
  auto load_tile = [&](int g, u32x4 (&dst)[KVT]) {
#pragma unroll
    for (int k = 0; k < KVT; ++k) {
      const int v = tid + k * NT, row = v / CPR, c = v - row * CPR;
      const int i = min(i0 + row, a.K_in - 1);
      dst[k] = ldg16(kbase + (size_t)i * kstride + (size_t)g * ROWB + c * 16);
    }
  };
  auto store_tile = [&](int buf, const u32x4 (&src)[KVT]) {
#pragma unroll
    for (int k = 0; k < KVT; ++k) {
      const int v = tid + k * NT, row = v / CPR, c = v - row * CPR;
      *reinterpret_cast<u32x4*>(&klds[buf][row * LROW + c * 16]) = src[k];
    }
  };

  float pm[VB];
#pragma unroll
  for (int vb = 0; vb < VB; ++vb) pm[vb] = 0.f;
  const int n_qblk = (Tb + 31) / 32;
  const int n_pass = (n_qblk + QW - 1) / QW;  // uniform over the workgroup (barriers below)
  for (int pass = 0; pass < n_pass; ++pass) {
    const int r0 = pass * QR;
    // text rows r0..r0+QR-1 of head index hi (rows past T_max re-read the
    // last row) and their log-sum-exps (float4s, every thread one; duplicates
    // store the same values; the row is padded to a multiple of 32)
    auto load_q = [&](int hi, u32x4 (&dst)[QVT], float4& ldst) {
      const int h = head_at(hi);
#pragma unroll
      for (int k = 0; k < QVT; ++k) {
        const int v = tid + k * NT, row = v / CPR, c = v - row * CPR;
        const int t = min(r0 + row, a.T_max - 1);
        dst[k] = ldg16(qtext + (size_t)t * qstride + (size_t)h * ROWB + c * 16);
      }
      ldst = *reinterpret_cast<const float4*>(a.lse2 + ((size_t)b * a.H_q + h) * a.T_pad +
                                              min(r0 + 4 * (tid % (QR / 4)), a.T_pad - 4));
    };
    auto store_q = [&](int buf, const u32x4 (&src)[QVT], float4 l) {
#pragma unroll
      for (int k = 0; k < QVT; ++k) {
        const int v = tid + k * NT, row = v / CPR, c = v - row * CPR;
        *reinterpret_cast<u32x4*>(&qlds[buf][row * LROW + c * 16]) = src[k];
      }
      *reinterpret_cast<float4*>(&llds[buf][4 * (tid % (QR / 4))]) = l;
    };
    float accs[VB][16];
#pragma unroll
    for (int vb = 0; vb < VB; ++vb)
#pragma unroll
      for (int rr = 0; rr < 16; ++rr) accs[vb][rr] = 0.f;
    auto process = [&](int qbuf, int kbuf) {
      const uint8_t* qp = &qlds[qbuf][(wave * 32 + col) * LROW + half * HALFB];
      u32x4 qf[NF][4];
#pragma unroll
      for (int f = 0; f < NF; ++f)
#pragma unroll
        for (int j = 0; j < 4; ++j) qf[f][j] = *reinterpret_cast<const u32x4*>(qp + f * 64 + j * 16);
      float4 lse[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) lse[j] = *reinterpret_cast<const float4*>(&llds[qbuf][wave * 32 + 8 * j + 4 * half]);
#pragma unroll
      for (int vb = 0; vb < VB; ++vb) {
        const uint8_t* p = &klds[kbuf][((vw * VB + vb) * 32 + col) * LROW + half * HALFB];
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
          accs[vb][4 * j + 0] += fast_exp2(fmaf(acc[4 * j + 0], a.scale_log2e, -lse[j].x));
          accs[vb][4 * j + 1] += fast_exp2(fmaf(acc[4 * j + 1], a.scale_log2e, -lse[j].y));
          accs[vb][4 * j + 2] += fast_exp2(fmaf(acc[4 * j + 2], a.scale_log2e, -lse[j].z));
          accs[vb][4 * j + 3] += fast_exp2(fmaf(acc[4 * j + 3], a.scale_log2e, -lse[j].w));
        }
      }
    };
    // group runs of H*: the first run's key tile goes to buffer 0, the next
    // run's tile waits in registers until its run starts
    u32x4 kst[KVT];
    load_tile(head_at(h_lo) / a.G, kst);
    store_tile(0, kst);
    int he = next_group(h_lo);
    if (he < h_hi) load_tile(head_at(he) / a.G, kst);
    int kbuf = 0;
    u32x4 qr[QVT];
    float4 lr;
    load_q(h_lo, qr, lr);
    for (int hi = h_lo; hi < h_hi; hi += 2) {
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        const int h = hi + c;
        if (h < h_hi) {  // uniform over the workgroup
          // Q buffer c was last read at head h - 2, before every wave passed
          // the barrier of head h - 1; a new group's key buffer was last
          // read two groups back, before the barrier of this group's start
          if (h > h_lo && h == he) {
            kbuf ^= 1;
            store_tile(kbuf, kst);
            he = next_group(h);
            if (he < h_hi) load_tile(head_at(he) / a.G, kst);
          }
          store_q(c, qr, lr);
          __syncthreads();
          load_q(h + 1, qr, lr);
          process(c, kbuf);
        }
      }
    }
    if (a.n_hsplit > 1) {  // this split's head sums of the valid rows; 32 lanes write 128 bytes
      float* hp = a.hpart + ((size_t)b * a.n_hsplit + hs) * a.T_max * a.K_in;
#pragma unroll
      for (int vb = 0; vb < VB; ++vb) {
        const int i = i0 + (vw * VB + vb) * 32 + col;
#pragma unroll
        for (int rr = 0; rr < 16; ++rr) {
          const int q = r0 + wave * 32 + mfma_row(rr, half);
          if (q < Tb && i < a.K_in) hp[(size_t)q * a.K_in + i] = accs[vb][rr];
        }
      }
    } else {
#pragma unroll
      for (int vb = 0; vb < VB; ++vb)
#pragma unroll
        for (int rr = 0; rr < 16; ++rr)
          if (r0 + wave * 32 + mfma_row(rr, half) < Tb) pm[vb] = fmaxf(pm[vb], accs[vb][rr]);
    }
    __syncthreads();  // the next pass restages every buffer
  }
  if (a.n_hsplit > 1) return;
  // operand A = text rows: a lane holds text rows of visual column
  // ((vw * VB + vb) * 32 + col)
#pragma unroll
  for (int vb = 0; vb < VB; ++vb) {
    const float v = fmaxf(pm[vb], __shfl_xor(pm[vb], 32, 64));
    if (half == 0) pmax[wave][(vw * VB + vb) * 32 + col] = v;
  }
  __syncthreads();
  for (int t = tid; t < V; t += NT) {
    if (i0 + t < a.K_in) {
      float v = pmax[0][t];
#pragma unroll
      for (int w = 1; w < QW; ++w) v = fmaxf(v, pmax[w][t]);
      a.p[(size_t)b * a.K_in + i0 + t] = v / (float)a.n_keep;
    }
  }
}

// ---------------------------------------------------------------------------
// Token-score merge after a head split: a workgroup owns 32 visual tokens of
// one sample, thread (g, t) the text rows g, g + 8, ... of token t.  It adds
// the splits' head sums of each row in split order and keeps the maximum
// over the valid text rows; the row groups meet in LDS and the result is
// divided by |H*| (Eq. (9)).
// ---------------------------------------------------------------------------
constexpr int kScoreMergeTokens = 32, kScoreMergeGroups = 8;

__global__ __launch_bounds__(kScoreMergeTokens * kScoreMergeGroups) void t2v_score_merge_kernel(ScoreArgs a) {
  __shared__ float red[kScoreMergeGroups][kScoreMergeTokens + 1];
  const int t = threadIdx.x % kScoreMergeTokens, g = threadIdx.x / kScoreMergeTokens;
  const int b = blockIdx.y, i = blockIdx.x * kScoreMergeTokens + t, ic = min(i, a.K_in - 1);
  const int S = a.n_hsplit, Tb = text_rows(a.text_len, b, a.T_max);
  // uniform split base plus a 32-bit lane offset
  const size_t sstride = (size_t)a.T_max * a.K_in;
  const float* pb = a.hpart + (size_t)b * S * sstride;
  float best = 0.f;  // attention sums are nonnegative
  for (int q = g; q < Tb; q += kScoreMergeGroups) {
    const int off = q * a.K_in + ic;
    float c = 0.f;
    for (int s0 = 0; s0 < S; s0 += 8) {  // 8 loads in flight, added in split order
      float v[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) v[k] = pb[min(s0 + k, S - 1) * sstride + off];
#pragma unroll
      for (int k = 0; k < 8; ++k) c += s0 + k < S ? v[k] : 0.f;
    }
    best = fmaxf(best, c);
  }
  red[g][t] = best;
  __syncthreads();
  if (g == 0 && i < a.K_in) {
    float v = red[0][t];
#pragma unroll
    for (int x = 1; x < kScoreMergeGroups; ++x) v = fmaxf(v, red[x][t]);
    a.p[(size_t)b * a.K_in + i] = v / (float)a.n_keep;
  }
}

// ---------------------------------------------------------------- launchers
// Selected heads are split over workgroups while the tiles leave compute
// units idle: up to one split per selected head, about one workgroup per CU.
int score_head_splits(int B, int n_vtiles, int n_keep) {
  const long tiles = (long)B * n_vtiles;
  return (int)std::max<long>(1, std::min<long>(n_keep, 256 / tiles));
}

int stats_waves(int G, int T_max) {
  const int nrb = (G * T_max + 31) / 32;
  return nrb >= 8 ? 8 : (nrb >= 4 ? 4 : (nrb >= 2 ? 2 : 1));
}

template <class In, int DH, bool CAUSAL>
static void launch_stats_c(const StatsArgs& a, hipStream_t s) {
  const dim3 grid(a.n_split * a.n_rgroups * a.H_kv * a.B);
  switch (stats_waves(a.G, a.T_max)) {
    case 8: hipLaunchKernelGGL((t2v_stats_kernel<In, DH, 8, CAUSAL>), grid, dim3(512), 0, s, a); break;
    case 4: hipLaunchKernelGGL((t2v_stats_kernel<In, DH, 4, CAUSAL>), grid, dim3(256), 0, s, a); break;
    case 2: hipLaunchKernelGGL((t2v_stats_kernel<In, DH, 2, CAUSAL>), grid, dim3(128), 0, s, a); break;
    default: hipLaunchKernelGGL((t2v_stats_kernel<In, DH, 1, CAUSAL>), grid, dim3(64), 0, s, a); break;
  }
}

template <class In, int DH>
static void launch_stats_t(const StatsArgs& a, hipStream_t s) {
  if (a.rest_len > 0)
    launch_stats_c<In, DH, true>(a, s);
  else
    launch_stats_c<In, DH, false>(a, s);
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
  hipLaunchKernelGGL(t2v_heads_kernel, dim3(a.H_q, a.B), dim3(kHeadThreads), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_heads_given(const float* row_stats, const HeadArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(heads_given_kernel, dim3(a.H_q, a.B), dim3(kHeadThreads), 0, s, row_stats, a);
  return hipGetLastError();
}

// 32-row text blocks per pass of the token-score workgroup (its waves); the
// Q rows of a pass are double-buffered in LDS, so long rows take fewer.
int score_qblocks(int T_max, int row_bytes) {
  const int qb = (T_max + 31) / 32;
  const int cap = row_bytes <= 256 ? 4 : (row_bytes <= 512 ? 2 : 1);
  return std::min(cap, qb >= 4 ? 4 : (qb >= 2 ? 2 : 1));
}

int score_tile_tokens(int dtype, int dh) {
  const int rowb = dh * (dtype == 1 ? 2 : 4);
  return rowb <= 256 ? 64 : 32;
}

template <class In, int DH>
static void launch_score_t(const ScoreArgs& a, hipStream_t s) {
  const dim3 grid(a.B * a.n_vtiles * a.n_hsplit);
  constexpr int ROWB = DH * In::kBytes;
  const int qw = score_qblocks(a.T_max, ROWB);
  if constexpr (ROWB <= 256) {
    if (qw == 4) {
      hipLaunchKernelGGL((t2v_score_kernel<In, DH, 4>), grid, dim3(256 * ScoreTile<ROWB>::WPB), 0, s, a);
      return;
    }
  }
  if constexpr (ROWB <= 512) {
    if (qw == 2) {
      hipLaunchKernelGGL((t2v_score_kernel<In, DH, 2>), grid, dim3(128 * ScoreTile<ROWB>::WPB), 0, s, a);
      return;
    }
  }
  hipLaunchKernelGGL((t2v_score_kernel<In, DH, 1>), grid, dim3(64 * ScoreTile<ROWB>::WPB), 0, s, a);
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
  if (a.n_hsplit > 1) {
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const dim3 grid((a.K_in + kScoreMergeTokens - 1) / kScoreMergeTokens, a.B);
    hipLaunchKernelGGL(t2v_score_merge_kernel, grid, dim3(kScoreMergeTokens * kScoreMergeGroups), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace trevs
