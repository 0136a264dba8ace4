// Workgroup-wide exact order statistics and stable top-K (one workgroup of
// 512 threads per sample; thread t owns the E consecutive elements
// [t*E, t*E + E), so a workgroup prefix sum walks the elements in index order).
#pragma once

#include "common.hpp"

namespace trevs {

constexpr int kSelThreads = 512;
constexpr int kSelWaves = kSelThreads / kWave;
constexpr int kRadixBits = 8;
constexpr int kRadixBins = 1 << kRadixBits;

struct SelectShared {
  uint32_t hist[2][kRadixBins];
  uint32_t mn[2][kSelWaves];
  uint32_t mx[2][kSelWaves];
  int wave_tot[kSelWaves];
  int wave_excl[kSelWaves];
  int total;
  uint32_t res_digit[2];
  uint32_t res_before[2];
  uint32_t res_count[2];
};

// Exclusive prefix sum of one int per thread over the workgroup.
__device__ __forceinline__ int block_excl_scan(int v, SelectShared& sh, int& total) {
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  const int inc = wave_incl_scan(v, lane);
  if (lane == kWave - 1) sh.wave_tot[wave] = inc;
  __syncthreads();
  if (wave == 0) {
    const int w = lane < kSelWaves ? sh.wave_tot[lane] : 0;
    const int wi = wave_incl_scan(w, lane);
    if (lane < kSelWaves) sh.wave_excl[lane] = wi - w;
    if (lane == kSelWaves - 1) sh.total = wi;
  }
  __syncthreads();
  total = sh.total;
  const int r = sh.wave_excl[wave] + inc - v;
  __syncthreads();
  return r;
}

// Histogram increment with wave aggregation of the first active lane's
// digit (many lanes share one digit when values cluster, e.g. exact zeros).
__device__ __forceinline__ void hist_add(uint32_t* hist, bool act, uint32_t digit, int lane) {
  const unsigned long long am = __ballot(act);
  if (am == 0ull) return;
  const int leader = __ffsll((long long)am) - 1;
  const uint32_t d0 = (uint32_t)__shfl((int)digit, leader, kWave);
  const unsigned long long same = __ballot(act && digit == d0);
  if (lane == leader) atomicAdd(&hist[d0], (uint32_t)__popcll(same));
  if (act && digit != d0) atomicAdd(&hist[digit], 1u);
}

// Exact rank selection on uint32 keys for NSET independent key sets at once.
// keyf(s, e) yields the key of this thread's element e in set s (recomputed
// on every pass rather than held in registers).  For set s returns the key of
// ascending 0-based rank rank[s] among the N valid keys, the number of keys
// strictly below it, and the number equal to it.  Radix passes of 8 bits
// start below the common prefix of the set's minimum and maximum key.
template <int NSET, int E, class KeyF>
__device__ void block_select(KeyF keyf, int base, int N, const int (&rank)[NSET],
                             uint32_t (&res)[NSET], int (&less)[NSET], int (&eq)[NSET],
                             SelectShared& sh) {
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  uint32_t mn[NSET], mx[NSET];
#pragma unroll
  for (int s = 0; s < NSET; ++s) {
    mn[s] = 0xffffffffu;
    mx[s] = 0u;
#pragma unroll
    for (int e = 0; e < E; ++e)
      if (base + e < N) {
        const uint32_t k = keyf(s, e);
        mn[s] = min(mn[s], k);
        mx[s] = max(mx[s], k);
      }
    mn[s] = wave_min_u32(mn[s]);
    mx[s] = wave_max_u32(mx[s]);
    if (lane == 0) {
      sh.mn[s][wave] = mn[s];
      sh.mx[s][wave] = mx[s];
    }
  }
  __syncthreads();
  int nb[NSET], krem[NSET];
  uint32_t prefix[NSET];
#pragma unroll
  for (int s = 0; s < NSET; ++s) {
    uint32_t a = 0xffffffffu, z = 0u;
    for (int w = 0; w < kSelWaves; ++w) {
      a = min(a, sh.mn[s][w]);
      z = max(z, sh.mx[s][w]);
    }
    const uint32_t diff = a ^ z;
    nb[s] = diff ? 32 - __clz(diff) : 0;
    prefix[s] = (uint32_t)(((uint64_t)a >> nb[s]) << nb[s]);
    krem[s] = rank[s];
    less[s] = 0;
    eq[s] = diff ? 0 : N;
  }
  __syncthreads();  // sh.mn / sh.mx are rewritten by the next call
  for (;;) {
    bool any = false;
#pragma unroll
    for (int s = 0; s < NSET; ++s) any |= nb[s] > 0;
    if (!any) break;
    for (int i = tid; i < NSET * kRadixBins; i += kSelThreads) sh.hist[i / kRadixBins][i % kRadixBins] = 0u;
    __syncthreads();
#pragma unroll
    for (int s = 0; s < NSET; ++s) {
      if (nb[s] == 0) continue;
      const int db = min(kRadixBits, nb[s]), shift = nb[s] - db;
      const uint32_t dmask = (1u << db) - 1u;
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const uint32_t k = keyf(s, e);
        const bool match = ((uint64_t)k >> nb[s]) == ((uint64_t)prefix[s] >> nb[s]);
        hist_add(sh.hist[s], base + e < N && match, (k >> shift) & dmask, lane);
      }
    }
    __syncthreads();
#pragma unroll
    for (int s = 0; s < NSET; ++s) {
      if (wave != s || nb[s] == 0) continue;
      uint32_t c[4];
      int lsum = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        c[j] = sh.hist[s][4 * lane + j];
        lsum += (int)c[j];
      }
      const int excl = wave_incl_scan(lsum, lane) - lsum;
      if (excl <= krem[s] && krem[s] < excl + lsum) {
        int run = excl;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          if (krem[s] < run + (int)c[j]) {
            sh.res_digit[s] = 4 * lane + j;
            sh.res_before[s] = run;
            sh.res_count[s] = c[j];
            break;
          }
          run += (int)c[j];
        }
      }
    }
    __syncthreads();
#pragma unroll
    for (int s = 0; s < NSET; ++s) {
      if (nb[s] == 0) continue;
      const int db = min(kRadixBits, nb[s]), shift = nb[s] - db;
      prefix[s] |= sh.res_digit[s] << shift;
      krem[s] -= (int)sh.res_before[s];
      less[s] += (int)sh.res_before[s];
      nb[s] = shift;
      if (shift == 0) eq[s] = (int)sh.res_count[s];
    }
  }
#pragma unroll
  for (int s = 0; s < NSET; ++s) res[s] = prefix[s];
}

// Stable top-K: keep every element whose score is above the K-th largest and
// the lowest-index elements equal to it, and write the kept indices in
// ascending order to out[0..K).
template <int E>
__device__ void block_topk_write(const float (&sc)[E], int base, int N, int K, int32_t* out,
                                 SelectShared& sh) {
  auto keyf = [&](int, int e) { return f2key(sc[e]); };
  const int rank[1] = {N - K};
  uint32_t res[1];
  int less[1], eq[1];
  block_select<1, E>(keyf, base, N, rank, res, less, eq, sh);
  const uint32_t thr = res[0];
  const int need_eq = K - (N - less[0] - eq[0]);
  int my_eq = 0;
#pragma unroll
  for (int e = 0; e < E; ++e) my_eq += (base + e < N && f2key(sc[e]) == thr) ? 1 : 0;
  int tot;
  int run = block_excl_scan(my_eq, sh, tot);
  bool keep[E];
  int my_keep = 0;
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const bool valid = base + e < N;
    const bool is_eq = valid && f2key(sc[e]) == thr;
    keep[e] = valid && (f2key(sc[e]) > thr || (is_eq && run < need_eq));
    run += is_eq ? 1 : 0;
    my_keep += keep[e] ? 1 : 0;
  }
  int pos = block_excl_scan(my_keep, sh, tot);
#pragma unroll
  for (int e = 0; e < E; ++e)
    if (keep[e] && pos < K) out[pos++] = base + e;  // exactly K are kept; the bound only guards memory
}

}  // namespace trevs
