// Workgroup-wide exact order statistics and stable top-K.  One workgroup of
// 1024 threads ranks one vector; thread t owns the E consecutive elements
// [t*E, t*E + E), so a workgroup prefix sum walks the elements in index order.
#pragma once

#include "common.hpp"

namespace trevs {

constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / kWave;
constexpr int kFirstBits = 11;                // digit width of the first radix pass
constexpr int kFirstBins = 1 << kFirstBits;
constexpr int kLaterBits = 8;                 // digit width of the candidate passes
constexpr int kCandCap = 4096;                // candidates kept in LDS after the first pass

struct SelectShared {
  uint32_t hist[kFirstBins];
  uint32_t cand[kCandCap];
  uint32_t mn[kSelWaves];
  uint32_t mx[kSelWaves];
  int wave_tot[kSelWaves];
  int wave_excl[kSelWaves];
  int total;
  uint32_t res_digit, res_before, res_count;
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

// Histogram increment.  The lanes that share the first active lane's digit
// are counted with one atomic (values cluster, e.g. exact zeros, which would
// otherwise serialise on one LDS address); the others add one each.  Must be
// called by every lane of the wave.
__device__ __forceinline__ void hist_add(uint32_t* hist, bool act, uint32_t digit) {
  const unsigned long long am = __ballot(act);
  if (am == 0ull) return;
  const int leader = __ffsll((long long)am) - 1;
  const uint32_t d0 = (uint32_t)__builtin_amdgcn_readlane((int)digit, leader);
  const unsigned long long same = __ballot(act && digit == d0);
  if ((int)(threadIdx.x & (kWave - 1)) == leader) atomicAdd(&hist[d0], (uint32_t)__popcll(same));
  if (act && digit != d0) atomicAdd(&hist[digit], 1u);
}

// Finds the bin holding rank krem in hist[0, nbins): every thread owns two
// bins, a workgroup scan orders them.  Result in sh.res_*.
__device__ __forceinline__ void block_find_bin(int nbins, int krem, SelectShared& sh) {
  const int t = threadIdx.x;
  const int c0 = 2 * t < nbins ? (int)sh.hist[2 * t] : 0;
  const int c1 = 2 * t + 1 < nbins ? (int)sh.hist[2 * t + 1] : 0;
  int tot;
  const int excl = block_excl_scan(c0 + c1, sh, tot);
  if (excl <= krem && krem < excl + c0 + c1) {
    const bool first = krem < excl + c0;
    sh.res_digit = 2 * t + (first ? 0 : 1);
    sh.res_before = first ? excl : excl + c0;
    sh.res_count = first ? c0 : c1;
  }
  __syncthreads();
}

// Finds the bin holding rank krem in hist[0, 256) with wave 0 alone.
__device__ __forceinline__ void wave0_find_bin(int krem, SelectShared& sh) {
  const int lane = threadIdx.x & (kWave - 1);
  if (threadIdx.x < kWave) {
    uint32_t c[4];
    int lsum = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      c[j] = sh.hist[4 * lane + j];
      lsum += (int)c[j];
    }
    const int excl = wave_incl_scan(lsum, lane) - lsum;
    if (excl <= krem && krem < excl + lsum) {
      int run = excl;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if (krem < run + (int)c[j]) {
          sh.res_digit = 4 * lane + j;
          sh.res_before = run;
          sh.res_count = c[j];
          break;
        }
        run += (int)c[j];
      }
    }
  }
  __syncthreads();
}

// Exact rank selection on uint32 keys.  keyf(e) yields the key of this
// thread's element e (recomputed on demand, not held).  Returns the key of
// ascending 0-based rank `rank` among the N valid keys, with the number of
// keys strictly below it (less) and equal to it (eq).
//   1. min and max; the bits above their highest differing bit are common.
//   2. one pass over all elements on the next (up to) 11 bits;
//   3. the elements in the chosen bin are compacted into LDS (if they fit)
//      and the remaining bits are resolved 8 at a time over them alone;
//      otherwise the remaining passes scan all elements.
template <int E, class KeyF>
__device__ void block_select(KeyF keyf, int base, int N, int rank, uint32_t& res, int& less,
                             int& eq, SelectShared& sh) {
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  uint32_t mn = 0xffffffffu, mx = 0u;
#pragma unroll
  for (int e = 0; e < E; ++e)
    if (base + e < N) {
      const uint32_t k = keyf(e);
      mn = min(mn, k);
      mx = max(mx, k);
    }
  mn = wave_min_u32(mn);
  mx = wave_max_u32(mx);
  if (lane == 0) {
    sh.mn[wave] = mn;
    sh.mx[wave] = mx;
  }
  __syncthreads();
  uint32_t a = 0xffffffffu, z = 0u;
#pragma unroll
  for (int w = 0; w < kSelWaves; ++w) {
    a = min(a, sh.mn[w]);
    z = max(z, sh.mx[w]);
  }
  __syncthreads();  // sh.mn / sh.mx are rewritten by the next call
  const uint32_t diff = a ^ z;
  less = 0;
  if (diff == 0u) {
    res = a;
    eq = N;
    return;
  }
  int nb = 32 - __clz(diff);
  uint32_t prefix = (uint32_t)(((uint64_t)a >> nb) << nb);
  int krem = rank;

  // ---- first pass: every element shares the prefix above bit nb
  {
    const int db = min(kFirstBits, nb), shift = nb - db;
    const uint32_t dmask = (1u << db) - 1u;
    for (int i = tid; i < (1 << db); i += kSelThreads) sh.hist[i] = 0u;
    __syncthreads();
#pragma unroll
    for (int e = 0; e < E; ++e) hist_add(sh.hist, base + e < N, (keyf(e) >> shift) & dmask);
    __syncthreads();
    block_find_bin(1 << db, krem, sh);
    prefix |= sh.res_digit << shift;
    krem -= (int)sh.res_before;
    less += (int)sh.res_before;
    nb = shift;
    eq = (int)sh.res_count;
  }
  if (nb == 0) {
    res = prefix;
    return;
  }
  const int ncand = eq;
  if (ncand <= kCandCap) {
    // ---- compact the candidates (keys sharing the prefix above bit nb)
    int mine = 0;
#pragma unroll
    for (int e = 0; e < E; ++e)
      mine += (base + e < N && ((uint64_t)keyf(e) >> nb) == ((uint64_t)prefix >> nb)) ? 1 : 0;
    int tot;
    int off = block_excl_scan(mine, sh, tot);
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const uint32_t k = keyf(e);
      if (base + e < N && ((uint64_t)k >> nb) == ((uint64_t)prefix >> nb) && off < kCandCap)
        sh.cand[off++] = k;
    }
    __syncthreads();
    const int rounds = (ncand + kSelThreads - 1) / kSelThreads;
    while (nb > 0) {
      const int db = min(kLaterBits, nb), shift = nb - db;
      const uint32_t dmask = (1u << db) - 1u;
      if (tid < (1 << kLaterBits)) sh.hist[tid] = 0u;
      __syncthreads();
      for (int r = 0; r < rounds; ++r) {
        const int c = r * kSelThreads + tid;
        const uint32_t k = c < ncand ? sh.cand[c] : 0u;
        const bool act = c < ncand && ((uint64_t)k >> nb) == ((uint64_t)prefix >> nb);
        hist_add(sh.hist, act, (k >> shift) & dmask);
      }
      __syncthreads();
      wave0_find_bin(krem, sh);
      prefix |= sh.res_digit << shift;
      krem -= (int)sh.res_before;
      less += (int)sh.res_before;
      eq = (int)sh.res_count;
      nb = shift;
      __syncthreads();  // sh.res_* and sh.hist are rewritten next round
    }
  } else {
    // ---- many keys share the first digit: resolve the rest over all elements
    while (nb > 0) {
      const int db = min(kLaterBits, nb), shift = nb - db;
      const uint32_t dmask = (1u << db) - 1u;
      if (tid < (1 << kLaterBits)) sh.hist[tid] = 0u;
      __syncthreads();
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const uint32_t k = keyf(e);
        const bool act = base + e < N && ((uint64_t)k >> nb) == ((uint64_t)prefix >> nb);
        hist_add(sh.hist, act, (k >> shift) & dmask);
      }
      __syncthreads();
      wave0_find_bin(krem, sh);
      prefix |= sh.res_digit << shift;
      krem -= (int)sh.res_before;
      less += (int)sh.res_before;
      eq = (int)sh.res_count;
      nb = shift;
      __syncthreads();
    }
  }
  res = prefix;
}

// Stable top-K: keep every element whose score is above the K-th largest and
// the lowest-index elements equal to it, and write the kept indices in
// ascending order to out[0..K).
template <int E>
__device__ void block_topk_write(const float (&sc)[E], int base, int N, int K, int32_t* out,
                                 SelectShared& sh) {
  auto keyf = [&](int e) { return f2key(sc[e]); };
  uint32_t thr;
  int less, eq;
  block_select<E>(keyf, base, N, N - K, thr, less, eq, sh);
  const int need_eq = K - (N - less - eq);
  int my_eq = 0;
#pragma unroll
  for (int e = 0; e < E; ++e) my_eq += (base + e < N && keyf(e) == thr) ? 1 : 0;
  int tot;
  int run = block_excl_scan(my_eq, sh, tot);
  uint32_t keep_mask = 0u;
  int my_keep = 0;
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const bool valid = base + e < N;
    const uint32_t k = keyf(e);
    const bool is_eq = valid && k == thr;
    const bool keep = valid && (k > thr || (is_eq && run < need_eq));
    run += is_eq ? 1 : 0;
    keep_mask |= keep ? (1u << e) : 0u;
    my_keep += keep ? 1 : 0;
  }
  int pos = block_excl_scan(my_keep, sh, tot);
#pragma unroll
  for (int e = 0; e < E; ++e)
    if (((keep_mask >> e) & 1u) && pos < K) out[pos++] = base + e;  // exactly K kept; bound guards memory
}

}  // namespace trevs
