// Workgroup-wide exact order statistics and stable top-K.  One workgroup of
// 1024 threads ranks one vector; thread t owns elements t, t + 1024, ...,
// (element e*1024 + t is its e-th), so loads and stores are coalesced.
#pragma once

#include <type_traits>

#include "common.hpp"

namespace trevs {

constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / kWave;
constexpr int kFirstBits = 11;                // digit width of the first radix pass
constexpr int kFirstBins = 1 << kFirstBits;
constexpr int kLaterBits = 8;                 // digit width of the candidate passes
constexpr int kCandCap = 4096;                // candidates kept in LDS after the first pass

constexpr int kMaxE = 64;                     // elements per thread (N <= 65536)

// One bit per element of a thread (bit e: element e*1024 + t).
template <int E>
using SelMask = typename std::conditional<(E > 32), uint64_t, uint32_t>::type;

struct SelectShared {
  uint32_t hist[kFirstBins];
  uint32_t cand[kCandCap];
  uint32_t wcnt[kMaxE * kSelWaves];           // per (element round, wave) counts
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
  // every wave scans the (few) wave totals itself
  const int wt = lane < kSelWaves ? sh.wave_tot[lane] : 0;
  const int wi = wave_incl_scan(wt, lane);
  const int before = __builtin_amdgcn_readlane(wi - wt, wave);
  total = __builtin_amdgcn_readlane(wi, kSelWaves - 1);
  __syncthreads();  // sh.wave_tot is rewritten by the next call
  return before + inc - v;
}

// Finds the bin holding rank krem in hist[0, nbins) (nbins <= 2 * 1024):
// thread t owns bins 2t and 2t+1, a workgroup scan orders them.
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

// A copy of v that the compiler cannot see through, so that compares on it are
// redone where they are used instead of being kept live (as one 64-bit lane
// mask per element) across a whole selection.
__device__ __forceinline__ int opaque(int v) {
  asm volatile("" : "+v"(v));
  return v;
}

// Number of this thread's valid elements: element e is valid iff e < rounds.
template <int E>
__device__ __forceinline__ int thread_rounds(int N) {
  const int t = (int)threadIdx.x;
  return N > t ? min(E, (N - t + kSelThreads - 1) / kSelThreads) : 0;
}

// Histogram pass over this thread's keys (all E of them: unused slots hold
// the minimum key, see block_select): keys equal to the set minimum
// `kmin` (often a large tie, e.g. exact zeros) are counted with one ballot per
// wave and added once; every other key adds one to its digit's bin (bits
// [shift, shift + db) of the key).
template <int E, class Match>
__device__ __forceinline__ void hist_pass(const uint32_t (&k)[E], Match match, uint32_t kmin,
                                          int shift, int db, SelectShared& sh) {
  const int lane = threadIdx.x & (kWave - 1);
  int nmin = 0;  // per lane, summed over the wave once
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const bool act = match(k[e]);
    nmin += (act && k[e] == kmin) ? 1 : 0;
    if (act && k[e] != kmin) atomicAdd(&sh.hist[__builtin_amdgcn_ubfe(k[e], shift, db)], 1u);
  }
  nmin = wave_reduce_bits(nmin, 0, [](int x, int y) { return x + y; });
  if (lane == 0 && nmin) atomicAdd(&sh.hist[__builtin_amdgcn_ubfe(kmin, shift, db)], (uint32_t)nmin);
}

// Exact rank selection on uint32 keys.  keyf(e) yields the key of this
// thread's element e; it is evaluated once per element and the keys are held
// in registers.  Returns the key of ascending 0-based rank `rank` among the N
// valid keys, with the number of keys strictly below it (less) and equal to it
// (eq).  If have_range, kmin and kmax are the minimum and maximum key, or
// bounds of them (else they are computed).  N <= E * 1024.
//   0. the E * 1024 - N unused slots take the key kmin: they sort first, so
//      rank r among the valid keys is rank r + (E * 1024 - N) among all
//      slots, and no pass tests validity;
//   1. the bits above the highest bit where min and max differ are common;
//   2. one pass over all elements on the next (up to) 11 bits;
//   3. the keys in the chosen bin are appended to LDS (if they fit) and the
//      remaining bits are resolved 8 at a time over them alone; otherwise the
//      remaining passes scan all elements.
template <int E, class KeyF>
__device__ void block_select(KeyF keyf, int N, int rank, uint32_t& res, int& less, int& eq,
                             SelectShared& sh, bool have_range = false, uint32_t kmin = 0u,
                             uint32_t kmax = 0u) {
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const int nv = thread_rounds<E>(N);
  uint32_t k[E];
#pragma unroll
  for (int e = 0; e < E; ++e) k[e] = keyf(e);
  uint32_t a = kmin, z = kmax;
  if (!have_range) {
    uint32_t mn = 0xffffffffu, mx = 0u;
#pragma unroll
    for (int e = 0; e < E; ++e)
      if (e < nv) {
        mn = min(mn, k[e]);
        mx = max(mx, k[e]);
      }
    mn = wave_min_u32(mn);
    mx = wave_max_u32(mx);
    if (lane == 0) {
      sh.mn[wave] = mn;
      sh.mx[wave] = mx;
    }
    __syncthreads();
    a = 0xffffffffu;
    z = 0u;
#pragma unroll
    for (int w = 0; w < kSelWaves; ++w) {
      a = min(a, sh.mn[w]);
      z = max(z, sh.mx[w]);
    }
    __syncthreads();  // sh.mn / sh.mx are rewritten by the next call
  }
  const uint32_t diff = a ^ z;
  less = 0;
  if (diff == 0u) {
    res = a;
    eq = N;
    return;
  }
  const int n_unused = E * kSelThreads - N;
  const int nv_sub = opaque(nv);
#pragma unroll
  for (int e = 0; e < E; ++e) k[e] = e < nv_sub ? k[e] : a;
  int nb = 32 - __clz(diff);
  uint32_t prefix = (uint32_t)(((uint64_t)a >> nb) << nb);
  int krem = rank + n_unused;

  // ---- first pass: every element shares the prefix above bit nb
  {
    const int db = min(kFirstBits, nb), shift = nb - db;
    const int nbins = 1 << db;
    for (int i = tid; i < nbins; i += kSelThreads) sh.hist[i] = 0u;
    if (tid == 0) sh.total = 0;
    __syncthreads();
    hist_pass<E>(k, [](uint32_t) { return true; }, a, shift, db, sh);
    __syncthreads();
    block_find_bin(nbins, krem, sh);
    prefix |= sh.res_digit << shift;
    krem -= (int)sh.res_before;
    less += (int)sh.res_before;
    nb = shift;
    eq = (int)sh.res_count;
  }
  // from here on nb <= 31: keys under the prefix share their bits above nb
  const auto under_prefix = [&](uint32_t key) { return (key >> nb) == (prefix >> nb); };
  const int ncand = eq;
  if (nb == 0) {
    // the first digit resolved every bit
  } else if (ncand <= kCandCap) {
    // ---- append the candidates (keys sharing the prefix above bit nb);
    // their order does not matter for a rank selection.  One LDS atomic per
    // wave reserves room for all of the wave's candidates.
    int wn = 0;
#pragma unroll
    for (int e = 0; e < E; ++e) wn += __popcll(__ballot(under_prefix(k[e])));
    int wbase = 0;
    if (lane == 0 && wn) wbase = atomicAdd(&sh.total, wn);
    wbase = __builtin_amdgcn_readfirstlane(wbase);
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const bool m = under_prefix(k[e]);
      const unsigned long long bal = __ballot(m);
      const int pos = wbase + (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(bal >> 32),
                                                             __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0u));
      if (m && pos < kCandCap) sh.cand[pos] = k[e];
      wbase += __popcll(bal);
    }
    __syncthreads();
    const int rounds = (ncand + kSelThreads - 1) / kSelThreads;
    while (nb > 0) {
      const int db = min(kLaterBits, nb), shift = nb - db;
      if (tid < (1 << kLaterBits)) sh.hist[tid] = 0u;
      __syncthreads();
      for (int r = 0; r < rounds; ++r) {
        const int c = r * kSelThreads + tid;
        const uint32_t key = c < ncand ? sh.cand[c] : 0u;
        if (c < ncand && under_prefix(key)) atomicAdd(&sh.hist[__builtin_amdgcn_ubfe(key, shift, db)], 1u);
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
      if (tid < (1 << kLaterBits)) sh.hist[tid] = 0u;
      __syncthreads();
      hist_pass<E>(k, under_prefix, a, shift, db, sh);
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
  // the unused slots hold the key a: below res, or tied with it
  if (res == a)
    eq -= n_unused;
  else
    less -= n_unused;
}

// Exclusive prefix sums of sh.wcnt[0, n) in place (n <= kMaxE * kSelWaves),
// by wave 0; entries are ordered (element round, wave), which is index order.
// Unsigned (wrapping) sums: packed entries carry a count in each 16-bit
// half, and only the exclusive sums, which stay below 2^16 in each half,
// are read.
__device__ __forceinline__ void wcnt_scan(int n, SelectShared& sh) {
  __syncthreads();
  if (threadIdx.x < kWave) {
    const int lane = threadIdx.x;
    const int per = (n + kWave - 1) / kWave;
    uint32_t* c = sh.wcnt + lane * per;
    uint32_t lsum = 0u;
    for (int j = 0; j < per; ++j)
      if (lane * per + j < n) lsum += c[j];
    uint32_t run = wave_incl_scan_u32(lsum) - lsum;
    for (int j = 0; j < per; ++j)
      if (lane * per + j < n) {
        const uint32_t v = c[j];
        c[j] = run;
        run += v;
      }
  }
  __syncthreads();
}

// Stable top-K as a mask: bit e of the result is set when this thread's
// element e is kept, i.e. its key is above the K-th largest, or equal to it
// and among the lowest-index elements of that key (K in 0..N).
template <int E, class KeyF>
__device__ SelMask<E> block_topk_mask(KeyF keyf, int N, int K, SelectShared& sh) {
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const int nv = thread_rounds<E>(N);
  auto valid = [&](int e) { return e < nv; };
  if (K <= 0) return SelMask<E>(0);
  if (K >= N) {
    SelMask<E> all = 0;
#pragma unroll
    for (int e = 0; e < E; ++e) all |= valid(e) ? (SelMask<E>(1) << e) : SelMask<E>(0);
    return all;
  }
  uint32_t key[E];
#pragma unroll
  for (int e = 0; e < E; ++e) key[e] = keyf(e);
  uint32_t thr;
  int less, eq;
  block_select<E>([&](int e) { return key[e]; }, N, N - K, thr, less, eq, sh);
  const int need_eq = K - (N - less - eq);
  auto lanes_below = [&](unsigned long long bal) {
    return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(bal >> 32),
                                          __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0u));
  };
  // rank of every tie among the ties, in index order (ballots are recomputed
  // after each scan rather than held)
  auto is_eq = [&](int e) { return valid(e) && key[e] == thr; };
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const unsigned long long bal = __ballot(is_eq(e));
    if (lane == 0) sh.wcnt[e * kSelWaves + wave] = __popcll(bal);
  }
  wcnt_scan(E * kSelWaves, sh);
  SelMask<E> keep_mask = 0;
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const bool eqe = is_eq(e);
    const int eq_rank = (int)sh.wcnt[e * kSelWaves + wave] + lanes_below(__ballot(eqe));
    const bool keep = valid(e) && (key[e] > thr || (eqe && eq_rank < need_eq));
    keep_mask |= keep ? (SelMask<E>(1) << e) : SelMask<E>(0);
  }
  __syncthreads();  // sh.wcnt is rewritten by the caller's next step
  return keep_mask;
}

// Writes the indices of the elements set in `mask` (K of them over the
// workgroup) in ascending order to out[0..K).
template <int E>
__device__ void block_write_mask(SelMask<E> mask, int K, int32_t* out, SelectShared& sh) {
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  auto lanes_below = [&](unsigned long long bal) {
    return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(bal >> 32),
                                          __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0u));
  };
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const unsigned long long bal = __ballot((mask >> e) & 1u);
    if (lane == 0) sh.wcnt[e * kSelWaves + wave] = __popcll(bal);
  }
  wcnt_scan(E * kSelWaves, sh);
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const bool kp = (mask >> e) & 1u;
    const int pos = (int)sh.wcnt[e * kSelWaves + wave] + lanes_below(__ballot(kp));
    if (kp && pos < K) out[pos] = e * kSelThreads + tid;  // exactly K kept; the bound guards memory
  }
}

// Stable top-K: keep every element whose score is above the K-th largest and
// the lowest-index elements equal to it, and write the kept indices in
// ascending order to out[0..K).  After the threshold selection one scan does
// the rest: element i goes to slot above(i) + min(ties(i), need), where
// above(i) and ties(i) count the elements before i (in index order) above the
// threshold and equal to it, and need is how many ties are kept.  The two
// counts travel packed in one word (low and high 16 bits: every exclusive
// count is below N <= 65536).
// have_range, kmin, kmax: bounds of the keys, as for block_select.
template <int E>
__device__ void block_topk_write(const float (&sc)[E], int N, int K, int32_t* out,
                                 SelectShared& sh, bool have_range = false, uint32_t kmin = 0u,
                                 uint32_t kmax = 0u) {
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const int nv = thread_rounds<E>(N);
  auto valid = [&](int e) { return e < nv; };
  if (K <= 0) return;
  if (K >= N) {
#pragma unroll
    for (int e = 0; e < E; ++e)
      if (valid(e)) out[e * kSelThreads + tid] = e * kSelThreads + tid;
    return;
  }
  uint32_t key[E];
#pragma unroll
  for (int e = 0; e < E; ++e) key[e] = f2key(sc[e]);
  uint32_t thr;
  int less, eq;
  block_select<E>([&](int e) { return key[e]; }, N, N - K, thr, less, eq, sh, have_range, kmin, kmax);
  const int need = K - (N - less - eq);  // ties kept, lowest index first
  auto lanes_below = [&](unsigned long long bal) {
    return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(bal >> 32),
                                          __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0u));
  };
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const uint32_t k = key[e];
    const unsigned long long ba = __ballot(valid(e) && k > thr);
    const unsigned long long bt = __ballot(valid(e) && k == thr);
    if (lane == 0) sh.wcnt[e * kSelWaves + wave] = (uint32_t)__popcll(ba) | ((uint32_t)__popcll(bt) << 16);
  }
  wcnt_scan(E * kSelWaves, sh);
  // the output base lives in a VGPR pair: held in SGPRs through the
  // selection it was spilled and re-read for every store
  uint64_t obase = (uint64_t)(uintptr_t)out;
  asm volatile("" : "+v"(obase));
  int32_t* const o = (int32_t*)(uintptr_t)obase;
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const uint32_t k = key[e];
    const bool above = valid(e) && k > thr, tie = valid(e) && k == thr;
    const unsigned long long ba = __ballot(above);
    const unsigned long long bt = __ballot(tie);
    const uint32_t base = sh.wcnt[e * kSelWaves + wave];
    const int na = (int)(base & 0xffffu) + lanes_below(ba);  // above the threshold, before this element
    const int nt = (int)(base >> 16) + lanes_below(bt);      // ties before this element
    if (above || (tie && nt < need)) {
      const int pos = na + min(nt, need);
      if (pos < K) o[pos] = e * kSelThreads + tid;  // exactly K kept; the bound guards memory
    }
  }
}

}  // namespace trevs
