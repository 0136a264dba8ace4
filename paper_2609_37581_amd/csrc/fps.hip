// Context preservation by farthest point sampling (Sec. 4.1, after Eq. (7)):
// K_d tokens are added one at a time to the pivot set, each the candidate
// whose cosine distance 1 - zbar_i . zbar_j to the nearest already-selected
// token is largest (ties to the lower index).
//
// The picks are sequential, and every pick needs the distances of all
// candidates to one more token.  Instead of re-reading Z for each pick, the
// Gram matrix G = Z Z^T of the sample is formed once on the matrix cores;
// a pick then reads one row of G (N floats).  ||z_i||^2 is its diagonal.
#include "common.hpp"
#include "kernels.hpp"
#include "select.hpp"

namespace trevs {

// ---------------------------------------------------------------------------
// Gram matrix.  G is symmetric, so only the tiles (tj, ti) with tj <= ti are
// computed: a workgroup of 4 waves computes the 128x128 tile of G[b] (rows j
// of the tile's first operand, columns i of the second), streaming the
// feature dimension in 128-byte slabs: each thread loads its share of both
// slabs with coalesced 16-byte loads (8 lanes per 128-byte row segment) into
// a ring of two register buffers, writes them to one of two LDS buffers
// (rows XOR-swizzled by 16-byte chunk), and the waves multiply on the matrix
// cores, each a 64x64 block.  Bytes past a row's end (a partial last slab)
// load as zero.  The tile is written in place and, off the diagonal, also
// transposed; both go through LDS and out as 16-byte runs of whole rows.
// Diagonal tiles also write 1/max(||z_i||, 1e-12) from G_ii.  G is written
// with nontemporal stores: the picks read it back long after it has left the
// caches, and cached stores would evict operand slabs the other resident
// workgroups still read.
// ---------------------------------------------------------------------------
constexpr int kGramTile = 128;
constexpr int kGramThreads = 256;

// Workgroup order: the tiles on and above the diagonal are walked in
// super-blocks of gs x gs tiles (gs = min(8, tiles per side)), so that the
// workgroups resident on one XCD at a time share 2*gs row blocks of Z and
// each slab they stream is reused from L2 by up to gs workgroups (in
// row-major tile order they shared one row block and streamed 64 distinct
// ones).  Super-blocks are numbered row-major over the pairs sj <= si, and
// every workgroup gets a tile: a diagonal super-block holds only its tiles
// on and above the diagonal (row-major), so the workgroups resident at one
// time cover compact runs of tiles instead of slots that exit at once.
__host__ __device__ constexpr int gram_super(int n_tiles) { return n_tiles < 8 ? n_tiles : 8; }
__host__ __device__ constexpr int gram_tiles(int n_tiles) { return n_tiles * (n_tiles + 1) / 2; }

// tile (tj, ti), tj <= ti, of dense index t in [0, gram_tiles(nT))
__device__ __forceinline__ void gram_tile_of(int t, int nT, int& tj, int& ti) {
  const int gs = gram_super(nT), nS = (nT + gs - 1) / gs;
  tj = 0;
  ti = 0;
  for (int sj = 0; sj < nS; ++sj) {
    const int h = min(gs, nT - sj * gs);
    for (int si = sj; si < nS; ++si) {
      const int w = min(gs, nT - si * gs);
      const int cnt = si == sj ? h * (h + 1) / 2 : h * w;
      if (t < cnt) {
        if (si == sj) {
          int r = 0;
          while (t >= h - r) {
            t -= h - r;
            ++r;
          }
          tj = sj * gs + r;
          ti = sj * gs + r + t;
        } else {
          tj = sj * gs + t / w;
          ti = si * gs + t % w;
        }
        return;
      }
      t -= cnt;
    }
  }
}

// Workgroup -> (sample b, dense tile index t).  With many tiles per sample
// (kGramStripe or more) XCD x takes the x-th eighth of every sample's tiles
// (a contiguous run in super-block order, for its L2), sample after sample,
// so that at any time all XCDs stream the same sample's Z, which fits the
// last-level cache (all samples together need not); workgroups go to the 8
// XCDs round-robin, and the grid, 8 * B * ceil(tiles / 8), has a few padding
// workgroups (false).  With few tiles per sample each XCD keeps whole
// samples instead (a contiguous range of workgroups per XCD), so that a
// sample's Z is loaded into one L2 only.
constexpr int kGramStripe = 64;
__device__ __forceinline__ bool gram_work(int per_b, int B, int& b, int& t) {
  if (per_b < kGramStripe) {
    const int lin = xcd_remap(blockIdx.x, gridDim.x);
    b = lin / per_b;
    t = lin - b * per_b;
    return true;
  }
  const int x = blockIdx.x & 7, k = blockIdx.x >> 3;
  const int r0 = (x * per_b) >> 3, L = (((x + 1) * per_b) >> 3) - r0;  // L >= 8
  b = k / L;
  t = r0 + (k - b * L);
  return b < B;
}
__host__ __device__ constexpr int gram_grid(int n_tiles, int B) {
  return gram_tiles(n_tiles) < kGramStripe ? B * gram_tiles(n_tiles) : 8 * B * ((gram_tiles(n_tiles) + 7) / 8);
}

__device__ __forceinline__ int gram_swizzle(int r, int c) { return c ^ ((r >> 1) & 7); }

template <class In>
__global__ __launch_bounds__(kGramThreads) void gram_kernel(GramArgs a) {
  constexpr int T = kGramTile;
  constexpr int SLAB = T * 128;                  // bytes of one operand slab
  constexpr int VPT = SLAB / 16 / kGramThreads;  // vectors per thread per operand
  constexpr int LDS = 4 * SLAB;                  // two stages of both operand slabs, then the output passes
  __shared__ __attribute__((aligned(1024))) uint8_t lds[LDS];
  uint8_t* l0 = lds;
  uint8_t* l1 = lds + 2 * SLAB;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, col = lane & 31;
  const int nT = a.n_tiles;
  int b, t, tj, ti;
  if (!gram_work(gram_tiles(nT), a.B, b, t)) return;  // the whole workgroup: no barrier has run
  gram_tile_of(t, nT, tj, ti);
  const int N = a.N, rb = a.row_bytes;
  const int n_slabs = (rb + 127) / 128;
  const int tail = rb & 127;  // bytes of a partial last slab, 0 if none
  const uint8_t* zb = reinterpret_cast<const uint8_t*>(a.Z) + (size_t)b * N * rb;
  const int cr = tid >> 3, cc = tid & 7;
  const uint8_t* src[2 * VPT];  // row starts (rows past N re-read row N - 1)
#pragma unroll
  for (int k = 0; k < VPT; ++k) {
    const int r = cr + (kGramThreads / 8) * k;
    src[k] = zb + (size_t)min(tj * T + r, N - 1) * rb;
    src[VPT + k] = zb + (size_t)min(ti * T + r, N - 1) * rb;
  }
  const int sdst = cr * 128 + gram_swizzle(cr, cc) * 16;  // rows 32 apart share the swizzle
  u32x4 g[2][2 * VPT];
  // chunk cc of slab s; a chunk past the row's end reads the row's first
  // chunk (in bounds), and the store overwrites its LDS copy with zeros (a
  // select on the loaded vectors made the compiler wait for every load in
  // flight at the top of each iteration); the padding steps past the last
  // slab re-read it and are never multiplied
  auto load = [&](int s, u32x4 (&dst)[2 * VPT]) {
    const int off = min(s, n_slabs - 1) * 128 + cc * 16;
    const int o = off < rb ? off : 0;
#pragma unroll
    for (int k = 0; k < 2 * VPT; ++k) dst[k] = ldg16(src[k] + o);
  };
  auto store = [&](uint8_t* st, const u32x4 (&v)[2 * VPT], int s) {
#pragma unroll
    for (int k = 0; k < VPT; ++k) {
      *reinterpret_cast<u32x4*>(st + sdst + k * (kGramThreads / 8) * 128) = v[k];
      *reinterpret_cast<u32x4*>(st + SLAB + sdst + k * (kGramThreads / 8) * 128) = v[VPT + k];
    }
    if (s == n_slabs - 1 && tail && cc * 16 >= tail) {  // chunks past the row's end hold zeros
#pragma unroll
      for (int k = 0; k < VPT; ++k) {
        *reinterpret_cast<u32x4*>(st + sdst + k * (kGramThreads / 8) * 128) = zero4();
        *reinterpret_cast<u32x4*>(st + SLAB + sdst + k * (kGramThreads / 8) * 128) = zero4();
      }
    }
  };
  const int wj = wave >> 1, wi = wave & 1;
  f32x16 acc[2][2];
#pragma unroll
  for (int m = 0; m < 2; ++m)
#pragma unroll
    for (int n = 0; n < 2; ++n)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[m][n][r] = 0.f;
  auto frag = [&](const uint8_t* base, int row, u32x4 (&f)[4]) {
#pragma unroll
    for (int q = 0; q < 4; ++q)
      f[q] = *reinterpret_cast<const u32x4*>(base + row * 128 + gram_swizzle(row, 4 * half + q) * 16);
  };
  auto compute = [&](const uint8_t* st) {
    u32x4 fa[2][4], fb[2][4];
#pragma unroll
    for (int m = 0; m < 2; ++m) frag(st, wj * 64 + m * 32 + col, fa[m]);
#pragma unroll
    for (int n = 0; n < 2; ++n) frag(st + SLAB, wi * 64 + n * 32 + col, fb[n]);
#pragma unroll
    for (int m = 0; m < 2; ++m)
#pragma unroll
      for (int n = 0; n < 2; ++n) acc[m][n] = mfma_frag(fa[m], fb[n], acc[m][n], In{});
  };
  // stage 0's loads go out first: loads complete in order, so the first
  // store then waits only for them, not for stage 1's as well
  load(0, g[0]);
  __builtin_amdgcn_sched_barrier(0);
  load(1, g[1]);
  const int n_iter = (n_slabs + 1) / 2;
  for (int it = 0; it < n_iter; ++it) {
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int s = 2 * it + c;
      uint8_t* st = c ? l1 : l0;
      // buffer c was last read at step s - 2, before every wave passed the
      // barrier of step s - 1
      store(st, g[c], s);
      load(s + 2, g[c]);
      __syncthreads();
      if (s < n_slabs) compute(st);
    }
  }
  // output: register r of block (m, n) is row wj*64 + m*32 + mfma_row(r),
  // column wi*64 + n*32 + col of the tile
  if (tj == ti) {  // the diagonal tile holds ||z_i||^2
#pragma unroll
    for (int m = 0; m < 2; ++m)
#pragma unroll
      for (int n = 0; n < 2; ++n)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int jl = wj * 64 + m * 32 + mfma_row(r, half), il = wi * 64 + n * 32 + col;
          const int i = ti * T + il;
          if (jl == il && i < N)
            a.inv_norm[(size_t)b * N + i] = 1.f / fmaxf(sqrtf(fmaxf(acc[m][n][r], 0.f)), 1e-12f);
        }
  }
  // The tile leaves through LDS, 32 rows j at a time, as 16-byte runs of
  // whole rows: tA (rows j, stride TA: 16-byte aligned rows, the half-waves'
  // writes on disjoint banks) for G[j, i]; off the diagonal tB (rows i, odd
  // stride TB) for the mirrored G[i, j].  Whole tiles of a matrix whose rows
  // are a multiple of 16 bytes store without bounds checks.
  constexpr int TA = T + 8, TB = 33, PR = 32;
  static_assert((PR * TA + T * TB) * 4 <= LDS, "output staging fits the LDS");
  float* tA = reinterpret_cast<float*>(lds);
  float* tB = tA + PR * TA;
  float* gb = a.G + (size_t)b * N * N;
  const bool mirror = tj != ti;
  const bool fast = (ti + 1) * T <= N && (N & 3) == 0;  // tj <= ti
#pragma unroll
  for (int p = 0; p < T / PR; ++p) {  // unrolled: the accumulator block m is a constant
    __syncthreads();  // the operand slabs, or the previous pass, are no longer read
    if (wj == p / 2) {
      const int m = p % 2;
#pragma unroll
      for (int n = 0; n < 2; ++n)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int jl = mfma_row(r, half), il = wi * 64 + n * 32 + col;
          tA[jl * TA + il] = acc[m][n][r];
          if (mirror) tB[il * TB + jl] = acc[m][n][r];
        }
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < PR * T / 4 / kGramThreads; ++k) {  // G[j, i]: PR rows of T / 4 runs
      const int e = tid + k * kGramThreads, row = e / (T / 4), q = e % (T / 4);
      const int j = tj * T + PR * p + row, i = ti * T + 4 * q;
      const u32x4 v = *reinterpret_cast<const u32x4*>(&tA[row * TA + 4 * q]);
      if (fast) {
        stg16_stream(&gb[(size_t)j * N + i], v);
      } else {
#pragma unroll
        for (int u = 0; u < 4; ++u)
          if (j < N && i + u < N) __builtin_nontemporal_store(__uint_as_float(v[u]), &gb[(size_t)j * N + i + u]);
      }
    }
    if (mirror) {  // G[i, j]: T rows of PR / 4 runs
#pragma unroll
      for (int k = 0; k < PR * T / 4 / kGramThreads; ++k) {
        const int e = tid + k * kGramThreads, il = e / (PR / 4), q = e % (PR / 4);
        const int i = ti * T + il, j = tj * T + PR * p + 4 * q;
        const float* src = &tB[il * TB + 4 * q];
        const u32x4 v = {__float_as_uint(src[0]), __float_as_uint(src[1]), __float_as_uint(src[2]),
                         __float_as_uint(src[3])};
        if (fast) {
          stg16_stream(&gb[(size_t)i * N + j], v);
        } else {
#pragma unroll
          for (int u = 0; u < 4; ++u)
            if (i < N && j + u < N) __builtin_nontemporal_store(__uint_as_float(v[u]), &gb[(size_t)i * N + j + u]);
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Gram matrix at 256x256 tiles, bf16 (N >= kGram256MinN, N + 256 rows of Z
// under 2 GB; fp32 inputs use gram_kernel; rows are a multiple of 16 bytes): a
// workgroup of 4 waves, one per SIMD, each a 128x128 block (4x4 MFMA tiles,
// 256 accumulation registers), so that each fragment byte read from LDS
// feeds 4 multiplies.  The feature dimension streams in 128-byte stages
// (four k-steps), loaded 8 lanes to a row (whole 128-byte lines: 4 lanes to
// a row, 64 bytes, cost about a tenth of the Gram's time) into a ring of two
// register stages, then into two LDS buffers.  Stage P runs in two halves:
// the first multiplies k-steps 0-1 while it stores stage P + 1 into the
// other buffer (free since the last barrier) and loads stage P + 3 into the
// register stage it frees; after a barrier, the second multiplies k-steps
// 2-3 while it reads stage P + 1's first fragments.  Every k-step's
// fragments are read during the previous k-step's multiplies, so each half
// starts on fragments already in registers.  The loads are buffer loads:
// chunks past a row's end, rows past N and stages past the last read zeros,
// which the multiplies add exactly, so the steps need no branches.  Rows are
// XOR-swizzled in 16-byte chunks (chunk ^ ((row >> 1) & 7)): the stores (2
// rows x 128 bytes per 16 lanes) and the fragment reads (16 rows at one
// chunk) hit all 64 banks.  Same super-block order and outputs as
// gram_kernel; both output tiles leave through LDS as 16-byte runs of whole
// rows.
// ---------------------------------------------------------------------------
constexpr int kGram256Threads = 256;
constexpr int kGram256MinN = 2048;

__global__ __launch_bounds__(kGram256Threads, 1) void gram256_kernel(GramArgs a) {
  constexpr int T = 256;
  constexpr int SLAB = T * 128;                     // bytes of one operand's 128-byte stage
  constexpr int VPT = SLAB / 16 / kGram256Threads;  // 8 vectors per thread per operand
  constexpr int RSTEP = kGram256Threads / 8;        // rows per load pass (8 lanes a row)
  constexpr int TA = T + 8, TB = 33, PR = 32;       // output staging (see below)
  constexpr int LDS_OPS = 4 * SLAB;
  constexpr int LDS_OUT = (PR * TA + T * TB) * 4;
  constexpr int LDS = LDS_OPS > LDS_OUT ? LDS_OPS : LDS_OUT;
  __shared__ __attribute__((aligned(1024))) uint8_t lds[LDS];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, col = lane & 31;
  const int nT = a.n_tiles;
  int b, t, tj, ti;
  if (!gram_work(gram_tiles(nT), a.B, b, t)) return;  // the whole workgroup: no barrier has run
  gram_tile_of(t, nT, tj, ti);
  const int N = a.N, rb = a.row_bytes;
  const int n_stages = (rb + 127) / 128;
  // rows past N read zeros (their offsets pass N * rb), and so do the chunks
  // of a stage that is past the row's end (offset + 2^31): with
  // (N + 256) * rb < 2^31 no offset wraps.  Rows and columns past N are never
  // stored.
  const __amdgpu_buffer_rsrc_t zs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(reinterpret_cast<const uint8_t*>(a.Z) + (size_t)b * N * rb), 0, N * rb,
      kBufferRsrcWord3);
  const int cr = tid >> 3, cc = tid & 7;
  // the thread loads chunk cc of rows cr + RSTEP * k of both operands
  const uint32_t rowA = (uint32_t)(tj * T + cr) * rb + cc * 16;
  const uint32_t rowB = (uint32_t)(ti * T + cr) * rb + cc * 16;
  const uint32_t kstride = (uint32_t)RSTEP * rb;
  // LDS: operand A of buffers 0 and 1, then operand B of buffers 0 and 1
  // (every fragment address is one register per k-step and operand plus an
  // immediate offset)
  const int sdst = cr * 128 + gram_swizzle(cr, cc) * 16;  // rows RSTEP apart share the swizzle
  u32x4 g[2][2 * VPT];
  // stage P; a chunk past the row's end (and every chunk past the last
  // stage) takes an offset outside the buffer and reads zeros
  auto load = [&](int P, u32x4 (&dst)[2 * VPT]) {
    const uint32_t so = P * 128 + cc * 16 < rb ? (uint32_t)P * 128u : 0x80000000u;
    const uint32_t oa = rowA + so, ob = rowB + so;
#pragma unroll
    for (int k = 0; k < VPT; ++k) {
      dst[k] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(zs, oa + k * kstride, 0, 0));
      dst[VPT + k] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(zs, ob + k * kstride, 0, 0));
    }
  };
  auto store = [&](int c, const u32x4 (&v)[2 * VPT]) {
#pragma unroll
    for (int k = 0; k < VPT; ++k) {
      *reinterpret_cast<u32x4*>(lds + c * SLAB + sdst + k * RSTEP * 128) = v[k];
      *reinterpret_cast<u32x4*>(lds + 2 * SLAB + c * SLAB + sdst + k * RSTEP * 128) = v[VPT + k];
    }
  };
  const int wj = wave >> 1, wi = wave & 1;  // rows wj*128.., columns wi*128.. of the tile
  f32x16 acc[4][4];
#pragma unroll
  for (int m = 0; m < 4; ++m)
#pragma unroll
    for (int n = 0; n < 4; ++n)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[m][n][r] = 0.f;
  // fragments of k-step q of a stage: half h holds logical chunk 2q + h.
  // Every row a lane reads (wj*128 + m*32 + col) has the swizzle of col.
  const int sw = (col >> 1) & 7;
  uint32_t fqa[4], fqb[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    fqa[q] = (wj * 128 + col) * 128 + ((2 * q + half) ^ sw) * 16;
    fqb[q] = 2 * SLAB + (wi * 128 + col) * 128 + ((2 * q + half) ^ sw) * 16;
  }
  auto frag = [&](int c, int q, u32x4 (&fa)[4][1], u32x4 (&fb)[4][1]) {
#pragma unroll
    for (int m = 0; m < 4; ++m) fa[m][0] = *reinterpret_cast<const u32x4*>(lds + fqa[q] + c * SLAB + m * 32 * 128);
#pragma unroll
    for (int n = 0; n < 4; ++n) fb[n][0] = *reinterpret_cast<const u32x4*>(lds + fqb[q] + c * SLAB + n * 32 * 128);
  };
  auto mfma16 = [&](const u32x4 (&fa)[4][1], const u32x4 (&fb)[4][1]) {
#pragma unroll
    for (int m = 0; m < 4; ++m)
#pragma unroll
      for (int n = 0; n < 4; ++n) acc[m][n] = mfma_frag(fa[m], fb[n], acc[m][n], BF16{});
  };
  // an MFMA group of `n` multiplies, each followed by `r` LDS reads, `w` LDS
  // writes and `l` global loads (the compiler's scheduler fills the groups
  // in this order)
  auto interleave = [](auto n, auto r, auto w, auto l) {
#pragma unroll
    for (int u = 0; u < decltype(n)::value; ++u) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      if (decltype(r)::value) __builtin_amdgcn_sched_group_barrier(0x100, decltype(r)::value, 0);
      if (decltype(w)::value) __builtin_amdgcn_sched_group_barrier(0x200, decltype(w)::value, 0);
      if (decltype(l)::value) __builtin_amdgcn_sched_group_barrier(0x020, decltype(l)::value, 0);
    }
  };
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  using I8 = std::integral_constant<int, 8>;
  // stage P sits in register stage P % 2 and LDS buffer P % 2
  load(0, g[0]);
  __builtin_amdgcn_sched_barrier(0);
  load(1, g[1]);
  __builtin_amdgcn_sched_barrier(0);
  store(0, g[0]);
  load(2, g[0]);
  __syncthreads();
  u32x4 fa0[4][1], fb0[4][1], fa1[4][1], fb1[4][1];
  frag(0, 0, fa0, fb0);
  const int n_iter = (n_stages + 1) / 2;
  for (int it = 0; it < n_iter; ++it) {
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int P = 2 * it + c;
      // first half: k-steps 0 and 1; stage P + 1 to LDS, stage P + 3 loaded
      __builtin_amdgcn_sched_barrier(0);
      frag(c, 1, fa1, fb1);
      mfma16(fa0, fb0);
      store(1 - c, g[1 - c]);
      load(P + 3, g[1 - c]);
      frag(c, 2, fa0, fb0);
      mfma16(fa1, fb1);
      interleave(I8{}, I1{}, I0{}, I0{});
      interleave(I8{}, I0{}, I1{}, I1{});  // the stores spread over 16 multiplies (8 cost 2% more)
      interleave(I8{}, I0{}, I1{}, I1{});
      interleave(I8{}, I1{}, I0{}, I0{});
      __syncthreads();
      // second half: k-steps 2 and 3; stage P + 1's first fragments
      __builtin_amdgcn_sched_barrier(0);
      frag(c, 3, fa1, fb1);
      mfma16(fa0, fb0);
      frag(1 - c, 0, fa0, fb0);
      mfma16(fa1, fb1);
      interleave(I8{}, I1{}, I0{}, I0{});
      interleave(I8{}, I0{}, I0{}, I0{});
      interleave(I8{}, I1{}, I0{}, I0{});
      interleave(I8{}, I0{}, I0{}, I0{});
      __syncthreads();
    }
  }
  // register r of block (m, n) is row wj*128 + m*32 + mfma_row(r), column
  // wi*128 + n*32 + col of the tile
  if (tj == ti) {  // the diagonal tile holds ||z_i||^2
#pragma unroll
    for (int m = 0; m < 4; ++m)
#pragma unroll
      for (int n = 0; n < 4; ++n)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int jl = wj * 128 + m * 32 + mfma_row(r, half), il = wi * 128 + n * 32 + col;
          const int i = ti * T + il;
          if (jl == il && i < N)
            a.inv_norm[(size_t)b * N + i] = 1.f / fmaxf(sqrtf(fmaxf(acc[m][n][r], 0.f)), 1e-12f);
        }
  }
  // The tile leaves through LDS, 32 rows j at a time, and is stored as
  // 16-byte runs of whole rows (each lane storing 4 bytes, or 16-byte runs
  // of a few bytes per row, writes G at a fraction of the rate): tA holds
  // the pass as rows j (stride TA: 16-byte aligned rows, the two half-waves'
  // writes on disjoint banks) for G[j, i]; off the diagonal tB holds it as
  // rows i (odd stride TB: the column writes spread over the banks) for the
  // mirrored G[i, j].  Whole tiles of a matrix whose rows are a multiple of
  // 16 bytes store without bounds checks.
  float* tA = reinterpret_cast<float*>(lds);
  float* tB = tA + PR * TA;
  float* gbm = a.G + (size_t)b * N * N;
  const bool mirror = tj != ti;
  const bool fast = (ti + 1) * T <= N && (N & 3) == 0;  // tj <= ti
#pragma unroll
  for (int p = 0; p < T / PR; ++p) {  // unrolled: the accumulator block m is a constant
    __syncthreads();  // the operand slabs, or the previous pass, are no longer read
    if (wj == p / 4) {
      const int m = p % 4;
#pragma unroll
      for (int n = 0; n < 4; ++n)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int jl = mfma_row(r, half), il = wi * 128 + n * 32 + col;
          tA[jl * TA + il] = acc[m][n][r];
          if (mirror) tB[il * TB + jl] = acc[m][n][r];
        }
    }
    __syncthreads();
    // G[j, i]: PR rows of T / 4 runs
#pragma unroll
    for (int k = 0; k < PR * T / 4 / kGram256Threads; ++k) {
      const int e = tid + k * kGram256Threads, row = e / (T / 4), q = e % (T / 4);
      const int j = tj * T + PR * p + row, i = ti * T + 4 * q;
      const u32x4 v = *reinterpret_cast<const u32x4*>(&tA[row * TA + 4 * q]);
      if (fast) {
        stg16_stream(&gbm[(size_t)j * N + i], v);
      } else {
#pragma unroll
        for (int u = 0; u < 4; ++u)
          if (j < N && i + u < N) __builtin_nontemporal_store(__uint_as_float(v[u]), &gbm[(size_t)j * N + i + u]);
      }
    }
    if (mirror) {  // G[i, j]: T rows of PR / 4 runs
#pragma unroll
      for (int k = 0; k < PR * T / 4 / kGram256Threads; ++k) {
        const int e = tid + k * kGram256Threads, il = e / (PR / 4), q = e % (PR / 4);
        const int i = ti * T + il, j = tj * T + PR * p + 4 * q;
        const float* srcp = &tB[il * TB + 4 * q];
        const u32x4 v = {__float_as_uint(srcp[0]), __float_as_uint(srcp[1]), __float_as_uint(srcp[2]),
                         __float_as_uint(srcp[3])};
        if (fast) {
          stg16_stream(&gbm[(size_t)i * N + j], v);
        } else {
#pragma unroll
          for (int u = 0; u < 4; ++u)
            if (i < N && j + u < N) __builtin_nontemporal_store(__uint_as_float(v[u]), &gbm[(size_t)i * N + j + u]);
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Initial distances: for every token i, 1 - max over the pivots j of
// cos(z_i, z_j) = G_ij / (||z_i|| ||z_j||), with the inverse norms the Gram
// pass wrote.  One thread per token; the pivots are split over n_psplit
// workgroups per token block (grid z), each writing the maximum of
// G_ij / ||z_j|| over its share; the picks kernel takes the maximum over the
// splits (exact, so the order does not matter) and forms the distance.  The
// pivot loop is unrolled so that several row reads of G are in flight (a
// pivot's row is read at consecutive columns by consecutive threads).
// ---------------------------------------------------------------------------
constexpr int kFpsInitThreads = 256;

__global__ __launch_bounds__(kFpsInitThreads) void fps_init_kernel(FpsArgs a) {
  const int b = blockIdx.y, split = blockIdx.z, N = a.N;
  const int i = min((int)(blockIdx.x * kFpsInitThreads + threadIdx.x), N - 1);
  const float* gb = a.G + (size_t)b * N * N;
  const float* inb = a.inv_norm + (size_t)b * N;
  const int per = (a.K_r + a.n_psplit - 1) / a.n_psplit;
  const int p_begin = min(split * per, a.K_r), p_end = min(p_begin + per, a.K_r);
  const int32_t* piv = a.pivots + (size_t)b * a.K_r;
  constexpr int U = 8;
  float mx = -INFINITY;
  int p = p_begin;
  for (; p + U <= p_end; p += U) {
    int j[U];
    float g[U], izj[U];
#pragma unroll
    for (int u = 0; u < U; ++u) j[u] = piv[p + u];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      g[u] = gb[(size_t)j[u] * N + i];
      izj[u] = inb[j[u]];
    }
#pragma unroll
    for (int u = 0; u < U; ++u) mx = fmaxf(mx, g[u] * izj[u]);
  }
  for (; p < p_end; ++p) {
    const int j = piv[p];
    mx = fmaxf(mx, gb[(size_t)j * N + i] * inb[j]);
  }
  if (blockIdx.x * kFpsInitThreads + threadIdx.x < N) a.dist[((size_t)split * a.B + b) * N + i] = mx;
}

// ---------------------------------------------------------------------------
// The picks: one workgroup per sample walks the K_d sequential steps with
// the distances of its tokens in registers (element e*1024 + t of thread t,
// as in the selection kernels), formed from the initial pass's per-split
// maxima.  Each step reduces (distance desc, index asc) over the unselected
// tokens, marks the winner, and lowers every distance with the winner's row
// of G.  The selected set (pivots and picks) is then written in ascending
// order.
// ---------------------------------------------------------------------------
template <int E>
__global__ __launch_bounds__(kSelThreads) void fps_pick_kernel(FpsArgs a) {
  __shared__ SelectShared sh;
  __shared__ float wv[2][kSelWaves];
  __shared__ int wi[2][kSelWaves];
  const int b = blockIdx.x, tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const int N = a.N, K_r = a.K_r;
  const int32_t* piv = a.pivots + (size_t)b * K_r;
  const float* gb = a.G + (size_t)b * N * N;
  auto valid = [&](int e) { return e * kSelThreads + tid < N; };
  // pivot membership: every thread marks its share of the pivot list in an
  // LDS bitmap, then reads the bits of its own elements
  __shared__ uint32_t pivbits[kMaxE * kSelThreads / 32];
  for (int w = tid; w < (N + 31) / 32; w += kSelThreads) pivbits[w] = 0u;
  float dist[E], iz[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int i = min(e * kSelThreads + tid, N - 1);
    float mx = a.dist[(size_t)b * N + i];
    for (int sp = 1; sp < a.n_psplit; ++sp) mx = fmaxf(mx, a.dist[((size_t)sp * a.B + b) * N + i]);
    iz[e] = a.inv_norm[(size_t)b * N + i];
    dist[e] = 1.f - mx * iz[e];
  }
  __syncthreads();
  for (int p = tid; p < K_r; p += kSelThreads) {
    const int j = min(max(piv[p], 0), N - 1);
    atomicOr(&pivbits[j >> 5], 1u << (j & 31));
  }
  __syncthreads();
  SelMask<E> sel = 0;  // bit e: element e is selected (a pivot or a pick)
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int i = e * kSelThreads + tid;
    if (valid(e) && ((pivbits[i >> 5] >> (i & 31)) & 1u)) sel |= SelMask<E>(1) << e;
  }
  // selected and padding elements hold distance -inf: they never win a step,
  // and the row updates (a minimum) keep them there, so neither the argmax
  // nor the update tests them
#pragma unroll
  for (int e = 0; e < E; ++e)
    if (!valid(e) || ((sel >> e) & 1u)) dist[e] = -INFINITY;
  for (int t = 0; t < a.K_d; ++t) {
    float v = -INFINITY;
    uint32_t idx = 0xffffffffu;
#pragma unroll
    for (int e = 0; e < E; ++e)
      if (dist[e] > v) {  // ascending e: the lower index wins ties
        v = dist[e];
        idx = (uint32_t)(e * kSelThreads + tid);
      }
    const float vm = wave_max(v);
    const uint32_t im = wave_min_u32(v == vm ? idx : 0xffffffffu);
    const int buf = t & 1;  // alternate slots: one barrier per step suffices
    if (lane == 0) {
      wv[buf][wave] = vm;
      wi[buf][wave] = (int)im;
    }
    __syncthreads();
    // every wave reduces the waves' winners itself (distance desc, index asc)
    const float v2 = lane < kSelWaves ? wv[buf][lane] : -INFINITY;
    const uint32_t i2 = lane < kSelWaves ? (uint32_t)wi[buf][lane] : 0xffffffffu;
    const float bv = wave_max(v2);
    int w = (int)wave_min_u32(v2 == bv ? i2 : 0xffffffffu);
    w = __builtin_amdgcn_readfirstlane(min(max(w, 0), N - 1));  // K_r + K_d <= N leaves a candidate
    if (tid == 0 && a.div_idx) a.div_idx[(size_t)b * a.K_d + t] = w;
    const int we = w / kSelThreads;
    const bool mine = (w & (kSelThreads - 1)) == tid;
    if (mine) sel |= SelMask<E>(1) << we;
#pragma unroll
    for (int e = 0; e < E; ++e)
      if (mine && e == we) dist[e] = -INFINITY;
    // the winner's row of G through a buffer resource: a uniform base and a
    // 32-bit offset per element (no 64-bit address per element), and the
    // elements past N read 0 (their distance is -inf already)
    const __amdgpu_buffer_rsrc_t row = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(gb + (size_t)w * N), 0, N * 4, kBufferRsrcWord3);
    const float izw = a.inv_norm[(size_t)b * N + w];
    // the row's loads go out before any is used, up to 16 at a time (one
    // round trip for N <= 16,384; 32 held values would spill)
    constexpr int CH = E < 16 ? E : 16;
#pragma unroll
    for (int c0 = 0; c0 < E; c0 += CH) {
      float gi[CH];
#pragma unroll
      for (int u = 0; u < CH; ++u)
        gi[u] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(row, ((c0 + u) * kSelThreads + tid) * 4, 0, 0));
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int u = 0; u < CH; ++u) {
        const float d = 1.f - gi[u] * iz[c0 + u] * izw;
        dist[c0 + u] = d < dist[c0 + u] ? d : dist[c0 + u];
      }
    }
  }
  block_write_mask<E>(sel, K_r + a.K_d, a.kept_idx + (size_t)b * (K_r + a.K_d), sh);
}

// ---------------------------------------------------------------- launchers
hipError_t launch_fps(const FpsArgs& f, const GramArgs& g, int dtype, int B, hipStream_t s) {
  // rows are a multiple of 16 bytes (checked at the boundary)
  if (dtype == 1 && g.N >= kGram256MinN && (size_t)(g.N + 256) * g.row_bytes < (1u << 31)) {
    GramArgs g2 = g;
    g2.n_tiles = (g.N + 255) / 256;
    const dim3 ggrid(gram_grid(g2.n_tiles, B));
    hipLaunchKernelGGL(gram256_kernel, ggrid, dim3(kGram256Threads), 0, s, g2);
  } else {
    const dim3 ggrid(gram_grid(g.n_tiles, B));
    if (dtype == 1)
      hipLaunchKernelGGL(gram_kernel<BF16>, ggrid, dim3(kGramThreads), 0, s, g);
    else
      hipLaunchKernelGGL(gram_kernel<F32>, ggrid, dim3(kGramThreads), 0, s, g);
  }
  hipLaunchKernelGGL(fps_init_kernel, dim3((f.N + kFpsInitThreads - 1) / kFpsInitThreads, B, f.n_psplit),
                     dim3(kFpsInitThreads), 0, s, f);
  const int E = select_e(f.N);
#define CALL(E_) hipLaunchKernelGGL(fps_pick_kernel<E_>, dim3(B), dim3(kSelThreads), 0, s, f)
  switch (E) {
    case 1: CALL(1); break;
    case 2: CALL(2); break;
    case 4: CALL(4); break;
    case 8: CALL(8); break;
    case 16: CALL(16); break;
    case 32: CALL(32); break;
    default: return hipErrorInvalidValue;
  }
#undef CALL
  return hipGetLastError();
}

}  // namespace trevs
