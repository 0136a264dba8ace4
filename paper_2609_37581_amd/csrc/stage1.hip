// Stage 1 (pre-LLM) kernels: [CLS] saliency, textual relevance, robust
// normalisation, fusion and pivot top-K (Sec. 4.1, Eq. (2)-(7)).
#include <algorithm>

#include "common.hpp"
#include "kernels.hpp"
#include "select.hpp"

namespace trevs {

// ---------------------------------------------------------------------------
// Prep.  Blocks [0, n_cls_blocks) take one ([CLS] head, segment) row each and
// reduce it in one pass to its softmax statistics (max and sum of exp, log2
// units, Eq. (2)); every later block takes 8 text rows, one per wave, and
// stores the inverse L2 norm of each (Sec. 4.1, before Eq. (4)).
// ---------------------------------------------------------------------------
constexpr int kPrepThreads = 512;

__device__ __forceinline__ void online_merge(float& m, float& s, float mo, float so) {
  const float mn = fmaxf(m, mo);
  if (mn == -INFINITY) return;
  s = s * __builtin_amdgcn_exp2f(m - mn) + so * __builtin_amdgcn_exp2f(mo - mn);
  m = mn;
}

template <class In>
__device__ __forceinline__ void online_vec(float& m, float& s, u32x4 w);
template <>
__device__ __forceinline__ void online_vec<BF16>(float& m, float& s, u32x4 w) {
  float x[8];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    x[2 * j] = bf16_lo(w[j]) * kLog2e;
    x[2 * j + 1] = bf16_hi(w[j]) * kLog2e;
  }
  float vm = x[0];
#pragma unroll
  for (int j = 1; j < 8; ++j) vm = fmaxf(vm, x[j]);
  const float mn = fmaxf(m, vm);
  float acc = s * __builtin_amdgcn_exp2f(m - mn);
#pragma unroll
  for (int j = 0; j < 8; ++j) acc += __builtin_amdgcn_exp2f(x[j] - mn);
  s = acc;
  m = mn;
}
template <>
__device__ __forceinline__ void online_vec<F32>(float& m, float& s, u32x4 w) {
  float x[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) x[j] = __uint_as_float(w[j]) * kLog2e;
  const float vm = fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3]));
  const float mn = fmaxf(m, vm);
  float acc = s * __builtin_amdgcn_exp2f(m - mn);
#pragma unroll
  for (int j = 0; j < 4; ++j) acc += __builtin_amdgcn_exp2f(x[j] - mn);
  s = acc;
  m = mn;
}

template <class In>
__global__ __launch_bounds__(kPrepThreads) void prep_kernel(PrepArgs a) {
  constexpr int NWV = kPrepThreads / 64;
  __shared__ float red_m[NWV], red_s[NWV];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if ((int)blockIdx.x < a.n_cls_blocks) {
    const int row = blockIdx.x;  // = (b*H + h)*n_seg + seg
    const int seg = row % a.n_seg, bh = row / a.n_seg;
    const size_t base = (size_t)bh * a.N + (size_t)seg * a.seg_len;
    float m = -INFINITY, s = 0.f;
    if (a.cls_vec16) {
      const uint8_t* p = reinterpret_cast<const uint8_t*>(a.cls) + base * In::kBytes;
      const int nvec = a.seg_len * In::kBytes / 16;
      for (int v = tid; v < nvec; v += 4 * kPrepThreads) {
        u32x4 w[4];
#pragma unroll
        for (int u = 0; u < 4; ++u)
          w[u] = v + u * kPrepThreads < nvec ? ldg16(p + (size_t)(v + u * kPrepThreads) * 16) : zero4();
#pragma unroll
        for (int u = 0; u < 4; ++u)
          if (v + u * kPrepThreads < nvec) online_vec<In>(m, s, w[u]);
      }
    } else {
      for (int i = tid; i < a.seg_len; i += kPrepThreads) {
        const float x = load_scalar(a.cls, base + i, In{}) * kLog2e;
        online_merge(m, s, x, 1.f);
      }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) online_merge(m, s, __shfl_xor(m, o, 64), __shfl_xor(s, o, 64));
    if (lane == 0) {
      red_m[wave] = m;
      red_s[wave] = s;
    }
    __syncthreads();
    if (tid == 0) {
      for (int w = 1; w < NWV; ++w) online_merge(m, s, red_m[w], red_s[w]);
      a.row_stats[row] = make_float2(m, 1.f / s);
    }
    return;
  }
  const int r = ((int)blockIdx.x - a.n_cls_blocks) * NWV + wave;  // = b*M_max + j
  if (r >= a.B * a.M_max) return;
  const int b = r / a.M_max, j = r - b * a.M_max;
  const int Mb = text_rows(a.text_len, b, a.M_max);
  float inv = 0.f;
  if (j < Mb) {
    const uint8_t* row = reinterpret_cast<const uint8_t*>(a.text) + (size_t)r * a.row_bytes;
    float s = 0.f;
    for (int off = lane * 16; off < a.row_bytes; off += 4 * 64 * 16) {
      u32x4 w[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) w[u] = off + u * 1024 < a.row_bytes ? ldg16(row + off + u * 1024) : zero4();
#pragma unroll
      for (int u = 0; u < 4; ++u) s += sumsq(w[u], In{});
    }
    s = wave_sum(s);
    inv = 1.f / fmaxf(sqrtf(s), 1e-12f);
  }
  if (lane == 0) a.inv_tnorm[r] = inv;
}

// Saliency (Eq. (2)-(3)) of the tokens [tok0, tok0 + VT) of sample b: the
// head mean of each [CLS] logit's softmax within its segment, from the
// per-(head, segment) max and 1/sum written by prep_kernel.  The head loop
// is unrolled by 8 with all loads of a group issued before the first use,
// so a tile pays about H/8 memory round trips instead of H.
template <class In>
__device__ __forceinline__ void tile_saliency(const RelArgs& a, int b, int tok0, int VT, int NT, int tid) {
  const int N = a.N, H = a.H;
  for (int t = tid; t < VT; t += NT) {
    const int i = tok0 + t;
    if (i < N) {
      const int seg = i / a.seg_len;
      float acc = 0.f;
      for (int h0 = 0; h0 < H; h0 += 8) {
        float2 st[8];
        float x[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int h = min(h0 + u, H - 1);
          st[u] = a.row_stats[((size_t)b * H + h) * a.n_seg + seg];
          x[u] = load_scalar(a.cls, ((size_t)b * H + h) * N + i, In{});
        }
#pragma unroll
        for (int u = 0; u < 8; ++u)
          if (h0 + u < H) acc = fmaf(__builtin_amdgcn_exp2f(fmaf(x[u], kLog2e, -st[u].x)), st[u].y, acc);
      }
      a.sal[(size_t)b * N + i] = acc / (float)H;
    }
  }
}

// ---------------------------------------------------------------------------
// Relevance: one pass over the visual features Z.  A workgroup owns 32*NW
// consecutive visual tokens of one sample; each wave owns 32 of them and
// computes C[text j][token i] = t_j . z_i on the matrix cores, streaming the
// feature dimension in slabs of SB bytes per row: the text slab goes through
// LDS (shared by the waves), each wave's Z rows go straight from HBM into
// registers.  Two register/LDS buffers alternate (A computes while B loads);
// every load is issued unconditionally (out-of-range lanes read an
// L2-resident dummy row and are masked where the data is used) so that the
// compiler can wait for exactly the older buffer.  The same Z registers give
// ||z_i||^2; the epilogue applies the norms, rectifies, squares and averages
// over the valid text rows (Eq. (4)-(5)).  The workgroup also finishes the
// head-mean saliency of its tokens from the prep statistics (Eq. (2)-(3)).
// ---------------------------------------------------------------------------
#ifndef TREVS_REL_NW
#define TREVS_REL_NW 4
#endif
#ifndef TREVS_REL_SB
#define TREVS_REL_SB 256
#endif
constexpr int kRelNW = TREVS_REL_NW;
constexpr int kRelSB = TREVS_REL_SB;

template <class In, int MT, int NW, int SB>
__global__ __launch_bounds__(64 * NW) void relevance_kernel(RelArgs a) {
  constexpr int MB = MT / 32;
  constexpr int NT = 64 * NW;
  constexpr int VT = 32 * NW;
  constexpr int NF = SB / 128;       // 64-byte fragments per lane per slab
  constexpr int HS = SB / 2;         // bytes of a slab row carried by one lane half
  constexpr int LROW = SB + 16;      // padded LDS row stride
  constexpr int CPR = SB / 16;       // 16-byte vectors per slab row
  constexpr int TV = MT * CPR;       // 16-byte vectors per text slab
  constexpr int TVT = (TV + NT - 1) / NT;
  __shared__ __attribute__((aligned(16))) uint8_t tlds[2][MT * LROW];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, col = lane & 31;
  const int tile = xcd_remap(blockIdx.x, gridDim.x);
  const int b = tile / a.tiles_per_sample;
  const int tok0 = (tile - b * a.tiles_per_sample) * VT;
  const int N = a.N, rb = a.row_bytes;
  const int Mb = text_rows(a.text_len, b, a.M_max);
  const int n_slabs = (rb + SB - 1) / SB;
  const int n_pairs = (n_slabs + 1) / 2;

  tile_saliency<In>(a, b, tok0, VT, NT, tid);

  const int tok = tok0 + wave * 32 + col;
  const bool tok_ok = tok < N;
  const uint8_t* tbase = reinterpret_cast<const uint8_t*>(a.T) + (size_t)b * a.M_max * rb;
  const uint8_t* dummy = tbase;  // always valid and hot in L2
  const uint8_t* zrow = reinterpret_cast<const uint8_t*>(a.Z) +
                        ((size_t)b * N + (tok_ok ? tok : N - 1)) * rb + half * HS;

  auto load_z = [&](int s, u32x4 (&dst)[NF][4]) {
#pragma unroll
    for (int f = 0; f < NF; ++f)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int off = s * SB + f * 64 + q * 16;
        dst[f][q] = ldg16_stream(off + half * HS < rb ? zrow + off : dummy);
      }
  };
  auto load_t = [&](int s, int j0, u32x4 (&dst)[TVT]) {
#pragma unroll
    for (int k = 0; k < TVT; ++k) {
      const int v = min(tid + k * NT, TV - 1), row = v / CPR, c = v - row * CPR;
      const int off = s * SB + c * 16;
      const bool ok = j0 + row < Mb && off < rb;
      dst[k] = ldg16(ok ? tbase + (size_t)(j0 + row) * rb + off : dummy);
    }
  };
  auto store_t = [&](int buf, int s, int j0, const u32x4 (&src)[TVT]) {
#pragma unroll
    for (int k = 0; k < TVT; ++k) {
      const int v = tid + k * NT;
      if (v < TV) {
        const int row = v / CPR, c = v - row * CPR;
        const bool ok = j0 + row < Mb && s * SB + c * 16 < rb;
        *reinterpret_cast<u32x4*>(&tlds[buf][row * LROW + c * 16]) = ok ? src[k] : zero4();
      }
    }
  };

  float zsq = 0.f, rsum = 0.f;
  for (int j0 = 0; j0 < Mb; j0 += MT) {
    f32x16 acc[MB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[mb][r] = 0.f;
    auto compute = [&](const u32x4 (&z)[NF][4], int buf, int s) {
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        const uint8_t* p = &tlds[buf][(mb * 32 + col) * LROW + half * HS];
#pragma unroll
        for (int f = 0; f < NF; ++f) {
          u32x4 af[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) af[q] = *reinterpret_cast<const u32x4*>(p + f * 64 + 16 * q);
          acc[mb] = mfma_frag(af, z[f], acc[mb], In{});
        }
      }
      if (j0 == 0) {
#pragma unroll
        for (int f = 0; f < NF; ++f)
#pragma unroll
          for (int q = 0; q < 4; ++q)
            zsq += (s * SB + half * HS + f * 64 + q * 16 < rb) ? sumsq(z[f][q], In{}) : 0.f;
      }
    };
    u32x4 zA[NF][4], zB[NF][4], tA[TVT], tB[TVT];
    load_t(0, j0, tA);
    load_z(0, zA);
    load_t(1, j0, tB);
    load_z(1, zB);
    store_t(0, 0, j0, tA);
    __syncthreads();
    for (int pr = 0; pr < n_pairs; ++pr) {
      const int s = 2 * pr;
      compute(zA, 0, s);
      store_t(1, s + 1, j0, tB);
      __syncthreads();
      load_t(s + 2, j0, tA);
      load_z(s + 2, zA);
      compute(zB, 1, s + 1);
      store_t(0, s + 2, j0, tA);
      __syncthreads();
      load_t(s + 3, j0, tB);
      load_z(s + 3, zB);
    }
    // ---- epilogue of this text chunk: sum_j max(t_j.z_i / ||t_j||, 0)^2
    const float* itn = a.inv_tnorm + (size_t)b * a.M_max;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      float w[16];  // every norm load before the first use
#pragma unroll
      for (int r = 0; r < 16; ++r) w[r] = itn[min(j0 + mb * 32 + mfma_row(r, half), a.M_max - 1)];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int j = j0 + mb * 32 + mfma_row(r, half);
        if (j < Mb) {
          const float c = fmaxf(acc[mb][r] * w[r], 0.f);
          rsum = fmaf(c, c, rsum);
        }
      }
    }
    __syncthreads();  // the next chunk refills both LDS buffers
  }
  const float zz = zsq + __shfl_xor(zsq, 32, 64);
  const float rr = rsum + __shfl_xor(rsum, 32, 64);
  const float iz = 1.f / fmaxf(sqrtf(zz), 1e-12f);
  if (half == 0 && tok_ok) a.rel[(size_t)b * N + tok] = sqrtf(rr * iz * iz / (float)Mb);
}

// ---------------------------------------------------------------------------
// Relevance, streaming variant for rows made of whole 128-byte slabs (text
// tiles of 32, 64 or 128 rows).  Same arithmetic as relevance_kernel; a
// workgroup of 4, 8 or 16 waves owns 256 tokens (12 waves own 192 tokens
// at 64 text rows).  Stage s is the 128-byte slab s of the tile's Z rows and
// of the MT text rows.  Every thread loads its share of a
// stage with coalesced 16-byte loads (8 lanes cover one 128-byte row
// segment) into a ring of R register buffers, so R stages are in flight; at
// each step the oldest buffer is written to one of two LDS buffers, the
// workgroup synchronises once, and the waves multiply the stage on the
// matrix cores (plain loads sustain a higher HBM rate on this chip than
// direct-to-LDS copies).  Rows are XOR-swizzled in 16-byte chunks so that
// both the stage writes and the MFMA fragment reads of 16 consecutive rows
// hit distinct banks.  Saliency (Eq. (2)-(3)) is computed while the first
// stages load.  With SPLIT the workgroup covers one range of slabs and
// writes raw partial products and ||z||^2 for relevance_merge_kernel.
// ---------------------------------------------------------------------------
constexpr int kStreamWaves = 8;
constexpr int kStreamTokens = 32 * kStreamWaves;
// register ring depth for text tiles of 128 and 64 rows
#ifndef TREVS_STREAM_R128
#define TREVS_STREAM_R128 2
#endif
#ifndef TREVS_STREAM_R64
#define TREVS_STREAM_R64 3
#endif
constexpr int kStreamR128 = TREVS_STREAM_R128, kStreamR64 = TREVS_STREAM_R64;
static_assert(kStreamR128 >= 2 && kStreamR128 <= 4 && kStreamR64 >= 2 && kStreamR64 <= 4,
              "register ring depth");

// Physical 16-byte chunk of logical chunk c in row r of a 128-byte slab row.
__device__ __forceinline__ int slab_swizzle(int r, int c) { return c ^ ((r >> 1) & 7); }

#ifndef TREVS_STREAM_TG128
#define TREVS_STREAM_TG128 2
#endif
#ifndef TREVS_STREAM_NW128
#define TREVS_STREAM_NW128 16
#endif
// Wave tiling of the stream kernel (VT = 32*VB tokens, MT text rows, NW
// waves): the waves form NTG token groups of 32*ZB tokens times TG text
// groups of MT/TG rows; wave w multiplies token group w % NTG against text
// group w / NTG.  Larger per-wave tiles read fewer fragment bytes from LDS
// per multiply (8 waves at 128 text rows: 64 x 64 tiles, 16 KB per wave and
// slab instead of 20 KB).  At 128 text rows the workgroup runs 16 waves
// (4 per SIMD, 32 x 64 tiles): with twice the waves of the 8-wave form each
// SIMD has work to issue while others wait on LDS or memory, and the kernel
// ran 6% faster at the 16,384-token workload (85 against 91 us).
// The 192-token tile (VB = 6, 64 text rows) runs 12 waves as 6 token groups
// times 2 text groups of 32 rows.
template <int MT, int NW, int VB = 8>
struct StreamTiling {
  static constexpr int TG = VB != 8 ? NW / VB : (NW == 16 ? 2 : (MT == 128 ? TREVS_STREAM_TG128 : 1));
  static constexpr int NTG = NW / TG;       // token groups
  static constexpr int ZB = VB / NTG;       // 32-token blocks per wave
  static constexpr int MBW = MT / 32 / TG;  // 32-row text blocks per wave
  static_assert(TG >= 1 && ZB >= 1 && NTG * ZB == VB && MBW * TG * 32 == MT, "stream tiling");
};

// (two waves per SIMD at four waves a workgroup: two workgroups per CU)
template <class In, int MT, int R, int NW, bool SPLIT, int VB = 8>
__global__ __launch_bounds__(64 * NW, NW == 4 ? 2 : 1) void relevance_stream_kernel(RelArgs a) {
  constexpr int NT = 64 * NW;
  constexpr int VT = 32 * VB;
  constexpr int TG = StreamTiling<MT, NW, VB>::TG;
  constexpr int ZB = StreamTiling<MT, NW, VB>::ZB;
  constexpr int MBW = StreamTiling<MT, NW, VB>::MBW;
  constexpr int NTG = StreamTiling<MT, NW, VB>::NTG;
  constexpr int ZBYTES = VT * 128;
  constexpr int STAGE = ZBYTES + MT * 128;
  constexpr int ZPT = ZBYTES / 16 / NT;        // Z chunks per thread per stage
  constexpr int TPT = (MT * 8 + NT - 1) / NT;  // text chunks per thread per stage
  constexpr bool TEXT_EXACT = TPT * NT == MT * 8;  // else the last chunks re-read text (not stored)
  constexpr int U = R % 2 ? 2 * R : R;         // steps per unrolled iteration
  static_assert(ZPT * NT * 16 == ZBYTES && (NT / 8) % 16 == 0, "stage split");
  __shared__ __attribute__((aligned(1024))) uint8_t l0[STAGE], l1[STAGE];
  __shared__ float tn[MT];
  __shared__ float rpart[TG][VT];  // per-text-group row sums of Eq. (5)

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, col = lane & 31;
  // the splits of one token tile are consecutive workgroups (one XCD, so
  // they share the text slabs in its L2)
  const int wid = xcd_remap(blockIdx.x, gridDim.x);
  const int tile = SPLIT ? wid / a.n_split : wid;
  const int split = SPLIT ? wid - tile * a.n_split : 0;
  const int b = tile / a.tiles_per_sample;
  const int tok0 = (tile - b * a.tiles_per_sample) * VT;
  const int N = a.N, rb = a.row_bytes;
  const int Mb = text_rows(a.text_len, b, a.M_max);
  const int s_begin = split * a.split_slabs;  // first slab of this split
  const int n_slabs = SPLIT ? min(rb >> 7, s_begin + a.split_slabs) - s_begin : rb >> 7;
  const int n_iter = (n_slabs + U - 1) / U;  // stages padded to the unroll

  const float* itn = a.inv_tnorm + (size_t)b * a.M_max;
  auto stage_norms = [&](int j0) {  // inverse text norms of a chunk, zero past the text
    if (tid < MT) tn[tid] = j0 + tid < Mb ? itn[j0 + tid] : 0.f;
  };

  // chunk k of this thread in a stage: row (tid / 8 + (NT / 8) k), chunk (tid % 8)
  const int cr = tid >> 3, cc = tid & 7;
  // (rows a multiple of 16 apart share the swizzle, so the LDS offsets
  // differ by (NT / 8) * 128 bytes)
  const uint8_t* zsrc[ZPT];
#pragma unroll
  for (int k = 0; k < ZPT; ++k) {
    const int r = cr + (NT / 8) * k;
    zsrc[k] = reinterpret_cast<const uint8_t*>(a.Z) + ((size_t)b * N + min(tok0 + r, N - 1)) * rb +
              s_begin * 128 + cc * 16;
  }
  const int sdst = cr * 128 + slab_swizzle(cr, cc) * 16;
  const uint8_t* tbase = reinterpret_cast<const uint8_t*>(a.T) + (size_t)b * a.M_max * rb;
  const int tgi = wave % NTG, xg = wave / NTG;  // token group, text group
  // this lane's Z rows in the stage (token block zb): tgi*32*ZB + zb*32 + col

  float zsq[ZB], rsum[ZB];
#pragma unroll
  for (int zb = 0; zb < ZB; ++zb) zsq[zb] = rsum[zb] = 0.f;
  for (int j0 = 0; j0 < Mb; j0 += MT) {
    const bool first = j0 == 0;
    if (!first && !SPLIT) {  // the previous chunk's epilogue has read its norms
      __syncthreads();
      stage_norms(j0);
    }
    const uint8_t* tsrc[TPT];
#pragma unroll
    for (int k = 0; k < TPT; ++k) {
      const int r = cr + (NT / 8) * k;
      tsrc[k] = tbase + (size_t)min(j0 + r, a.M_max - 1) * rb + s_begin * 128 + cc * 16;
    }
    // stage s into register buffer g; the padding stages past the last slab
    // re-read the last slab (still in L2) and are never multiplied
    u32x4 g[R][ZPT + TPT];
    auto load = [&](int s, u32x4 (&dst)[ZPT + TPT]) {
      const int off = min(s, n_slabs - 1) * 128;
#pragma unroll
      for (int k = 0; k < ZPT; ++k) dst[k] = ldg16_stream(zsrc[k] + off);
#pragma unroll
      for (int k = 0; k < TPT; ++k) dst[ZPT + k] = ldg16(tsrc[k] + off);
    };
    auto store = [&](uint8_t* st, const u32x4 (&src)[ZPT + TPT]) {
#pragma unroll
      for (int k = 0; k < ZPT; ++k) *reinterpret_cast<u32x4*>(st + sdst + k * (NT / 8) * 128) = src[k];
#pragma unroll
      for (int k = 0; k < TPT; ++k)
        if (TEXT_EXACT || cr + (NT / 8) * k < MT)
          *reinterpret_cast<u32x4*>(st + ZBYTES + sdst + k * (NT / 8) * 128) = src[ZPT + k];
    };
    f32x16 acc[ZB][MBW];
#pragma unroll
    for (int zb = 0; zb < ZB; ++zb)
#pragma unroll
      for (int mb = 0; mb < MBW; ++mb)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[zb][mb][r] = 0.f;
    auto compute = [&](const uint8_t* st) {
      u32x4 zf[ZB][4];
#pragma unroll
      for (int zb = 0; zb < ZB; ++zb) {
        const int zr = (tgi * ZB + zb) * 32 + col;
#pragma unroll
        for (int q = 0; q < 4; ++q)
          zf[zb][q] = *reinterpret_cast<const u32x4*>(st + zr * 128 + slab_swizzle(zr, 4 * half + q) * 16);
      }
      if (j0 == 0 && xg == 0) {  // ||z||^2 once per token
#pragma unroll
        for (int zb = 0; zb < ZB; ++zb)
#pragma unroll
          for (int q = 0; q < 4; ++q) zsq[zb] += sumsq(zf[zb][q], In{});
      }
#pragma unroll
      for (int mb = 0; mb < MBW; ++mb) {
        const int row = (xg * MBW + mb) * 32 + col;
        u32x4 af[4];
#pragma unroll
        for (int q = 0; q < 4; ++q)
          af[q] = *reinterpret_cast<const u32x4*>(st + ZBYTES + row * 128 + slab_swizzle(row, 4 * half + q) * 16);
#pragma unroll
        for (int zb = 0; zb < ZB; ++zb) acc[zb][mb] = mfma_frag(af, zf[zb], acc[zb][mb], In{});
      }
    };
#pragma unroll
    for (int c = 0; c < R; ++c) load(c, g[c]);
    if (first) {
      if (split == 0) tile_saliency<In>(a, b, tok0, VT, NT, tid);
      if (!SPLIT) stage_norms(0);
    }
    for (int it = 0; it < n_iter; ++it) {
#pragma unroll
      for (int c = 0; c < U; ++c) {
        const int s = it * U + c;
        uint8_t* st = c % 2 ? l1 : l0;
        // buffer (s % 2) was last read at step s - 2, before every wave
        // passed the barrier of step s - 1
        store(st, g[c % R]);
        load(s + R, g[c % R]);
        __syncthreads();
        if (s < n_slabs) compute(st);
      }
    }
    __syncthreads();  // the LDS buffers are refilled by the next text chunk
    if constexpr (SPLIT) {  // partial products of the valid rows; 32 lanes write 128 bytes
      float* pp = a.part + (size_t)(b * a.n_split + split) * a.M_max * N;
#pragma unroll
      for (int zb = 0; zb < ZB; ++zb) {
        const int t = tok0 + (tgi * ZB + zb) * 32 + col;
#pragma unroll
        for (int mb = 0; mb < MBW; ++mb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int j = j0 + (xg * MBW + mb) * 32 + mfma_row(r, half);
            if (j < Mb && t < N) pp[(size_t)j * N + t] = acc[zb][mb][r];
          }
      }
      continue;
    }
    // ---- epilogue of this text chunk: sum_j max(t_j.z_i / ||t_j||, 0)^2
    // (the staged norm is zero for rows past the text, which drops them)
#pragma unroll
    for (int zb = 0; zb < ZB; ++zb)
#pragma unroll
      for (int mb = 0; mb < MBW; ++mb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float c = fmaxf(acc[zb][mb][r] * tn[(xg * MBW + mb) * 32 + mfma_row(r, half)], 0.f);
          rsum[zb] = fmaf(c, c, rsum[zb]);
        }
  }
  if constexpr (SPLIT) {
    if (xg == 0)
#pragma unroll
      for (int zb = 0; zb < ZB; ++zb) {
        const int t = tok0 + (tgi * ZB + zb) * 32 + col;
        const float zz = zsq[zb] + __shfl_xor(zsq[zb], 32, 64);
        if (half == 0 && t < N) a.zpart[(size_t)(b * a.n_split + split) * N + t] = zz;
      }
    return;
  }
  // row sums of the text groups meet in LDS (a fixed order of additions)
#pragma unroll
  for (int zb = 0; zb < ZB; ++zb) {
    const float rr = rsum[zb] + __shfl_xor(rsum[zb], 32, 64);
    if (half == 0) rpart[xg][(tgi * ZB + zb) * 32 + col] = rr;
  }
  __syncthreads();
  if (xg == 0) {
#pragma unroll
    for (int zb = 0; zb < ZB; ++zb) {
      const int t = (tgi * ZB + zb) * 32 + col;
      float rr = rpart[0][t];
#pragma unroll
      for (int x = 1; x < TG; ++x) rr += rpart[x][t];
      const float zz = zsq[zb] + __shfl_xor(zsq[zb], 32, 64);
      const float iz = 1.f / fmaxf(sqrtf(zz), 1e-12f);
      if (half == 0 && tok0 + t < N) a.rel[(size_t)b * N + tok0 + t] = sqrtf(rr * iz * iz / (float)Mb);
    }
  }
}

// ---------------------------------------------------------------------------
// Relevance merge after a feature-dimension split: a workgroup owns 32
// tokens of one sample, thread (g, t) the text rows g, g + 32, ... of token
// t.  It adds the n_split partial products of each row in split order,
// applies the inverse text norm, rectifies and squares (Eq. (4)); the row
// sums meet in LDS and the first row group divides by ||z_i||^2 (summed over
// the splits) and by the text length (Eq. (5)).
// ---------------------------------------------------------------------------
constexpr int kMergeTokens = 32, kMergeGroups = 32;

// (64 registers: two workgroups per CU)
__global__ __launch_bounds__(kMergeTokens * kMergeGroups, 8) void relevance_merge_kernel(RelArgs a) {
  __shared__ float red[kMergeGroups][kMergeTokens + 1], zred[kMergeGroups][kMergeTokens + 1];
  const int t = threadIdx.x % kMergeTokens, g = threadIdx.x / kMergeTokens;
  const int b = blockIdx.y, N = a.N, S = a.n_split;
  const int i = blockIdx.x * kMergeTokens + t, ic = min(i, N - 1);
  const int Mb = text_rows(a.text_len, b, a.M_max);
  // uniform split base plus a 32-bit lane offset: the loads take their
  // address from scalar registers
  const size_t sstride = (size_t)a.M_max * N;
  const float* pb = a.part + (size_t)b * S * sstride;
  const float* itn = a.inv_tnorm + (size_t)b * a.M_max;
  float r = 0.f;
  for (int j = g; j < Mb; j += kMergeGroups) {
    const int off = j * N + ic;
    float c = 0.f;
    for (int s0 = 0; s0 < S; s0 += 16) {  // 16 loads in flight, added in split order
      float v[16];
#pragma unroll
      for (int k = 0; k < 16; ++k) v[k] = pb[min(s0 + k, S - 1) * sstride + off];
#pragma unroll
      for (int k = 0; k < 16; ++k) c += s0 + k < S ? v[k] : 0.f;
    }
    c = fmaxf(c * itn[j], 0.f);
    r = fmaf(c, c, r);
  }
  float z = 0.f;  // ||z_i||^2: split sp goes to row group sp % 32
  const float* zb = a.zpart + (size_t)b * S * N;
  for (int sp = g; sp < S; sp += kMergeGroups) z += zb[(size_t)sp * N + ic];
  red[g][t] = r;
  zred[g][t] = z;
  __syncthreads();
  if (g == 0 && i < N) {
    float rr = red[0][t], zz = zred[0][t];
#pragma unroll 4
    for (int x = 1; x < kMergeGroups; ++x) {
      rr += red[x][t];
      zz += zred[x][t];
    }
    const float iz = 1.f / fmaxf(sqrtf(zz), 1e-12f);
    a.rel[(size_t)b * N + i] = sqrtf(rr * iz * iz / (float)Mb);
  }
}

// ---------------------------------------------------------------------------
// Robust statistics: one workgroup per (branch, sample), branch 0 = s^v,
// branch 1 = s^t.  Lower median and MAD as exact order statistics (Eq. (6)).
// ---------------------------------------------------------------------------
template <int E>
__global__ __launch_bounds__(kSelThreads) void norm_stats_kernel(NormArgs a) {
  __shared__ SelectShared sh;
  __shared__ float red_lo[kSelWaves], red_hi[kSelWaves];
  const int branch = blockIdx.x, b = blockIdx.y, tid = threadIdx.x, N = a.N;
  const float* src = (branch ? a.rel : a.sal) + (size_t)b * N;
  float x[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int i = e * kSelThreads + tid;
    x[e] = i < N ? src[i] : 0.f;
  }
  // min and max of the scores, then the median
  float lo = INFINITY, hi = -INFINITY;
#pragma unroll
  for (int e = 0; e < E; ++e)
    if (e * kSelThreads + tid < N) {
      lo = fminf(lo, x[e]);
      hi = fmaxf(hi, x[e]);
    }
  lo = -wave_max(-lo);
  hi = wave_max(hi);
  if ((tid & 63) == 0) {
    red_lo[tid >> 6] = lo;
    red_hi[tid >> 6] = hi;
  }
  __syncthreads();
  lo = INFINITY;
  hi = -INFINITY;
#pragma unroll
  for (int w = 0; w < kSelWaves; ++w) {
    lo = fminf(lo, red_lo[w]);
    hi = fmaxf(hi, red_hi[w]);
  }
  const int rmed = (N - 1) / 2;
  uint32_t k;
  int less, eq;
  block_select<E>([&](int e) { return f2key(x[e]); }, N, rmed, k, less, eq, sh, true, f2key(lo),
                  f2key(hi));
  const float med = key2f(k);
  // the deviations |x - Med| range from 0 (the median itself) to the larger
  // distance of the extremes, computed with the same fp32 operation
  block_select<E>([&](int e) { return f2key(fabsf(x[e] - med)); }, N, rmed, k, less, eq, sh, true,
                  f2key(0.f), f2key(fmaxf(fabsf(lo - med), fabsf(hi - med))));
  if (tid == 0) {
    a.stats[4 * b + 2 * branch] = med;
    a.stats[4 * b + 2 * branch + 1] = key2f(k);
  }
}

// ---------------------------------------------------------------------------
// Fusion and pivot selection: one workgroup per sample.  Normalised scores
// with temperature (Eq. (6)), branch weights and the consistency reward
// (Eq. (7)), then the stable top-K.
// ---------------------------------------------------------------------------
template <int E>
__global__ __launch_bounds__(kSelThreads) void fuse_topk_kernel(SelArgs a) {
  __shared__ SelectShared sh;
  const int b = blockIdx.x, tid = threadIdx.x, N = a.N;
  const float* sv_p = a.sal + (size_t)b * N;
  const float* st_p = a.rel + (size_t)b * N;
  const float med_v = a.stats[4 * b + 0], mad_v = a.stats[4 * b + 1];
  const float med_t = a.stats[4 * b + 2], mad_t = a.stats[4 * b + 3];
  // one workgroup holds a whole sample, so the per-token arithmetic is kept
  // to multiplies: the branch weight, 1/(MAD + eps) and 1/tau are folded into
  // one factor per branch, and the square root is the hardware one (a few
  // ulp from the exactly rounded expression of Eq. (6)-(7))
  const float cv = a.wv / ((mad_v + a.eps) * a.tau_v);
  const float ct = a.wt / ((mad_t + a.eps) * a.tau_t);
  // every load before the first store: a store to score_out may alias the
  // inputs as far as the compiler knows, which would serialise the loads
  float sv[E], st[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int i = min(e * kSelThreads + tid, N - 1);
    sv[e] = sv_p[i];
    st[e] = st_p[i];
  }
  float sc[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const float dv = fmaxf(sv[e] - med_v, 0.f), dt = fmaxf(st[e] - med_t, 0.f);
    const float av = dv > 0.f ? dv * cv : 0.f;  // clamped tokens stay exactly 0
    const float bt = dt > 0.f ? dt * ct : 0.f;
    sc[e] = e * kSelThreads + tid < N ? fmaxf(av, bt) + a.lam * __builtin_amdgcn_sqrtf(av * bt) : 0.f;
  }
  if (a.score_out) {
#pragma unroll
    for (int e = 0; e < E; ++e)
      if (e * kSelThreads + tid < N) a.score_out[(size_t)b * N + e * kSelThreads + tid] = sc[e];
  }
  if (a.norm_stats && tid < 4) a.norm_stats[4 * b + tid] = a.stats[4 * b + tid];
  // with lam >= 0 every score is a sum of non-negative terms, so the keys lie
  // in [key(+0), 0xffffffff] and the selection needs no min/max reduction
  // (the bound spans the same 31 bits as the exact range once any score is 0)
  block_topk_write<E>(sc, N, a.K, a.kept_idx + (size_t)b * a.K, sh, a.lam >= 0.f, f2key(0.f),
                      0xffffffffu);
}

// ---------------------------------------------------------------------------
// Budget-split selection: one workgroup per sample.  The textual ratio read
// as the share of the token budget given to textual relevance (the analysis
// of Sec. 3): the K_t tokens with the highest s^t, then the K - K_t tokens
// with the highest s^v among the rest (both stable: score descending, lower
// index first), kept in ascending order.  Tokens already taken get the
// smallest key in the second selection, below every finite score.
// ---------------------------------------------------------------------------
template <int E>
__global__ __launch_bounds__(kSelThreads) void budget_topk_kernel(SelArgs a) {
  __shared__ SelectShared sh;
  const int b = blockIdx.x, tid = threadIdx.x, N = a.N;
  float sv[E], st[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int i = min(e * kSelThreads + tid, N - 1);  // out-of-range elements are never valid below
    sv[e] = a.sal[(size_t)b * N + i];
    st[e] = a.rel[(size_t)b * N + i];
  }
  const SelMask<E> by_text = block_topk_mask<E>([&](int e) { return f2key(st[e]); }, N, a.K_t, sh);
  const SelMask<E> by_sal = block_topk_mask<E>(
      [&](int e) { return (by_text >> e) & 1u ? 0u : f2key(sv[e]); }, N, a.K - a.K_t, sh);
  block_write_mask<E>(by_text | by_sal, a.K, a.kept_idx + (size_t)b * a.K, sh);
}

template <int E>
__global__ __launch_bounds__(kSelThreads) void topk_kernel(const float* scores, int N, int K,
                                                           int32_t* out, bool nonneg) {
  __shared__ SelectShared sh;
  const int b = blockIdx.x, tid = threadIdx.x;
  const float* p = scores + (size_t)b * N;
  float sc[E];
#pragma unroll
  for (int e = 0; e < E; ++e) sc[e] = p[min(e * kSelThreads + tid, N - 1)];  // unconditional loads
#pragma unroll
  for (int e = 0; e < E; ++e)
    if (e * kSelThreads + tid >= N) sc[e] = 0.f;
  // scores known to be >= 0 bound the keys by [key(+0), 0xffffffff]: no min/max reduction
  block_topk_write<E>(sc, N, K, out + (size_t)b * K, sh, nonneg, f2key(0.f), 0xffffffffu);
}

// ---------------------------------------------------------------- launchers
hipError_t launch_prep(const PrepArgs& a, int dtype, hipStream_t s) {
  const int rows_per_block = kPrepThreads / 64;
  const int text_blocks = (a.B * a.M_max + rows_per_block - 1) / rows_per_block;
  const dim3 grid(a.n_cls_blocks + text_blocks);
  if (dtype == 1)
    hipLaunchKernelGGL(prep_kernel<BF16>, grid, dim3(kPrepThreads), 0, s, a);
  else
    hipLaunchKernelGGL(prep_kernel<F32>, grid, dim3(kPrepThreads), 0, s, a);
  return hipGetLastError();
}

// Feature-dimension split.  The stream kernel keeps one workgroup per CU at
// text tiles of 64 or 128 rows and two at 32 rows; a grid with fewer token
// tiles than half of that resident capacity (256 CUs) leaves compute units
// idle, so each tile is split along the feature dimension into as many
// slab ranges as kSplitRounds resident rounds hold, keeping at least
// kSplitMinSlabs 128-byte slabs per range.  The partial products cost 8
// bytes per (text row, token, split) of extra traffic plus a merge pass, which
// pays only while compute units would otherwise stand idle.
#ifndef TREVS_REL_SPLIT_ROUNDS
#define TREVS_REL_SPLIT_ROUNDS 1
#endif
#ifndef TREVS_REL_SPLIT_MIN_SLABS
#define TREVS_REL_SPLIT_MIN_SLABS 4
#endif
#ifndef TREVS_STREAM_R32
#define TREVS_STREAM_R32 2
#endif
constexpr int kNumCUs = 256;
constexpr int kTile192 = 192;  // 64 text rows: 12 waves, VB = 6
constexpr int kSplitRounds = TREVS_REL_SPLIT_ROUNDS, kSplitMinSlabs = TREVS_REL_SPLIT_MIN_SLABS;
constexpr size_t kSplitMaxBytes = size_t(256) << 20;  // cap on the partial products
constexpr int kStreamR32 = TREVS_STREAM_R32;

size_t RelPlan::part_floats() const {
  return n_split > 1 ? (size_t)n_split * B * ((size_t)M_max + 1) * N : 0;
}

RelPlan relevance_plan(int B, int N, int M_max, int row_bytes) {
  RelPlan p;
  p.B = B;
  p.N = N;
  p.M_max = M_max;
  p.MT = M_max <= 32 ? 32 : (M_max <= 64 ? 64 : 128);
  p.stream = row_bytes % 128 == 0;
  p.tile_tokens = p.stream ? kStreamTokens : 32 * kRelNW;
  p.tiles_per_sample = (N + p.tile_tokens - 1) / p.tile_tokens;
  p.n_split = 1;
  p.split_slabs = row_bytes / 128;
  const long tiles = (long)B * p.tiles_per_sample;
  const long resident = (long)kNumCUs * (p.MT == 32 ? 2 : 1);
  // At 64 text rows a 192-token tile is taken when it streams fewer rows per
  // CU (tile rows times resident rounds): 576 = 3 x 192 tokens leave no
  // half-empty tile, and LLaVA-1.5 batch 64 ran 74.6 -> 69.0 us.
  if (p.stream && p.MT == 64 && 2 * tiles > resident) {
    const long t192 = (long)B * ((N + kTile192 - 1) / kTile192);
    const long rows256 = kStreamTokens * ((tiles + resident - 1) / resident);
    const long rows192 = kTile192 * ((t192 + resident - 1) / resident);
    if (rows192 < rows256) {
      p.tile_tokens = kTile192;
      p.tiles_per_sample = (N + kTile192 - 1) / kTile192;
    }
  }
  if (p.stream && 2 * tiles <= resident) {
    const int slabs = row_bytes / 128;
    const int want = (int)std::min<long>(kSplitRounds * resident / tiles, std::max(slabs / kSplitMinSlabs, 1));
    if (want > 1) {
      p.split_slabs = (slabs + want - 1) / want;
      p.n_split = (slabs + p.split_slabs - 1) / p.split_slabs;
      if (p.part_floats() * sizeof(float) > kSplitMaxBytes) {  // very long texts: no split
        p.n_split = 1;
        p.split_slabs = slabs;
      }
    }
  }
  return p;
}

template <class In>
static void launch_rel_t(const RelArgs& a, int MT, hipStream_t s) {
  const dim3 grid(a.B * a.tiles_per_sample), block(64 * kRelNW);
  if (MT == 32)
    hipLaunchKernelGGL((relevance_kernel<In, 32, kRelNW, kRelSB>), grid, block, 0, s, a);
  else if (MT == 64)
    hipLaunchKernelGGL((relevance_kernel<In, 64, kRelNW, kRelSB>), grid, block, 0, s, a);
  else
    hipLaunchKernelGGL((relevance_kernel<In, 128, kRelNW, kRelSB>), grid, block, 0, s, a);
}

template <class In, bool SPLIT>
static void launch_rel_stream_t(const RelArgs& a, const RelPlan& p, hipStream_t s) {
  const dim3 grid(a.B * a.tiles_per_sample * a.n_split);
  constexpr int NW128 = TREVS_STREAM_NW128;
  const int MT = p.MT;
  if constexpr (!SPLIT) {  // the split runs on 256-token tiles only
    if (MT == 64 && p.tile_tokens == kTile192) {
      hipLaunchKernelGGL((relevance_stream_kernel<In, 64, 2, 12, false, 6>), grid, dim3(64 * 12), 0, s, a);
      return;
    }
  }
  if (MT == 32)
    hipLaunchKernelGGL((relevance_stream_kernel<In, 32, kStreamR32, 4, SPLIT>), grid, dim3(64 * 4), 0, s, a);
  else if (MT == 64)
    hipLaunchKernelGGL((relevance_stream_kernel<In, 64, kStreamR64, kStreamWaves, SPLIT>), grid,
                       dim3(64 * kStreamWaves), 0, s, a);
  else
    hipLaunchKernelGGL((relevance_stream_kernel<In, 128, kStreamR128, NW128, SPLIT>), grid,
                       dim3(64 * NW128), 0, s, a);
}

hipError_t launch_relevance(const RelArgs& a, const RelPlan& p, int dtype, hipStream_t s) {
  if (!p.stream) {
    if (dtype == 1)
      launch_rel_t<BF16>(a, p.MT, s);
    else
      launch_rel_t<F32>(a, p.MT, s);
    return hipGetLastError();
  }
  if (p.n_split > 1) {
    if (dtype == 1)
      launch_rel_stream_t<BF16, true>(a, p, s);
    else
      launch_rel_stream_t<F32, true>(a, p, s);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const dim3 grid((a.N + kMergeTokens - 1) / kMergeTokens, a.B);
    hipLaunchKernelGGL(relevance_merge_kernel, grid, dim3(kMergeTokens * kMergeGroups), 0, s, a);
  } else if (dtype == 1) {
    launch_rel_stream_t<BF16, false>(a, p, s);
  } else {
    launch_rel_stream_t<F32, false>(a, p, s);
  }
  return hipGetLastError();
}


#define TREVS_SELECT_SWITCH(E_, CALL)   \
  switch (E_) {                         \
    case 1: CALL(1); break;             \
    case 2: CALL(2); break;             \
    case 4: CALL(4); break;             \
    case 8: CALL(8); break;             \
    case 16: CALL(16); break;           \
    case 32: CALL(32); break;           \
    case 64: CALL(64); break;           \
    default: return hipErrorInvalidValue; \
  }

hipError_t launch_norm_stats(const NormArgs& a, int B, hipStream_t s) {
#define CALL(E) hipLaunchKernelGGL(norm_stats_kernel<E>, dim3(2, B), dim3(kSelThreads), 0, s, a)
  TREVS_SELECT_SWITCH(select_e(a.N), CALL)
#undef CALL
  return hipGetLastError();
}

hipError_t launch_prellm_select(const SelArgs& a, int B, hipStream_t s) {
#define CALL(E) hipLaunchKernelGGL(fuse_topk_kernel<E>, dim3(B), dim3(kSelThreads), 0, s, a)
  TREVS_SELECT_SWITCH(select_e(a.N), CALL)
#undef CALL
  return hipGetLastError();
}

hipError_t launch_budget_select(const SelArgs& a, int B, hipStream_t s) {
#define CALL(E) hipLaunchKernelGGL(budget_topk_kernel<E>, dim3(B), dim3(kSelThreads), 0, s, a)
  TREVS_SELECT_SWITCH(select_e(a.N), CALL)
#undef CALL
  return hipGetLastError();
}

hipError_t launch_topk(const float* scores, int B, int N, int K, int32_t* out, hipStream_t s,
                       bool nonneg) {
#define CALL(E) hipLaunchKernelGGL(topk_kernel<E>, dim3(B), dim3(kSelThreads), 0, s, scores, N, K, out, nonneg)
  TREVS_SELECT_SWITCH(select_e(N), CALL)
#undef CALL
  return hipGetLastError();
}

}  // namespace trevs
