// Stage 1 (pre-LLM) kernels: [CLS] saliency, textual relevance, robust
// normalisation, fusion and pivot top-K (Sec. 4.1, Eq. (2)-(7)).
#include "common.hpp"
#include "kernels.hpp"
#include "select.hpp"

namespace trevs {

// ---------------------------------------------------------------------------
// Prep: per ([CLS] head, segment) softmax statistics, and per text row the
// inverse L2 norm.  Blocks [0, n_cls_blocks) take one [CLS] row each; every
// later block takes 4 text rows, one per wave.
// ---------------------------------------------------------------------------
template <class In>
__global__ __launch_bounds__(256) void prep_kernel(PrepArgs a) {
  __shared__ float red[4];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if ((int)blockIdx.x < a.n_cls_blocks) {
    const int row = blockIdx.x;  // = (b*H + h)*n_seg + seg
    const int seg = row % a.n_seg, bh = row / a.n_seg;
    const size_t base = (size_t)bh * a.N + (size_t)seg * a.seg_len;
    float m = -INFINITY;
    for (int i = tid; i < a.seg_len; i += 256) m = fmaxf(m, load_scalar(a.cls, base + i, In{}));
    m = wave_max(m);
    if (lane == 0) red[wave] = m;
    __syncthreads();
    m = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3])) * kLog2e;
    __syncthreads();
    float s = 0.f;
    for (int i = tid; i < a.seg_len; i += 256)
      s += exp2f(fmaf(load_scalar(a.cls, base + i, In{}), kLog2e, -m));
    s = wave_sum(s);
    if (lane == 0) red[wave] = s;
    __syncthreads();
    if (tid == 0) a.row_stats[row] = make_float2(m, 1.f / ((red[0] + red[1]) + (red[2] + red[3])));
    return;
  }
  const int r = ((int)blockIdx.x - a.n_cls_blocks) * 4 + wave;  // = b*M_max + j
  if (r >= a.B * a.M_max) return;
  const int b = r / a.M_max, j = r - b * a.M_max;
  const int Mb = a.text_len ? a.text_len[b] : a.M_max;
  float inv = 0.f;
  if (j < Mb) {
    const uint8_t* row = reinterpret_cast<const uint8_t*>(a.text) + (size_t)r * a.row_bytes;
    float s = 0.f;
    for (int off = lane * 16; off < a.row_bytes; off += 64 * 16) s += sumsq(ldg16(row + off), In{});
    s = wave_sum(s);
    inv = 1.f / fmaxf(sqrtf(s), 1e-12f);
  }
  if (lane == 0) a.inv_tnorm[r] = inv;
}

// ---------------------------------------------------------------------------
// Relevance: one pass over the visual features Z.  A workgroup owns VT
// consecutive visual tokens of one sample; each wave owns NB blocks of 32
// tokens and computes C[text j][token i] = t_j . z_i on the matrix cores
// (text tile from LDS, Z straight from HBM into registers, 128-byte row
// slabs double buffered).  The same Z registers give ||z_i||^2; the epilogue
// applies the norms, rectifies, squares and averages over the valid text
// rows (Eq. (4)-(5)).  The workgroup also finishes the head-mean saliency of
// its tokens from the prep statistics (Eq. (2)-(3)).
// ---------------------------------------------------------------------------
constexpr int kRelNB = 1;
constexpr int kRelNW = 4;
constexpr int kLdsRow = 128 + 16;  // padded LDS row stride (bytes) of a 128-byte text slab row

template <class In, int MT, int NB, int NW>
__global__ __launch_bounds__(64 * NW) void relevance_kernel(RelArgs a) {
  constexpr int MB = MT / 32;
  constexpr int NT = 64 * NW;
  constexpr int VT = 32 * NB * NW;
  constexpr int TV = MT * 8;  // 16-byte vectors in one text slab
  constexpr int TVT = (TV + NT - 1) / NT;
  __shared__ __attribute__((aligned(16))) uint8_t tlds[2][MT * kLdsRow];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, col = lane & 31;
  const int tile = xcd_remap(blockIdx.x, gridDim.x);
  const int b = tile / a.tiles_per_sample;
  const int tok0 = (tile - b * a.tiles_per_sample) * VT;
  const int N = a.N, rb = a.row_bytes;
  const int Mb = a.text_len ? a.text_len[b] : a.M_max;
  const int n_slabs = (rb + 127) >> 7;

  // ---- saliency of this tile's tokens
  for (int t = tid; t < VT; t += NT) {
    const int i = tok0 + t;
    if (i < N) {
      const int seg = i / a.seg_len;
      float acc = 0.f;
      for (int h = 0; h < a.H; ++h) {
        const float2 st = a.row_stats[((size_t)b * a.H + h) * a.n_seg + seg];
        const float x = load_scalar(a.cls, ((size_t)b * a.H + h) * N + i, In{});
        acc = fmaf(exp2f(fmaf(x, kLog2e, -st.x)), st.y, acc);
      }
      a.sal[(size_t)b * N + i] = acc / (float)a.H;
    }
  }

  // ---- visual rows carried by this lane
  const uint8_t* zrow[NB];
  bool zvalid[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int i = tok0 + (wave * NB + nb) * 32 + col;
    zvalid[nb] = i < N;
    zrow[nb] = reinterpret_cast<const uint8_t*>(a.Z) + ((size_t)b * N + (zvalid[nb] ? i : N - 1)) * rb +
               half * 64;
  }
  const uint8_t* tbase = reinterpret_cast<const uint8_t*>(a.T) + (size_t)b * a.M_max * rb;

  auto load_z = [&](int s, u32x4 (&dst)[NB][4]) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int off = s * 128 + q * 16;
        dst[nb][q] = (off + half * 64 < rb) ? ldg16_stream(zrow[nb] + off) : zero4();
      }
  };
  auto load_t = [&](int s, int j0, u32x4 (&dst)[TVT]) {
#pragma unroll
    for (int k = 0; k < TVT; ++k) {
      const int v = tid + k * NT, row = v >> 3, c = v & 7;
      const int off = s * 128 + c * 16;
      dst[k] = (v < TV && j0 + row < Mb && off < rb) ? ldg16(tbase + (size_t)(j0 + row) * rb + off)
                                                     : zero4();
    }
  };
  auto store_t = [&](int buf, const u32x4 (&src)[TVT]) {
#pragma unroll
    for (int k = 0; k < TVT; ++k) {
      const int v = tid + k * NT, row = v >> 3, c = v & 7;
      if (v < TV) *reinterpret_cast<u32x4*>(&tlds[buf][row * kLdsRow + c * 16]) = src[k];
    }
  };

  float zsq[NB], rsum[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) zsq[nb] = rsum[nb] = 0.f;

  for (int j0 = 0; j0 < Mb; j0 += MT) {
    f32x16 acc[MB][NB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[mb][nb][r] = 0.f;
    u32x4 zc[NB][4], zn[NB][4], tv[TVT];
    load_t(0, j0, tv);
    load_z(0, zc);
    store_t(0, tv);
    __syncthreads();
    for (int s = 0; s < n_slabs; ++s) {
      const bool more = s + 1 < n_slabs;
      if (more) {
        load_z(s + 1, zn);
        load_t(s + 1, j0, tv);
      }
      const uint8_t* buf = tlds[s & 1];
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        u32x4 af[4];
        const uint8_t* p = buf + (mb * 32 + col) * kLdsRow + half * 64;
#pragma unroll
        for (int q = 0; q < 4; ++q) af[q] = *reinterpret_cast<const u32x4*>(p + 16 * q);
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) acc[mb][nb] = mfma_frag(af, zc[nb], acc[mb][nb], In{});
      }
      if (j0 == 0) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
          for (int q = 0; q < 4; ++q) zsq[nb] += sumsq(zc[nb][q], In{});
      }
      if (more) store_t((s + 1) & 1, tv);
      __syncthreads();
      if (more) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
          for (int q = 0; q < 4; ++q) zc[nb][q] = zn[nb][q];
      }
    }
    // ---- epilogue of this text chunk: sum_j max(t_j.z_i / ||t_j||, 0)^2
    const float* itn = a.inv_tnorm + (size_t)b * a.M_max;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int j = j0 + mb * 32 + mfma_row(r, half);
        if (j < Mb) {
          const float it = itn[j];
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) {
            const float c = fmaxf(acc[mb][nb][r] * it, 0.f);
            rsum[nb] = fmaf(c, c, rsum[nb]);
          }
        }
      }
  }
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const float zz = zsq[nb] + __shfl_xor(zsq[nb], 32, 64);
    const float rr = rsum[nb] + __shfl_xor(rsum[nb], 32, 64);
    const float iz = 1.f / fmaxf(sqrtf(zz), 1e-12f);
    const int i = tok0 + (wave * NB + nb) * 32 + col;
    if (half == 0 && zvalid[nb]) a.rel[(size_t)b * N + i] = sqrtf(rr * iz * iz / (float)Mb);
  }
}

// ---------------------------------------------------------------------------
// Select: one workgroup per sample.  Lower medians and MADs of s^v and s^t
// (Eq. (6)), the fused score (Eq. (7)) and its stable top-K.
// ---------------------------------------------------------------------------
template <int E>
__global__ __launch_bounds__(kSelThreads) void prellm_select_kernel(SelArgs a) {
  __shared__ SelectShared sh;
  const int b = blockIdx.x, tid = threadIdx.x, N = a.N, base = tid * E;
  const float* sv_p = a.sal + (size_t)b * N;
  const float* st_p = a.rel + (size_t)b * N;
  float sv[E], st[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const bool ok = base + e < N;
    sv[e] = ok ? sv_p[base + e] : 0.f;
    st[e] = ok ? st_p[base + e] : 0.f;
  }
  const int rmed = (N - 1) / 2;
  const int rank[2] = {rmed, rmed};
  uint32_t res[2];
  int less[2], eq[2];
  auto raw_key = [&](int set, int e) { return f2key(set ? st[e] : sv[e]); };
  block_select<2, E>(raw_key, base, N, rank, res, less, eq, sh);
  const float med_v = key2f(res[0]), med_t = key2f(res[1]);
  auto dev_key = [&](int set, int e) {
    return f2key(set ? fabsf(st[e] - med_t) : fabsf(sv[e] - med_v));
  };
  block_select<2, E>(dev_key, base, N, rank, res, less, eq, sh);
  const float mad_v = key2f(res[0]), mad_t = key2f(res[1]);
  if (a.norm_stats && tid == 0) {
    a.norm_stats[4 * b + 0] = med_v;
    a.norm_stats[4 * b + 1] = mad_v;
    a.norm_stats[4 * b + 2] = med_t;
    a.norm_stats[4 * b + 3] = mad_t;
  }
  const float den_v = mad_v + a.eps, den_t = mad_t + a.eps;
  float sc[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const float av = a.wv * (fmaxf((sv[e] - med_v) / den_v, 0.f) / a.tau_v);
    const float bt = a.wt * (fmaxf((st[e] - med_t) / den_t, 0.f) / a.tau_t);
    sc[e] = fmaxf(av, bt) + a.lam * sqrtf(av * bt);
  }
  if (a.score_out) {
#pragma unroll
    for (int e = 0; e < E; ++e)
      if (base + e < N) a.score_out[(size_t)b * N + base + e] = sc[e];
  }
  block_topk_write<E>(sc, base, N, a.K, a.kept_idx + (size_t)b * a.K, sh);
}

template <int E>
__global__ __launch_bounds__(kSelThreads) void topk_kernel(const float* scores, int N, int K,
                                                           int32_t* out) {
  __shared__ SelectShared sh;
  const int b = blockIdx.x, base = threadIdx.x * E;
  const float* p = scores + (size_t)b * N;
  float sc[E];
#pragma unroll
  for (int e = 0; e < E; ++e) sc[e] = base + e < N ? p[base + e] : 0.f;
  block_topk_write<E>(sc, base, N, K, out + (size_t)b * K, sh);
}

// ---------------------------------------------------------------- launchers
hipError_t launch_prep(const PrepArgs& a, int dtype, hipStream_t s) {
  const int text_blocks = (a.B * a.M_max + 3) / 4;
  const dim3 grid(a.n_cls_blocks + text_blocks);
  if (dtype == 1)
    hipLaunchKernelGGL(prep_kernel<BF16>, grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(prep_kernel<F32>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

int relevance_tile_tokens() { return 32 * kRelNB * kRelNW; }

template <class In>
static void launch_rel_t(const RelArgs& a, int MT, hipStream_t s) {
  const dim3 grid(a.B * a.tiles_per_sample), block(64 * kRelNW);
  if (MT == 32)
    hipLaunchKernelGGL((relevance_kernel<In, 32, kRelNB, kRelNW>), grid, block, 0, s, a);
  else if (MT == 64)
    hipLaunchKernelGGL((relevance_kernel<In, 64, kRelNB, kRelNW>), grid, block, 0, s, a);
  else
    hipLaunchKernelGGL((relevance_kernel<In, 128, kRelNB, kRelNW>), grid, block, 0, s, a);
}

hipError_t launch_relevance(const RelArgs& a, int dtype, int MT, hipStream_t s) {
  if (dtype == 1)
    launch_rel_t<BF16>(a, MT, s);
  else
    launch_rel_t<F32>(a, MT, s);
  return hipGetLastError();
}

static int select_e(int N) {
  int e = 1;
  while (e * kSelThreads < N) e <<= 1;
  return e;
}

hipError_t launch_prellm_select(const SelArgs& a, int B, hipStream_t s) {
  const dim3 grid(B), block(kSelThreads);
  switch (select_e(a.N)) {
    case 1: hipLaunchKernelGGL(prellm_select_kernel<1>, grid, block, 0, s, a); break;
    case 2: hipLaunchKernelGGL(prellm_select_kernel<2>, grid, block, 0, s, a); break;
    case 4: hipLaunchKernelGGL(prellm_select_kernel<4>, grid, block, 0, s, a); break;
    case 8: hipLaunchKernelGGL(prellm_select_kernel<8>, grid, block, 0, s, a); break;
    case 16: hipLaunchKernelGGL(prellm_select_kernel<16>, grid, block, 0, s, a); break;
    case 32: hipLaunchKernelGGL(prellm_select_kernel<32>, grid, block, 0, s, a); break;
    case 64: hipLaunchKernelGGL(prellm_select_kernel<64>, grid, block, 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_topk(const float* scores, int B, int N, int K, int32_t* out, hipStream_t s) {
  const dim3 grid(B), block(kSelThreads);
  switch (select_e(N)) {
    case 1: hipLaunchKernelGGL(topk_kernel<1>, grid, block, 0, s, scores, N, K, out); break;
    case 2: hipLaunchKernelGGL(topk_kernel<2>, grid, block, 0, s, scores, N, K, out); break;
    case 4: hipLaunchKernelGGL(topk_kernel<4>, grid, block, 0, s, scores, N, K, out); break;
    case 8: hipLaunchKernelGGL(topk_kernel<8>, grid, block, 0, s, scores, N, K, out); break;
    case 16: hipLaunchKernelGGL(topk_kernel<16>, grid, block, 0, s, scores, N, K, out); break;
    case 32: hipLaunchKernelGGL(topk_kernel<32>, grid, block, 0, s, scores, N, K, out); break;
    case 64: hipLaunchKernelGGL(topk_kernel<64>, grid, block, 0, s, scores, N, K, out); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace trevs
