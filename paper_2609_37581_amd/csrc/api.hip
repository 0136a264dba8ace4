// Host side of the C ABI: argument validation, workspace layout and the
// launch sequence of each stage.  Nothing here allocates device memory or
// waits for the device.
#include <cmath>
#include <math.h>
#include <string.h>

#include <algorithm>

#include "../../include/trevs.h"
#include "common.hpp"
#include "kernels.hpp"

using namespace trevs;

namespace {

constexpr size_t kWsAlign = 256;

size_t align_up(size_t x) { return (x + kWsAlign - 1) / kWsAlign * kWsAlign; }
bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }
bool finite(float x) { return isfinite(x) != 0; }
int elem_bytes(int dtype) { return dtype == TREVS_BF16 ? 2 : 4; }

struct Span {
  const void* p;
  size_t n;
};
bool overlap(Span a, Span b) {
  if (!a.p || !b.p || a.n == 0 || b.n == 0) return false;
  const uintptr_t a0 = reinterpret_cast<uintptr_t>(a.p), b0 = reinterpret_cast<uintptr_t>(b.p);
  return a0 < b0 + b.n && b0 < a0 + a.n;
}
// Every output span must be disjoint from every input span and from the
// other outputs.
bool any_overlap(const Span* out, int n_out, const Span* in, int n_in) {
  for (int i = 0; i < n_out; ++i) {
    for (int j = 0; j < n_in; ++j)
      if (overlap(out[i], in[j])) return true;
    for (int j = i + 1; j < n_out; ++j)
      if (overlap(out[i], out[j])) return true;
  }
  return false;
}

trevs_status record(void* const* events, int slot, hipStream_t s) {
  if (events && events[slot]) {
    if (hipEventRecord(reinterpret_cast<hipEvent_t>(events[slot]), s) != hipSuccess) return TREVS_ERR_HIP;
  }
  return TREVS_OK;
}

// ------------------------------------------------------------------ stage 1
struct PrellmLayout {
  size_t row_stats, inv_tnorm, sal, rel, stats, rel_part, pivots, gram, dist, inv_norm, total;
  RelPlan rel_plan;
};

trevs_status validate_prellm(const trevs_prellm_args* a) {
  if (!a || a->struct_size != sizeof(trevs_prellm_args)) return TREVS_ERR_INVALID_ARG;
  if (a->dtype != TREVS_F32 && a->dtype != TREVS_BF16) return TREVS_ERR_INVALID_ARG;
  if (a->B < 1 || a->N < 1 || a->n_seg < 1 || a->H_v < 1 || a->d < 1 || a->M_max < 1)
    return TREVS_ERR_INVALID_ARG;
  if (a->N % a->n_seg) return TREVS_ERR_INVALID_ARG;
  if (a->k_keep < 1 || a->k_keep > a->N) return TREVS_ERR_INVALID_ARG;
  if (a->k_div < 0 || a->k_div >= a->k_keep) return TREVS_ERR_INVALID_ARG;
  const int e = elem_bytes(a->dtype);
  if (((int64_t)a->d * e) % 16) return TREVS_ERR_INVALID_ARG;
  if (!finite(a->textual_ratio) || a->textual_ratio < 0.f || a->textual_ratio > 1.f)
    return TREVS_ERR_INVALID_ARG;
  if (!finite(a->tau_v) || !finite(a->tau_t) || a->tau_v <= 0.f || a->tau_t <= 0.f)
    return TREVS_ERR_INVALID_ARG;
  if (!finite(a->lambda_) || a->lambda_ < 0.f || !finite(a->eps) || a->eps < 0.f)
    return TREVS_ERR_INVALID_ARG;
  if (!a->cls_logits || !a->vis_feats || !a->text_emb || !a->kept_idx || !a->kept_feats)
    return TREVS_ERR_INVALID_ARG;
  if (!aligned(a->vis_feats, 16) || !aligned(a->text_emb, 16) || !aligned(a->kept_feats, 16) ||
      !aligned(a->cls_logits, e) || !aligned(a->kept_idx, 4) || !aligned(a->text_len, 4) ||
      !aligned(a->score_out, 4) || !aligned(a->sal_out, 4) || !aligned(a->rel_out, 4) ||
      !aligned(a->norm_stats, 4))
    return TREVS_ERR_INVALID_ARG;
  if ((int64_t)a->B * a->M_max > INT32_MAX || (int64_t)a->B * a->H_v * a->n_seg > INT32_MAX ||
      (int64_t)a->B * a->N > INT32_MAX)
    return TREVS_ERR_UNSUPPORTED;
  const size_t B = a->B, N = a->N;
  const Span in[] = {{a->cls_logits, B * a->H_v * N * e},
                     {a->vis_feats, B * N * a->d * e},
                     {a->text_emb, B * a->M_max * a->d * e},
                     {a->text_len, a->text_len ? B * 4 : 0}};
  const Span out[] = {{a->kept_idx, B * a->k_keep * 4},
                      {a->kept_feats, B * a->k_keep * a->d * e},
                      {a->score_out, a->score_out ? B * N * 4 : 0},
                      {a->sal_out, a->sal_out ? B * N * 4 : 0},
                      {a->rel_out, a->rel_out ? B * N * 4 : 0},
                      {a->norm_stats, a->norm_stats ? B * 16 : 0},
                      {a->div_idx, a->div_idx ? B * a->k_div * 4 : 0}};
  if (any_overlap(out, 7, in, 4)) return TREVS_ERR_INVALID_ARG;
  if (!aligned(a->div_idx, 4)) return TREVS_ERR_INVALID_ARG;
  if (a->ratio_mode != TREVS_RATIO_WEIGHTS && a->ratio_mode != TREVS_RATIO_BUDGET) return TREVS_ERR_INVALID_ARG;
  if (a->ratio_mode == TREVS_RATIO_BUDGET && (a->score_out || a->norm_stats)) return TREVS_ERR_INVALID_ARG;
  if (a->N > TREVS_MAX_SELECT_N) return TREVS_ERR_UNSUPPORTED;
  if (a->k_div > 0 && a->N > TREVS_MAX_FPS_N) return TREVS_ERR_UNSUPPORTED;
  return TREVS_OK;
}

// Tokens chosen by textual relevance in the budget-split mode: floor(rho K + 1/2).
int budget_text_count(float rho, int K) {
  const int kt = (int)std::floor((double)rho * K + 0.5);
  return std::min(std::max(kt, 0), K);
}

PrellmLayout prellm_layout(const trevs_prellm_args* a) {
  PrellmLayout L;
  size_t off = 0;
  L.row_stats = off;
  off = align_up(off + (size_t)a->B * a->H_v * a->n_seg * sizeof(float2));
  L.inv_tnorm = off;
  off = align_up(off + (size_t)a->B * a->M_max * sizeof(float));
  L.sal = off;
  off = align_up(off + (size_t)a->B * a->N * sizeof(float));
  L.rel = off;
  off = align_up(off + (size_t)a->B * a->N * sizeof(float));
  L.stats = off;
  off = align_up(off + (size_t)a->B * 4 * sizeof(float));
  L.rel_plan = relevance_plan(a->B, a->N, a->M_max, a->d * elem_bytes(a->dtype));
  L.rel_part = off;  // partial products of a feature-dimension split
  off = align_up(off + L.rel_plan.part_floats() * sizeof(float));
  L.pivots = L.gram = L.dist = L.inv_norm = off;
  if (a->k_div > 0) {  // farthest point sampling: pivot list, Gram matrices, distances
    L.pivots = off;
    off = align_up(off + (size_t)a->B * (a->k_keep - a->k_div) * sizeof(int32_t));
    L.gram = off;
    off = align_up(off + (size_t)a->B * a->N * a->N * sizeof(float));
    L.dist = off;
    off = align_up(off + (size_t)fps_init_splits(a->k_keep - a->k_div) * a->B * a->N * sizeof(float));
    L.inv_norm = off;
    off = align_up(off + (size_t)a->B * a->N * sizeof(float));
  }
  L.total = off;
  return L;
}

// ------------------------------------------------------------------ stage 2
struct InllmPlan {
  int n_split, split_len, n_rgroups, rest_len;
  int n_vtiles, n_hsplit, hps;  // token-score tiles per sample, head splits, heads per split
  size_t part, part_rest, lse2, head_var, head_sel, score, hpart, total;
};

trevs_status validate_inllm(const trevs_inllm_args* a) {
  if (!a || a->struct_size != sizeof(trevs_inllm_args)) return TREVS_ERR_INVALID_ARG;
  if (a->dtype != TREVS_F32 && a->dtype != TREVS_BF16) return TREVS_ERR_INVALID_ARG;
  if (a->B < 1 || a->S < 1 || a->P < 0 || a->K_in < 1 || a->T_max < 1) return TREVS_ERR_INVALID_ARG;
  if ((int64_t)a->P + a->K_in + a->T_max > a->S) return TREVS_ERR_INVALID_ARG;
  if (a->H_q < 1 || a->H_kv < 1 || a->H_q % a->H_kv) return TREVS_ERR_INVALID_ARG;
  if (a->d_head < 1 || a->D < 1 || a->n_pos < 1) return TREVS_ERR_INVALID_ARG;
  const int e = elem_bytes(a->dtype);
  if (((int64_t)a->D * e) % 16 || ((int64_t)a->H_kv * a->d_head * e) % 16) return TREVS_ERR_INVALID_ARG;
  if (a->n_keep_heads < 1 || a->n_keep_heads > a->H_q) return TREVS_ERR_INVALID_ARG;
  if (a->k_keep < 1 || a->k_keep > a->K_in) return TREVS_ERR_INVALID_ARG;
  if (!finite(a->scale) || a->scale <= 0.f) return TREVS_ERR_INVALID_ARG;
  if (a->softmax != TREVS_SOFTMAX_VISUAL && a->softmax != TREVS_SOFTMAX_CAUSAL) return TREVS_ERR_INVALID_ARG;
  if (a->softmax == TREVS_SOFTMAX_CAUSAL && a->lse_rest) return TREVS_ERR_INVALID_ARG;
  if (a->row_stats && a->lse_rest) return TREVS_ERR_INVALID_ARG;  // the given statistics hold the domain
  if (!aligned(a->row_stats, 4)) return TREVS_ERR_INVALID_ARG;
  if (!a->q || !a->k || !a->v || !a->hidden || !a->pos || !a->kept_idx || !a->hidden_out ||
      !a->k_out || !a->v_out || !a->pos_out)
    return TREVS_ERR_INVALID_ARG;
  if (!aligned(a->q, 16) || !aligned(a->k, 16) || !aligned(a->v, 16) || !aligned(a->hidden, 16) ||
      !aligned(a->hidden_out, 16) || !aligned(a->k_out, 16) || !aligned(a->v_out, 16) ||
      !aligned(a->pos, 8) || !aligned(a->pos_out, 8) || !aligned(a->text_len, 4) ||
      !aligned(a->lse_rest, 4) || !aligned(a->kept_idx, 4) || !aligned(a->head_sel, 4) ||
      !aligned(a->head_var, 4) || !aligned(a->score_out, 4))
    return TREVS_ERR_INVALID_ARG;
  if ((int64_t)a->B * a->S > INT32_MAX || (int64_t)a->n_pos * a->B * a->S > INT32_MAX ||
      (int64_t)a->B * a->H_q * a->T_max > INT32_MAX)
    return TREVS_ERR_UNSUPPORTED;
  const size_t B = a->B, S = a->S, So = (size_t)a->S - a->K_in + a->k_keep;
  const size_t kvrow = (size_t)a->H_kv * a->d_head * e;
  const Span in[] = {{a->q, B * S * a->H_q * a->d_head * e},
                     {a->k, B * S * kvrow},
                     {a->v, B * S * kvrow},
                     {a->hidden, B * S * a->D * e},
                     {a->pos, (size_t)a->n_pos * B * S * 8},
                     {a->text_len, a->text_len ? B * 4 : 0},
                     {a->lse_rest, a->lse_rest ? B * a->H_q * a->T_max * 4 : 0},
                     {a->row_stats, a->row_stats ? B * a->H_q * a->T_max * 12 : 0}};
  const Span out[] = {{a->kept_idx, B * a->k_keep * 4},
                      {a->hidden_out, B * So * a->D * e},
                      {a->k_out, B * So * kvrow},
                      {a->v_out, B * So * kvrow},
                      {a->pos_out, (size_t)a->n_pos * B * So * 8},
                      {a->head_sel, a->head_sel ? B * a->n_keep_heads * 4 : 0},
                      {a->head_var, a->head_var ? B * a->H_q * 4 : 0},
                      {a->score_out, a->score_out ? B * a->K_in * 4 : 0}};
  if (any_overlap(out, 8, in, 8)) return TREVS_ERR_INVALID_ARG;
  if (a->d_head != 64 && a->d_head != 128 && a->d_head != 256) return TREVS_ERR_UNSUPPORTED;
  if (a->H_q > 256) return TREVS_ERR_UNSUPPORTED;
  if (a->K_in > TREVS_MAX_SELECT_N) return TREVS_ERR_UNSUPPORTED;
  return TREVS_OK;
}

// Split of the visual keys for the statistics pass: enough workgroups to fill
// the GPU (>= 2 per CU), each split at least 64 keys, lengths multiples of 64
// (the pass consumes key tiles in pairs of 32).
struct StatsPlan {
  int n_split, split_len, n_rgroups;
  int rest_len;  // causal non-visual keys per split, multiple of 32 (0: visual-only softmax)
};
StatsPlan stats_plan(int B, int K_in, int T_max, int H_q, int H_kv, int softmax, int P) {
  StatsPlan p;
  const int G = H_q / H_kv;
  const int nrb = (G * T_max + 31) / 32;
  const int nw = stats_waves(G, T_max);
  p.n_rgroups = (nrb + nw - 1) / nw;
  const int64_t base_wgs = (int64_t)B * H_kv * p.n_rgroups;
  int n_split = (int)std::min<int64_t>((512 + base_wgs - 1) / base_wgs, (K_in + 63) / 64);
  n_split = std::max(n_split, 1);
  p.split_len = ((K_in + n_split - 1) / n_split + 63) / 64 * 64;
  p.n_split = (K_in + p.split_len - 1) / p.split_len;
  // the causal non-visual keys (P prefix + T_max text) shared evenly by the splits
  p.rest_len = softmax == TREVS_SOFTMAX_CAUSAL ? ((P + T_max + p.n_split - 1) / p.n_split + 31) / 32 * 32 : 0;
  return p;
}

size_t lse_rows_padded(int T_max) { return (size_t)(T_max + 31) / 32 * 32; }

InllmPlan inllm_plan(const trevs_inllm_args* a) {
  InllmPlan p;
  const StatsPlan sp = stats_plan(a->B, a->K_in, a->T_max, a->H_q, a->H_kv,
                                  a->row_stats ? TREVS_SOFTMAX_VISUAL : a->softmax, a->P);
  p.n_split = sp.n_split;
  p.split_len = sp.split_len;
  p.n_rgroups = sp.n_rgroups;
  p.rest_len = sp.rest_len;
  const size_t rows = (size_t)a->B * a->H_q * a->T_max;
  size_t off = 0;
  p.part = off;  // split statistics (none with the caller's row statistics)
  off = align_up(off + (a->row_stats ? 0 : rows * p.n_split * sizeof(float4)));
  p.part_rest = off;
  off = align_up(off + (p.rest_len ? rows * p.n_split * sizeof(float4) : 0));
  p.lse2 = off;
  off = align_up(off + (size_t)a->B * a->H_q * lse_rows_padded(a->T_max) * sizeof(float));
  p.head_var = off;
  off = align_up(off + (size_t)a->B * a->H_q * sizeof(float));
  p.head_sel = off;
  off = align_up(off + (size_t)a->B * a->n_keep_heads * sizeof(int32_t));
  p.score = off;
  off = align_up(off + (size_t)a->B * a->K_in * sizeof(float));
  const int vt = score_tile_tokens(a->dtype, a->d_head);
  p.n_vtiles = (a->K_in + vt - 1) / vt;
  const int hs = score_head_splits(a->B, p.n_vtiles, a->n_keep_heads);
  p.hps = (a->n_keep_heads + hs - 1) / hs;
  p.n_hsplit = (a->n_keep_heads + p.hps - 1) / p.hps;  // no split is empty
  if ((size_t)a->B * p.n_hsplit * a->T_max * a->K_in * sizeof(float) > (size_t(256) << 20)) {
    p.n_hsplit = 1;  // very long texts: the head sums would outgrow a modest workspace
    p.hps = a->n_keep_heads;
  }
  p.hpart = off;  // per-split head sums of the token-score pass
  off = align_up(off + (p.n_hsplit > 1 ? (size_t)a->B * p.n_hsplit * a->T_max * a->K_in * sizeof(float) : 0));
  p.total = off;
  return p;
}

// ------------------------------------------------------------------ analysis
trevs_status validate_sensitivity(const trevs_sensitivity_args* a) {
  if (!a || a->struct_size != sizeof(trevs_sensitivity_args)) return TREVS_ERR_INVALID_ARG;
  if (a->dtype != TREVS_F32 && a->dtype != TREVS_BF16) return TREVS_ERR_INVALID_ARG;
  if (a->B < 1 || a->S < 1 || a->P < 0 || a->K_in < 1 || a->T_max < 1) return TREVS_ERR_INVALID_ARG;
  if ((int64_t)a->P + a->K_in + a->T_max > a->S) return TREVS_ERR_INVALID_ARG;
  if (a->H_q < 1 || a->H_kv < 1 || a->H_q % a->H_kv || a->d_head < 1) return TREVS_ERR_INVALID_ARG;
  if (!finite(a->scale) || a->scale <= 0.f) return TREVS_ERR_INVALID_ARG;
  if (a->softmax != TREVS_SOFTMAX_VISUAL && a->softmax != TREVS_SOFTMAX_CAUSAL) return TREVS_ERR_INVALID_ARG;
  if (a->softmax == TREVS_SOFTMAX_CAUSAL && (a->lse_rest[0] || a->lse_rest[1])) return TREVS_ERR_INVALID_ARG;
  if (!a->ts || !aligned(a->ts, 4)) return TREVS_ERR_INVALID_ARG;
  const int e = elem_bytes(a->dtype);
  const size_t B = a->B, S = a->S;
  Span in[8], out[5];
  out[0] = Span{a->ts, B * a->H_q * 4};
  for (int c = 0; c < 2; ++c) {
    if (!a->q[c] || !a->k[c] || !aligned(a->q[c], 16) || !aligned(a->k[c], 16) ||
        !aligned(a->text_len[c], 4) || !aligned(a->lse_rest[c], 4) || !aligned(a->profile[c], 4) ||
        !aligned(a->head_var[c], 4))
      return TREVS_ERR_INVALID_ARG;
    in[4 * c + 0] = Span{a->q[c], B * S * a->H_q * a->d_head * e};
    in[4 * c + 1] = Span{a->k[c], B * S * a->H_kv * a->d_head * e};
    in[4 * c + 2] = Span{a->text_len[c], a->text_len[c] ? B * 4 : 0};
    in[4 * c + 3] = Span{a->lse_rest[c], a->lse_rest[c] ? B * a->H_q * a->T_max * 4 : 0};
    out[1 + 2 * c] = Span{a->profile[c], a->profile[c] ? B * a->H_q * a->K_in * 4 : 0};
    out[2 + 2 * c] = Span{a->head_var[c], a->head_var[c] ? B * a->H_q * 4 : 0};
  }
  if (any_overlap(out, 5, in, 8)) return TREVS_ERR_INVALID_ARG;
  if ((int64_t)a->B * a->S > INT32_MAX || (int64_t)a->B * a->H_q * a->T_max > INT32_MAX ||
      (int64_t)a->B * a->H_q * a->K_in > INT32_MAX)
    return TREVS_ERR_UNSUPPORTED;
  if (a->d_head != 64 && a->d_head != 128 && a->d_head != 256) return TREVS_ERR_UNSUPPORTED;
  return TREVS_OK;
}

struct SensitivityLayout {
  StatsPlan sp;
  size_t part[2], part_rest[2], lse2[2], head_var[2], profile[2], total;
};

SensitivityLayout sensitivity_layout(const trevs_sensitivity_args* a) {
  SensitivityLayout L;
  L.sp = stats_plan(a->B, a->K_in, a->T_max, a->H_q, a->H_kv, a->softmax, a->P);
  const size_t heads = (size_t)a->B * a->H_q;
  size_t off = 0;
  for (int c = 0; c < 2; ++c) {
    L.part[c] = off;
    off = align_up(off + heads * a->T_max * L.sp.n_split * sizeof(float4));
    L.part_rest[c] = off;
    off = align_up(off + (L.sp.rest_len ? heads * a->T_max * L.sp.n_split * sizeof(float4) : 0));
    L.lse2[c] = off;
    off = align_up(off + heads * lse_rows_padded(a->T_max) * sizeof(float));
    L.head_var[c] = off;
    off = align_up(off + heads * sizeof(float));
    L.profile[c] = off;
    off = align_up(off + heads * a->K_in * sizeof(float));
  }
  L.total = off;
  return L;
}

size_t spearman_tiles(int K) { return (size_t)(K + kRankTile - 1) / kRankTile; }

trevs_status validate_spearman(const float* sv, const float* st, int32_t B, int32_t N, int32_t K,
                               const double* rho, const int32_t* kept_idx) {
  if (!sv || !st || !rho || B < 1 || N < 1 || K < 1 || K > N) return TREVS_ERR_INVALID_ARG;
  if (!aligned(sv, 4) || !aligned(st, 4) || !aligned(rho, 8) || !aligned(kept_idx, 4))
    return TREVS_ERR_INVALID_ARG;
  const Span in[] = {{sv, (size_t)B * N * 4}, {st, (size_t)B * N * 4}};
  const Span out[] = {{rho, (size_t)B * 8}, {kept_idx, kept_idx ? (size_t)B * K * 4 : 0}};
  if (any_overlap(out, 2, in, 2)) return TREVS_ERR_INVALID_ARG;
  if ((int64_t)B * N > INT32_MAX) return TREVS_ERR_UNSUPPORTED;
  if (N > TREVS_MAX_SELECT_N) return TREVS_ERR_UNSUPPORTED;
  return TREVS_OK;
}

size_t spearman_ws_part(int32_t B, int32_t K) { return align_up((size_t)B * K * sizeof(int32_t)); }

trevs_status check_ws(void* ws, size_t ws_bytes, size_t need) {
  if (need == 0) return TREVS_OK;
  if (!ws || ws_bytes < need || !aligned(ws, kWsAlign)) return TREVS_ERR_WORKSPACE;
  return TREVS_OK;
}

}  // namespace

#define TREVS_TRY(x)                            \
  do {                                          \
    const trevs_status st_ = (x);               \
    if (st_ != TREVS_OK) return st_;            \
  } while (0)
#define TREVS_HIP(x)                                   \
  do {                                                 \
    if ((x) != hipSuccess) return TREVS_ERR_HIP;       \
  } while (0)

extern "C" {

size_t trevs_prellm_args_size(void) { return sizeof(trevs_prellm_args); }
size_t trevs_inllm_args_size(void) { return sizeof(trevs_inllm_args); }
size_t trevs_sensitivity_args_size(void) { return sizeof(trevs_sensitivity_args); }

const char* trevs_status_string(trevs_status s) {
  switch (s) {
    case TREVS_OK: return "ok";
    case TREVS_ERR_INVALID_ARG: return "invalid argument";
    case TREVS_ERR_UNSUPPORTED: return "unsupported by this implementation";
    case TREVS_ERR_WORKSPACE: return "workspace missing, misaligned or too small";
    case TREVS_ERR_HIP: return "HIP launch or event error";
  }
  return "unknown status";
}

int32_t trevs_keep_count(float ratio, int32_t n) {
  if (n < 1) return 0;
  const double k = floor((double)ratio * n + 0.5);
  if (!(k >= 1.0)) return 1;
  return k > n ? n : (int32_t)k;
}

size_t trevs_prellm_workspace_size(const trevs_prellm_args* a) {
  const trevs_status st = validate_prellm(a);
  if (st != TREVS_OK) return 0;
  return prellm_layout(a).total;
}

size_t trevs_inllm_workspace_size(const trevs_inllm_args* a) {
  const trevs_status st = validate_inllm(a);
  if (st != TREVS_OK) return 0;
  return inllm_plan(a).total;
}

size_t trevs_topk_workspace_size(int32_t, int32_t, int32_t) { return 0; }

trevs_status trevs_prellm_prune(const trevs_prellm_args* a, void* ws, size_t ws_bytes, void* stream) {
  TREVS_TRY(validate_prellm(a));
  const PrellmLayout L = prellm_layout(a);
  TREVS_TRY(check_ws(ws, ws_bytes, L.total));
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  uint8_t* w = reinterpret_cast<uint8_t*>(ws);
  const int e = elem_bytes(a->dtype);
  float2* row_stats = reinterpret_cast<float2*>(w + L.row_stats);
  float* inv_tnorm = reinterpret_cast<float*>(w + L.inv_tnorm);
  float* sal = a->sal_out ? a->sal_out : reinterpret_cast<float*>(w + L.sal);
  float* rel = a->rel_out ? a->rel_out : reinterpret_cast<float*>(w + L.rel);

  PrepArgs pa;
  pa.cls = a->cls_logits;
  pa.B = a->B;
  pa.H = a->H_v;
  pa.N = a->N;
  pa.n_seg = a->n_seg;
  pa.seg_len = a->N / a->n_seg;
  pa.row_stats = row_stats;
  pa.text = a->text_emb;
  pa.text_len = a->text_len;
  pa.M_max = a->M_max;
  pa.row_bytes = a->d * e;
  pa.inv_tnorm = inv_tnorm;
  pa.n_cls_blocks = a->B * a->H_v * a->n_seg;
  pa.cls_vec16 = aligned(a->cls_logits, 16) && ((size_t)a->N * e) % 16 == 0 &&
                 ((size_t)(a->N / a->n_seg) * e) % 16 == 0;
  TREVS_TRY(record(a->events, 0, s));
  TREVS_HIP(launch_prep(pa, a->dtype, s));
  TREVS_TRY(record(a->events, 1, s));

  RelArgs ra;
  ra.cls = a->cls_logits;
  ra.row_stats = row_stats;
  ra.H = a->H_v;
  ra.n_seg = a->n_seg;
  ra.seg_len = a->N / a->n_seg;
  ra.Z = a->vis_feats;
  ra.T = a->text_emb;
  ra.text_len = a->text_len;
  ra.inv_tnorm = inv_tnorm;
  ra.B = a->B;
  ra.N = a->N;
  ra.M_max = a->M_max;
  ra.row_bytes = a->d * e;
  const RelPlan& rp = L.rel_plan;
  ra.tiles_per_sample = rp.tiles_per_sample;
  ra.sal = sal;
  ra.rel = rel;
  ra.n_split = rp.n_split;
  ra.split_slabs = rp.split_slabs;
  ra.part = reinterpret_cast<float*>(w + L.rel_part);
  ra.zpart = ra.part + (size_t)rp.n_split * a->B * a->M_max * a->N;
  TREVS_TRY(record(a->events, 2, s));
  TREVS_HIP(launch_relevance(ra, rp, a->dtype, s));
  TREVS_TRY(record(a->events, 3, s));

  const bool budget = a->ratio_mode == TREVS_RATIO_BUDGET;
  float* stats = reinterpret_cast<float*>(w + L.stats);
  NormArgs na;
  na.sal = sal;
  na.rel = rel;
  na.N = a->N;
  na.stats = stats;
  TREVS_TRY(record(a->events, 4, s));
  if (!budget) TREVS_HIP(launch_norm_stats(na, a->B, s));  // the budget split ranks raw scores
  TREVS_TRY(record(a->events, 5, s));

  SelArgs sa;
  sa.sal = sal;
  sa.rel = rel;
  sa.stats = stats;
  sa.N = a->N;
  sa.K = a->k_keep;
  sa.wv = (float)(2.0 * (1.0 - (double)a->textual_ratio));
  sa.wt = (float)(2.0 * (double)a->textual_ratio);
  sa.tau_v = a->tau_v;
  sa.tau_t = a->tau_t;
  sa.lam = a->lambda_;
  sa.eps = a->eps;
  sa.score_out = a->score_out;
  sa.norm_stats = a->norm_stats;
  // with a diversity set the top-K keeps the K_r pivots, and farthest point
  // sampling adds the other K_d tokens and writes the kept list
  const int K_r = a->k_keep - a->k_div;
  int32_t* pivots = reinterpret_cast<int32_t*>(w + L.pivots);
  sa.K = K_r;
  sa.kept_idx = a->k_div > 0 ? pivots : a->kept_idx;
  sa.K_t = budget_text_count(a->textual_ratio, K_r);
  TREVS_TRY(record(a->events, 6, s));
  if (budget)
    TREVS_HIP(launch_budget_select(sa, a->B, s));
  else
    TREVS_HIP(launch_prellm_select(sa, a->B, s));
  if (a->k_div > 0) {
    GramArgs ga;
    ga.Z = a->vis_feats;
    ga.B = a->B;
    ga.N = a->N;
    ga.row_bytes = a->d * e;
    ga.n_tiles = (a->N + 127) / 128;
    ga.G = reinterpret_cast<float*>(w + L.gram);
    ga.inv_norm = reinterpret_cast<float*>(w + L.inv_norm);
    FpsArgs fa;
    fa.G = ga.G;
    fa.pivots = pivots;
    fa.N = a->N;
    fa.K_r = K_r;
    fa.K_d = a->k_div;
    fa.B = a->B;
    fa.n_psplit = fps_init_splits(K_r);
    fa.dist = reinterpret_cast<float*>(w + L.dist);
    fa.inv_norm = reinterpret_cast<float*>(w + L.inv_norm);
    fa.kept_idx = a->kept_idx;
    fa.div_idx = a->div_idx;
    TREVS_HIP(launch_fps(fa, ga, a->dtype, a->B, s));
  }
  TREVS_TRY(record(a->events, 7, s));

  GatherArgs ga;
  memset(&ga, 0, sizeof(ga));
  ga.t[0].src = reinterpret_cast<const uint8_t*>(a->vis_feats);
  ga.t[0].dst = reinterpret_cast<uint8_t*>(a->kept_feats);
  ga.t[0].row_bytes = a->d * e;
  ga.t[0].src_bstride = (long long)a->N * a->d * e;
  ga.t[0].dst_bstride = (long long)a->k_keep * a->d * e;
  ga.n_tensors = 1;
  ga.idx = a->kept_idx;
  ga.B = a->B;
  ga.rows_out = a->k_keep;
  ga.P = 0;
  ga.K_in = a->N;
  ga.n_kept = a->k_keep;
  TREVS_TRY(record(a->events, 8, s));
  TREVS_HIP(launch_gather(ga, s));
  TREVS_TRY(record(a->events, 9, s));
  return TREVS_OK;
}

trevs_status trevs_inllm_prune(const trevs_inllm_args* a, void* ws, size_t ws_bytes, void* stream) {
  TREVS_TRY(validate_inllm(a));
  const InllmPlan p = inllm_plan(a);
  TREVS_TRY(check_ws(ws, ws_bytes, p.total));
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  uint8_t* w = reinterpret_cast<uint8_t*>(ws);
  const int e = elem_bytes(a->dtype);
  const int G = a->H_q / a->H_kv;
  const float scale_log2e = a->scale * kLog2e;
  float4* part = reinterpret_cast<float4*>(w + p.part);
  float4* part_rest = p.rest_len ? reinterpret_cast<float4*>(w + p.part_rest) : nullptr;
  float* lse2 = reinterpret_cast<float*>(w + p.lse2);
  float* head_var = a->head_var ? a->head_var : reinterpret_cast<float*>(w + p.head_var);
  float* score = a->score_out ? a->score_out : reinterpret_cast<float*>(w + p.score);

  StatsArgs ta;
  ta.q = a->q;
  ta.k = a->k;
  ta.B = a->B;
  ta.S = a->S;
  ta.P = a->P;
  ta.K_in = a->K_in;
  ta.T_max = a->T_max;
  ta.H_q = a->H_q;
  ta.H_kv = a->H_kv;
  ta.G = G;
  ta.scale_log2e = scale_log2e;
  ta.n_split = p.n_split;
  ta.split_len = p.split_len;
  ta.n_rgroups = p.n_rgroups;
  ta.part = part;
  ta.rest_len = p.rest_len;
  ta.part_rest = part_rest;
  TREVS_TRY(record(a->events, 0, s));
  if (!a->row_stats) TREVS_HIP(launch_stats(ta, a->dtype, a->d_head, s));
  TREVS_TRY(record(a->events, 1, s));

  HeadArgs ha;
  ha.part = part;
  ha.B = a->B;
  ha.H_q = a->H_q;
  ha.T_max = a->T_max;
  ha.T_pad = (int)lse_rows_padded(a->T_max);
  ha.K_in = a->K_in;
  ha.n_split = p.n_split;
  ha.text_len = a->text_len;
  ha.lse_rest = a->lse_rest;
  ha.part_rest = part_rest;
  ha.lse2 = lse2;
  ha.head_var = head_var;
  TREVS_TRY(record(a->events, 2, s));
  if (a->row_stats)
    TREVS_HIP(launch_heads_given(a->row_stats, ha, s));
  else
    TREVS_HIP(launch_heads(ha, s));
  TREVS_TRY(record(a->events, 3, s));

  ScoreArgs sa;
  sa.q = a->q;
  sa.k = a->k;
  sa.B = a->B;
  sa.S = a->S;
  sa.P = a->P;
  sa.K_in = a->K_in;
  sa.T_max = a->T_max;
  sa.T_pad = (int)lse_rows_padded(a->T_max);
  sa.H_q = a->H_q;
  sa.H_kv = a->H_kv;
  sa.G = G;
  sa.n_keep = a->n_keep_heads;
  sa.n_vtiles = p.n_vtiles;
  sa.n_hsplit = p.n_hsplit;
  sa.hps = p.hps;
  sa.hpart = reinterpret_cast<float*>(w + p.hpart);
  sa.scale_log2e = scale_log2e;
  sa.lse2 = lse2;
  sa.head_var = head_var;
  sa.head_sel = a->head_sel;
  sa.text_len = a->text_len;
  sa.p = score;
  TREVS_TRY(record(a->events, 4, s));
  TREVS_HIP(launch_score(sa, a->dtype, a->d_head, s));
  TREVS_TRY(record(a->events, 5, s));

  TREVS_TRY(record(a->events, 6, s));
  TREVS_HIP(launch_topk(score, a->B, a->K_in, a->k_keep, a->kept_idx, s, /*nonneg=*/true));  // means of probabilities
  TREVS_TRY(record(a->events, 7, s));

  const int So = a->S - a->K_in + a->k_keep;
  const int kvrow = a->H_kv * a->d_head * e;
  GatherArgs ga;
  memset(&ga, 0, sizeof(ga));
  const void* srcs[3] = {a->hidden, a->k, a->v};
  void* dsts[3] = {a->hidden_out, a->k_out, a->v_out};
  const int rowb[3] = {a->D * e, kvrow, kvrow};
  for (int t = 0; t < 3; ++t) {
    ga.t[t].src = reinterpret_cast<const uint8_t*>(srcs[t]);
    ga.t[t].dst = reinterpret_cast<uint8_t*>(dsts[t]);
    ga.t[t].row_bytes = rowb[t];
    ga.t[t].src_bstride = (long long)a->S * rowb[t];
    ga.t[t].dst_bstride = (long long)So * rowb[t];
  }
  ga.n_tensors = 3;
  ga.idx = a->kept_idx;
  ga.B = a->B;
  ga.rows_out = So;
  ga.P = a->P;
  ga.K_in = a->K_in;
  ga.n_kept = a->k_keep;
  ga.pos = a->pos;
  ga.pos_out = a->pos_out;
  ga.n_pos = a->n_pos;
  ga.S = a->S;
  TREVS_TRY(record(a->events, 8, s));
  TREVS_HIP(launch_gather(ga, s));
  TREVS_TRY(record(a->events, 9, s));
  return TREVS_OK;
}

trevs_status trevs_topk_select(const float* scores, int32_t B, int32_t N, int32_t K, int32_t* kept_idx,
                               void* ws, size_t ws_bytes, void* stream) {
  (void)ws;
  (void)ws_bytes;
  if (!scores || !kept_idx || B < 1 || N < 1 || K < 1 || K > N) return TREVS_ERR_INVALID_ARG;
  if (!aligned(scores, 4) || !aligned(kept_idx, 4)) return TREVS_ERR_INVALID_ARG;
  if (overlap(Span{scores, (size_t)B * N * 4}, Span{kept_idx, (size_t)B * K * 4}))
    return TREVS_ERR_INVALID_ARG;
  if (N > TREVS_MAX_SELECT_N) return TREVS_ERR_UNSUPPORTED;
  TREVS_HIP(launch_topk(scores, B, N, K, kept_idx, reinterpret_cast<hipStream_t>(stream)));
  return TREVS_OK;
}

size_t trevs_sensitivity_workspace_size(const trevs_sensitivity_args* a) {
  if (validate_sensitivity(a) != TREVS_OK) return 0;
  return sensitivity_layout(a).total;
}

trevs_status trevs_text_sensitivity(const trevs_sensitivity_args* a, void* ws, size_t ws_bytes, void* stream) {
  TREVS_TRY(validate_sensitivity(a));
  const SensitivityLayout L = sensitivity_layout(a);
  TREVS_TRY(check_ws(ws, ws_bytes, L.total));
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  uint8_t* w = reinterpret_cast<uint8_t*>(ws);
  const int G = a->H_q / a->H_kv;
  const int T_pad = (int)lse_rows_padded(a->T_max);
  // profile splits: about 1024 workgroups, each split 128..kProfileSplitMax keys
  int n_split = (int)std::min<int64_t>((1024 + (int64_t)a->B * a->H_q - 1) / ((int64_t)a->B * a->H_q),
                                       (a->K_in + 127) / 128);
  n_split = std::max(std::max(n_split, 1), (a->K_in + kProfileSplitMax - 1) / kProfileSplitMax);
  const int split_len = ((a->K_in + n_split - 1) / n_split + 31) / 32 * 32;
  n_split = (a->K_in + split_len - 1) / split_len;
  SensitivityArgs sa;
  sa.H_q = a->H_q;
  sa.K_in = a->K_in;
  sa.ts = a->ts;
  for (int c = 0; c < 2; ++c) {
    float4* part = reinterpret_cast<float4*>(w + L.part[c]);
    float4* part_rest = L.sp.rest_len ? reinterpret_cast<float4*>(w + L.part_rest[c]) : nullptr;
    float* lse2 = reinterpret_cast<float*>(w + L.lse2[c]);
    float* head_var = a->head_var[c] ? a->head_var[c] : reinterpret_cast<float*>(w + L.head_var[c]);
    float* profile = a->profile[c] ? a->profile[c] : reinterpret_cast<float*>(w + L.profile[c]);
    StatsArgs ta;
    ta.q = a->q[c];
    ta.k = a->k[c];
    ta.B = a->B;
    ta.S = a->S;
    ta.P = a->P;
    ta.K_in = a->K_in;
    ta.T_max = a->T_max;
    ta.H_q = a->H_q;
    ta.H_kv = a->H_kv;
    ta.G = G;
    ta.scale_log2e = a->scale * kLog2e;
    ta.n_split = L.sp.n_split;
    ta.split_len = L.sp.split_len;
    ta.n_rgroups = L.sp.n_rgroups;
    ta.part = part;
    ta.rest_len = L.sp.rest_len;
    ta.part_rest = part_rest;
    TREVS_TRY(record(a->events, 6 * c + 0, s));
    TREVS_HIP(launch_stats(ta, a->dtype, a->d_head, s));
    TREVS_TRY(record(a->events, 6 * c + 1, s));
    HeadArgs ha;
    ha.part = part;
    ha.B = a->B;
    ha.H_q = a->H_q;
    ha.T_max = a->T_max;
    ha.T_pad = T_pad;
    ha.K_in = a->K_in;
    ha.n_split = L.sp.n_split;
    ha.text_len = a->text_len[c];
    ha.lse_rest = a->lse_rest[c];
    ha.part_rest = part_rest;
    ha.lse2 = lse2;
    ha.head_var = head_var;
    TREVS_TRY(record(a->events, 6 * c + 2, s));
    TREVS_HIP(launch_heads(ha, s));
    TREVS_TRY(record(a->events, 6 * c + 3, s));
    ProfileArgs pa;
    pa.q = a->q[c];
    pa.k = a->k[c];
    pa.B = a->B;
    pa.S = a->S;
    pa.P = a->P;
    pa.K_in = a->K_in;
    pa.T_max = a->T_max;
    pa.T_pad = T_pad;
    pa.H_q = a->H_q;
    pa.H_kv = a->H_kv;
    pa.G = G;
    pa.n_split = n_split;
    pa.split_len = split_len;
    pa.scale_log2e = a->scale * kLog2e;
    pa.lse2 = lse2;
    pa.text_len = a->text_len[c];
    pa.profile = profile;
    TREVS_TRY(record(a->events, 6 * c + 4, s));
    TREVS_HIP(launch_profile(pa, a->dtype, a->d_head, s));
    TREVS_TRY(record(a->events, 6 * c + 5, s));
    sa.profile[c] = profile;
  }
  TREVS_TRY(record(a->events, 12, s));
  TREVS_HIP(launch_sensitivity(sa, a->B, s));
  TREVS_TRY(record(a->events, 13, s));
  return TREVS_OK;
}

size_t trevs_spearman_workspace_size(int32_t B, int32_t N, int32_t K) {
  if (B < 1 || N < 1 || K < 1 || K > N || N > TREVS_MAX_SELECT_N || (int64_t)B * N > INT32_MAX) return 0;
  return spearman_ws_part(B, K) + align_up((size_t)B * spearman_tiles(K) * 4 * sizeof(long long));
}

trevs_status trevs_topk_spearman(const float* sv, const float* st, int32_t B, int32_t N, int32_t K, double* rho,
                                 int32_t* kept_idx, void* ws, size_t ws_bytes, void* stream) {
  TREVS_TRY(validate_spearman(sv, st, B, N, K, rho, kept_idx));
  TREVS_TRY(check_ws(ws, ws_bytes, trevs_spearman_workspace_size(B, N, K)));
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  uint8_t* w = reinterpret_cast<uint8_t*>(ws);
  int32_t* idx = kept_idx ? kept_idx : reinterpret_cast<int32_t*>(w);
  TREVS_HIP(launch_topk(sv, B, N, K, idx, s));
  SpearmanArgs pa;
  pa.sv = sv;
  pa.st = st;
  pa.idx = idx;
  pa.N = N;
  pa.K = K;
  pa.n_tiles = (int)spearman_tiles(K);
  pa.part = reinterpret_cast<long long*>(w + spearman_ws_part(B, K));
  pa.rho = rho;
  TREVS_HIP(launch_spearman(pa, B, s));
  return TREVS_OK;
}

}  // extern "C"
