// Internal kernel argument blocks and launchers (not part of the C ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace trevs {

// ---------------------------------------------------------------- stage 1
struct PrepArgs {
  const void* cls;           // [B,H,N]
  int B, H, N, n_seg, seg_len;
  float2* row_stats;         // [B*H*n_seg]: (row max * log2 e, 1 / sum of exp)
  const void* text;          // [B,M_max,d]
  const int32_t* text_len;   // [B] or null
  int M_max, row_bytes;      // row_bytes = d * elem
  float* inv_tnorm;          // [B*M_max]: 1/max(||t_j||, 1e-12), 0 for j >= M_b
  int n_cls_blocks;          // blocks [0, n_cls_blocks) do [CLS] rows, the rest text rows
  int cls_vec16;             // every [CLS] segment row starts 16-byte aligned
};

struct RelArgs {
  const void* cls;
  const float2* row_stats;
  int H, n_seg, seg_len;
  const void* Z;             // [B,N,d]
  const void* T;             // [B,M_max,d]
  const int32_t* text_len;
  const float* inv_tnorm;
  int B, N, M_max, row_bytes, tiles_per_sample;
  float* sal;                // [B,N]
  float* rel;                // [B,N]
  // feature-dimension split (n_split > 1): workgroup (tile, split) covers
  // the 128-byte slabs [split*split_slabs, ...) and writes its partial dot
  // products t_j.z_i to part [B,n_split,M_max,N] and its partial ||z_i||^2
  // to zpart [B,n_split,N]; a merge pass finishes Eq. (4)-(5)
  int n_split, split_slabs;
  float* part;
  float* zpart;
};

// Launch shape of the relevance pass for one problem size.
struct RelPlan {
  bool stream;           // streaming kernel (rows of whole 128-byte slabs)
  int MT;                // text rows per tile (32, 64 or 128)
  int tile_tokens;       // visual tokens per workgroup
  int tiles_per_sample;
  int n_split, split_slabs;
  size_t part_floats() const;  // floats of part + zpart (0 without a split)
  int B, N, M_max;
};

struct NormArgs {
  const float* sal;
  const float* rel;
  int N;
  float* stats;              // [B,4]: Med(s^v), MAD(s^v), Med(s^t), MAD(s^t)
};

struct SelArgs {
  const float* sal;
  const float* rel;
  const float* stats;        // [B,4] from the robust-statistics kernel
  int N, K;
  int K_t;                   // budget-split mode: tokens taken by s^t first
  float wv, wt, tau_v, tau_t, lam, eps;
  float* score_out;          // [B,N] or null
  float* norm_stats;         // [B,4] or null
  int32_t* kept_idx;         // [B,K]
};

// ---------------------------------------------------------------- stage 2
struct StatsArgs {
  const void* q;             // [B,S,H_q,dh]
  const void* k;             // [B,S,H_kv,dh]
  int B, S, P, K_in, T_max, H_q, H_kv, G;
  float scale_log2e;         // scale * log2 e
  int n_split, split_len;    // visual columns per split (multiple of 32)
  int n_rgroups;             // workgroups along the (head-in-group, text row) axis
  float4* part;              // [B,H_q,T_max,n_split]: (max, sum e, sum e^2, -) in log2 units
  // Causal softmax domain: split s also reduces the non-visual causal keys
  // [s*rest_len, (s+1)*rest_len) of each text row (key j < P is prefix row j,
  // j >= P text row j - P, valid for text row q while j - P <= q).
  int rest_len;              // multiple of 32; 0 for the visual-only domain
  float4* part_rest;         // [B,H_q,T_max,n_split]: as part, over the non-visual keys
};

struct HeadArgs {
  const float4* part;
  int B, H_q, T_max, T_pad, K_in, n_split;
  const int32_t* text_len;
  const float* lse_rest;     // [B,H_q,T_max] natural log, or null
  const float4* part_rest;   // [B,H_q,T_max,n_split] non-visual causal statistics, or null
  float* lse2;               // [B,H_q,T_pad] row log-sum-exp in log2 units (T_pad = T_max rounded up to 32)
  float* head_var;           // [B,H_q] u_h
};

struct ScoreArgs {
  const void* q;
  const void* k;
  int B, S, P, K_in, T_max, T_pad, H_q, H_kv, G, n_keep;
  int n_vtiles;              // workgroups per sample (score_tile_tokens visual tokens each)
  float scale_log2e;
  const float* lse2;
  const float* head_var;     // [B,H_q] u_h
  int32_t* head_sel;         // [B,n_keep] H* ascending, or null
  const int32_t* text_len;
  float* p;                  // [B,K_in]
  // head split (n_hsplit > 1): workgroup (tile, split) sums the attention of
  // the selected heads [split*hps, (split+1)*hps) and writes it per (text
  // row, token) to hpart [B,n_hsplit,T_max,K_in]; a merge pass adds the
  // splits and takes the max over text rows
  int n_hsplit, hps;
  float* hpart;
};

// ---------------------------------------------------------------- diversity set
struct GramArgs {
  const void* Z;             // [B,N,d]
  int B, N, row_bytes, n_tiles; // n_tiles = ceil(N / tile rows)
  float* G;                  // [B,N,N] fp32 dot products z_j . z_i
  float* inv_norm;           // [B,N] 1 / max(||z_i||, 1e-12)
};
struct FpsArgs {
  const float* G;            // [B,N,N]
  const int32_t* pivots;     // [B,K_r] ascending
  int N, K_r, K_d;
  int B;
  int n_psplit;              // pivot splits of the initial distances (fps_init_splits)
  float* dist;               // [n_psplit,B,N] work: per split, max over its pivots j of G_ij / ||z_j||
  float* inv_norm;           // [B,N] work: 1 / max(||z_i||, 1e-12), from the Gram pass
  int32_t* kept_idx;         // [B,K_r+K_d] ascending
  int32_t* div_idx;          // [B,K_d] picks in pick order, or null
};
// Gram matrix, initial distances and the K_d sequential picks.
hipError_t launch_fps(const FpsArgs& f, const GramArgs& g, int dtype, int B, hipStream_t s);
// Pivot splits of the initial-distance pass (workgroups per token block):
// about 256 pivots each, at most 8.
inline int fps_init_splits(int K_r) {
  const int s = K_r / 256;
  return s < 1 ? 1 : (s > 8 ? 8 : s);
}

// ---------------------------------------------------------------- analysis
struct ProfileArgs {
  const void* q;
  const void* k;
  int B, S, P, K_in, T_max, T_pad, H_q, H_kv, G;
  int n_split, split_len;    // visual columns per workgroup (multiple of 32, <= kProfileSplitMax)
  float scale_log2e;
  const float* lse2;         // [B,H_q,T_pad] row log-sum-exp in log2 units
  const int32_t* text_len;
  float* profile;            // [B,H_q,K_in] mean attention over the valid text rows
};
constexpr int kProfileSplitMax = 2048;
struct SensitivityArgs {
  const float* profile[2];   // [B,H_q,K_in] per question
  int H_q, K_in;
  float* ts;                 // [B,H_q]
};
struct SpearmanArgs {
  const float* sv;           // [B,N]
  const float* st;           // [B,N]
  const int32_t* idx;        // [B,K] the top-K saliency set
  int N, K, n_tiles;         // n_tiles = ceil(K / kRankTile)
  long long* part;           // [B,n_tiles,4] partial sums of the centred rank products
  double* rho;               // [B]
};
constexpr int kRankTile = 64;  // tokens ranked per workgroup (one per lane)
// Visual profiles of every head for one question, the sensitivity of each
// head between two questions, and the rank correlation within a top-K set.
hipError_t launch_profile(const ProfileArgs& a, int dtype, int dh, hipStream_t s);
hipError_t launch_sensitivity(const SensitivityArgs& a, int B, hipStream_t s);
hipError_t launch_spearman(const SpearmanArgs& a, int B, hipStream_t s);

// ---------------------------------------------------------------- gather
constexpr int kGatherMaxTensors = 4;
struct GatherTensor {
  const uint8_t* src;
  uint8_t* dst;
  long long src_bstride, dst_bstride;  // bytes per sample
  int row_bytes;                       // multiple of 16
};
struct GatherArgs {
  GatherTensor t[kGatherMaxTensors];
  int n_tensors;
  const int32_t* idx;        // [B,n_kept] kept rows relative to the selected block
  int B, rows_out, P, K_in, n_kept;
  const int64_t* pos;        // [n_pos,B,S] or null
  int64_t* pos_out;          // [n_pos,B,rows_out]
  int n_pos, S;
};
constexpr int kGatherRowsPerBlock = 4;  // one row per wave
constexpr int kGatherThreads = 256;
constexpr int kGatherBatch = 8;  // 16-byte loads in flight per lane
constexpr int kGatherShortRows = 8;  // rows of at most 1 KB per wave

// Elements per thread of a 1024-thread selection workgroup over N values
// (a power of two, the template argument of the selection kernels).
inline int select_e(int N) {
  int e = 1;
  while (e * 1024 < N) e <<= 1;
  return e;
}

hipError_t launch_prep(const PrepArgs& a, int dtype, hipStream_t s);
RelPlan relevance_plan(int B, int N, int M_max, int row_bytes);
hipError_t launch_relevance(const RelArgs& a, const RelPlan& p, int dtype, hipStream_t s);
hipError_t launch_norm_stats(const NormArgs& a, int B, hipStream_t s);
hipError_t launch_prellm_select(const SelArgs& a, int B, hipStream_t s);
// Budget-split selection: the K_t highest s^t, then the K - K_t highest s^v
// among the other tokens.
hipError_t launch_budget_select(const SelArgs& a, int B, hipStream_t s);
// Stable top-K per row; nonneg: every score is >= 0 (lets the selection skip
// its min/max reduction).
hipError_t launch_topk(const float* scores, int B, int N, int K, int32_t* out, hipStream_t s,
                       bool nonneg = false);
hipError_t launch_stats(const StatsArgs& a, int dtype, int dh, hipStream_t s);
hipError_t launch_heads(const HeadArgs& a, hipStream_t s);
// u_h and the row log-sum-exps from the caller's per-row statistics
// [B,H_q,T_max,3] = (log-sum-exp, sum A, sum A^2) instead of the
// statistics pass.
hipError_t launch_heads_given(const float* row_stats, const HeadArgs& a, hipStream_t s);
hipError_t launch_score(const ScoreArgs& a, int dtype, int dh, hipStream_t s);
hipError_t launch_gather(const GatherArgs& a, hipStream_t s);

// Waves per workgroup of the statistics pass (column blocks of 32 rows).
int stats_waves(int G, int T_max);
// Visual tokens per workgroup of the token-score pass.
int score_tile_tokens(int dtype, int dh);
// Head splits of the token-score pass (1: none).
int score_head_splits(int B, int n_vtiles, int n_keep);

}  // namespace trevs
