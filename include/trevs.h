/*
 * trevs.h - C ABI of the TReVS visual-token pruning library for MI355X (gfx950).
 *
 * TReVS ("Integrating Textual Relevance and Visual Saliency for Efficient
 * Vision-Language Model Token Pruning", arxiv 2609.37581) prunes the visual
 * tokens of a vision-language model in two stages:
 *   Stage 1, before the LLM (Sec. 4.1, Eq. (2)-(7)): fuse the vision
 *     encoder's [CLS] attention saliency with the textual relevance of each
 *     visual token, take a stable top-K_1, and gather the kept tokens.
 *   Stage 2, inside the LLM at one layer (Sec. 4.2, Eq. (8)-(9)): compute the
 *     text->vision attention, keep the high-variance heads, score each visual
 *     token by its max-over-text attention averaged over those heads, take a
 *     stable top-K_2, and compact hidden states, position ids and K/V rows.
 *
 * Conventions for every entry point:
 *   - Tensor pointers are DEVICE pointers to dense row-major tensors.  Float
 *     tensors share one element type per call (trevs_dtype).  Pointers that
 *     are read or written as 16-byte vectors (named below) must be 16-byte
 *     aligned; every other tensor must be aligned to its element size.
 *   - The caller owns every buffer, including the workspace; the library
 *     never allocates, frees or keeps state between calls.  Calls are
 *     reentrant and thread-safe.
 *   - Work is enqueued asynchronously on `stream` (a hipStream_t; NULL means
 *     the default stream); the host never waits for the device.
 *   - Arguments are validated on the host before anything is launched;
 *     invalid arguments return an error and launch nothing.  Values that live
 *     in device memory (text lengths) cannot be checked without a device
 *     synchronisation: the kernels clamp a text length into 1..M_max (or
 *     1..T_max), so an out-of-range length computes with the nearest valid
 *     one and never reads or writes outside the buffers.
 *   - Inputs must be finite.  Output buffers must not overlap the inputs or
 *     each other.  Outputs are undefined when an error is returned.
 *   - Index lists are int32, ascending and unique.  Top-K order is score
 *     descending with ties going to the lower index.
 *   - Optional `events`: NULL, or an array of 2*TREVS_*_NUM_KERNELS
 *     hipEvent_t handles (entries may be NULL).  Event 2k is recorded on the
 *     stream right before kernel k of the call and event 2k+1 right after
 *     it, for per-kernel timing by the caller.
 */
#ifndef TREVS_H
#define TREVS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum trevs_status {
  TREVS_OK = 0,
  TREVS_ERR_INVALID_ARG = 1, /* a size, ratio, pointer or alignment is invalid */
  TREVS_ERR_UNSUPPORTED = 2, /* valid, but beyond this implementation's limits */
  TREVS_ERR_WORKSPACE = 3,   /* workspace NULL, misaligned or too small */
  TREVS_ERR_HIP = 4          /* a HIP launch or event call failed */
} trevs_status;

typedef enum trevs_dtype { TREVS_F32 = 0, TREVS_BF16 = 1 } trevs_dtype;

/* Implementation limits (TREVS_ERR_UNSUPPORTED beyond them). */
#define TREVS_MAX_SELECT_N 65536 /* tokens ranked per sample by one top-K */
#define TREVS_MAX_FPS_N 32768    /* tokens per sample with a diversity set (k_div > 0) */
#define TREVS_PRELLM_NUM_KERNELS 5 /* prep, relevance, robust stats, fuse+top-K (+ diversity set), gather */
#define TREVS_INLLM_NUM_KERNELS 5  /* t2v stats (+ causal rest keys), head variance, head set+token score, top-K, compaction */
#define TREVS_SENSITIVITY_NUM_KERNELS 7 /* per question: t2v stats, head variance, profile; then Eq. (1) */

/* ------------------------------------------------------------------------
 * Stage 1 (pre-LLM), Sec. 4.1.  Per sample b:
 *   s^v_i  = (1/H_v) sum_h softmax(cls_logits[b,h,segment(i)])[i]   Eq. (2)-(3)
 *            the softmax runs over the N/n_seg patch logits of the segment
 *            (image tile or video frame) holding patch i.
 *   s^t_i  = sqrt((1/M_b) sum_{j<M_b} max(tbar_j . zbar_i, 0)^2)     Eq. (4)-(5)
 *            zbar, tbar: rows of vis_feats / text_emb over their L2 norm
 *            (norm floored at 1e-12); M_b = text_len[b].
 *   shat^c = max((s^c - Med(s^c)) / (MAD(s^c) + eps), 0) / tau_c     Eq. (6)
 *            Med = lower median (0-based rank floor((N-1)/2)), MAD = lower
 *            median of |s^c - Med|.
 *   s_i    = max(a_i, b_i) + lambda sqrt(a_i b_i),                   Eq. (7)
 *            a = 2(1-rho) shat^v, b = 2 rho shat^t  (rho = textual_ratio;
 *            rho = 0.5 is Eq. (7) exactly, rho = 0 is [CLS]-only saliency).
 *   kept_idx[b]   = TopK(s, k_keep) in ascending order
 *   kept_feats[b] = vis_feats[b, kept_idx[b], :]  (bit copy)
 * With k_div = K_d > 0 the top-K above keeps K_r = k_keep - K_d pivots, and
 * K_d more tokens are added by farthest point sampling (context
 * preservation, Sec. 4.1 after Eq. (7)): one at a time, the token outside
 * the selected set whose cosine distance 1 - zbar_i . zbar_j to its nearest
 * selected token is largest (ties to the lower index).  This forms the Gram
 * matrix Z Z^T of every sample in the workspace (B*N*N floats beyond the
 * k_div = 0 size, e.g. 4.3 GB at B = 4, N = 16,384; 85 MB at B = 64,
 * N = 576); trevs_prellm_workspace_size includes it, and the call itself
 * allocates nothing.
 * With ratio_mode = TREVS_RATIO_BUDGET the textual ratio is instead the
 * share of the token budget given to textual relevance (the reading of the
 * preliminary analysis, Sec. 3): K_t = floor(rho * k_keep + 1/2) tokens with
 * the highest s^t, then the k_keep - K_t tokens with the highest s^v among
 * the others; Eq. (6)-(7) are not used, and score_out and norm_stats must
 * be NULL.  Every top-K is stable (score descending, lower index first).
 * ---------------------------------------------------------------------- */
typedef enum trevs_ratio_mode {
  TREVS_RATIO_WEIGHTS = 0, /* branch weights 2(1-rho), 2rho inside Eq. (7) */
  TREVS_RATIO_BUDGET = 1   /* budget split between s^t and s^v */
} trevs_ratio_mode;

typedef struct trevs_prellm_args {
  uint32_t struct_size;      /* sizeof(trevs_prellm_args) */
  int32_t B;                 /* samples */
  int32_t N;                 /* visual tokens per sample, 1..TREVS_MAX_SELECT_N */
  int32_t n_seg;             /* [CLS] softmax segments; N % n_seg == 0 */
  int32_t H_v;               /* vision-encoder heads, >= 1 */
  int32_t d;                 /* projected width d'; d * elem_size % 16 == 0 */
  int32_t M_max;             /* padded text rows, >= 1 */
  int32_t k_keep;            /* K_1 = K_r + K_d, 1..N */
  int32_t k_div;             /* K_d farthest-point diversity tokens, 0..k_keep-1; N <= TREVS_MAX_FPS_N when > 0 */
  float textual_ratio;       /* rho in [0, 1]; 0.5 reproduces Eq. (7) */
  float tau_v, tau_t;        /* temperatures > 0 (paper: 1.4, 1.0) */
  float lambda_;             /* consistency reward weight >= 0 (paper: 1.0) */
  float eps;                 /* MAD stabiliser >= 0 (default 1e-8) */
  int32_t dtype;             /* trevs_dtype of cls_logits, vis_feats, text_emb, kept_feats */
  const void* cls_logits;    /* [B,H_v,N] pre-softmax [CLS]->patch logits, scaled by 1/sqrt(d_h) */
  const void* vis_feats;     /* [B,N,d] projected visual features Z (16-byte aligned) */
  const void* text_emb;      /* [B,M_max,d] text embeddings (16-byte aligned) */
  const int32_t* text_len;   /* [B] valid text rows M_b in 1..M_max, or NULL (= M_max) */
  int32_t* kept_idx;         /* OUT [B,k_keep] ascending */
  void* kept_feats;          /* OUT [B,k_keep,d] gathered rows (16-byte aligned) */
  float* score_out;          /* OPTIONAL OUT [B,N] fused score s */
  float* sal_out;            /* OPTIONAL OUT [B,N] s^v */
  float* rel_out;            /* OPTIONAL OUT [B,N] s^t */
  float* norm_stats;         /* OPTIONAL OUT [B,4] Med(s^v), MAD(s^v), Med(s^t), MAD(s^t) */
  void* const* events;       /* OPTIONAL [2*TREVS_PRELLM_NUM_KERNELS] hipEvent_t */
  int32_t ratio_mode;        /* trevs_ratio_mode */
  int32_t* div_idx;          /* OPTIONAL OUT [B,k_div] diversity tokens in pick order */
} trevs_prellm_args;

/* ------------------------------------------------------------------------
 * Stage 2 (in-LLM, at the pruning layer), Sec. 4.2.  Sequence layout per
 * sample: rows [0,P) prefix, [P,P+K_in) visual, [P+K_in, P+K_in+T_max) text,
 * then any further rows up to S.  Per sample b with G = H_q/H_kv and
 * T_b = text_len[b]:
 *   x[h,q,i] = scale * q[b,P+K_in+q,h,:] . k[b,P+i,h/G,:]   (q < T_b, i < K_in)
 *   A[h,q,:] = exp(x[h,q,:] - LSE[h,q]) over the visual columns, where the
 *              softmax domain (trevs_softmax) sets LSE[h,q]:
 *              VISUAL: logsumexp_i x[h,q,i] over the K_in visual keys; when
 *                lse_rest is given, logaddexp(that, lse_rest[b,h,q]), the
 *                full-row softmax with the non-visual part supplied by the
 *                caller;
 *              CAUSAL: the log-sum-exp of the row's whole causal attention
 *                row at this layer, computed from q and k: the prefix keys
 *                [0,P), the visual keys, and the text keys P+K_in .. P+K_in+q
 *                (the row's own position and those before it); every key
 *                uses the row's KV head h/G.  A thus holds the visual columns
 *                of the layer's own attention matrix (Sec. 4.2).
 *   u_h      = (1/T_b) sum_q Var_i A[h,q,i]  (population variance)    Eq. (8)
 *              (with row_stats: (1/T_b) sum_q [S2/K_in - (S1/K_in)^2] from the
 *              caller's per-row sums S1 = sum_i A, S2 = sum_i A^2, and the
 *              row log-sum-exp from row_stats as well)
 *   H*       = the n_keep_heads heads first under (u desc, h asc)
 *   p_i      = max_{q<T_b} (1/|H*|) sum_{h in H*} A[h,q,i]            Eq. (9)
 *   kept_idx = TopK(p, k_keep) ascending, relative to the visual block
 *   rows     = [0,P) ++ (P + kept_idx) ++ [P+K_in, S);  S' = S - K_in + k_keep
 *   hidden_out[b] = hidden[b,rows], k_out[b] = k[b,rows], v_out[b] = v[b,rows],
 *   pos_out[p,b]  = pos[p,b,rows]   (bit copies; position ids are not renumbered)
 * ---------------------------------------------------------------------- */
typedef enum trevs_softmax {
  TREVS_SOFTMAX_VISUAL = 0,  /* softmax over the visual keys (plus lse_rest, if given) */
  TREVS_SOFTMAX_CAUSAL = 1   /* softmax over each text row's causal row of the sequence */
} trevs_softmax;

typedef struct trevs_inllm_args {
  uint32_t struct_size;      /* sizeof(trevs_inllm_args) */
  int32_t B;                 /* samples */
  int32_t S;                 /* sequence rows at the pruning layer */
  int32_t P;                 /* prefix rows before the visual block, >= 0 */
  int32_t K_in;              /* visual rows K_1, 1..TREVS_MAX_SELECT_N */
  int32_t T_max;             /* padded text rows; P + K_in + T_max <= S */
  int32_t H_q, H_kv;         /* query / key-value heads; H_q % H_kv == 0 */
  int32_t d_head;            /* 64, 128 or 256 */
  int32_t D;                 /* hidden size; D * elem_size % 16 == 0 */
  int32_t n_pos;             /* position-id planes (1, or 3 for M-RoPE), >= 1 */
  int32_t n_keep_heads;      /* |H*|, 1..H_q (paper: H_q / 2) */
  int32_t k_keep;            /* K_2, 1..K_in */
  float scale;               /* logit scale > 0, normally 1/sqrt(d_head) */
  int32_t dtype;             /* trevs_dtype of q, k, v, hidden and their outputs */
  const void* q;             /* [B,S,H_q,d_head] (16-byte aligned) */
  const void* k;             /* [B,S,H_kv,d_head] (16-byte aligned) */
  const void* v;             /* [B,S,H_kv,d_head] (16-byte aligned) */
  const void* hidden;        /* [B,S,D] (16-byte aligned) */
  const int64_t* pos;        /* [n_pos,B,S] */
  const int32_t* text_len;   /* [B] T_b in 1..T_max, or NULL (= T_max) */
  const float* lse_rest;     /* OPTIONAL [B,H_q,T_max] log-sum-exp of each text row's non-visual
                                logits (natural log); VISUAL softmax only, NULL with CAUSAL */
  int32_t* kept_idx;         /* OUT [B,k_keep] ascending, relative to the visual block */
  void* hidden_out;          /* OUT [B,S',D] (16-byte aligned) */
  void* k_out;               /* OUT [B,S',H_kv,d_head] (16-byte aligned) */
  void* v_out;               /* OUT [B,S',H_kv,d_head] (16-byte aligned) */
  int64_t* pos_out;          /* OUT [n_pos,B,S'] */
  int32_t* head_sel;         /* OPTIONAL OUT [B,n_keep_heads] H*, ascending */
  float* head_var;           /* OPTIONAL OUT [B,H_q] u_h */
  float* score_out;          /* OPTIONAL OUT [B,K_in] p_i */
  void* const* events;       /* OPTIONAL [2*TREVS_INLLM_NUM_KERNELS] hipEvent_t */
  int32_t softmax;           /* trevs_softmax: domain of the attention softmax (0 = VISUAL) */
  const float* row_stats;    /* OPTIONAL [B,H_q,T_max,3] per text row, from the layer's own
                                attention pass: (log-sum-exp of the row's logits over its
                                softmax domain, natural log; sum and sum of squares of A over
                                the K_in visual columns).  When given, u_h is formed from them
                                and the row log-sum-exp is taken from them instead of being
                                recomputed from q and k (softmax is then ignored and lse_rest
                                must be NULL); the token score still recomputes the logits of
                                the H* heads.  Rows q >= T_b are not read for u_h. */
} trevs_inllm_args;

/* ------------------------------------------------------------------------
 * Diagnostics of the preliminary analysis (Sec. 3), computed on the same
 * tensors as the pruning stages.
 *
 * Text sensitivity of the attention heads (Eq. (1)).  One image paired with
 * two questions gives two stage-2 inputs of one shape, each laid out as for
 * trevs_inllm_prune (visual rows [P,P+K_in), text rows after them).  For
 * question c in {0,1} with T^c_b = text_len[c][b] valid text rows:
 *   A^c[h,q,:]  = the text->vision attention of trevs_inllm_prune, in the
 *                 same softmax domain (VISUAL, with lse_rest[c] if given, or
 *                 CAUSAL computed from q[c] and k[c])
 *   s^c_h       = (1/T^c_b) sum_{q<T^c_b} A^c[h,q,:]   the head's attention
 *                 distribution over the visual tokens for that question
 *   ts[b,h]     = 1 - cos(s^0_h, s^1_h)                                 Eq. (1)
 * head_var[c] optionally receives u_h of Eq. (8) for question c, so that the
 * heads can be ranked by attention variance as in the analysis.
 * ---------------------------------------------------------------------- */
typedef struct trevs_sensitivity_args {
  uint32_t struct_size;      /* sizeof(trevs_sensitivity_args) */
  int32_t B, S, P, K_in, T_max;  /* as in trevs_inllm_args; P + K_in + T_max <= S */
  int32_t H_q, H_kv;         /* query / key-value heads; H_q % H_kv == 0 */
  int32_t d_head;            /* 64, 128 or 256 */
  float scale;               /* logit scale > 0 */
  int32_t dtype;             /* trevs_dtype of q and k */
  const void* q[2];          /* per question [B,S,H_q,d_head] (16-byte aligned) */
  const void* k[2];          /* per question [B,S,H_kv,d_head] (16-byte aligned); may be one buffer */
  const int32_t* text_len[2];  /* per question [B] in 1..T_max, or NULL (= T_max) */
  const float* lse_rest[2];  /* OPTIONAL per question [B,H_q,T_max] non-visual log-sum-exp
                                (VISUAL softmax only) */
  float* ts;                 /* OUT [B,H_q] text sensitivity */
  float* profile[2];         /* OPTIONAL OUT per question [B,H_q,K_in] s^c_h */
  float* head_var[2];        /* OPTIONAL OUT per question [B,H_q] u_h */
  void* const* events;       /* OPTIONAL [2*TREVS_SENSITIVITY_NUM_KERNELS] hipEvent_t */
  int32_t softmax;           /* trevs_softmax, as in trevs_inllm_args (0 = VISUAL) */
} trevs_sensitivity_args;

size_t trevs_sensitivity_workspace_size(const trevs_sensitivity_args* args);
trevs_status trevs_text_sensitivity(const trevs_sensitivity_args* args, void* workspace,
                                    size_t workspace_bytes, void* stream);

/* Spearman rank correlation between visual saliency and textual relevance
 * within the top-K saliency set (Sec. 3).  sv, st [B,N] are s^v and s^t
 * (device, finite fp32; e.g. sal_out and rel_out of trevs_prellm_prune).
 * Per sample b: the K tokens first under (sv desc, index asc), the same
 * stable top-K as the pruning; the 1-based ranks of sv and of st over those
 * K tokens, tied values sharing the mean of the ranks they span; rho[b] =
 * the Pearson correlation of the two rank vectors, NaN when either is
 * constant (always for K = 1).  The rank sums are exact integers, so rho is
 * correctly rounded up to one division and one square root in double.
 * kept_idx: OPTIONAL OUT [B,K] the set, ascending.  N in
 * 1..TREVS_MAX_SELECT_N, K in 1..N. */
size_t trevs_spearman_workspace_size(int32_t B, int32_t N, int32_t K);
trevs_status trevs_topk_spearman(const float* sv, const float* st, int32_t B, int32_t N, int32_t K,
                                 double* rho, int32_t* kept_idx, void* workspace,
                                 size_t workspace_bytes, void* stream);

/* Workspace bytes the call needs for these arguments (0 on invalid args).
 * The workspace must be 256-byte aligned; its contents need no initialisation
 * and are garbage afterwards. */
size_t trevs_prellm_workspace_size(const trevs_prellm_args* args);
size_t trevs_inllm_workspace_size(const trevs_inllm_args* args);
size_t trevs_topk_workspace_size(int32_t B, int32_t N, int32_t K);

/* Stage 1 (Sec. 4.1, Eq. (2)-(7) and the pivot Top-K). */
trevs_status trevs_prellm_prune(const trevs_prellm_args* args, void* workspace,
                                size_t workspace_bytes, void* stream);

/* Stage 2 (Sec. 4.2, Eq. (8)-(9), Top-K_2 and compaction). */
trevs_status trevs_inllm_prune(const trevs_inllm_args* args, void* workspace,
                               size_t workspace_bytes, void* stream);

/* Stage 2 exactly as trevs_inllm_prune, for callers that cannot allocate
 * device memory: code under HIP graph capture, tight serving loops, and
 * harnesses that forbid allocation.  The caller passes inputs and outputs
 * only; the workspace is a static device array of
 * TREVS_NOALLOC_SCRATCH_BYTES inside the library, one per GPU, held from the
 * first call on that GPU until the process ends.  The call allocates and
 * frees nothing.
 *   - Runs on the calling thread's current device, which must be the
 *     stream's device.  The first call on a device looks up the array's
 *     address there (hipGetSymbolAddress); make that first call before
 *     capturing a graph.
 *   - Arguments whose workspace (trevs_inllm_workspace_size) exceeds
 *     TREVS_NOALLOC_SCRATCH_BYTES return TREVS_ERR_WORKSPACE before any
 *     launch; invalid arguments return the status trevs_inllm_prune gives.
 *   - Every call on a GPU shares that GPU's array: calls that overlap on one
 *     GPU (different streams, or host threads) race and give undefined
 *     results.  Serialise them, e.g. on one stream.  Calls in order on one
 *     stream are safe; no state carries from one call to the next. */
#define TREVS_NOALLOC_SCRATCH_BYTES ((size_t)16 << 20)
trevs_status trevs_inllm_prune_noalloc(const trevs_inllm_args* args, void* stream);

/* Stable top-K of each row of scores [B,N] (device, finite fp32): writes the
 * K kept indices of row b, ascending, to kept_idx [B,K].  N in
 * 1..TREVS_MAX_SELECT_N, K in 1..N.  Needs no workspace (pass NULL, 0). */
trevs_status trevs_topk_select(const float* scores, int32_t B, int32_t N, int32_t K,
                               int32_t* kept_idx, void* workspace, size_t workspace_bytes,
                               void* stream);

/* Static description of a status code. */
const char* trevs_status_string(trevs_status status);

/* Budget bookkeeping: floor(ratio * n + 1/2) clamped to [1, n] (0 if n < 1). */
int32_t trevs_keep_count(float ratio, int32_t n);

/* sizeof() of the argument structs as compiled into the library, for
 * bindings that mirror them. */
size_t trevs_prellm_args_size(void);
size_t trevs_inllm_args_size(void);
size_t trevs_sensitivity_args_size(void);

#ifdef __cplusplus
}
#endif

#endif /* TREVS_H */
