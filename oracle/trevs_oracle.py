"""CPU oracle of the TReVS two-stage visual-token pruning path.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this module.  It shares no code with
the HIP library: it is a plain, slow, obviously-correct NumPy restatement of
the method, computed in float64 from the exact upcast of the input bits.

Paper: "TReVS: Integrating Textual Relevance and Visual Saliency for Efficient
Vision-Language Model Token Pruning" (arxiv 2609.37581).  Citations below name
the section and equation of the paper.

Stage 1 (Sec. 4.1, "Query-Aware Visual Redundancy Reduction"):
    Eq. (2)  [CLS]->patch attention softmax per head
    Eq. (3)  visual saliency s^v = head mean of that attention
    Eq. (4)  rectified cosine between L2-normalised text and visual features
    Eq. (5)  textual relevance s^t = RMS of Eq. (4) over the text tokens
    Eq. (6)  median/MAD robust normalisation, clamp, temperature
    Eq. (7)  fused pivot score with the consistency reward, then Top-K_r
    (context preservation by farthest point sampling follows Eq. (7))
Stage 2 (Sec. 4.2, "Query-Driven Visual Token Compression"):
    Eq. (8)  per-head text->vision attention variance u_h; top heads H*
    Eq. (9)  token score p_i = max over text rows of the H*-mean attention,
             then Top-K_2 and compaction of the sequence for later layers.
Diagnostics (Sec. 3, preliminary analysis):
    Eq. (1)  text sensitivity TS_h of a head between two questions
    the Spearman correlation of s^v and s^t inside the top-K saliency set

Readings where the paper is silent (each also listed in the design notes):
  * median = LOWER median, the order statistic of 0-based rank floor((n-1)/2);
    MAD = lower median of |s - Med|.
  * "textual ratio" rho: branch weights w_v = 2(1-rho), w_t = 2 rho applied to
    the normalised scores before Eq. (7); rho = 0.5 is Eq. (7) exactly.
  * top-K order: score descending, ties to the lower index; kept index lists
    are returned ascending.
  * multi-segment [CLS] input (tiles / frames): the softmax of Eq. (2) runs
    per segment of N / n_seg logits.
  * text padding: Eq. (5)'s mean runs over the M_b valid text rows; a zero
    vector is normalised with a norm floor of 1e-12.
  * Eq. (8) Var is the population variance (divide by K_1); text rows are the
    T_b valid ones; heads are query heads (under GQA, query head h reads KV
    head h // (H_q / H_kv)).
  * Eq. (8)/(9) softmax domain: the K_1 visual keys only, unless a per-row
    log-sum-exp of the non-visual keys ("lse_rest") is supplied, which gives
    the full-sequence softmax restricted to the visual columns; or the whole
    causal row computed from the sequence (softmax="causal": prefix keys,
    visual keys and the text keys up to the row itself).
  * compaction keeps the prefix rows, the K_2 selected visual rows (ascending)
    and the text rows, and copies the original position ids unchanged.
  * Eq. (1) (analysis of Sec. 3): a head's visual-token attention
    distribution for a question is the mean of its text->vision attention
    rows over the valid text rows; the Spearman correlation of Sec. 3 uses
    average ranks for ties and is NaN when either ranking is constant.
"""

import math

import numpy as np

# ----------------------------------------------------------------------------
# input decoding (the oracle's own; the library never calls this)
# ----------------------------------------------------------------------------


def to_f64(arr, dtype):
    """Exact float64 value of an input array given as float32 or as the raw
    uint16 bit patterns of bfloat16."""
    if dtype == "f32":
        return np.asarray(arr, dtype=np.float32).astype(np.float64)
    if dtype == "bf16":
        bits = np.asarray(arr, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
        return bits.view(np.float32).astype(np.float64)
    raise ValueError(f"unknown dtype {dtype!r}")


# ----------------------------------------------------------------------------
# Stage 1 steps, one sample at a time
# ----------------------------------------------------------------------------


def cls_saliency(cls_logits, n_seg=1):
    """Eq. (2)-(3), Sec. 4.1 "Visual saliency score".

    cls_logits: [H, N] pre-softmax [CLS]->patch logits (already scaled by
    1/sqrt(d_h)).  The softmax runs over the patch keys only, separately for
    each of the n_seg segments of N / n_seg patches; the saliency of patch i
    is the mean of its attention over the H heads.  Returns s^v, shape [N].
    """
    x = np.asarray(cls_logits, dtype=np.float64)
    H, N = x.shape
    if N % n_seg:
        raise ValueError("N must be a multiple of n_seg")
    seg = x.reshape(H, n_seg, N // n_seg)
    e = np.exp(seg - seg.max(axis=-1, keepdims=True))
    attn = e / e.sum(axis=-1, keepdims=True)
    return attn.reshape(H, N).sum(axis=0) / H


def l2_normalise_rows(x, floor=1e-12):
    """z / ||z||_2 per row (Sec. 4.1, before Eq. (4)), norm floored at 1e-12."""
    x = np.asarray(x, dtype=np.float64)
    n = np.sqrt((x * x).sum(axis=-1, keepdims=True))
    return x / np.maximum(n, floor)


def text_relevance(Z, T):
    """Eq. (4)-(5), Sec. 4.1 "Textual-relevance score".

    Z: [N, d'] projected visual features; T: [M, d'] embeddings of the M valid
    text tokens.  m_{j,i} = max(tbar_j . zbar_i, 0) and
    s^t_i = sqrt((1/M) sum_j m_{j,i}^2).  Returns s^t, shape [N].
    """
    zbar = l2_normalise_rows(Z)
    tbar = l2_normalise_rows(T)
    m = np.maximum(tbar @ zbar.T, 0.0)  # [M, N]
    return np.sqrt((m * m).sum(axis=0) / tbar.shape[0])


def lower_median(x):
    """Order statistic of 0-based rank floor((n-1)/2) (the 'Med' of Eq. (6))."""
    x = np.sort(np.asarray(x, dtype=np.float64))
    return x[(x.size - 1) // 2]


def median_abs_deviation(x, med):
    """MAD of Eq. (6): lower median of |x - Med|."""
    return lower_median(np.abs(np.asarray(x, dtype=np.float64) - med))


def robust_normalise(s, tau, eps):
    """Eq. (6): [(s - Med(s)) / (MAD(s) + eps)]_+ / tau.

    Returns (s_hat, Med, MAD)."""
    s = np.asarray(s, dtype=np.float64)
    med = lower_median(s)
    mad = median_abs_deviation(s, med)
    s_hat = np.maximum((s - med) / (mad + eps), 0.0) / tau
    return s_hat, med, mad


def fuse_scores(sv_hat, st_hat, rho=0.5, lam=1.0):
    """Eq. (7), Sec. 4.1 "Pivot token selection", with the textual-ratio
    branch weights a = 2(1-rho) sv_hat, b = 2 rho st_hat:
    s = max(a, b) + lam * sqrt(a * b)."""
    a = 2.0 * (1.0 - rho) * np.asarray(sv_hat, dtype=np.float64)
    b = 2.0 * rho * np.asarray(st_hat, dtype=np.float64)
    return np.maximum(a, b) + lam * np.sqrt(a * b)


def topk_ascending(scores, k):
    """TopK of Eq. (7) / Sec. 4.2: the k entries that come first under the
    order (score descending, index ascending), returned as ascending indices."""
    scores = np.asarray(scores, dtype=np.float64)
    n = scores.size
    if not 0 <= k <= n:
        raise ValueError("k out of range")
    order = sorted(range(n), key=lambda i: (-scores[i], i))
    return np.array(sorted(order[:k]), dtype=np.int64)


def budget_split_topk(sv, st, k, rho):
    """The "textual ratio" read as in the preliminary analysis (Sec. 3): the
    share of a token budget filled by textual relevance.  K_t = floor(rho k +
    1/2) tokens with the highest s^t, then the k - K_t tokens with the highest
    s^v among the others (each ranking: score descending, index ascending).
    Returns the union as ascending indices."""
    sv = np.asarray(sv, dtype=np.float64)
    st = np.asarray(st, dtype=np.float64)
    n = sv.size
    if not 0 <= k <= n:
        raise ValueError("k out of range")
    k_t = min(max(int(math.floor(rho * k + 0.5)), 0), k)
    by_text = [i for i in sorted(range(n), key=lambda i: (-st[i], i))][:k_t]
    taken = set(by_text)
    rest = [i for i in sorted(range(n), key=lambda i: (-sv[i], i)) if i not in taken]
    return np.array(sorted(by_text + rest[:k - k_t]), dtype=np.int64)


def farthest_point_sampling(Z, selected, k_div):
    """Context preservation (Sec. 4.1, after Eq. (7)): k_div tokens taken one at
    a time from the candidates outside `selected`, each the candidate whose
    cosine distance 1 - zbar_i . zbar_j to the nearest already-selected token
    is largest (ties to the lower index).  If nothing is selected yet the first
    pick is the lowest-index candidate.  Returns the picks in pick order."""
    zbar = l2_normalise_rows(Z)
    N = zbar.shape[0]
    sel = [int(i) for i in selected]
    picks = []
    for _ in range(k_div):
        taken = set(sel)
        cand = np.array([i for i in range(N) if i not in taken], dtype=np.int64)
        if cand.size == 0:
            break
        if sel:
            # distance of every candidate to its nearest selected token
            d = (1.0 - zbar[cand] @ zbar[np.array(sel)].T).min(axis=1)
            best = int(cand[int(np.argmax(d))])  # argmax returns the first max
        else:
            best = int(cand[0])
        picks.append(best)
        sel.append(best)
    return np.array(picks, dtype=np.int64)


def prellm_sample(cls_logits, Z, T, *, n_seg=1, k_keep, k_div=0, rho=0.5,
                  tau_v=1.4, tau_t=1.0, lam=1.0, eps=1e-8, ratio_mode="weights"):
    """Stage 1 for one sample (Sec. 4.1), all inputs float64.

    cls_logits [H_v, N]; Z [N, d']; T [M_b, d'] (valid text rows only).
    Returns a dict with s^v, s^t, the normalised scores, the fused score s,
    the medians / MADs, and kept_idx (ascending, K_1 = k_keep entries).
    ratio_mode "budget" takes the pivots by budget_split_topk on the raw
    scores instead of Eq. (6)-(7)."""
    sv = cls_saliency(cls_logits, n_seg)
    st = text_relevance(Z, T)
    sv_hat, med_v, mad_v = robust_normalise(sv, tau_v, eps)
    st_hat, med_t, mad_t = robust_normalise(st, tau_t, eps)
    s = fuse_scores(sv_hat, st_hat, rho, lam)
    k_piv = k_keep - k_div
    if ratio_mode == "budget":
        pivots = budget_split_topk(sv, st, k_piv, rho)
    elif ratio_mode == "weights":
        pivots = topk_ascending(s, k_piv)
    else:
        raise ValueError("ratio_mode")
    extra = farthest_point_sampling(Z, pivots, k_div) if k_div else np.zeros(0, np.int64)
    kept = np.sort(np.concatenate([pivots, extra]))
    return dict(sal=sv, rel=st, sal_hat=sv_hat, rel_hat=st_hat, score=s,
                med_v=med_v, mad_v=mad_v, med_t=med_t, mad_t=mad_t,
                pivots=pivots, diverse=extra, kept_idx=kept)


def prellm(cls_logits, Z, T, text_len, dtype, *, n_seg=1, k_keep, k_div=0,
           rho=0.5, tau_v=1.4, tau_t=1.0, lam=1.0, eps=1e-8, ratio_mode="weights"):
    """Stage 1 over a batch.  Array inputs are in the library's storage form
    (float32, or uint16 bf16 bits): cls_logits [B,H_v,N], Z [B,N,d'],
    T [B,M_max,d'], text_len [B] or None.  kept_feats is the row gather of the
    ORIGINAL input rows (bit copy)."""
    B = cls_logits.shape[0]
    M_max = T.shape[1]
    out = {k: [] for k in ("sal", "rel", "score", "kept_idx", "kept_feats",
                           "med_v", "mad_v", "med_t", "mad_t", "pivots", "diverse")}
    for b in range(B):
        mb = M_max if text_len is None else int(text_len[b])
        if not 1 <= mb <= M_max:
            raise ValueError("text_len out of range")
        r = prellm_sample(to_f64(cls_logits[b], dtype), to_f64(Z[b], dtype),
                          to_f64(T[b, :mb], dtype), n_seg=n_seg, k_keep=k_keep,
                          k_div=k_div, rho=rho, tau_v=tau_v, tau_t=tau_t,
                          lam=lam, eps=eps, ratio_mode=ratio_mode)
        for key in ("sal", "rel", "score", "kept_idx", "med_v", "mad_v",
                    "med_t", "mad_t", "pivots", "diverse"):
            out[key].append(r[key])
        out["kept_feats"].append(np.asarray(Z[b])[r["kept_idx"]])
    return {k: np.stack(v) if isinstance(v[0], np.ndarray) else np.array(v)
            for k, v in out.items()}


# ----------------------------------------------------------------------------
# Stage 2 steps, one sample at a time
# ----------------------------------------------------------------------------


def t2v_logits(q_text, k_vis, scale):
    """Scaled text->vision logits of the attention at layer l* (Sec. 4.2).

    q_text [T_b, H_q, d_h] query rows of the text tokens; k_vis [K_1, H_kv,
    d_h] key rows of the visual tokens.  Query head h reads KV head
    h // (H_q / H_kv).  Returns x [H_q, T_b, K_1]."""
    Tb, Hq, dh = q_text.shape
    K1, Hkv, _ = k_vis.shape
    G = Hq // Hkv
    x = np.empty((Hq, Tb, K1))
    for h in range(Hq):
        x[h] = scale * (q_text[:, h, :] @ k_vis[:, h // G, :].T)
    return x


def t2v_attention(x, lse_rest=None):
    """A_{T->V}[h, q, i] = exp(x - LSE[h, q]) where LSE is the log-sum-exp over
    the visual logits of the row, or, given lse_rest [H_q, T_b] (log-sum-exp of
    the row's non-visual logits), over the whole row.  Returns (A, LSE)."""
    m = x.max(axis=-1, keepdims=True)
    lse = m[..., 0] + np.log(np.exp(x - m).sum(axis=-1))
    if lse_rest is not None:
        lse = np.logaddexp(lse, np.asarray(lse_rest, dtype=np.float64))
    return np.exp(x - lse[..., None]), lse


def causal_rest_lse(q, k, *, P, K1, T_b, scale):
    """Log-sum-exp of each text row's non-visual logits over its causal row,
    from the sequence itself (the full-sequence softmax of Sec. 4.2 read as
    the model's causal attention at layer l*): text row t, at position
    P+K1+t, sees the prefix rows [0, P) and the text rows P+K1 .. P+K1+t.
    q [S, H_q, d_h], k [S, H_kv, d_h] float64 -> [H_q, T_b]."""
    Hq = q.shape[1]
    G = Hq // k.shape[1]
    out = np.empty((Hq, T_b))
    for h in range(Hq):
        qt = q[P + K1:P + K1 + T_b, h, :]
        kr = np.concatenate([k[:P, h // G, :], k[P + K1:P + K1 + T_b, h // G, :]])
        x = scale * (qt @ kr.T)
        for t in range(T_b):
            x[t, P + t + 1:] = -np.inf
        m = x.max(axis=1)
        out[h] = m + np.log(np.exp(x - m[:, None]).sum(axis=1))
    return out


def head_variance(A):
    """Eq. (8): u_h = mean over text rows q of the population variance over
    the K_1 visual columns of A[h, q, :].  A: [H_q, T_b, K_1] -> u [H_q]."""
    mean = A.mean(axis=-1, keepdims=True)
    var = ((A - mean) ** 2).mean(axis=-1)
    return var.mean(axis=-1)


def select_heads(u, n_keep):
    """High-variance head set H* (Sec. 4.2): the n_keep heads first under
    (u descending, head index ascending), returned ascending."""
    return topk_ascending(u, n_keep)


def token_score(A, heads):
    """Eq. (9): p_i = max over text rows q of (1/|H*|) sum_{h in H*} A[h,q,i]."""
    heads = np.asarray(heads, dtype=np.int64)
    return (A[heads].sum(axis=0) / heads.size).max(axis=0)


def compaction_rows(S, P, K1, kept):
    """Row map of the compacted sequence (Sec. 4.2, last paragraph): prefix
    rows [0, P), the kept visual rows P + kept (ascending), then every row
    after the visual block, [P + K1, S)."""
    kept = np.asarray(kept, dtype=np.int64)
    return np.concatenate([np.arange(P), P + kept, np.arange(P + K1, S)])


def inllm_sample(q, k, *, P, K1, T_b, n_keep, k_keep, scale, lse_rest=None,
                 heads=None, softmax="visual"):
    """Stage 2 scoring for one sample, inputs float64: q [S, H_q, d_h],
    k [S, H_kv, d_h] with visual rows [P, P+K1) and text rows
    [P+K1, P+K1+T_b).  `heads`, when given, replaces the selected head set
    (used to score with another side's head choice).  softmax="causal" takes
    each text row's softmax over its whole causal row (causal_rest_lse)
    instead of over the visual keys only.  Returns a dict."""
    if softmax == "causal":
        if lse_rest is not None:
            raise ValueError("lse_rest is for the visual softmax domain only")
        lse_rest = causal_rest_lse(q, k, P=P, K1=K1, T_b=T_b, scale=scale)
    x = t2v_logits(q[P + K1:P + K1 + T_b], k[P:P + K1], scale)
    A, lse = t2v_attention(x, lse_rest)
    u = head_variance(A)
    hsel = select_heads(u, n_keep) if heads is None else np.sort(np.asarray(heads))
    p = token_score(A, hsel)
    kept = topk_ascending(p, k_keep)
    return dict(head_var=u, head_sel=hsel, score=p, kept_idx=kept, lse=lse)


def inllm(q, k, v, hidden, pos, text_len, dtype, *, P, K1, n_keep, k_keep,
          scale, lse_rest=None, heads=None, softmax="visual"):
    """Stage 2 over a batch.  q [B,S,H_q,d_h], k, v [B,S,H_kv,d_h],
    hidden [B,S,D] in storage form; pos int64 [n_pos,B,S]; text_len [B] or
    None (= T_max = S - P - K1).  Outputs the compacted tensors as bit copies
    of the input rows.  `heads` optionally fixes H* per sample ([B, n_keep])."""
    B, S = hidden.shape[:2]
    T_max = S - P - K1
    res = {key: [] for key in ("head_var", "head_sel", "score", "kept_idx")}
    rows = []
    for b in range(B):
        tb = T_max if text_len is None else int(text_len[b])
        if not 1 <= tb <= T_max:
            raise ValueError("text_len out of range")
        r = inllm_sample(to_f64(q[b], dtype), to_f64(k[b], dtype), P=P, K1=K1,
                         T_b=tb, n_keep=n_keep, k_keep=k_keep, scale=scale,
                         lse_rest=None if lse_rest is None else lse_rest[b][:, :tb],
                         heads=None if heads is None else heads[b], softmax=softmax)
        for key in res:
            res[key].append(r[key])
        rows.append(compaction_rows(S, P, K1, r["kept_idx"]))
    rows = np.stack(rows)
    bidx = np.arange(B)[:, None]
    out = {key: np.stack(val) for key, val in res.items()}
    out["rows"] = rows
    out["hidden_out"] = np.asarray(hidden)[bidx, rows]
    out["k_out"] = np.asarray(k)[bidx, rows]
    out["v_out"] = np.asarray(v)[bidx, rows]
    out["pos_out"] = np.asarray(pos)[:, bidx, rows]
    return out


# ----------------------------------------------------------------------------
# Diagnostic quantities of the preliminary analysis (Sec. 3)
# ----------------------------------------------------------------------------


def visual_profile(A):
    """The attention distribution of each head over the visual tokens for one
    question (the s_h of Eq. (1)), read as the mean of A_{T->V}[h, q, :] over
    the question's valid text rows.  A [H_q, T_b, K_1] -> [H_q, K_1]."""
    return A.mean(axis=1)


def text_sensitivity(s1, s2):
    """Eq. (1): TS_h = 1 - cos(s_h^(1), s_h^(2)) between a head's visual
    profiles under two questions.  s1, s2 [H_q, K_1] -> [H_q]."""
    dot = (s1 * s2).sum(axis=-1)
    return 1.0 - dot / (np.linalg.norm(s1, axis=-1) * np.linalg.norm(s2, axis=-1))


def sensitivity_sample(q1, k1, q2, k2, *, P, K1, T1, T2, scale, lse_rest1=None,
                       lse_rest2=None, softmax="visual"):
    """Text sensitivity of every head for one image paired with two questions
    (Sec. 3, Eq. (1)).  Each question is a stage-2 input of the layout of
    inllm_sample (float64 q [S, H_q, d_h], k [S, H_kv, d_h]) with T1 / T2
    valid text rows.  Returns the sensitivities, both profiles and both
    questions' head variances u_h of Eq. (8)."""
    out = {}
    for c, (q, k, tb, rest) in enumerate(((q1, k1, T1, lse_rest1), (q2, k2, T2, lse_rest2))):
        if softmax == "causal":
            if rest is not None:
                raise ValueError("lse_rest is for the visual softmax domain only")
            rest = causal_rest_lse(q, k, P=P, K1=K1, T_b=tb, scale=scale)
        x = t2v_logits(q[P + K1:P + K1 + tb], k[P:P + K1], scale)
        A, _ = t2v_attention(x, rest)
        out[f"profile{c}"] = visual_profile(A)
        out[f"head_var{c}"] = head_variance(A)
    out["ts"] = text_sensitivity(out["profile0"], out["profile1"])
    return out


def sensitivity(q1, k1, q2, k2, text_len1, text_len2, dtype, *, P, K1, scale,
                lse_rest1=None, lse_rest2=None, softmax="visual"):
    """Batch form of sensitivity_sample on storage-form inputs
    ([B, S, H, d_h]); text_len* [B] or None (= T_max = S - P - K1)."""
    B, S = q1.shape[:2]
    T_max = S - P - K1
    keys = ("ts", "profile0", "profile1", "head_var0", "head_var1")
    res = {key: [] for key in keys}
    for b in range(B):
        t1 = T_max if text_len1 is None else int(text_len1[b])
        t2 = T_max if text_len2 is None else int(text_len2[b])
        if not (1 <= t1 <= T_max and 1 <= t2 <= T_max):
            raise ValueError("text_len out of range")
        r = sensitivity_sample(
            to_f64(q1[b], dtype), to_f64(k1[b], dtype), to_f64(q2[b], dtype), to_f64(k2[b], dtype),
            P=P, K1=K1, T1=t1, T2=t2, scale=scale,
            lse_rest1=None if lse_rest1 is None else lse_rest1[b][:, :t1],
            lse_rest2=None if lse_rest2 is None else lse_rest2[b][:, :t2], softmax=softmax)
        for key in keys:
            res[key].append(r[key])
    return {key: np.stack(val) for key, val in res.items()}


def average_ranks(x):
    """1-based ranks of x in ascending order; tied values share the mean of
    the ranks they span."""
    x = np.asarray(x, dtype=np.float64)
    n = x.size
    order = np.argsort(x, kind="stable")
    xs = x[order]
    ranks = np.empty(n)
    i = 0
    while i < n:
        j = i
        while j + 1 < n and xs[j + 1] == xs[i]:
            j += 1
        ranks[order[i:j + 1]] = (i + j) / 2.0 + 1.0
        i = j + 1
    return ranks


def spearman(x, y):
    """Spearman rank correlation: the Pearson correlation of the average ranks
    of x and of y; NaN when either rank vector is constant."""
    rx, ry = average_ranks(x), average_ranks(y)
    dx, dy = rx - rx.mean(), ry - ry.mean()
    den = math.sqrt((dx * dx).sum() * (dy * dy).sum())
    return float("nan") if den == 0.0 else float((dx * dy).sum() / den)


def topk_saliency_spearman(sv, st, k):
    """Sec. 3 analysis: the Spearman correlation between visual saliency and
    textual relevance over the k tokens with the highest saliency (the same
    stable top-K as the pruning).  Returns (rho, kept indices ascending)."""
    sv = np.asarray(sv, dtype=np.float64)
    st = np.asarray(st, dtype=np.float64)
    idx = topk_ascending(sv, k)
    return spearman(sv[idx], st[idx]), idx


def keep_count(ratio, n):
    """Budget bookkeeping: floor(ratio * n + 1/2) clamped to [1, n]."""
    return int(min(max(math.floor(ratio * n + 0.5), 1), n))
