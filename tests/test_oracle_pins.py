"""Oracle pinned to library routines, closed forms, invariants and brute force.

Each test checks the oracle against something other than itself: SciPy /
scikit-learn / NumPy / PyTorch routines that compute the same textbook
quantity, exhaustive search on tiny inputs, or a closed form of the paper's
definitions (Sec. 4.1, Eq. (2)-(7); Sec. 4.2, Eq. (8)-(9))."""
import itertools
import math

import numpy as np
import pytest
import scipy.special
import scipy.stats
import torch
from sklearn.metrics.pairwise import cosine_similarity

import oracle

RNG = np.random.default_rng(1234)


# ---------------------------------------------------------------- Eq. (2)-(3)
@pytest.mark.parametrize("H,N,n_seg", [(16, 576, 1), (4, 60, 5), (3, 7, 1)])
def test_saliency_matches_library_softmax(H, N, n_seg):
    x = RNG.standard_normal((H, N)) * 3
    want = np.zeros(N)
    L = N // n_seg
    for s in range(n_seg):
        want[s * L:(s + 1) * L] = scipy.special.softmax(x[:, s * L:(s + 1) * L], axis=1).mean(0)
    np.testing.assert_allclose(oracle.cls_saliency(x, n_seg), want, rtol=1e-13)


@pytest.mark.parametrize("n_seg", [1, 2, 5])
def test_saliency_sums_to_segments_and_uniform_case(n_seg):
    x = RNG.standard_normal((5, 40 * n_seg))
    assert oracle.cls_saliency(x, n_seg).sum() == pytest.approx(n_seg, rel=1e-13)
    c = np.full((5, 40 * n_seg), 2.5)
    np.testing.assert_allclose(oracle.cls_saliency(c, n_seg), n_seg / (40 * n_seg), rtol=1e-14)


# ---------------------------------------------------------------- Eq. (4)-(5)
def test_relevance_matches_sklearn_cosine():
    Z = RNG.standard_normal((50, 33))
    T = RNG.standard_normal((7, 33))
    cos = cosine_similarity(T, Z)  # [M, N]
    want = np.sqrt((np.maximum(cos, 0) ** 2).mean(axis=0))
    np.testing.assert_allclose(oracle.text_relevance(Z, T), want, rtol=1e-12)


def test_relevance_invariants():
    Z = RNG.standard_normal((40, 16))
    T = RNG.standard_normal((5, 16))
    st = oracle.text_relevance(Z, T)
    assert np.all(st >= 0) and np.all(st <= 1 + 1e-15)
    # scale invariance of both operands (cosine)
    np.testing.assert_allclose(oracle.text_relevance(3.0 * Z, 0.1 * T), st, rtol=1e-12)
    # text row order does not matter; a duplicated row of a one-row query
    # leaves the mean of squares unchanged
    np.testing.assert_allclose(oracle.text_relevance(Z, T[::-1]), st, rtol=1e-12)
    t1 = T[:1]
    np.testing.assert_allclose(oracle.text_relevance(Z, np.vstack([t1, t1, t1])),
                               oracle.text_relevance(Z, t1), rtol=1e-12)
    # with one text row the RMS is the rectified cosine itself
    np.testing.assert_allclose(oracle.text_relevance(Z, t1)[:, None].T,
                               np.maximum(cosine_similarity(t1, Z), 0), rtol=1e-12, atol=1e-15)
    # a visual token parallel to every text row scores 1; orthogonal scores 0
    t = np.zeros((3, 16)); t[:, 0] = [1, 2, 5]
    z = np.zeros((2, 16)); z[0, 0] = 4; z[1, 3] = 1
    np.testing.assert_allclose(oracle.text_relevance(z, t), [1.0, 0.0], atol=1e-15)


def test_relevance_zero_vector_guard():
    Z = np.zeros((3, 8)); Z[1, 2] = 1.0
    T = np.ones((2, 8))
    st = oracle.text_relevance(Z, T)
    assert np.all(np.isfinite(st)) and st[0] == 0.0 and st[2] == 0.0


# ---------------------------------------------------------------- Eq. (6)
@pytest.mark.parametrize("n", [1, 3, 5, 101, 577])
def test_lower_median_odd_equals_library_median(n):
    x = RNG.standard_normal(n)
    med = oracle.lower_median(x)
    assert med == np.median(x)
    mad = oracle.median_abs_deviation(x, med)
    assert mad == pytest.approx(scipy.stats.median_abs_deviation(x, scale=1.0), rel=1e-15)


@pytest.mark.parametrize("n", [2, 4, 6, 576, 2880])
def test_lower_median_even_is_the_rank_statistic(n):
    x = RNG.integers(0, 20, size=n).astype(float)  # with ties
    med = oracle.lower_median(x)
    k = (n - 1) // 2
    # order-statistic definition by counting, no sorting
    assert np.sum(x < med) <= k < np.sum(x <= med)
    assert med in x


def test_robust_normalise_shift_scale_equivariance():
    s = RNG.standard_normal(301)
    h1, m1, d1 = oracle.robust_normalise(s, 1.4, 0.0)
    h2, m2, d2 = oracle.robust_normalise(5.0 + 3.0 * s, 1.4, 0.0)
    assert m2 == pytest.approx(5.0 + 3.0 * m1) and d2 == pytest.approx(3.0 * d1)
    np.testing.assert_allclose(h1, h2, rtol=1e-12, atol=1e-12)
    # clamp: exactly the tokens at or below the median map to zero
    assert np.all((h1 == 0) == (s <= m1))


# ---------------------------------------------------------------- Eq. (7)
def test_fusion_special_cases():
    a = np.abs(RNG.standard_normal(100))
    b = np.abs(RNG.standard_normal(100))
    # rho = 0: pure saliency branch, rho = 1: pure text branch
    np.testing.assert_allclose(oracle.fuse_scores(a, b, 0.0, 1.0), 2 * a, rtol=1e-15)
    np.testing.assert_allclose(oracle.fuse_scores(a, b, 1.0, 1.0), 2 * b, rtol=1e-15)
    # lambda = 0 at rho = 0.5: the max of the two normalised scores
    np.testing.assert_allclose(oracle.fuse_scores(a, b, 0.5, 0.0), np.maximum(a, b), rtol=1e-15)
    # swap symmetry (s^v, rho) <-> (s^t, 1 - rho)
    for rho in (0.1, 0.3, 0.5, 0.9):
        np.testing.assert_allclose(oracle.fuse_scores(a, b, rho, 1.0),
                                   oracle.fuse_scores(b, a, 1 - rho, 1.0), rtol=1e-14)


def test_textual_ratio_zero_is_cls_only_selection():
    """rho = 0 keeps exactly the top-K of the raw [CLS] saliency when
    K <= #{s^v > Med} (the clamp only merges tokens below the median)."""
    for seed in range(5):
        rng = np.random.default_rng(seed)
        L = rng.standard_normal((4, 64))
        Z = rng.standard_normal((64, 12))
        T = rng.standard_normal((3, 12))
        r = oracle.prellm_sample(L, Z, T, k_keep=20, rho=0.0)
        sv = oracle.cls_saliency(L)
        assert np.sum(sv > np.sort(sv)[31]) >= 20
        assert r["kept_idx"].tolist() == sorted(np.argsort(-sv, kind="stable")[:20].tolist())
        r1 = oracle.prellm_sample(L, Z, T, k_keep=20, rho=1.0)
        st = oracle.text_relevance(Z, T)
        assert r1["kept_idx"].tolist() == sorted(np.argsort(-st, kind="stable")[:20].tolist())


# ---------------------------------------------------------------- Top-K
def _brute_topk(s, k):
    n = len(s)
    found = []
    for S in itertools.combinations(range(n), k):
        Sset = set(S)
        ok = all((s[i] > s[j]) or (s[i] == s[j] and i < j)
                 for i in Sset for j in range(n) if j not in Sset)
        if ok:
            found.append(list(S))
    assert len(found) == 1  # the (score desc, index asc) order is total
    return found[0]


@pytest.mark.parametrize("seed", range(6))
def test_topk_brute_force(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 11))
    s = rng.integers(0, 4, size=n).astype(float)  # many ties
    for k in range(0, n + 1):
        got = oracle.topk_ascending(s, k)
        assert got.tolist() == _brute_topk(s, k)
        assert np.all(np.diff(got) > 0)


def test_topk_matches_stable_argsort_and_identity():
    s = RNG.integers(0, 50, size=3000).astype(float)
    got = oracle.topk_ascending(s, 700)
    assert got.tolist() == sorted(np.argsort(-s, kind="stable")[:700].tolist())
    assert oracle.topk_ascending(s, 3000).tolist() == list(range(3000))


def test_stage1_brute_force_selection():
    """On a tiny sample the kept set is the unique K-subset that no excluded
    token beats under (fused score desc, index asc)."""
    rng = np.random.default_rng(7)
    L = rng.standard_normal((2, 9))
    Z = rng.standard_normal((9, 5))
    T = rng.standard_normal((2, 5))
    for k in (1, 3, 5, 9):
        r = oracle.prellm_sample(L, Z, T, k_keep=k)
        assert r["kept_idx"].tolist() == _brute_topk(r["score"], k)


# ---------------------------------------------------------------- FPS
def test_fps_on_circle():
    ang = np.deg2rad([0, 90, 180, 45, 200])
    Z = np.stack([np.cos(ang), np.sin(ang)], axis=1)
    # from {0 deg}: 180 (dist 2) first, then 90 (dist 1 to both 0 and 180)
    picks = oracle.farthest_point_sampling(Z, [0], 2)
    assert picks.tolist() == [2, 1]
    # from nothing: the lowest index candidate first
    assert oracle.farthest_point_sampling(Z, [], 1).tolist() == [0]


# ---------------------------------------------------------------- Eq. (8)-(9)
def _torch_attention(q_text, k_vis, scale):
    """Reference text->vision softmax with PyTorch (GQA by repeat_interleave)."""
    Hq, Hkv = q_text.shape[1], k_vis.shape[1]
    q = torch.from_numpy(q_text).permute(1, 0, 2)                 # [Hq, T, d]
    k = torch.from_numpy(k_vis).permute(1, 0, 2)                  # [Hkv, K, d]
    k = torch.repeat_interleave(k, Hq // Hkv, dim=0)
    return torch.softmax(scale * q @ k.transpose(1, 2), dim=-1).numpy()


@pytest.mark.parametrize("Hq,Hkv", [(4, 4), (6, 2), (8, 1)])
def test_t2v_attention_matches_torch_gqa(Hq, Hkv):
    q = RNG.standard_normal((5, Hq, 16))
    k = RNG.standard_normal((11, Hkv, 16))
    x = oracle.t2v_logits(q, k, 0.25)
    A, lse = oracle.t2v_attention(x)
    np.testing.assert_allclose(A, _torch_attention(q, k, 0.25), rtol=1e-12)
    np.testing.assert_allclose(lse, scipy.special.logsumexp(x, axis=-1), rtol=1e-13)


def test_lse_rest_gives_full_row_softmax():
    """Given the log-sum-exp of a row's non-visual logits, A equals the visual
    columns of the softmax over the whole row."""
    full = RNG.standard_normal((3, 4, 30)) * 2
    vis = slice(10, 22)
    rest = np.concatenate([full[..., :10], full[..., 22:]], axis=-1)
    A, _ = oracle.t2v_attention(full[..., vis], scipy.special.logsumexp(rest, axis=-1))
    np.testing.assert_allclose(A, scipy.special.softmax(full, axis=-1)[..., vis], rtol=1e-12)


def test_head_variance_library_and_closed_forms():
    x = RNG.standard_normal((6, 5, 40))
    A, _ = oracle.t2v_attention(x)
    u = oracle.head_variance(A)
    np.testing.assert_allclose(u, np.var(A, axis=-1, ddof=0).mean(-1), rtol=1e-12)
    # visual-only softmax rows sum to 1: Var = mean(A^2) - 1/K^2
    np.testing.assert_allclose(u, ((A ** 2).mean(-1) - 1 / 40 ** 2).mean(-1), rtol=1e-10)
    # uniform attention -> 0; a one-hot row -> (1/K)(1 - 1/K)
    assert oracle.head_variance(np.full((1, 2, 8), 1 / 8))[0] == pytest.approx(0, abs=1e-18)
    oh = np.zeros((1, 1, 8)); oh[0, 0, 3] = 1
    assert oracle.head_variance(oh)[0] == pytest.approx((1 / 8) * (1 - 1 / 8), rel=1e-14)


def test_head_ranking_permutation_equivariance():
    q = RNG.standard_normal((6, 8, 16)) * np.linspace(0.5, 2, 8)[None, :, None]
    k = RNG.standard_normal((20, 8, 16))
    u = oracle.head_variance(oracle.t2v_attention(oracle.t2v_logits(q, k, 0.25))[0])
    perm = RNG.permutation(8)
    up = oracle.head_variance(oracle.t2v_attention(
        oracle.t2v_logits(q[:, perm], k[:, perm], 0.25))[0])
    np.testing.assert_allclose(up, u[perm], rtol=1e-12)
    sel = oracle.select_heads(u, 4)
    selp = oracle.select_heads(up, 4)
    assert sorted(perm[selp].tolist()) == sel.tolist()


def test_token_score_special_cases():
    x = RNG.standard_normal((4, 1, 12))
    A, _ = oracle.t2v_attention(x)
    # one text row, one head: the score is that head's softmax row
    np.testing.assert_allclose(oracle.token_score(A, [2]), scipy.special.softmax(x[2, 0]), rtol=1e-13)
    # all heads: the all-head mean used by the ablation's "All Heads" variant
    x2 = RNG.standard_normal((4, 3, 12))
    A2, _ = oracle.t2v_attention(x2)
    np.testing.assert_allclose(oracle.token_score(A2, range(4)),
                               A2.mean(axis=0).max(axis=0), rtol=1e-13)


def test_inllm_identity_when_keeping_everything():
    B, S, P, K1, T = 2, 14, 3, 6, 5
    q = RNG.standard_normal((B, S, 4, 8)).astype(np.float32)
    k = RNG.standard_normal((B, S, 2, 8)).astype(np.float32)
    v = RNG.standard_normal((B, S, 2, 8)).astype(np.float32)
    hid = RNG.standard_normal((B, S, 10)).astype(np.float32)
    pos = np.tile(np.arange(S), (3, B, 1))
    r = oracle.inllm(q, k, v, hid, pos, None, "f32", P=P, K1=K1, n_keep=2,
                     k_keep=K1, scale=1 / math.sqrt(8))
    assert np.array_equal(r["hidden_out"], hid)
    assert np.array_equal(r["k_out"], k) and np.array_equal(r["pos_out"], pos)


def test_keep_counts_of_the_sweep():
    k1 = [oracle.keep_count(r, 576) for r in (0.5, 0.25, 1 / 9, 1 / 18)]
    assert k1 == [288, 144, 64, 32]
    assert [oracle.keep_count(1 / 3, k) for k in k1] == [96, 48, 21, 11]


def test_bf16_decoding():
    bits = np.array([0x3F80, 0xC000, 0x0000, 0x8000, 0x3E80], dtype=np.uint16)
    np.testing.assert_array_equal(oracle.to_f64(bits, "bf16"), [1.0, -2.0, 0.0, -0.0, 0.25])
    t = torch.tensor([1.5, -3.25, 1e-3], dtype=torch.bfloat16)
    np.testing.assert_array_equal(oracle.to_f64(t.view(torch.uint16).numpy(), "bf16"),
                                  t.double().numpy())


# ---------------------------------------------- textual ratio as a budget split
@pytest.mark.parametrize("seed", range(4))
def test_budget_split_extremes_and_invariants(seed):
    """rho = 0 and rho = 1 reduce to one plain top-K; in general the kept set
    holds the K_t best by s^t, the rest come from the top-k by s^v, and the
    budget is spent exactly."""
    rng = np.random.default_rng(seed)
    n, k = 40, 13
    sv = rng.integers(0, 9, size=n).astype(float)   # many ties
    st = rng.integers(0, 9, size=n).astype(float)
    assert oracle.budget_split_topk(sv, st, k, 0.0).tolist() == oracle.topk_ascending(sv, k).tolist()
    assert oracle.budget_split_topk(sv, st, k, 1.0).tolist() == oracle.topk_ascending(st, k).tolist()
    for rho in (0.2, 0.5, 0.8):
        got = oracle.budget_split_topk(sv, st, k, rho)
        k_t = int(np.floor(rho * k + 0.5))
        assert got.size == k and np.all(np.diff(got) > 0)
        by_text = set(oracle.topk_ascending(st, k_t).tolist())
        assert by_text <= set(got.tolist())
        assert set(got.tolist()) - by_text <= set(oracle.topk_ascending(sv, k).tolist())


def test_budget_split_brute_force_small():
    """Exhaustive check on tiny inputs: among all k-subsets, the kept set is the
    one whose s^t part is the K_t first tokens in (s^t desc, index asc) order
    and whose remaining part is lexicographically best in (s^v desc, index
    asc) order among the subsets that contain that s^t part."""
    rng = np.random.default_rng(7)
    for _ in range(20):
        n = int(rng.integers(2, 8))
        k = int(rng.integers(1, n + 1))
        rho = float(rng.choice([0.0, 0.3, 0.5, 0.75, 1.0]))
        sv = rng.integers(0, 3, size=n).astype(float)
        st = rng.integers(0, 3, size=n).astype(float)
        k_t = int(np.floor(rho * k + 0.5))
        first_t = sorted(range(n), key=lambda i: (-st[i], i))[:k_t]
        best = None
        for S in itertools.combinations(range(n), k):
            if not set(first_t) <= set(S):
                continue
            rest = sorted((i for i in S if i not in first_t), key=lambda i: (-sv[i], i))
            key = [(-sv[i], i) for i in rest]
            if best is None or key < best[0]:
                best = (key, list(S))
        assert oracle.budget_split_topk(sv, st, k, rho).tolist() == best[1]


# ------------------------------------------------------- Sec. 3 diagnostics
def test_visual_profile_rows_and_single_row():
    """Under the visual-only softmax each attention row sums to 1, so a
    head's profile (the mean over text rows) sums to 1; with one text row it
    is that row's softmax (library softmax)."""
    x = RNG.standard_normal((4, 7, 30)) * 2
    A, _ = oracle.t2v_attention(x)
    prof = oracle.visual_profile(A)
    assert prof.shape == (4, 30)
    np.testing.assert_allclose(prof.sum(axis=-1), 1.0, rtol=1e-13)
    one, _ = oracle.t2v_attention(x[:, :1])
    np.testing.assert_allclose(oracle.visual_profile(one), scipy.special.softmax(x[:, 0], axis=-1),
                               rtol=1e-13)


def test_text_sensitivity_library_and_closed_forms():
    """Eq. (1) against scikit-learn's cosine similarity, plus closed forms:
    identical profiles give 0, profiles on disjoint tokens give 1, uniform
    against one-hot over K tokens gives 1 - 1/sqrt(K); scaling a profile
    changes nothing and the measure is symmetric."""
    s1 = RNG.random((6, 50))
    s2 = RNG.random((6, 50))
    want = 1.0 - np.diag(cosine_similarity(s1, s2))
    np.testing.assert_allclose(oracle.text_sensitivity(s1, s2), want, rtol=1e-12)
    np.testing.assert_allclose(oracle.text_sensitivity(s2, s1), want, rtol=1e-12)
    np.testing.assert_allclose(oracle.text_sensitivity(3.0 * s1, 0.5 * s2), want, rtol=1e-12)
    np.testing.assert_allclose(oracle.text_sensitivity(s1, s1), 0.0, atol=1e-15)
    K = 64
    uni = np.full((1, K), 1.0 / K)
    hot = np.zeros((1, K))
    hot[0, 5] = 1.0
    assert oracle.text_sensitivity(uni, hot)[0] == pytest.approx(1 - 1 / math.sqrt(K), rel=1e-14)
    a = np.zeros((1, K))
    b = np.zeros((1, K))
    a[0, :10] = RNG.random(10)
    b[0, 10:] = RNG.random(K - 10)
    assert oracle.text_sensitivity(a, b)[0] == 1.0


@pytest.mark.parametrize("Hq,Hkv", [(4, 4), (6, 2)])
def test_sensitivity_sample_matches_torch(Hq, Hkv):
    """Both questions' profiles, head variances and sensitivities against an
    independent float64 PyTorch computation (GQA by repeat_interleave,
    library softmax), with different text lengths per question."""
    S, P, K1, dh = 40, 3, 20, 16
    q1, q2 = RNG.standard_normal((2, S, Hq, dh))
    k1, k2 = RNG.standard_normal((2, S, Hkv, dh))
    T1, T2, scale = 9, 4, 0.3
    r = oracle.sensitivity_sample(q1, k1, q2, k2, P=P, K1=K1, T1=T1, T2=T2, scale=scale)
    prof = []
    for q, k, tb in ((q1, k1, T1), (q2, k2, T2)):
        qt = torch.from_numpy(q[P + K1:P + K1 + tb]).permute(1, 0, 2)
        kv = torch.from_numpy(k[P:P + K1]).permute(1, 0, 2).repeat_interleave(Hq // Hkv, dim=0)
        A = torch.softmax(scale * qt @ kv.transpose(1, 2), dim=-1)
        prof.append(A.mean(dim=1).numpy())
        c = len(prof) - 1
        np.testing.assert_allclose(r[f"profile{c}"], prof[c], rtol=1e-12)
        np.testing.assert_allclose(r[f"head_var{c}"], A.var(dim=-1, unbiased=False).mean(dim=1).numpy(),
                                   rtol=1e-11)
    want = 1.0 - np.diag(cosine_similarity(prof[0], prof[1]))
    np.testing.assert_allclose(r["ts"], want, rtol=1e-10)
    same = oracle.sensitivity_sample(q1, k1, q1, k1, P=P, K1=K1, T1=T1, T2=T1, scale=scale)
    np.testing.assert_allclose(same["ts"], 0.0, atol=1e-14)


def test_average_ranks_library_and_hand_example():
    assert oracle.average_ranks([10.0, 20.0, 20.0, 5.0]).tolist() == [2.0, 3.5, 3.5, 1.0]
    for _ in range(5):
        x = RNG.integers(0, 7, size=40).astype(np.float64)
        np.testing.assert_array_equal(oracle.average_ranks(x), scipy.stats.rankdata(x, method="average"))
    x = np.array([0.0, -0.0, 1.0])
    assert oracle.average_ranks(x).tolist() == [1.5, 1.5, 3.0]


def test_spearman_library_closed_form_and_invariants():
    """Against SciPy (with ties), the tie-free closed form
    1 - 6 sum d^2 / (n (n^2 - 1)), invariance under increasing maps, the
    perfectly (anti)monotone cases and the constant case."""
    for n in (5, 33, 200):
        x = RNG.integers(0, 9, size=n).astype(np.float64)
        y = RNG.integers(0, 5, size=n).astype(np.float64)
        assert oracle.spearman(x, y) == pytest.approx(scipy.stats.spearmanr(x, y)[0], rel=1e-12, abs=1e-15)
        x = RNG.permutation(n).astype(np.float64)
        y = RNG.permutation(n).astype(np.float64)
        d = x - y
        closed = 1 - 6 * (d * d).sum() / (n * (n * n - 1))
        assert oracle.spearman(x, y) == pytest.approx(closed, rel=1e-12, abs=1e-15)
        assert oracle.spearman(np.exp(x / n), y ** 3) == pytest.approx(closed, rel=1e-12, abs=1e-15)
        assert oracle.spearman(x, 2 * x + 1) == pytest.approx(1.0, rel=1e-15)
        assert oracle.spearman(x, -x) == pytest.approx(-1.0, rel=1e-15)
    assert math.isnan(oracle.spearman(np.ones(5), np.arange(5.0)))
    assert math.isnan(oracle.spearman([1.0], [2.0]))


def test_topk_saliency_spearman_brute_force():
    """The set is the top-K of s^v in the pruning's stable order, found here
    by sorting (-s^v, index) tuples; K = N correlates the whole vectors."""
    for seed in range(6):
        rng = np.random.default_rng(seed)
        N = 25
        sv = rng.integers(0, 6, size=N).astype(np.float64)
        st = rng.standard_normal(N)
        st[rng.random(N) < 0.3] = 0.0
        K = int(rng.integers(2, N))
        idx = sorted(sorted(range(N), key=lambda i: (-sv[i], i))[:K])
        rho, got = oracle.topk_saliency_spearman(sv, st, K)
        assert got.tolist() == idx
        want = scipy.stats.spearmanr(sv[idx], st[idx])[0]
        if math.isnan(want):
            assert math.isnan(rho)
        else:
            assert rho == pytest.approx(want, rel=1e-12, abs=1e-15)
        full, _ = oracle.topk_saliency_spearman(sv, st, N)
        assert full == pytest.approx(scipy.stats.spearmanr(sv, st)[0], rel=1e-12, abs=1e-15)


@pytest.mark.parametrize("Hq,Hkv,P", [(4, 4, 3), (6, 2, 0)])
def test_causal_softmax_matches_torch_masked_attention(Hq, Hkv, P):
    """softmax="causal": the visual columns of each text row's softmax over
    its whole causal row, against an independent float64 PyTorch causal
    attention over the full sequence (GQA by repeat_interleave), and u_h and
    p of Eq. (8)-(9) on those attention rows."""
    K1, T, dh, scale = 13, 7, 8, 0.4
    S = P + K1 + T + 2  # rows after the text are not attended by it
    q = RNG.standard_normal((S, Hq, dh))
    k = RNG.standard_normal((S, Hkv, dh))
    Tb = 5
    qt = torch.from_numpy(q).permute(1, 0, 2)
    kt = torch.from_numpy(k).permute(1, 0, 2).repeat_interleave(Hq // Hkv, dim=0)
    x = scale * qt @ kt.transpose(1, 2)
    pos = torch.arange(S)
    x = x.masked_fill(pos[None, :] > pos[:, None], float("-inf"))
    A_full = torch.softmax(x, dim=-1)[:, P + K1:P + K1 + Tb, P:P + K1].numpy()
    r = oracle.inllm_sample(q, k, P=P, K1=K1, T_b=Tb, n_keep=2, k_keep=4, scale=scale,
                            softmax="causal")
    u = ((A_full - A_full.mean(-1, keepdims=True)) ** 2).mean(-1).mean(-1)
    np.testing.assert_allclose(r["head_var"], u, rtol=1e-10)
    p = (A_full[r["head_sel"]].sum(0) / 2).max(0)
    np.testing.assert_allclose(r["score"], p, rtol=1e-10)
    rest = oracle.causal_rest_lse(q, k, P=P, K1=K1, T_b=Tb, scale=scale)
    A, _ = oracle.t2v_attention(oracle.t2v_logits(q[P + K1:P + K1 + Tb], k[P:P + K1], scale), rest)
    np.testing.assert_allclose(A, A_full, rtol=1e-11)
    # each row's attention over the visual block sums to less than 1
    assert (A.sum(-1) < 1).all()
