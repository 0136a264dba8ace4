"""Oracle pinned to hand-derived values (tests/golden/*.json, each citing the
equation it follows and giving its derivation)."""
import json
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


@pytest.mark.parametrize("name", ["mad_odd.json", "mad_even.json"])
def test_median_mad_normalise(name):
    g = load(name)
    s = np.array(g["s"], dtype=np.float64)
    s_hat, med, mad = oracle.robust_normalise(s, g["tau"], g["eps"])
    assert med == pytest.approx(g["med"], abs=1e-15)
    assert mad == pytest.approx(g["mad"], abs=1e-15)
    np.testing.assert_allclose(s_hat, g["s_hat"], rtol=1e-12, atol=1e-12)


def test_fusion():
    g = load("fusion.json")
    s = oracle.fuse_scores(g["sv_hat"], g["st_hat"], g["rho"], g["lam"])
    np.testing.assert_allclose(s, g["s"], rtol=1e-15)


def test_cosine_rms():
    g = load("cosine_rms.json")
    st = oracle.text_relevance(np.array(g["Z"], float), np.array(g["T"], float))
    np.testing.assert_allclose(st, g["s_t"], rtol=1e-12, atol=1e-15)


@pytest.mark.parametrize("name", ["cls_saliency.json", "cls_saliency_segments.json"])
def test_cls_saliency(name):
    g = load(name)
    sv = oracle.cls_saliency(np.array(g["logits"], float), g["n_seg"])
    np.testing.assert_allclose(sv, g["s_v"], rtol=1e-12)


def test_head_variance():
    g = load("head_variance.json")
    A, _ = oracle.t2v_attention(np.array(g["logits"], float))
    np.testing.assert_allclose(oracle.head_variance(A), g["u"], rtol=1e-12)


def test_token_score():
    g = load("token_score.json")
    A = np.array(g["A"], float)
    # feed the attention in as logits ln A: the softmax returns A itself
    A2, _ = oracle.t2v_attention(np.log(A))
    np.testing.assert_allclose(A2, A, rtol=1e-12)
    p = oracle.token_score(A2, g["heads"])
    np.testing.assert_allclose(p, g["p"], rtol=1e-12)


def test_topk_ties():
    g = load("topk_ties.json")
    for k, want in g["cases"]:
        assert oracle.topk_ascending(g["scores"], k).tolist() == want


def test_compaction_rows():
    g = load("compaction.json")
    rows = oracle.compaction_rows(g["S"], g["P"], g["K1"], g["kept"])
    assert rows.tolist() == g["rows"]


def test_budget_split():
    g = load("budget_split.json")
    for c in g["cases"]:
        got = oracle.budget_split_topk(c["sv"], c["st"], c["k"], c["rho"])
        assert got.tolist() == c["kept"], c
