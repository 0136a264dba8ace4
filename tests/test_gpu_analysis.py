"""Diagnostics of the preliminary analysis (Sec. 3) on the GPU through the C
ABI, against the CPU oracle on the same seeded inputs: the text sensitivity
of every attention head between two questions (Eq. (1)), and the Spearman
correlation of s^v and s^t inside the top-K saliency set."""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2609_37581_amd import trevs
from parity import assert_scores_close, dev_tensor
from synthetic import WORKLOADS, sensitivity_inputs, stage1_inputs

pytestmark = pytest.mark.gpu


def run_sensitivity(inp, w, use_lse_rest=False, shared_k=True, softmax="visual"):
    q0 = dev_tensor(inp["q0"], w.dtype)
    q1 = dev_tensor(inp["q1"], w.dtype)
    k0 = dev_tensor(inp["k"], w.dtype)
    k1 = k0 if shared_k else k0.clone()
    tl0 = torch.from_numpy(inp["text_len0"]).cuda()
    tl1 = torch.from_numpy(inp["text_len1"]).cuda()
    lr0 = torch.from_numpy(inp["lse_rest0"]).cuda() if use_lse_rest else None
    lr1 = torch.from_numpy(inp["lse_rest1"]).cuda() if use_lse_rest else None
    ts, prof, hv = trevs.text_sensitivity(q0, k0, q1, k1, tl0, tl1, P=w.P, K_in=w.K1,
                                          lse_rest=lr0, lse_rest2=lr1, softmax=softmax)
    torch.cuda.synchronize()
    return dict(ts=ts.cpu().numpy(), profile0=prof[0].cpu().numpy(),
                profile1=prof[1].cpu().numpy(), head_var0=hv[0].cpu().numpy(),
                head_var1=hv[1].cpu().numpy())


def oracle_sensitivity(inp, w, use_lse_rest=False, softmax="visual"):
    return oracle.sensitivity(inp["q0"], inp["k"], inp["q1"], inp["k"], inp["text_len0"],
                              inp["text_len1"], w.dtype, P=w.P, K1=w.K1,
                              scale=1.0 / math.sqrt(w.d_h),
                              lse_rest1=inp["lse_rest0"] if use_lse_rest else None,
                              lse_rest2=inp["lse_rest1"] if use_lse_rest else None,
                              softmax=softmax)


# TS lies in [0, 1]; besides the relative bar it gets an absolute floor of
# 1e-6, the size of one fp32 rounding of the profiles it is computed from (a
# sample whose every head has TS = 0 leaves the relative bar no room at all).
TS_ATOL = 1e-6


def check_sensitivity(g, o):
    for key in ("profile0", "profile1", "head_var0", "head_var1"):
        assert_scores_close(g[key], o[key], key)
    err = np.abs(g["ts"] - o["ts"])
    tol = 1e-3 * np.abs(o["ts"]) + TS_ATOL
    assert (err <= tol).all(), (g["ts"], o["ts"])


SENS_CASES = {
    "llava15-b2-f32": WORKLOADS["llava15-b1-f32"].with_(B=2, text_len=("uniform", 5, 32)),
    "llava15-b4-bf16-ragged-text": WORKLOADS["llava15-b64-bf16"].with_(B=4),
    "qwen25vl-b1-bf16-gqa": WORKLOADS["qwen25vl-b4-bf16"].with_(B=1),
    # visual and text rows not multiples of 32, no prefix, GQA 12/3, d_head 64
    "ragged-bf16-dh64": WORKLOADS["llava15-b64-bf16"].with_(
        B=3, K1=77, M_max=45, text_len=("uniform", 1, 45), P=0, H_q=12, H_kv=3, d_h=64),
    "f32-dh256": WORKLOADS["llava15-b1-f32"].with_(B=2, K1=50, M_max=10, H_q=4, H_kv=2, d_h=256),
    "bf16-dh256-mqa": WORKLOADS["llava15-b64-bf16"].with_(
        B=2, K1=130, M_max=33, text_len=("uniform", 20, 33), H_q=8, H_kv=1, d_h=256),
    "one-visual-one-text-row": WORKLOADS["llava15-b1-f32"].with_(B=2, K1=1, M_max=1, H_q=4,
                                                                H_kv=4),
}


@pytest.mark.parametrize("name", list(SENS_CASES))
def test_text_sensitivity_parity(name):
    w = SENS_CASES[name]
    print(f"[sensitivity] {name}: B={w.B} K1={w.K1} T={w.T_max} H={w.H_q}/{w.H_kv} "
          f"dh={w.d_h} {w.dtype}", flush=True)
    inp = sensitivity_inputs(w)
    g = run_sensitivity(inp, w, shared_k=(w.B % 2 == 0))
    check_sensitivity(g, oracle_sensitivity(inp, w))


def test_text_sensitivity_full_row_softmax():
    w = WORKLOADS["llava15-b64-bf16"].with_(B=3)
    print("[sensitivity] lse_rest", flush=True)
    inp = sensitivity_inputs(w, with_lse_rest=True)
    g = run_sensitivity(inp, w, use_lse_rest=True)
    check_sensitivity(g, oracle_sensitivity(inp, w, use_lse_rest=True))


@pytest.mark.parametrize("name", ["llava15-b4-bf16-ragged-text", "ragged-bf16-dh64",
                                  "qwen25vl-b1-bf16-gqa"])
def test_text_sensitivity_causal_softmax(name):
    """Eq. (1) on the visual columns of each text row's whole causal
    attention row, computed by the library from q and k."""
    w = SENS_CASES[name]
    print(f"[sensitivity] causal {name}", flush=True)
    inp = sensitivity_inputs(w)
    g = run_sensitivity(inp, w, softmax="causal")
    check_sensitivity(g, oracle_sensitivity(inp, w, softmax="causal"))
    # a causal profile carries only the visual share of each row
    assert (g["profile0"].sum(-1) < 1).all()


def test_text_sensitivity_same_question_is_zero():
    """The same question twice gives bit-identical profiles, so Eq. (1) is 0
    up to the rounding of one square root."""
    w = WORKLOADS["llava15-b64-bf16"].with_(B=2)
    inp = sensitivity_inputs(w)
    inp["q1"] = inp["q0"]
    inp["text_len1"] = inp["text_len0"]
    g = run_sensitivity(inp, w, shared_k=False)
    assert np.array_equal(g["profile0"], g["profile1"])
    assert np.abs(g["ts"]).max() <= 1e-7


def test_text_sensitivity_planted_heads():
    """The planted question-dependent heads are the most text-sensitive ones
    (a property of the synthetic inputs, checked on the kernel's output)."""
    w = WORKLOADS["llava15-b64-bf16"].with_(B=2)
    inp = sensitivity_inputs(w)
    g = run_sensitivity(inp, w)
    for b in range(w.B):
        sens = inp["sensitive"][b]
        top = np.argsort(-g["ts"][b], kind="stable")[:sens.size]
        assert set(top.tolist()) == set(sens.tolist())


# ---------------------------------------------------------------- Spearman
def check_spearman(sv, st, k):
    rho, idx = trevs.topk_spearman(torch.from_numpy(sv).cuda(), torch.from_numpy(st).cuda(), k)
    rho = rho.cpu().numpy()
    idx = idx.cpu().numpy()
    for b in range(sv.shape[0]):
        want, want_idx = oracle.topk_saliency_spearman(sv[b].astype(np.float64),
                                                       st[b].astype(np.float64), k)
        assert idx[b].tolist() == want_idx.tolist(), b
        if math.isnan(want):
            assert math.isnan(rho[b]), (b, rho[b])
        else:
            # exact integer rank sums on both sides: one division and one sqrt apart
            assert abs(rho[b] - want) <= 1e-12, (b, rho[b], want)
    return rho


@pytest.mark.parametrize("N,K", [(1, 1), (7, 3), (576, 192), (577, 64), (2880, 640),
                                 (16384, 4096), (32768, 32768), (1000, 999), (100, 2)])
def test_spearman_random_with_ties(N, K):
    print(f"[spearman] N={N} K={K}", flush=True)
    rng = np.random.default_rng(N * 3 + K)
    sv = rng.random((3, N)).astype(np.float32)
    st = rng.random((3, N)).astype(np.float32)
    # ties in both signals: table values in s^v, exact zeros in s^t
    table = rng.random(32).astype(np.float32)
    m = rng.random((3, N)) < 0.3
    sv[m] = table[rng.integers(0, 32, size=m.sum())]
    st[rng.random((3, N)) < 0.2] = 0.0
    rho = check_spearman(sv, st, K)
    if K == 1:
        assert np.isnan(rho).all()


def test_spearman_monotone_and_constant_cases():
    N = 300
    x = np.random.default_rng(5).random(N).astype(np.float32)
    sv = np.stack([x, x, x, x])
    st = np.stack([2 * x + 1, -x, np.full(N, 0.5, np.float32), x * x])
    rho = check_spearman(sv, st, 120)
    assert rho[0] == 1.0 and rho[1] == -1.0 and math.isnan(rho[2]) and rho[3] == 1.0


def test_spearman_on_stage1_scores():
    """The analysis of Sec. 3 on the library's own s^v and s^t (stage 1 of the
    LLaVA-1.5 batch), top-K = K_1."""
    w = WORKLOADS["llava15-b64-bf16"].with_(B=8)
    inp = stage1_inputs(w)
    call = trevs.Prellm(dev_tensor(inp["cls_logits"], w.dtype), dev_tensor(inp["vis_feats"], w.dtype),
                        dev_tensor(inp["text_emb"], w.dtype), torch.from_numpy(inp["text_len"]).cuda(),
                        k_keep=w.K1, want_scores=True)
    call()
    torch.cuda.synchronize()
    check_spearman(call.sal.cpu().numpy(), call.rel.cpu().numpy(), w.K1)
