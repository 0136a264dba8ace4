"""The seeded generators: determinism, planted structure, storage rounding."""
import numpy as np
import torch

import oracle
from synthetic import WORKLOADS, stage1_inputs, stage2_inputs, sweep, to_storage


def small(name, **kw):
    return WORKLOADS[name].with_(**kw)


def test_same_seed_same_bytes():
    w = small("llava15-b64-bf16", B=3)
    a, b = stage1_inputs(w), stage1_inputs(w)
    for key in ("cls_logits", "vis_feats", "text_emb", "text_len"):
        assert a[key].tobytes() == b[key].tobytes()
    c, d = stage2_inputs(w), stage2_inputs(w)
    for key in ("q", "k", "v", "hidden", "pos"):
        assert c[key].tobytes() == d[key].tobytes()


def test_planted_cosine_and_padding():
    w = small("llava15-b64-bf16", B=4)
    s = stage1_inputs(w)
    for b in range(w.B):
        L = int(s["text_len"][b])
        assert 16 <= L <= 64
        assert not s["text_emb"][b, L:].any()
    w32 = WORKLOADS["llava15-b1-f32"]
    s = stage1_inputs(w32)
    Z = oracle.to_f64(s["vis_feats"][0], "f32")
    T = oracle.to_f64(s["text_emb"][0], "f32")
    u = T.mean(0) / np.linalg.norm(T.mean(0))
    cos = Z[s["matched"][0]] @ u / np.linalg.norm(Z[s["matched"][0]], axis=1)
    np.testing.assert_allclose(cos, 0.6, atol=1e-6)


def test_bf16_storage_is_round_to_nearest_even():
    x = np.random.default_rng(0).standard_normal(10000) * 10
    ours = to_storage(x, "bf16")
    ref = torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).view(torch.uint16).numpy()
    assert np.array_equal(ours, ref)


def test_block_tokens_and_positions_qwen_layout():
    w = WORKLOADS["qwen25vl-b4-bf16"].with_(B=1, N=16384, d=8, D=8, K1=64, K2=16, M_max=4)
    s = stage1_inputs(w)
    qm = s["matched"][0]
    assert qm.size == 256 and np.unique(qm).size == 256
    s2 = stage2_inputs(w)
    assert s2["pos"].shape == (3, 1, w.S)


def test_sweep_grid():
    g = sweep()
    assert len(g) == 4 * 5 * 4
    assert sorted({(c.K1, c.K2) for c in g}) == [(32, 11), (64, 21), (144, 48), (288, 96)]


def test_stage2_tie_stress_copies_visual_key_rows():
    w = WORKLOADS["sweep-llava15-b32-bf16"].with_(B=2, K1=144, D=8, tie_stress=True)
    s = stage2_inputs(w)
    for b in range(w.B):
        vis = s["k"][b, w.P:w.P + w.K1].reshape(w.K1, -1)
        n_distinct = np.unique(vis, axis=0).shape[0]
        assert n_distinct == w.K1 - w.K1 // 4  # every copy repeats a prototype row
    plain = stage2_inputs(w.with_(tie_stress=False))
    assert np.unique(plain["k"][0, w.P:w.P + w.K1].reshape(w.K1, -1), axis=0).shape[0] == w.K1
