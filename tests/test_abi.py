"""The C ABI without a GPU: the library loads, exports every function the
header declares, mirrors the argument structs, and rejects invalid arguments
on the host before any HIP call."""
import ctypes
import os
import re
import subprocess

import pytest

from paper_2609_37581_amd import trevs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "trevs.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(trevs_\w+)\s*\(", text)))


def test_header_compiles_as_c99():
    r = subprocess.run(["gcc", "-std=c99", "-Wall", "-Werror", "-fsyntax-only", "-x", "c", HEADER],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr


def test_every_declared_symbol_is_exported():
    L = trevs.lib()
    names = declared_functions()
    assert len(names) >= 10
    for n in names:
        assert hasattr(L, n), n
    out = subprocess.run(["nm", "-D", "--defined-only", trevs.LIB_PATH], capture_output=True,
                         text=True).stdout
    exported = set(re.findall(r" T (trevs_\w+)", out))
    assert set(names) <= exported


def test_struct_mirror_sizes():
    L = trevs.lib()
    assert L.trevs_prellm_args_size() == ctypes.sizeof(trevs.PrellmArgs) == 168
    assert L.trevs_inllm_args_size() == ctypes.sizeof(trevs.InllmArgs) == 208
    assert L.trevs_sensitivity_args_size() == ctypes.sizeof(trevs.SensitivityArgs) == 168


def test_status_strings_and_keep_count():
    L = trevs.lib()
    for s in range(5):
        assert L.trevs_status_string(s)
    assert [trevs.keep_count(r, 576) for r in (0.5, 0.25, 1 / 9, 1 / 18)] == [288, 144, 64, 32]
    assert trevs.keep_count(0.0, 10) == 1 and trevs.keep_count(2.0, 10) == 10
    assert trevs.keep_count(0.5, 0) == 0


def _prellm(**kw):
    a = trevs.PrellmArgs()
    a.struct_size = ctypes.sizeof(a)
    a.B, a.N, a.n_seg, a.H_v, a.d, a.M_max, a.k_keep = 2, 576, 1, 16, 4096, 32, 192
    a.textual_ratio, a.tau_v, a.tau_t, a.lambda_, a.eps = 0.5, 1.4, 1.0, 1.0, 1e-8
    a.dtype = trevs.TREVS_BF16
    base = 1 << 40
    a.cls_logits, a.vis_feats, a.text_emb = base, base + (1 << 32), base + (2 << 32)
    a.kept_idx, a.kept_feats = base + (3 << 32), base + (4 << 32)
    for k, v in kw.items():
        setattr(a, k, v)
    return a


def _inllm(**kw):
    a = trevs.InllmArgs()
    a.struct_size = ctypes.sizeof(a)
    a.B, a.S, a.P, a.K_in, a.T_max = 2, 259, 35, 192, 32
    a.H_q, a.H_kv, a.d_head, a.D, a.n_pos = 32, 32, 128, 4096, 1
    a.n_keep_heads, a.k_keep, a.scale, a.dtype = 16, 64, 128 ** -0.5, trevs.TREVS_BF16
    base = 1 << 40
    for i, name in enumerate(["q", "k", "v", "hidden", "pos", "kept_idx", "hidden_out", "k_out",
                              "v_out", "pos_out"]):
        setattr(a, name, base + (i << 32))
    for k, v in kw.items():
        setattr(a, k, v)
    return a


def test_workspace_size_is_positive_for_valid_args():
    L = trevs.lib()
    assert L.trevs_prellm_workspace_size(ctypes.byref(_prellm())) > 0
    assert L.trevs_prellm_workspace_size(ctypes.byref(_prellm(ratio_mode=1))) > 0
    # the diversity set adds the Gram matrices of the batch: B * N * N floats
    plain = L.trevs_prellm_workspace_size(ctypes.byref(_prellm()))
    assert L.trevs_prellm_workspace_size(ctypes.byref(_prellm(k_div=48))) >= plain + 2 * 576 * 576 * 4
    assert L.trevs_inllm_workspace_size(ctypes.byref(_inllm())) > 0
    # the causal softmax adds the non-visual statistics of every text row
    vis = L.trevs_inllm_workspace_size(ctypes.byref(_inllm()))
    assert L.trevs_inllm_workspace_size(ctypes.byref(_inllm(softmax=1))) >= vis + 2 * 32 * 32 * 16


def test_small_grids_reserve_split_partials():
    """A grid with fewer tiles than compute units splits the relevance pass
    over the feature dimension and the token score over the selected heads;
    the partial sums those splits write live in the workspace, so its size
    must cover at least two splits' worth."""
    L = trevs.lib()
    # 2 samples x 3 token tiles: split; 200 samples: one tile per CU or more
    small = L.trevs_prellm_workspace_size(ctypes.byref(_prellm()))
    big = L.trevs_prellm_workspace_size(ctypes.byref(_prellm(B=200)))
    assert small >= 2 * 2 * (32 + 1) * 576 * 4  # [B, splits >= 2, M_max + 1, N] floats
    assert big < 200 * 576 * 64                  # no partials: about 40 bytes per token
    # token score: 2 samples x 3 tiles of 64 keys split the 16 selected heads
    small = L.trevs_inllm_workspace_size(ctypes.byref(_inllm()))
    assert small >= 2 * 2 * 32 * 192 * 4        # [B, splits >= 2, T_max, K_in] floats
    # a text so long that the split's partials would pass 256 MB runs unsplit
    long_text = L.trevs_prellm_workspace_size(ctypes.byref(_prellm(B=1, M_max=16384)))
    assert 0 < long_text < (64 << 20)


@pytest.mark.parametrize("bad,code", [
    (dict(k_keep=0), 1), (dict(k_keep=577), 1), (dict(n_seg=5), 1), (dict(d=4095), 1),
    (dict(textual_ratio=-0.1), 1), (dict(textual_ratio=float("nan")), 1), (dict(tau_v=0.0), 1),
    (dict(eps=-1.0), 1), (dict(dtype=7), 1), (dict(vis_feats=None), 1),
    (dict(kept_feats=(1 << 40) + 8), 1), (dict(struct_size=10), 1), (dict(k_div=192), 1),
    (dict(k_div=-1), 1), (dict(k_div=3, div_idx=(1 << 40) + (5 << 32) + 2), 1),
    (dict(N=70000, k_keep=10, n_seg=1), 2),
    (dict(N=40000, k_keep=10, n_seg=1, k_div=3), 2),  # diversity set: N <= 32768
    (dict(kept_feats=(1 << 40) + (1 << 32) + 4096 * 64), 1),  # overlaps vis_feats
    (dict(ratio_mode=2), 1), (dict(ratio_mode=1, score_out=(1 << 40) + (5 << 32)), 1),
    (dict(ratio_mode=1, norm_stats=(1 << 40) + (5 << 32)), 1),
])
def test_prellm_rejects_before_launch(bad, code):
    L = trevs.lib()
    a = _prellm(**bad)
    assert L.trevs_prellm_workspace_size(ctypes.byref(a)) == 0
    assert L.trevs_prellm_prune(ctypes.byref(a), None, 0, None) == code


def test_selection_limits():
    """One selection ranks up to 65,536 tokens (64 per thread); the diversity
    set's Gram matrix limits it to 32,768."""
    L = trevs.lib()
    assert trevs.MAX_SELECT_N == 65536 and trevs.MAX_FPS_N == 32768
    assert L.trevs_prellm_workspace_size(ctypes.byref(_prellm(N=65536, k_keep=10, n_seg=1))) > 0
    assert L.trevs_prellm_workspace_size(ctypes.byref(_prellm(N=65537, k_keep=10, n_seg=1))) == 0
    assert L.trevs_prellm_workspace_size(ctypes.byref(_prellm(N=32768, k_keep=10, n_seg=1, k_div=3))) > 0
    assert L.trevs_prellm_workspace_size(ctypes.byref(_prellm(N=32769, k_keep=10, n_seg=1, k_div=3))) == 0
    assert L.trevs_inllm_workspace_size(ctypes.byref(_inllm(K_in=65536, S=65600, T_max=10))) > 0


def test_prellm_workspace_errors():
    L = trevs.lib()
    a = _prellm()
    need = L.trevs_prellm_workspace_size(ctypes.byref(a))
    assert L.trevs_prellm_prune(ctypes.byref(a), None, 0, None) == 3
    assert L.trevs_prellm_prune(ctypes.byref(a), 1 << 44, need - 1, None) == 3
    assert L.trevs_prellm_prune(ctypes.byref(a), (1 << 44) + 16, need, None) == 3


@pytest.mark.parametrize("bad,code", [
    (dict(T_max=300), 1), (dict(H_kv=5), 1), (dict(n_keep_heads=0), 1),
    (dict(n_keep_heads=33), 1), (dict(k_keep=193), 1), (dict(scale=0.0), 1), (dict(P=-1), 1),
    (dict(hidden_out=None), 1), (dict(d_head=96), 2), (dict(D=4095), 1), (dict(pos=(1 << 40) + 4), 1),
    (dict(K_in=70000, S=70100, T_max=10), 2),
    (dict(k_out=(1 << 40) + (1 << 32) + 1024), 1),  # overlaps k
    (dict(softmax=2), 1), (dict(softmax=-1), 1),
    (dict(softmax=1, lse_rest=(1 << 40) + (11 << 32)), 1),  # lse_rest is for the visual domain
])
def test_inllm_rejects_before_launch(bad, code):
    L = trevs.lib()
    a = _inllm(**bad)
    assert L.trevs_inllm_workspace_size(ctypes.byref(a)) == 0
    assert L.trevs_inllm_prune(ctypes.byref(a), None, 0, None) == code


def test_topk_rejects_before_launch():
    L = trevs.lib()
    assert L.trevs_topk_select(1 << 40, 1, 10, 11, (1 << 40) + (1 << 32), None, 0, None) == 1
    assert L.trevs_topk_select(None, 1, 10, 1, (1 << 40) + (1 << 32), None, 0, None) == 1
    assert L.trevs_topk_select(1 << 40, 1, 70000, 1, (1 << 40) + (1 << 32), None, 0, None) == 2
    assert L.trevs_topk_select(1 << 40, 1, 10, 5, (1 << 40) + 8, None, 0, None) == 1  # overlap


def _sens(**kw):
    a = trevs.SensitivityArgs()
    a.struct_size = ctypes.sizeof(a)
    a.B, a.S, a.P, a.K_in, a.T_max = 2, 259, 35, 192, 32
    a.H_q, a.H_kv, a.d_head, a.scale, a.dtype = 32, 32, 128, 128 ** -0.5, trevs.TREVS_BF16
    base = 1 << 40
    a.q[0], a.q[1] = base, base + (1 << 32)
    a.k[0] = a.k[1] = base + (2 << 32)  # one image: both questions may share the keys
    a.ts = base + (3 << 32)
    for k, v in kw.items():
        if isinstance(v, tuple):
            getattr(a, k)[v[0]] = v[1]
        else:
            setattr(a, k, v)
    return a


def test_sensitivity_workspace_covers_both_questions():
    L = trevs.lib()
    a = _sens()
    ws = L.trevs_sensitivity_workspace_size(ctypes.byref(a))
    # both questions' profiles [B,H_q,K_in] live in the workspace when not requested
    assert ws >= 2 * 2 * 32 * 192 * 4
    assert L.trevs_text_sensitivity(ctypes.byref(a), None, 0, None) == 3


@pytest.mark.parametrize("bad,code", [
    (dict(T_max=300), 1), (dict(H_kv=5), 1), (dict(scale=float("inf")), 1), (dict(P=-1), 1),
    (dict(ts=None), 1), (dict(q=(1, None)), 1), (dict(k=(0, (1 << 40) + 8)), 1),
    (dict(d_head=96), 2), (dict(struct_size=8), 1), (dict(dtype=3), 1),
    (dict(ts=(1 << 40) + (2 << 32) + 64), 1),  # overlaps the keys
    (dict(profile=(1, (1 << 40) + 1024)), 1),  # overlaps question 0's queries
    (dict(head_var=(0, (1 << 40) + (5 << 32) + 2)), 1),  # misaligned
    (dict(softmax=5), 1), (dict(softmax=1, lse_rest=(1, (1 << 40) + (6 << 32))), 1),
])
def test_sensitivity_rejects_before_launch(bad, code):
    L = trevs.lib()
    a = _sens(**bad)
    assert L.trevs_sensitivity_workspace_size(ctypes.byref(a)) == 0
    assert L.trevs_text_sensitivity(ctypes.byref(a), None, 0, None) == code


def test_spearman_rejects_before_launch():
    L = trevs.lib()
    sv, st, rho, idx = 1 << 40, (1 << 40) + (1 << 32), (1 << 40) + (2 << 32), (1 << 40) + (3 << 32)
    assert L.trevs_spearman_workspace_size(2, 100, 30) > 0
    assert L.trevs_spearman_workspace_size(2, 100, 101) == 0
    ws = 1 << 44
    need = L.trevs_spearman_workspace_size(2, 100, 30)
    assert L.trevs_topk_spearman(sv, st, 2, 100, 101, rho, idx, ws, need, None) == 1
    assert L.trevs_topk_spearman(sv, st, 2, 100, 0, rho, idx, ws, need, None) == 1
    assert L.trevs_topk_spearman(None, st, 2, 100, 30, rho, idx, ws, need, None) == 1
    assert L.trevs_topk_spearman(sv, st, 2, 100, 30, rho + 4, idx, ws, need, None) == 1
    assert L.trevs_topk_spearman(sv, st, 2, 100, 30, sv + 8, idx, ws, need, None) == 1
    assert L.trevs_topk_spearman(sv, st, 2, 70000, 30, rho, idx, ws, need, None) == 2
    assert L.trevs_topk_spearman(sv, st, 2, 100, 30, rho, idx, ws, need - 1, None) == 3
    assert L.trevs_topk_spearman(sv, st, 2, 100, 30, rho, idx, None, 0, None) == 3


def test_noalloc_rejects_on_the_host():
    """The allocation-free stage-2 entry point returns the regular entry
    point's status for invalid arguments, and TREVS_ERR_WORKSPACE when the
    call would need more than its static workspace, both before any HIP call."""
    L = trevs.lib()
    a = _inllm(k_keep=0)
    assert L.trevs_inllm_prune_noalloc(ctypes.byref(a), None) == 1
    # 64 samples x 32 heads x 1024 text rows of split statistics: > 16 MiB
    big = _inllm(B=64, T_max=1024, S=35 + 192 + 1024)
    need = L.trevs_inllm_workspace_size(ctypes.byref(big))
    assert need > 16 << 20
    assert L.trevs_inllm_prune_noalloc(ctypes.byref(big), None) == 3


def test_inllm_row_stats_rejections():
    """Caller-given row statistics exclude lse_rest, must be 4-byte aligned
    and must not overlap an output."""
    L = trevs.lib()
    base = 1 << 40
    a = _inllm(row_stats=base + (20 << 32), lse_rest=base + (21 << 32))
    assert L.trevs_inllm_workspace_size(ctypes.byref(a)) == 0
    a = _inllm(row_stats=base + (20 << 32) + 2)
    assert L.trevs_inllm_workspace_size(ctypes.byref(a)) == 0
    a = _inllm(row_stats=base + (6 << 32))  # inside hidden_out
    assert L.trevs_inllm_workspace_size(ctypes.byref(a)) == 0
    ok = _inllm(row_stats=base + (20 << 32))
    plain = _inllm()
    # no statistics pass: its split partials leave the workspace
    assert 0 < L.trevs_inllm_workspace_size(ctypes.byref(ok)) < L.trevs_inllm_workspace_size(ctypes.byref(plain))
