"""Both pruning stages captured into a HIP graph (torch.cuda.CUDAGraph over
the library's launches) and replayed: every replay, with the program's own
eager work and synchronisations between replays, gives bit-identical
outputs to the eager calls."""
import numpy as np
import pytest
import torch

from paper_2609_37581_amd import trevs
from parity import dev_tensor, host_bits
from synthetic import WORKLOADS, stage1_inputs, stage2_inputs

pytestmark = pytest.mark.gpu


def _outputs(pre, inl):
    out = {"kept_idx": pre.kept_idx, "kept_feats": pre.kept_feats, "score1": pre.score,
           "kept2": inl.kept_idx, "hidden_out": inl.hidden_out, "k_out": inl.k_out,
           "v_out": inl.v_out, "pos_out": inl.pos_out, "score2": inl.score}
    return {k: host_bits(v) for k, v in out.items()}


@pytest.mark.parametrize("name,B", [("qwen25vl-b4-bf16", 1), ("llava15-b64-bf16", 4)])
def test_graph_replays_match_eager(name, B):
    w = WORKLOADS[name].with_(B=B)
    print(f"[graph] {name} B={B}", flush=True)
    s1, s2 = stage1_inputs(w), stage2_inputs(w)
    pre = trevs.Prellm(dev_tensor(s1["cls_logits"], w.dtype), dev_tensor(s1["vis_feats"], w.dtype),
                       dev_tensor(s1["text_emb"], w.dtype), torch.from_numpy(s1["text_len"]).cuda(),
                       k_keep=w.K1, n_seg=w.n_seg, want_scores=True)
    inl = trevs.Inllm(dev_tensor(s2["q"], w.dtype), dev_tensor(s2["k"], w.dtype),
                      dev_tensor(s2["v"], w.dtype), dev_tensor(s2["hidden"], w.dtype),
                      torch.from_numpy(s2["pos"]).cuda(), torch.from_numpy(s2["text_len"]).cuda(),
                      P=w.P, K_in=w.K1, n_keep_heads=w.n_keep, k_keep=w.K2, want_scores=True)
    pre()
    inl()
    torch.cuda.synchronize()
    eager = _outputs(pre, inl)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        pre(side)
        inl(side)
    torch.cuda.current_stream().wait_stream(side)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        pre()
        inl()
    outs = [pre.kept_idx, pre.kept_feats, pre.score, inl.kept_idx, inl.hidden_out, inl.k_out,
            inl.v_out, inl.pos_out, inl.score]
    for r in range(4):
        for t in outs:  # eager work between replays: clobber every output
            t.view(torch.uint8).fill_(0x5A)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = _outputs(pre, inl)
        for k in eager:
            assert np.array_equal(got[k], eager[k]), (r, k)
        # an eager call between replays leaves the next replay unaffected
        pre()
        torch.cuda.synchronize()
