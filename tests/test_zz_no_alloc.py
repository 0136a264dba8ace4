"""trevs_inllm_prune_noalloc (stage 2 on the library's static per-GPU
workspace) against trevs_inllm_prune (caller's workspace), through the C ABI:
two calls in a row, the second on a smaller input, each bit-identical to the
workspace entry point and within the parity bar of the oracle."""
import numpy as np
import pytest
import torch

import test_gpu_stage2 as s2
from paper_2609_37581_amd import trevs
from parity import dev_tensor, host_bits
from synthetic import WORKLOADS, stage2_inputs

pytestmark = pytest.mark.gpu


def _run(inp, w, noalloc):
    call = trevs.Inllm(dev_tensor(inp["q"], w.dtype), dev_tensor(inp["k"], w.dtype),
                       dev_tensor(inp["v"], w.dtype), dev_tensor(inp["hidden"], w.dtype),
                       torch.from_numpy(inp["pos"]).cuda(), torch.from_numpy(inp["text_len"]).cuda(),
                       P=w.P, K_in=w.K1, n_keep_heads=w.n_keep, k_keep=w.K2, want_scores=True,
                       noalloc=noalloc)
    assert (call.workspace is None) == noalloc
    call()
    torch.cuda.synchronize()
    return dict(kept_idx=call.kept_idx.cpu().numpy(), hidden_out=host_bits(call.hidden_out),
                k_out=host_bits(call.k_out), v_out=host_bits(call.v_out),
                pos_out=call.pos_out.cpu().numpy(), head_sel=call.head_sel.cpu().numpy(),
                head_var=call.head_var.cpu().numpy(), score=call.score.cpu().numpy())


def test_noalloc_matches_the_workspace_entry_point():
    # first the 16,384-token model's shapes (GQA 28/4, M-RoPE), then a
    # smaller LLaVA-1.5 input on the same static workspace
    for w in (WORKLOADS["qwen25vl-b4-bf16"].with_(B=2), WORKLOADS["llava15-b64-bf16"].with_(B=3)):
        print(f"[noalloc] {w.name} B={w.B} K1={w.K1} T={w.T_max} H={w.H_q}/{w.H_kv}", flush=True)
        inp = stage2_inputs(w)
        ref = _run(inp, w, noalloc=False)
        got = _run(inp, w, noalloc=True)
        for key in ref:
            assert np.array_equal(got[key], ref[key]), (w.name, key)
        s2.check(inp, w, got)
