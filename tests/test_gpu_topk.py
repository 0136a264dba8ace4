"""trevs_topk_select: stable top-K on the GPU, bit-exact against the oracle's
(score desc, index asc) order on the same fp32 scores."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_37581_amd import trevs

pytestmark = pytest.mark.gpu


def check(scores, k):
    got = trevs.topk_select(torch.from_numpy(scores).cuda(), k).cpu().numpy()
    for b in range(scores.shape[0]):
        want = oracle.topk_ascending(scores[b].astype(np.float64), k)
        assert got[b].tolist() == want.tolist(), (b, k)


@pytest.mark.parametrize("N,K", [(1, 1), (5, 3), (576, 192), (577, 64), (2880, 640),
                                 (4096, 1024), (16384, 4096), (32768, 1), (32768, 32768),
                                 (1000, 999), (50000, 12345), (65536, 1), (65536, 40000),
                                 (65536, 65536)])
def test_topk_random_with_quantised_ties(N, K):
    print(f"[topk] N={N} K={K}", flush=True)
    rng = np.random.default_rng(N * 7 + K)
    s = rng.random((3, N)).astype(np.float32)
    # a quarter of the scores drawn from a 64-entry table
    table = rng.random(64).astype(np.float32)
    mask = rng.random((3, N)) < 0.25
    s[mask] = table[rng.integers(0, 64, size=mask.sum())]
    check(s, K)


def test_topk_signs_zeros_and_all_equal():
    s = np.array([[0.0, -0.0, -1.5, 2.0, -0.0, 0.0, -3.0, 2.0, 1e-30, -1e-30]], dtype=np.float32)
    for k in range(1, 11):
        check(s, k)
    eq = np.full((2, 1000), 0.25, dtype=np.float32)
    for k in (1, 17, 1000):
        check(eq, k)
    # two distinct values, heavy contention in every radix pass
    two = np.where(np.arange(5000) % 3 == 0, 1.0, 0.5).astype(np.float32)[None]
    for k in (1, 1667, 1668, 4999):
        check(two, k)


def test_topk_crowded_first_digit_bin():
    """More than 4096 keys share the threshold's first 11-bit digit, so the
    selection resolves the remaining bits over all elements instead of an LDS
    candidate list; once with the crowded bin above the minimum, once with
    the minimum itself in it (its ties counted by ballot)."""
    rng = np.random.default_rng(11)
    for N in (16384, 32768, 65536):
        above = rng.random((2, N)).astype(np.float32)
        crowd = rng.random((2, N)) < 0.4
        above[crowd] = np.float32(2.0) + rng.integers(0, 3, size=crowd.sum()).astype(np.float32) * np.float32(2.0 ** -22)
        above[:, :50] = np.float32(7.0)
        for k in (60, N // 3, N // 2):
            print(f"[topk crowded] N={N} K={k}", flush=True)
            check(above, k)
        low = (np.float32(0.1) + rng.random((2, N)).astype(np.float32)).astype(np.float32)
        at_min = rng.random((2, N)) < 0.5
        low[at_min] = np.float32(0.1)
        near = rng.random((2, N)) < 0.05
        low[near & ~at_min] = np.float32(0.1) + np.float32(2.0 ** -26)
        for k in (N - 10, N - N // 3, N // 2):
            print(f"[topk crowded min] N={N} K={k}", flush=True)
            check(low, k)


def test_topk_batch_of_many_rows():
    rng = np.random.default_rng(3)
    s = rng.standard_normal((257, 300)).astype(np.float32)
    check(s, 100)


def test_topk_rejects_bad_arguments():
    s = torch.zeros((2, 10), device="cuda")
    with pytest.raises(trevs.TrevsError):
        trevs.topk_select(s, 11)
    with pytest.raises(trevs.TrevsError) as e:
        trevs.topk_select(torch.zeros((1, 70000), device="cuda"), 5)
    assert e.value.status == 2
