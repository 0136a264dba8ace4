"""Parity checks between the HIP library and the CPU oracle.

Tolerances: scores agree within 1e-3 relative plus 1e-6 of the largest
magnitude (fp32 accumulation from bf16 inputs against the float64 oracle);
kept index sets agree exactly outside the band of candidates whose oracle
score lies within that tolerance of the K-th score; gathered rows are bit
exact."""
import numpy as np
import torch

import oracle

RTOL = 1e-3
ATOL_FRAC = 1e-6


def dev_tensor(arr, dtype, device="cuda"):
    """Storage-form numpy array (float32 / uint16 bf16 bits / ints) -> device tensor."""
    t = torch.from_numpy(np.ascontiguousarray(arr))
    if dtype == "bf16" and t.dtype == torch.uint16:
        t = t.view(torch.bfloat16)
    elif dtype == "bf16" and t.dtype == torch.int16:
        t = t.view(torch.bfloat16)
    return t.to(device)


def host_bits(t):
    """Device tensor -> numpy array of its raw bits (bf16 -> uint16)."""
    t = t.detach().cpu()
    if t.dtype == torch.bfloat16:
        t = t.view(torch.uint16)
    return t.numpy()


def assert_scores_close(gpu, ora, name):
    gpu = np.asarray(gpu, dtype=np.float64)
    ora = np.asarray(ora, dtype=np.float64)
    assert gpu.shape == ora.shape, (name, gpu.shape, ora.shape)
    g2 = gpu.reshape(-1, gpu.shape[-1]) if gpu.ndim > 1 else gpu[None]
    o2 = ora.reshape(-1, ora.shape[-1]) if ora.ndim > 1 else ora[None]
    for r in range(o2.shape[0]):
        scale = np.abs(o2[r]).max()
        tol = RTOL * np.abs(o2[r]) + ATOL_FRAC * scale
        err = np.abs(g2[r] - o2[r])
        bad = np.nonzero(~(err <= tol))[0]
        assert bad.size == 0, (
            f"{name} row {r}: {bad.size} of {o2.shape[1]} outside tolerance; first at "
            f"{bad[0]}: gpu={g2[r, bad[0]]!r} oracle={o2[r, bad[0]]!r}")


def band(ora_scores, k):
    """Indices whose oracle score is within tolerance of the k-th largest."""
    s = np.asarray(ora_scores, dtype=np.float64)
    kth = np.sort(s)[::-1][k - 1]
    tol = RTOL * abs(kth) + ATOL_FRAC * np.abs(s).max()
    return set(np.nonzero(np.abs(s - kth) <= tol)[0].tolist())


def assert_kept_band(gpu_idx, ora_scores, k, name):
    gpu_idx = np.asarray(gpu_idx)
    for b in range(gpu_idx.shape[0]):
        g = gpu_idx[b].tolist()
        assert len(g) == k, (name, b, len(g))
        assert all(x < y for x, y in zip(g, g[1:])), f"{name}[{b}]: not ascending/unique"
        assert 0 <= g[0] and g[-1] < len(ora_scores[b]), f"{name}[{b}]: index out of range"
        o = set(oracle.topk_ascending(ora_scores[b], k).tolist())
        bd = band(ora_scores[b], k)
        gs = set(g)
        assert gs - bd == o - bd, (
            f"{name}[{b}]: differs outside the tie band: gpu-only {sorted((gs - o) - bd)[:8]}, "
            f"oracle-only {sorted((o - gs) - bd)[:8]}")


def assert_kept_exact_on_own_scores(gpu_idx, gpu_scores, k, name):
    """The selection is exactly the stable top-k of the kernel's own fp32
    scores (same precision decision on both sides)."""
    gpu_idx = np.asarray(gpu_idx)
    for b in range(gpu_idx.shape[0]):
        want = oracle.topk_ascending(np.asarray(gpu_scores[b], dtype=np.float32).astype(np.float64), k)
        assert gpu_idx[b].tolist() == want.tolist(), f"{name}[{b}]: not the top-k of its own scores"
