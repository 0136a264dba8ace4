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


FPS_TIE = 1e-5  # oracle distances this close are a genuine near-tie


def check_fps_picks(Z64, pivots, picks, want=None):
    """Every pick of the GPU sequence is valid against the GPU's own selected
    set so far: it is not yet selected, and its float64 distance to its
    nearest selected token is within FPS_TIE of the largest over the
    unselected tokens.  Where the largest leads by more than FPS_TIE this
    forces the unique farthest token, so the sequence equals the oracle's
    `want` until a genuine near-tie, and every later pick is still checked
    against the history the GPU actually took.  Returns the number of picks
    equal to the oracle's before the first difference (0 without `want`)."""
    zbar = oracle.l2_normalise_rows(Z64)
    N = zbar.shape[0]
    picks = np.asarray(picks, dtype=np.int64)
    taken = np.zeros(N, dtype=bool)
    taken[np.asarray(pivots, dtype=np.int64)] = True
    dist = (1.0 - zbar @ zbar[np.asarray(pivots, dtype=np.int64)].T).min(axis=1) if len(pivots) \
        else np.zeros(N)
    # the cosine similarities of every pick to every token in one product
    # (row t is zbar @ zbar[picks[t]]); indices are checked before each use
    rows = zbar[np.clip(picks, 0, N - 1)] @ zbar.T
    same = 0
    for t, p in enumerate(picks):
        p = int(p)
        assert 0 <= p < N and not taken[p], (t, p)
        if not taken.any():  # nothing selected yet: the lowest index
            assert p == 0, (t, p)
        best = dist[~taken].max()
        assert dist[p] >= best - FPS_TIE, (t, p, dist[p], best)
        if want is not None and same == t and p == int(want[t]):
            same += 1
        taken[p] = True
        dist = np.minimum(dist, 1.0 - rows[t])
    return same
