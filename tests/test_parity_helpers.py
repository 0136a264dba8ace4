"""The GPU tests' diversity-set checker accepts exactly the valid pick
sequences (runs on the CPU with oracle sequences and planted bad ones)."""
import numpy as np
import pytest

import oracle
from parity import check_fps_picks


def _inputs(seed, N=80, d=6, n_piv=8):
    rng = np.random.default_rng(seed)
    Z = rng.standard_normal((N, d)) * rng.uniform(0.1, 5.0, size=(N, 1))
    pivots = np.sort(rng.choice(N, size=n_piv, replace=False))
    return Z, pivots


@pytest.mark.parametrize("seed", range(3))
def test_checker_accepts_the_oracle_sequence(seed):
    Z, pivots = _inputs(seed)
    want = oracle.farthest_point_sampling(Z, pivots, 20)
    assert check_fps_picks(Z, pivots, want, want) == 20


def test_checker_rejects_a_wrong_pick_duplicate_or_pivot():
    Z, pivots = _inputs(7)
    want = oracle.farthest_point_sampling(Z, pivots, 10)
    bad = want.copy()
    # a candidate that is not the farthest at step 3
    zbar = oracle.l2_normalise_rows(Z)
    sel = list(pivots) + list(want[:3])
    d = (1.0 - zbar @ zbar[sel].T).min(axis=1)
    d[sel] = np.inf
    bad[3] = int(np.argmin(d))
    with pytest.raises(AssertionError):
        check_fps_picks(Z, pivots, bad, want)
    dup = want.copy()
    dup[5] = dup[2]
    with pytest.raises(AssertionError):
        check_fps_picks(Z, pivots, dup, want)
    piv = want.copy()
    piv[0] = pivots[0]
    with pytest.raises(AssertionError):
        check_fps_picks(Z, pivots, piv, want)


def test_checker_follows_the_gpu_history_after_a_tie():
    """Two candidates exactly equidistant: either may come first, and the
    later picks are checked against the history actually taken."""
    Z = np.array([[1.0, 0.0], [0.0, 1.0], [0.0, -1.0], [-1.0, 0.0], [0.7, 0.7]])
    want = oracle.farthest_point_sampling(Z, [0, 3], 2)
    assert want.tolist() == [1, 2]
    assert check_fps_picks(Z, [0, 3], [2, 1], want) == 0
    with pytest.raises(AssertionError):  # 4 is nearer to 0 than 1 and 2 are
        check_fps_picks(Z, [0, 3], [2, 4], want)


def test_checker_without_pivots_takes_the_lowest_index_first():
    Z = np.array([[1.0, 0.0], [0.0, 1.0], [-1.0, 0.0]])
    assert check_fps_picks(Z, [], [0, 2], [0, 2]) == 2
    with pytest.raises(AssertionError):
        check_fps_picks(Z, [], [1, 2], [0, 2])
