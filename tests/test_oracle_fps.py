"""Pins of the oracle's farthest point sampling (Sec. 4.1, context
preservation after Eq. (7)): each pick is the candidate whose cosine distance
to its nearest already-selected token is largest, ties to the lower index.

The pins come from outside the oracle: exact rational arithmetic on a
hand-derived fixture whose points separate the rule from its plausible
misreadings, an exhaustive search over every pick sequence on tiny inputs,
and invariances of cosine distance (row scale, rotation).  The last tests
plant mistakes in the oracle on the CPU and check that the pins catch them."""
import itertools
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
import oracle.trevs_oracle as oracle_mod

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "fps_nearest.json")


def _golden():
    with open(GOLDEN) as f:
        return json.load(f)


def _isqrt_norm(p):
    n2 = sum(c * c for c in p)
    n = math.isqrt(n2)
    assert n * n == n2, "fixture points have integer norms"
    return n


def _exact_dist(p, q):
    """1 - cos(p, q) as an exact fraction (integer points with integer norms)."""
    return 1 - Fraction(sum(a * b for a, b in zip(p, q)), _isqrt_norm(p) * _isqrt_norm(q))


def _greedy_exact(points, pivots, k, value):
    """Greedy picks with an exact per-candidate value (largest first, lower
    index on ties); value(i, selected) is the rule under test."""
    sel, picks = list(pivots), []
    for _ in range(k):
        best = None
        for i in range(len(points)):
            if i in sel:
                continue
            v = value(i, sel)
            if best is None or v > best[0]:
                best = (v, i)
        picks.append(best[1])
        sel.append(best[1])
    return picks


# ---------------------------------------------------------------- fixture
def test_fps_fixture_nearest_rule():
    g = _golden()
    Z = np.array(g["points"], dtype=np.float64)
    got = oracle.farthest_point_sampling(Z, g["pivots"], g["k_div"])
    assert got.tolist() == g["picks"]
    # the fixture's stated minimum distances of the picks, in exact arithmetic
    pts = g["points"]
    sel = list(g["pivots"])
    for pick, (num, den) in zip(g["picks"], g["min_dist_of_picks"]):
        assert min(_exact_dist(pts[pick], pts[j]) for j in sel) == Fraction(num, den)
        sel.append(pick)


def test_fps_fixture_exact_greedy_agrees():
    """The nearest-selected rule evaluated in exact rational arithmetic gives
    the fixture's sequence, with every winner clear of the runner-up."""
    g = _golden()
    pts = g["points"]
    near = lambda i, sel: min(_exact_dist(pts[i], pts[j]) for j in sel)  # noqa: E731
    assert _greedy_exact(pts, g["pivots"], g["k_div"], near) == g["picks"]
    sel = list(g["pivots"])
    for pick in g["picks"]:
        vals = sorted((near(i, sel) for i in range(len(pts)) if i not in sel), reverse=True)
        assert vals[0] - vals[1] >= Fraction(56, 125)
        sel.append(pick)


def test_fps_fixture_separates_misreadings():
    """Each misreading of the rule, evaluated exactly on the fixture's points,
    gives the sequence the fixture records for it, and none of those is the
    true sequence: a mistake of any of these kinds cannot pass the fixture."""
    g = _golden()
    pts = g["points"]
    d = _exact_dist
    dot = lambda p, q: sum(a * b for a, b in zip(p, q))  # noqa: E731
    rules = {
        "sum_of_distances": lambda i, sel: sum(d(pts[i], pts[j]) for j in sel),
        "last_pick_only": lambda i, sel: d(pts[i], pts[sel[-1]]),
        "first_pivot_only": lambda i, sel: d(pts[i], pts[sel[0]]),
        "no_normalisation": lambda i, sel: min(1 - dot(pts[i], pts[j]) for j in sel),
        "selected_side_normalised_only": lambda i, sel: min(
            1 - Fraction(dot(pts[i], pts[j]), _isqrt_norm(pts[j]) ** 2) for j in sel),
        "max_over_selected": lambda i, sel: max(d(pts[i], pts[j]) for j in sel),
        "argmin": lambda i, sel: -min(d(pts[i], pts[j]) for j in sel),
        "squared_euclidean": lambda i, sel: min(
            sum((a - b) ** 2 for a, b in zip(pts[i], pts[j])) for j in sel),
    }
    assert set(rules) == set(g["wrong_rules"])
    for name, rule in rules.items():
        seq = _greedy_exact(pts, g["pivots"], g["k_div"], rule)
        assert seq == g["wrong_rules"][name], name
        assert seq != g["picks"], name


def test_fps_fixture_ties_and_empty_selection():
    g = _golden()
    for case in (g["ties"], g["no_pivot"]):
        Z = np.array(case["points"], dtype=np.float64)
        assert oracle.farthest_point_sampling(Z, case["pivots"], case["k_div"]).tolist() == case["picks"]


# ---------------------------------------------------------------- brute force
def _loop_cos_dist(a, b):
    na = math.sqrt(math.fsum(x * x for x in a))
    nb = math.sqrt(math.fsum(x * x for x in b))
    return 1.0 - math.fsum(x * y for x, y in zip(a, b)) / (na * nb)


def _lex_max_sequence(Z, pivots, k):
    """Exhaustive search: among all ordered sequences of k distinct
    candidates, the one whose per-step key (distance to the nearest token
    selected so far, descending; index, ascending) is lexicographically
    best.  With no token selected yet every candidate's distance counts as
    equal."""
    rows = [list(r) for r in Z]
    cand = [i for i in range(len(rows)) if i not in set(pivots)]
    best_key, best_seq = None, None
    for seq in itertools.permutations(cand, k):
        sel = list(pivots)
        key = []
        for i in seq:
            dist = min(_loop_cos_dist(rows[i], rows[j]) for j in sel) if sel else 0.0
            key.extend([dist, -i])
            sel.append(i)
        if best_key is None or key > best_key:
            best_key, best_seq = key, list(seq)
    return best_seq


@pytest.mark.parametrize("seed", range(12))
def test_fps_brute_force_lex_max(seed):
    rng = np.random.default_rng(100 + seed)
    n = int(rng.integers(4, 8))
    d = int(rng.integers(2, 5))
    # rows of very different norms: the rule is scale-free per row
    Z = rng.standard_normal((n, d)) * rng.uniform(0.05, 20.0, size=(n, 1))
    n_piv = int(rng.integers(0, 3))
    pivots = sorted(rng.choice(n, size=n_piv, replace=False).tolist())
    k = int(min(3, n - n_piv))
    got = oracle.farthest_point_sampling(Z, pivots, k).tolist()
    assert got == _lex_max_sequence(Z, pivots, k)


# ---------------------------------------------------------------- invariances
@pytest.mark.parametrize("seed", range(4))
def test_fps_invariant_under_row_scale_and_rotation(seed):
    rng = np.random.default_rng(200 + seed)
    N, d = 60, 8
    Z = rng.standard_normal((N, d))
    pivots = np.sort(rng.choice(N, size=10, replace=False))
    want = oracle.farthest_point_sampling(Z, pivots, 12)
    Q, _ = np.linalg.qr(rng.standard_normal((d, d)))
    scaled = Z * rng.uniform(0.01, 100.0, size=(N, 1))
    assert np.array_equal(oracle.farthest_point_sampling(scaled, pivots, 12), want)
    assert np.array_equal(oracle.farthest_point_sampling(Z @ Q, pivots, 12), want)


# ---------------------------------------------------------------- planted mistakes
def test_planted_missing_normalisation_is_caught(monkeypatch):
    """Plant 'no L2 normalisation' in the oracle: the fixture rejects it."""
    g = _golden()
    Z = np.array(g["points"], dtype=np.float64)
    monkeypatch.setattr(oracle_mod, "l2_normalise_rows", lambda X: np.asarray(X, dtype=np.float64))
    assert oracle.farthest_point_sampling(Z, g["pivots"], g["k_div"]).tolist() != g["picks"]


def _fps_variant(Z, selected, k_div, reduce_fn):
    """The oracle's own loop with the reduction over the selected set
    replaced (a planted mistake)."""
    zbar = oracle.l2_normalise_rows(Z)
    sel = [int(i) for i in selected]
    picks = []
    for _ in range(k_div):
        cand = np.array([i for i in range(zbar.shape[0]) if i not in set(sel)], dtype=np.int64)
        d = reduce_fn(1.0 - zbar[cand] @ zbar[np.array(sel)].T, sel)
        best = int(cand[int(np.argmax(d))])
        picks.append(best)
        sel.append(best)
    return picks


@pytest.mark.parametrize("name,reduce_fn", [
    ("sum", lambda D, sel: D.sum(axis=1)),
    ("mean", lambda D, sel: D.mean(axis=1)),
    ("last pick only", lambda D, sel: D[:, -1]),
])
def test_planted_wrong_reduction_is_caught(name, reduce_fn):
    """Reductions other than the nearest selected token fail the fixture,
    the exhaustive search, or both."""
    g = _golden()
    Z = np.array(g["points"], dtype=np.float64)
    assert _fps_variant(Z, g["pivots"], g["k_div"], lambda D, sel: D.min(axis=1)) == g["picks"]
    assert _fps_variant(Z, g["pivots"], g["k_div"], reduce_fn) != g["picks"], name
