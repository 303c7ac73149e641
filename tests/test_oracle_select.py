"""Pins for the oracle's top-tau block selection (Alg. 1 step 7, Alg. 2
step 6, Sec. 4.1 forced first/last blocks)."""
import itertools
import math

import numpy as np
import pytest

import oracle as O


def _best_subset_bruteforce(values, cand, m):
    """Among all m-subsets of the candidates, the one whose members sorted
    by (value desc, index asc) is lexicographically best."""
    best, best_key = None, None
    for sub in itertools.combinations(cand, m):
        key = sorted((-values[j], j) for j in sub)
        if best_key is None or key < best_key:
            best, best_key = sub, key
    return sorted(best) if best is not None else []


@pytest.mark.parametrize("seed", range(6))
def test_selection_matches_exhaustive_search(seed):
    rng = np.random.default_rng(seed)
    for avail in range(1, 9):
        vals = rng.integers(0, 4, size=avail).astype(np.float64)   # many ties
        for flags in (0, O.FORCE_FIRST, O.FORCE_LAST, O.FORCE_BOTH):
            for k in range(1, avail + 1):
                F = O.forced_set(avail - 1, flags)
                tau = O.row_budget(avail, len(F), k=k)
                got, _ = O.select_row(vals, avail, F, tau)
                cand = [j for j in range(avail) if j not in F]
                want = sorted(set(F) | set(_best_subset_bruteforce(vals, cand, tau - len(F))))
                assert got == want, (avail, flags, k)
                assert len(got) == tau
                assert set(F) <= set(got)
                assert got == sorted(set(got)) and all(0 <= j < avail for j in got)


def test_budget_is_integer_ceiling():
    # 15 * 0.2 is 3.0000000000000004 in floating point; the integer ceiling is 3
    assert O.row_budget(15, 1, pct=20) == 3
    assert O.row_budget(5, 2, pct=20) == 2        # ceil(1.0) = 1, raised to |F|
    assert O.row_budget(11, 2, pct=20) == 3       # ceil(2.2)
    assert O.row_budget(1, 1, pct=20) == 1
    assert O.row_budget(37, 2, pct=100) == 37
    assert O.row_budget(8, 2, k=20) == 8          # fixed k clamps to what exists
    assert O.row_budget(8, 2, k=1) == 2


def test_density_100_selects_every_causal_block():
    rng = np.random.default_rng(7)
    R = np.tril(rng.uniform(size=(9, 9)))
    sel, gaps = O.select_blocks(R, pct=100)
    for i in range(9):
        assert sel[i] == list(range(i + 1))
        assert math.isinf(gaps[i])


def test_causal_density_counts():
    """Sum of tau_i over the rows of a b-block sequence at 20% density."""
    b = 32
    total = sum(O.row_budget(i + 1, len(O.forced_set(i, O.FORCE_BOTH)), pct=20) for i in range(b))
    # rows 1..9 are raised to the 2 forced blocks; hand count of the ceilings
    want = 1 + sum(max(2, math.ceil((i + 1) * 20 / 100)) for i in range(1, b))
    assert total == want == 123


def test_gap_reports_relative_boundary_gap():
    vals = np.array([5.0, 4.0, 3.0, 2.0])
    chosen, gap = O.select_row(vals, 4, [], 2)
    assert chosen == [0, 1] and gap == pytest.approx(0.25)
    chosen, gap = O.select_row(vals, 4, [], 4)
    assert math.isinf(gap)
