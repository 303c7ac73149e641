"""Pins for the oracle's walk (Sec. 2.3, Alg. 1 step 6, appendix lemmas on
walk accumulation, block selection and multi-hop information flow)."""
import itertools
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _lower(rng, b, zero_frac=0.0):
    W = np.tril(rng.uniform(0.1, 1.0, size=(b, b)))
    if zero_frac:
        W = W * (rng.uniform(size=(b, b)) > zero_frac)
    return W


def test_power_worked_example():
    """Element-wise power of A / c, computed by hand:
    A = [[2, 0], [1, -3]], c = 3."""
    A = np.array([[2.0, 0.0], [1.0, -3.0]])
    np.testing.assert_allclose(O.walk_weights(A, 3.0, 2), [[4 / 9, 0], [1 / 9, 1]], rtol=1e-15)
    np.testing.assert_allclose(O.walk_weights(A, 3.0, 3), [[8 / 27, 0], [1 / 27, -1]], rtol=1e-15)
    np.testing.assert_allclose(O.walk_weights(A, 3.0, 1), A / 3.0, rtol=1e-15)
    with pytest.raises(ValueError):
        O.walk_weights(A, 3.0, 0)
    with pytest.raises(ValueError):
        O.walk_weights(A, 3.0, 2.5)


@pytest.mark.parametrize("b,L", [(3, 2), (4, 3), (5, 4)])
def test_walk_equals_path_sum(b, L):
    """Lemma on walk selection, step 2 (path expansion): R_k[i, j] is the sum
    over every (k+1)-hop block path from i to j of the product of the
    per-layer weights. Enumerated by brute force over all paths."""
    rng = np.random.default_rng(10 + b)
    Ws = [rng.uniform(-1.0, 1.0, size=(b, b)) for _ in range(L)]   # non-symmetric
    R = None
    for W in Ws:
        R = O.walk_step(R, W, normalize=False)
    for i in range(b):
        for j in range(b):
            total = 0.0
            for mids in itertools.product(range(b), repeat=L - 1):
                path = (i,) + mids + (j,)
                prod = 1.0
                for ell in range(L):
                    prod *= Ws[ell][path[ell], path[ell + 1]]
                total += prod
            assert abs(R[i, j] - total) < 1e-12, (i, j)


def test_walk_incremental_equals_ordered_product():
    """R_k = W_0 W_1 ... W_k (main theorem, part 1, step 1.1)."""
    rng = np.random.default_rng(11)
    Ws = [_lower(rng, 6) for _ in range(4)]
    R = None
    for W in Ws:
        R = O.walk_step(R, W, normalize=False)
    np.testing.assert_allclose(R, np.linalg.multi_dot(Ws), rtol=1e-13)


def test_walk_support_is_reachability():
    """Lemma on multi-hop information flow, step 6: with non-negative
    weights, R_L[i, j] > 0 exactly when a path with all weights positive
    leads from i to j."""
    rng = np.random.default_rng(12)
    b, L = 6, 3
    Ws = [_lower(rng, b, zero_frac=0.6) for _ in range(L)]
    R = None
    for W in Ws:
        R = O.walk_step(R, W)
    reach = [{i} for i in range(b)]
    for W in Ws:
        reach = [{j for m in reach[i] for j in range(b) if W[m, j] > 0} for i in range(b)]
    for i in range(b):
        for j in range(b):
            assert (R[i, j] > 0) == (j in reach[i]), (i, j)


def test_walk_stays_lower_triangular_and_nonnegative_for_even_s():
    rng = np.random.default_rng(13)
    h, n, d, B = 2, 64, 16, 8
    R = None
    signs = rng.choice([-1, 1], size=d)
    cols = rng.choice(d, size=8, replace=False)
    for _ in range(3):
        Q = rng.normal(size=(h, n, d))
        K = rng.normal(size=(h, n, d))
        sk = O.sketch_scores(Q, K, B, signs, cols)
        W = O.walk_weights(sk["A"], sk["c"], 8)
        assert (W >= 0).all()
        R = O.walk_step(R, W)
        assert np.allclose(np.triu(R, 1), 0.0)
        assert (R >= 0).all()
        assert np.allclose(np.max(np.abs(R), axis=1)[np.any(R != 0, axis=1)], 1.0)


def _exact_select(R_rows, pct, flags):
    """Selection by exact rational ranking (Fractions), no floats."""
    b = len(R_rows)
    out = []
    for i in range(b):
        F = O.forced_set(i, flags)
        tau = O.row_budget(i + 1, len(F), pct=pct)
        cand = sorted((j for j in range(i + 1) if j not in F), key=lambda j: (-R_rows[i][j], j))
        out.append(sorted(set(F) | set(cand[:tau - len(F)])))
    return out


@pytest.mark.parametrize("s", [2, 3, 8])
def test_rescaling_leaves_selection_unchanged_exactly(s):
    """The per-layer scale c and the per-row normalization multiply rows by
    positive factors; the selection from the raw, unscaled product computed
    in exact rational arithmetic must be identical."""
    rng = np.random.default_rng(20 + s)
    b, L, pct = 7, 3, 40
    As = []
    for _ in range(L):
        A = np.tril(rng.integers(-6, 7, size=(b, b)).astype(np.float64) / 4.0)  # dyadic
        As.append(A)
    # exact raw walk: R = prod_l (A_l)^s, no scaling at all
    Rx = None
    for A in As:
        Wx = [[Fraction(A[i, j]) ** s for j in range(b)] for i in range(b)]
        if Rx is None:
            Rx = Wx
        else:
            Rx = [[sum(Rx[i][m] * Wx[m][j] for m in range(b)) for j in range(b)] for i in range(b)]
    want = _exact_select(Rx, pct, O.FORCE_BOTH)
    # oracle walk with scale c and row normalization, in float64
    R = None
    for A in As:
        R = O.walk_step(R, O.walk_weights(A, O.score_scale(A), s))
    got, _ = O.select_blocks(R, pct=pct, flags=O.FORCE_BOTH)
    assert got == want


def test_one_hop_s1_selection_is_argsort_of_scores():
    """s = 1, one layer, nothing forced: the selection is the k largest
    scores of each causal row (stable library sort on the negated row)."""
    rng = np.random.default_rng(30)
    b, k = 9, 3
    A = np.tril(rng.normal(size=(b, b)))
    R = O.walk_step(None, O.walk_weights(A, O.score_scale(A), 1))
    sel, _ = O.select_blocks(R, k=k, flags=0)
    for i in range(b):
        want = sorted(np.argsort(-A[i, :i + 1], kind="stable")[:min(k, i + 1)].tolist())
        assert sel[i] == want, i


def test_remark_nonmetric_two_hop():
    """Appendix remark (inner product violates the triangle inequality): the
    walk reaches block k through j, which direct scores cannot."""
    with open(os.path.join(GOLDEN, "remark_nonmetric.json")) as f:
        g = json.load(f)
    d, B = g["d"], g["B"]
    signs = np.ones(d)
    cols = np.arange(d)
    q0 = np.array(g["layers"][0]["q"])
    k0 = np.array(g["layers"][0]["k"])
    # the remark's dot products, as printed
    np.testing.assert_allclose(k0 @ q0[2], g["direct_dots_layer0_row_i"])
    assert float(np.dot(k0[1], k0[0])) == 1.0
    R = None
    sk = None
    for layer in g["layers"]:
        Q = np.array(layer["q"])[None]
        K = np.array(layer["k"])[None]
        sk = O.sketch_scores(Q, K, B, signs, cols)
        R = O.walk_step(R, O.walk_weights(sk["A"], sk["c"], 8))
    i = g["query_block"]
    walk_sel, _ = O.select_blocks(R, k=g["k_select"], flags=0)
    hop_sel, _ = O.select_blocks(sk["A"], k=g["k_select"], flags=0)
    assert walk_sel[i] == g["walk_pick_layer1"]
    assert hop_sel[i] == g["one_hop_pick_layer1"]
    assert math.isclose(R[i, 0], 1.0) and R[i, 1] < 1e-2
