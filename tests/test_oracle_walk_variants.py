"""Pins for the oracle's walk transition variants: the power after clipping
negative scores, the causal row softmax (the transition matrix of the
appendix lemma on the walk's stationary structure, step 1) and the matrix
power (the within-layer multi-hop walk of Sec. 1 and Fig. 2)."""
import itertools
import math

import numpy as np
import pytest
import scipy.special

import oracle as O


def _signed_lower(rng, b):
    return np.tril(rng.uniform(-1.0, 1.0, size=(b, b)))


# ---------------------------------------------------------------- ReLU power

def test_relu_worked_example():
    """By hand: A = [[2, 0], [1, -3]], c = 3. The -3 entry is clipped first,
    so it contributes 0 instead of (-1)^s."""
    A = np.array([[2.0, 0.0], [1.0, -3.0]])
    np.testing.assert_allclose(O.walk_weights_relu(A, 3.0, 2), [[4 / 9, 0], [1 / 9, 0]], rtol=1e-15)
    np.testing.assert_allclose(O.walk_weights_relu(A, 3.0, 3), [[8 / 27, 0], [1 / 27, 0]],
                               rtol=1e-15)


@pytest.mark.parametrize("s", [1, 2, 3, 7, 8])
def test_relu_relation_to_plain_power(s):
    """Odd s keeps the sign, so clipping after the power gives the same W;
    even s agrees with the plain power on non-negative scores and is zero on
    negative ones."""
    rng = np.random.default_rng(40 + s)
    A = _signed_lower(rng, 9)
    c = O.score_scale(A)
    Wr = O.walk_weights_relu(A, c, s)
    Wp = O.walk_weights(A, c, s)
    if s % 2:
        np.testing.assert_array_equal(Wr, np.maximum(Wp, 0.0))
    else:
        np.testing.assert_array_equal(Wr[A >= 0], Wp[A >= 0])
        assert np.all(Wr[A < 0] == 0.0)
    assert np.all(Wr >= 0.0)


def test_relu_equals_power_on_nonnegative_scores():
    rng = np.random.default_rng(47)
    A = np.abs(_signed_lower(rng, 7))
    np.testing.assert_array_equal(O.walk_weights_relu(A, 0.9, 8), O.walk_weights(A, 0.9, 8))


# ----------------------------------------------------------- softmax rows

def test_softmax_worked_example():
    """By hand: logit scale 1, A = [[0, 0], [ln 3, 0]]: row 0 has one causal
    block (weight 1); row 1 has weights e^{ln 3} : e^0 = 3 : 1."""
    A = np.array([[0.0, 0.0], [math.log(3.0), 0.0]])
    np.testing.assert_allclose(O.walk_weights_softmax(A, 1.0), [[1.0, 0.0], [0.75, 0.25]],
                               rtol=1e-15)


def test_softmax_rows_are_distributions_over_causal_blocks():
    rng = np.random.default_rng(48)
    A = _signed_lower(rng, 11) * 5.0
    W = O.walk_weights_softmax(A, 0.7)
    np.testing.assert_allclose(W.sum(axis=1), np.ones(11), rtol=1e-14)
    assert np.all(np.triu(W, 1) == 0.0)
    assert np.all(W[np.tril_indices(11)] > 0.0)


def test_softmax_matches_library_softmax_per_row():
    rng = np.random.default_rng(49)
    A = _signed_lower(rng, 10) * 3.0
    t = math.sqrt(32 / 128)
    W = O.walk_weights_softmax(A, t)
    for i in range(10):
        ref = scipy.special.softmax(t * A[i, :i + 1])
        np.testing.assert_allclose(W[i, :i + 1], ref, rtol=1e-13)


def test_softmax_zero_logit_scale_is_uniform():
    """Closed form: equal logits give 1 / (i + 1) on every causal block."""
    rng = np.random.default_rng(50)
    W = O.walk_weights_softmax(_signed_lower(rng, 8), 0.0)
    for i in range(8):
        np.testing.assert_allclose(W[i, :i + 1], np.full(i + 1, 1.0 / (i + 1)), rtol=1e-15)


def test_softmax_is_invariant_to_per_row_shift():
    rng = np.random.default_rng(51)
    A = _signed_lower(rng, 9)
    shift = rng.uniform(-4.0, 4.0, size=9)
    A2 = np.tril(A + shift[:, None])
    np.testing.assert_allclose(O.walk_weights_softmax(A2, 1.3), O.walk_weights_softmax(A, 1.3),
                               rtol=1e-12, atol=1e-15)


def test_softmax_large_scale_tends_to_row_argmax():
    rng = np.random.default_rng(52)
    A = _signed_lower(rng, 9)
    W = O.walk_weights_softmax(A, 1e4)
    for i in range(1, 9):
        j = int(np.argmax(A[i, :i + 1]))
        assert W[i, j] > 1.0 - 1e-12


# ---------------------------------------------------------- matrix power

@pytest.mark.parametrize("s", [1, 2, 3, 8])
def test_matpow_matches_library_matrix_power(s):
    rng = np.random.default_rng(60 + s)
    A = _signed_lower(rng, 12)
    c = O.score_scale(A)
    np.testing.assert_allclose(O.walk_weights_matpow(A, c, s),
                               np.linalg.matrix_power(A / c, s), rtol=1e-12, atol=1e-15)


def test_matpow_is_sum_over_s_hop_paths():
    """Entry (i, j) of (A/c)^3 sums X[i,m1] X[m1,m2] X[m2,j] over every
    path, enumerated by brute force; the result is lower triangular."""
    rng = np.random.default_rng(64)
    b = 5
    A = _signed_lower(rng, b)
    c = 0.8
    X = A / c
    W = O.walk_weights_matpow(A, c, 3)
    for i in range(b):
        for j in range(b):
            total = 0.0
            for m1, m2 in itertools.product(range(b), repeat=2):
                total += X[i, m1] * X[m1, m2] * X[m2, j]
            assert abs(W[i, j] - total) < 1e-13, (i, j)
    assert np.all(np.triu(W, 1) == 0.0)


def test_matpow_diagonal_and_nilpotent_closed_forms():
    """For a lower triangular X the diagonal of X^s is the diagonal of X to
    the power s. For a strictly lower triangular b x b matrix, X^(b-1) has
    the single entry (b-1, 0) equal to the product of the subdiagonal, and
    X^b = 0."""
    rng = np.random.default_rng(65)
    A = _signed_lower(rng, 6)
    np.testing.assert_allclose(np.diag(O.walk_weights_matpow(A, 1.0, 5)), np.diag(A) ** 5,
                               rtol=1e-13)
    b = 5
    N = np.tril(rng.uniform(0.5, 1.5, size=(b, b)), -1)
    P = O.walk_weights_matpow(N, 1.0, b - 1)
    expect = np.zeros((b, b))
    expect[b - 1, 0] = np.prod([N[m + 1, m] for m in range(b - 1)])
    np.testing.assert_allclose(P, expect, rtol=1e-14, atol=0.0)
    assert np.all(O.walk_weights_matpow(N, 1.0, b) == 0.0)


def test_matpow_s1_is_scaled_scores_and_rejects_bad_s():
    A = np.array([[2.0, 0.0], [1.0, -3.0]])
    np.testing.assert_array_equal(O.walk_weights_matpow(A, 2.0, 1), A / 2.0)
    with pytest.raises(ValueError):
        O.walk_weights_matpow(A, 1.0, 0)


# ------------------------------------------------------------- dispatcher

def test_variant_dispatch():
    rng = np.random.default_rng(70)
    A = _signed_lower(rng, 6)
    c = O.score_scale(A)
    np.testing.assert_array_equal(O.walk_weights_variant(O.WALK_POWER, A, c, 8),
                                  O.walk_weights(A, c, 8))
    np.testing.assert_array_equal(O.walk_weights_variant(O.WALK_RELU, A, c, 8),
                                  O.walk_weights_relu(A, c, 8))
    np.testing.assert_array_equal(O.walk_weights_variant(O.WALK_SOFTMAX, A, c, 8, 0.5),
                                  O.walk_weights_softmax(A, 0.5))
    np.testing.assert_array_equal(O.walk_weights_variant(O.WALK_MATPOW, A, c, 3),
                                  O.walk_weights_matpow(A, c, 3))
    with pytest.raises(ValueError):
        O.walk_weights_variant(9, A, c, 8)


def test_decode_relu_walk_row_equals_row_of_full_product():
    """Decode with the clipped power: the walk row is the current query
    block's row of the product of the per-layer clipped weights."""
    rng = np.random.default_rng(71)
    h_q, h_kv, d, B, n0, layers = 4, 2, 8, 4, 21, 3
    T = n0 + 3
    Q = [rng.normal(size=(h_q, T, d)) for _ in range(layers)]
    K = [rng.normal(size=(h_kv, T, d)) for _ in range(layers)]
    signs = rng.choice([-1, 1], size=d)
    cols = rng.permutation(d)
    b_max = -(-T // B)
    sts = [O.decode_state_from_prefill(Q[l][:, :n0], K[l][:, :n0], B, signs, cols, b_max)
           for l in range(layers)]
    for p in range(n0, T):
        r = None
        for l in range(layers):
            r, _, _ = O.decode_layer_step(sts[l], Q[l][:, p], K[l][:, p], p, r, B, signs, cols, 8,
                                          pct=40, variant=O.WALK_RELU)
    bq = (T - 1) // B
    mats = [np.power(np.maximum(st.A[:bq + 1, :bq + 1], 0.0) / st.c, 8) for st in sts]
    full = np.linalg.multi_dot(mats)
    np.testing.assert_allclose(r, full[bq] / np.max(np.abs(full[bq])), rtol=1e-10, atol=1e-14)
