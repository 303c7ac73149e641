"""Pins for the oracle's sketching steps (Sec. 2.1-2.2, Alg. 1 steps 1-5).

Each test checks the oracle against something other than itself: a library
routine, a closed form, the definition written as a brute-force double sum,
or a statistical property the paper proves.
"""
import math

import numpy as np
import pytest
import scipy.linalg

import oracle as O


@pytest.mark.parametrize("d", [1, 2, 4, 8, 16, 32, 64, 128])
def test_hadamard_is_sylvester_and_orthogonal(d):
    H = O.sylvester_hadamard(d)
    # library routine (Sylvester construction, natural order)
    np.testing.assert_array_equal(H, scipy.linalg.hadamard(d).astype(np.float64))
    # closed form H H^T = d I
    np.testing.assert_array_equal(H @ H.T, d * np.eye(d))


def test_hadamard_rejects_non_power_of_two():
    with pytest.raises(ValueError):
        O.sylvester_hadamard(12)


@pytest.mark.parametrize("d", [8, 64, 128])
def test_srht_of_unit_vectors_recovers_rows(d):
    """With D = I and all columns kept, transforming e_a gives row a of the
    Sylvester matrix scaled by 1/sqrt(d)."""
    signs = np.ones(d, dtype=np.int8)
    cols = np.arange(d)
    E = np.eye(d)
    Y = O.srht(E, signs, cols)
    np.testing.assert_allclose(Y * math.sqrt(d), scipy.linalg.hadamard(d), atol=1e-12)


@pytest.mark.parametrize("d,r", [(8, 3), (64, 16), (128, 64)])
def test_srht_of_unit_vectors_with_signs_and_sampling(d, r):
    """e_a picks row a of D W: its sketch is signs[a] times the sampled
    entries of Sylvester row a, scaled by 1/sqrt(r) (sqrt(d/r) / sqrt(d))."""
    rng = np.random.default_rng(d + r)
    signs = rng.choice([-1, 1], size=d)
    cols = rng.choice(d, size=r, replace=False)
    Y = O.srht(np.eye(d), signs, cols)
    H = scipy.linalg.hadamard(d).astype(np.float64)
    for a in range(d):
        np.testing.assert_allclose(Y[a] * math.sqrt(r), signs[a] * H[a, cols], atol=1e-12)


@pytest.mark.parametrize("d", [16, 64])
def test_srht_exact_inner_products_at_full_dim(d):
    """At r = d the transform is orthogonal: sketched inner products equal
    the block-mean inner products."""
    rng = np.random.default_rng(1)
    X = rng.normal(size=(5, d))
    Y = rng.normal(size=(7, d))
    signs = rng.choice([-1, 1], size=d)
    cols = rng.permutation(d)
    G = O.srht(X, signs, cols) @ O.srht(Y, signs, cols).T
    np.testing.assert_allclose(G, X @ Y.T, rtol=1e-12, atol=1e-12)


def test_srht_column_order_is_irrelevant_for_scores():
    rng = np.random.default_rng(2)
    d, r = 32, 8
    X = rng.normal(size=(6, d))
    signs = rng.choice([-1, 1], size=d)
    cols = rng.choice(d, size=r, replace=False)
    A1 = O.block_scores(O.srht(X, signs, cols), O.srht(X, signs, cols))
    perm = rng.permutation(r)
    A2 = O.block_scores(O.srht(X, signs, cols[perm]), O.srht(X, signs, cols[perm]))
    np.testing.assert_allclose(A1, A2, rtol=1e-13, atol=1e-15)


def test_srht_inner_product_is_unbiased():
    """Appendix lemma on the Hadamard transform guarantee, step 3: over
    random signs and sampled columns, E[u~ . v~] = u . v."""
    rng = np.random.default_rng(3)
    d, r, draws = 32, 8, 20000
    u = rng.normal(size=d)
    v = u + 0.5 * rng.normal(size=d)
    W = scipy.linalg.hadamard(d).astype(np.float64)   # independent +-1 matrix
    vals = np.empty(draws)
    for t in range(draws):
        signs = rng.choice([-1.0, 1.0], size=d)
        cols = rng.choice(d, size=r, replace=False)
        us = O.srht(u[None, :], signs, cols)[0]
        vs = O.srht(v[None, :], signs, cols)[0]
        vals[t] = us @ vs
    se = vals.std(ddof=1) / math.sqrt(draws)
    assert abs(vals.mean() - u @ v) < 5 * se, (vals.mean(), u @ v, se)
    # and the estimate is not trivially exact (r < d really subsamples)
    assert vals.std() > 1e-3
    del W


def test_head_mean_matches_loop_and_gqa_expansion():
    rng = np.random.default_rng(4)
    h_kv, G, n, d = 2, 3, 5, 4
    K = rng.normal(size=(h_kv, n, d))
    loop = np.zeros((n, d))
    for g in range(h_kv):
        loop += K[g]
    loop /= h_kv
    np.testing.assert_allclose(O.head_mean(K), loop, rtol=1e-15, atol=1e-15)
    # averaging the KV heads equals averaging the GQA-expanded key heads
    expanded = np.repeat(K, G, axis=0)
    np.testing.assert_allclose(O.head_mean(expanded), O.head_mean(K), rtol=1e-14, atol=1e-15)


def test_block_means_with_partial_last_block():
    X = np.arange(30, dtype=np.float64).reshape(10, 3)
    M = O.block_means(X, 4)
    assert M.shape == (3, 3)
    np.testing.assert_array_equal(M[0], X[0:4].mean(axis=0))
    np.testing.assert_array_equal(M[1], X[4:8].mean(axis=0))
    np.testing.assert_array_equal(M[2], X[8:10].mean(axis=0))


def test_sketched_scores_equal_block_attention_definition_at_full_dim():
    """Def. Block Attention Score (Sec. 2.1): with r = d the sketch is exact,
    so every causal entry equals the brute-force B*B double sum / sqrt(d)."""
    rng = np.random.default_rng(5)
    h, n, d, B = 3, 12, 8, 4
    Q = rng.normal(size=(h, n, d))
    K = rng.normal(size=(h, n, d))
    signs = rng.choice([-1, 1], size=d)
    cols = rng.permutation(d)
    sk = O.sketch_scores(Q, K, B, signs, cols)
    Qa = O.head_mean(Q)
    Ka = O.head_mean(K)
    b = n // B
    for i in range(b):
        for j in range(b):
            want = O.block_score_true(Qa, Ka, B, i, j) if j <= i else 0.0
            assert abs(sk["A"][i, j] - want) < 1e-13, (i, j)
    assert sk["c"] == pytest.approx(np.max(np.abs(sk["A"])))


def test_score_scale_of_zero_matrix_is_one():
    assert O.score_scale(np.zeros((3, 3))) == 1.0
