"""Pins for the oracle's block-sparse attention (Alg. 1 step 8) and the dense
causal reference it must reduce to."""
import math

import numpy as np
import pytest
import torch

import oracle as O


def _qkv(seed, h_q, h_kv, n, d):
    rng = np.random.default_rng(seed)
    return (rng.normal(size=(h_q, n, d)), rng.normal(size=(h_kv, n, d)),
            rng.normal(size=(h_kv, n, d)))


@pytest.mark.parametrize("h_q,h_kv,n,d", [(1, 1, 17, 8), (4, 2, 40, 16), (6, 2, 33, 8)])
def test_dense_matches_torch_sdpa_float64(h_q, h_kv, n, d):
    Q, K, V = _qkv(1, h_q, h_kv, n, d)
    G = h_q // h_kv
    tq = torch.from_numpy(Q)[None]
    tk = torch.from_numpy(np.repeat(K, G, axis=0))[None]
    tv = torch.from_numpy(np.repeat(V, G, axis=0))[None]
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, is_causal=True)[0].numpy()
    np.testing.assert_allclose(O.dense_causal_attention(Q, K, V), ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("n,B", [(64, 8), (70, 8), (33, 16)])
def test_full_selection_equals_dense(n, B):
    """Density 100% is dense causal attention, including a ragged tail."""
    Q, K, V = _qkv(2, 4, 2, n, 16)
    b = -(-n // B)
    sel = [list(range(i + 1)) for i in range(b)]
    np.testing.assert_allclose(O.sparse_attention_prefill(Q, K, V, B, sel),
                               O.dense_causal_attention(Q, K, V), rtol=1e-12, atol=1e-12)


def test_sparse_equals_dense_with_additive_mask():
    """Masked attention written as dense softmax plus a -inf mask built token
    by token from the selection."""
    n, B, d = 48, 8, 8
    Q, K, V = _qkv(3, 2, 1, n, d)
    rng = np.random.default_rng(3)
    b = n // B
    sel = []
    for i in range(b):
        others = [j for j in range(1, i) if rng.uniform() < 0.4]
        sel.append(sorted(set([0, i] + others)))
    got = O.sparse_attention_prefill(Q, K, V, B, sel)
    for u in range(2):
        S = Q[u] @ K[0].T / math.sqrt(d)
        mask = np.full((n, n), -np.inf)
        for p in range(n):
            for t in range(n):
                if t <= p and (t // B) in sel[p // B]:
                    mask[p, t] = 0.0
        P = np.exp(S + mask - np.max(S + mask, axis=1, keepdims=True))
        P /= P.sum(axis=1, keepdims=True)
        np.testing.assert_allclose(got[u], P @ V[0], rtol=1e-12, atol=1e-12)


def test_constant_values_give_constant_output():
    n, B, d = 32, 8, 8
    Q, K, _ = _qkv(4, 2, 2, n, d)
    V = np.broadcast_to(np.arange(d, dtype=np.float64), (2, n, d)).copy()
    sel = [[0, i] if i else [0] for i in range(n // B)]
    out = O.sparse_attention_prefill(Q, K, V, B, sel)
    np.testing.assert_allclose(out, np.broadcast_to(np.arange(d), out.shape), rtol=1e-13, atol=1e-13)


def test_diagonal_only_is_blockwise_causal_softmax():
    n, B, d = 24, 8, 4
    Q, K, V = _qkv(5, 1, 1, n, d)
    sel = [[i] for i in range(n // B)]
    out = O.sparse_attention_prefill(Q, K, V, B, sel)
    for i in range(n // B):
        sl = slice(i * B, (i + 1) * B)
        want = O.dense_causal_attention(Q[:, sl], K[:, sl], V[:, sl])
        np.testing.assert_allclose(out[:, sl], want, rtol=1e-12, atol=1e-12)


def test_executed_flops_of_full_selection():
    n, B, h, d = 100, 16, 3, 8
    b = -(-n // B)
    sel = [list(range(i + 1)) for i in range(b)]
    assert O.executed_attention_flops([n], B, h, d, [sel]) == 4 * d * h * n * (n + 1) // 2
