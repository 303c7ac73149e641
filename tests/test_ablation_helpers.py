"""CPU checks of the ablation harness's measuring helpers (bench.py) and of
the synthetic generator's needle plan: the dense block attention mass
against a per-token brute force, the selection masks, the best-possible
selection, and the needle positions against the planted keys."""
import math

import numpy as np
import pytest
import torch

import bench
import synth


def _brute_block_mass(Q, K, B):
    h_q, n, d = Q.shape
    G = h_q // K.shape[0]
    b = -(-n // B)
    M = np.zeros((b, b))
    for u in range(h_q):
        for t in range(n):
            z = np.array([Q[u, t] @ K[u // G, k] / math.sqrt(d) for k in range(t + 1)])
            e = np.exp(z - z.max())
            pr = e / e.sum()
            for k in range(t + 1):
                M[t // B, k // B] += pr[k]
    for i in range(b):
        M[i] /= h_q * min(B, n - i * B)
    return M


def test_block_attention_mass_matches_brute_force():
    rng = np.random.default_rng(3)
    Q = rng.normal(size=(4, 37, 8))
    K = rng.normal(size=(2, 37, 8))
    got = bench.block_attention_mass(torch.tensor(Q, dtype=torch.float32),
                                     torch.tensor(K, dtype=torch.float32), 8, chunk=16).numpy()
    ref = _brute_block_mass(Q.astype(np.float32).astype(np.float64),
                            K.astype(np.float32).astype(np.float64), 8)
    np.testing.assert_allclose(got, ref, atol=2e-6)
    np.testing.assert_allclose(got.sum(axis=1), np.ones(got.shape[0]), atol=1e-6)
    assert np.all(np.triu(got, 1) == 0.0)


def test_selection_mask_from_padded_indices():
    idx = torch.tensor([[0, -1, -1], [0, 1, -1], [0, 2, 1]], dtype=torch.int32)
    cnt = torch.tensor([1, 2, 2], dtype=torch.int32)
    m = bench.selection_mask(idx, cnt, 3).numpy()
    np.testing.assert_array_equal(m, [[1, 0, 0], [1, 1, 0], [1, 0, 1]])


def test_best_mask_budget_and_forced_blocks():
    rng = np.random.default_rng(5)
    b = 23
    M = torch.tensor(np.tril(rng.uniform(size=(b, b))))
    for pct in (10, 20, 50, 100):
        m = bench.best_mask(M, pct).numpy()
        for i in range(b):
            tau = min(max(-(-(i + 1) * pct // 100), len({0, i})), i + 1)
            assert m[i].sum() == tau and m[i, 0] and m[i, i]
            assert not m[i, i + 1:].any()
            chosen = [j for j in range(1, i) if m[i, j]]
            dropped = [j for j in range(1, i) if not m[i, j]]
            if chosen and dropped:
                assert min(M[i, j] for j in chosen) >= max(M[i, j] for j in dropped)
    assert bench.best_mask(M, 100).numpy().sum() == b * (b + 1) // 2


def test_needle_plan_matches_planted_keys():
    """Each planted needle block holds the group-mean query of position p
    plus N(0, 0.1^2) noise."""
    w = synth.scaled(synth.WORKLOADS["tiny"], needles=3)
    _, _, _, (Q, K, _) = synth.prefill_layer_inputs(w, 1, keep_fp32=True)
    plan = synth.needle_plan(w, 1)
    assert len(plan) == 1 and len(plan[0]) == 3
    for jstar, p in plan[0]:
        assert p >= (jstar + 1) * w.B
        blk = K[0, jstar * w.B:(jstar + 1) * w.B]
        dev = (blk - Q[0, p][None, :]).numpy()
        assert 0.05 < dev.std() < 0.2 and np.abs(dev).max() < 0.8
