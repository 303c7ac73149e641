"""Pins for the oracle's decode path (Alg. 2): running block means, the
incremental score updates, the walk row, selection and single-token
attention."""
import math

import numpy as np
import pytest

import oracle as O


def _setup(seed=0, h_q=4, h_kv=2, n0=21, steps=14, d=8, B=4, layers=3):
    rng = np.random.default_rng(seed)
    T = n0 + steps
    Qs = [rng.normal(size=(h_q, T, d)) for _ in range(layers)]
    Ks = [rng.normal(size=(h_kv, T, d)) for _ in range(layers)]
    Vs = [rng.normal(size=(h_kv, T, d)) for _ in range(layers)]
    signs = rng.choice([-1, 1], size=d)
    cols = rng.permutation(d)          # r = d: exact sketch
    b_max = -(-T // B)
    states = [O.decode_state_from_prefill(Qs[l][:, :n0], Ks[l][:, :n0], B, signs, cols, b_max)
              for l in range(layers)]
    return dict(Q=Qs, K=Ks, V=Vs, signs=signs, cols=cols, states=states, n0=n0, T=T, B=B, d=d)


def _run(env, p_from, p_to, states, pct=40):
    out = []
    for p in range(p_from, p_to):
        r = None
        per_layer = []
        for l, st in enumerate(states):
            r, sel, gap = O.decode_layer_step(st, env["Q"][l][:, p], env["K"][l][:, p], p, r,
                                              env["B"], env["signs"], env["cols"], 8, pct=pct)
            per_layer.append((r.copy(), sel))
        out.append(per_layer)
    return out


def test_open_block_mean_equals_block_mean():
    env = _setup()
    _run(env, env["n0"], env["T"], env["states"])
    B, T = env["B"], env["T"]
    for l, st in enumerate(env["states"]):
        kb = O.block_means(O.head_mean(env["K"][l][:, :T]), B)
        qb = O.block_means(O.head_mean(env["Q"][l][:, :T]), B)
        np.testing.assert_allclose(st.kbar[:kb.shape[0]], kb, rtol=1e-12, atol=1e-13)
        np.testing.assert_allclose(st.qbar[:qb.shape[0]], qb, rtol=1e-12, atol=1e-13)
        assert st.ktok.shape[0] == st.qtok.shape[0] == T - (kb.shape[0] - 1) * B


def test_score_row_and_column_follow_their_definitions():
    """At r = d: the new query row holds (token query . key block mean)/sqrt(d)
    and the last column holds (query block mean . open key block mean)/sqrt(d)."""
    env = _setup(seed=1)
    p = env["n0"]
    st = env["states"][0]
    O.decode_layer_step(st, env["Q"][0][:, p], env["K"][0][:, p], p, None, env["B"],
                        env["signs"], env["cols"], 8, pct=40)
    B, d = env["B"], env["d"]
    bc = p // B
    qa = O.head_mean(env["Q"][0][:, p:p + 1])[0]
    kb = O.block_means(O.head_mean(env["K"][0][:, :p + 1]), B)
    qb = O.block_means(O.head_mean(env["Q"][0][:, :p + 1]), B)
    for j in range(bc):
        assert abs(st.A[bc, j] - qa @ kb[j] / math.sqrt(d)) < 1e-12
    for m in range(bc + 1):
        assert abs(st.A[m, bc] - qb[m] @ kb[bc] / math.sqrt(d)) < 1e-12


def test_walk_row_equals_row_of_full_product():
    env = _setup(seed=2)
    res = _run(env, env["n0"], env["n0"] + 5, env["states"])
    p = env["n0"] + 4
    bq = p // env["B"]
    mats = []
    for st in env["states"]:
        A = st.A[:bq + 1, :bq + 1]
        mats.append(np.power(A / st.c, 8))
    full = np.linalg.multi_dot(mats) if len(mats) > 1 else mats[0]
    row = full[bq] / np.max(np.abs(full[bq]))
    np.testing.assert_allclose(res[-1][-1][0], row, rtol=1e-10, atol=1e-14)


def test_current_and_first_block_always_selected():
    env = _setup(seed=3)
    res = _run(env, env["n0"], env["T"], env["states"], pct=10)
    for k, per_layer in enumerate(res):
        p = env["n0"] + k
        for _, sel in per_layer:
            assert p // env["B"] in sel and 0 in sel
            tau = O.row_budget(p // env["B"] + 1, len(O.forced_set(p // env["B"], O.FORCE_BOTH)), pct=10)
            assert len(sel) == tau


def test_decode_attention_equals_prefill_row():
    """Decode attention at position p equals row p of the prefill sparse
    attention given the same block selection (two independent code paths)."""
    env = _setup(seed=4)
    B = env["B"]
    Q, K, V = env["Q"][0], env["K"][0], env["V"][0]
    for p in (env["n0"], env["n0"] + 3, env["T"] - 1):
        bq = p // B
        sel = sorted({0, bq} | ({1} if bq > 2 else set()))
        dec = O.decode_attention(Q[:, p], K[:, :p + 1], V[:, :p + 1], sel, p, B)
        for u in range(Q.shape[0]):
            blk = O.sparse_attention_block(Q[:, :p + 1], K[:, :p + 1], V[:, :p + 1], B, sel, u, bq)
            np.testing.assert_allclose(dec[u], blk[p - bq * B], rtol=1e-12, atol=1e-12)


def test_state_round_trip_is_bit_identical():
    env = _setup(seed=5)
    a = [st.copy() for st in env["states"]]
    b = [st.copy() for st in env["states"]]
    n0, T = env["n0"], env["T"]
    mid = (n0 + T) // 2
    ra = _run(env, n0, T, a)
    _run(env, n0, mid, b)
    saved = [st.copy() for st in b]          # checkpoint
    rb = _run(env, mid, T, saved)
    for (x, y) in zip(ra[mid - n0:], rb):
        for (rx, sx), (ry, sy) in zip(x, y):
            assert sx == sy
            np.testing.assert_array_equal(rx, ry)


def test_state_from_prefill_places_the_prompt_scores():
    """The decode caches taken over from an n-token prompt (n not a multiple
    of B): at r = d the score cache holds the Sec. 2.1 block score (the
    literal double sum over token pairs divided by sqrt(d)) at (i, j) for
    j <= i < b, zero everywhere else of the b_max x b_max cache; the block
    representatives are the per-block token means and the open block's token
    list holds the head-averaged tokens of the prompt's last block."""
    rng = np.random.default_rng(11)
    h_q, h_kv, d, B, n, b_max = 4, 2, 8, 4, 18, 9
    Q = rng.normal(size=(h_q, n, d))
    K = rng.normal(size=(h_kv, n, d))
    signs = rng.choice([-1, 1], size=d)
    cols = rng.permutation(d)
    st = O.decode_state_from_prefill(Q, K, B, signs, cols, b_max)
    b = -(-n // B)
    Qa = np.array([[sum(Q[u, t, e] for u in range(h_q)) / h_q for e in range(d)] for t in range(n)])
    Ka = np.array([[sum(K[g, t, e] for g in range(h_kv)) / h_kv for e in range(d)] for t in range(n)])
    want = np.zeros((b_max, b_max))
    for i in range(b):
        for j in range(i + 1):
            want[i, j] = O.block_score_true(Qa, Ka, B, i, j)
    np.testing.assert_allclose(st.A, want, rtol=1e-12, atol=1e-13)
    assert st.c == pytest.approx(np.max(np.abs(want)), rel=1e-12)
    for i in range(b):
        lo, hi = i * B, min(n, (i + 1) * B)
        np.testing.assert_allclose(st.qbar[i], Qa[lo:hi].mean(axis=0), rtol=1e-12, atol=1e-14)
        np.testing.assert_allclose(st.kbar[i], Ka[lo:hi].mean(axis=0), rtol=1e-12, atol=1e-14)
    assert not st.qbar[b:].any() and not st.kbar[b:].any()
    np.testing.assert_allclose(st.qtok, Qa[(b - 1) * B:], rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(st.ktok, Ka[(b - 1) * B:], rtol=1e-12, atol=1e-14)
