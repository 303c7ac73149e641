"""GPU parity of the prefill hot path against the fp64 oracle, through the
C ABI: sketch scores, walk update, top-tau selection and block-sparse
attention, each in isolation and end to end."""
import math

import numpy as np
import pytest
import torch

import oracle as O
import synth
from paper_2602_07397_amd import binding as sw

pytestmark = pytest.mark.gpu

U = pytest.importorskip("_gpu_util")


def _bf16_case(seqlens, h_q=8, h_kv=2, d=128, B=128, seed_index=40, needles=2):
    w = synth.Workload("case", seed_index, layers=1, h_q=h_q, h_kv=h_kv, d=d, B=B,
                       dtype="bf16", pct=20, seqlens=tuple(seqlens), needles=needles)
    return w


# ---------------------------------------------------------------------------
# sketch_scores
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("n", [2048, 1000])
def test_sketch_matches_oracle_fp32(n):
    w = synth.scaled(synth.WORKLOADS["tiny"], seqlens=(n,))
    Q, K, _ = synth.prefill_layer_inputs(w, 0)
    signs, cols, ts, tc = U.srht_dev(w.d, w.r, w.seed)
    cu = synth.cu_seqlens(w.seqlens)
    sk = sw.sketch_scores(U.to_dev(Q), U.to_dev(K), cu, w.B, ts, tc, want_means=True)
    ref = O.sketch_scores(Q, K, w.B, signs, cols)
    A = sk["A"].cpu().numpy().reshape(ref["A"].shape)
    scale = np.max(np.abs(ref["A"]))
    assert U.max_abs(A, ref["A"]) <= 1e-12 * scale
    np.testing.assert_allclose(sk["Qbar"].cpu().numpy(), ref["qbar"], rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(sk["Kbar"].cpu().numpy(), ref["kbar"], rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(sk["Qs"].cpu().numpy(), ref["Qs"], rtol=1e-11, atol=1e-14)
    np.testing.assert_allclose(sk["Ks"].cpu().numpy(), ref["Ks"], rtol=1e-11, atol=1e-14)
    assert sk["A_scale"].item() == pytest.approx(ref["c"], rel=1e-12)


@pytest.mark.parametrize("B,d", [(128, 128), (64, 128), (64, 64), (16, 32), (32, 256), (16, 16)])
def test_sketch_matches_oracle_bf16_gqa_varlen(B, d):
    w = _bf16_case((1000, 384, 257, 64), d=d, B=B)
    Q, K, _ = synth.prefill_layer_inputs(w, 0)
    r = min(64, d)
    signs, cols, ts, tc = U.srht_dev(d, r, w.seed)
    cu = synth.cu_seqlens(w.seqlens)
    sk = sw.sketch_scores(U.to_dev(Q), U.to_dev(K), cu, B, ts, tc, want_means=True)
    As = U.split_mats(sk["A"].cpu().numpy(), cu, B)
    Qs = U.split_rows(sk["Qs"].cpu().numpy(), cu, B)
    Qb = U.split_rows(sk["Qbar"].cpu().numpy(), cu, B)
    scales = sk["A_scale"].cpu().numpy()
    for si, (a, e) in enumerate(zip(cu[:-1], cu[1:])):
        ref = O.sketch_scores(Q[:, a:e], K[:, a:e], B, signs, cols)
        c = np.max(np.abs(ref["A"]))
        assert U.max_abs(As[si], ref["A"]) <= 1e-12 * c, si
        np.testing.assert_allclose(Qs[si], ref["Qs"], rtol=1e-10, atol=1e-14)
        np.testing.assert_allclose(Qb[si], ref["qbar"], rtol=1e-12, atol=1e-15)
        assert scales[si] == pytest.approx(ref["c"], rel=1e-12)
        assert np.all(np.triu(As[si], 1) == 0.0)


# ---------------------------------------------------------------------------
# walk_update
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("s", [1, 2, 8])
def test_walk_matches_oracle_over_layers(s):
    bs = [5, 17, 40, 1]
    B = 16
    cu = synth.cu_seqlens([b * B for b in bs])
    rng = np.random.default_rng(100 + s)
    R_gpu = None
    R_ref = [None] * len(bs)
    for layer in range(4):
        mats = [np.tril(rng.normal(size=(b, b))) for b in bs]
        if layer == 2:
            mats[1] = np.zeros_like(mats[1])          # an all-zero layer: c falls back to 1
        flat = np.concatenate([m.ravel() for m in mats])
        scales = np.array([O.score_scale(m) if np.any(m) else 0.0 for m in mats])
        R_gpu = sw.walk_update(U.to_dev(flat), U.to_dev(scales), s, cu, B, R_gpu)
        for k, m in enumerate(mats):
            R_ref[k] = O.walk_step(R_ref[k], O.walk_weights(m, O.score_scale(m), s))
        got = U.split_mats(R_gpu.cpu().numpy(), cu, B)
        for k in range(len(bs)):
            assert U.max_abs(got[k], R_ref[k]) <= 1e-12, (layer, k)
            assert np.all(np.triu(got[k], 1) == 0.0)


# ---------------------------------------------------------------------------
# select_topk_blocks (values are the same fp64 bits on both sides: exact)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("kind", ["continuous", "ties", "zeros"])
@pytest.mark.parametrize("mode", [(0, 20, 3), (0, 100, 3), (0, 37, 1), (4, 0, 0), (3, 0, 2), (1, 0, 3)])
def test_select_is_exact(kind, mode):
    k, pct, flags = mode
    bs = [1, 2, 7, 33, 130, 300]
    B = 16
    cu = synth.cu_seqlens([b * B for b in bs])
    rng = np.random.default_rng(7)
    mats = []
    for b in bs:
        if kind == "continuous":
            m = rng.uniform(0, 1, size=(b, b))
        elif kind == "ties":
            m = rng.integers(0, 3, size=(b, b)).astype(np.float64)
        else:
            m = np.zeros((b, b))
        mats.append(np.tril(m))
    flat = np.concatenate([m.ravel() for m in mats])
    idx, cnt, kmax = sw.select_topk_blocks(U.to_dev(flat), cu, B, k=k, density_pct=max(pct, 1),
                                           flags=flags)
    got = U.gpu_selection(idx, cnt)
    ih = idx.cpu().numpy()
    r = 0
    for m in mats:
        ref, _ = O.select_blocks(m, pct=pct, k=k, flags=flags)
        for i, want in enumerate(ref):
            assert got[r] == want, (kind, mode, r, got[r], want)
            assert np.all(ih[r, len(want):] == -1)
            r += 1


def test_select_handles_negative_values_and_negative_zero():
    B = 16
    m = np.tril(np.array([[0.0, 0, 0, 0], [-0.0, 0.0, 0, 0], [-1.0, -0.0, 0.5, 0], [-2.0, 3.0, -0.0, 0.0]]))
    m[1, 0] = -0.0
    idx, cnt, kmax = sw.select_topk_blocks(U.to_dev(m.ravel()), [0, 4 * B], B, k=2, flags=0)
    ref, _ = O.select_blocks(m, k=2, flags=0)
    assert U.gpu_selection(idx, cnt) == ref


# ---------------------------------------------------------------------------
# sparse_attn_prefill (same selection on both sides)
# ---------------------------------------------------------------------------

def _random_selection(cu, B, rng, p=0.3):
    sel = []
    for a, e in zip(cu[:-1], cu[1:]):
        b = -(-(int(e) - int(a)) // B)
        for i in range(b):
            others = [j for j in range(1, i) if rng.uniform() < p]
            sel.append(sorted(set([0, i] + others)))
    return sel


def _pack(sel):
    kmax = max(len(s) for s in sel)
    idx = np.full((len(sel), kmax), -1, dtype=np.int32)
    cnt = np.zeros(len(sel), dtype=np.int32)
    for r, s in enumerate(sel):
        idx[r, :len(s)] = s
        cnt[r] = len(s)
    return U.to_dev(idx), U.to_dev(cnt), kmax


def _oracle_attention(Q, K, V, cu, B, sel):
    outs = []
    r = 0
    for a, e in zip(cu[:-1], cu[1:]):
        b = -(-(int(e) - int(a)) // B)
        outs.append(O.sparse_attention_prefill(Q[:, a:e], K[:, a:e], V[:, a:e], B, sel[r:r + b]))
        r += b
    return np.concatenate(outs, axis=1)


@pytest.mark.parametrize("n,B,d", [(2048, 64, 64), (1000, 64, 64), (700, 128, 128), (333, 64, 128)])
def test_attention_fp32_matches_oracle(n, B, d):
    w = synth.Workload("f32case", 41, layers=1, h_q=2, h_kv=1, d=d, B=B, dtype="f32", pct=20,
                       seqlens=(n,), needles=2, local_window=False)
    Q, K, V = synth.prefill_layer_inputs(w, 0)
    cu = synth.cu_seqlens(w.seqlens)
    sel = _random_selection(cu, B, np.random.default_rng(n))
    idx, cnt, kmax = _pack(sel)
    out, lse = sw.sparse_attn_prefill(U.to_dev(Q), U.to_dev(K), U.to_dev(V), cu, B, idx, cnt, kmax,
                                      want_lse=True)
    ref = _oracle_attention(Q, K, V, cu, B, sel)
    assert U.max_abs(out.cpu().numpy(), ref) <= U.ATOL_F32
    assert torch.isfinite(lse).all()


@pytest.mark.parametrize("seqlens,h_q,h_kv,d,B", [
    ((1000,), 8, 2, 128, 128),
    ((700, 256, 129), 8, 2, 128, 128),
    ((500,), 4, 1, 128, 64),
    ((640,), 4, 4, 128, 64),
    ((384, 200), 6, 2, 64, 128),
    ((300,), 3, 1, 64, 64),
])
def test_attention_bf16_matches_oracle(seqlens, h_q, h_kv, d, B):
    w = _bf16_case(seqlens, h_q=h_q, h_kv=h_kv, d=d, B=B, seed_index=42)
    Q, K, V = synth.prefill_layer_inputs(w, 0)
    cu = synth.cu_seqlens(w.seqlens)
    sel = _random_selection(cu, B, np.random.default_rng(sum(seqlens)))
    idx, cnt, kmax = _pack(sel)
    out = sw.sparse_attn_prefill(U.to_dev(Q), U.to_dev(K), U.to_dev(V), cu, B, idx, cnt, kmax)
    ref = _oracle_attention(Q, K, V, cu, B, sel)
    assert U.max_abs(out.float().cpu().numpy(), ref) <= U.ATOL_BF16


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_density_100_equals_dense_causal(dtype):
    n, B = 777, 64 if dtype == "f32" else 128
    w = synth.Workload("dense", 43, layers=1, h_q=4, h_kv=2, d=128, B=B, dtype=dtype, pct=100,
                       seqlens=(n,), needles=2)
    Q, K, V = synth.prefill_layer_inputs(w, 0)
    signs, cols, ts, tc = U.srht_dev(w.d, w.r, w.seed)
    cu = synth.cu_seqlens(w.seqlens)
    res = U.gpu_prefill_layer(U.to_dev(Q), U.to_dev(K), U.to_dev(V), cu, B, ts, tc, 8, None, pct=100)
    b = -(-n // B)
    assert U.gpu_selection(res["idx"], res["cnt"]) == [list(range(i + 1)) for i in range(b)]
    ref = O.dense_causal_attention(Q, K, V)
    tol = U.ATOL_BF16 if dtype == "bf16" else U.ATOL_F32
    assert U.max_abs(res["O"].float().cpu().numpy(), ref) <= tol


# ---------------------------------------------------------------------------
# end to end
# ---------------------------------------------------------------------------

def test_tiny_workload_end_to_end():
    """2 layers x 1 head, n=2048, d=64, B=64, fp32, density 20%, planted sink
    and needles: selections exact where the oracle gap exceeds 1e-4, outputs
    within 1e-5 of the oracle's masked attention."""
    w = synth.WORKLOADS["tiny"]
    signs, cols, ts, tc = U.srht_dev(w.d, w.r, w.seed)
    cu = synth.cu_seqlens(w.seqlens)
    R_gpu, R_ref = None, None
    for layer in range(w.layers):
        Q, K, V = synth.prefill_layer_inputs(w, layer)
        res = U.gpu_prefill_layer(U.to_dev(Q), U.to_dev(K), U.to_dev(V), cu, w.B, ts, tc, w.s,
                                  R_gpu, pct=w.pct)
        R_gpu = res["R"]
        ref = O.prefill_layer(Q, K, V, w.B, signs, cols, w.s, R_ref, pct=w.pct, attention=False)
        R_ref = ref["R"]
        got = U.gpu_selection(res["idx"], res["cnt"])
        U.check_selection(got, ref["sel"], ref["gaps"], R_ref)
        assert U.max_abs(res["R"].cpu().numpy().reshape(R_ref.shape), R_ref) <= 1e-9
        out = O.sparse_attention_prefill(Q, K, V, w.B, got)
        assert U.max_abs(res["O"].cpu().numpy(), out) <= U.ATOL_F32
        # with identical selections the outputs agree with the oracle pipeline too
        full = O.sparse_attention_prefill(Q, K, V, w.B, ref["sel"])
        same = [i for i in range(len(got)) if got[i] == ref["sel"][i]]
        rows = np.concatenate([np.arange(i * w.B, (i + 1) * w.B) for i in same])
        assert U.max_abs(res["O"].cpu().numpy()[:, rows], full[:, rows]) <= U.ATOL_F32


def test_outputs_are_deterministic():
    w = _bf16_case((1500, 300), seed_index=44)
    Q, K, V = [U.to_dev(x) for x in synth.prefill_layer_inputs(w, 0)]
    signs, cols, ts, tc = U.srht_dev(w.d, w.r, w.seed)
    cu = synth.cu_seqlens(w.seqlens)
    a = U.gpu_prefill_layer(Q, K, V, cu, w.B, ts, tc, 8, None)
    b = U.gpu_prefill_layer(Q, K, V, cu, w.B, ts, tc, 8, None)
    for key in ("A", "A_scale", "Qs", "Ks", "R", "idx", "cnt", "O"):
        assert torch.equal(a[key], b[key]), key
