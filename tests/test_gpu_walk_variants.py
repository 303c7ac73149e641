"""GPU parity of the walk transition variants against the fp64 oracle,
through the C ABI: the power after clipping negative scores, the causal row
softmax and the matrix power, in prefill; the clipped power in decode."""
import math

import numpy as np
import pytest

import oracle as O
import synth
from paper_2602_07397_amd import binding as sw

pytestmark = pytest.mark.gpu

U = pytest.importorskip("_gpu_util")

EPS = np.finfo(np.float64).eps

ORACLE_VARIANT = {sw.WALK_POWER: O.WALK_POWER, sw.WALK_RELU: O.WALK_RELU,
                  sw.WALK_SOFTMAX: O.WALK_SOFTMAX, sw.WALK_MATPOW: O.WALK_MATPOW}


def _matpow_row_tol(A, c, s, R_prev):
    """Forward error bound of R = normalize(R_prev (A/c)^s) per row.
    A product of b-term dot products errs by at most gamma_b |X||Y|
    (gamma_b = b eps / (1 - b eps)); a chain of squarings and products for
    the power s accumulates at most (s + 2) such terms, on each side (the
    oracle's s - 1 successive products and the library's binary
    exponentiation), measured against |R_prev| |A/c|^s and divided by the
    row's largest magnitude."""
    b = A.shape[0]
    gamma = b * EPS / (1.0 - b * EPS)
    absW = O.walk_weights_matpow(np.abs(A), c, s)
    Rp = np.eye(b) if R_prev is None else np.abs(R_prev)
    absP = Rp @ absW
    P = O.walk_step(R_prev, O.walk_weights_matpow(A, c, s), normalize=False)
    tol = np.zeros(b)
    for i in range(b):
        m = np.max(np.abs(P[i]))
        tol[i] = 0.0 if m == 0.0 else 4.0 * (s + 2) * gamma * np.max(absP[i]) / m
    return tol + 1e-15


@pytest.mark.parametrize("variant,s", [(sw.WALK_RELU, 8), (sw.WALK_RELU, 3), (sw.WALK_SOFTMAX, 8),
                                       (sw.WALK_MATPOW, 2), (sw.WALK_MATPOW, 3),
                                       (sw.WALK_MATPOW, 8), (sw.WALK_MATPOW, 1),
                                       (sw.WALK_POWER, 8)])
def test_walk_variant_matches_oracle_per_layer(variant, s):
    """Four layers of signed lower triangular scores on ragged sizes (one
    sequence of a single block, tiles with a ragged edge, an all-zero layer
    whose scale falls back to 1). Each layer starts from the oracle's R_prev,
    so the comparison bounds one layer's rounding."""
    bs = [5, 17, 40, 1]
    B = 16
    cu = synth.cu_seqlens([b * B for b in bs])
    rng = np.random.default_rng(300 + 10 * variant + s)
    t = math.sqrt(32 / 128)
    R_ref = [None] * len(bs)
    for layer in range(4):
        mats = [np.tril(rng.normal(size=(b, b))) for b in bs]
        if layer == 2:
            mats[1] = np.zeros_like(mats[1])
        flat = np.concatenate([m.ravel() for m in mats])
        scales = np.array([O.score_scale(m) if np.any(m) else 0.0 for m in mats])
        R_prev = None if layer == 0 else U.to_dev(np.concatenate([r.ravel() for r in R_ref]))
        R_gpu = sw.walk_update_variant(variant, U.to_dev(flat), U.to_dev(scales), s, cu, B, R_prev,
                                       logit_scale=t)
        got = U.split_mats(R_gpu.cpu().numpy(), cu, B)
        for k, m in enumerate(mats):
            c = O.score_scale(m)
            W = O.walk_weights_variant(ORACLE_VARIANT[variant], m, c, s, t)
            ref = O.walk_step(R_ref[k], W)
            assert np.all(np.triu(got[k], 1) == 0.0), (layer, k)
            if variant == sw.WALK_MATPOW:
                tol = _matpow_row_tol(m, c, s, R_ref[k])
                err = np.max(np.abs(got[k] - ref), axis=1)
                assert np.all(err <= tol), (layer, k, err, tol)
            else:
                assert U.max_abs(got[k], ref) <= 1e-12, (layer, k)
            R_ref[k] = ref


@pytest.mark.parametrize("variant", [sw.WALK_RELU, sw.WALK_SOFTMAX, sw.WALK_MATPOW])
def test_walk_variant_selection_on_workload(variant):
    """The small fp32 workload (n = 2048, d = 64, B = 64, planted sink and
    needles) through sketch, variant walk and selection over its layers on
    both sides: selections exact wherever the oracle's boundary gap exceeds
    1e-4."""
    w = synth.WORKLOADS["tiny"]
    signs, cols, ts, tc = U.srht_dev(w.d, w.r, w.seed)
    cu = synth.cu_seqlens(w.seqlens)
    t = math.sqrt(w.r / w.d)
    R_gpu, R_ref = None, None
    for layer in range(w.layers):
        Q, K, _ = synth.prefill_layer_inputs(w, layer)
        sk = sw.sketch_scores(U.to_dev(Q), U.to_dev(K), cu, w.B, ts, tc)
        R_gpu = sw.walk_update_variant(variant, sk["A"], sk["A_scale"], w.s, cu, w.B, R_gpu,
                                       logit_scale=t)
        idx, cnt, _ = sw.select_topk_blocks(R_gpu, cu, w.B, density_pct=w.pct)
        ref = O.sketch_scores(Q, K, w.B, signs, cols)
        W = O.walk_weights_variant(ORACLE_VARIANT[variant], ref["A"], ref["c"], w.s, t)
        R_ref = O.walk_step(R_ref, W)
        sel, gaps = O.select_blocks(R_ref, pct=w.pct)
        near = U.check_selection(U.gpu_selection(idx, cnt), sel, gaps, R_ref)
        assert near <= 0.05 * len(sel), (layer, near)
        Rg = R_gpu.cpu().numpy().reshape(R_ref.shape)
        assert U.max_abs(Rg, R_ref) <= (1e-6 if variant == sw.WALK_MATPOW else 1e-9)


def test_walk_variant_rejects_bad_arguments():
    cu = [0, 64]
    A = U.to_dev(np.zeros(16))
    c = U.to_dev(np.ones(1))
    with pytest.raises(sw.SketchWalkError):
        sw.walk_update_variant(7, A, c, 8, cu, 16)
    with pytest.raises(sw.SketchWalkError):
        sw.walk_update_variant(sw.WALK_MATPOW, A, c, 65, cu, 16)
    with pytest.raises(sw.SketchWalkError):
        sw.walk_update_variant(sw.WALK_SOFTMAX, A, c, 8, cu, 16, logit_scale=float("nan"))
    ws = U.to_dev(np.zeros(1, dtype=np.uint8))
    with pytest.raises(sw.SketchWalkError):   # matrix power needs 2 * 16 doubles of workspace
        rc = sw.load().sw_walk_update_variant(
            sw.WALK_MATPOW, A.data_ptr(), c.data_ptr(), 8, 1.0, 1, sw._cu(cu)[0], 16, None,
            U.to_dev(np.zeros(16)).data_ptr(), ws.data_ptr(), 1, None)
        sw._check(rc, "sw_walk_update_variant")


def test_decode_relu_walk_matches_oracle():
    """Decode (Alg. 2 steps 2-7) with the clipped power in the walk row."""
    test_gpu_decode = pytest.importorskip("test_gpu_decode")
    w = synth.Workload("dec", 45, layers=3, h_q=8, h_kv=2, d=128, B=64, dtype="bf16", pct=20,
                       needles=2, batch=3, kv_len=1000, steps=60)
    run = test_gpu_decode.DecodeRun(w, prompts=[1000, 640, 65], steps=40, variant=sw.WALK_RELU)
    near = rows = 0
    for k in range(run.steps):
        st = run.step(k)
        assert st["werr"] <= 1e-4, (k, st)
        assert st["err"] <= U.ATOL_BF16, (k, st)
        near += st["near"]
        rows += st["rows"]
    assert near <= 0.05 * rows


def test_decode_softmax_and_matpow_are_unsupported():
    state = sw.new_decode_state(1, 64, 16, 4, U.DEV)
    pos = U.to_dev(np.array([3], dtype=np.int32))
    for v in (sw.WALK_SOFTMAX, sw.WALK_MATPOW):
        with pytest.raises(sw.SketchWalkError, match="code 2"):
            sw.walk_update_decode_variant(v, state, 1, 64, 16, 4, 16, pos, 8)
