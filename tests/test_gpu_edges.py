"""Edge cases of the prefill path through the C ABI, against the oracle: the
largest supported block count per sequence (walk product and selection),
one-token and one-block sequences mixed into a varlen batch, all-zero
queries and keys (every score 0: the scale falls back to 1, the walk state is
zero and the selection is decided by the tie rule), and sizes past the
supported maximum (rejected before any launch)."""
import numpy as np
import pytest
import torch

import oracle as O
import synth
from paper_2602_07397_amd import binding as sw

pytestmark = pytest.mark.gpu

U = pytest.importorskip("_gpu_util")


def test_walk_and_select_at_max_blocks():
    """One sequence of SW_MAX_BLOCKS blocks: the walk product of two layers
    and the 20 % selection, checked on sampled rows (every selection row is
    checked for size, order and forced blocks)."""
    b = sw.MAX_BLOCKS
    B = 16
    cu = [0, b * B]
    rng = np.random.default_rng(900)
    A0 = np.tril(rng.uniform(-1.0, 1.0, size=(b, b)))
    A1 = np.tril(rng.uniform(-1.0, 1.0, size=(b, b)))
    c0, c1 = O.score_scale(A0), O.score_scale(A1)
    R0 = sw.walk_update(U.to_dev(A0.ravel()), U.to_dev(np.array([c0])), 8, cu, B)
    R1 = sw.walk_update(U.to_dev(A1.ravel()), U.to_dev(np.array([c1])), 8, cu, B, R0)
    idx, cnt, kmax = sw.select_topk_blocks(R1, cu, B, density_pct=20)
    W0 = O.walk_weights(A0, c0, 8)
    W1 = O.walk_weights(A1, c1, 8)
    ref0 = O.walk_step(None, W0)
    rows = [0, 1, 2, 100, 1000, 2047, 2048, 3333, b - 2, b - 1]
    got1 = R1.cpu().numpy().reshape(b, b)
    ref1_rows = O.normalize_rows(ref0[rows] @ W1)
    assert U.max_abs(got1[rows], ref1_rows) <= 1e-12
    assert np.all(np.triu(got1, 1) == 0.0)
    sel = U.gpu_selection(idx, cnt)
    for i in rows:
        want, gap = O.select_row(ref1_rows[rows.index(i)], i + 1, O.forced_set(i, O.FORCE_BOTH),
                                 O.row_budget(i + 1, len(O.forced_set(i, O.FORCE_BOTH)), pct=20))
        if gap > U.GAP_TOL:
            assert sel[i] == want, i
    for i, s in enumerate(sel):
        tau = O.row_budget(i + 1, len(O.forced_set(i, O.FORCE_BOTH)), pct=20)
        assert len(s) == tau and s == sorted(set(s)) and 0 in s and i in s and s[-1] <= i


def test_sizes_past_the_maximum_are_rejected():
    B = 16
    cu = [0, (sw.MAX_BLOCKS + 1) * B]
    A = torch.zeros(1, dtype=torch.float64, device=U.DEV)
    with pytest.raises(sw.SketchWalkError, match="code 2"):
        sw.walk_update(A, A, 8, cu, B)
    with pytest.raises(sw.SketchWalkError, match="code 1"):
        sw.walk_update(A, A, 8, [0] + [B] * (sw.MAX_SEQS + 1), B)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_one_token_and_one_block_sequences(dtype):
    """A varlen batch with sequences of 1, 2, 63, 64 and 65 tokens (B = 64):
    partial single blocks, an exact block and a one-token second block, end
    to end (sketch, walk, select, attention) against the oracle."""
    seqlens = (1, 65, 2, 64, 63)
    w = synth.Workload("edge", 47, layers=1, h_q=4, h_kv=2, d=64, B=64, dtype=dtype, pct=20,
                       seqlens=seqlens, needles=0, local_window=False)
    Q, K, V = synth.prefill_layer_inputs(w, 0)
    signs, cols, ts, tc = U.srht_dev(w.d, w.r, w.seed)
    cu = synth.cu_seqlens(seqlens)
    res = U.gpu_prefill_layer(U.to_dev(Q), U.to_dev(K), U.to_dev(V), cu, w.B, ts, tc, 8, None,
                              pct=w.pct)
    got = U.gpu_selection(res["idx"], res["cnt"])
    Og = res["O"].float().cpu().numpy()
    Rg = U.split_mats(res["R"].cpu().numpy(), cu, w.B)
    r = 0
    tol = U.ATOL_BF16 if dtype == "bf16" else U.ATOL_F32
    for si, (a, e) in enumerate(zip(cu[:-1], cu[1:])):
        ref = O.prefill_layer(Q[:, a:e], K[:, a:e], V[:, a:e], w.B, signs, cols, 8, None, pct=w.pct)
        bs = len(ref["sel"])
        assert U.max_abs(Rg[si], ref["R"]) <= 1e-12
        U.check_selection(got[r:r + bs], ref["sel"], ref["gaps"], ref["R"])
        out = O.sparse_attention_prefill(Q[:, a:e], K[:, a:e], V[:, a:e], w.B, got[r:r + bs])
        assert U.max_abs(Og[:, a:e], out) <= tol, si
        r += bs


def test_all_zero_queries_and_keys():
    """Q = K = 0: A = 0, the scale falls back to 1, W = R = 0, every row ties,
    so the selection is the forced blocks plus the lowest-index others; the
    attention weights are uniform over the selected causal keys."""
    n, B, d = 640, 64, 64
    Q = torch.zeros((2, n, d), dtype=torch.float32)
    K = torch.zeros((1, n, d), dtype=torch.float32)
    V = torch.randn((1, n, d), generator=torch.Generator().manual_seed(5), dtype=torch.float32)
    signs, cols, ts, tc = U.srht_dev(d, 32, 48)
    cu = [0, n]
    res = U.gpu_prefill_layer(U.to_dev(Q), U.to_dev(K), U.to_dev(V), cu, B, ts, tc, 8, None, pct=30)
    assert res["A_scale"].item() == 0.0
    assert torch.count_nonzero(res["R"]).item() == 0
    got = U.gpu_selection(res["idx"], res["cnt"])
    ref = O.prefill_layer(Q.numpy(), K.numpy(), V.numpy(), B, signs, cols, 8, None, pct=30)
    assert got == ref["sel"]
    out = O.sparse_attention_prefill(Q.numpy(), K.numpy(), V.numpy(), B, got)
    assert U.max_abs(res["O"].cpu().numpy(), out) <= U.ATOL_F32
