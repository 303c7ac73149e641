"""Seeded random configurations of the block-sparse prefill attention against
the oracle (the kernel given a selection): ragged varlen batches with 1- to
1500-token sequences, GQA group sizes 1-8 (odd ones leave wavefronts of a
workgroup without rows), B in {64, 128}, d in {64, 128}, bf16 and fp32, and
selections that are random subsets with or without the diagonal block, the
diagonal alone, every block, or padded with entries the kernel must skip
(-1 and blocks after the row)."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2602_07397_amd import binding as sw

pytestmark = pytest.mark.gpu

U = pytest.importorskip("_gpu_util")

N_CASES = 24


def _case(seed):
    rng = np.random.default_rng(1000 + seed)
    dtype = "f32" if seed % 6 == 5 else "bf16"
    B = int(rng.choice([64, 128]))
    d = int(rng.choice([64, 128]))
    h_kv = int(rng.choice([1, 2]))
    G = int(rng.choice([1, 2, 3, 4, 7, 8]))
    nseq = int(rng.integers(1, 5))
    seqlens = [int(rng.integers(1, 1500)) for _ in range(nseq)]
    mode = ["random", "random", "no_diag", "diag_only", "all", "padded"][seed % 6]
    return rng, dtype, B, d, h_kv, G, seqlens, mode


def _selection(rng, cu, B, mode):
    """(rows passed to the kernel, rows the oracle uses)."""
    given, used = [], []
    for a, e in zip(cu[:-1], cu[1:]):
        b = -(-(e - a) // B)
        for i in range(b):
            if mode == "diag_only":
                s = [i]
            elif mode == "all":
                s = list(range(i + 1))
            else:
                p = rng.uniform(0.1, 0.9)
                s = sorted({j for j in range(i) if rng.uniform() < p} | ({i} if mode != "no_diag" else set()))
            g = list(s)
            if mode == "padded":
                g = sorted(g + [-1] * int(rng.integers(0, 3)) + [i + 1 + int(x) for x in
                                                                  range(int(rng.integers(0, 3)))])
            given.append(g)
            used.append([j for j in s if 0 <= j <= i])
    return given, used


@pytest.mark.parametrize("seed", range(N_CASES))
def test_random_configuration_matches_oracle(seed):
    rng, dtype, B, d, h_kv, G, seqlens, mode = _case(seed)
    h_q = G * h_kv
    cu = [0] + list(np.cumsum(seqlens).astype(int))
    N = cu[-1]
    g = torch.Generator().manual_seed(seed)
    Q = torch.randn((h_q, N, d), generator=g)
    K = torch.randn((h_kv, N, d), generator=g)
    V = torch.randn((h_kv, N, d), generator=g)
    td = torch.bfloat16 if dtype == "bf16" else torch.float32
    Q, K, V = Q.to(td), K.to(td), V.to(td)
    given, used = _selection(rng, cu, B, mode)
    kmax = max(1, max(len(s) for s in given))
    idx = np.full((len(given), kmax), -1, dtype=np.int32)
    cnt = np.zeros(len(given), dtype=np.int32)
    for r, s in enumerate(given):
        idx[r, :len(s)] = s
        cnt[r] = len(s)
    out = sw.sparse_attn_prefill(U.to_dev(Q), U.to_dev(K), U.to_dev(V), cu, B, U.to_dev(idx),
                                 U.to_dev(cnt), kmax)
    got = out.float().cpu().numpy()
    tol = U.ATOL_BF16 if dtype == "bf16" else U.ATOL_F32
    Qh, Kh, Vh = O.f64(Q), O.f64(K), O.f64(V)
    r = 0
    for s, (a, e) in enumerate(zip(cu[:-1], cu[1:])):
        b = -(-(e - a) // B)
        rows = used[r:r + b]
        ref = np.zeros((h_q, e - a, d))
        for u in range(h_q):
            for i in range(b):
                if rows[i]:
                    ref[u, i * B:min(e - a, (i + 1) * B)] = O.sparse_attention_block(
                        Qh[:, a:e], Kh[:, a:e], Vh[:, a:e], B, rows[i], u, i)
        # a row whose selection admits no key has no defined softmax: the
        # kernel writes zeros there (rows of a no-diagonal selection before any
        # selected key cannot occur, since every selected block precedes them)
        assert np.isfinite(got[:, a:e]).all(), (seed, s)
        assert U.max_abs(got[:, a:e], ref) <= tol, (seed, s, dtype, B, d, G, mode)
        r += b


def test_rows_selecting_every_block_at_max_blocks():
    """One sequence of SW_MAX_BLOCKS blocks (B = 64): the last rows select
    every block (the longest lists the kernel compacts in LDS), the others
    only their diagonal block."""
    B, d, h_q, h_kv = 64, 64, 2, 1
    b = sw.MAX_BLOCKS
    N = b * B
    g = torch.Generator().manual_seed(91)
    Q = torch.randn((h_q, N, d), generator=g).to(torch.bfloat16)
    K = torch.randn((h_kv, N, d), generator=g).to(torch.bfloat16)
    V = torch.randn((h_kv, N, d), generator=g).to(torch.bfloat16)
    full = {b - 1, b - 2, b - 5}
    sel = [list(range(i + 1)) if i in full else [i] for i in range(b)]
    kmax = b
    idx = np.full((b, kmax), -1, dtype=np.int32)
    cnt = np.array([len(s) for s in sel], dtype=np.int32)
    for r, s in enumerate(sel):
        idx[r, :len(s)] = s
    out = sw.sparse_attn_prefill(U.to_dev(Q), U.to_dev(K), U.to_dev(V), [0, N], B, U.to_dev(idx),
                                 U.to_dev(cnt), kmax)
    got = out.float().cpu().numpy()
    Qh, Kh, Vh = O.f64(Q), O.f64(K), O.f64(V)
    for i in sorted(full) + [0, 1, 1000]:
        for u in range(h_q):
            ref = O.sparse_attention_block(Qh, Kh, Vh, B, sel[i], u, i)
            assert U.max_abs(got[u, i * B:(i + 1) * B], ref) <= U.ATOL_BF16, (i, u)
