"""Helpers shared by the GPU parity tests (not collected by pytest).

They run the HIP path through the C ABI binding and compare it with the fp64
oracle on the same seeded inputs.
"""
from __future__ import annotations

import math
from typing import Dict, List, Sequence

import numpy as np
import torch

import oracle as O
import synth
from paper_2602_07397_amd import binding as sw

DEV = torch.device("cuda:0")

# Tolerances: attention outputs vs the fp64 oracle given the same selection.
ATOL_BF16 = 2e-2
ATOL_F32 = 1e-5
# Selection indices must match exactly on rows whose oracle boundary gap is
# larger than this (relative).
GAP_TOL = 1e-4


def to_dev(x, dtype=None):
    t = torch.as_tensor(x)
    if dtype is not None:
        t = t.to(dtype)
    return t.contiguous().to(DEV)


def srht_dev(d: int, r: int, seed: int):
    signs, cols = synth.srht_params(d, r, seed)
    return signs, cols, to_dev(signs), to_dev(cols)


def gpu_prefill_layer(Q, K, V, cu, B, ts, tc, s, R_prev, pct=20, k=0, flags=sw.FORCE_BOTH,
                      attention=True) -> Dict:
    sk = sw.sketch_scores(Q, K, cu, B, ts, tc, want_means=True)
    R = sw.walk_update(sk["A"], sk["A_scale"], s, cu, B, R_prev)
    idx, cnt, kmax = sw.select_topk_blocks(R, cu, B, k=k, density_pct=pct, flags=flags)
    out = dict(sk, R=R, idx=idx, cnt=cnt, kmax=kmax)
    if attention:
        out["O"] = sw.sparse_attn_prefill(Q, K, V, cu, B, idx, cnt, kmax)
    return out


def split_rows(flat: np.ndarray, cu, B) -> List[np.ndarray]:
    """Per-sequence views of a [nb][...] array."""
    out, r = [], 0
    for a, e in zip(cu[:-1], cu[1:]):
        b = -(-(int(e) - int(a)) // B)
        out.append(flat[r:r + b])
        r += b
    return out


def split_mats(flat: np.ndarray, cu, B) -> List[np.ndarray]:
    out, o = [], 0
    for a, e in zip(cu[:-1], cu[1:]):
        b = -(-(int(e) - int(a)) // B)
        out.append(flat[o:o + b * b].reshape(b, b))
        o += b * b
    return out


def gpu_selection(idx: torch.Tensor, cnt: torch.Tensor) -> List[List[int]]:
    ih, ch = idx.cpu().numpy(), cnt.cpu().numpy()
    return [ih[r, :ch[r]].tolist() for r in range(ih.shape[0])]


def check_selection(got: Sequence[List[int]], ref: Sequence[List[int]], gaps, R_rows,
                    flags=sw.FORCE_BOTH, gap_tol=GAP_TOL) -> int:
    """Exact on rows whose gap exceeds gap_tol; on the others the two sets
    have the same size, contain the forced blocks and differ only in blocks
    whose oracle values are within gap_tol of the boundary. Returns the
    number of near-tie rows."""
    near = 0
    for i, (g, r) in enumerate(zip(got, ref)):
        assert g == sorted(set(g)), (i, g)
        if gaps[i] > gap_tol:
            assert g == r, (i, g, r)
            continue
        near += 1
        assert len(g) == len(r), (i, g, r)
        F = set(O.forced_set(i, flags))
        assert F <= set(g), (i, g)
        vals = R_rows[i]
        ranked = [j for j in r if j not in F]
        if not ranked:
            continue
        vb = min(float(vals[j]) for j in ranked)
        scale = max(abs(vb), 1e-300)
        for j in set(g) ^ set(r):
            assert abs(float(vals[j]) - vb) <= 2 * gap_tol * scale, (i, j, vals[j], vb)
    return near


def max_abs(a, b) -> float:
    return float(np.max(np.abs(np.asarray(a, dtype=np.float64) - np.asarray(b, dtype=np.float64))))
