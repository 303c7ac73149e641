"""Host-side parts of the benchmark that its numbers rest on: the executed
attention FLOP count (checked against brute-force enumeration of the
(query, key) pairs a selection admits), the source-hash guard of the measured
HBM traffic, and the one-GPU contract of the command line."""
import os
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def _brute_pairs(n, B, sel):
    """Unmasked (query t, key k) pairs: k in a selected block of t's block,
    k <= t, both inside the sequence; full blocks (tile count) alongside."""
    alg = tile = 0
    b = -(-n // B)
    for i in range(b):
        for j in sel[i]:
            qs = range(i * B, min(n, (i + 1) * B))
            ks = range(j * B, min(n, (j + 1) * B))
            tile += len(qs) * len(ks)
            alg += sum(1 for t in qs for k in ks if k <= t)
    return alg, tile


def test_attention_flops_counts_admitted_pairs():
    rng = np.random.default_rng(7)
    B, h_q, d = 16, 3, 32
    seqlens = [50, 16, 1, 37]
    cu = np.concatenate([[0], np.cumsum(seqlens)]).astype(np.int64)
    rows, sels = [], []
    for n in seqlens:
        b = -(-n // B)
        sel = [sorted({i} | {j for j in range(i) if rng.uniform() < 0.5}) for i in range(b)]
        sels.append(sel)
        rows.extend(sel)
    kmax = max(len(s) for s in rows)
    idx = np.full((len(rows), kmax), -1, dtype=np.int32)
    cnt = np.array([len(s) for s in rows], dtype=np.int32)
    for r, s in enumerate(rows):
        idx[r, :len(s)] = s
    alg, tile = bench.attention_flops(idx, cnt, cu, B, h_q, d)
    ref_alg = ref_tile = 0
    for n, sel in zip(seqlens, sels):
        a, t = _brute_pairs(n, B, sel)
        ref_alg += a
        ref_tile += t
    assert alg == 4 * d * h_q * ref_alg
    assert tile == 4 * d * h_q * ref_tile


def test_measured_traffic_guarded_by_source_hash(monkeypatch):
    for src in bench.MEASURED_TRAFFIC:
        digest, fetch, write = bench.MEASURED_TRAFFIC[src]
        value = bench.measured_traffic(src)
        path = os.path.join(ROOT, "paper_2602_07397_amd", "csrc", src)
        import hashlib
        matches = hashlib.sha256(open(path, "rb").read()).hexdigest() == digest
        if matches:
            assert value == pytest.approx(bench.FETCH_SCALE * fetch + bench.WRITE_SCALE * write)
        else:
            assert value is None
        monkeypatch.setitem(bench.MEASURED_TRAFFIC, src, ("0" * 64, fetch, write))
        assert bench.measured_traffic(src) is None


def test_more_than_one_gpu_is_refused():
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                         capture_output=True, text=True, timeout=120)
    assert res.returncode == 2
    assert "one GPU" in res.stderr or "one GPU" in res.stdout


def test_decode_step_bytes_follow_the_selection_rule():
    """The decode byte count takes tau - 1 whole earlier blocks and the
    current block's tokens up to p (tau from the oracle's budget rule with the
    first and current blocks forced), and the score-cache entries of the lower
    triangle plus the decode-filled columns."""
    import oracle as O
    B, h_q, h_kv, d, r, pct = 64, 32, 8, 128, 64, 20
    for n0, p in ((65536, 65536), (65536, 65600), (65532, 65533), (100, 130)):
        got = bench.decode_step_bytes(p, n0, B, h_q, h_kv, d, r, pct)
        bc = p // B
        tau = O.row_budget(bc + 1, len(O.forced_set(bc, O.FORCE_BOTH)), pct=pct)
        toks = (tau - 1) * B + (p - bc * B + 1)
        assert got["kv"] == toks * h_kv * d * 2 * 2
        col0 = n0 // B
        entries = sum(1 for m in range(bc + 1) for j in range(bc + 1) if j <= m or j >= col0)
        assert got["walk"] == entries * 4
        assert got["sketch"] == 2 * bc * r * 8
