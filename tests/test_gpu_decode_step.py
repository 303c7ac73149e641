"""The one-call decode step (sw_decode_step) against the per-layer calls:
every output of every layer and step bit-identical (the per-layer path is
itself checked against the oracle in the same run), the caches and decode
states bit-identical afterwards, and the clipped-power walk through the same
call."""
import numpy as np
import pytest
import torch

import synth
from paper_2602_07397_amd import binding as sw

pytestmark = pytest.mark.gpu

U = pytest.importorskip("_gpu_util")
D = pytest.importorskip("test_gpu_decode")


def _stacked_inputs(w, k, batch):
    qs, ks, vs = [], [], []
    for l in range(w.layers):
        q, kk, v = synth.decode_step_inputs(w, k, l, batch=batch)
        qs.append(q)
        ks.append(kk)
        vs.append(v)
    return (U.to_dev(torch.stack(qs)), U.to_dev(torch.stack(ks)), U.to_dev(torch.stack(vs)))


@pytest.mark.parametrize("dtype,h_q,h_kv,d,variant", [("bf16", 8, 2, 128, sw.WALK_POWER),
                                                      ("f32", 4, 2, 64, sw.WALK_POWER),
                                                      ("bf16", 8, 1, 64, sw.WALK_RELU)])
def test_decode_step_is_bit_identical_to_per_layer_calls(dtype, h_q, h_kv, d, variant):
    w = synth.Workload("dec", 45, layers=3, h_q=h_q, h_kv=h_kv, d=d, B=64, dtype=dtype, pct=20,
                       needles=2, batch=3, kv_len=1000, steps=70)
    run = D.DecodeRun(w, prompts=[1000, 640, 65], steps=70, variant=variant)
    _check_against_per_layer(w, run, dtype, h_q, h_kv, d, variant)


def test_decode_step_with_decode_columns_across_strips():
    """Blocks of 16 tokens, so that decode fills several columns of the score
    cache: 193..199 inside one 32-column strip (two column quads, the rows
    above the strip), and 62..68 across the boundary of strips 1 and 2; the
    cache has 7 strips (three pairs and a single strip)."""
    w = synth.Workload("dec", 48, layers=2, h_q=4, h_kv=1, d=64, B=16, dtype="bf16", pct=20,
                       needles=2, batch=2, kv_len=3100, steps=100)
    run = D.DecodeRun(w, prompts=[3100, 1000], steps=100)
    _check_against_per_layer(w, run, "bf16", 4, 1, 64, sw.WALK_POWER)


def test_decode_step_with_a_long_cache():
    """2307 blocks of 16 tokens (the selection holds 16 values per thread):
    the open block moves from 2303 to 2304 during the run, so the closed
    decode column 2303 lies in strip 71 and the open one in strip 72, and
    the rows above strip 71 (2272) extend past the 2048 whose loads the walk
    issues ahead."""
    w = synth.Workload("dec", 47, layers=2, h_q=4, h_kv=1, d=64, B=16, dtype="bf16", pct=20,
                       needles=2, batch=1, kv_len=36858, steps=12)
    run = D.DecodeRun(w, prompts=[36858], steps=12, T_extra=42)
    assert run.b_max == 2307
    _check_against_per_layer(w, run, "bf16", 4, 1, 64, sw.WALK_POWER)


def _check_against_per_layer(w, run, dtype, h_q, h_kv, d, variant):
    Kc = torch.stack(run.Kc).contiguous()
    Vc = torch.stack(run.Vc).contiguous()
    state = torch.stack(run.state).contiguous()
    out = None
    ws = torch.empty((sw.load().sw_decode_step_workspace_bytes(run.batch, h_q, h_kv, d),),
                     dtype=torch.uint8, device=U.DEV)
    for k in range(run.steps):
        q, kk, v = _stacked_inputs(w, k, run.batch)
        pos = U.to_dev(np.array([n + k for n in run.prompts], dtype=np.int32))
        out = sw.decode_step(q, kk, v, Kc, Vc, state, pos, run.ts, run.tc, run.B, run.b_max,
                             s=run.s, walk_variant=variant, density_pct=w.pct, kmax=run.kmax,
                             out=out, workspace=ws)
        st = run.step(k)                           # per-layer path, checked against the oracle
        for l, (r, idx, cnt, o) in enumerate(run.last):
            assert torch.equal(out["rows"][l], r), (k, l)
            assert torch.equal(out["cnt"][l], cnt), (k, l)
            assert torch.equal(out["idx"][l], idx), (k, l)
            assert torch.equal(out["O"][l], o), (k, l)
        assert st["werr"] <= 1e-4 and st["err"] <= (U.ATOL_BF16 if dtype == "bf16" else U.ATOL_F32)
    torch.cuda.synchronize()
    for l in range(w.layers):
        assert torch.equal(Kc[l], run.Kc[l])
        assert torch.equal(Vc[l], run.Vc[l])
        assert torch.equal(state[l], run.state[l])


def test_decode_step_rejects_bad_arguments():
    w = synth.Workload("dec", 46, layers=2, h_q=8, h_kv=2, d=128, B=64, dtype="bf16", pct=20,
                       batch=2, kv_len=100, steps=4)
    L, b, T = 2, 2, 128
    q = torch.zeros((L, b, 8, 128), dtype=torch.bfloat16, device=U.DEV)
    kv = torch.zeros((L, b, 2, 128), dtype=torch.bfloat16, device=U.DEV)
    cache = torch.zeros((L, b, 2, T, 128), dtype=torch.bfloat16, device=U.DEV)
    state = torch.zeros((L, sw.decode_state_bytes(b, 128, 64, 2)), dtype=torch.uint8, device=U.DEV)
    pos = U.to_dev(np.array([100, 101], dtype=np.int32))
    signs, cols, ts, tc = U.srht_dev(128, 64, w.seed)
    with pytest.raises(sw.SketchWalkError, match="code 2"):
        sw.decode_step(q, kv, kv, cache, cache.clone(), state, pos, ts, tc, 64, 2,
                       walk_variant=sw.WALK_SOFTMAX)
    with pytest.raises(sw.SketchWalkError, match="T_max"):
        sw.decode_step(q, kv, kv, cache, cache.clone(), state, pos, ts, tc, 64, 1)


def test_inactive_sequence_is_skipped():
    """A sequence whose position is -1 in a step: its state, caches, walk rows
    and selection keep their previous bytes and its attention output is zero;
    the active sequences get exactly the bits of a step without it."""
    w = synth.Workload("dec", 49, layers=2, h_q=8, h_kv=2, d=128, B=64, dtype="bf16", pct=20,
                       needles=2, batch=3, kv_len=500, steps=4)
    runs = [D.DecodeRun(w, prompts=[500, 300, 129], steps=4) for _ in range(2)]
    outs = []
    for which, run in enumerate(runs):
        Kc = torch.stack(run.Kc).contiguous()
        Vc = torch.stack(run.Vc).contiguous()
        state = torch.stack(run.state).contiguous()
        q, kk, v = _stacked_inputs(w, 0, run.batch)
        pos_h = np.array([500, 300, 129], dtype=np.int32)
        if which == 1:
            pos_h[1] = -1
        pos = U.to_dev(pos_h)
        out = {"rows": torch.full((w.layers, 3, run.b_max), 7.0, dtype=torch.float64, device=U.DEV),
               "idx": torch.full((w.layers, 3, run.kmax), 5, dtype=torch.int32, device=U.DEV),
               "cnt": torch.full((w.layers, 3), 5, dtype=torch.int32, device=U.DEV),
               "O": torch.full_like(q, 3.0)}
        state0, K0 = state.clone(), Kc.clone()
        sw.decode_step(q, kk, v, Kc, Vc, state, pos, run.ts, run.tc, run.B, run.b_max, s=w.s,
                       density_pct=w.pct, kmax=run.kmax, out=out)
        torch.cuda.synchronize()
        outs.append((out, state, Kc, state0, K0))
    full, part = outs[0], outs[1]
    for name in ("rows", "idx", "cnt", "O"):
        for b in (0, 2):
            assert torch.equal(full[0][name][:, b], part[0][name][:, b]), name
    assert torch.all(part[0]["rows"][:, 1] == 7.0)
    assert torch.all(part[0]["idx"][:, 1] == 5) and torch.all(part[0]["cnt"][:, 1] == 5)
    assert torch.all(part[0]["O"][:, 1] == 0)
    assert torch.equal(part[2][:, 1], part[4][:, 1])      # cache of the skipped sequence
