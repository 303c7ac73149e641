"""GPU parity of the decode path (Alg. 2) against the fp64 oracle, through
the C ABI: prefill-to-decode state hand-off, KV append, incremental sketch,
walk row, row selection and split-K decode attention."""
import math

import numpy as np
import pytest
import torch

import oracle as O
import synth
from paper_2602_07397_amd import binding as sw

pytestmark = pytest.mark.gpu

U = pytest.importorskip("_gpu_util")


class DecodeRun:
    """Runs the same decode on the GPU (through the C ABI) and on the oracle."""

    def __init__(self, w, prompts, steps, T_extra=0, variant=sw.WALK_POWER, s=None):
        self.w = w
        self.variant = variant
        self.s = w.s if s is None else s
        self.B = w.B
        self.d = w.d
        self.r = w.r
        self.batch = len(prompts)
        self.prompts = list(prompts)
        self.steps = steps
        self.T_max = max(prompts) + steps + T_extra
        self.b_max = -(-self.T_max // self.B)
        self.signs, self.cols, self.ts, self.tc = U.srht_dev(w.d, w.r, w.seed)
        L, H, Hk = w.layers, w.h_q, w.h_kv
        dt = w.torch_dtype
        self.Kc = [torch.zeros((self.batch, Hk, self.T_max, w.d), dtype=dt, device=U.DEV) for _ in range(L)]
        self.Vc = [torch.zeros_like(self.Kc[0]) for _ in range(L)]
        self.state = [sw.new_decode_state(self.batch, w.d, w.r, self.b_max, U.DEV) for _ in range(L)]
        self.Kh = [[None] * self.batch for _ in range(L)]   # host fp64 caches for the oracle
        self.Vh = [[None] * self.batch for _ in range(L)]
        self.ost = [[None] * self.batch for _ in range(L)]
        for l in range(L):
            for b, n in enumerate(prompts):
                Q, K, V = synth.decode_prefix_inputs(w, l, b, kv_len=n)
                Qd, Kd = U.to_dev(Q), U.to_dev(K)
                sk = sw.sketch_scores(Qd, Kd, [0, n], self.B, self.ts, self.tc, want_means=True)
                sw.decode_state_init(self.state[l], self.batch, w.d, w.r, self.b_max, b, n, self.B, sk)
                self.Kc[l][b, :, :n] = Kd
                self.Vc[l][b, :, :n] = U.to_dev(V)
                Kf = np.zeros((Hk, self.T_max, w.d))
                Vf = np.zeros((Hk, self.T_max, w.d))
                Kf[:, :n] = O.f64(K)
                Vf[:, :n] = O.f64(V)
                self.Kh[l][b] = Kf
                self.Vh[l][b] = Vf
                self.ost[l][b] = O.decode_state_from_prefill(Q, K, self.B, self.signs, self.cols, self.b_max)
        self.kmax = sw.select_max_count_decode(self.b_max, density_pct=w.pct)
        torch.cuda.synchronize()

    def step(self, k, check=True):
        w = self.w
        pos_h = np.array([n + k for n in self.prompts], dtype=np.int32)
        pos = U.to_dev(pos_h)
        r_gpu = None
        r_ref = [None] * self.batch
        stats = dict(near=0, rows=0, err=0.0, werr=0.0)
        self.last = []                     # per layer: walk row, idx, cnt, O of this step
        for l in range(w.layers):
            q, kk, v = synth.decode_step_inputs(w, k, l, batch=self.batch)
            qd, kd, vd = U.to_dev(q), U.to_dev(kk), U.to_dev(v)
            sw.kv_append(kd, vd, self.Kc[l], self.Vc[l], pos)
            sw.sketch_scores_decode(qd, kd, self.B, pos, self.ts, self.tc, self.b_max, self.state[l])
            if self.variant == sw.WALK_POWER:
                r_gpu = sw.walk_update_decode(self.state[l], self.batch, w.d, w.r, self.b_max, self.B,
                                              pos, self.s, r_prev=r_gpu)
            else:
                r_gpu = sw.walk_update_decode_variant(self.variant, self.state[l], self.batch, w.d,
                                                      w.r, self.b_max, self.B, pos, self.s,
                                                      r_prev=r_gpu)
            idx, cnt, _ = sw.select_topk_blocks_decode(r_gpu, self.B, pos, density_pct=w.pct,
                                                       kmax=self.kmax)
            out = sw.sparse_attn_decode(qd, self.Kc[l], self.Vc[l], self.B, pos, idx, cnt, self.kmax)
            self.last.append((r_gpu.clone(), idx, cnt, out))
            if not check:
                continue
            rg = r_gpu.cpu().numpy()
            got = U.gpu_selection(idx, cnt)
            og = out.float().cpu().numpy()
            qh, kh, vh = O.f64(q), O.f64(kk), O.f64(v)
            for b in range(self.batch):
                p = int(pos_h[b])
                bc = p // self.B
                self.Kh[l][b][:, p] = kh[b]
                self.Vh[l][b][:, p] = vh[b]
                row, sel, gap = O.decode_layer_step(self.ost[l][b], qh[b], kh[b], p, r_ref[b], self.B,
                                                    self.signs, self.cols, self.s, pct=w.pct,
                                                    variant=self.variant)
                r_ref[b] = row
                stats["werr"] = max(stats["werr"], U.max_abs(rg[b, :bc + 1], row))
                assert np.all(rg[b, bc + 1:] == 0.0)
                stats["rows"] += 1
                if gap > U.GAP_TOL:
                    assert got[b] == sel, (k, l, b, got[b], sel)
                else:
                    stats["near"] += 1
                    assert len(got[b]) == len(sel) and {0, bc} <= set(got[b])
                ref = O.decode_attention(qh[b], self.Kh[l][b], self.Vh[l][b], got[b], p, self.B)
                stats["err"] = max(stats["err"], U.max_abs(og[b], ref))
        return stats


def _small(dtype="bf16", h_q=8, h_kv=2, d=128, B=64, layers=3):
    return synth.Workload("dec", 45, layers=layers, h_q=h_q, h_kv=h_kv, d=d, B=B, dtype=dtype,
                          pct=20, needles=2, batch=3, kv_len=1000, steps=150)


@pytest.mark.parametrize("dtype,h_q,h_kv,d", [("bf16", 8, 2, 128), ("f32", 4, 2, 64),
                                               ("bf16", 8, 1, 64), ("bf16", 4, 4, 128)])
def test_decode_matches_oracle(dtype, h_q, h_kv, d):
    w = _small(dtype, h_q, h_kv, d)
    run = DecodeRun(w, prompts=[1000, 640, 65], steps=140)
    tol = U.ATOL_BF16 if dtype == "bf16" else U.ATOL_F32
    worst = dict(err=0.0, werr=0.0, near=0, rows=0)
    for k in range(run.steps):
        st = run.step(k)
        worst["err"] = max(worst["err"], st["err"])
        worst["werr"] = max(worst["werr"], st["werr"])
        worst["near"] += st["near"]
        worst["rows"] += st["rows"]
    # walk rows: fp32 score cache, fp64 arithmetic
    assert worst["werr"] <= 1e-4, worst
    assert worst["err"] <= tol, worst
    assert worst["near"] <= 0.05 * worst["rows"], worst
    # the caches hold exactly what was appended
    for l in range(w.layers):
        for b in range(run.batch):
            n_end = run.prompts[b] + run.steps
            got = run.Kc[l][b, :, :n_end].double().cpu().numpy()
            np.testing.assert_array_equal(got, run.Kh[l][b][:, :n_end])


def test_decode_state_round_trip_is_bit_identical():
    w = _small(layers=2)
    a = DecodeRun(w, prompts=[300, 128], steps=80)
    for k in range(40):
        a.step(k, check=False)
    saved = [s.clone() for s in a.state]
    savedK = [x.clone() for x in a.Kc]
    savedV = [x.clone() for x in a.Vc]
    outs = []
    for rep in range(2):
        for l in range(w.layers):
            a.state[l].copy_(saved[l])
            a.Kc[l].copy_(savedK[l])
            a.Vc[l].copy_(savedV[l])
        for k in range(40, 80):
            a.step(k, check=False)
        outs.append([s.clone() for s in a.state])
    for x, y in zip(*outs):
        assert torch.equal(x, y)


def test_first_layer_walk_row_is_power_of_score_row():
    """Alg. 2 step 5 at the first walked layer: the row is W[b_q, :]."""
    w = _small(layers=1)
    run = DecodeRun(w, prompts=[200], steps=3)
    pos = U.to_dev(np.array([200], dtype=np.int32))
    q, k, v = synth.decode_step_inputs(w, 0, 0, batch=1)
    sw.sketch_scores_decode(U.to_dev(q), U.to_dev(k), w.B, pos, run.ts, run.tc, run.b_max, run.state[0])
    r = sw.walk_update_decode(run.state[0], 1, w.d, w.r, run.b_max, w.B, pos, w.s)
    row, _, _ = O.decode_layer_step(run.ost[0][0], q[0], k[0], 200, None, w.B, run.signs, run.cols,
                                    w.s, pct=w.pct)
    assert U.max_abs(r.cpu().numpy()[0, :200 // w.B + 1], row) <= 1e-5


def _fixed_step_fn(run, bufs, outs):
    """One decode step over all layers reading fixed input buffers and writing
    per-layer outputs (so that it can be captured in a graph)."""
    w = run.w
    bq, bk, bv, pos = bufs

    def body():
        r = None
        for l in range(w.layers):
            sw.kv_append(bk[l], bv[l], run.Kc[l], run.Vc[l], pos)
            sw.sketch_scores_decode(bq[l], bk[l], run.B, pos, run.ts, run.tc, run.b_max, run.state[l])
            r = sw.walk_update_decode(run.state[l], run.batch, w.d, w.r, run.b_max, run.B, pos, w.s,
                                      r_prev=r, r_out=outs["r"][l])
            sw.select_topk_blocks_decode(r, run.B, pos, density_pct=w.pct, kmax=run.kmax,
                                         idx=outs["idx"][l], cnt=outs["cnt"][l])
            sw.sparse_attn_decode(bq[l], run.Kc[l], run.Vc[l], run.B, pos, outs["idx"][l],
                                  outs["cnt"][l], run.kmax, O=outs["O"][l], workspace=outs["wsa"])
        pos.add_(1)
    return body


def test_decode_graph_replay_matches_eager():
    """A decode step captured in a HIP graph and replayed several times (with
    eager work and synchronisation between replays) gives, at every replay,
    the bits of the same step launched eagerly."""
    w = _small(layers=3)
    prompts = [300, 128, 75]
    steps = 6
    runs = [DecodeRun(w, prompts=prompts, steps=steps) for _ in range(2)]
    inputs = [[synth.decode_step_inputs(w, k, l, batch=len(prompts)) for l in range(w.layers)]
              for k in range(steps)]
    results = []
    for mode, run in zip(("eager", "graph"), runs):
        bq = torch.stack([U.to_dev(inputs[0][l][0]) for l in range(w.layers)])
        bk = torch.stack([U.to_dev(inputs[0][l][1]) for l in range(w.layers)])
        bv = torch.stack([U.to_dev(inputs[0][l][2]) for l in range(w.layers)])
        pos = U.to_dev(np.array(prompts, dtype=np.int32))
        outs = {
            "r": [torch.empty((run.batch, run.b_max), dtype=torch.float64, device=U.DEV) for _ in range(w.layers)],
            "idx": [torch.empty((run.batch, run.kmax), dtype=torch.int32, device=U.DEV) for _ in range(w.layers)],
            "cnt": [torch.empty((run.batch,), dtype=torch.int32, device=U.DEV) for _ in range(w.layers)],
            "O": [torch.empty((run.batch, w.h_q, w.d), dtype=torch.bfloat16, device=U.DEV) for _ in range(w.layers)],
            "wsa": torch.empty((sw.decode_attn_workspace_bytes(run.batch, w.h_q, w.h_kv, w.d),),
                               dtype=torch.uint8, device=U.DEV),
        }
        body = _fixed_step_fn(run, (bq, bk, bv, pos), outs)
        graph = None
        if mode == "graph":
            torch.cuda.synchronize()
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph):
                body()
            torch.cuda.synchronize()
        per_step = []
        for k in range(steps):
            for l in range(w.layers):
                bq[l].copy_(U.to_dev(inputs[k][l][0]))
                bk[l].copy_(U.to_dev(inputs[k][l][1]))
                bv[l].copy_(U.to_dev(inputs[k][l][2]))
            if graph is not None:
                graph.replay()
            else:
                body()
            torch.cuda.synchronize()
            _ = (torch.ones(8, device=U.DEV) * 2).sum().item()   # eager work between replays
            per_step.append({key: [t.clone() for t in outs[key]] for key in ("r", "idx", "cnt", "O")})
        results.append(per_step)
    for k in range(steps):
        for key in ("r", "idx", "cnt", "O"):
            for l in range(w.layers):
                assert torch.equal(results[0][k][key][l], results[1][k][key][l]), (k, key, l)
