"""Benchmark of the Sketch&Walk prefill hot path on one MI355X.

One step = every layer of the Llama-3-8B-shaped workload (32 layers, 32 query
/ 8 KV heads, head dim 128, 32768 tokens, block 128, bf16, density 20%) run
through the full path: sketch scores, walk update, top-tau selection and
block-sparse attention, with inputs already resident in HBM.

Prints one JSON line. ``value`` is the sparse-prefill throughput in TFLOP/s on
the attention FLOPs the selection makes the kernel execute (unmasked query/key
pairs, 4*d flop each), divided by the wall time of the whole step (sketch,
walk and selection included). ``roofline`` describes the attention kernel
alone: its algorithmic FLOPs per launch over its average launch time measured
with HIP events on the launch stream, against the bf16 dense MFMA peak.
``cpu_baseline`` is the fp64 oracle timed on a bounded sample of the same
layer on this host's cores.

The same line carries the decode workload (``decode``: tok/s, the attention
kernel's roofline and the whole step's HBM fraction), the other prefill
workloads (``configs``: the 131072-token layer at 10/20/40/100% and the
variable-length batch) and the sparse/dense ratios at 16K-128K tokens
(``speedup``); ``--no-extras`` leaves out the last two.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0

# HBM bytes per launch from rocprofv3 FETCH_SIZE / WRITE_SIZE passes (KiB per
# dispatch), scaled by the counters' reading for a plain 1 GiB device copy
# (FETCH_SIZE reads 0.5 GiB -> x2.0, WRITE_SIZE reads 1 GiB -> x1.0); see
# profiles/*_traffic.md. Keyed by the sha256 of the kernel source they were
# measured on: a changed source reports null.
FETCH_SCALE, WRITE_SCALE = 2.0, 1.0
MEASURED_TRAFFIC = {
    "attn_prefill.hip": ("2149d18851d90f262dfc6f4961c3e5831781851fa204e37a2fc0bb1999ee0fa0",
                         334347.4 * 1024, 262144.0 * 1024),
    "attn_decode.hip": ("63befefed809dbbb7d18ce6f2ea196fd42b541d037ae887a09056ecb2c0f901d",
                        419749.8 * 1024, 1088.0 * 1024),
}


def measured_traffic(src: str):
    """Scaled HBM bytes per launch for the kernel in csrc/<src>, or None when
    the source changed since the counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "paper_2602_07397_amd", "csrc", src)
    digest, fetch_kib_bytes, write_kib_bytes = MEASURED_TRAFFIC[src]
    with open(path, "rb") as f:
        if hashlib.sha256(f.read()).hexdigest() != digest:
            return None
    return FETCH_SCALE * fetch_kib_bytes + WRITE_SCALE * write_kib_bytes


def attention_flops(idx: np.ndarray, cnt: np.ndarray, cu, B: int, h_q: int, d: int):
    """(unmasked, tile) FLOPs of one layer's sparse attention: 4*d per
    (query, key) pair the selection admits; tile FLOPs count the diagonal
    block in full."""
    alg = 0
    tile = 0
    r = 0
    for a, e in zip(cu[:-1], cu[1:]):
        n = int(e) - int(a)
        b = -(-n // B)
        for i in range(b):
            ci = min(B, n - i * B)
            for j in idx[r, :cnt[r]]:
                cj = min(B, n - int(j) * B)
                alg += ci * (ci + 1) // 2 if j == i else ci * cj
                tile += ci * cj
            r += 1
    return 4 * d * h_q * alg, 4 * d * h_q * tile


def host_cpu_model() -> str:
    """The host CPU's model name (as lscpu reports it)."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def cpu_baseline(Qh, Kh, Vh, cu, B, signs, cols, s, pct, pairs, needle_blocks=(), seed=0):
    """Times the fp64 oracle on one layer: the full selection path (sketch,
    walk, select) plus masked attention on a stratified sample of `pairs`
    (head, query block) pairs: every head of the query blocks that hold a
    planted needle's query, every head of the first and the last block, the
    rest drawn at random; the attention time is scaled to the whole layer by
    the executed FLOPs."""
    import oracle as O
    try:
        from threadpoolctl import threadpool_info
        cores = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    except Exception:  # pragma: no cover
        cores = os.cpu_count() or 1
    t0 = time.perf_counter()
    Q = O.f64(Qh)
    K = O.f64(Kh)
    V = O.f64(Vh)
    t_conv = time.perf_counter() - t0
    t0 = time.perf_counter()
    sk = O.sketch_scores(Q, K, B, signs, cols)
    R = O.walk_step(None, O.walk_weights(sk["A"], sk["c"], s))
    sel, _ = O.select_blocks(R, pct=pct)
    t_sel = time.perf_counter() - t0
    h_q = Q.shape[0]
    b = len(sel)
    rng = np.random.default_rng(seed)
    strata = sorted({int(i) for i in needle_blocks if 0 <= int(i) < b} | {0, b - 1})
    samp = [(u, i) for i in strata for u in range(h_q)]
    n_fixed = len(samp)
    samp += [(int(rng.integers(h_q)), int(rng.integers(b))) for _ in range(max(0, pairs - n_fixed))]
    t0 = time.perf_counter()
    flops_s = 0
    n = Q.shape[1]
    d = Q.shape[2]
    for (u, i) in samp:
        O.sparse_attention_block(Q, K, V, B, sel[i], u, i)
        ci = min(B, n - i * B)
        for j in sel[i]:
            cj = min(B, n - j * B)
            flops_s += 4 * d * (ci * (ci + 1) // 2 if j == i else ci * cj)
    t_attn = time.perf_counter() - t0
    total_pairs = h_q * b
    flops_layer = 0
    for i in range(b):
        ci = min(B, n - i * B)
        for j in sel[i]:
            cj = min(B, n - j * B)
            flops_layer += 4 * d * h_q * (ci * (ci + 1) // 2 if j == i else ci * cj)
    t_layer = t_sel + t_attn * (flops_layer / max(flops_s, 1))
    return {
        "value": flops_layer / t_layer / 1e12,
        "unit": "TFLOP/s",
        "cores": int(cores),
        "cpu_model": host_cpu_model(),
        "kind": "oracle",
        "sample": (f"layer 0 of the workload: full fp64 selection path ({t_sel:.1f} s) + masked "
                   f"attention on {len(samp)} (head, query-block) pairs of {total_pairs}: every "
                   f"head of the needle query blocks and of blocks 0 and b-1 ({n_fixed} pairs), "
                   f"the rest random ({t_attn:.1f} s); attention time scaled by executed FLOPs "
                   f"to the layer; input conversion ({t_conv:.1f} s) excluded"),
        "layer_seconds_extrapolated": t_layer,
    }


def cpu_baseline_decode(budget_s: float = 10.0, layers: int = 4, seed: int = 0) -> dict:
    """Times the fp64 oracle's decode (Alg. 2 steps 2-7: decode_layer_step
    and decode_attention) for one sequence of the decode workload at its full
    shapes, over `layers` layers and as many steps as fit in about
    `budget_s` seconds, and scales it to tokens per second of the whole
    batch. The per-layer state and caches hold seeded random values of the
    workload's shapes (the oracle's work does not depend on the values); the
    caches are built in fp64 once, outside the timed region."""
    import oracle as O
    import synth
    try:
        from threadpoolctl import threadpool_info
        cores = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    except Exception:  # pragma: no cover
        cores = os.cpu_count() or 1
    w = synth.WORKLOADS["decode"]
    B, d, r = w.B, w.d, w.r
    n0 = w.kv_len
    T = n0 + w.steps
    b_max = -(-T // B)
    b0 = -(-n0 // B)
    signs, cols = synth.srht_params(d, r, w.seed)
    rng = np.random.default_rng(seed)
    states = []
    for _ in range(layers):
        A = np.zeros((b_max, b_max))
        A[:b0, :b0] = np.tril(rng.standard_normal((b0, b0)))
        qbar = np.zeros((b_max, d))
        kbar = np.zeros((b_max, d))
        qbar[:b0] = rng.standard_normal((b0, d))
        kbar[:b0] = rng.standard_normal((b0, d))
        last = n0 - (b0 - 1) * B
        qtok = rng.standard_normal((last, d))
        ktok = rng.standard_normal((last, d))
        states.append(O.DecodeLayerState(qbar, kbar, qtok, ktok, A, float(np.abs(A).max())))
    Kc = rng.standard_normal((w.h_kv, T, d))
    Vc = rng.standard_normal((w.h_kv, T, d))
    t0 = time.perf_counter()
    done = 0
    p = n0
    while True:
        r_prev = None
        for st in states:
            q_new = rng.standard_normal((w.h_q, d))
            k_new = rng.standard_normal((w.h_kv, d))
            row, sel, _ = O.decode_layer_step(st, q_new, k_new, p, r_prev, B, signs, cols, w.s,
                                              pct=w.pct)
            O.decode_attention(q_new, Kc, Vc, sel, p, B)
            r_prev = row
            done += 1
        p += 1
        if time.perf_counter() - t0 > budget_s:
            break
    t_layer_step = (time.perf_counter() - t0) / done
    step_s = t_layer_step * w.layers * w.batch          # one step of every sequence and layer
    return {
        "value": w.batch / step_s,
        "unit": "tok/s",
        "cores": int(cores),
        "cpu_model": host_cpu_model(),
        "kind": "oracle",
        "sample": (f"one sequence, {layers} layers x {done // layers} steps of the decode workload's "
                   f"shapes (65536-token caches, b_max {b_max}): {t_layer_step * 1e3:.0f} ms per "
                   f"(sequence, layer) step, scaled to {w.batch} sequences x {w.layers} layers"),
    }


def decode_step_bytes(p: int, n0: int, B: int, h_q: int, h_kv: int, d: int, r: int, pct: int,
                      esz: int = 2) -> dict:
    """Algorithmic HBM bytes of one (sequence, layer) decode step for the
    token at position p of a sequence whose prompt had n0 tokens (density
    pct, forced first and current blocks), by category:
      kv      K and V of the selected tokens: tau - 1 whole blocks plus the
              current block's tokens up to p (the current block is always
              selected, every other selected block precedes it);
      qo      the query and the output of every query head;
      walk    the score-cache entries the walk row reads (fp32): row m holds
              blocks j <= m, and the columns decode filled (col0..b_cur) hold
              every row;
      sketch  the block sketches the score updates read (fp64 Qs and Ks of
              the earlier blocks);
      writes  the appended K/V token and the new score row and column."""
    bc = p // B
    col0 = n0 // B
    tau = min(max((bc + 1) * pct // 100 + (1 if (bc + 1) * pct % 100 else 0), 2), bc + 1)
    toks = (tau - 1) * B + (p - bc * B + 1)
    walk_entries = (bc + 1) * (bc + 2) // 2 + sum(range(col0, bc + 1))
    return {
        "kv": toks * h_kv * d * esz * 2,
        "qo": 2 * h_q * d * esz,
        "walk": walk_entries * 4,
        "sketch": 2 * bc * r * 8,
        "writes": 2 * h_kv * d * esz + (2 * bc + 1) * 4,
    }


def run_decode(args, dev) -> dict:
    """Decode workload: batch 16, 65536-token prompt per sequence, 32 layers,
    256 single-token steps, every layer walked. Returns the decode block of
    the JSON line."""
    import torch
    import synth
    from paper_2602_07397_amd import binding as sw

    w = synth.WORKLOADS["decode"]
    L = args.decode_layers or w.layers
    steps = args.decode_steps
    batch, n0, B = w.batch, w.kv_len, w.B
    T_max = n0 + steps
    b_max = -(-T_max // B)
    signs, cols = synth.srht_params(w.d, w.r, w.seed)
    ts = torch.from_numpy(signs).to(dev)
    tc = torch.from_numpy(cols).to(dev)
    t0 = time.perf_counter()
    # layer-stacked caches and states (per-layer views for the setup and the
    # per-layer launch mode)
    Kst = torch.empty((L, batch, w.h_kv, T_max, w.d), dtype=torch.bfloat16, device=dev)
    Vst = torch.empty_like(Kst)
    Sst = torch.zeros((L, sw.decode_state_bytes(batch, w.d, w.r, b_max)), dtype=torch.uint8,
                      device=dev)
    Kc, Vc, state = list(Kst), list(Vst), list(Sst)
    for l in range(L):
        for b in range(batch):
            Q, K, V = synth.decode_prefix_inputs(w, l, b, device=dev)
            sk = sw.sketch_scores(Q, K, [0, n0], B, ts, tc, want_means=True)
            sw.decode_state_init(state[l], batch, w.d, w.r, b_max, b, n0, B, sk)
            Kc[l][b, :, :n0] = K
            Vc[l][b, :, :n0] = V
            del Q, K, V, sk
    toks = [[synth.decode_step_inputs(w, k, l, device=dev) for l in range(L)] for k in range(steps)]
    torch.cuda.synchronize(dev)
    print(f"[bench] decode setup {time.perf_counter() - t0:.1f} s", file=sys.stderr, flush=True)

    kmax = sw.select_max_count_decode(b_max, density_pct=w.pct)
    pos = torch.full((batch,), n0, dtype=torch.int32, device=dev)
    rbuf = [torch.empty((batch, b_max), dtype=torch.float64, device=dev) for _ in range(2)]
    idx = torch.empty((batch, kmax), dtype=torch.int32, device=dev)
    cnt = torch.empty((batch,), dtype=torch.int32, device=dev)
    obuf = torch.empty((batch, w.h_q, w.d), dtype=torch.bfloat16, device=dev)
    wsa = torch.empty((sw.decode_attn_workspace_bytes(batch, w.h_q, w.h_kv, w.d),), dtype=torch.uint8,
                      device=dev)
    stream = torch.cuda.current_stream(dev)

    # inputs for every step, and the fixed per-step buffers a captured graph reads
    tq = torch.stack([torch.stack([toks[k][l][0] for l in range(L)]) for k in range(steps)])
    tk = torch.stack([torch.stack([toks[k][l][1] for l in range(L)]) for k in range(steps)])
    tv = torch.stack([torch.stack([toks[k][l][2] for l in range(L)]) for k in range(steps)])
    del toks
    bq, bk, bv = torch.empty_like(tq[0]), torch.empty_like(tk[0]), torch.empty_like(tv[0])

    step_out = {"rows": torch.empty((L, batch, b_max), dtype=torch.float64, device=dev),
                "idx": torch.empty((L, batch, kmax), dtype=torch.int32, device=dev),
                "cnt": torch.empty((L, batch), dtype=torch.int32, device=dev),
                "O": torch.empty((L, batch, w.h_q, w.d), dtype=torch.bfloat16, device=dev)}
    wss = torch.empty((sw.load().sw_decode_step_workspace_bytes(batch, w.h_q, w.h_kv, w.d),),
                      dtype=torch.uint8, device=dev)

    def body(sel_log=None):
        nonlocal step_out
        if not args.decode_per_layer:
            step_out = sw.decode_step(bq, bk, bv, Kst, Vst, Sst, pos, ts, tc, B, b_max, s=w.s,
                                      density_pct=w.pct, kmax=kmax, out=step_out, workspace=wss)
            if sel_log is not None:
                for l in range(L):
                    sel_log.append((step_out["idx"][l].clone(), step_out["cnt"][l].clone()))
            pos.add_(1)
            return
        r = None
        for l in range(L):
            sw.kv_append(bk[l], bv[l], Kc[l], Vc[l], pos)
            sw.sketch_scores_decode(bq[l], bk[l], B, pos, ts, tc, b_max, state[l])
            r = sw.walk_update_decode(state[l], batch, w.d, w.r, b_max, B, pos, w.s, r_prev=r,
                                      r_out=rbuf[l & 1])
            sw.select_topk_blocks_decode(r, B, pos, density_pct=w.pct, kmax=kmax, idx=idx, cnt=cnt)
            if sel_log is not None:
                sel_log.append((idx.clone(), cnt.clone()))
            sw.sparse_attn_decode(bq[l], Kc[l], Vc[l], B, pos, idx, cnt, kmax, O=obuf, workspace=wsa)
        pos.add_(1)

    def load_inputs(k):
        bq.copy_(tq[k])
        bk.copy_(tk[k])
        bv.copy_(tv[k])

    graph = None
    if not args.decode_eager:
        torch.cuda.synchronize(dev)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            body()
        torch.cuda.synchronize(dev)

    # timed: steps 0..steps-2, each the whole path for all layers (input copy,
    # KV append, sketch, walk, select, attention)
    torch.cuda.synchronize(dev)
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for k in range(steps - 1):
        load_inputs(k)
        if graph is not None:
            graph.replay()
        else:
            body()
    e1.record(stream)
    torch.cuda.synchronize(dev)
    total_ms = e0.elapsed_time(e1)
    n_timed = steps - 1
    wall_tok_s = batch * n_timed / (total_ms * 1e-3)

    # last step with the selections kept, then the attention launches alone,
    # back to back (the queue stays ahead of the host), for the roofline
    sel_log = []
    load_inputs(steps - 1)
    body(sel_log=sel_log)
    pos.sub_(1)
    torch.cuda.synchronize(dev)
    reps = 3
    a0 = torch.cuda.Event(enable_timing=True)
    a1 = torch.cuda.Event(enable_timing=True)
    a0.record(stream)
    for _ in range(reps):
        for l in range(L):
            sw.sparse_attn_decode(bq[l], Kc[l], Vc[l], B, pos, sel_log[l][0], sel_log[l][1], kmax, O=obuf,
                                  workspace=wsa)
    a1.record(stream)
    torch.cuda.synchronize(dev)
    attn_ms = a0.elapsed_time(a1) / (reps * L)
    p = n0 + steps - 1
    bc = p // B
    kv_bytes = 0
    for (it, ct) in sel_log:
        ih, ch = it.cpu().numpy(), ct.cpu().numpy()
        for b in range(batch):
            toks_sel = 0
            for j in ih[b, :ch[b]]:
                toks_sel += B if j < bc else (p - bc * B + 1)
            kv_bytes += toks_sel * w.h_kv * w.d * 2 * 2
    qo_bytes = 2 * batch * w.h_q * w.d * 2 * L
    attn_bytes = (kv_bytes + qo_bytes) / L
    achieved = attn_bytes / (attn_ms * 1e-3) / 1e9
    step_ms = total_ms / n_timed
    sel_ms = step_ms / L - attn_ms
    # algorithmic bytes of the timed steps (positions n0 .. n0 + n_timed - 1)
    cats = {}
    for k in range(n_timed):
        for key, v in decode_step_bytes(n0 + k, n0, B, w.h_q, w.h_kv, w.d, w.r, w.pct).items():
            cats[key] = cats.get(key, 0) + v * batch * L
    step_bytes = sum(cats.values()) / n_timed
    step_gbs = step_bytes / (step_ms * 1e-3) / 1e9
    return {
        "workload": "decode: batch 16, 65536-token KV cache, 32 q / 8 kv heads, head_dim 128, block 64, "
                    "bf16, 32 layers, 256 steps, density 20%",
        "tok_per_s": round(wall_tok_s, 1),
        "ms_per_step": round(step_ms, 3),
        "timed_steps": n_timed, "layers": L,
        "launch": ("eager" if graph is None else "hip graph of the 32-layer step") + (
            ", per-layer calls" if args.decode_per_layer else ", one sw_decode_step call"),
        "attention_ms_per_layer": round(attn_ms, 4),
        "rest_ms_per_layer": round(sel_ms, 4),
        "overhead_pct": round(100.0 * max(sel_ms, 0.0) / (step_ms / L), 2),
        "hbm_step": {
            "what": "algorithmic bytes of the whole step (selected K/V, q/o, walk-row score-cache "
                    "reads, block-sketch reads, appends and score writes) over the step time",
            "bytes_per_step": round(step_bytes), "achieved": round(step_gbs, 1),
            "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": round(step_gbs / PEAK_HBM_GBS, 4),
            "share": {key: round(v / n_timed / step_bytes, 4) for key, v in cats.items()},
        },
        "roofline": {
            "kernel": "attn_decode_mfma_kernel<128> + attn_merge_kernel",
            "bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
            "frac": round(achieved / PEAK_HBM_GBS, 4), "traffic": measured_traffic("attn_decode.hip"),
            "avg_launch_ms": round(attn_ms, 4), "bytes_per_launch": attn_bytes,
        },
    }


def run_prefill(args, dev):
    """Prefill workload (32 layers of the Llama-3-8B shape). Returns the
    JSON fields and a host copy of layer 0's inputs for the CPU baseline."""
    import torch
    import synth
    from paper_2602_07397_amd import binding as sw

    dev = torch.device("cuda:0")
    w = synth.WORKLOADS["llama8b"]
    L = args.layers or w.layers
    cu = synth.cu_seqlens(w.seqlens)
    B = w.B
    signs, cols = synth.srht_params(w.d, w.r, w.seed)
    ts = torch.from_numpy(signs).to(dev)
    tc = torch.from_numpy(cols).to(dev)

    t0 = time.perf_counter()
    layers = [synth.prefill_layer_inputs(w, l, device=dev) for l in range(L)]
    torch.cuda.synchronize(dev)
    print(f"[bench] generated {L} layers in {time.perf_counter() - t0:.1f} s", file=sys.stderr,
          flush=True)

    nb, nm, _ = sw.layout(cu, B)
    kmax = sw.select_max_count(cu, B, density_pct=w.pct)
    f64 = dict(dtype=torch.float64, device=dev)
    bufs = {
        "Qs": torch.empty((nb, w.r), **f64), "Ks": torch.empty((nb, w.r), **f64),
        "A": torch.empty((nm,), **f64), "A_scale": torch.empty((1,), **f64),
    }
    ws = torch.empty((sw.sketch_workspace_bytes(w.h_q, w.h_kv, w.d, cu, B),), dtype=torch.uint8,
                     device=dev)
    Rbuf = [torch.empty((nm,), **f64), torch.empty((nm,), **f64)]
    idx = [torch.empty((nb, kmax), dtype=torch.int32, device=dev) for _ in range(L)]
    cnt = [torch.empty((nb,), dtype=torch.int32, device=dev) for _ in range(L)]
    Obuf = torch.empty_like(layers[0][0])
    stream = torch.cuda.current_stream(dev)

    def step(events=None):
        R = None
        for l in range(L):
            Q, K, V = layers[l]
            if events is not None:
                events[l][0].record(stream)
            sk = sw.sketch_scores(Q, K, cu, B, ts, tc, out=bufs, workspace=ws)
            if events is not None:
                events[l][1].record(stream)
            Rn = sw.walk_update(sk["A"], sk["A_scale"], w.s, cu, B, R, R_out=Rbuf[l & 1])
            R = Rn
            if events is not None:
                events[l][2].record(stream)
            sw.select_topk_blocks(R, cu, B, density_pct=w.pct, kmax=kmax, idx=idx[l], cnt=cnt[l])
            if events is not None:
                events[l][3].record(stream)
            sw.sparse_attn_prefill(Q, K, V, cu, B, idx[l], cnt[l], kmax, O=Obuf)
            if events is not None:
                events[l][4].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize(dev)
    print("[bench] warmup done", file=sys.stderr, flush=True)

    flops_alg = 0
    flops_tile = 0
    per_layer_alg = []
    for l in range(L):
        a, t = attention_flops(idx[l].cpu().numpy(), cnt[l].cpu().numpy(), cu, B, w.h_q, w.d)
        flops_alg += a
        flops_tile += t
        per_layer_alg.append(a)

    # whole-step wall time
    torch.cuda.synchronize(dev)
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    for _ in range(args.steps):
        step()
    ev1.record(stream)
    torch.cuda.synchronize(dev)
    ms_per_step = ev0.elapsed_time(ev1) / args.steps
    print(f"[bench] timed {args.steps} steps: {ms_per_step:.2f} ms/step", file=sys.stderr, flush=True)

    # per-phase breakdown (separate pass with events between the calls)
    phase = np.zeros(4)
    attn_times = []
    for _ in range(max(1, min(args.steps, 3))):
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(L)]
        step(evs)
        torch.cuda.synchronize(dev)
        for l in range(L):
            for p in range(4):
                phase[p] += evs[l][p].elapsed_time(evs[l][p + 1])
            attn_times.append(evs[l][3].elapsed_time(evs[l][4]))
    phase_frac = phase / phase.sum()
    attn_ms = float(np.mean(attn_times))
    achieved = (flops_alg / L) / (attn_ms * 1e-3) / 1e12

    value = flops_alg / (ms_per_step * 1e-3) / 1e12
    # the sketch reads Q and K once: its algorithmic bytes per layer
    sketch_bytes = (w.h_q + w.h_kv) * int(cu[-1]) * w.d * 2
    sketch_ms = float(phase[0]) / max(1, min(args.steps, 3)) / L
    out = {
        "metric": "sparse prefill TFLOP/s + decode tok/s at 20% density; sketch+select overhead %",
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) with planted sink, local window and needles)",
        "config": {
            "workload": "llama8b-shaped sparse prefill: 32 layers, 32 q / 8 kv heads, head_dim 128, "
                        "seq 32768, block 128, density 20%",
            "layers": L, "h_q": w.h_q, "h_kv": w.h_kv, "head_dim": w.d, "seq_len": w.seqlens[0],
            "block": B, "density_pct": w.pct, "sketch_dim": w.r, "sparsity_exponent": w.s,
            "parallelism": "single GPU",
        },
        "executed_tflop_per_step": flops_alg / 1e12,
        "tile_tflop_per_step": flops_tile / 1e12,
        "overhead_pct": round(100.0 * float(phase_frac[:3].sum()), 3),
        "sketch_hbm": {
            "call": "sw_sketch_scores (Q/K pooling, FWHT, block scores)",
            "bytes_per_layer": sketch_bytes,
            "ms_per_layer": round(sketch_ms, 4),
            "achieved": round(sketch_bytes / (sketch_ms * 1e-3) / 1e9, 1),
            "peak": PEAK_HBM_GBS,
            "unit": "GB/s",
            "frac": round(sketch_bytes / (sketch_ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
        },
        "phase_ms_per_step": {k: round(float(v) / max(1, min(args.steps, 3)), 4)
                              for k, v in zip(("sketch", "walk", "select", "attention"), phase)},
        "roofline": {
            "kernel": "attn_prefill_bf16_kernel<128,128>",
            "bound": "mfma",
            "achieved": round(achieved, 2),
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
            "traffic": measured_traffic("attn_prefill.hip"),
            "avg_launch_ms": round(attn_ms, 4),
            "flop_per_launch": flops_alg / L,
        },
    }
    Q, K, V = layers[0]
    cpu_layer = (Q.cpu(), K.cpu(), V.cpu())
    return out, cpu_layer


def run_configs(args, dev) -> dict:
    """The other prefill workloads, measured like the benchmark's attention
    kernel: the single-layer stress shape at every density of its sweep and
    the varlen batch (2 walked layers). Per layer: the whole path (sketch,
    walk, select, attention) and the attention kernel alone, with the FLOPs
    the selection executes."""
    import torch
    import synth
    from paper_2602_07397_amd import binding as sw

    out = []
    for name in ("stress", "varlen"):
        w = synth.WORKLOADS[name]
        cu = synth.cu_seqlens(w.seqlens)
        B = w.B
        signs, cols = synth.srht_params(w.d, w.r, w.seed)
        ts = torch.from_numpy(signs).to(dev)
        tc = torch.from_numpy(cols).to(dev)
        layers = [synth.prefill_layer_inputs(w, l, device=dev) for l in range(w.layers)]
        pcts = synth.STRESS_DENSITIES if name == "stress" else (w.pct,)
        for pct in pcts:
            kmax = sw.select_max_count(cu, B, density_pct=pct)
            sel = []

            def path(events=None):
                R = None
                sel.clear()
                for l, (Q, K, V) in enumerate(layers):
                    sk = sw.sketch_scores(Q, K, cu, B, ts, tc)
                    R = sw.walk_update(sk["A"], sk["A_scale"], w.s, cu, B, R)
                    idx, cnt, _ = sw.select_topk_blocks(R, cu, B, density_pct=pct, kmax=kmax)
                    if events is not None:
                        events[l][0].record()
                    sw.sparse_attn_prefill(Q, K, V, cu, B, idx, cnt, kmax)
                    if events is not None:
                        events[l][1].record()
                    sel.append((idx, cnt))

            path()
            torch.cuda.synchronize(dev)
            flops = sum(attention_flops(i.cpu().numpy(), c.cpu().numpy(), cu, B, w.h_q, w.d)[0]
                        for i, c in sel)
            # the same passes give both times: events around all of them and
            # around every attention launch inside them
            reps = 3
            evs = [[[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in layers]
                   for _ in range(reps)]
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record()
            for r in range(reps):
                path(evs[r])
            e1.record()
            torch.cuda.synchronize(dev)
            path_ms = e0.elapsed_time(e1) / reps
            attn_ms = sum(a.elapsed_time(b) for er in evs for a, b in er) / reps
            rec = {"workload": name, "layers": len(layers), "density_pct": pct,
                   "tokens": int(cu[-1]), "sequences": len(cu) - 1,
                   "path_ms": round(path_ms, 3), "attention_ms": round(attn_ms, 3),
                   "executed_tflop": round(flops / 1e12, 4),
                   "attention_tflops": round(flops / (attn_ms * 1e-3) / 1e12, 1),
                   "attention_frac_of_peak": round(flops / (attn_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
                   "path_tflops": round(flops / (path_ms * 1e-3) / 1e12, 1),
                   "overhead_pct": round(100.0 * (path_ms - attn_ms) / path_ms, 2)}
            print(f"[bench] configs {rec}", file=sys.stderr, flush=True)
            out.append(rec)
        del layers
        torch.cuda.empty_cache()
    return {"prefill": out,
            "note": "synthetic inputs of each workload's recipe; attention time from HIP events "
                    "around the kernel, path time from events around whole passes"}


def run_speedup(args, dev) -> dict:
    """Sparse vs dense at 16K-128K tokens (one layer of the Llama-3-8B
    shape; the paper reports only such ratios, against FlashAttention).
    Prefill: the whole sparse path (sketch, walk product, select, attention
    at 20%) against dense causal attention, run by this library's kernel
    with every block selected and by torch's flash SDPA when available.
    Decode (batch 16, block 64): one step of the sparse path (KV append,
    sketch, walk row, select, attention) against KV append + dense
    attention over every cached token, both as captured HIP graphs."""
    import torch
    import synth
    from paper_2602_07397_amd import binding as sw

    lengths = [int(x) for x in args.speedup_lengths.split(",")]
    stream = torch.cuda.current_stream(dev)

    def timed(fn, reps):
        fn()
        torch.cuda.synchronize(dev)
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize(dev)
        return e0.elapsed_time(e1) / reps

    pre = []
    base = synth.WORKLOADS["llama8b"]
    for n in lengths:
        w = synth.scaled(base, seqlens=(n,), layers=1)
        cu = synth.cu_seqlens(w.seqlens)
        B = w.B
        signs, cols = synth.srht_params(w.d, w.r, w.seed)
        ts, tc = torch.from_numpy(signs).to(dev), torch.from_numpy(cols).to(dev)
        Q, K, V = synth.prefill_layer_inputs(w, 0, device=dev)
        nb, nm, _ = sw.layout(cu, B)
        f64 = dict(dtype=torch.float64, device=dev)
        bufs = {"Qs": torch.empty((nb, w.r), **f64), "Ks": torch.empty((nb, w.r), **f64),
                "A": torch.empty((nm,), **f64), "A_scale": torch.empty((1,), **f64)}
        ws = torch.empty((sw.sketch_workspace_bytes(w.h_q, w.h_kv, w.d, cu, B),), dtype=torch.uint8,
                         device=dev)
        kmax = sw.select_max_count(cu, B, density_pct=w.pct)
        kd = sw.select_max_count(cu, B, density_pct=100)
        idx = torch.empty((nb, kmax), dtype=torch.int32, device=dev)
        cnt = torch.empty((nb,), dtype=torch.int32, device=dev)
        O = torch.empty_like(Q)
        sk = sw.sketch_scores(Q, K, cu, B, ts, tc, out=bufs, workspace=ws)
        R0 = sw.walk_update(sk["A"], sk["A_scale"], w.s, cu, B, None).clone()
        Rb = torch.empty_like(R0)

        def sparse_path():
            s2 = sw.sketch_scores(Q, K, cu, B, ts, tc, out=bufs, workspace=ws)
            R = sw.walk_update(s2["A"], s2["A_scale"], w.s, cu, B, R0, R_out=Rb)
            sw.select_topk_blocks(R, cu, B, density_pct=w.pct, kmax=kmax, idx=idx, cnt=cnt)
            sw.sparse_attn_prefill(Q, K, V, cu, B, idx, cnt, kmax, O=O)

        reps = max(2, min(10, int(4e5 // n)))
        t_path = timed(sparse_path, reps)
        t_attn = timed(lambda: sw.sparse_attn_prefill(Q, K, V, cu, B, idx, cnt, kmax, O=O), reps)
        idx_d, cnt_d, _ = sw.select_topk_blocks(R0, cu, B, density_pct=100, kmax=kd)
        t_dense = timed(lambda: sw.sparse_attn_prefill(Q, K, V, cu, B, idx_d, cnt_d, kd, O=O), reps)
        t_sdpa = None
        try:
            from torch.nn.attention import SDPBackend, sdpa_kernel
            q4 = Q.unsqueeze(0)
            k4 = K.repeat_interleave(w.h_q // w.h_kv, dim=0).unsqueeze(0)
            v4 = V.repeat_interleave(w.h_q // w.h_kv, dim=0).unsqueeze(0)
            with sdpa_kernel([SDPBackend.FLASH_ATTENTION]):
                t_sdpa = timed(lambda: torch.nn.functional.scaled_dot_product_attention(
                    q4, k4, v4, is_causal=True), reps)
            del q4, k4, v4
        except Exception as e:  # backend not built into this torch
            print(f"[bench] flash SDPA unavailable: {type(e).__name__}: {e}", file=sys.stderr)
        row = {"n": n, "sparse_path_ms": round(t_path, 3), "sparse_attention_ms": round(t_attn, 3),
               "dense_ms_this_kernel": round(t_dense, 3),
               "speedup_vs_dense_this_kernel": round(t_dense / t_path, 2)}
        if t_sdpa is not None:
            row["dense_ms_torch_flash_sdpa"] = round(t_sdpa, 3)
            row["speedup_vs_torch_flash_sdpa"] = round(t_sdpa / t_path, 2)
        pre.append(row)
        print(f"[bench] speedup prefill {row}", file=sys.stderr, flush=True)
        del Q, K, V, O, sk, bufs, ws, idx, cnt, idx_d, cnt_d, R0, Rb
        torch.cuda.empty_cache()

    dec = []
    dbase = synth.WORKLOADS["decode"]
    steps = 32
    for n0 in lengths:
        w = synth.scaled(dbase, kv_len=n0, layers=1)
        batch, B = w.batch, w.B
        T_max = n0 + steps + 1
        b_max = -(-T_max // B)
        signs, cols = synth.srht_params(w.d, w.r, w.seed)
        ts, tc = torch.from_numpy(signs).to(dev), torch.from_numpy(cols).to(dev)
        Kc = torch.empty((batch, w.h_kv, T_max, w.d), dtype=torch.bfloat16, device=dev)
        Vc = torch.empty_like(Kc)
        state = sw.new_decode_state(batch, w.d, w.r, b_max, dev)
        for b in range(batch):
            Qp, Kp, Vp = synth.decode_prefix_inputs(w, 0, b, device=dev)
            skp = sw.sketch_scores(Qp, Kp, [0, n0], B, ts, tc, want_means=True)
            sw.decode_state_init(state, batch, w.d, w.r, b_max, b, n0, B, skp)
            Kc[b, :, :n0] = Kp
            Vc[b, :, :n0] = Vp
            del Qp, Kp, Vp, skp
        q, kn, vn = synth.decode_step_inputs(w, 0, 0, device=dev)
        pos = torch.full((batch,), n0, dtype=torch.int32, device=dev)
        kmax = sw.select_max_count_decode(b_max, density_pct=w.pct)
        idx = torch.empty((batch, kmax), dtype=torch.int32, device=dev)
        cnt = torch.empty((batch,), dtype=torch.int32, device=dev)
        r_prev = torch.ones((batch, b_max), dtype=torch.float64, device=dev)
        r_out = torch.empty_like(r_prev)
        o = torch.empty_like(q)
        wsa = torch.empty((sw.decode_attn_workspace_bytes(batch, w.h_q, w.h_kv, w.d),), dtype=torch.uint8,
                          device=dev)
        bc = (n0 + steps) // B
        idx_d = torch.arange(bc + 1, dtype=torch.int32, device=dev).repeat(batch, 1).contiguous()
        cnt_d = torch.full((batch,), bc + 1, dtype=torch.int32, device=dev)

        def sparse_step():
            sw.kv_append(kn, vn, Kc, Vc, pos)
            sw.sketch_scores_decode(q, kn, B, pos, ts, tc, b_max, state)
            rr = sw.walk_update_decode(state, batch, w.d, w.r, b_max, B, pos, w.s, r_prev=r_prev,
                                       r_out=r_out)
            sw.select_topk_blocks_decode(rr, B, pos, density_pct=w.pct, kmax=kmax, idx=idx, cnt=cnt)
            sw.sparse_attn_decode(q, Kc, Vc, B, pos, idx, cnt, kmax, O=o, workspace=wsa)
            pos.add_(1)

        def dense_step():
            sw.kv_append(kn, vn, Kc, Vc, pos)
            sw.sparse_attn_decode(q, Kc, Vc, B, pos, idx_d, cnt_d, bc + 1, O=o, workspace=wsa)
            pos.add_(1)

        res = {}
        for name, fn in (("sparse", sparse_step), ("dense", dense_step)):
            torch.cuda.synchronize(dev)
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                fn()
            pos.fill_(n0)
            torch.cuda.synchronize(dev)
            res[name] = timed(g.replay, steps)
            pos.fill_(n0)
        row = {"kv_len": n0, "batch": batch, "sparse_step_us": round(res["sparse"] * 1e3, 1),
               "dense_step_us": round(res["dense"] * 1e3, 1),
               "speedup_vs_dense_this_kernel": round(res["dense"] / res["sparse"], 2)}
        dec.append(row)
        print(f"[bench] speedup decode {row}", file=sys.stderr, flush=True)
        del Kc, Vc, state, idx_d
        torch.cuda.empty_cache()
    return {
        "prefill_one_layer": pre,
        "decode_one_layer": dec,
        "note": "per layer of the Llama-3-8B shape (32 q / 8 kv heads, head_dim 128), density 20%; "
                "the paper's ratios (against FlashAttention on an H100, whole model) are context only",
    }


def run_walk_variants(args, dev) -> dict:
    """Walk transition variants at the Llama-3-8B shape (one layer, block
    128) for each prompt length in --speedup-lengths: time of one walk update
    with a previous walk state (the per-layer call after the first layer),
    the fp64 MFMA rate of its block products, and how much of the default
    variant's selection at 20% each variant keeps."""
    import torch
    import synth
    from paper_2602_07397_amd import binding as sw

    names = {sw.WALK_POWER: "power", sw.WALK_RELU: "relu_power", sw.WALK_SOFTMAX: "row_softmax",
             sw.WALK_MATPOW: "matrix_power"}
    stream = torch.cuda.current_stream(dev)
    base = synth.WORKLOADS["llama8b"]
    rows = []
    for n in [int(x) for x in args.speedup_lengths.split(",")]:
        w = synth.scaled(base, seqlens=(n,), layers=2)
        cu = synth.cu_seqlens(w.seqlens)
        B = w.B
        signs, cols = synth.srht_params(w.d, w.r, w.seed)
        ts, tc = torch.from_numpy(signs).to(dev), torch.from_numpy(cols).to(dev)
        sks = []
        for layer in range(2):
            Q, K, _ = synth.prefill_layer_inputs(w, layer, device=dev)
            sks.append(sw.sketch_scores(Q, K, cu, B, ts, tc))
            del Q, K
        b = -(-n // B)
        macs = b * (b + 1) * (b + 2) // 6          # one lower x lower triangular product
        t = math.sqrt(w.r / w.d)
        kmax = sw.select_max_count(cu, B, density_pct=w.pct)
        base_sel = None
        for v in (sw.WALK_POWER, sw.WALK_RELU, sw.WALK_SOFTMAX, sw.WALK_MATPOW):
            R0 = sw.walk_update_variant(v, sks[0]["A"], sks[0]["A_scale"], w.s, cu, B, logit_scale=t)
            R1 = torch.empty_like(R0)
            wsb = sw.walk_workspace_bytes(v, cu, B)
            ws = torch.empty((max(wsb, 256),), dtype=torch.uint8, device=dev)

            def step():
                sw.walk_update_variant(v, sks[1]["A"], sks[1]["A_scale"], w.s, cu, B, R0, R1,
                                       logit_scale=t, workspace=ws)

            step()
            torch.cuda.synchronize(dev)
            reps = 50
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(reps):
                step()
            e1.record(stream)
            torch.cuda.synchronize(dev)
            ms = e0.elapsed_time(e1) / reps
            if v == sw.WALK_MATPOW:
                top = w.s.bit_length() - 1
                nprod = sum(1 + ((w.s >> bit) & 1) for bit in range(top - 1, -1, -1)) + 1
            else:
                nprod = 1
            idx, cnt, _ = sw.select_topk_blocks(R1, cu, B, density_pct=w.pct, kmax=kmax)
            sel = [set(r[:c].tolist()) for r, c in zip(idx.cpu().numpy(), cnt.cpu().numpy())]
            if base_sel is None:
                base_sel = sel
            kept = sum(len(a & b_) for a, b_ in zip(sel, base_sel)) / sum(len(a) for a in base_sel)
            rows.append({"n": n, "blocks": b, "variant": names[v], "ms": round(ms, 4),
                         "block_products": nprod,
                         "fp64_tflops": round(2.0 * macs * nprod / (ms * 1e-3) / 1e12, 2),
                         "kept_of_power_selection": round(kept, 4)})
            print(f"[bench] walk {names[v]} n={n}: {ms:.4f} ms", file=sys.stderr, flush=True)
        del sks
        torch.cuda.empty_cache()
    return {"rows": rows, "s": base.s, "density_pct": base.pct, "block": base.B,
            "fp64_mfma_peak_tflops": 78.6,
            "note": "one walk update with a previous state (second layer); the softmax variant "
                    "uses logit scale sqrt(r/d)"}


def block_attention_mass(Q, K, B: int, chunk: int = 2048):
    """Dense causal attention mass between blocks of one sequence, averaged
    over the query heads and over the query tokens of each block:
    M[i][j] = mean over heads u and tokens t of query block i of the softmax
    probability (scale 1/sqrt(d), keys k <= t) that falls in key block j.
    Rows sum to 1. Q [h_q][n][d], K [h_kv][n][d]; fp32 arithmetic, fp64 sums.
    Ground truth for the ablation's mass recall (an evaluation, not a step of
    the method)."""
    import torch
    h_q, n, d = Q.shape
    G = h_q // K.shape[0]
    b = -(-n // B)
    dev = Q.device
    M = torch.zeros((b, b), dtype=torch.float64, device=dev)
    chunk = max(B, chunk // B * B)
    for u in range(h_q):
        Kg = K[u // G].float()
        for c0 in range(0, n, chunk):
            c1 = min(n, c0 + chunk)
            sc = (Q[u, c0:c1].float() @ Kg[:c1].T) * (1.0 / math.sqrt(d))
            tq = torch.arange(c0, c1, device=dev).unsqueeze(1)
            tk = torch.arange(c1, device=dev).unsqueeze(0)
            sc.masked_fill_(tk > tq, float("-inf"))
            pr = torch.softmax(sc, dim=1)
            nkb = -(-c1 // B)
            pr = torch.nn.functional.pad(pr, (0, nkb * B - c1)).view(c1 - c0, nkb, B).sum(-1)
            qb = torch.arange(c0, c1, device=dev) // B
            M[:, :nkb].index_add_(0, qb, pr.double())
    cnt = torch.full((b,), float(B), dtype=torch.float64, device=dev)
    cnt[-1] = n - (b - 1) * B
    return M / (cnt[:, None] * h_q)


def selection_mask(idx, cnt, b: int):
    """[b][b] bool: row i marks the key blocks selected for query block i."""
    import torch
    k = idx.shape[1]
    valid = torch.arange(k, device=idx.device)[None, :] < cnt[:, None].long()
    mask = torch.zeros((b, b + 1), dtype=torch.bool, device=idx.device)
    cols = torch.where(valid, idx.long(), torch.full_like(idx.long(), b))
    mask.scatter_(1, cols, True)
    return mask[:, :b]


def best_mask(M, pct: int):
    """Per query block, the forced blocks {0, i} plus the key blocks of
    largest true mass up to the same budget tau_i = ceil((i + 1) pct / 100):
    the most attention mass any block selection of that size can cover."""
    import torch
    b = M.shape[0]
    Mh = M.cpu().numpy()
    mask = np.zeros((b, b), dtype=bool)
    for i in range(b):
        forced = {0, i}
        tau = min(max(((i + 1) * pct + 99) // 100, len(forced)), i + 1)
        rest = sorted((j for j in range(i + 1) if j not in forced), key=lambda j: (-Mh[i, j], j))
        for j in list(forced) + rest[:tau - len(forced)]:
            mask[i, j] = True
    return torch.from_numpy(mask).to(M.device)


def run_ablation(args, dev, record=None) -> dict:
    """Recall of the block selection on synthetic data, one factor
    at a time around the default (r = 64, s = 8, 20 %, walk across layers,
    element-wise power): the sketch dimension r, the exponent s, the density,
    the cross-layer walk (off = each layer ranks its own W; "walk_layers" k =
    the walk restarts every k layers, so it accumulates at most k layers),
    and the walk transition. Two measures per configuration, averaged over
    layers:
    mass recall = the share of the dense attention mass (all query heads)
    that the selected blocks hold; needle recall = the share of planted
    needle blocks selected for the query block that holds the needle's
    query. "best" rows select by the true mass itself (an upper bound at
    each density). The default configuration's recall is also reported per
    layer (after 1, 2, ... walked layers). ``record``, if a dict, receives
    every configuration's selection per layer: record[(axis, value, layer)]
    = (idx, cnt) on the host."""
    import torch
    import synth
    from paper_2602_07397_amd import binding as sw

    w = synth.scaled(synth.WORKLOADS["llama8b"], seqlens=(args.ablation_tokens,),
                     layers=args.ablation_layers, needles=args.ablation_needles)
    n, B, d = w.seqlens[0], w.B, w.d
    b = -(-n // B)
    cu = synth.cu_seqlens(w.seqlens)
    base = dict(r=64, s=8, pct=20, walk=True, window=0, variant=sw.WALK_POWER)
    names = {sw.WALK_POWER: "power", sw.WALK_RELU: "relu_power", sw.WALK_SOFTMAX: "row_softmax",
             sw.WALK_MATPOW: "matrix_power"}
    configs = [("default", "-", dict(base))]
    for r in (16, 32, 128):
        configs.append(("r", r, dict(base, r=r)))
    for s_ in (1, 2, 4, 16):
        configs.append(("s", s_, dict(base, s=s_)))
    for pct in (10, 30, 50, 100):
        configs.append(("pct", pct, dict(base, pct=pct)))
    configs.append(("walk", "off", dict(base, walk=False)))
    for k in (2, 4):
        if k < w.layers:
            configs.append(("walk_layers", k, dict(base, window=k)))
    for v in (sw.WALK_RELU, sw.WALK_SOFTMAX, sw.WALK_MATPOW):
        configs.append(("variant", names[v], dict(base, variant=v)))
    rs = sorted({c["r"] for _, _, c in configs})
    srht = {}
    for r in rs:
        sg, cl = synth.srht_params(d, r, w.seed)
        srht[r] = (torch.from_numpy(sg).to(dev), torch.from_numpy(cl).to(dev))
    state = [None] * len(configs)
    acc = [dict(mass=0.0, needle_hits=0, needles=0, density=0.0) for _ in configs]
    best = {p: dict(mass=0.0, needle_hits=0, needles=0) for p in sorted({c["pct"] for _, _, c in configs})}
    causal_pairs = b * (b + 1) / 2
    depth = []                       # the default configuration's recall per layer
    t0 = time.perf_counter()
    for layer in range(w.layers):
        if args.ablation_data == "topics":
            Q, K, _ = synth.topic_layer_inputs(w, layer, device=dev, drift=args.ablation_drift)
            plan = []
        else:
            Q, K, _ = synth.prefill_layer_inputs(w, layer, device=dev)
            # a later needle in the same key block overwrites an earlier one
            plan = sorted({jstar: p for jstar, p in synth.needle_plan(w, layer)[0]}.items())
        M = block_attention_mass(Q, K, B)
        best_masks = {pct: best_mask(M, pct) for pct in best}
        sks = {r: sw.sketch_scores(Q, K, cu, B, *srht[r]) for r in rs}
        del Q, K
        for ci, (_, _, c) in enumerate(configs):
            sk = sks[c["r"]]
            restart = (not c["walk"]) or (c["window"] > 0 and layer % c["window"] == 0)
            R = sw.walk_update_variant(c["variant"], sk["A"], sk["A_scale"], c["s"], cu, B,
                                       None if restart else state[ci],
                                       logit_scale=math.sqrt(c["r"] / d))
            state[ci] = R
            idx, cnt, _ = sw.select_topk_blocks(R, cu, B, density_pct=c["pct"])
            if record is not None:
                record[(configs[ci][0], configs[ci][1], layer)] = (idx.cpu(), cnt.cpu())
            mask = selection_mask(idx, cnt, b)
            a = acc[ci]
            m_layer = float((M * mask).sum(dim=1).mean())
            a["mass"] += m_layer
            if ci == 0:
                depth.append(round(m_layer, 4))
            a["density"] += float(cnt.sum()) / causal_pairs
            a["best_overlap"] = a.get("best_overlap", 0.0) + float(
                (mask & best_masks[c["pct"]]).sum()) / float(best_masks[c["pct"]].sum())
            mh = mask.cpu().numpy()
            for (jstar, p) in plan:
                a["needles"] += 1
                a["needle_hits"] += int(mh[p // B, jstar])
        for pct, bacc in best.items():
            bm = best_masks[pct]
            bacc["mass"] += float((M * bm).sum(dim=1).mean())
            bmh = bm.cpu().numpy()
            for (jstar, p) in plan:
                bacc["needles"] += 1
                bacc["needle_hits"] += int(bmh[p // B, jstar])
        print(f"[bench] ablation layer {layer} done ({time.perf_counter() - t0:.1f} s)",
              file=sys.stderr, flush=True)
    L = w.layers
    rows = []
    for (axis, value, c), a in zip(configs, acc):
        rows.append({"axis": axis, "value": value, "r": c["r"], "s": c["s"], "pct": c["pct"],
                     "walk": c["walk"], "walk_layers": c["window"] or (L if c["walk"] else 1),
                     "variant": names[c["variant"]],
                     "mass_recall": round(a["mass"] / L, 4),
                     "best_overlap": round(a["best_overlap"] / L, 4),
                     "needle_recall": (round(a["needle_hits"] / a["needles"], 4)
                                       if a["needles"] else None),
                     "selected_fraction": round(a["density"] / L, 4)})
    for pct, bacc in best.items():
        rows.append({"axis": "best", "value": pct, "pct": pct,
                     "mass_recall": round(bacc["mass"] / L, 4),
                     "needle_recall": (round(bacc["needle_hits"] / bacc["needles"], 4)
                                       if bacc["needles"] else None)})
    return {"rows": rows,
            "default_recall_per_layer": depth,
            "workload": {"tokens": n, "layers": L, "h_q": w.h_q, "h_kv": w.h_kv, "d": d, "B": B,
                         "data": args.ablation_data, "dtype": w.dtype,
                         "topic_drift": args.ablation_drift if args.ablation_data == "topics" else None,
                         "needles_per_layer": w.needles if args.ablation_data == "planted" else 0},
            "note": "synthetic data; recall is measured against the dense attention of the same "
                    "inputs; best_overlap = share of the best-by-mass selection's blocks kept"}


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--layers", type=int, default=None, help="override layer count (debug only)")
    ap.add_argument("--cpu-pairs", type=int, default=3000)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-decode", action="store_true")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the stress/varlen workloads and the sparse/dense ratios")
    ap.add_argument("--decode-steps", type=int, default=256)
    ap.add_argument("--decode-layers", type=int, default=None, help="override (debug only)")
    ap.add_argument("--decode-eager", action="store_true", help="launch the decode step eagerly")
    ap.add_argument("--decode-per-layer", action="store_true",
                    help="run the decode step as per-layer calls instead of one sw_decode_step")
    ap.add_argument("--configs", action="store_true",
                    help="instead of the benchmark line, measure the stress density sweep and "
                         "the varlen batch")
    ap.add_argument("--speedup", action="store_true",
                    help="instead of the benchmark line, print sparse-vs-dense ratios at several lengths")
    ap.add_argument("--speedup-lengths", default="16384,32768,65536,131072")
    ap.add_argument("--ablation", action="store_true",
                    help="instead of the benchmark line, print selection recall on planted "
                         "synthetic data against r, s, density, walk on/off and transition")
    ap.add_argument("--ablation-tokens", type=int, default=16384)
    ap.add_argument("--ablation-layers", type=int, default=8)
    ap.add_argument("--ablation-needles", type=int, default=16)
    ap.add_argument("--ablation-drift", type=float, default=0.0,
                    help="topic data: share of blocks that change topic at each layer")
    ap.add_argument("--ablation-data", choices=("topics", "planted"), default="topics",
                    help="block-topic data with heavy-tailed attention, or the benchmark's "
                         "planted sink / local window / needles")
    ap.add_argument("--walk-variants", action="store_true",
                    help="instead of the benchmark line, time the walk transition variants at the "
                         "--speedup-lengths")
    ap.add_argument("--only", choices=("prefill", "decode", "copy"), default=None,
                    help="run one workload only (profiling); 'copy' runs the plain 1 GiB device "
                         "copy used to calibrate the FETCH_SIZE / WRITE_SIZE counters")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU; --gpus must be 1"}))
        print("bench.py: only --gpus 1 is supported (one GPU per run)", file=sys.stderr)
        return 2

    import torch
    dev = torch.device("cuda:0")
    if args.only == "copy":
        src = torch.empty((1 << 30,), dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize(dev)
        print(json.dumps({"copy_bytes": 1 << 30, "copies": 5}), flush=True)
        return 0
    if args.speedup:
        print(json.dumps({"speedup": run_speedup(args, dev)}), flush=True)
        return 0
    if args.configs:
        print(json.dumps({"configs": run_configs(args, dev)}), flush=True)
        return 0
    if args.ablation:
        print(json.dumps({"ablation": run_ablation(args, dev)}), flush=True)
        return 0
    if args.walk_variants:
        print(json.dumps({"walk_variants": run_walk_variants(args, dev)}), flush=True)
        return 0
    out = {}
    cpu_layer = None
    if args.only != "decode":
        out, cpu_layer = run_prefill(args, dev)
        torch.cuda.empty_cache()
    if args.only != "prefill" and not args.no_decode:
        out["decode"] = run_decode(args, dev)
        torch.cuda.empty_cache()
    if args.only is None and not args.no_extras:
        # the other workloads and the sparse/dense ratios, measured in the same run
        out["configs"] = run_configs(args, dev)["prefill"]
        torch.cuda.empty_cache()
        out["speedup"] = run_speedup(args, dev)
        torch.cuda.empty_cache()
    if "decode" in out and args.only != "decode" and not args.no_cpu_baseline:
        print("[bench] timing the oracle's decode on the host", file=sys.stderr, flush=True)
        out["decode"]["cpu_baseline"] = cpu_baseline_decode()
    if cpu_layer is not None and not args.no_cpu_baseline:
        import synth
        w = synth.WORKLOADS["llama8b"]
        signs, cols = synth.srht_params(w.d, w.r, w.seed)
        print("[bench] timing the oracle on the host", file=sys.stderr, flush=True)
        needles = [p // w.B for (_, p) in synth.needle_plan(w, 0)[0]]
        out["cpu_baseline"] = cpu_baseline(*cpu_layer, synth.cu_seqlens(w.seqlens), w.B, signs, cols,
                                           w.s, w.pct, args.cpu_pairs, needle_blocks=needles)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
