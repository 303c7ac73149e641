"""Seeded random configurations of the one-call decode step (Alg. 2 over
every layer in one sw_decode_step call) against the per-layer calls, which
the same run checks against the oracle: head dims 64 and 128, GQA groups
1-8, blocks of 16-128 tokens, bf16 and fp32, the element-wise and the
clipped power with exponents 1-8, densities 10-50 %, 1-4 sequences whose
prompts (1-2500 tokens) and 20-60 steps put the open block anywhere in a
32-column strip of the score cache."""
import numpy as np
import pytest

import synth
from paper_2602_07397_amd import binding as sw

pytestmark = pytest.mark.gpu

D = pytest.importorskip("test_gpu_decode")
S = pytest.importorskip("test_gpu_decode_step")

N_CASES = 8


@pytest.mark.parametrize("seed", range(N_CASES))
def test_random_decode_step_matches_per_layer_calls_and_oracle(seed):
    rng = np.random.default_rng(3000 + seed)
    d = int(rng.choice([64, 128]))
    h_kv = int(rng.choice([1, 2, 4]))
    G = int(rng.choice([1, 2, 4, 8]))
    B = int(rng.choice([16, 64, 128]))
    dtype = "f32" if seed % 3 == 2 else "bf16"
    variant = sw.WALK_RELU if seed % 2 else sw.WALK_POWER
    s = int(rng.choice([1, 2, 3, 5, 8]))
    pct = int(rng.choice([10, 20, 50]))
    layers = int(rng.integers(2, 4))
    batch = int(rng.integers(1, 5))
    prompts = [int(x) for x in rng.integers(1, 2501, size=batch)]
    steps = int(rng.integers(20, 61))
    w = synth.Workload("dec", 60 + seed, layers=layers, h_q=G * h_kv, h_kv=h_kv, d=d, B=B,
                       dtype=dtype, pct=pct, needles=2, batch=batch, kv_len=max(prompts),
                       steps=steps)
    print(f"seed {seed}: d={d} h_q={G * h_kv} h_kv={h_kv} B={B} {dtype} variant={variant} s={s} "
          f"pct={pct} layers={layers} prompts={prompts} steps={steps}", flush=True)
    run = D.DecodeRun(w, prompts=prompts, steps=steps, variant=variant, s=s)
    S._check_against_per_layer(w, run, dtype, G * h_kv, h_kv, d, variant)
