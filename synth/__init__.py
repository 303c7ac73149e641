"""Seeded synthetic inputs for the sketch-and-walk attention hot path.

This module only draws random tensors and plants structure in them. It holds
none of the method's arithmetic (no pooling, transform, score, walk, selection
or attention step): both the GPU library and the fp64 oracle consume what it
returns, so it is the one piece of code the two sides share.

Workloads (shapes follow the paper's models: Llama-3.1-8B has 32 layers,
32 query / 8 KV heads, head dim 128; Qwen2-7B has 28 / 4 heads):

* ``tiny``     2 layers x 1 head, causal prefill, n=2048, d=64, B=64, fp32.
* ``llama8b``  32 layers, 32/8 heads, d=128, n=32768, B=128, bf16.
* ``stress``   1 layer, 32/8 heads, d=128, n=131072, B=128, bf16.
* ``decode``   batch 16, 65536-token KV cache, 32/8 heads, d=128, B=64,
               bf16, 32 layers, 256 single-token steps.
* ``varlen``   8 sequences, lengths uniform in [8192, 131072] rounded to 128,
               28/4 heads, d=128, B=128, bf16, log-normal key-block scales.

Planted structure (the paper assumes heavy-tailed, block-coherent attention;
these plants emulate it on random data):

* sink: for each KV group g, the keys of block 0 get ``3 * unit(mean query of
  group g)`` added;
* local window (not in ``tiny``): key t gets ``0.5 * (group-mean query at
  t + B)`` added, so block i-1 is salient for query block i;
* needles: a key block j* is overwritten with the group-mean query of one
  later position p plus N(0, 0.1^2) noise;
* ``varlen`` only: every (sequence, group, key block) is scaled by
  exp(0.5 z), z ~ N(0, 1).

Values are drawn in fp32 from N(0, 1) with torch's generator (Philox on the
GPU), planted in fp32, then rounded to the workload dtype. Discrete choices
(needle positions, sequence lengths, the transform's signs and columns) come
from numpy's seeded generator.
"""

from __future__ import annotations

import dataclasses
from typing import List, Optional, Sequence, Tuple

import numpy as np
import torch

BASE_SEED = 20260000


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    index: int            # position in the workload list; seeds derive from it
    layers: int
    h_q: int
    h_kv: int
    d: int
    B: int
    dtype: str            # "f32" or "bf16"
    pct: int              # density in integer percent of causal block pairs
    seqlens: Tuple[int, ...] = ()
    needles: int = 2
    local_window: bool = True
    lognormal_sigma: float = 0.0
    # decode-only fields
    batch: int = 0
    kv_len: int = 0
    steps: int = 0

    @property
    def seed(self) -> int:
        return BASE_SEED + self.index

    @property
    def r(self) -> int:
        """Sketch dimension: 64 (the paper's default), capped at d."""
        return min(64, self.d)

    @property
    def s(self) -> int:
        """Sparsity exponent: 8 (the paper's default)."""
        return 8

    @property
    def torch_dtype(self) -> torch.dtype:
        return torch.float32 if self.dtype == "f32" else torch.bfloat16


def _varlen_lengths(seed: int, count: int, lo: int, hi: int, mult: int) -> Tuple[int, ...]:
    rng = np.random.default_rng(seed + 77)
    raw = rng.integers(lo, hi + 1, size=count)
    out = [int(max(lo, min(hi, mult * int(round(x / mult))))) for x in raw]
    return tuple(out)


WORKLOADS = {
    "tiny": Workload("tiny", 0, layers=2, h_q=1, h_kv=1, d=64, B=64, dtype="f32",
                     pct=20, seqlens=(2048,), needles=2, local_window=False),
    "llama8b": Workload("llama8b", 1, layers=32, h_q=32, h_kv=8, d=128, B=128,
                        dtype="bf16", pct=20, seqlens=(32768,), needles=4),
    "stress": Workload("stress", 2, layers=1, h_q=32, h_kv=8, d=128, B=128,
                       dtype="bf16", pct=20, seqlens=(131072,), needles=4),
    "decode": Workload("decode", 3, layers=32, h_q=32, h_kv=8, d=128, B=64,
                       dtype="bf16", pct=20, needles=4, batch=16, kv_len=65536,
                       steps=256),
    "varlen": Workload("varlen", 4, layers=2, h_q=28, h_kv=4, d=128, B=128,
                       dtype="bf16", pct=20,
                       seqlens=_varlen_lengths(BASE_SEED + 4, 8, 8192, 131072, 128),
                       needles=4, lognormal_sigma=0.5),
}

STRESS_DENSITIES = (10, 20, 40, 100)


def scaled(w: Workload, **changes) -> Workload:
    """A copy of a workload with some fields replaced (smaller test shapes)."""
    return dataclasses.replace(w, **changes)


def srht_params(d: int, r: int, seed: int) -> Tuple[np.ndarray, np.ndarray]:
    """Random signs (int8, +-1) and sampled columns (int32, distinct) of the
    subsampled randomized Hadamard transform. One set serves every layer."""
    rng = np.random.default_rng(seed + 999)
    signs = rng.choice(np.array([-1, 1], dtype=np.int8), size=d).astype(np.int8)
    if r == d:
        cols = rng.permutation(d).astype(np.int32)
    else:
        cols = rng.choice(d, size=r, replace=False).astype(np.int32)
    return signs, cols


def cu_seqlens(seqlens: Sequence[int]) -> np.ndarray:
    out = np.zeros(len(seqlens) + 1, dtype=np.int32)
    out[1:] = np.cumsum(np.asarray(seqlens, dtype=np.int64))
    return out


def _needle_plan(rng: np.random.Generator, n: int, B: int, count: int) -> List[Tuple[int, int]]:
    """(needle key block, query position) pairs with the query after the block."""
    b = -(-n // B)
    plan = []
    if b < 3:
        return plan
    for _ in range(count):
        jstar = int(rng.integers(1, b - 1))
        p = int(rng.integers((jstar + 1) * B, n))
        plan.append((jstar, p))
    return plan


def _layer_seed(w: Workload, layer: int, salt: int = 0) -> int:
    return (w.seed * 1009 + layer * 17 + salt) % (2**62)


def needle_plan(w: Workload, layer: int,
                seqlens: Optional[Sequence[int]] = None) -> List[List[Tuple[int, int]]]:
    """The planted needles of one layer, per sequence: (key block j*, query
    position p) pairs, positions relative to the sequence start. Draws the
    same numbers as prefill_layer_inputs."""
    seqlens = tuple(seqlens if seqlens is not None else w.seqlens)
    rng = np.random.default_rng(_layer_seed(w, layer, 1))
    return [_needle_plan(rng, n, w.B, w.needles) for n in seqlens]


def prefill_layer_inputs(w: Workload, layer: int, device="cpu",
                         seqlens: Optional[Sequence[int]] = None,
                         keep_fp32: bool = False):
    """Q [h_q][N][d], K [h_kv][N][d], V [h_kv][N][d] for one layer.

    Sequences are concatenated along the token axis (N = sum of lengths).
    Returns torch tensors in the workload dtype (fp32 copies as well when
    ``keep_fp32`` is set, for tests that want the pre-rounding values)."""
    seqlens = tuple(seqlens if seqlens is not None else w.seqlens)
    N = int(sum(seqlens))
    dev = torch.device(device)
    gen = torch.Generator(device=dev)
    gen.manual_seed(_layer_seed(w, layer))
    Q = torch.randn((w.h_q, N, w.d), generator=gen, device=dev, dtype=torch.float32)
    K = torch.randn((w.h_kv, N, w.d), generator=gen, device=dev, dtype=torch.float32)
    V = torch.randn((w.h_kv, N, w.d), generator=gen, device=dev, dtype=torch.float32)
    rng = np.random.default_rng(_layer_seed(w, layer, 1))
    G = w.h_q // w.h_kv
    start = 0
    for n in seqlens:
        _plant(w, Q, K, start, n, G, rng, gen)
        start += n
    if keep_fp32:
        return Q.to(w.torch_dtype), K.to(w.torch_dtype), V.to(w.torch_dtype), (Q, K, V)
    return Q.to(w.torch_dtype), K.to(w.torch_dtype), V.to(w.torch_dtype)


def _plant(w: Workload, Q, K, a: int, n: int, G: int, rng, gen) -> None:
    B = w.B
    plan = _needle_plan(rng, n, B, w.needles)
    b = -(-n // B)
    z = None
    if w.lognormal_sigma > 0.0:
        z = torch.randn((w.h_kv, b), generator=gen, device=K.device, dtype=torch.float32)
    for g in range(w.h_kv):
        qg = Q[g * G:(g + 1) * G, a:a + n].mean(dim=0)          # [n][d]
        mu = qg.mean(dim=0)
        nrm = torch.linalg.vector_norm(mu)
        if float(nrm) > 0.0:
            K[g, a:a + min(B, n)] += 3.0 * (mu / nrm)
        if w.local_window and n > B:
            K[g, a:a + n - B] += 0.5 * qg[B:]
        for (jstar, p) in plan:
            lo = a + jstar * B
            hi = min(a + n, lo + B)
            noise = torch.randn((hi - lo, w.d), generator=gen, device=K.device,
                                dtype=torch.float32)
            K[g, lo:hi] = qg[p][None, :] + 0.1 * noise
        if z is not None:
            scale = torch.exp(w.lognormal_sigma * z[g])           # [b]
            tok = torch.repeat_interleave(scale, B)[:n]
            K[g, a:a + n] *= tok[:, None]
        del qg


def topic_layer_inputs(w: Workload, layer: int, device="cpu", topics: int = 16,
                       logit_boost: float = 3.0, drift: float = 0.25):
    """Q, K, V [heads][n][d] of one layer with block-coherent, heavy-tailed
    attention (the structure the paper's analysis assumes), for accuracy
    ablations. Every block of tokens carries a topic; a token's query and key
    are N(0, 1) plus a * u_topic with unit topic vectors u shared by all
    layers and heads and a^2 = logit_boost * sqrt(d), so a query and a key of
    the same topic gain about ``logit_boost`` in q.k / sqrt(d). Block topics
    persist across layers; at each layer a fraction ``drift`` of the blocks
    draws a new topic. One sequence (w.seqlens[0] tokens)."""
    n = int(w.seqlens[0])
    b = -(-n // w.B)
    rng0 = np.random.default_rng(w.seed + 31)
    U = rng0.normal(size=(topics, w.d))
    U /= np.linalg.norm(U, axis=1, keepdims=True)
    z = rng0.integers(0, topics, size=b)
    for ell in range(1, layer + 1):
        rl = np.random.default_rng(_layer_seed(w, ell, 2))
        redraw = rl.uniform(size=b) < drift
        z = np.where(redraw, rl.integers(0, topics, size=b), z)
    a = float(np.sqrt(logit_boost * np.sqrt(w.d)))
    dev = torch.device(device)
    tok = torch.from_numpy(a * U[np.repeat(z, w.B)[:n]]).to(dev, torch.float32)     # [n][d]
    gen = torch.Generator(device=dev)
    gen.manual_seed(_layer_seed(w, layer, 3))
    Q = torch.randn((w.h_q, n, w.d), generator=gen, device=dev, dtype=torch.float32) + tok
    K = torch.randn((w.h_kv, n, w.d), generator=gen, device=dev, dtype=torch.float32) + tok
    V = torch.randn((w.h_kv, n, w.d), generator=gen, device=dev, dtype=torch.float32)
    return Q.to(w.torch_dtype), K.to(w.torch_dtype), V.to(w.torch_dtype)


def decode_prefix_inputs(w: Workload, layer: int, seq: int, device="cpu",
                         kv_len: Optional[int] = None):
    """Prompt Q/K/V of one decode sequence at one layer (planted like prefill).
    Shapes: Q [h_q][T][d], K/V [h_kv][T][d]."""
    T = int(kv_len if kv_len is not None else w.kv_len)
    sub = dataclasses.replace(w, index=w.index * 100 + 7 + seq)
    return prefill_layer_inputs(sub, layer, device=device, seqlens=(T,))


def decode_step_inputs(w: Workload, step: int, layer: int, device="cpu",
                       batch: Optional[int] = None):
    """New-token q [batch][h_q][d], k and v [batch][h_kv][d] for one step of
    one layer, N(0,1) in the workload dtype."""
    bsz = int(batch if batch is not None else w.batch)
    dev = torch.device(device)
    gen = torch.Generator(device=dev)
    gen.manual_seed(_layer_seed(w, layer, 1000 + step))
    q = torch.randn((bsz, w.h_q, w.d), generator=gen, device=dev, dtype=torch.float32)
    k = torch.randn((bsz, w.h_kv, w.d), generator=gen, device=dev, dtype=torch.float32)
    v = torch.randn((bsz, w.h_kv, w.d), generator=gen, device=dev, dtype=torch.float32)
    return q.to(w.torch_dtype), k.to(w.torch_dtype), v.to(w.torch_dtype)


def random_matrix(shape, seed: int, lo: float = -1.0, hi: float = 1.0) -> np.ndarray:
    """Uniform fp64 test matrix (for tests that feed the walk or the
    selection directly)."""
    rng = np.random.default_rng(seed)
    return rng.uniform(lo, hi, size=shape)
