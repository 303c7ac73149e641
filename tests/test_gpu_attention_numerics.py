"""Numerical edge cases of the block-sparse prefill attention against the
oracle: key blocks whose scores grow along the selection (so the exponent
reference set by earlier blocks is far below later scores and the kernel's
exact-reference fix-up runs), very large logits, and identical keys (ties,
uniform weights); plus the log-sum-exp output against its definition."""
import math

import numpy as np
import pytest
import torch

import oracle as O
from paper_2602_07397_amd import binding as sw

pytestmark = pytest.mark.gpu

U = pytest.importorskip("_gpu_util")


def _all_causal(b):
    return [list(range(i + 1)) for i in range(b)]


def _pack(sel):
    kmax = max(len(s) for s in sel)
    idx = np.full((len(sel), kmax), -1, dtype=np.int32)
    cnt = np.zeros(len(sel), dtype=np.int32)
    for r, s in enumerate(sel):
        idx[r, :len(s)] = s
        cnt[r] = len(s)
    return U.to_dev(idx), U.to_dev(cnt), kmax


def _f32_bound(Q, K, V, scale=None):
    """Forward error bound of fp32 attention against the exact result on the
    same inputs. A length-d fp32 dot product is within gamma_d * sum|q_i k_i|
    of the exact one (gamma_d = d u / (1 - d u), u = 2^-24); the scaling and
    the exponential add a few ulps of |z|. A perturbation of at most delta in
    every logit moves each normalised weight by a factor within e^(+-2 delta),
    so the output moves by at most (e^(2 delta) - 1) max|V|."""
    Qh, Kh, Vh = (np.abs(x.double().numpy()) for x in (Q, K, V))
    h_q, _, d = Qh.shape
    G = h_q // Kh.shape[0]
    sc = 1.0 / math.sqrt(d) if scale is None else scale
    u = 2.0 ** -24
    gamma = d * u / (1 - d * u)
    dots = max(float((Qh[h] @ Kh[h // G].T).max()) for h in range(h_q)) * sc
    delta = gamma * dots + 4 * u * dots
    return math.expm1(2 * delta) * float(Vh.max()) + U.ATOL_F32


def _f32_tol(Q, K, V, cap):
    """The fp32 tolerance where the logits reach hundreds: the worst-case
    bound above, capped at `cap`, a fixed ceiling a few times the error the
    kernel shows on these inputs, so that a rescaling mistake well inside the
    (loose) worst-case bound still fails."""
    return min(_f32_bound(Q, K, V), cap)


def _inputs(n, h_q, h_kv, d, seed, kscale=None):
    g = torch.Generator().manual_seed(seed)
    Q = torch.randn((h_q, n, d), generator=g)
    K = torch.randn((h_kv, n, d), generator=g)
    V = torch.randn((h_kv, n, d), generator=g)
    if kscale is not None:
        K = K * kscale[None, :, None]
    return Q, K, V


@pytest.mark.parametrize("dtype,B", [("bf16", 128), ("bf16", 64), ("f32", 64)])
def test_growing_scores_force_reference_fixups(dtype, B):
    """Key block j is scaled by 1 + 1.5 j, so every later block's scores
    exceed the reference the earlier ones set by many powers of two."""
    n, h_q, h_kv, d = 1024, 4, 2, 128 if dtype == "bf16" else 64
    blk = torch.arange(n) // B
    Q, K, V = _inputs(n, h_q, h_kv, d, 11, kscale=1.0 + 1.5 * blk.float())
    td = torch.bfloat16 if dtype == "bf16" else torch.float32
    Q, K, V = Q.to(td), K.to(td), V.to(td)
    sel = _all_causal(-(-n // B))
    idx, cnt, kmax = _pack(sel)
    out, lse = sw.sparse_attn_prefill(U.to_dev(Q), U.to_dev(K), U.to_dev(V), [0, n], B, idx, cnt,
                                      kmax, want_lse=True)
    ref = O.sparse_attention_prefill(Q, K, V, B, sel)
    # fp32: logits up to ~300; observed max-abs error 1.9e-5
    tol = U.ATOL_BF16 if dtype == "bf16" else _f32_tol(Q, K, V, 5e-5)
    assert torch.isfinite(out.float()).all() and torch.isfinite(lse).all()
    err = U.max_abs(out.float().cpu().numpy(), ref)
    print(f"\n[numerics] growing scores {dtype} B={B}: max-abs {err:.2e}, tolerance {tol:.2e}")
    assert err <= tol


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_large_logits_stay_finite(dtype):
    """Scores of several hundred (logits far beyond exp range in fp32 without
    a reference) give finite outputs equal to the oracle's."""
    n, B, h_q, h_kv, d = 700, 64, 2, 1, 64
    Q, K, V = _inputs(n, h_q, h_kv, d, 12)
    Q = Q * 12.0
    K = K * 12.0
    td = torch.bfloat16 if dtype == "bf16" else torch.float32
    Q, K, V = Q.to(td), K.to(td), V.to(td)
    rng = np.random.default_rng(3)
    sel = [sorted({0, i} | {j for j in range(1, i) if rng.uniform() < 0.4}) for i in range(-(-n // B))]
    idx, cnt, kmax = _pack(sel)
    out = sw.sparse_attn_prefill(U.to_dev(Q), U.to_dev(K), U.to_dev(V), [0, n], B, idx, cnt, kmax)
    ref = O.sparse_attention_prefill(Q, K, V, B, sel)
    # fp32: logits of several hundred; observed max-abs error 1.2e-4
    tol = U.ATOL_BF16 if dtype == "bf16" else _f32_tol(Q, K, V, 3e-4)
    assert torch.isfinite(out.float()).all()
    err = U.max_abs(out.float().cpu().numpy(), ref)
    print(f"\n[numerics] large logits {dtype}: max-abs {err:.2e}, tolerance {tol:.2e}")
    assert err <= tol


def test_identical_keys_give_uniform_weights():
    """All keys equal: every causal selected key has the same weight, so each
    output row is the mean of the selected values up to the query."""
    n, B, h_q, h_kv, d = 500, 64, 2, 1, 128
    Q, _, V = _inputs(n, h_q, h_kv, d, 13)
    K = torch.ones((h_kv, n, d)) * 0.25
    Q, K, V = Q.to(torch.bfloat16), K.to(torch.bfloat16), V.to(torch.bfloat16)
    sel = _all_causal(-(-n // B))
    idx, cnt, kmax = _pack(sel)
    out = sw.sparse_attn_prefill(U.to_dev(Q), U.to_dev(K), U.to_dev(V), [0, n], B, idx, cnt, kmax)
    Vh = V.double().numpy()[0]
    mean = np.cumsum(Vh, axis=0) / np.arange(1, n + 1)[:, None]
    for u in range(h_q):
        assert U.max_abs(out[u].float().cpu().numpy(), mean) <= U.ATOL_BF16


def test_lse_matches_definition():
    """lse = log of the softmax denominator over the selected causal keys
    (natural log, scale 1/sqrt(d))."""
    n, B, h_q, h_kv, d = 300, 64, 2, 1, 64
    Q, K, V = _inputs(n, h_q, h_kv, d, 14)
    rng = np.random.default_rng(4)
    b = -(-n // B)
    sel = [sorted({0, i} | {j for j in range(1, i) if rng.uniform() < 0.5}) for i in range(b)]
    idx, cnt, kmax = _pack(sel)
    _, lse = sw.sparse_attn_prefill(U.to_dev(Q), U.to_dev(K), U.to_dev(V), [0, n], B, idx, cnt, kmax,
                                    want_lse=True)
    Qh, Kh = Q.double().numpy(), K.double().numpy()
    got = lse.cpu().numpy()
    for u in range(h_q):
        for t in range(0, n, 7):
            i = t // B
            toks = np.concatenate([np.arange(j * B, min(n, (j + 1) * B)) for j in sel[i]])
            toks = toks[toks <= t]
            z = Kh[0, toks] @ Qh[u, t] / math.sqrt(d)
            ref = z.max() + math.log(np.exp(z - z.max()).sum())
            assert abs(got[u, t] - ref) <= 1e-4 * max(1.0, abs(ref)), (u, t)
