"""The allocation-free decode attention (sw_sparse_attn_decode_noalloc)
against the workspace entry point (sw_sparse_attn_decode) through the C ABI:
two calls in a row, the second with a smaller batch, cache and selection,
both bit-identical to the workspace call on the same inputs and within the
bf16 / fp32 tolerance of the oracle; an oversize call is refused."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2602_07397_amd import binding as sw

pytestmark = pytest.mark.gpu

U = pytest.importorskip("_gpu_util")


def _case(seed, batch, h_q, h_kv, d, B, T_max, dtype):
    rng = np.random.default_rng(seed)
    g = torch.Generator().manual_seed(seed)
    td = torch.bfloat16 if dtype == "bf16" else torch.float32
    q = torch.randn((batch, h_q, d), generator=g).to(td)
    Kc = torch.randn((batch, h_kv, T_max, d), generator=g).to(td)
    Vc = torch.randn((batch, h_kv, T_max, d), generator=g).to(td)
    pos = [int(rng.integers(0, T_max)) for _ in range(batch)]
    if batch > 2:
        pos[1] = -1                                   # an inactive sequence
    sels = []
    for p in pos:
        if p < 0:
            sels.append([0])
            continue
        bc = p // B
        sels.append(sorted({0, bc} | {j for j in range(1, bc) if rng.uniform() < 0.3}))
    kmax = max(len(s) for s in sels)
    idx = np.full((batch, kmax), -1, dtype=np.int32)
    for b, s in enumerate(sels):
        idx[b, :len(s)] = s
    cnt = np.array([len(s) for s in sels], dtype=np.int32)
    return dict(q=q, Kc=Kc, Vc=Vc, pos=pos, sels=sels, idx=idx, cnt=cnt, kmax=kmax, B=B)


def _run_both(c):
    q, Kc, Vc = U.to_dev(c["q"]), U.to_dev(c["Kc"]), U.to_dev(c["Vc"])
    pos = U.to_dev(np.array(c["pos"], dtype=np.int32))
    idx, cnt = U.to_dev(c["idx"]), U.to_dev(c["cnt"])
    ref = sw.sparse_attn_decode(q, Kc, Vc, c["B"], pos, idx, cnt, c["kmax"])
    O_out = torch.full_like(q, 7.0)
    got = sw.sparse_attn_decode_noalloc(q, Kc, Vc, c["B"], pos, idx, cnt, c["kmax"], O=O_out)
    torch.cuda.synchronize()
    return ref, got


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_noalloc_decode_attention_equals_workspace_call(dtype):
    big = _case(71, 16, 32, 8, 128, 64, 6000, dtype)
    small = _case(72, 3, 8, 2, 64, 16, 700, dtype)
    tol = U.ATOL_BF16 if dtype == "bf16" else U.ATOL_F32
    for c in (big, small):                           # two calls, the second smaller
        ref, got = _run_both(c)
        assert torch.equal(ref, got)
        og = got.float().cpu().numpy()
        for b, p in enumerate(c["pos"]):
            if p < 0:
                assert np.all(og[b] == 0.0)
                continue
            want = O.decode_attention(c["q"][b], c["Kc"][b], c["Vc"][b], c["sels"][b], p, c["B"])
            assert U.max_abs(og[b], want) <= tol, (b, p)


def test_noalloc_refuses_calls_beyond_its_scratch():
    batch, h_q, h_kv, d = 4096, 32, 8, 128
    need = sw.decode_attn_workspace_bytes(batch, h_q, h_kv, d)
    assert need > sw.NOALLOC_SCRATCH_BYTES
    q = torch.zeros((batch, h_q, d), dtype=torch.bfloat16, device=U.DEV)
    Kc = torch.zeros((batch, h_kv, 16, d), dtype=torch.bfloat16, device=U.DEV)
    pos = torch.zeros((batch,), dtype=torch.int32, device=U.DEV)
    idx = torch.zeros((batch, 1), dtype=torch.int32, device=U.DEV)
    with pytest.raises(sw.SketchWalkError, match="scratch"):
        sw.sparse_attn_decode_noalloc(q, Kc, Kc, 16, pos, idx, pos, 1)
