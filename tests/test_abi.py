"""CPU checks of the C ABI: the library loads, exports every function the
public header declares, and rejects invalid arguments on the host before any
GPU work (no compute call is made here)."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2602_07397_amd import binding as sw

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sketchwalk.h")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sw_[a-z0-9_]+)\s*\(", text)))


def test_library_loads_and_reports_version():
    lib = sw.load()
    assert lib.sw_abi_version() == 1


def test_every_declared_function_is_exported_and_bound():
    lib = sw.load()
    names = _declared_functions()
    assert len(names) >= 9
    for name in names:
        assert hasattr(lib, name), name
        assert name in sw.exported_symbols(), f"{name} missing from the binding"


def test_layout_and_budget_queries():
    assert sw.layout([0, 2048], 64) == (32, 1024, 32)
    assert sw.layout(np.cumsum([0, 100, 300, 64]), 64) == (2 + 5 + 1, 4 + 25 + 1, 5)
    # tiny workload at 20%: largest row budget is ceil(32 * 20 / 100) = 7
    assert sw.select_max_count([0, 2048], 64, density_pct=20) == 7
    assert sw.select_max_count([0, 2048], 64, density_pct=100) == 32
    assert sw.select_max_count([0, 2048], 64, k=3, flags=0) == 3
    assert sw.sketch_workspace_bytes(32, 8, 128, [0, 32768], 128) >= 0


def _err(fn, *args):
    lib = sw.load()
    rc = getattr(lib, fn)(*args)
    return rc, lib.sw_last_error().decode()


def _cu(vals):
    arr = (ctypes.c_int32 * len(vals))(*vals)
    return arr


FAKE = 1 << 20   # 16-byte aligned non-null address; never dereferenced


def test_sketch_rejects_bad_arguments():
    cu = _cu([0, 256])
    base = [sw.SW_BF16, FAKE, FAKE, 4, 2, 64, 1, cu, 64, FAKE, FAKE, 32,
            FAKE, FAKE, FAKE, FAKE, None, None, FAKE, 1 << 30, None]
    # every case below must fail host validation: nothing is ever launched
    cases = {
        "dtype": (0, 7),
        "heads": (4, 3),          # h_q=4 not a multiple of h_kv=3
        "d": (5, 48),             # not a power of two
        "r": (11, 65),            # r > d
        "B": (8, 24),             # not a multiple of 16
        "nseq": (6, 0),
        "Q null": (1, None),
        "Q misaligned": (1, FAKE + 2),
        "Qs null": (12, None),
    }
    for name, (pos, val) in cases.items():
        args = list(base)
        args[pos] = val
        rc, msg = _err("sw_sketch_scores", *args)
        assert rc == 1, (name, rc, msg)
        assert msg, name


def test_sketch_rejects_bad_cu_seqlens():
    args = [sw.SW_BF16, FAKE, FAKE, 4, 2, 64, 2, _cu([0, 100, 100]), 64, FAKE, FAKE, 32,
            FAKE, FAKE, FAKE, FAKE, None, None, FAKE, 1 << 30, None]
    rc, msg = _err("sw_sketch_scores", *args)
    assert rc == 1 and "length" in msg
    args[7] = _cu([5, 100, 200])
    rc, msg = _err("sw_sketch_scores", *args)
    assert rc == 1


def test_walk_select_attention_reject_bad_arguments():
    cu = _cu([0, 256])
    rc, msg = _err("sw_walk_update", FAKE, FAKE, 0, 1, cu, 64, None, FAKE + 256, None)
    assert rc == 1 and "s=" in msg
    rc, msg = _err("sw_walk_update", FAKE, FAKE, 8, 1, cu, 64, FAKE, FAKE, None)
    assert rc == 1 and "alias" in msg
    # kmax below the largest budget
    rc, msg = _err("sw_select_topk_blocks", FAKE, 1, cu, 64, 0, 50, 3, FAKE, FAKE, 1, None)
    assert rc == 1 and "kmax" in msg
    rc, msg = _err("sw_select_topk_blocks", FAKE, 1, cu, 64, 0, 0, 3, FAKE, FAKE, 8, None)
    assert rc == 1 and "density" in msg
    rc, msg = _err("sw_select_topk_blocks", FAKE, 1, cu, 64, 0, 20, 8, FAKE, FAKE, 8, None)
    assert rc == 1 and "flags" in msg
    # attention: unsupported head dim / block size
    rc, msg = _err("sw_sparse_attn_prefill", sw.SW_BF16, FAKE, FAKE, FAKE, 4, 2, 96, 1, cu, 64,
                   FAKE, FAKE, 4, ctypes.c_float(0.0), FAKE, None, None)
    assert rc == 2
    rc, msg = _err("sw_sparse_attn_prefill", sw.SW_BF16, FAKE, FAKE, FAKE, 4, 2, 128, 1, cu, 32,
                   FAKE, FAKE, 4, ctypes.c_float(0.0), FAKE, None, None)
    assert rc == 2
    rc, msg = _err("sw_sparse_attn_prefill", sw.SW_BF16, FAKE, FAKE, FAKE, 4, 3, 128, 1, cu, 64,
                   FAKE, FAKE, 4, ctypes.c_float(0.0), FAKE, None, None)
    assert rc == 1


@pytest.mark.parametrize("B", [0, 8, 40, 1040])
def test_decode_attention_rejects_block_sizes_off_the_16_token_grid(B):
    """The decode attention walks each selected block in 16-token groups: a
    block size that is not a multiple of 16 in [16, 1024] is refused before
    anything is enqueued."""
    rc, msg = _err("sw_sparse_attn_decode", sw.SW_BF16, FAKE, FAKE, FAKE, 2, 8, 2, 128, 4096, B,
                   FAKE, FAKE, FAKE, 8, ctypes.c_float(0.0), FAKE, FAKE, 1 << 30, None)
    assert rc == 1 and "B=" in msg, msg


def test_binding_refuses_cpu_tensors():
    import torch
    x = torch.zeros((1, 64, 64))
    with pytest.raises(sw.SketchWalkError):
        sw.sparse_attn_prefill(x, x, x, [0, 64], 64, torch.zeros((1, 1), dtype=torch.int32),
                               torch.zeros(1, dtype=torch.int32), 1)


def _compile_and_run_c(tmp_path, lang):
    import shutil
    import subprocess
    cc = shutil.which("gcc" if lang == "c" else "g++")
    if cc is None:
        pytest.skip("no host compiler")
    exe = str(tmp_path / f"abi_check_{lang}")
    src = os.path.join(ROOT, "tests", "abi_check.c")
    libdir = os.path.dirname(sw.LIB_PATH)
    std = ["-std=c99", "-pedantic"] if lang == "c" else ["-x", "c++", "-std=c++17"]
    cmd = [cc, *std, "-Wall", "-Wextra", "-Werror", "-I", os.path.join(ROOT, "include"), src,
           "-L", libdir, f"-Wl,-rpath,{libdir}", "-l:libsketchwalk.so", "-o", exe]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    out = subprocess.run([exe], check=True, capture_output=True, text=True).stdout
    return dict((line.split(" ", 1)[0], line.split(" ", 1)[1]) for line in out.strip().splitlines())


@pytest.mark.parametrize("lang", ["c", "c++"])
def test_header_compiles_and_links_from_c(tmp_path, lang):
    """The public header compiles as C99 and as C++ with warnings as errors,
    every call links against the built library, and the host-side answers
    agree with the binding's."""
    r = _compile_and_run_c(tmp_path, lang)
    cu = [0, 100, 400]
    assert r["version"] == "1"
    nb, nm, mb = sw.layout(cu, 64)
    assert r["layout"] == f"0 {nb} {nm} {mb}"
    assert r["max_count"] == f"0 {sw.select_max_count(cu, 64, density_pct=20)}"
    assert r["sketch_ws"] == str(sw.sketch_workspace_bytes(32, 8, 128, cu, 64))
    assert r["walk_ws"] == f"{sw.walk_workspace_bytes(sw.WALK_MATPOW, cu, 64)} 0"
    assert r["state_bytes"] == str(sw.decode_state_bytes(16, 128, 64, 1028))
    assert int(r["step_ws"]) > 0
    assert r["bad_variant"].startswith("1 ") and "variant" in r["bad_variant"]
    assert r["too_many_blocks"] == "2"


def test_noalloc_decode_attention_refuses_oversize_calls_on_the_host():
    """A call whose split-K partials exceed the fixed scratch is refused
    before any device work (no GPU needed to see it)."""
    batch, h_q, h_kv, d = 4096, 32, 8, 128
    assert sw.decode_attn_workspace_bytes(batch, h_q, h_kv, d) > sw.NOALLOC_SCRATCH_BYTES
    rc, msg = _err("sw_sparse_attn_decode_noalloc", sw.SW_BF16, FAKE, FAKE, FAKE, batch, h_q, h_kv,
                   d, 4096, 64, FAKE, FAKE, FAKE, 8, ctypes.c_float(0.0), FAKE, None)
    assert rc == 1 and "scratch" in msg, msg
