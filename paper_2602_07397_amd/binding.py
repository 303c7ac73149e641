"""Thin ctypes binding over libsketchwalk.so.

Argument marshalling only: every function here checks tensor placement,
dtype and contiguity, allocates outputs with torch and passes raw pointers to
the C ABI of the same name (without the ``sw_`` prefix). All computation runs
in the library's HIP kernels; there is no fallback path. If the library is not
built or cannot be loaded, every call raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence, Tuple

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsketchwalk.so")

SW_OK = 0
SW_F32 = 0
SW_BF16 = 1
FORCE_FIRST = 1
FORCE_LAST = 2
FORCE_BOTH = 3
WALK_POWER = 0
WALK_RELU = 1
WALK_SOFTMAX = 2
WALK_MATPOW = 3
MAX_SEQS = 64
MAX_BLOCKS = 4096

_c_int = ctypes.c_int
_c_i64 = ctypes.c_int64
_vp = ctypes.c_void_p
_i32p = ctypes.POINTER(ctypes.c_int32)
_i64p = ctypes.POINTER(ctypes.c_int64)

# name -> (restype, argtypes)
_SIGNATURES = {
    "sw_last_error": (ctypes.c_char_p, []),
    "sw_abi_version": (_c_int, []),
    "sw_layout": (_c_int, [_c_int, _i32p, _c_int, _i64p, _i64p, _i32p]),
    "sw_sketch_workspace_bytes": (_c_i64, [_c_int, _c_int, _c_int, _c_int, _i32p, _c_int]),
    "sw_select_max_count": (_c_int, [_c_int, _i32p, _c_int, _c_int, _c_int, ctypes.c_uint32, _i32p]),
    "sw_sketch_scores": (_c_int, [_c_int, _vp, _vp, _c_int, _c_int, _c_int, _c_int, _i32p, _c_int,
                                  _vp, _vp, _c_int, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _c_i64, _vp]),
    "sw_walk_update": (_c_int, [_vp, _vp, _c_int, _c_int, _i32p, _c_int, _vp, _vp, _vp]),
    "sw_walk_workspace_bytes": (_c_i64, [_c_int, _c_int, _i32p, _c_int]),
    "sw_walk_update_variant": (_c_int, [_c_int, _vp, _vp, _c_int, ctypes.c_double, _c_int, _i32p,
                                        _c_int, _vp, _vp, _vp, _c_i64, _vp]),
    "sw_select_topk_blocks": (_c_int, [_vp, _c_int, _i32p, _c_int, _c_int, _c_int, ctypes.c_uint32,
                                       _vp, _vp, _c_int, _vp]),
    "sw_sparse_attn_prefill": (_c_int, [_c_int, _vp, _vp, _vp, _c_int, _c_int, _c_int, _c_int, _i32p,
                                        _c_int, _vp, _vp, _c_int, ctypes.c_float, _vp, _vp, _vp]),
    "sw_decode_state_bytes": (_c_i64, [_c_int, _c_int, _c_int, _c_int]),
    "sw_decode_state_init": (_c_int, [_vp, _c_int, _c_int, _c_int, _c_int, _c_int, _c_int, _c_int,
                                      _vp, _vp, _vp, _vp, _vp, _vp, _vp]),
    "sw_kv_append": (_c_int, [_c_int, _vp, _vp, _vp, _vp, _c_int, _c_int, _c_int, _c_int, _vp, _vp]),
    "sw_sketch_scores_decode": (_c_int, [_c_int, _vp, _vp, _c_int, _c_int, _c_int, _c_int, _c_int, _vp,
                                         _vp, _vp, _c_int, _c_int, _vp, _vp]),
    "sw_walk_update_decode": (_c_int, [_vp, _c_int, _c_int, _c_int, _c_int, _c_int, _vp, _c_int, _vp,
                                       _vp, _vp]),
    "sw_walk_update_decode_variant": (_c_int, [_c_int, _vp, _c_int, _c_int, _c_int, _c_int, _c_int,
                                               _vp, _c_int, _vp, _vp, _vp]),
    "sw_select_max_count_decode": (_c_int, [_c_int, _c_int, _c_int, ctypes.c_uint32, _i32p]),
    "sw_select_topk_blocks_decode": (_c_int, [_vp, _c_int, _c_int, _c_int, _vp, _c_int, _c_int,
                                              ctypes.c_uint32, _vp, _vp, _c_int, _vp]),
    "sw_decode_attn_workspace_bytes": (_c_i64, [_c_int, _c_int, _c_int, _c_int]),
    "sw_decode_step_workspace_bytes": (_c_i64, [_c_int, _c_int, _c_int, _c_int]),
    "sw_decode_step": (_c_int, [_c_int, _c_int, _c_int, _c_int, _c_int, _c_int, _c_int, _c_int,
                                _c_int, _c_int, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                                _c_int, _c_int, _c_int, _c_int, ctypes.c_uint32, _c_int,
                                ctypes.c_float, _vp, _vp, _vp, _vp, _vp, _c_i64, _vp]),
    "sw_sparse_attn_decode": (_c_int, [_c_int, _vp, _vp, _vp, _c_int, _c_int, _c_int, _c_int, _c_int,
                                       _c_int, _vp, _vp, _vp, _c_int, ctypes.c_float, _vp, _vp, _c_i64,
                                       _vp]),
    "sw_sparse_attn_decode_noalloc": (_c_int, [_c_int, _vp, _vp, _vp, _c_int, _c_int, _c_int, _c_int,
                                               _c_int, _c_int, _vp, _vp, _vp, _c_int, ctypes.c_float,
                                               _vp, _vp]),
}

NOALLOC_SCRATCH_BYTES = 8 * 1024 * 1024

_lib = None


class SketchWalkError(RuntimeError):
    pass


def load() -> ctypes.CDLL:
    """Loads the built library (raises if it is missing)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise SketchWalkError(
            f"{LIB_PATH} is not built; run `python -m paper_2602_07397_amd.build` first")
    lib = ctypes.CDLL(LIB_PATH)
    for name, (res, args) in _SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def exported_symbols() -> Sequence[str]:
    return tuple(_SIGNATURES)


def _check(rc: int, what: str) -> None:
    if rc != SW_OK:
        msg = load().sw_last_error().decode(errors="replace")
        raise SketchWalkError(f"{what} failed with code {rc}: {msg}")


def _cu(cu_seqlens) -> Tuple[ctypes.Array, int]:
    arr = np.ascontiguousarray(np.asarray(cu_seqlens, dtype=np.int32))
    buf = (ctypes.c_int32 * arr.size)(*arr.tolist())
    return buf, arr.size - 1


def _dev(t: torch.Tensor, name: str, dtype=None) -> int:
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
        raise SketchWalkError(f"{name} must be a CUDA (HIP) tensor")
    if not t.is_contiguous():
        raise SketchWalkError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise SketchWalkError(f"{name} must have dtype {dtype}, got {t.dtype}")
    return t.data_ptr()


def _opt(t: Optional[torch.Tensor], name: str, dtype=None) -> Optional[int]:
    return None if t is None else _dev(t, name, dtype)


def _stream(dev: torch.device) -> int:
    return torch.cuda.current_stream(dev).cuda_stream


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return SW_BF16
    if t.dtype == torch.float32:
        return SW_F32
    raise SketchWalkError(f"unsupported dtype {t.dtype}")


def abi_version() -> int:
    return load().sw_abi_version()


def layout(cu_seqlens, B: int) -> Tuple[int, int, int]:
    """(nb, nm, max_b): total block rows, total matrix elements, largest b_s."""
    cu, n = _cu(cu_seqlens)
    nb, nm, mb = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int32()
    _check(load().sw_layout(n, cu, B, ctypes.byref(nb), ctypes.byref(nm), ctypes.byref(mb)), "sw_layout")
    return nb.value, nm.value, mb.value


def sketch_workspace_bytes(h_q: int, h_kv: int, d: int, cu_seqlens, B: int) -> int:
    cu, n = _cu(cu_seqlens)
    v = load().sw_sketch_workspace_bytes(h_q, h_kv, d, n, cu, B)
    if v < 0:
        _check(1, "sw_sketch_workspace_bytes")
    return int(v)


def select_max_count(cu_seqlens, B: int, k: int = 0, density_pct: int = 20,
                     flags: int = FORCE_BOTH) -> int:
    cu, n = _cu(cu_seqlens)
    out = ctypes.c_int32()
    _check(load().sw_select_max_count(n, cu, B, k, density_pct, flags, ctypes.byref(out)),
           "sw_select_max_count")
    return out.value


def sketch_scores(Q: torch.Tensor, K: torch.Tensor, cu_seqlens, B: int, signs: torch.Tensor,
                  cols: torch.Tensor, want_means: bool = False, out: Optional[dict] = None,
                  workspace: Optional[torch.Tensor] = None) -> dict:
    """Q [h_q][N][d], K [h_kv][N][d] (bf16 or fp32). Returns dict with Qs, Ks
    [nb][r], A [nm], A_scale [n_seqs] (float64) and Qbar, Kbar [nb][d] when
    ``want_means``. Pre-allocated outputs may be passed in ``out``."""
    lib = load()
    dev = Q.device
    h_q, N, d = Q.shape
    h_kv = K.shape[0]
    r = int(cols.numel())
    nb, nm, _ = layout(cu_seqlens, B)
    cu, n = _cu(cu_seqlens)
    o = dict(out or {})
    f64 = dict(dtype=torch.float64, device=dev)
    o.setdefault("Qs", torch.empty((nb, r), **f64))
    o.setdefault("Ks", torch.empty((nb, r), **f64))
    o.setdefault("A", torch.empty((nm,), **f64))
    o.setdefault("A_scale", torch.empty((n,), **f64))
    if want_means:
        o.setdefault("Qbar", torch.empty((nb, d), **f64))
        o.setdefault("Kbar", torch.empty((nb, d), **f64))
    wsb = sketch_workspace_bytes(h_q, h_kv, d, cu_seqlens, B)
    if workspace is None or workspace.numel() < wsb:
        workspace = torch.empty((max(wsb, 256),), dtype=torch.uint8, device=dev)
    if K.dtype != Q.dtype:
        raise SketchWalkError("Q and K must share a dtype")
    rc = lib.sw_sketch_scores(
        _dtype_code(Q), _dev(Q, "Q"), _dev(K, "K"), h_q, h_kv, d, n, cu, B,
        _dev(signs, "signs", torch.int8), _dev(cols, "cols", torch.int32), r,
        _dev(o["Qs"], "Qs", torch.float64), _dev(o["Ks"], "Ks", torch.float64),
        _dev(o["A"], "A", torch.float64), _dev(o["A_scale"], "A_scale", torch.float64),
        _opt(o.get("Qbar"), "Qbar", torch.float64), _opt(o.get("Kbar"), "Kbar", torch.float64),
        _dev(workspace, "workspace"), workspace.numel(), _stream(dev))
    _check(rc, "sw_sketch_scores")
    return o


def walk_update(A: torch.Tensor, A_scale: torch.Tensor, s: int, cu_seqlens, B: int,
                R_prev: Optional[torch.Tensor] = None,
                R_out: Optional[torch.Tensor] = None) -> torch.Tensor:
    lib = load()
    cu, n = _cu(cu_seqlens)
    if R_out is None:
        R_out = torch.empty_like(A)
    rc = lib.sw_walk_update(_dev(A, "A", torch.float64), _dev(A_scale, "A_scale", torch.float64), s,
                            n, cu, B, _opt(R_prev, "R_prev", torch.float64),
                            _dev(R_out, "R_out", torch.float64), _stream(A.device))
    _check(rc, "sw_walk_update")
    return R_out


def walk_workspace_bytes(variant: int, cu_seqlens, B: int) -> int:
    cu, n = _cu(cu_seqlens)
    v = load().sw_walk_workspace_bytes(variant, n, cu, B)
    if v < 0:
        _check(1, "sw_walk_workspace_bytes")
    return int(v)


def walk_update_variant(variant: int, A: torch.Tensor, A_scale: torch.Tensor, s: int, cu_seqlens,
                        B: int, R_prev: Optional[torch.Tensor] = None,
                        R_out: Optional[torch.Tensor] = None, logit_scale: float = 1.0,
                        workspace: Optional[torch.Tensor] = None) -> torch.Tensor:
    """variant: WALK_POWER, WALK_RELU, WALK_SOFTMAX (uses ``logit_scale``,
    not ``s``) or WALK_MATPOW."""
    lib = load()
    cu, n = _cu(cu_seqlens)
    if R_out is None:
        R_out = torch.empty_like(A)
    wsb = walk_workspace_bytes(variant, cu_seqlens, B)
    if wsb > 0 and (workspace is None or workspace.numel() < wsb):
        workspace = torch.empty((wsb,), dtype=torch.uint8, device=A.device)
    rc = lib.sw_walk_update_variant(
        variant, _dev(A, "A", torch.float64), _dev(A_scale, "A_scale", torch.float64), s,
        float(logit_scale), n, cu, B, _opt(R_prev, "R_prev", torch.float64),
        _dev(R_out, "R_out", torch.float64), _opt(workspace, "workspace"),
        0 if workspace is None else workspace.numel(), _stream(A.device))
    _check(rc, "sw_walk_update_variant")
    return R_out


def select_topk_blocks(R: torch.Tensor, cu_seqlens, B: int, k: int = 0, density_pct: int = 20,
                       flags: int = FORCE_BOTH, kmax: Optional[int] = None,
                       idx: Optional[torch.Tensor] = None,
                       cnt: Optional[torch.Tensor] = None) -> Tuple[torch.Tensor, torch.Tensor, int]:
    lib = load()
    cu, n = _cu(cu_seqlens)
    nb, _, _ = layout(cu_seqlens, B)
    if kmax is None:
        kmax = select_max_count(cu_seqlens, B, k, density_pct, flags)
    if idx is None:
        idx = torch.empty((nb, kmax), dtype=torch.int32, device=R.device)
    if cnt is None:
        cnt = torch.empty((nb,), dtype=torch.int32, device=R.device)
    rc = lib.sw_select_topk_blocks(_dev(R, "R", torch.float64), n, cu, B, k, density_pct, flags,
                                   _dev(idx, "idx", torch.int32), _dev(cnt, "cnt", torch.int32),
                                   kmax, _stream(R.device))
    _check(rc, "sw_select_topk_blocks")
    return idx, cnt, kmax


def sparse_attn_prefill(Q: torch.Tensor, K: torch.Tensor, V: torch.Tensor, cu_seqlens, B: int,
                        idx: torch.Tensor, cnt: torch.Tensor, kmax: int, scale: float = 0.0,
                        want_lse: bool = False, O: Optional[torch.Tensor] = None):
    lib = load()
    cu, n = _cu(cu_seqlens)
    h_q, N, d = Q.shape
    h_kv = K.shape[0]
    if O is None:
        O = torch.empty_like(Q)
    lse = torch.empty((h_q, N), dtype=torch.float32, device=Q.device) if want_lse else None
    if not (K.dtype == V.dtype == Q.dtype == O.dtype):
        raise SketchWalkError("Q, K, V, O must share a dtype")
    rc = lib.sw_sparse_attn_prefill(_dtype_code(Q), _dev(Q, "Q"), _dev(K, "K"), _dev(V, "V"), h_q,
                                    h_kv, d, n, cu, B, _dev(idx, "idx", torch.int32),
                                    _dev(cnt, "cnt", torch.int32), kmax, float(scale),
                                    _dev(O, "O"), _opt(lse, "lse", torch.float32),
                                    _stream(Q.device))
    _check(rc, "sw_sparse_attn_prefill")
    return (O, lse) if want_lse else O


# ---------------------------------------------------------------------------
# decode (Alg. 2)
# ---------------------------------------------------------------------------

def decode_state_bytes(batch: int, d: int, r: int, b_max: int) -> int:
    v = load().sw_decode_state_bytes(batch, d, r, b_max)
    if v < 0:
        _check(1, "sw_decode_state_bytes")
    return int(v)


def new_decode_state(batch: int, d: int, r: int, b_max: int, device) -> torch.Tensor:
    """A zero-filled byte buffer holding one layer's decode state."""
    return torch.zeros((decode_state_bytes(batch, d, r, b_max),), dtype=torch.uint8, device=device)


def decode_state_init(state: torch.Tensor, batch: int, d: int, r: int, b_max: int, seq: int, n: int,
                      B: int, sk: dict) -> None:
    """Initialises sequence ``seq`` of ``state`` from one sequence's
    sketch_scores output (computed with want_means=True)."""
    rc = load().sw_decode_state_init(
        _dev(state, "state", torch.uint8), batch, d, r, b_max, seq, n, B,
        _dev(sk["Qs"], "Qs", torch.float64), _dev(sk["Ks"], "Ks", torch.float64),
        _dev(sk["A"], "A", torch.float64), _dev(sk["A_scale"], "A_scale", torch.float64),
        _dev(sk["Qbar"], "Qbar", torch.float64), _dev(sk["Kbar"], "Kbar", torch.float64),
        _stream(state.device))
    _check(rc, "sw_decode_state_init")


def kv_append(k_new: torch.Tensor, v_new: torch.Tensor, Kc: torch.Tensor, Vc: torch.Tensor,
              pos: torch.Tensor) -> None:
    batch, h_kv, T_max, d = Kc.shape
    rc = load().sw_kv_append(_dtype_code(Kc), _dev(k_new, "k_new", Kc.dtype), _dev(v_new, "v_new", Kc.dtype),
                             _dev(Kc, "Kc"), _dev(Vc, "Vc", Kc.dtype), batch, h_kv, d, T_max,
                             _dev(pos, "pos", torch.int32), _stream(Kc.device))
    _check(rc, "sw_kv_append")


def sketch_scores_decode(q_new: torch.Tensor, k_new: torch.Tensor, B: int, pos: torch.Tensor,
                         signs: torch.Tensor, cols: torch.Tensor, b_max: int,
                         state: torch.Tensor) -> None:
    batch, h_q, d = q_new.shape
    h_kv = k_new.shape[1]
    rc = load().sw_sketch_scores_decode(
        _dtype_code(q_new), _dev(q_new, "q_new"), _dev(k_new, "k_new", q_new.dtype), batch, h_q, h_kv,
        d, B, _dev(pos, "pos", torch.int32), _dev(signs, "signs", torch.int8),
        _dev(cols, "cols", torch.int32), int(cols.numel()), b_max, _dev(state, "state", torch.uint8),
        _stream(q_new.device))
    _check(rc, "sw_sketch_scores_decode")


def walk_update_decode(state: torch.Tensor, batch: int, d: int, r: int, b_max: int, B: int,
                       pos: torch.Tensor, s: int, r_prev: Optional[torch.Tensor] = None,
                       r_out: Optional[torch.Tensor] = None) -> torch.Tensor:
    dev = state.device
    if r_out is None:
        r_out = torch.empty((batch, b_max), dtype=torch.float64, device=dev)
    rc = load().sw_walk_update_decode(_dev(state, "state", torch.uint8), batch, d, r, b_max, B,
                                      _dev(pos, "pos", torch.int32), s,
                                      _opt(r_prev, "r_prev", torch.float64),
                                      _dev(r_out, "r_out", torch.float64), _stream(dev))
    _check(rc, "sw_walk_update_decode")
    return r_out


def walk_update_decode_variant(variant: int, state: torch.Tensor, batch: int, d: int, r: int,
                               b_max: int, B: int, pos: torch.Tensor, s: int,
                               r_prev: Optional[torch.Tensor] = None,
                               r_out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """variant: WALK_POWER or WALK_RELU (the others raise: unsupported)."""
    dev = state.device
    if r_out is None:
        r_out = torch.empty((batch, b_max), dtype=torch.float64, device=dev)
    rc = load().sw_walk_update_decode_variant(variant, _dev(state, "state", torch.uint8), batch, d,
                                              r, b_max, B, _dev(pos, "pos", torch.int32), s,
                                              _opt(r_prev, "r_prev", torch.float64),
                                              _dev(r_out, "r_out", torch.float64), _stream(dev))
    _check(rc, "sw_walk_update_decode_variant")
    return r_out


def select_max_count_decode(b_max: int, k: int = 0, density_pct: int = 20,
                            flags: int = FORCE_BOTH) -> int:
    out = ctypes.c_int32()
    _check(load().sw_select_max_count_decode(b_max, k, density_pct, flags, ctypes.byref(out)),
           "sw_select_max_count_decode")
    return out.value


def select_topk_blocks_decode(rows: torch.Tensor, B: int, pos: torch.Tensor, k: int = 0,
                              density_pct: int = 20, flags: int = FORCE_BOTH,
                              kmax: Optional[int] = None, idx: Optional[torch.Tensor] = None,
                              cnt: Optional[torch.Tensor] = None):
    batch, b_max = rows.shape
    if kmax is None:
        kmax = select_max_count_decode(b_max, k, density_pct, flags)
    if idx is None:
        idx = torch.empty((batch, kmax), dtype=torch.int32, device=rows.device)
    if cnt is None:
        cnt = torch.empty((batch,), dtype=torch.int32, device=rows.device)
    rc = load().sw_select_topk_blocks_decode(_dev(rows, "rows", torch.float64), batch, b_max, B,
                                             _dev(pos, "pos", torch.int32), k, density_pct, flags,
                                             _dev(idx, "idx", torch.int32), _dev(cnt, "cnt", torch.int32),
                                             kmax, _stream(rows.device))
    _check(rc, "sw_select_topk_blocks_decode")
    return idx, cnt, kmax


def decode_attn_workspace_bytes(batch: int, h_q: int, h_kv: int, d: int) -> int:
    v = load().sw_decode_attn_workspace_bytes(batch, h_q, h_kv, d)
    if v < 0:
        _check(1, "sw_decode_attn_workspace_bytes")
    return int(v)


def sparse_attn_decode(q: torch.Tensor, Kc: torch.Tensor, Vc: torch.Tensor, B: int, pos: torch.Tensor,
                       idx: torch.Tensor, cnt: torch.Tensor, kmax: int, scale: float = 0.0,
                       O: Optional[torch.Tensor] = None,
                       workspace: Optional[torch.Tensor] = None) -> torch.Tensor:
    batch, h_q, d = q.shape
    _, h_kv, T_max, _ = Kc.shape
    dev = q.device
    if O is None:
        O = torch.empty_like(q)
    wsb = decode_attn_workspace_bytes(batch, h_q, h_kv, d)
    if workspace is None or workspace.numel() < wsb:
        workspace = torch.empty((max(wsb, 256),), dtype=torch.uint8, device=dev)
    if not (Kc.dtype == Vc.dtype == q.dtype == O.dtype):
        raise SketchWalkError("q, Kc, Vc, O must share a dtype")
    rc = load().sw_sparse_attn_decode(_dtype_code(q), _dev(q, "q"), _dev(Kc, "Kc"), _dev(Vc, "Vc"),
                                      batch, h_q, h_kv, d, T_max, B, _dev(pos, "pos", torch.int32),
                                      _dev(idx, "idx", torch.int32), _dev(cnt, "cnt", torch.int32), kmax,
                                      float(scale), _dev(O, "O"), _dev(workspace, "workspace"),
                                      workspace.numel(), _stream(dev))
    _check(rc, "sw_sparse_attn_decode")
    return O


def sparse_attn_decode_noalloc(q: torch.Tensor, Kc: torch.Tensor, Vc: torch.Tensor, B: int,
                               pos: torch.Tensor, idx: torch.Tensor, cnt: torch.Tensor, kmax: int,
                               scale: float = 0.0, O: Optional[torch.Tensor] = None) -> torch.Tensor:
    """sparse_attn_decode without a workspace: the library's fixed per-GPU
    scratch holds the split-K partials (pass a pre-allocated ``O`` to make
    the whole call allocation-free)."""
    batch, h_q, d = q.shape
    _, h_kv, T_max, _ = Kc.shape
    if O is None:
        O = torch.empty_like(q)
    if not (Kc.dtype == Vc.dtype == q.dtype == O.dtype):
        raise SketchWalkError("q, Kc, Vc, O must share a dtype")
    rc = load().sw_sparse_attn_decode_noalloc(_dtype_code(q), _dev(q, "q"), _dev(Kc, "Kc"),
                                              _dev(Vc, "Vc"), batch, h_q, h_kv, d, T_max, B,
                                              _dev(pos, "pos", torch.int32),
                                              _dev(idx, "idx", torch.int32),
                                              _dev(cnt, "cnt", torch.int32), kmax, float(scale),
                                              _dev(O, "O"), _stream(q.device))
    _check(rc, "sw_sparse_attn_decode_noalloc")
    return O


def decode_step(q_new: torch.Tensor, k_new: torch.Tensor, v_new: torch.Tensor, Kc: torch.Tensor,
                Vc: torch.Tensor, state: torch.Tensor, pos: torch.Tensor, signs: torch.Tensor,
                cols: torch.Tensor, B: int, b_max: int, s: int = 8, walk_variant: int = WALK_POWER,
                k: int = 0, density_pct: int = 20, flags: int = FORCE_BOTH,
                kmax: Optional[int] = None, scale: float = 0.0, out: Optional[dict] = None,
                workspace: Optional[torch.Tensor] = None) -> dict:
    """One decode step of every layer (layer-stacked tensors):
    q_new [L][batch][h_q][d], k_new/v_new [L][batch][h_kv][d], Kc/Vc
    [L][batch][h_kv][T_max][d], state [L][state_bytes] uint8. Returns dict with
    rows [L][batch][b_max], idx [L][batch][kmax], cnt [L][batch], O
    [L][batch][h_q][d]; pre-allocated outputs may be passed in ``out``."""
    L, batch, h_q, d = q_new.shape
    h_kv = k_new.shape[2]
    T_max = Kc.shape[3]
    r = int(cols.numel())
    dev = q_new.device
    if kmax is None:
        kmax = select_max_count_decode(b_max, k=k, density_pct=density_pct, flags=flags)
    o = dict(out or {})
    o.setdefault("rows", torch.empty((L, batch, b_max), dtype=torch.float64, device=dev))
    o.setdefault("idx", torch.empty((L, batch, kmax), dtype=torch.int32, device=dev))
    o.setdefault("cnt", torch.empty((L, batch), dtype=torch.int32, device=dev))
    o.setdefault("O", torch.empty_like(q_new))
    wsb = int(load().sw_decode_step_workspace_bytes(batch, h_q, h_kv, d))
    if wsb < 0:
        _check(1, "sw_decode_step_workspace_bytes")
    if workspace is None or workspace.numel() < wsb:
        workspace = torch.empty((max(wsb, 256),), dtype=torch.uint8, device=dev)
    for name, t in (("k_new", k_new), ("v_new", v_new), ("Kc", Kc), ("Vc", Vc)):
        if t.dtype != q_new.dtype:
            raise SketchWalkError(f"{name} must have dtype {q_new.dtype}")
    rc = load().sw_decode_step(
        _dtype_code(q_new), L, batch, h_q, h_kv, d, r, T_max, B, b_max, _dev(q_new, "q_new"),
        _dev(k_new, "k_new"), _dev(v_new, "v_new"), _dev(Kc, "Kc"), _dev(Vc, "Vc"),
        _dev(state, "state", torch.uint8), _dev(pos, "pos", torch.int32),
        _dev(signs, "signs", torch.int8), _dev(cols, "cols", torch.int32), s, walk_variant, k,
        density_pct, flags, kmax, float(scale), _dev(o["rows"], "rows", torch.float64),
        _dev(o["idx"], "idx", torch.int32), _dev(o["cnt"], "cnt", torch.int32),
        _dev(o["O"], "O", q_new.dtype), _dev(workspace, "workspace"), workspace.numel(),
        _stream(dev))
    _check(rc, "sw_decode_step")
    return o
