"""Thin ctypes binding of libpisa (the C ABI declared in include/pisa.h).

Each ``pisa_*`` function here has the name and argument order of its C
counterpart; tensors are passed as device pointers and the stream defaults to
torch's current stream.  Every step of the computation runs in the HIP
library: this module only marshals arguments, allocates outputs with torch and
turns negative status codes into :class:`PisaError`.  It raises at import time
if the library has not been built (there is no fallback path).
"""
from __future__ import annotations

import ctypes
import os

import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libpisa.so")

PISA_DTYPE_F32 = 0
PISA_DTYPE_BF16 = 1
PISA_SCHEDULE_AUTO = 0
PISA_SCHEDULE_TWO_STAGE = 1
PISA_SCHEDULE_FUSED = 2
PISA_SCHEDULE_SPLIT = 3
PISA_SCORE_LSE = 0
PISA_SCORE_MEAN = 1
PISA_SCORE_MEAN_VAR = 2

PISA_OK = 0
PISA_ERR_INVALID_ARG = -1
PISA_ERR_UNSUPPORTED = -2
PISA_ERR_WORKSPACE = -3
PISA_ERR_DEVICE = -4

EXPORTS = (
    "pisa_num_levels", "pisa_pyramid_layout", "pisa_pyramid_bytes",
    "pisa_select_workspace_bytes", "pisa_bsa_workspace_bytes", "pisa_attn_workspace_bytes",
    "pisa_build_pyramid", "pisa_pyramid_append", "pisa_cache_capacity", "pisa_cache_grow", "pisa_select", "pisa_select_static", "pisa_select_flat_bsa",
    "pisa_sparse_attn_fwd", "pisa_attn_union_min_tiles",
    "pisa_attn_bwd_workspace_bytes", "pisa_sparse_attn_bwd",
    "pisa_quality_workspace_bytes", "pisa_selection_quality",
    "pisa_profile_enable", "pisa_profile_report", "pisa_status_string", "pisa_last_error",
)


class PisaError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        super().__init__(f"{where} failed with status {status}: {detail}")
        self.status = status


class Problem(ctypes.Structure):
    """Mirror of ``pisa_problem``."""
    _fields_ = [(n, ctypes.c_int32) for n in
                ("B", "H", "Hkv", "Nq", "N", "d", "C", "fanout", "K", "causal", "dtype", "schedule", "Ncap",
                 "score")]

    def __repr__(self):
        return "Problem(" + ", ".join(f"{n}={getattr(self, n)}" for n, _ in self._fields_) + ")"


def make_problem(B, H, Hkv, Nq, N, d, C, fanout, K, causal=1, dtype="bf16", schedule=PISA_SCHEDULE_AUTO, Ncap=0,
                 score=0):
    """A pisa_problem; Ncap > N reserves rows of k, v and the pyramid for a growing N;
    score picks the selection's block score (PISA_SCORE_LSE / _MEAN / _MEAN_VAR)."""
    dt = {"bf16": PISA_DTYPE_BF16, "f32": PISA_DTYPE_F32,
          torch.bfloat16: PISA_DTYPE_BF16, torch.float32: PISA_DTYPE_F32}[dtype]
    return Problem(B, H, Hkv, Nq, N, d, C, fanout, K, int(causal), dt, schedule, Ncap, score)


def _load():
    if not os.path.exists(_LIB_PATH):
        raise ImportError(f"{_LIB_PATH} is missing: build it with `python -m paper_2609_31093_amd.build`")
    lib = ctypes.CDLL(_LIB_PATH)
    P = ctypes.POINTER(Problem)
    vp, sz, i32 = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int32
    sig = {
        "pisa_num_levels": (ctypes.c_int, [i32, i32, i32]),
        "pisa_pyramid_layout": (ctypes.c_int, [P, ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(ctypes.c_int64)]),
        "pisa_pyramid_bytes": (sz, [P]),
        "pisa_select_workspace_bytes": (sz, [P]),
        "pisa_bsa_workspace_bytes": (sz, [P]),
        "pisa_attn_workspace_bytes": (sz, [P]),
        "pisa_build_pyramid": (ctypes.c_int, [P, vp, vp, vp]),
        "pisa_pyramid_append": (ctypes.c_int, [P, vp, vp, i32, vp]),
        "pisa_cache_capacity": (ctypes.c_int32, [i32, i32, i32]),
        "pisa_cache_grow": (ctypes.c_int, [P, i32, vp, vp, vp, vp, vp, vp, vp]),
        "pisa_select": (ctypes.c_int, [P, vp, vp, vp, vp, vp, vp, sz, vp]),
        "pisa_select_static": (ctypes.c_int, [P, vp, vp, vp, vp, vp, vp]),
        "pisa_select_flat_bsa": (ctypes.c_int, [P, vp, vp, vp, vp, sz, vp]),
        "pisa_sparse_attn_fwd": (ctypes.c_int, [P, vp, vp, vp, vp, vp, vp, vp, sz, vp]),
        "pisa_attn_union_min_tiles": (ctypes.c_int, [i32]),
        "pisa_attn_bwd_workspace_bytes": (sz, [P]),
        "pisa_sparse_attn_bwd": (ctypes.c_int, [P, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]),
        "pisa_quality_workspace_bytes": (sz, [P, i32]),
        "pisa_selection_quality": (ctypes.c_int, [P, vp, vp, vp, vp, i32, vp, vp, vp, sz, vp]),
        "pisa_profile_enable": (ctypes.c_int, [ctypes.c_int]),
        "pisa_profile_report": (ctypes.c_int, [ctypes.c_char_p, sz]),
        "pisa_status_string": (ctypes.c_char_p, [ctypes.c_int]),
        "pisa_last_error": (ctypes.c_char_p, []),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


_lib = _load()


def library():
    """The loaded ctypes.CDLL (its path is ``library()._name``)."""
    return _lib


def _ptr(x):
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(stream):
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _check(status: int, where: str):
    if status != PISA_OK:
        raise PisaError(status, where, _lib.pisa_last_error().decode())
    return status


# ------------------------------------------------------------ C entry points ---

def pisa_num_levels(N: int, C: int, fanout: int) -> int:
    L = _lib.pisa_num_levels(N, C, fanout)
    return _check(L, "pisa_num_levels") if L < 0 else L


def pisa_pyramid_layout(p: Problem):
    offs = (ctypes.c_int64 * 64)()
    R = ctypes.c_int64()
    L = _lib.pisa_pyramid_layout(ctypes.byref(p), offs, ctypes.byref(R))
    if L < 0:
        _check(L, "pisa_pyramid_layout")
    return [offs[i] for i in range(L)], R.value


def pisa_pyramid_bytes(p: Problem) -> int:
    return _lib.pisa_pyramid_bytes(ctypes.byref(p))


def pisa_select_workspace_bytes(p: Problem) -> int:
    return _lib.pisa_select_workspace_bytes(ctypes.byref(p))


def pisa_bsa_workspace_bytes(p: Problem) -> int:
    return _lib.pisa_bsa_workspace_bytes(ctypes.byref(p))


def pisa_attn_workspace_bytes(p: Problem) -> int:
    return _lib.pisa_attn_workspace_bytes(ctypes.byref(p))


def pisa_build_pyramid(p: Problem, k, pyramid, stream=None) -> int:
    return _check(_lib.pisa_build_pyramid(ctypes.byref(p), _ptr(k), _ptr(pyramid), _stream(stream)),
                  "pisa_build_pyramid")


def pisa_pyramid_append(p: Problem, k, pyramid, n_old: int, stream=None) -> int:
    return _check(_lib.pisa_pyramid_append(ctypes.byref(p), _ptr(k), _ptr(pyramid), n_old, _stream(stream)),
                  "pisa_pyramid_append")


def pisa_cache_capacity(cap: int, need: int, C: int) -> int:
    r = _lib.pisa_cache_capacity(cap, need, C)
    return _check(r, "pisa_cache_capacity") if r < 0 else r


def pisa_cache_grow(p: Problem, new_cap: int, pyr_old, pyr_new, k_old=None, k_new=None, v_old=None, v_new=None,
                    stream=None) -> int:
    return _check(_lib.pisa_cache_grow(ctypes.byref(p), new_cap, _ptr(pyr_old), _ptr(pyr_new), _ptr(k_old), _ptr(k_new),
                                       _ptr(v_old), _ptr(v_new), _stream(stream)), "pisa_cache_grow")


def pisa_select(p: Problem, q, k, pyramid, block_idx, block_score=None, ws=None, ws_bytes=0, stream=None) -> int:
    return _check(_lib.pisa_select(ctypes.byref(p), _ptr(q), _ptr(k), _ptr(pyramid), _ptr(block_idx),
                                   _ptr(block_score), _ptr(ws), ws_bytes, _stream(stream)), "pisa_select")


def pisa_select_static(p: Problem, q, k, pyramid, block_idx, block_score=None, stream=None) -> int:
    return _check(_lib.pisa_select_static(ctypes.byref(p), _ptr(q), _ptr(k), _ptr(pyramid), _ptr(block_idx),
                                          _ptr(block_score), _stream(stream)), "pisa_select_static")


PISA_STATIC_SCRATCH_BYTES = 32 << 20  # include/pisa.h


def pisa_select_flat_bsa(p: Problem, q, pyramid, block_idx, ws=None, ws_bytes=0, stream=None) -> int:
    return _check(_lib.pisa_select_flat_bsa(ctypes.byref(p), _ptr(q), _ptr(pyramid), _ptr(block_idx),
                                            _ptr(ws), ws_bytes, _stream(stream)), "pisa_select_flat_bsa")


def pisa_sparse_attn_fwd(p: Problem, q, k, v, block_idx, o, lse=None, ws=None, ws_bytes=0, stream=None) -> int:
    return _check(_lib.pisa_sparse_attn_fwd(ctypes.byref(p), _ptr(q), _ptr(k), _ptr(v), _ptr(block_idx),
                                            _ptr(o), _ptr(lse), _ptr(ws), ws_bytes, _stream(stream)),
                  "pisa_sparse_attn_fwd")


def pisa_attn_bwd_workspace_bytes(p: Problem) -> int:
    return _lib.pisa_attn_bwd_workspace_bytes(ctypes.byref(p))


def pisa_sparse_attn_bwd(p: Problem, q, k, v, block_idx, o, lse, d_o, dq, dk, dv, ws=None, ws_bytes=0,
                         stream=None) -> int:
    return _check(_lib.pisa_sparse_attn_bwd(ctypes.byref(p), _ptr(q), _ptr(k), _ptr(v), _ptr(block_idx), _ptr(o),
                                            _ptr(lse), _ptr(d_o), _ptr(dq), _ptr(dk), _ptr(dv), _ptr(ws), ws_bytes,
                                            _stream(stream)), "pisa_sparse_attn_bwd")


def pisa_quality_workspace_bytes(p: Problem, n_rows: int) -> int:
    return _lib.pisa_quality_workspace_bytes(ctypes.byref(p), n_rows)


def pisa_selection_quality(p: Problem, q, k, block_idx, rows, n_rows: int, metrics, ref_idx=None, ws=None,
                           ws_bytes=0, stream=None) -> int:
    return _check(_lib.pisa_selection_quality(ctypes.byref(p), _ptr(q), _ptr(k), _ptr(block_idx), _ptr(rows), n_rows,
                                              _ptr(metrics), _ptr(ref_idx), _ptr(ws), ws_bytes, _stream(stream)),
                  "pisa_selection_quality")


def pisa_attn_union_min_tiles(n: int) -> int:
    """Sets the row-tile union threshold of pisa_sparse_attn_fwd (n < 0: off); returns the previous one."""
    return _lib.pisa_attn_union_min_tiles(int(n))


def pisa_profile_enable(on: bool) -> int:
    return _lib.pisa_profile_enable(1 if on else 0)


def pisa_profile_report() -> dict:
    """{kernel: (launches, total_ms)} since the last report (waits for the events)."""
    cap = 1 << 16
    buf = ctypes.create_string_buffer(cap)
    _lib.pisa_profile_report(buf, cap)
    out = {}
    for line in buf.value.decode().splitlines():
        name, cnt, ms = line.split()
        out[name] = (int(cnt), float(ms))
    return out


def pisa_status_string(status: int) -> str:
    return _lib.pisa_status_string(status).decode()


def pisa_last_error() -> str:
    return _lib.pisa_last_error().decode()


# ----------------------------------------------- allocation-side conveniences ---

def _workspace(nbytes: int, device):
    if nbytes == 0:
        return None
    return torch.empty(nbytes, dtype=torch.uint8, device=device)


def build_pyramid(p: Problem, k, stream=None):
    """Allocate [B, Hkv, R, d] float32 and fill it with pisa_build_pyramid."""
    _, R = pisa_pyramid_layout(p)
    pyr = torch.empty((p.B, p.Hkv, R, p.d), dtype=torch.float32, device=k.device)
    pisa_build_pyramid(p, k, pyr, stream)
    return pyr


def grow_cache(p: Problem, new_cap: int, pyramid, k=None, v=None, stream=None):
    """Allocate buffers for new_cap tokens and move the cache of problem p into
    them with pisa_cache_grow.  Returns (problem with Ncap = new_cap, pyramid,
    k, v); k and v are None when not given."""
    pn = Problem(*[getattr(p, n) for n, _ in Problem._fields_])
    pn.Ncap = new_cap
    _, R = pisa_pyramid_layout(pn)
    pyr = torch.empty((p.B, p.Hkv, R, p.d), dtype=torch.float32, device=pyramid.device)
    kn = vn = None
    if k is not None:
        kn = torch.empty((p.B, p.Hkv, new_cap, p.d), dtype=k.dtype, device=k.device)
        vn = torch.empty((p.B, p.Hkv, new_cap, p.d), dtype=v.dtype, device=v.device)
    pisa_cache_grow(p, new_cap, pyramid, pyr, k, kn, v, vn, stream)
    return pn, pyr, kn, vn


def select(p: Problem, q, k, pyramid, with_score=False, stream=None):
    """Allocate outputs and workspace, run pisa_select; returns idx (and scores)."""
    idx = torch.empty((p.B, p.Hkv, p.Nq, p.K), dtype=torch.int32, device=q.device)
    sc = torch.empty((p.B, p.Hkv, p.Nq, p.K), dtype=torch.float32, device=q.device) if with_score else None
    nb = pisa_select_workspace_bytes(p)
    ws = _workspace(nb, q.device)
    pisa_select(p, q, k, pyramid, idx, sc, ws, nb, stream)
    return (idx, sc) if with_score else idx


def select_flat_bsa(p: Problem, q, pyramid, stream=None):
    idx = torch.empty((p.B, p.Hkv, p.Nq, p.K), dtype=torch.int32, device=q.device)
    nb = pisa_bsa_workspace_bytes(p)
    pisa_select_flat_bsa(p, q, pyramid, idx, _workspace(nb, q.device), nb, stream)
    return idx


def sparse_attn_fwd(p: Problem, q, k, v, block_idx, stream=None):
    o = torch.empty_like(q)
    lse = torch.empty((p.B, p.H, p.Nq), dtype=torch.float32, device=q.device)
    nb = pisa_attn_workspace_bytes(p)
    pisa_sparse_attn_fwd(p, q, k, v, block_idx, o, lse, _workspace(nb, q.device), nb, stream)
    return o, lse


def selection_quality(p: Problem, q, k, block_idx, rows, stream=None):
    """Allocate outputs and workspace, run pisa_selection_quality on the listed
    rows (a device int32 tensor); returns (metrics [B,Hkv,n,3], ref [B,Hkv,n,K])."""
    n = int(rows.numel())
    met = torch.empty((p.B, p.Hkv, n, 3), dtype=torch.float32, device=q.device)
    ref = torch.empty((p.B, p.Hkv, n, p.K), dtype=torch.int32, device=q.device)
    nb = pisa_quality_workspace_bytes(p, n)
    pisa_selection_quality(p, q, k, block_idx, rows, n, met, ref, _workspace(nb, q.device), nb, stream)
    return met, ref


def sparse_attn_bwd(p: Problem, q, k, v, block_idx, o, lse, d_o, stream=None):
    """Allocate gradients and workspace, run pisa_sparse_attn_bwd; returns (dq, dk, dv)."""
    dq = torch.empty_like(q)
    dk = torch.empty_like(k)
    dv = torch.empty_like(v)
    nb = pisa_attn_bwd_workspace_bytes(p)
    pisa_sparse_attn_bwd(p, q, k, v, block_idx, o, lse, d_o, dq, dk, dv, _workspace(nb, q.device), nb, stream)
    return dq, dk, dv
