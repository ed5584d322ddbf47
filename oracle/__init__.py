"""fp64 CPU oracle of spliced single-query GQA decode attention.

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, ``__graft_entry__.smoke()``
and the CPU-baseline leg of ``bench.py``; the GPU library never uses it.

The arithmetic lives in ``splice_oracle.c`` (plain C, IEEE double), which
follows the paper's definition of the splice intervention (Section 3 and
Algorithm 1) and of softmax attention; this module only loads it and
marshals numpy arrays.  Inputs are the exact stored bits: bf16 tensors are
passed as uint16 arrays, f32 tensors as float32 arrays.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence, Tuple

import numpy as np

from .build import LIB
from .build import build as build_library

_lib = None


class OracleShape(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "n_cells", "n_q_heads", "n_kv_heads", "head_dim", "prompt_len", "span_lo",
        "span_hi", "gen_capacity", "donor_zero", "elem_bytes")]


class OracleCall(ctypes.Structure):
    _fields_ = [("layer", ctypes.c_int32), ("step", ctypes.c_int32),
                ("window", ctypes.c_int32), ("scale", ctypes.c_double)]


SRC_CLEAN, SRC_DONOR, SRC_ZERO, SRC_GEN = 0, 1, 2, 3


def load(path: str = LIB):
    global _lib
    if _lib is not None and path == LIB:
        return _lib
    if not os.path.exists(path):
        build_library()
    lib = ctypes.CDLL(path)
    vp, i32p = ctypes.c_void_p, ctypes.POINTER(ctypes.c_int32)
    lib.oracle_spliced.argtypes = [ctypes.c_int] * 4
    lib.oracle_spliced.restype = ctypes.c_int
    lib.oracle_visible_len.argtypes = [ctypes.POINTER(OracleShape), ctypes.c_int, ctypes.c_int]
    lib.oracle_visible_len.restype = ctypes.c_int
    lib.oracle_gather.argtypes = [ctypes.POINTER(OracleShape), ctypes.POINTER(OracleCall), i32p,
                                  vp, vp, vp, vp, vp, vp, vp, vp, vp]
    lib.oracle_gather.restype = ctypes.c_int
    lib.oracle_attn.argtypes = [ctypes.POINTER(OracleShape), ctypes.POINTER(OracleCall), i32p,
                                vp, vp, vp, vp, vp, vp, vp, i32p, ctypes.c_int,
                                vp, vp, ctypes.c_int]
    lib.oracle_attn.restype = ctypes.c_int
    lib.oracle_max_threads.restype = ctypes.c_int
    if path == LIB:
        _lib = lib
    return lib


def make_shape(n_cells, n_q_heads, n_kv_heads, head_dim, prompt_len, span, gen_capacity,
               donor_zero: bool, elem_bytes: int) -> OracleShape:
    return OracleShape(n_cells, n_q_heads, n_kv_heads, head_dim, prompt_len, span[0], span[1],
                       gen_capacity, 1 if donor_zero else 0, elem_bytes)


def shape_of(w, n_cells: Optional[int] = None, gen_capacity: Optional[int] = None) -> OracleShape:
    """Oracle shape for a ``workloads.Workload``."""
    return make_shape(w.n_cells if n_cells is None else n_cells, w.n_q_heads, w.n_kv_heads,
                      w.head_dim, w.prompt_len, w.span,
                      w.n_steps if gen_capacity is None else gen_capacity,
                      w.donor == "zero", w.elem_bytes)


def _ptr(a: Optional[np.ndarray]):
    if a is None:
        return None
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(ctypes.c_void_p)


def _i32(a: np.ndarray):
    a = np.ascontiguousarray(a, dtype=np.int32)
    return a, a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))


def spliced(layer: int, step: int, L: int, W: int, lib=None) -> bool:
    return bool((lib or load()).oracle_spliced(layer, step, L, W))


def visible_len(shape: OracleShape, step: int, window: int, lib=None) -> int:
    return (lib or load()).oracle_visible_len(ctypes.byref(shape), step, window)


def gather(shape: OracleShape, layer: int, step: int, window: int, cell_lw: np.ndarray,
           clean_k, clean_v, donor_k, donor_v, gen_k, gen_v, lib=None
           ) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Materialised visible K, V [C][Hkv][n_vis][D] (stored bits) and source map [C][n_vis]."""
    lib = lib or load()
    call = OracleCall(layer, step, window, 0.0)
    n_vis = visible_len(shape, step, window, lib)
    dt = clean_k.dtype
    ok = np.empty((shape.n_cells, shape.n_kv_heads, n_vis, shape.head_dim), dtype=dt)
    ov = np.empty_like(ok)
    src = np.empty((shape.n_cells, n_vis), dtype=np.uint8)
    lw, lwp = _i32(cell_lw)
    rc = lib.oracle_gather(ctypes.byref(shape), ctypes.byref(call), lwp,
                           _ptr(clean_k), _ptr(clean_v), _ptr(donor_k), _ptr(donor_v),
                           _ptr(gen_k), _ptr(gen_v), _ptr(ok), _ptr(ov),
                           src.ctypes.data_as(ctypes.c_void_p))
    if rc != 0:
        raise RuntimeError(f"oracle_gather failed: {rc}")
    return ok, ov, src


def attn(shape: OracleShape, layer: int, step: int, window: int, scale: float,
         cell_lw: np.ndarray, q, clean_k, clean_v, donor_k, donor_v, gen_k, gen_v,
         rows: Optional[Sequence[Tuple[int, int]]] = None, n_threads: int = 0, lib=None
         ) -> Tuple[np.ndarray, np.ndarray]:
    """fp64 attention.  Without ``rows``: out [C][Hq][D], lse [C][Hq].
    With ``rows`` (a list of (c, h)): out [n][D], lse [n]."""
    lib = lib or load()
    call = OracleCall(layer, step, window, float(scale))
    lw, lwp = _i32(cell_lw)
    if rows is None:
        n = shape.n_cells * shape.n_q_heads
        rp = None
    else:
        ra, rp = _i32(np.asarray(rows, dtype=np.int32).reshape(-1, 2))
        n = ra.shape[0]
    out = np.empty((n, shape.head_dim), dtype=np.float64)
    lse = np.empty((n,), dtype=np.float64)
    rc = lib.oracle_attn(ctypes.byref(shape), ctypes.byref(call), lwp, _ptr(q),
                         _ptr(clean_k), _ptr(clean_v), _ptr(donor_k), _ptr(donor_v),
                         _ptr(gen_k), _ptr(gen_v), rp, n,
                         out.ctypes.data_as(ctypes.c_void_p), lse.ctypes.data_as(ctypes.c_void_p),
                         int(n_threads))
    if rc != 0:
        raise RuntimeError(f"oracle_attn failed: {rc}")
    if rows is None:
        return (out.reshape(shape.n_cells, shape.n_q_heads, shape.head_dim),
                lse.reshape(shape.n_cells, shape.n_q_heads))
    return out, lse


def max_threads(lib=None) -> int:
    return (lib or load()).oracle_max_threads()
