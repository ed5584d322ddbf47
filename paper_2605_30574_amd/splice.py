"""Python binding of the C ABI in include/splice_attn.h (ctypes).

Argument marshalling only: every step of the computation runs in the HIP
library.  Functions have the C names.  Tensor arguments are torch tensors
on the GPU; before calling into C the binding checks each tensor's device,
dtype, contiguity and element count against the shape, so that no call can
make a kernel read or write outside a buffer.  A negative status from C
raises SpliceError.  The library must be built
(``python -m paper_2605_30574_amd.build``); there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libsplice_attn.so")

SPLICE_OK, SPLICE_EINVAL, SPLICE_ESHAPE, SPLICE_EWORKSPACE, SPLICE_EUNSUPPORTED, SPLICE_EHIP = 0, -1, -2, -3, -4, -5
SPLICE_DONOR_BUFFER, SPLICE_DONOR_ZERO = 0, 1
SPLICE_BF16, SPLICE_F32 = 0, 1
SPLICE_SRC_CLEAN, SPLICE_SRC_DONOR, SPLICE_SRC_ZERO, SPLICE_SRC_GEN = 0, 1, 2, 3
SPLICE_MAX_CELLS = 256
SPLICE_ABI_VERSION = 6   # layout of SpliceShape / SpliceCall below

EXPORTS = ("splice_abi_version", "splice_status_str", "splice_visible_len", "splice_kv_build",
           "splice_decode_attn_workspace_bytes", "splice_workspace_init", "splice_decode_attn",
           "splice_decode_step", "splice_decode_forked", "splice_workspace_handovers",
           "splice_decode_attn_noalloc")
SPLICE_NOALLOC_WORKSPACE_BYTES = 32 << 20


class SpliceShape(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "n_cells", "n_layers", "n_q_heads", "n_kv_heads", "head_dim", "prompt_len",
        "span_lo", "span_hi", "gen_capacity", "donor_kind", "dtype")]


class SpliceCall(ctypes.Structure):
    _fields_ = [("layer", ctypes.c_int32), ("step", ctypes.c_int32), ("window", ctypes.c_int32),
                ("scale", ctypes.c_float), ("split_keys", ctypes.c_int32), ("merge_wait", ctypes.c_int32)]


class SpliceError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {status_name(status)} ({status})")


_lib = None


def load_library(path: str = LIB_PATH):
    """Load libsplice_attn.so (after torch, so both share one HIP runtime)."""
    global _lib
    if _lib is not None:
        return _lib
    import torch  # noqa: F401  -- maps torch's libamdhip64 before ours resolves it
    if not os.path.exists(path):
        raise ImportError(f"{path} is not built; run `python -m paper_2605_30574_amd.build`")
    lib = ctypes.CDLL(path)
    vp, i32 = ctypes.c_void_p, ctypes.c_int32
    shp, cal = ctypes.POINTER(SpliceShape), ctypes.POINTER(SpliceCall)
    i32p = ctypes.POINTER(ctypes.c_int32)
    lib.splice_abi_version.restype = i32
    lib.splice_abi_version.argtypes = []
    lib.splice_status_str.restype = ctypes.c_char_p
    lib.splice_status_str.argtypes = [i32]
    lib.splice_visible_len.restype = i32
    lib.splice_visible_len.argtypes = [shp, cal]
    lib.splice_kv_build.restype = i32
    lib.splice_kv_build.argtypes = [shp, cal, i32p, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
    lib.splice_decode_attn_workspace_bytes.restype = ctypes.c_int64
    lib.splice_decode_attn_workspace_bytes.argtypes = [shp, cal]
    lib.splice_workspace_init.restype = i32
    lib.splice_workspace_init.argtypes = [vp, ctypes.c_size_t, vp]
    lib.splice_workspace_handovers.restype = ctypes.c_int64
    lib.splice_workspace_handovers.argtypes = [vp, ctypes.c_size_t, vp]
    lib.splice_decode_attn.restype = i32
    lib.splice_decode_attn.argtypes = [shp, cal, i32p, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                       ctypes.c_size_t, vp]
    lib.splice_decode_attn_noalloc.restype = i32
    lib.splice_decode_attn_noalloc.argtypes = [shp, cal, i32p, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
    lib.splice_decode_step.restype = i32
    lib.splice_decode_step.argtypes = [shp, cal, i32p, i32p, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                       vp, ctypes.c_size_t, vp]
    lib.splice_decode_forked.restype = i32
    lib.splice_decode_forked.argtypes = [shp, cal, i32p, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                         ctypes.c_size_t, vp]
    got = lib.splice_abi_version()
    if got != SPLICE_ABI_VERSION:
        raise ImportError(f"{path} has ABI version {got}, this binding expects {SPLICE_ABI_VERSION}: rebuild it")
    _lib = lib
    return lib


def status_name(status: int) -> str:
    try:
        return load_library().splice_status_str(int(status)).decode()
    except ImportError:
        return "unknown"


def _check(rc: int, where: str) -> int:
    if rc < 0:
        raise SpliceError(rc, where)
    return rc


# ------------------------------------------------------------------ helpers

def make_shape(n_cells: int, n_layers: int, n_q_heads: int, n_kv_heads: int, head_dim: int,
               prompt_len: int, span: Sequence[int], gen_capacity: int, donor_zero: bool,
               dtype: str) -> SpliceShape:
    return SpliceShape(n_cells, n_layers, n_q_heads, n_kv_heads, head_dim, prompt_len,
                       int(span[0]), int(span[1]), gen_capacity,
                       SPLICE_DONOR_ZERO if donor_zero else SPLICE_DONOR_BUFFER,
                       SPLICE_BF16 if dtype == "bf16" else SPLICE_F32)


def make_call(layer: int, step: int, window: int, scale: float, split_keys: int = 0,
              merge_wait: int = 0) -> SpliceCall:
    return SpliceCall(layer, step, window, float(scale), split_keys, merge_wait)


def _cells(cell_LW, n_cells: int):
    a = np.ascontiguousarray(np.asarray(cell_LW, dtype=np.int32).reshape(-1, 2))
    if a.shape[0] != n_cells:
        raise ValueError(f"cell_LW has {a.shape[0]} rows, shape says {n_cells} cells")
    return a, a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))


def _torch_dtype(shape: SpliceShape):
    import torch
    return torch.bfloat16 if shape.dtype == SPLICE_BF16 else torch.float32


def _dev_ptr(t, name: str, numel: int, dtype, device=None, optional: bool = False):
    """Pointer of a contiguous GPU tensor of exactly ``numel`` elements."""
    if t is None:
        if optional:
            return None, device
        raise ValueError(f"{name} is required")
    if numel == 0 and t.numel() == 0:
        return None, (t.device if device is None else device)   # empty buffer: NULL
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} has dtype {t.dtype}, expected {dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if numel is not None and t.numel() != numel:
        raise ValueError(f"{name} has {t.numel()} elements, expected {numel}")
    if device is not None and t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")
    return ctypes.c_void_p(t.data_ptr()), t.device


def _stream_ptr(stream, device):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream(device)
    if isinstance(stream, int):
        return ctypes.c_void_p(stream)
    return ctypes.c_void_p(stream.cuda_stream)


def _donors(shape: SpliceShape, donor_k, donor_v, dt, n_prompt, dev):
    if shape.donor_kind == SPLICE_DONOR_ZERO:
        if donor_k is not None or donor_v is not None:
            raise ValueError("the ZERO donor takes no donor buffers")
        return None, None
    dk, _ = _dev_ptr(donor_k, "donor_k", n_prompt, dt, dev)
    dv, _ = _dev_ptr(donor_v, "donor_v", n_prompt, dt, dev)
    return dk, dv


# ------------------------------------------------------------------ C entry points

def splice_abi_version() -> int:
    return load_library().splice_abi_version()


def splice_status_str(status: int) -> str:
    return load_library().splice_status_str(int(status)).decode()


def splice_visible_len(shape: SpliceShape, call: SpliceCall) -> int:
    return _check(load_library().splice_visible_len(ctypes.byref(shape), ctypes.byref(call)),
                  "splice_visible_len")


def splice_decode_attn_workspace_bytes(shape: SpliceShape, call: Optional[SpliceCall] = None) -> int:
    lib = load_library()
    return _check(lib.splice_decode_attn_workspace_bytes(
        ctypes.byref(shape), ctypes.byref(call) if call is not None else None),
        "splice_decode_attn_workspace_bytes")


def splice_workspace_init(workspace, stream=None) -> None:
    p, dev = _dev_ptr(workspace, "workspace", None, None)
    nbytes = workspace.numel() * workspace.element_size()
    _check(load_library().splice_workspace_init(p, nbytes, _stream_ptr(stream, dev)), "splice_workspace_init")


def splice_workspace_handovers(workspace, stream=None) -> int:
    """Merges handed over since the workspace was initialised (synchronises ``stream``)."""
    p, dev = _dev_ptr(workspace, "workspace", None, None)
    nbytes = workspace.numel() * workspace.element_size()
    return _check(load_library().splice_workspace_handovers(p, nbytes, _stream_ptr(stream, dev)),
                  "splice_workspace_handovers")


def new_workspace(shape: SpliceShape, call: Optional[SpliceCall] = None, device="cuda", stream=None):
    """Allocate (torch) and prepare a workspace for ``shape`` (and ``call``)."""
    import torch
    nbytes = splice_decode_attn_workspace_bytes(shape, call)
    ws = torch.empty(max(256, (nbytes + 255) // 256 * 256), dtype=torch.uint8, device=device)
    splice_workspace_init(ws, stream)
    return ws


def splice_kv_build(shape: SpliceShape, call: SpliceCall, cell_LW, clean_k, clean_v, donor_k, donor_v,
                    gen_k, gen_v, out_k, out_v, out_src, stream=None) -> None:
    import torch
    lib = load_library()
    C, Hkv, D = shape.n_cells, shape.n_kv_heads, shape.head_dim
    n_vis = splice_visible_len(shape, call)
    dt = _torch_dtype(shape)
    n_prompt = Hkv * shape.prompt_len * D
    ck, dev = _dev_ptr(clean_k, "clean_k", n_prompt, dt)
    cv, _ = _dev_ptr(clean_v, "clean_v", n_prompt, dt, dev)
    dk, dv = _donors(shape, donor_k, donor_v, dt, n_prompt, dev)
    gk, _ = _dev_ptr(gen_k, "gen_k", C * Hkv * shape.gen_capacity * D, dt, dev)
    gv, _ = _dev_ptr(gen_v, "gen_v", C * Hkv * shape.gen_capacity * D, dt, dev)
    ok, _ = _dev_ptr(out_k, "out_k", C * Hkv * n_vis * D, dt, dev)
    ov, _ = _dev_ptr(out_v, "out_v", C * Hkv * n_vis * D, dt, dev)
    os_, _ = _dev_ptr(out_src, "out_src", C * n_vis, torch.uint8, dev)
    lw, lwp = _cells(cell_LW, C)
    _check(lib.splice_kv_build(ctypes.byref(shape), ctypes.byref(call), lwp, ck, cv, dk, dv, gk, gv,
                               ok, ov, os_, _stream_ptr(stream, dev)), "splice_kv_build")


def splice_decode_attn(shape: SpliceShape, call: SpliceCall, cell_LW, q, clean_k, clean_v, donor_k,
                       donor_v, gen_k, gen_v, out, lse, workspace, stream=None) -> None:
    import torch
    lib = load_library()
    C, Hq, Hkv, D = shape.n_cells, shape.n_q_heads, shape.n_kv_heads, shape.head_dim
    dt = _torch_dtype(shape)
    n_prompt = Hkv * shape.prompt_len * D
    qp, dev = _dev_ptr(q, "q", C * Hq * D, dt)
    ck, _ = _dev_ptr(clean_k, "clean_k", n_prompt, dt, dev)
    cv, _ = _dev_ptr(clean_v, "clean_v", n_prompt, dt, dev)
    dk, dv = _donors(shape, donor_k, donor_v, dt, n_prompt, dev)
    gk, _ = _dev_ptr(gen_k, "gen_k", C * Hkv * shape.gen_capacity * D, dt, dev)
    gv, _ = _dev_ptr(gen_v, "gen_v", C * Hkv * shape.gen_capacity * D, dt, dev)
    op, _ = _dev_ptr(out, "out", C * Hq * D, torch.float32, dev)
    lp, _ = _dev_ptr(lse, "lse", C * Hq, torch.float32, dev)
    wp, _ = _dev_ptr(workspace, "workspace", None, None, dev)
    wbytes = workspace.numel() * workspace.element_size()
    lw, lwp = _cells(cell_LW, C)
    _check(lib.splice_decode_attn(ctypes.byref(shape), ctypes.byref(call), lwp, qp, ck, cv, dk, dv, gk, gv,
                                  op, lp, wp, wbytes, _stream_ptr(stream, dev)), "splice_decode_attn")


def splice_decode_attn_noalloc(shape: SpliceShape, call: SpliceCall, cell_LW, q, clean_k, clean_v, donor_k,
                               donor_v, gen_k, gen_v, out, lse, stream=None) -> None:
    """splice_decode_attn with the library's own per-GPU workspace array
    (no workspace argument, nothing allocated)."""
    import torch
    lib = load_library()
    C, Hq, Hkv, D = shape.n_cells, shape.n_q_heads, shape.n_kv_heads, shape.head_dim
    dt = _torch_dtype(shape)
    n_prompt = Hkv * shape.prompt_len * D
    qp, dev = _dev_ptr(q, "q", C * Hq * D, dt)
    ck, _ = _dev_ptr(clean_k, "clean_k", n_prompt, dt, dev)
    cv, _ = _dev_ptr(clean_v, "clean_v", n_prompt, dt, dev)
    dk, dv = _donors(shape, donor_k, donor_v, dt, n_prompt, dev)
    gk, _ = _dev_ptr(gen_k, "gen_k", C * Hkv * shape.gen_capacity * D, dt, dev)
    gv, _ = _dev_ptr(gen_v, "gen_v", C * Hkv * shape.gen_capacity * D, dt, dev)
    op, _ = _dev_ptr(out, "out", C * Hq * D, torch.float32, dev)
    lp, _ = _dev_ptr(lse, "lse", C * Hq, torch.float32, dev)
    lw, lwp = _cells(cell_LW, C)
    _check(lib.splice_decode_attn_noalloc(ctypes.byref(shape), ctypes.byref(call), lwp, qp, ck, cv, dk, dv, gk, gv,
                                          op, lp, _stream_ptr(stream, dev)), "splice_decode_attn_noalloc")


def _steps(cell_step, n_cells: int):
    a = np.ascontiguousarray(np.asarray(cell_step, dtype=np.int32).reshape(-1))
    if a.shape[0] != n_cells:
        raise ValueError(f"cell_step has {a.shape[0]} entries, shape says {n_cells} cells")
    return a, a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))


def splice_decode_step(shape: SpliceShape, call: SpliceCall, cell_LW, cell_step, q, k_new, v_new, clean_k,
                       clean_v, donor_k, donor_v, gen_k, gen_v, out, lse, workspace, stream=None) -> None:
    """One decode pass with each cell at its own step ``cell_step[c]`` (< 0: finished).

    Appends ``k_new[c]``, ``v_new[c]`` ([C, Hkv, D]) as row ``cell_step[c]`` of the
    cell's generated caches, then attends as ``splice_decode_attn`` at that step.
    """
    import torch
    lib = load_library()
    C, Hq, Hkv, D = shape.n_cells, shape.n_q_heads, shape.n_kv_heads, shape.head_dim
    dt = _torch_dtype(shape)
    n_prompt = Hkv * shape.prompt_len * D
    qp, dev = _dev_ptr(q, "q", C * Hq * D, dt)
    kn, _ = _dev_ptr(k_new, "k_new", C * Hkv * D, dt, dev)
    vn, _ = _dev_ptr(v_new, "v_new", C * Hkv * D, dt, dev)
    ck, _ = _dev_ptr(clean_k, "clean_k", n_prompt, dt, dev)
    cv, _ = _dev_ptr(clean_v, "clean_v", n_prompt, dt, dev)
    dk, dv = _donors(shape, donor_k, donor_v, dt, n_prompt, dev)
    gk, _ = _dev_ptr(gen_k, "gen_k", C * Hkv * shape.gen_capacity * D, dt, dev)
    gv, _ = _dev_ptr(gen_v, "gen_v", C * Hkv * shape.gen_capacity * D, dt, dev)
    op, _ = _dev_ptr(out, "out", C * Hq * D, torch.float32, dev)
    lp, _ = _dev_ptr(lse, "lse", C * Hq, torch.float32, dev)
    wp, _ = _dev_ptr(workspace, "workspace", None, None, dev)
    wbytes = workspace.numel() * workspace.element_size()
    lw, lwp = _cells(cell_LW, C)
    st, stp = _steps(cell_step, C)
    _check(lib.splice_decode_step(ctypes.byref(shape), ctypes.byref(call), lwp, stp, qp, kn, vn, ck, cv, dk, dv,
                                  gk, gv, op, lp, wp, wbytes, _stream_ptr(stream, dev)), "splice_decode_step")


def splice_decode_forked(shape: SpliceShape, call: SpliceCall, cell_LW, trunk: int, q, clean_k, clean_v,
                         donor_k, donor_v, gen_k, gen_v, out, lse, workspace, stream=None) -> None:
    """Attention of a forked sweep: cell ``trunk`` is the clean run; a cell that
    has diverged reads its generated rows below its onset W from the trunk, and
    a cell that has not takes the trunk's out and lse."""
    import torch
    lib = load_library()
    C, Hq, Hkv, D = shape.n_cells, shape.n_q_heads, shape.n_kv_heads, shape.head_dim
    dt = _torch_dtype(shape)
    n_prompt = Hkv * shape.prompt_len * D
    qp, dev = _dev_ptr(q, "q", C * Hq * D, dt)
    ck, _ = _dev_ptr(clean_k, "clean_k", n_prompt, dt, dev)
    cv, _ = _dev_ptr(clean_v, "clean_v", n_prompt, dt, dev)
    dk, dv = _donors(shape, donor_k, donor_v, dt, n_prompt, dev)
    gk, _ = _dev_ptr(gen_k, "gen_k", C * Hkv * shape.gen_capacity * D, dt, dev)
    gv, _ = _dev_ptr(gen_v, "gen_v", C * Hkv * shape.gen_capacity * D, dt, dev)
    op, _ = _dev_ptr(out, "out", C * Hq * D, torch.float32, dev)
    lp, _ = _dev_ptr(lse, "lse", C * Hq, torch.float32, dev)
    wp, _ = _dev_ptr(workspace, "workspace", None, None, dev)
    wbytes = workspace.numel() * workspace.element_size()
    lw, lwp = _cells(cell_LW, C)
    _check(lib.splice_decode_forked(ctypes.byref(shape), ctypes.byref(call), lwp, int(trunk), qp, ck, cv, dk, dv,
                                    gk, gv, op, lp, wp, wbytes, _stream_ptr(stream, dev)), "splice_decode_forked")
