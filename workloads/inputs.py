"""Seeded synthetic tensors for a workload, on any torch device.

Layouts (row-major, contiguous):
  q                 [C][Hq][D]
  clean_k, clean_v  [Hkv][T_p][D]       prefill cache of one layer
  donor_k, donor_v  [Hkv][T_p][D]       donor cache (None for the ZERO donor)
  gen_k,  gen_v     [C][Hkv][S][D]      generated-span cache of every cell

Values: N(0,1) in float32 from a seeded torch generator, K multiplied by the
workload's pre-scale, the sink outlier (prompt position 0, channels 0..3 of
K, times the sink factor) applied to clean and donor caches, then rounded to
the workload's element type (bf16 conversion is round-to-nearest-even).
Donors (Table 1 of the paper): BLANK keeps the clean prefix/suffix and
redraws the user span; the diff-family donor is an independent draw of the
whole prompt; ZERO has no buffer at all.  Generated rows are drawn for the
full capacity S once: the method never modifies a generated entry.

Nothing here computes any part of the splice or of the attention; the same
tensors feed both the oracle and the GPU library.
"""
from __future__ import annotations

from typing import Dict, Optional

import numpy as np
import torch

from .configs import DONOR_BLANK, DONOR_DIFF, DONOR_ZERO, Workload

# tensor kinds, one seed stream each
KIND_Q, KIND_CLEAN_K, KIND_CLEAN_V, KIND_DONOR_K, KIND_DONOR_V, KIND_GEN_K, KIND_GEN_V = range(7)
KIND_NEW_K, KIND_NEW_V, KIND_STEPS = 7, 8, 9


def derive_seed(base: int, workload_index: int, kind: int, layer: int, step: int = 0) -> int:
    """A 63-bit seed for one tensor, from numpy's SeedSequence."""
    ss = np.random.SeedSequence([int(base) & 0xFFFFFFFF, workload_index, kind, layer, step])
    return int(ss.generate_state(1, dtype=np.uint64)[0] & np.uint64(0x7FFFFFFFFFFFFFFF))


def _randn(shape, seed: int, device) -> torch.Tensor:
    dev = torch.device(device)
    g = torch.Generator(device=dev)
    g.manual_seed(seed)
    return torch.randn(*shape, generator=g, device=dev, dtype=torch.float32)


def torch_dtype(w: Workload):
    return torch.bfloat16 if w.dtype == "bf16" else torch.float32


def _finish_k(w: Workload, k: torch.Tensor, prompt: bool) -> torch.Tensor:
    if w.k_prescale != 1.0:
        k = k * w.k_prescale
    if prompt and w.sink and k.shape[-2] > 0:
        k[..., 0, 0:4] *= w.sink_factor
    return k


def make_layer(w: Workload, layer: int, seed: int = 0, device="cpu",
               n_cells: Optional[int] = None, gen_capacity: Optional[int] = None
               ) -> Dict[str, Optional[torch.Tensor]]:
    """Prompt caches (clean, donor) and generated caches of one layer."""
    C = w.n_cells if n_cells is None else n_cells
    S = w.n_steps if gen_capacity is None else gen_capacity
    Hkv, Tp, D = w.n_kv_heads, w.prompt_len, w.head_dim
    dt = torch_dtype(w)
    a, b = w.span

    ck = _finish_k(w, _randn((Hkv, Tp, D), derive_seed(seed, w.index, KIND_CLEAN_K, layer), device), True)
    cv = _randn((Hkv, Tp, D), derive_seed(seed, w.index, KIND_CLEAN_V, layer), device)

    dk = dv = None
    if w.donor == DONOR_BLANK:
        rk = _finish_k(w, _randn((Hkv, Tp, D), derive_seed(seed, w.index, KIND_DONOR_K, layer), device), True)
        rv = _randn((Hkv, Tp, D), derive_seed(seed, w.index, KIND_DONOR_V, layer), device)
        dk = ck.clone()
        dv = cv.clone()
        dk[:, a:b] = rk[:, a:b]
        dv[:, a:b] = rv[:, a:b]
    elif w.donor == DONOR_DIFF:
        dk = _finish_k(w, _randn((Hkv, Tp, D), derive_seed(seed, w.index, KIND_DONOR_K, layer), device), True)
        dv = _randn((Hkv, Tp, D), derive_seed(seed, w.index, KIND_DONOR_V, layer), device)
    elif w.donor != DONOR_ZERO:
        raise ValueError(f"unknown donor {w.donor!r}")

    gk = _finish_k(w, _randn((C, Hkv, S, D), derive_seed(seed, w.index, KIND_GEN_K, layer), device), False)
    gv = _randn((C, Hkv, S, D), derive_seed(seed, w.index, KIND_GEN_V, layer), device)

    out = dict(clean_k=ck, clean_v=cv, donor_k=dk, donor_v=dv, gen_k=gk, gen_v=gv)
    return {k: (None if v is None else v.to(dt).contiguous()) for k, v in out.items()}


def make_q(w: Workload, layer: int, step: int, seed: int = 0, device="cpu",
           n_cells: Optional[int] = None) -> torch.Tensor:
    C = w.n_cells if n_cells is None else n_cells
    q = _randn((C, w.n_q_heads, w.head_dim), derive_seed(seed, w.index, KIND_Q, layer, step), device)
    return q.to(torch_dtype(w)).contiguous()


def make_new_rows(w: Workload, layer: int, step: int, seed: int = 0, device="cpu",
                  n_cells: Optional[int] = None) -> Dict[str, torch.Tensor]:
    """The K, V rows [C][Hkv][D] the current token of every cell appends at one
    decode pass (drawn like generated rows)."""
    C = w.n_cells if n_cells is None else n_cells
    shp = (C, w.n_kv_heads, w.head_dim)
    kn = _finish_k(w, _randn(shp, derive_seed(seed, w.index, KIND_NEW_K, layer, step), device), False)
    vn = _randn(shp, derive_seed(seed, w.index, KIND_NEW_V, layer, step), device)
    dt = torch_dtype(w)
    return dict(k_new=kn.to(dt).contiguous(), v_new=vn.to(dt).contiguous())


def cell_steps(w: Workload, seed: int = 0, n_cells: Optional[int] = None, finished: float = 0.125,
               max_step: Optional[int] = None) -> np.ndarray:
    """int32 [C]: a mix of per-cell decode steps, as in a batch whose slots are
    refilled with new cells as others stop -- uniform in [0, max_step], about
    ``finished`` of the cells stopped (-1), and steps 0 and max_step present
    when there are at least two cells."""
    C = w.n_cells if n_cells is None else n_cells
    top = w.n_steps - 1 if max_step is None else max_step
    rng = np.random.default_rng(derive_seed(seed, w.index, KIND_STEPS, 0))
    st = rng.integers(0, top + 1, size=C).astype(np.int32)
    st[rng.random(C) < finished] = -1
    if C >= 2:
        st[0], st[C - 1] = 0, top
    return np.ascontiguousarray(st)


def cell_lw(w: Workload, cells=None) -> np.ndarray:
    """int32 [C][2] array of (L_c, W_c)."""
    cells = w.cells if cells is None else cells
    return np.ascontiguousarray(np.array(cells, dtype=np.int32).reshape(-1, 2))


def to_numpy(t: Optional[torch.Tensor]) -> Optional[np.ndarray]:
    """Host copy keeping the exact bits: bf16 -> uint16, f32 -> float32."""
    if t is None:
        return None
    t = t.detach().contiguous().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16).copy()
    return t.numpy().copy()
