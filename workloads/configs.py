"""Synthetic sweep workloads shaped like the paper's four models.

The paper evaluates Qwen3-4B, Gemma-3-4B-IT, Qwen3-8B and Llama-3-8B-Instruct
(Section 2, "Models and Datasets") and sweeps a grid of layer cutoffs L and
splice onsets W (Section 3, "Sweep and reporting").  Neither the weights nor
the datasets are used here: each workload below reproduces only the attention
shapes of one model plus a prompt layout, a donor form (Table 1) and a cell
grid.  Every tensor is synthetic and seeded (see ``workloads.inputs``).

Readings for details the paper leaves open:
  * span placement for the Llama/Gemma/Qwen3-8B shapes: prefix =
    round(2/3 of the non-span tokens), suffix = the rest;
  * the Llama shape folds the 1/sqrt(128) softmax scale into K, so its
    attention scale is 1.0;
  * Gemma local layers (l mod 6 != 5) use a 1024-token sliding window,
    global layers see every key;
  * the sink outlier sits at prompt position 0, channels 0..3 of K, x50.
This module holds shapes and grids only: no part of the attention or of the
splice arithmetic.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List, Optional, Tuple

DONOR_ZERO = "zero"      # Table 1: all-zero K, V at every patched layer
DONOR_BLANK = "blank"    # Table 1: scaffold kept, user content replaced
DONOR_DIFF = "diff"      # Table 1: diff-family donor (independent content)


@dataclass(frozen=True)
class Workload:
    name: str
    index: int
    n_layers: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    prompt_len: int
    span: Tuple[int, int]
    n_steps: int
    cells: Tuple[Tuple[int, int], ...]
    donor: str
    dtype: str                 # "f32" or "bf16": element type of q, K, V
    scale: float               # softmax scale applied to q.k
    k_prescale: float = 1.0    # factor folded into K when it is drawn
    sink: bool = False         # K[pos 0, ch 0..3] *= sink_factor
    sink_factor: float = 50.0
    local_window: int = 0      # sliding window of local layers (0: none)
    global_period: int = 0     # layer l is global iff l % period == period-1
    note: str = ""

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    @property
    def n_cells(self) -> int:
        return len(self.cells)

    @property
    def elem_bytes(self) -> int:
        return 2 if self.dtype == "bf16" else 4

    def window(self, layer: int) -> int:
        """Sliding window of ``layer``: 0 means every key is visible."""
        if self.local_window <= 0:
            return 0
        if self.global_period > 0 and layer % self.global_period == self.global_period - 1:
            return 0
        return self.local_window

    def with_(self, **kw) -> "Workload":
        d = dict(self.__dict__)
        d.update(kw)
        return Workload(**d)


def _grid(Ls, Ws, limit: Optional[int] = None):
    cells = [(L, W) for L in Ls for W in Ws]   # L-major order
    if limit is not None:
        cells = cells[:limit]
    return tuple(cells)


def _span_two_thirds(prompt_len: int, span_len: int) -> Tuple[int, int]:
    rest = prompt_len - span_len
    prefix = int(math.floor(rest * 2.0 / 3.0 + 0.5))
    return (prefix, prefix + span_len)


_W8 = (0, 1, 2, 4, 8, 16, 32, 64)

WORKLOADS: List[Workload] = [
    Workload(
        name="tiny-f32", index=0, n_layers=2, n_q_heads=4, n_kv_heads=2,
        head_dim=64, prompt_len=32, span=(4, 28), n_steps=16,
        cells=_grid((0, 1, 2), (0, 4)), donor=DONOR_ZERO, dtype="f32",
        scale=1.0 / 8.0,
        note="tiny fp32 sweep, CPU-seconds"),
    Workload(
        name="qwen3-4b", index=1, n_layers=36, n_q_heads=32, n_kv_heads=8,
        head_dim=128, prompt_len=256, span=(40, 236), n_steps=512,
        cells=_grid(range(0, 37, 4), _W8), donor=DONOR_BLANK, dtype="bf16",
        scale=1.0 / math.sqrt(128.0), sink=True,
        note="Qwen3-4B-shaped, 40-token prefix, 196-token user span"),
    Workload(
        name="llama3-8b", index=2, n_layers=32, n_q_heads=32, n_kv_heads=8,
        head_dim=128, prompt_len=1024, span=_span_two_thirds(1024, 960),
        n_steps=256, cells=_grid(range(0, 29, 4), _W8), donor=DONOR_ZERO,
        dtype="bf16", scale=1.0, k_prescale=1.0 / math.sqrt(128.0), sink=True,
        note="Llama-3-8B-shaped, K pre-scaled by 1/sqrt(128)"),
    Workload(
        name="gemma3-4b", index=3, n_layers=34, n_q_heads=8, n_kv_heads=4,
        head_dim=256, prompt_len=4096, span=_span_two_thirds(4096, 4000),
        n_steps=128, cells=_grid(range(0, 31, 6), _W8), donor=DONOR_BLANK,
        dtype="bf16", scale=1.0 / 16.0, sink=True, local_window=1024,
        global_period=6,
        note="Gemma-3-4B-shaped, 5:1 local:global, 1024-token window"),
    Workload(
        name="qwen3-8b", index=4, n_layers=36, n_q_heads=32, n_kv_heads=8,
        head_dim=128, prompt_len=8192, span=_span_two_thirds(8192, 8000),
        n_steps=1024,
        cells=_grid(range(0, 37, 3), _W8 + (128, 256), limit=128),
        donor=DONOR_DIFF, dtype="bf16", scale=1.0 / math.sqrt(128.0),
        sink=True,
        note="Qwen3-8B-shaped long context, diff-family donor"),
]

BY_NAME = {w.name: w for w in WORKLOADS}


def get(name_or_index) -> Workload:
    if isinstance(name_or_index, int):
        return WORKLOADS[name_or_index]
    return BY_NAME[name_or_index]
