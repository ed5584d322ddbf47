"""fp64 CPU reference of the greedy decode loop around the spliced attention.

TEST INFRASTRUCTURE ONLY: imported by ``tests/``; the GPU library never uses
it.  It follows Algorithm 1 of the paper: per decode step one forward pass
through every layer -- at each layer the step's K/V appended to the cell's
generated cache (as generated row s), then the attention the splice defines
(this package's fp64 oracle, ``oracle.attn``, one cell at a time) -- then the
argmax token, and a cell stops at EOS or T_max.

The model around the attention is the synthetic stand-in the paper's models
are replaced by (weights from ``workloads.model``), written out here in plain
numpy float64:
  * RMSNorm: x / sqrt(mean(x^2) + eps) * gain;
  * q, k, v = h W_q, h W_k, h W_v; rotary embedding on q and k: pairs
    (i, i + D/2) rotated by the angle pos * theta^(-2i/D), pos = T_p + s;
  * q, k, v rounded to bf16 (round to nearest even) -- the precision the
    attention and its caches are kept in;
  * x += attn W_o; x += (silu(h2 W_gate) * (h2 W_up)) W_down with h2 the
    normed x; logits = norm(x) lm_head;
  * next token: the lowest index of the maximal logit.
Only the q/k/v rounding is shared with the GPU path's precision; everything
else is float64.
"""
from __future__ import annotations

from typing import Dict, List

import numpy as np

from . import attn, make_shape


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round to float32, then to bf16 (round to nearest even): uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    r = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return r.astype(np.uint16)


def from_bf16_bits(b: np.ndarray) -> np.ndarray:
    return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def _rms_norm(x: np.ndarray, gain: np.ndarray, eps: float) -> np.ndarray:
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * gain


def _rope(x: np.ndarray, pos: np.ndarray, theta: float) -> np.ndarray:
    """x [C][H][D]: pair (i, i + D/2) rotated by pos * theta^(-2i/D)."""
    D = x.shape[-1]
    half = D // 2
    ang = pos.astype(np.float64)[:, None] * theta ** (-np.arange(half, dtype=np.float64) * 2.0 / D)[None, :]
    c, s = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
    a, b = x[..., :half], x[..., half:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def _silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


class ReferenceDecoder:
    """w: a workloads.Workload (attention shape, prompt layout, donor);
    m: a workloads.model.ModelConfig; weights: float64 numpy arrays in the
    layout of workloads.model.make_weights; prompts[l]: dict of the exact
    bits (uint16) of clean_k, clean_v, donor_k, donor_v of layer l."""

    def __init__(self, w, m, weights: Dict, prompts: List[Dict], cell_LW):
        self.w, self.m, self.wt, self.prompts = w, m, weights, prompts
        self.lw = np.ascontiguousarray(np.asarray(cell_LW, dtype=np.int32).reshape(-1, 2))
        C, N = self.lw.shape[0], len(weights["layers"])
        self.C, self.N = C, N
        shp = (C, w.n_kv_heads, w.n_steps, w.head_dim)
        self.gen_k = [np.zeros(shp, dtype=np.uint16) for _ in range(N)]
        self.gen_v = [np.zeros(shp, dtype=np.uint16) for _ in range(N)]
        self.osh = make_shape(1, w.n_q_heads, w.n_kv_heads, w.head_dim, w.prompt_len, w.span, w.n_steps,
                              w.donor == "zero", 2)

    def attend(self, l: int, c: int, s: int, q_c: np.ndarray) -> np.ndarray:
        """Attention output [Hq][D] of cell c at layer l, step s (q_c: bf16
        bits [Hq][D]) over its spliced prompt and generated rows 0..s."""
        w, pr = self.w, self.prompts[l]
        oc, _ = attn(self.osh, l, s, w.window(l), w.head_dim ** -0.5, self.lw[c:c + 1],
                     np.ascontiguousarray(q_c[None]), pr["clean_k"], pr["clean_v"], pr["donor_k"], pr["donor_v"],
                     np.ascontiguousarray(self.gen_k[l][c:c + 1]), np.ascontiguousarray(self.gen_v[l][c:c + 1]))
        return oc[0]

    def forward(self, tokens: np.ndarray, steps: np.ndarray) -> np.ndarray:
        """Logits [C][V] of one decode pass (rows of finished cells are not
        meaningful); steps[c] < 0 marks a finished cell."""
        w, m, wt = self.w, self.m, self.wt
        C, Hq, Hkv, D = self.C, w.n_q_heads, w.n_kv_heads, w.head_dim
        pos = w.prompt_len + np.maximum(steps, 0)
        x = wt["embed"][tokens].astype(np.float64)
        for l in range(self.N):
            p = wt["layers"][l]
            h = _rms_norm(x, p["norm_1"], m.rms_eps)
            q = to_bf16_bits(_rope((h @ p["w_q"]).reshape(C, Hq, D), pos, m.rope_theta))
            k = to_bf16_bits(_rope((h @ p["w_k"]).reshape(C, Hkv, D), pos, m.rope_theta))
            v = to_bf16_bits((h @ p["w_v"]).reshape(C, Hkv, D))
            o = np.zeros((C, Hq, D))
            for c in range(C):
                s = int(steps[c])
                if s < 0:
                    continue
                self.gen_k[l][c, :, s] = k[c]
                self.gen_v[l][c, :, s] = v[c]
                o[c] = self.attend(l, c, s, q[c])
            x = x + o.reshape(C, Hq * D) @ p["w_o"]
            h2 = _rms_norm(x, p["norm_2"], m.rms_eps)
            x = x + (_silu(h2 @ p["w_gate"]) * (h2 @ p["w_up"])) @ p["w_down"]
        return _rms_norm(x, wt["norm_f"], m.rms_eps) @ wt["lm_head"]


def greedy(logits: np.ndarray) -> np.ndarray:
    """Lowest index of the maximal logit, per row."""
    return np.argmax(logits, axis=-1)
