"""Greedy decode of a sweep around the spliced attention (Algorithm 1 of the
paper: per decode step one forward pass, which appends the step's K/V to the
generated cache and attends, then the argmax token; a trajectory stops at
EOS or T_max).

The decoder is a stand-in with synthetic weights (``workloads.model``):
pre-norm blocks of grouped-query attention and a gated MLP.  Per layer and
step the attention -- the current token's K/V appended to each cell's
generated cache, then single-query attention over the cell's spliced prompt
and its generated rows -- is one ``splice_decode_step`` launch of this
library's kernel; the projections, norms, rotary embedding and MLP are plain
PyTorch operations (library GEMMs), outside the measured hot path.

Readings of what the paper leaves to the model (the same on the CPU
reference in ``oracle.decoder``):
  * RMSNorm x / sqrt(mean(x^2) + eps) * gain; residual stream in float32;
  * rotary embedding on q and k, pairs (i, i + D/2), angle
    pos * theta^(-2i/D), position T_p + s for decode step s;
  * MLP down(silu(gate(h)) * up(h)); logits from the final norm;
  * the next token is the lowest index of the maximal logit; a cell that
    emits EOS stops (its step becomes -1) and is skipped from then on.
"""
from __future__ import annotations

from typing import List, Optional

import numpy as np
import torch

from . import splice as S


def rms_norm(x: torch.Tensor, gain: torch.Tensor, eps: float) -> torch.Tensor:
    xf = x.float()
    return xf * torch.rsqrt(xf.pow(2).mean(-1, keepdim=True) + eps) * gain.float()


def rope(x: torch.Tensor, pos: torch.Tensor, theta: float) -> torch.Tensor:
    """x [C][H][D] float32, pos [C]: rotate pairs (i, i + D/2) by pos * theta^(-2i/D)."""
    D = x.shape[-1]
    half = D // 2
    inv = theta ** (-torch.arange(0, half, device=x.device, dtype=torch.float64) * 2.0 / D)
    ang = (pos.to(torch.float64)[:, None] * inv[None, :]).to(torch.float32)   # [C][D/2]
    cos, sin = torch.cos(ang)[:, None, :], torch.sin(ang)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return torch.cat([x1 * cos - x2 * sin, x2 * cos + x1 * sin], dim=-1)


class SweepDecoder:
    """C sweep cells (L_c, W_c) decoding over one prompt, all N layers.

    ``weights`` as drawn by ``workloads.model.make_weights`` (on the device);
    ``caches[l]``: dict clean_k, clean_v, donor_k, donor_v (prompt caches of
    layer l, shared by the cells) and gen_k, gen_v ([C][Hkv][S][D], rows
    written by the decode itself)."""

    def __init__(self, w, m, weights, caches: List[dict], cell_LW, device="cuda"):
        self.w, self.m, self.wt, self.caches = w, m, weights, caches
        self.lw = np.ascontiguousarray(np.asarray(cell_LW, dtype=np.int32).reshape(-1, 2))
        C = self.lw.shape[0]
        self.C, self.N = C, len(weights["layers"])
        self.shape = S.make_shape(C, self.N, w.n_q_heads, w.n_kv_heads, w.head_dim, w.prompt_len, w.span,
                                  w.n_steps, w.donor == "zero", "bf16")
        self.ws = S.new_workspace(self.shape, device=device)
        self.out = torch.empty((C, w.n_q_heads, w.head_dim), dtype=torch.float32, device=device)
        self.lse = torch.empty((C, w.n_q_heads), dtype=torch.float32, device=device)
        self.calls = [S.make_call(l, 0, w.window(l), w.head_dim ** -0.5) for l in range(self.N)]
        self.device = device

    def positions(self, steps: np.ndarray) -> torch.Tensor:
        """Device positions T_p + s of the cells' current tokens."""
        return torch.as_tensor(self.w.prompt_len + np.maximum(steps, 0), device=self.device)

    def forward(self, tokens: torch.Tensor, steps: np.ndarray, pos: Optional[torch.Tensor] = None) -> torch.Tensor:
        """Logits [C][V] (float32) of one decode pass; steps[c] < 0: finished.
        pos: the device positions (self.positions(steps)), given when the pass
        is captured in a graph."""
        w, m, wt = self.w, self.m, self.wt
        C, Hq, Hkv, D = self.C, w.n_q_heads, w.n_kv_heads, w.head_dim
        cdt = wt["embed"].dtype
        if pos is None:
            pos = self.positions(steps)
        x = wt["embed"][tokens].float()
        for l in range(self.N):
            p = wt["layers"][l]
            h = rms_norm(x, p["norm_1"], m.rms_eps).to(cdt)
            q = rope((h @ p["w_q"]).float().view(C, Hq, D), pos, m.rope_theta)
            k = rope((h @ p["w_k"]).float().view(C, Hkv, D), pos, m.rope_theta)
            v = (h @ p["w_v"]).float().view(C, Hkv, D)
            c = self.caches[l]
            S.splice_decode_step(self.shape, self.calls[l], self.lw, steps,
                                 q.to(torch.bfloat16).contiguous(), k.to(torch.bfloat16).contiguous(),
                                 v.to(torch.bfloat16).contiguous(), c["clean_k"], c["clean_v"], c["donor_k"],
                                 c["donor_v"], c["gen_k"], c["gen_v"], self.out, self.lse, self.ws)
            x = x + (self.out.view(C, Hq * D).to(cdt) @ p["w_o"]).float()
            h = rms_norm(x, p["norm_2"], m.rms_eps).to(cdt)
            x = x + ((torch.nn.functional.silu((h @ p["w_gate"]).float()).to(cdt) * (h @ p["w_up"]))
                     @ p["w_down"]).float()
        return (rms_norm(x, wt["norm_f"], m.rms_eps).to(cdt) @ wt["lm_head"]).float()

    def step(self, tokens: torch.Tensor, steps: np.ndarray, pos: Optional[torch.Tensor] = None):
        """One decode pass: (next tokens [C] int64, logits [C][V]).  argmax
        returns the first maximal index, the lowest-index tie-break."""
        logits = self.forward(tokens, steps, pos)
        return torch.argmax(logits, dim=-1), logits


def advance(steps: np.ndarray, next_tokens: np.ndarray, eos: int, n_steps: int) -> np.ndarray:
    """The cells' steps after a pass: +1, or -1 for a cell that emitted EOS or
    reached T_max (= the generated-cache capacity)."""
    s = steps.copy()
    act = s >= 0
    s[act] += 1
    s[act & (next_tokens == eos)] = -1
    s[s >= n_steps] = -1
    return s
