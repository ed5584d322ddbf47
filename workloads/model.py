"""Seeded synthetic weights for the greedy decode loop around the attention
(Algorithm 1 of the paper: one forward pass per decode step, the argmax
token, a stop at EOS).  No trained checkpoint exists here, so the decoder is
a stand-in with the attention shapes of a workload: pre-norm blocks with
grouped-query attention and a gated MLP, the layout of the paper's Qwen3 and
Llama models.  This module only draws tensors; none of the forward pass
lives here.

Weights are N(0, 1/fan_in) (so activations keep unit scale), the norm
gains 1, in float32, then rounded to the requested dtype.  Layouts
(row-major): embed [V][d], w_q [d][Hq*D], w_k / w_v [d][Hkv*D],
w_o [Hq*D][d], w_gate / w_up [d][F], w_down [F][d], lm_head [d][V].
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Dict, List

import numpy as np
import torch

from .configs import Workload
from .inputs import derive_seed


@dataclass(frozen=True)
class ModelConfig:
    d_model: int
    d_ff: int
    vocab: int
    eos: int                 # token id that ends a cell's decode
    rope_theta: float = 1.0e6
    rms_eps: float = 1.0e-6


# one model per attention shape: the hidden sizes of the paper's models
MODELS = {
    "qwen3-4b": ModelConfig(d_model=2560, d_ff=9728, vocab=151936, eos=151645),
    "llama3-8b": ModelConfig(d_model=4096, d_ff=14336, vocab=128256, eos=128009),
    "qwen3-8b": ModelConfig(d_model=4096, d_ff=12288, vocab=151936, eos=151645),
}

KIND_MODEL = 100   # seed stream of the weights (per layer, per tensor index)


def _randn(shape, seed: int, std: float, device="cpu") -> torch.Tensor:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return torch.randn(*shape, generator=g, dtype=torch.float32, device=device) * std


def make_weights(w: Workload, m: ModelConfig, seed: int = 0, dtype=torch.bfloat16, device="cpu",
                 n_layers: int = None, draw_on_device: bool = False) -> Dict[str, object]:
    """{'embed', 'lm_head', 'norm_f', 'layers': [{'norm_1', 'w_q', 'w_k', 'w_v', 'w_o',
    'norm_2', 'w_gate', 'w_up', 'w_down'}]} for the first n_layers layers.  Drawn
    on the CPU (the same values for every device) unless draw_on_device, which
    is faster for full-size models and gives other values."""
    N = w.n_layers if n_layers is None else n_layers
    d, F, V = m.d_model, m.d_ff, m.vocab
    HqD, HkvD = w.n_q_heads * w.head_dim, w.n_kv_heads * w.head_dim

    def t(shape, layer, idx, fan_in):
        x = _randn(shape, derive_seed(seed, w.index, KIND_MODEL + idx, layer), fan_in ** -0.5,
                   device if draw_on_device else "cpu")
        return x.to(dtype).to(device).contiguous()

    layers: List[Dict[str, torch.Tensor]] = []
    for l in range(N):
        layers.append(dict(
            norm_1=torch.ones(d, dtype=dtype, device=device),
            w_q=t((d, HqD), l, 0, d), w_k=t((d, HkvD), l, 1, d), w_v=t((d, HkvD), l, 2, d),
            w_o=t((HqD, d), l, 3, HqD),
            norm_2=torch.ones(d, dtype=dtype, device=device),
            w_gate=t((d, F), l, 4, d), w_up=t((d, F), l, 5, d), w_down=t((F, d), l, 6, F)))
    return dict(embed=t((V, d), N, 7, 1), lm_head=t((d, V), N, 8, d),
                norm_f=torch.ones(d, dtype=dtype, device=device), layers=layers)


def first_tokens(m: ModelConfig, n_cells: int, seed: int = 0) -> np.ndarray:
    """int64 [C]: the token each cell's decode starts from (the prompt's last)."""
    rng = np.random.default_rng(derive_seed(seed, 0, KIND_MODEL + 9, 0))
    return rng.integers(0, m.vocab, size=n_cells).astype(np.int64)
