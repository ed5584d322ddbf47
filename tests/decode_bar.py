"""Bars of the decode-loop GPU test (tests/test_gpu_decode.py), derived on
the CPU from the attention bar alone.

The GPU decode loop and the float64 reference (oracle.decoder) differ by the
attention library's own error, carried through the layers: q, k, v and the
caches are bf16 on both sides.  A conforming attention kernel errs by at
most 1e-2 (max abs) and 1e-3 (mean abs) per call on out.  The bars are
what a kernel at the mean limit produces: the reference decoder runs once
as is and once with every attention output perturbed, both teacher-forced
on the unperturbed run's tokens.  Two families of perturbation, each with a
mean absolute value of exactly 1e-3 per (cell, layer, step) and clipped at
1e-2:

  * independent: Gaussian noise on every output element;
  * coherent: the whole output of the call scaled by 1 + e, one e per call
    (random sign) -- an error shared by every element, like a misjudged
    normaliser or a rounded dominant weight, which the independent family
    averages away in the projections that follow.

Over DRAWS draws of each family on each test case, the derivation records

  * the largest logit deviation relative to max(1, |largest logit|);
  * on the appended cache rows at layers >= 1 (layer 0's rows depend on the
    embeddings alone), the largest absolute deviation of an element relative
    to the root mean square of that layer's K (or V) rows, and the fraction
    of elements whose bits differ.  (A distance in units in the last place
    is no measure here: the perturbation moves k by an amount set by the
    layer's scale, so an element near zero can change sign, thousands of
    ulps away.)

Each bar is twice the worst value observed, rounded up to two digits.  The GPU test's constants must equal derive()'s
(test_decode_bar.py checks it), so a bar moves only with this derivation.
"""
from __future__ import annotations

import math

import numpy as np
import torch

import oracle_pins
from oracle import decoder as ref
import workloads
from workloads.model import ModelConfig, make_weights

ATTN_MEAN_ABS = 1e-3     # the attention bar (the benchmark spec): mean abs error of out per call
ATTN_MAX_ABS = 1e-2      # ... and max abs error
DRAWS = 6
MODEL = ModelConfig(d_model=96, d_ff=160, vocab=64, eos=5)


def case(name: str):
    """The decode-loop test's workloads (tiny, bf16 attention)."""
    t = oracle_pins.tiny
    return {"blank-sink": lambda: t(dtype="bf16", donor="blank", sink=True),
            "zero-window5": lambda: t(dtype="bf16", donor="zero", window=5),
            "diff-G8": lambda: t(dtype="bf16", donor="diff").with_(n_q_heads=16, n_kv_heads=2)}[name]()


CASES = ("blank-sink", "zero-window5", "diff-G8")


def f64_weights(wt):
    f = lambda t: t.double().numpy()
    return dict(embed=f(wt["embed"]), lm_head=f(wt["lm_head"]), norm_f=f(wt["norm_f"]),
                layers=[{k: f(v) for k, v in L.items()} for L in wt["layers"]])


def row_deviation(want_bits: np.ndarray, got_bits: np.ndarray):
    """(max |got - want| / rms(want), fraction of differing elements) over
    the written rows (nonzero reference bits) of one layer's K or V cache."""
    written = want_bits != 0
    want = ref.from_bf16_bits(want_bits[written])
    got = ref.from_bf16_bits(got_bits[written])
    rms = float(np.sqrt(np.mean(want * want)))
    return float(np.abs(got - want).max()) / rms, float((want_bits[written] != got_bits[written]).mean())


class PerturbedDecoder(ref.ReferenceDecoder):
    """The reference decoder with each attention output moved at the
    attention bar: mean |change| = ATTN_MEAN_ABS over the call's Hq x D
    outputs, each change clipped at ATTN_MAX_ABS; `coherent` scales the
    output by one random-signed factor, else independent Gaussian noise."""

    def __init__(self, *a, rng=None, coherent=False, **kw):
        super().__init__(*a, **kw)
        self.rng, self.coherent = rng, coherent

    def attend(self, l, c, s, q_c):
        o = super().attend(l, c, s, q_c)
        z = o * self.rng.choice((-1.0, 1.0)) if self.coherent else self.rng.standard_normal(o.shape)
        z *= ATTN_MEAN_ABS / np.abs(z).mean()
        return o + np.clip(z, -ATTN_MAX_ABS, ATTN_MAX_ABS)


def prompt_bits(w, C):
    out = []
    for l in range(w.n_layers):
        a = oracle_pins.layer_arrays(w, l)
        out.append({k: a[k] for k in ("clean_k", "clean_v", "donor_k", "donor_v")})
    return out


def run_case(name: str, draws: int = DRAWS):
    """(worst relative logit deviation, worst row deviation relative to the
    rows' rms, worst flip fraction) of the perturbed reference against the
    reference, teacher-forced on the reference's tokens, over `draws`
    perturbations of each family."""
    w = case(name)
    lw = workloads.cell_lw(w)
    C = lw.shape[0]
    wt = f64_weights(make_weights(w, MODEL, dtype=torch.float32))
    prompts = prompt_bits(w, C)
    worst_logit, worst_row, worst_flip = 0.0, 0.0, 0.0
    for d in range(2 * draws):
        a = ref.ReferenceDecoder(w, MODEL, wt, prompts, lw)
        b = PerturbedDecoder(w, MODEL, wt, prompts, lw, rng=np.random.default_rng(1000 + d), coherent=d % 2 == 1)
        steps = np.zeros(C, dtype=np.int32)
        tokens = np.full(C, 11, dtype=np.int64)
        eos = None
        for _ in range(w.n_steps):
            if (steps < 0).all():
                break
            ra = a.forward(tokens, steps)
            rb = b.forward(tokens, steps)
            act = steps >= 0
            scale = max(1.0, float(np.abs(ra[act]).max()))
            worst_logit = max(worst_logit, float(np.abs(rb[act] - ra[act]).max()) / scale)
            nxt = ref.greedy(ra)
            if eos is None:
                eos = int(nxt[2])
            s = steps.copy()
            s[act] += 1
            s[act & (nxt == eos)] = -1
            s[s >= w.n_steps] = -1
            tokens = np.where(s >= 0, nxt, tokens)
            steps = s
        for l in range(1, w.n_layers):
            for ka, kb in ((a.gen_k[l], b.gen_k[l]), (a.gen_v[l], b.gen_v[l])):
                dev, flip = row_deviation(ka, kb)
                worst_row, worst_flip = max(worst_row, dev), max(worst_flip, flip)
    return worst_logit, worst_row, worst_flip


def derive(draws: int = DRAWS):
    """The bars {'logit_rel', 'row_rel', 'row_flip_frac'}: twice the worst
    observed value, rounded up to two significant digits (the flip fraction
    capped at 1)."""
    lg, row, flip = 0.0, 0.0, 0.0
    for name in CASES:
        a, b, c = run_case(name, draws)
        lg, row, flip = max(lg, a), max(row, b), max(flip, c)

    def up2(x):
        e = math.floor(math.log10(x)) - 1
        return round(math.ceil(round(x / 10 ** e, 9)) * 10 ** e, 12)

    return {"logit_rel": up2(2 * lg), "row_rel": up2(2 * row), "row_flip_frac": min(1.0, up2(2 * flip)),
            "observed": {"logit_rel": lg, "row_rel": row, "row_flip_frac": flip}}


if __name__ == "__main__":
    print(derive())
