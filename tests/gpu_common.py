"""Shared helpers of the GPU tests: run the library and the oracle on the same
seeded inputs and compare them to the acceptance bar.

Bar (out fp32 vs oracle fp64 on the same bf16/f32 inputs): max abs error
<= 1e-2 and mean abs error <= 1e-3 per call on out; relative error <= 1e-4
on lse, relative to max(1, |lse|).  Gather output and source map: bit-exact.
"""
from __future__ import annotations

import sys
from typing import Optional

import numpy as np
import torch

import oracle
import paper_2605_30574_amd as sp
import workloads

OUT_MAX_ABS = 1e-2
OUT_MEAN_ABS = 1e-3
LSE_REL = 1e-4


def announce(msg: str) -> None:
    """Name the case on the real stderr before a GPU step (survives capture)."""
    sys.__stderr__.write(f"[gpu] {msg}\n")
    sys.__stderr__.flush()


def shape_of(w: workloads.Workload, n_cells: Optional[int] = None) -> sp.SpliceShape:
    return sp.make_shape(w.n_cells if n_cells is None else n_cells, w.n_layers, w.n_q_heads,
                         w.n_kv_heads, w.head_dim, w.prompt_len, w.span, w.n_steps,
                         w.donor == workloads.DONOR_ZERO, w.dtype)


def gpu_layer(w, layer, seed=0, n_cells=None):
    return workloads.make_layer(w, layer, seed=seed, device="cuda", n_cells=n_cells)


def host(bufs):
    return {k: workloads.to_numpy(v) for k, v in bufs.items()}


def run_attn(w, layer, step, bufs, q, lw, split=0, ws=None, shape=None, merge_wait=0):
    shape = shape or shape_of(w, n_cells=q.shape[0])
    call = sp.make_call(layer, step, w.window(layer), w.scale, split, merge_wait)
    C = shape.n_cells
    out = torch.full((C, w.n_q_heads, w.head_dim), float("nan"), device="cuda", dtype=torch.float32)
    lse = torch.full((C, w.n_q_heads), float("nan"), device="cuda", dtype=torch.float32)
    if ws is None:
        ws = sp.new_workspace(shape, call)
    sp.splice_decode_attn(shape, call, lw, q, bufs["clean_k"], bufs["clean_v"], bufs["donor_k"],
                          bufs["donor_v"], bufs["gen_k"], bufs["gen_v"], out, lse, ws)
    torch.cuda.synchronize()
    return out.cpu().numpy().astype(np.float64), lse.cpu().numpy().astype(np.float64)


def run_gather(w, layer, step, bufs, lw, shape=None):
    shape = shape or shape_of(w, n_cells=lw.shape[0])
    call = sp.make_call(layer, step, w.window(layer), w.scale)
    n_vis = sp.splice_visible_len(shape, call)
    C = shape.n_cells
    dt = workloads.torch_dtype(w)
    ok = torch.empty((C, w.n_kv_heads, n_vis, w.head_dim), dtype=dt, device="cuda")
    ov = torch.empty_like(ok)
    src = torch.full((C, n_vis), 255, dtype=torch.uint8, device="cuda")
    sp.splice_kv_build(shape, call, lw, bufs["clean_k"], bufs["clean_v"], bufs["donor_k"],
                       bufs["donor_v"], bufs["gen_k"], bufs["gen_v"], ok, ov, src)
    torch.cuda.synchronize()
    return workloads.to_numpy(ok), workloads.to_numpy(ov), src.cpu().numpy()


def run_oracle(w, layer, step, hbufs, q_np, lw, rows=None, n_cells=None):
    osh = oracle.shape_of(w, n_cells=lw.shape[0] if n_cells is None else n_cells)
    return oracle.attn(osh, layer, step, w.window(layer), w.scale, lw, q_np, hbufs["clean_k"],
                       hbufs["clean_v"], hbufs["donor_k"], hbufs["donor_v"], hbufs["gen_k"],
                       hbufs["gen_v"], rows=rows)


def run_oracle_gather(w, layer, step, hbufs, lw):
    osh = oracle.shape_of(w, n_cells=lw.shape[0])
    return oracle.gather(osh, layer, step, w.window(layer), lw, hbufs["clean_k"], hbufs["clean_v"],
                         hbufs["donor_k"], hbufs["donor_v"], hbufs["gen_k"], hbufs["gen_v"])


def attn_errors(out, lse, ref_out, ref_lse):
    err = np.abs(out - ref_out)
    rel = np.abs(lse - ref_lse) / np.maximum(1.0, np.abs(ref_lse))
    return float(err.max()), float(err.mean()), float(rel.max())


def assert_attn_close(out, lse, ref_out, ref_lse, what=""):
    assert np.all(np.isfinite(out)) and np.all(np.isfinite(lse)), f"{what}: non-finite output"
    mx, mean, rel = attn_errors(out, lse, ref_out, ref_lse)
    assert mx <= OUT_MAX_ABS, f"{what}: out max abs {mx:.3e}"
    assert mean <= OUT_MEAN_ABS, f"{what}: out mean abs {mean:.3e}"
    assert rel <= LSE_REL, f"{what}: lse rel {rel:.3e}"
    return mx, mean, rel
