"""GPU parity of splice_decode_step: each cell at its own decode step, the
current token's K/V appended to the generated caches, finished cells (EOS)
skipped (Algorithm 1's decode loop: append, attend, stop at EOS).

The oracle has no notion of a decode step: it is run per cell (C = 1) at
that cell's step, over host caches in which row s_c was replaced by the new
row.  Appended rows and every other cache byte: bit-exact.  out, lse of
active cells: the attention bar of the other parity tests.  Finished cells:
no output written (the NaN sentinel survives) and their caches unchanged."""
import numpy as np
import pytest
import torch

import gpu_common as gc
import oracle
import oracle_pins
import paper_2605_30574_amd as sp
import workloads
from workloads import DONOR_BLANK, DONOR_DIFF, DONOR_ZERO

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    sp.load_library()


def spread_cells(w, n):
    """n of the workload's sweep cells, spread over its (L, W) grid."""
    lw = workloads.cell_lw(w)
    idx = np.linspace(0, lw.shape[0] - 1, n).round().astype(int)
    return np.ascontiguousarray(lw[idx])


def run_step(w, layer, lw, steps, bufs, q, new, split=0, merge_wait=0):
    C = lw.shape[0]
    shape = gc.shape_of(w, n_cells=C)
    call = sp.make_call(layer, 0, w.window(layer), w.scale, split, merge_wait)
    active = steps[steps >= 0]
    if split and active.size:   # an explicit split: size the workspace for the smallest step
        ws = sp.new_workspace(shape, sp.make_call(layer, int(active.min()), w.window(layer), w.scale, split))
    else:
        ws = sp.new_workspace(shape)
    out = torch.full((C, w.n_q_heads, w.head_dim), float("nan"), device="cuda", dtype=torch.float32)
    lse = torch.full((C, w.n_q_heads), float("nan"), device="cuda", dtype=torch.float32)
    sp.splice_decode_step(shape, call, lw, steps, q, new["k_new"], new["v_new"], bufs["clean_k"],
                          bufs["clean_v"], bufs["donor_k"], bufs["donor_v"], bufs["gen_k"], bufs["gen_v"],
                          out, lse, ws)
    torch.cuda.synchronize()
    return out.cpu().numpy().astype(np.float64), lse.cpu().numpy().astype(np.float64)


def append_on_host(hb, new_h, steps):
    """Host caches after the pass: row s_c of each active cell set to its new row."""
    gk, gv = hb["gen_k"].copy(), hb["gen_v"].copy()
    for c, s in enumerate(steps):
        if s >= 0:
            gk[c, :, s, :] = new_h["k_new"][c]
            gv[c, :, s, :] = new_h["v_new"][c]
    out = dict(hb)
    out["gen_k"], out["gen_v"] = gk, gv
    return out


def oracle_step(w, layer, lw, steps, hb, q_np):
    """fp64 out, lse of every active cell, each at its own step (C = 1 per call)."""
    C = lw.shape[0]
    ref_o = np.full((C, w.n_q_heads, w.head_dim), np.nan)
    ref_l = np.full((C, w.n_q_heads), np.nan)
    osh = oracle.shape_of(w, n_cells=1)
    for c, s in enumerate(steps):
        if s < 0:
            continue
        o, l = oracle.attn(osh, layer, int(s), w.window(layer), w.scale, lw[c:c + 1],
                           np.ascontiguousarray(q_np[c:c + 1]), hb["clean_k"], hb["clean_v"], hb["donor_k"],
                           hb["donor_v"], np.ascontiguousarray(hb["gen_k"][c:c + 1]),
                           np.ascontiguousarray(hb["gen_v"][c:c + 1]))
        ref_o[c], ref_l[c] = o[0], l[0]
    return ref_o, ref_l


def check_pass(w, layer, lw, steps, bufs, hb, q, new, what, split=0, merge_wait=0):
    """Run one pass on the GPU and check it; returns the host caches after it."""
    gc.announce(f"decode_step {what} layer={layer} C={lw.shape[0]} split={split} wait={merge_wait} "
                f"steps={steps.tolist()}")
    out, lse = run_step(w, layer, lw, steps, bufs, q, new, split, merge_wait)
    after = append_on_host(hb, gc.host(new), steps)
    got = gc.host(bufs)
    for name in ("gen_k", "gen_v"):
        assert np.array_equal(got[name], after[name]), f"{what}: {name} after the append"
    act = steps >= 0
    assert np.all(np.isnan(out[~act])) and np.all(np.isnan(lse[~act])), f"{what}: a finished cell was written"
    if act.any():
        ref_o, ref_l = oracle_step(w, layer, lw, steps, after, workloads.to_numpy(q))
        gc.assert_attn_close(out[act], lse[act], ref_o[act], ref_l[act], what)
    return after


def _case(name):
    t = oracle_pins.tiny
    return {
        # (workload, layer, cells)
        "qwen3-4b": (workloads.get("qwen3-4b"), 16, 24),
        "qwen3-4b-window100": (workloads.get("qwen3-4b").with_(local_window=100), 8, 24),
        "llama3-8b-zero": (workloads.get("llama3-8b"), 12, 16),
        "gemma3-4b-local": (workloads.get("gemma3-4b"), 6, 12),
        "gemma3-4b-global": (workloads.get("gemma3-4b"), 5, 12),
        "qwen3-8b-diff": (workloads.get("qwen3-8b"), 9, 8),
        "tiny-bf16-G8-zero-window5": (t(dtype="bf16", donor=DONOR_ZERO, window=5)
                                      .with_(n_q_heads=16, n_kv_heads=2), 1, 6),
        "tiny-bf16-G1-D256-blank": (t(dtype="bf16", donor=DONOR_BLANK, sink=True)
                                    .with_(n_q_heads=2, n_kv_heads=2, head_dim=256, scale=1 / 16), 1, 6),
        "tiny-bf16-noprompt": (t(dtype="bf16", donor=DONOR_DIFF).with_(prompt_len=0, span=(0, 0)), 0, 6),
    }[name]


CASES = ["qwen3-4b", "qwen3-4b-window100", "llama3-8b-zero", "gemma3-4b-local", "gemma3-4b-global",
         "qwen3-8b-diff", "tiny-bf16-G8-zero-window5", "tiny-bf16-G1-D256-blank", "tiny-bf16-noprompt"]


@pytest.mark.parametrize("name", CASES)
def test_step_matches_oracle_per_cell(name):
    w, layer, C = _case(name)
    lw = spread_cells(w, C)
    steps = workloads.cell_steps(w, seed=3, n_cells=C)
    bufs = gc.gpu_layer(w, layer, n_cells=C)
    hb = gc.host(bufs)
    q = workloads.make_q(w, layer, 0, device="cuda", n_cells=C)
    new = workloads.make_new_rows(w, layer, 0, device="cuda", n_cells=C)
    check_pass(w, layer, lw, steps, bufs, hb, q, new, name)


@pytest.mark.parametrize("name,split,merge_wait", [
    ("qwen3-4b-window100", 64, 0),     # prompt chunks of 64 keys, rows masked per cell
    ("llama3-8b-zero", 64, -1),        # 16 chunks; the last item to finish merges
    ("qwen3-8b-diff", 256, 0),         # 32 chunks: more than one round of merge loads
    ("gemma3-4b-local", 128, -1),
])
def test_step_split_and_merge_site(name, split, merge_wait):
    w, layer, C = _case(name)
    lw = spread_cells(w, C)
    steps = workloads.cell_steps(w, seed=5, n_cells=C)
    bufs = gc.gpu_layer(w, layer, n_cells=C)
    hb = gc.host(bufs)
    q = workloads.make_q(w, layer, 1, device="cuda", n_cells=C)
    new = workloads.make_new_rows(w, layer, 1, device="cuda", n_cells=C)
    check_pass(w, layer, lw, steps, bufs, hb, q, new, f"{name} split={split}", split, merge_wait)


def test_all_cells_finished_is_a_no_op():
    w, layer, C = _case("qwen3-4b")
    lw = spread_cells(w, C)
    steps = np.full(C, -1, dtype=np.int32)
    bufs = gc.gpu_layer(w, layer, n_cells=C)
    hb = gc.host(bufs)
    q = workloads.make_q(w, layer, 0, device="cuda", n_cells=C)
    new = workloads.make_new_rows(w, layer, 0, device="cuda", n_cells=C)
    check_pass(w, layer, lw, steps, bufs, hb, q, new, "all finished")


def test_same_step_everywhere():
    """Every cell at one step: the lockstep sweep, through the decode-step entry."""
    w, layer, C = _case("llama3-8b-zero")
    lw = spread_cells(w, C)
    for s in (0, 37, w.n_steps - 1):
        steps = np.full(C, s, dtype=np.int32)
        bufs = gc.gpu_layer(w, layer, n_cells=C)
        hb = gc.host(bufs)
        q = workloads.make_q(w, layer, s, device="cuda", n_cells=C)
        new = workloads.make_new_rows(w, layer, s, device="cuda", n_cells=C)
        check_pass(w, layer, lw, steps, bufs, hb, q, new, f"lockstep s={s}")


def test_decode_loop_with_refills():
    """Consecutive passes over one set of caches: cells advance one step per
    pass, some stop, and a stopped slot is refilled with a new cell at step 0."""
    w, layer, C = _case("qwen3-4b-window100")
    lw = spread_cells(w, C)
    steps = workloads.cell_steps(w, seed=11, n_cells=C, max_step=w.n_steps - 6)
    bufs = gc.gpu_layer(w, layer, n_cells=C)
    hb = gc.host(bufs)
    rng = np.random.default_rng(7)
    for p in range(5):
        q = workloads.make_q(w, layer, 100 + p, device="cuda", n_cells=C)
        new = workloads.make_new_rows(w, layer, 100 + p, device="cuda", n_cells=C)
        hb = check_pass(w, layer, lw, steps, bufs, hb, q, new, f"loop pass {p}")
        nxt = np.where(steps >= 0, steps + 1, -1).astype(np.int32)
        stop = rng.random(C) < 0.2
        nxt[stop & (nxt >= 0)] = -1            # EOS
        refill = (steps < 0) & (rng.random(C) < 0.5)
        nxt[refill] = 0                         # a new cell in a freed slot
        lw = lw.copy()
        lw[refill] = spread_cells(w, C)[rng.integers(0, C, size=int(refill.sum()))]
        steps = np.ascontiguousarray(nxt)
