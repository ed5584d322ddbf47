"""GPU parity of splice_decode_forked: a sweep decoded as one clean run (the
trunk) that each cell forks from at its onset W (Section 3: nothing is
spliced before step W, so a cell is the clean run until then).

A cell that has diverged attends over its prompt as usual and over generated
rows that are the trunk's below W and its own from W on; the oracle sees that
cache materialised on the host (run per cell, C = 1).  A cell that has not
diverged gets the trunk's out and lse bit for bit.  The rows a diverged cell
must not read (its own rows below W) hold NaN, so reading one fails the
test."""
import numpy as np
import pytest
import torch

import gpu_common as gc
import oracle
import oracle_pins
import paper_2605_30574_amd as sp
import workloads
from workloads import DONOR_BLANK, DONOR_ZERO

pytestmark = pytest.mark.gpu

BF16_NAN = 0x7FC0


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    sp.load_library()


def sweep_cells(w, n):
    """n sweep cells spread over the grid, plus a never-spliced trunk cell
    (L = n_layers) if the grid has none; returns (cell_LW, trunk index)."""
    lw = workloads.cell_lw(w)
    idx = np.linspace(0, lw.shape[0] - 1, n).round().astype(int)
    lw = lw[idx]
    never = np.nonzero(lw[:, 0] >= w.n_layers)[0]
    if never.size:
        return np.ascontiguousarray(lw), int(never[0])
    lw = np.concatenate([lw, np.array([[w.n_layers, 0]], dtype=np.int32)])
    return np.ascontiguousarray(lw), lw.shape[0] - 1


def diverged(w, lw, trunk, step):
    return np.array([c == trunk or (lw[c, 0] < w.n_layers and step >= lw[c, 1]) for c in range(lw.shape[0])])


def check_forked(w, layer, step, lw, trunk, what, split=0, merge_wait=0):
    C = lw.shape[0]
    gc.announce(f"forked {what} layer={layer} step={step} C={C} trunk={trunk} split={split} wait={merge_wait}")
    bufs = gc.gpu_layer(w, layer, n_cells=C)
    # a diverged cell's own rows below its onset are never read: poison them
    for c in range(C):
        if c != trunk and lw[c, 1] > 0:
            for name in ("gen_k", "gen_v"):
                bufs[name][c, :, :lw[c, 1]].view(torch.int16).fill_(BF16_NAN)
    hb = gc.host(bufs)
    q = workloads.make_q(w, layer, step, device="cuda", n_cells=C)
    shape = gc.shape_of(w, n_cells=C)
    call = sp.make_call(layer, step, w.window(layer), w.scale, split, merge_wait)
    ws = sp.new_workspace(shape, call)
    out = torch.full((C, w.n_q_heads, w.head_dim), float("nan"), device="cuda", dtype=torch.float32)
    lse = torch.full((C, w.n_q_heads), float("nan"), device="cuda", dtype=torch.float32)
    sp.splice_decode_forked(shape, call, lw, trunk, q, bufs["clean_k"], bufs["clean_v"], bufs["donor_k"],
                            bufs["donor_v"], bufs["gen_k"], bufs["gen_v"], out, lse, ws)
    torch.cuda.synchronize()
    o = out.cpu().numpy()
    l = lse.cpu().numpy()
    div = diverged(w, lw, trunk, step)
    # not diverged: the trunk's bits
    for c in np.nonzero(~div)[0]:
        assert np.array_equal(o[c], o[trunk]) and np.array_equal(l[c], l[trunk]), f"{what}: cell {c} != trunk"
    # diverged: the oracle over the materialised cache
    osh = oracle.shape_of(w, n_cells=1)
    qn = workloads.to_numpy(q)
    for c in np.nonzero(div)[0]:
        gk = hb["gen_k"][c:c + 1].copy()
        gv = hb["gen_v"][c:c + 1].copy()
        if c != trunk:
            W = lw[c, 1]
            gk[0, :, :W] = hb["gen_k"][trunk, :, :W]
            gv[0, :, :W] = hb["gen_v"][trunk, :, :W]
        ro, rl = oracle.attn(osh, layer, step, w.window(layer), w.scale, lw[c:c + 1], np.ascontiguousarray(qn[c:c + 1]),
                             hb["clean_k"], hb["clean_v"], hb["donor_k"], hb["donor_v"], gk, gv)
        gc.assert_attn_close(o[c:c + 1].astype(np.float64), l[c:c + 1].astype(np.float64), ro, rl,
                             f"{what} cell {c} (L={lw[c, 0]}, W={lw[c, 1]})")
    return int(div.sum())


def _case(name):
    t = oracle_pins.tiny
    return {
        # (workload, layer, cells)
        "qwen3-4b": (workloads.get("qwen3-4b"), 16, 30),
        "llama3-8b-zero": (workloads.get("llama3-8b"), 12, 24),
        "gemma3-4b-local": (workloads.get("gemma3-4b"), 6, 16),
        "qwen3-8b": (workloads.get("qwen3-8b"), 9, 12),
        "tiny-bf16-window5": (t(dtype="bf16", donor=DONOR_BLANK, window=5, sink=True), 1, 6),
        "tiny-bf16-zero-G8": (t(dtype="bf16", donor=DONOR_ZERO).with_(n_q_heads=16, n_kv_heads=2), 0, 6),
    }[name]


@pytest.mark.parametrize("name", ["qwen3-4b", "llama3-8b-zero", "gemma3-4b-local", "qwen3-8b",
                                  "tiny-bf16-window5", "tiny-bf16-zero-G8"])
def test_forked_matches_oracle(name):
    w, layer, n = _case(name)
    lw, trunk = sweep_cells(w, n)
    onsets = sorted({int(x) for x in lw[:, 1]})
    steps = sorted({0, 1} | {min(w.n_steps - 1, x) for W in onsets for x in (max(W - 1, 0), W)} | {w.n_steps - 1})
    for step in steps:
        check_forked(w, layer, step, lw, trunk, name)


def test_forked_split_and_merge_site():
    w, layer, n = _case("llama3-8b-zero")
    lw, trunk = sweep_cells(w, n)
    for step, split, mw in ((3, 64, -1), (40, 128, 0), (255, 64, 1)):
        check_forked(w, layer, step, lw, trunk, f"llama split={split}", split, mw)


def test_every_cell_dormant_but_the_trunk():
    """At step 0 every cell with W > 0 is still the clean run."""
    w, layer, n = _case("qwen3-4b")
    lw, trunk = sweep_cells(w, n)
    lw = lw.copy()
    lw[:, 1] = np.where(np.arange(lw.shape[0]) == trunk, lw[:, 1], 5)
    assert check_forked(w, layer, 0, lw, trunk, "all dormant") == 1
