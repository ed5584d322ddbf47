"""Invariants of the method, reproduced by the GPU library itself:
donor == clean and onsets past the step are bit-identical to unspliced, a
cell's result does not depend on its batch-mates, repeat calls are
bit-identical, and the split of the key list changes only rounding."""
import sys

import numpy as np
import pytest
import torch

import gpu_common as gc
import oracle_pins
import paper_2605_30574_amd as sp
import workloads
from workloads import DONOR_BLANK, DONOR_ZERO

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    sp.load_library()


def _w():
    return oracle_pins.tiny(dtype="bf16", donor=DONOR_BLANK, sink=True, n_steps=200).with_(
        prompt_len=500, span=(40, 460), head_dim=128, scale=128 ** -0.5)


@pytest.mark.parametrize("split", [0, 64])
def test_donor_equal_clean_and_late_onset_are_unspliced(split):
    w = _w()
    lw = workloads.cell_lw(w)
    never = np.array([[w.n_layers, 0]] * w.n_cells, dtype=np.int32)
    for layer in range(w.n_layers):
        bufs = gc.gpu_layer(w, layer)
        same = dict(bufs, donor_k=bufs["clean_k"], donor_v=bufs["clean_v"])
        for step in (0, 4, 199):
            q = workloads.make_q(w, layer, step, device="cuda")
            gc.announce(f"invariants layer={layer} step={step} split={split}")
            o_u, l_u = gc.run_attn(w, layer, step, bufs, q, never, split=split)
            o_s, l_s = gc.run_attn(w, layer, step, same, q, lw, split=split)
            assert np.array_equal(o_u, o_s) and np.array_equal(l_u, l_s)
            late = lw.copy()
            late[:, 1] = step + 1
            o_l, l_l = gc.run_attn(w, layer, step, bufs, q, late, split=split)
            assert np.array_equal(o_u, o_l) and np.array_equal(l_u, l_l)


def test_batch_independence_and_determinism():
    w = _w()
    lw = workloads.cell_lw(w)
    layer, step = 1, 150
    bufs = gc.gpu_layer(w, layer)
    q = workloads.make_q(w, layer, step, device="cuda")
    gc.announce("batch independence")
    o_b, l_b = gc.run_attn(w, layer, step, bufs, q, lw, split=128)
    o_r, l_r = gc.run_attn(w, layer, step, bufs, q, lw, split=128)
    assert np.array_equal(o_b, o_r) and np.array_equal(l_b, l_r), "repeat call not bit-identical"
    for c in range(w.n_cells):
        one = dict(bufs, gen_k=bufs["gen_k"][c:c + 1].contiguous(), gen_v=bufs["gen_v"][c:c + 1].contiguous())
        o1, l1 = gc.run_attn(w, layer, step, one, q[c:c + 1].contiguous(), lw[c:c + 1].copy(), split=128)
        assert np.array_equal(o1[0], o_b[c]) and np.array_equal(l1[0], l_b[c]), f"cell {c}"
    # reversed batch order
    perm = np.arange(w.n_cells)[::-1].copy()
    pb = dict(bufs, gen_k=bufs["gen_k"][perm].contiguous(), gen_v=bufs["gen_v"][perm].contiguous())
    o_p, l_p = gc.run_attn(w, layer, step, pb, q[perm].contiguous(), lw[perm].copy(), split=128)
    assert np.array_equal(o_p, o_b[perm]) and np.array_equal(l_p, l_b[perm])


@pytest.mark.parametrize("donor", [DONOR_BLANK, DONOR_ZERO])
def test_merge_site_does_not_change_bits(donor):
    """A generated-row item merges its (cell, KV head) in place after waiting
    for the prompt partials, or -- past its polling bound -- leaves the merge
    to the last item to finish.  Both follow one fold order, so the bits are
    the same whichever item merged.  merge_wait < 0 never polls, so every
    pair takes the hand-over route (the workspace counts C * Hkv hand-overs);
    the default bound takes none; 1 poll mixes the two within a call."""
    w = _w().with_(donor=donor)
    lw = workloads.cell_lw(w)
    layer, step = 1, 150
    bufs = gc.gpu_layer(w, layer)
    hb = gc.host(bufs)
    q = workloads.make_q(w, layer, step, device="cuda")
    ref_o, ref_l = gc.run_oracle(w, layer, step, hb, workloads.to_numpy(q), lw)
    shape = gc.shape_of(w)
    pairs = w.n_cells * w.n_kv_heads
    gc.announce(f"merge site donor={donor}: in place")
    ws = sp.new_workspace(shape, sp.make_call(layer, step, 0, w.scale, 64))
    o_w, l_w = gc.run_attn(w, layer, step, bufs, q, lw, split=64, ws=ws)
    gc.assert_attn_close(o_w, l_w, ref_o, ref_l, "in place")
    assert sp.splice_workspace_handovers(ws) == 0, "the default bound handed a merge over"
    for mw in (-1, 1):
        gc.announce(f"merge site donor={donor}: merge_wait={mw}")
        ws = sp.new_workspace(shape, sp.make_call(layer, step, 0, w.scale, 64))
        o_h, l_h = gc.run_attn(w, layer, step, bufs, q, lw, split=64, merge_wait=mw, ws=ws)
        assert np.array_equal(o_h, o_w) and np.array_equal(l_h, l_w), f"merge_wait={mw}"
        n = sp.splice_workspace_handovers(ws)
        if mw < 0:
            assert n == pairs, f"merge_wait=-1 handed over {n} of {pairs} merges"
        else:
            assert 0 <= n <= pairs


@pytest.mark.parametrize("merge_wait", [0, -1])
def test_large_values_scale_exactly(merge_wait):
    """V scaled by 2^17 scales out by 2^17 and leaves lse as it was: every
    product and sum of P.V moves by a power of two, and a prompt partial of
    a bf16 call, kept in fp16 as o / (l sc), takes a power-of-two range
    factor sc once the row's largest |o / l| passes the fp16 limit (here it
    does: |v| reaches about 5 * 2^17), so its rounding moves with the scale
    too.  The only slack allowed is for partial values below the fp16
    normal range at scale 1, which are kept more precisely at 2^17.  Both
    merge sites (in place, and the hand-over merge) read such slots."""
    w = _w()
    lw = workloads.cell_lw(w)
    layer, step = 1, 150
    bufs = gc.gpu_layer(w, layer)
    f = float(2 ** 17)
    big = dict(bufs, clean_v=bufs["clean_v"] * f, donor_v=bufs["donor_v"] * f, gen_v=bufs["gen_v"] * f)
    assert torch.equal(big["gen_v"] / f, bufs["gen_v"])   # the scaling itself is exact in bf16
    q = workloads.make_q(w, layer, step, device="cuda")
    gc.announce(f"scale 2^17 merge_wait={merge_wait}")
    o, l = gc.run_attn(w, layer, step, bufs, q, lw, split=64, merge_wait=merge_wait)
    ob, lb = gc.run_attn(w, layer, step, big, q, lw, split=64, merge_wait=merge_wait)
    assert np.all(np.isfinite(ob)) and np.array_equal(l, lb)
    assert np.abs(ob / f - o).max() <= 1e-6 * max(1.0, np.abs(o).max())
    hb = gc.host(big)
    ref_o, ref_l = gc.run_oracle(w, layer, step, hb, workloads.to_numpy(q), lw)
    gc.assert_attn_close(ob / f, lb, ref_o / f, ref_l, "V x 2^17")


def test_split_changes_only_rounding():
    w = _w()
    lw = workloads.cell_lw(w)
    layer, step = 0, 180
    bufs = gc.gpu_layer(w, layer)
    hb = gc.host(bufs)
    q = workloads.make_q(w, layer, step, device="cuda")
    ref_o, ref_l = gc.run_oracle(w, layer, step, hb, workloads.to_numpy(q), lw)
    results = []
    for split in (64, 128, 320, 704, 0):
        gc.announce(f"split {split}")
        o, l = gc.run_attn(w, layer, step, bufs, q, lw, split=split)
        gc.assert_attn_close(o, l, ref_o, ref_l, f"split={split}")
        results.append((o, l))
    for o, l in results[1:]:
        gc.assert_attn_close(o, l, results[0][0], results[0][1], "split vs split")


def test_workspace_reuse_across_steps_and_splits():
    """One workspace serves a sequence of calls of different sizes; each
    call writes every partial slot it reads, so stale contents never leak."""
    w = _w()
    lw = workloads.cell_lw(w)
    shape = gc.shape_of(w)
    ws = sp.new_workspace(shape, sp.make_call(1, w.n_steps - 1, 0, w.scale, 64))
    assert ws.numel() >= sp.splice_decode_attn_workspace_bytes(shape)
    bufs = gc.gpu_layer(w, 1)
    hb = gc.host(bufs)
    for step in (199, 3, 120, 0, 199):
        for split in (64, 0):
            q = workloads.make_q(w, 1, step, device="cuda")
            gc.announce(f"workspace reuse step={step} split={split}")
            o, l = gc.run_attn(w, 1, step, bufs, q, lw, split=split, ws=ws)
            ref_o, ref_l = gc.run_oracle(w, 1, step, hb, workloads.to_numpy(q), lw)
            gc.assert_attn_close(o, l, ref_o, ref_l, f"reuse s={step} split={split}")


def test_graph_replay_matches_eager():
    """Calls captured in a HIP graph and replayed several times, with eager
    work and synchronisation in between, give the eager bits every time."""
    w = _w()
    lw = workloads.cell_lw(w)
    shape = gc.shape_of(w)
    ws = sp.new_workspace(shape)
    bufs = [gc.gpu_layer(w, layer) for layer in range(w.n_layers)]
    steps = (0, 77, 199)
    qs = {(l, s): workloads.make_q(w, l, s, device="cuda") for l in range(w.n_layers) for s in steps}
    outs = {k: torch.empty((w.n_cells, w.n_q_heads, w.head_dim), device="cuda") for k in qs}
    lses = {k: torch.empty((w.n_cells, w.n_q_heads), device="cuda") for k in qs}

    def issue():
        for (l, s) in qs:
            b = bufs[l]
            sp.splice_decode_attn(shape, sp.make_call(l, s, 0, w.scale), lw, qs[(l, s)], b["clean_k"],
                                  b["clean_v"], b["donor_k"], b["donor_v"], b["gen_k"], b["gen_v"],
                                  outs[(l, s)], lses[(l, s)], ws)

    gc.announce("graph replay: eager reference")
    issue()
    torch.cuda.synchronize()
    ref = {k: (outs[k].clone(), lses[k].clone()) for k in qs}
    stream = torch.cuda.Stream()
    stream.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=stream):
        issue()
    torch.cuda.synchronize()
    for rep in range(4):
        for k in qs:
            outs[k].fill_(float("nan"))
            lses[k].fill_(float("nan"))
        torch.cuda.synchronize()
        gc.announce(f"graph replay {rep}")
        g.replay()
        torch.cuda.synchronize()
        for k in qs:
            assert torch.equal(outs[k], ref[k][0]) and torch.equal(lses[k], ref[k][1]), (rep, k)
        issue()                                  # eager work between replays
        torch.cuda.synchronize()


_FIRST_CALL_IN_GRAPH = r"""
import sys
import torch
import paper_2605_30574_amd as sp
import workloads
w = workloads.get("qwen3-4b")
layer, step = 17, 300
lw = workloads.cell_lw(w)
b = workloads.make_layer(w, layer, device="cuda")
q = workloads.make_q(w, layer, step, device="cuda")
shape = sp.make_shape(w.n_cells, w.n_layers, w.n_q_heads, w.n_kv_heads, w.head_dim, w.prompt_len, w.span,
                      w.n_steps, w.donor == workloads.DONOR_ZERO, w.dtype)
call = sp.make_call(layer, step, w.window(layer), w.scale)
ws = sp.new_workspace(shape)
out = [torch.full((w.n_cells, w.n_q_heads, w.head_dim), float("nan"), device="cuda") for _ in range(2)]
lse = [torch.full((w.n_cells, w.n_q_heads), float("nan"), device="cuda") for _ in range(2)]
def run(i):
    sp.splice_decode_attn(shape, call, lw, q, b["clean_k"], b["clean_v"], b["donor_k"], b["donor_v"],
                          b["gen_k"], b["gen_v"], out[i], lse[i], ws)
torch.cuda.synchronize()
stream = torch.cuda.Stream()
stream.wait_stream(torch.cuda.current_stream())
g = torch.cuda.CUDAGraph()
with torch.cuda.graph(g, stream=stream):   # the process's first attention call
    run(0)
g.replay()
torch.cuda.synchronize()
run(1)
torch.cuda.synchronize()
ok = torch.equal(out[0], out[1]) and torch.equal(lse[0], lse[1]) and bool(torch.isfinite(out[0]).all())
print("first-call-in-graph", "ok" if ok else "MISMATCH", flush=True)
sys.exit(0 if ok else 1)
"""


def test_first_call_inside_graph_capture():
    """The library asks HIP for the device's compute units and the kernel's
    residency on its first call on a device; when that first call is being
    captured into a graph, the queries must not break the capture, and the
    replay must give the eager call's bits.  Run in a fresh process, whose
    first attention call is the captured one."""
    import os
    import subprocess
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    gc.announce("first call inside graph capture (subprocess)")
    env = dict(os.environ, PYTHONPATH=root + os.pathsep + os.environ.get("PYTHONPATH", ""))
    res = subprocess.run([sys.executable, "-c", _FIRST_CALL_IN_GRAPH], cwd=root, env=env, capture_output=True,
                         text=True, timeout=240)
    assert res.returncode == 0 and "first-call-in-graph ok" in res.stdout, (res.stdout[-2000:], res.stderr[-2000:])


def test_workspace_reuse_gives_fresh_workspace_bits():
    """One workspace serves a sequence of calls that change the slot count
    (the split), hand every merge over (merge_wait < 0) or mix both merge
    sites (1), and skip finished cells (a ragged decode step).  Every call
    must give the bits the same call gives on a fresh workspace: what a call
    leaves behind (partial slots, arrival counters) never reaches the next
    one."""
    w = _w().with_(prompt_len=1100, span=(40, 1060))
    lw = workloads.cell_lw(w)
    C = lw.shape[0]
    layer = 1
    shape = gc.shape_of(w, n_cells=C)
    bufs = gc.gpu_layer(w, layer)
    # sized for the call with the most slots (64-key chunks)
    shared = sp.new_workspace(shape, sp.make_call(layer, 150, w.window(layer), w.scale, 64))
    finished = workloads.cell_steps(w, seed=3, n_cells=C, finished=0.25) < 0
    plan = [  # (split_keys, merge_wait, step, ragged decode step?)
        (512, 0, 10, False), (64, 0, 150, False), (256, 1, 40, False), (128, -1, 150, False),
        (0, 0, 60, True), (512, -1, 150, False), (256, 0, 199, False), (64, 1, 3, False),
        (0, 0, 61, True), (512, 0, 150, False), (128, 0, 20, False), (256, -1, 150, False)]
    for i, (split, mw, step, ragged) in enumerate(plan):
        gc.announce(f"workspace reuse call {i}: split={split} wait={mw} step={step} ragged={ragged}")
        q = workloads.make_q(w, layer, step, device="cuda")
        if not ragged:
            got = gc.run_attn(w, layer, step, bufs, q, lw, split=split, ws=shared, shape=shape, merge_wait=mw)
            want = gc.run_attn(w, layer, step, bufs, q, lw, split=split, shape=shape, merge_wait=mw)
        else:
            steps = np.where(finished, -1, step).astype(np.int32)
            new = workloads.make_new_rows(w, layer, step, device="cuda", n_cells=C)
            call = sp.make_call(layer, 0, w.window(layer), w.scale, split, mw)
            res = []
            for ws in (shared, sp.new_workspace(shape)):
                out = torch.full((C, w.n_q_heads, w.head_dim), float("nan"), device="cuda")
                lse = torch.full((C, w.n_q_heads), float("nan"), device="cuda")
                sp.splice_decode_step(shape, call, lw, steps, q, new["k_new"], new["v_new"], bufs["clean_k"],
                                      bufs["clean_v"], bufs["donor_k"], bufs["donor_v"], bufs["gen_k"],
                                      bufs["gen_v"], out, lse, ws)
                torch.cuda.synchronize()
                res.append((out.cpu().numpy(), lse.cpu().numpy()))
            got, want = res
        assert np.array_equal(got[0], want[0], equal_nan=True), f"call {i}: out"
        assert np.array_equal(got[1], want[1], equal_nan=True), f"call {i}: lse"
