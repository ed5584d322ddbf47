"""The allocation-free entry point (splice_decode_attn_noalloc, through the
C ABI) against splice_decode_attn on a workspace the caller allocated: the
same kernels and plan, so the same bits.  Two calls and more in a row on
one device -- the later ones smaller (fewer cells, an earlier step, another
layer, the f32 path) -- so a call must not depend on what the previous one
left in the library's array; each result is also checked against the
oracle."""
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


def _pair(w, layer, step, bufs, q, lw):
    """(noalloc out, lse), (workspace out, lse) for one call, as float64 arrays."""
    shape = gc.shape_of(w, n_cells=lw.shape[0])
    call = sp.make_call(layer, step, w.window(layer), w.scale)
    res = []
    for noalloc in (True, False):
        C = shape.n_cells
        out = torch.full((C, w.n_q_heads, w.head_dim), float("nan"), device="cuda")
        lse = torch.full((C, w.n_q_heads), float("nan"), device="cuda")
        args = (shape, call, lw, q, bufs["clean_k"], bufs["clean_v"], bufs["donor_k"], bufs["donor_v"],
                bufs["gen_k"], bufs["gen_v"], out, lse)
        if noalloc:
            sp.splice_decode_attn_noalloc(*args)
        else:
            sp.splice_decode_attn(*args, sp.new_workspace(shape, call))
        torch.cuda.synchronize()
        res.append((out.cpu().numpy().astype(np.float64), lse.cpu().numpy().astype(np.float64)))
    return res


def test_noalloc_gives_the_workspace_bits_call_after_call():
    big = oracle_pins.tiny(dtype="bf16", donor=DONOR_BLANK, sink=True, n_steps=200).with_(
        prompt_len=1100, span=(40, 1060), head_dim=128, scale=128 ** -0.5)
    small = big.with_(donor=DONOR_ZERO, prompt_len=300, span=(20, 280))
    tiny = oracle_pins.tiny()   # f32
    plan = [(big, 1, 199, None), (small, 0, 20, 3), (big, 0, 77, 4), (tiny, 1, 9, None)]
    for i, (w, layer, step, n_cells) in enumerate(plan):
        lw = workloads.cell_lw(w)[: n_cells or None].copy()
        C = lw.shape[0]
        gc.announce(f"noalloc call {i}: {w.name} dtype={w.dtype} T_p={w.prompt_len} layer={layer} step={step} cells={C}")
        bufs = gc.gpu_layer(w, layer, n_cells=C)
        q = workloads.make_q(w, layer, step, device="cuda", n_cells=C)
        (o_n, l_n), (o_w, l_w) = _pair(w, layer, step, bufs, q, lw)
        assert np.array_equal(o_n, o_w) and np.array_equal(l_n, l_w), f"call {i}: noalloc bits differ"
        ref_o, ref_l = gc.run_oracle(w, layer, step, gc.host(bufs), workloads.to_numpy(q), lw)
        gc.assert_attn_close(o_n, l_n, ref_o, ref_l, f"noalloc call {i}")
