"""Workload shapes and the seeded input recipe (CPU only)."""
import numpy as np
import torch

import workloads
from workloads import DONOR_BLANK, DONOR_DIFF, DONOR_ZERO


def test_shapes_and_grids():
    w = workloads.WORKLOADS
    assert [x.n_cells for x in w] == [6, 80, 64, 48, 128]
    assert [x.prompt_len for x in w] == [32, 256, 1024, 4096, 8192]
    assert [x.span for x in w] == [(4, 28), (40, 236), (43, 1003), (64, 4064), (128, 8128)]
    assert [x.n_steps for x in w] == [16, 512, 256, 128, 1024]
    assert [x.donor for x in w] == [DONOR_ZERO, DONOR_BLANK, DONOR_ZERO, DONOR_BLANK, DONOR_DIFF]
    assert [x.group for x in w] == [2, 4, 4, 2, 4]
    assert w[4].cells[-1] == (36, 64) and (36, 128) not in w[4].cells
    g = w[3]
    assert [g.window(l) for l in range(12)] == [1024] * 5 + [0] + [1024] * 5 + [0]
    assert all(x.window(0) == 0 for x in (w[0], w[1], w[2], w[4]))


def test_inputs_deterministic_and_shaped():
    w = workloads.get(1).with_(n_steps=8, cells=((0, 0), (4, 1), (36, 2)))
    a = workloads.make_layer(w, 3, seed=7)
    b = workloads.make_layer(w, 3, seed=7)
    c = workloads.make_layer(w, 4, seed=7)
    for k in a:
        assert torch.equal(a[k], b[k])
        assert not torch.equal(a[k], c[k])
    assert a["clean_k"].shape == (8, 256, 128) and a["clean_k"].dtype == torch.bfloat16
    assert a["gen_k"].shape == (3, 8, 8, 128)
    span = slice(*w.span)
    # BLANK donor: scaffold identical, span redrawn
    assert torch.equal(a["donor_k"][:, :40], a["clean_k"][:, :40])
    assert torch.equal(a["donor_v"][:, 236:], a["clean_v"][:, 236:])
    assert not torch.equal(a["donor_k"][:, span], a["clean_k"][:, span])
    # sink outlier at prompt position 0, channels 0..3 of K
    assert a["clean_k"][:, 0, :4].float().abs().mean() > 10 * a["clean_k"][:, 1:, :4].float().abs().mean()
    q = workloads.make_q(w, 3, 5, seed=7)
    assert q.shape == (3, 32, 128)
    assert np.array_equal(workloads.to_numpy(q), workloads.to_numpy(workloads.make_q(w, 3, 5, seed=7)))


def test_zero_and_diff_donors():
    z = workloads.make_layer(workloads.get(0), 0)
    assert z["donor_k"] is None and z["donor_v"] is None
    w = workloads.get(4).with_(prompt_len=64, span=(4, 60), n_steps=4, cells=((0, 0),))
    d = workloads.make_layer(w, 0)
    assert not torch.equal(d["donor_k"][:, :4], d["clean_k"][:, :4])
