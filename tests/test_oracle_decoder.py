"""Pins of the fp64 decode-loop reference (oracle.decoder) on the CPU: each
piece against a property or a library routine that fixes it, and the wiring
of one layer against a closed form."""
import numpy as np
import torch

import oracle
import oracle_pins
from oracle import decoder as ref
import workloads
from workloads.model import ModelConfig, make_weights


def test_bf16_rounding_matches_the_library_conversion():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(20000) * 10.0 ** rng.integers(-6, 6, 20000),
                        [0.0, -0.0, 1.0, 1.00390625, 1.0078125, 1.01171875, 65504.0]])
    want = torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ref.to_bf16_bits(x), want)
    assert np.array_equal(ref.from_bf16_bits(want), torch.from_numpy(want.view(np.int16)).view(torch.bfloat16)
                          .to(torch.float64).numpy())


def test_rope_is_a_rotation_of_relative_position():
    rng = np.random.default_rng(1)
    q, k = rng.standard_normal((3, 2, 64)), rng.standard_normal((3, 2, 64))
    assert np.allclose(ref._rope(q, np.zeros(3), 1e6), q)                      # position 0: identity
    r = ref._rope(q, np.array([5, 40, 1000]), 1e4)
    assert np.allclose(np.linalg.norm(r, axis=-1), np.linalg.norm(q, axis=-1))  # norms kept
    # q.k after rotation depends on the position difference only
    d1 = np.sum(ref._rope(q, np.array([7, 7, 7]), 1e4) * ref._rope(k, np.array([3, 3, 3]), 1e4), -1)
    d2 = np.sum(ref._rope(q, np.array([104, 104, 104]), 1e4) * ref._rope(k, np.array([100, 100, 100]), 1e4), -1)
    assert np.allclose(d1, d2)
    # one pair by hand: (x_0, x_{D/2}) turned by the angle pos
    x = np.zeros((1, 1, 4)); x[0, 0, 0] = 1.0
    y = ref._rope(x, np.array([0.5]), 1e4)
    assert np.allclose(y[0, 0], [np.cos(0.5), 0.0, np.sin(0.5), 0.0])


def test_rms_norm_has_unit_rms():
    x = np.random.default_rng(2).standard_normal((5, 96)) * 3.0
    y = ref._rms_norm(x, np.ones(96), 0.0)
    assert np.allclose(np.sqrt(np.mean(y * y, -1)), 1.0)


def _tiny():
    w = oracle_pins.tiny(dtype="bf16", donor="blank", sink=True)
    m = ModelConfig(d_model=96, d_ff=160, vocab=64, eos=5)
    return w, m


def _f64(wt):
    f = lambda t: t.double().numpy()
    return dict(embed=f(wt["embed"]), lm_head=f(wt["lm_head"]), norm_f=f(wt["norm_f"]),
                layers=[{k: f(v) for k, v in L.items()} for L in wt["layers"]])


def test_one_layer_without_a_prompt_is_its_closed_form():
    """T_p = 0 and step 0: each cell's only key is its own row, so the
    attention output is v (as stored, bf16) in every head of the group."""
    w, m = _tiny()
    w = w.with_(prompt_len=0, span=(0, 0), n_layers=1, sink=False)
    wt = _f64(make_weights(w, m, dtype=torch.float32, n_layers=1))
    C = 3
    e = np.zeros((w.n_kv_heads, 0, w.head_dim), dtype=np.uint16)
    prompts = [dict(clean_k=e, clean_v=e, donor_k=e, donor_v=e)]
    dec = ref.ReferenceDecoder(w, m, wt, prompts, [[0, 0]] * C)
    tokens = np.array([3, 17, 60])
    got = dec.forward(tokens, np.zeros(C, dtype=np.int32))
    # closed form
    p = wt["layers"][0]
    x = wt["embed"][tokens]
    h = x / np.sqrt(np.mean(x * x, -1, keepdims=True) + m.rms_eps)
    v = ref.from_bf16_bits(ref.to_bf16_bits((h @ p["w_v"]).reshape(C, w.n_kv_heads, w.head_dim)))
    G = w.n_q_heads // w.n_kv_heads
    o = np.repeat(v, G, axis=1).reshape(C, -1)
    x = x + o @ p["w_o"]
    h2 = x / np.sqrt(np.mean(x * x, -1, keepdims=True) + m.rms_eps)
    g = h2 @ p["w_gate"]
    x = x + (g / (1 + np.exp(-g)) * (h2 @ p["w_up"])) @ p["w_down"]
    want = x / np.sqrt(np.mean(x * x, -1, keepdims=True) + m.rms_eps) @ wt["lm_head"]
    assert np.allclose(got, want, rtol=1e-12, atol=1e-12)
    # the appended rows are the stored k, v
    assert np.array_equal(dec.gen_v[0][:, :, 0], ref.to_bf16_bits((h @ p["w_v"]).reshape(C, w.n_kv_heads, w.head_dim)))


def test_greedy_takes_the_lowest_index_of_a_tie():
    assert list(ref.greedy(np.array([[1.0, 3.0, 3.0, 2.0], [5.0, 5.0, 5.0, 5.0]]))) == [1, 0]
