"""Pins of the fp64 decode-loop reference (oracle.decoder) on the CPU: each
piece against a property or a library routine that fixes it, and the wiring
of one layer against a closed form."""
import numpy as np
import pytest
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


def test_silu_matches_the_library_routine():
    x = np.concatenate([np.linspace(-40.0, 40.0, 4001), np.random.default_rng(3).standard_normal(5000) * 6.0])
    want = torch.nn.functional.silu(torch.from_numpy(x)).numpy()
    assert np.allclose(ref._silu(x), want, rtol=1e-12, atol=1e-300)


def test_rms_norm_with_gain_and_eps_matches_the_library_routine():
    rng = np.random.default_rng(4)
    x = rng.standard_normal((7, 96)) * np.array([[1e-3], [1e-2], [0.3], [1.0], [3.0], [40.0], [1e-4]])
    gain = 1.0 + 0.5 * rng.standard_normal(96)
    for eps in (1e-6, 1e-2, 0.7):
        want = torch.nn.functional.rms_norm(torch.from_numpy(x), (96,), weight=torch.from_numpy(gain), eps=eps)
        assert np.allclose(ref._rms_norm(x, gain, eps), want.numpy(), rtol=1e-12, atol=1e-15), eps


def _torch_decode_pass(w, m, wt, prompts, lw, gen, tokens, steps):
    """One decode pass of the same model written from torch.nn.functional in
    float64, independently of oracle.decoder: RMSNorm and the projections as
    library calls, the rotary embedding as a complex rotation of the pairs
    (i, i + D/2), q, k, v rounded to bf16 through float32 by torch's own
    conversion, the splice as a list of visible keys (layer >= L and step >= W
    read the span from the donor, or zeros for ZERO) and the attention as
    library SDPA over that list.  gen[l] = (K, V) float64 [C][Hkv][S][D],
    written in place."""
    F = torch.nn.functional
    t = torch.from_numpy
    C, Hq, Hkv, D = len(tokens), w.n_q_heads, w.n_kv_heads, w.head_dim
    G, Tp, half = Hq // Hkv, w.prompt_len, D // 2
    d = m.d_model
    pos = t((Tp + np.maximum(steps, 0)).astype(np.float64))
    ang = pos[:, None] * m.rope_theta ** (-torch.arange(half, dtype=torch.float64) * 2.0 / D)[None, :]
    turn = torch.polar(torch.ones_like(ang), ang)[:, None, :]

    def rotate(x):
        z = torch.complex(x[..., :half], x[..., half:]) * turn
        return torch.cat([z.real, z.imag], dim=-1)

    def bf16(x):
        return x.float().to(torch.bfloat16).to(torch.float64)

    x = t(wt["embed"])[t(tokens)]
    for l, p in enumerate(wt["layers"]):
        P = {k: t(v) for k, v in p.items()}
        h = F.rms_norm(x, (d,), weight=P["norm_1"], eps=m.rms_eps)
        q = bf16(rotate(F.linear(h, P["w_q"].T).view(C, Hq, D)))
        k = bf16(rotate(F.linear(h, P["w_k"].T).view(C, Hkv, D)))
        v = bf16(F.linear(h, P["w_v"].T).view(C, Hkv, D))
        pk = {n: t(prompts[l][n].view(np.int16)).view(torch.bfloat16).to(torch.float64)
              if prompts[l][n] is not None else None for n in ("clean_k", "clean_v", "donor_k", "donor_v")}
        o = torch.zeros(C, Hq, D, dtype=torch.float64)
        for c in range(C):
            s = int(steps[c])
            if s < 0:
                continue
            gen[l][0][c, :, s], gen[l][1][c, :, s] = k[c], v[c]
            p_q = Tp + s
            win = w.window(l)
            vis = [j for j in range(Tp) if win == 0 or j > p_q - win]
            spl = l >= lw[c][0] and s >= lw[c][1]
            ks, vs = [], []
            for j in vis:
                if spl and w.span[0] <= j < w.span[1]:
                    if w.donor == "zero":
                        ks.append(torch.zeros(Hkv, D, dtype=torch.float64))
                        vs.append(torch.zeros(Hkv, D, dtype=torch.float64))
                    else:
                        ks.append(pk["donor_k"][:, j]); vs.append(pk["donor_v"][:, j])
                else:
                    ks.append(pk["clean_k"][:, j]); vs.append(pk["clean_v"][:, j])
            for i in range(s + 1):
                if win == 0 or Tp + i > p_q - win:
                    ks.append(gen[l][0][c, :, i]); vs.append(gen[l][1][c, :, i])
            K = torch.stack(ks, dim=1).repeat_interleave(G, dim=0)   # [Hq][n][D]
            V = torch.stack(vs, dim=1).repeat_interleave(G, dim=0)
            o[c] = F.scaled_dot_product_attention(q[c][:, None, :], K, V, scale=D ** -0.5)[:, 0, :]
        x = x + F.linear(o.reshape(C, Hq * D), P["w_o"].T)
        h2 = F.rms_norm(x, (d,), weight=P["norm_2"], eps=m.rms_eps)
        x = x + F.linear(F.silu(F.linear(h2, P["w_gate"].T)) * F.linear(h2, P["w_up"].T), P["w_down"].T)
    return F.linear(F.rms_norm(x, (d,), weight=t(wt["norm_f"]), eps=m.rms_eps), t(wt["lm_head"]).T).numpy()


@pytest.mark.parametrize("donor,window", [("blank", 0), ("zero", 5), ("diff", 0)])
def test_decode_passes_match_a_torch_functional_model(donor, window):
    """Two layers, a prompt with a spliced span, non-unit norm gains and
    eps > 0, cells spliced at different (L, W), one cell finishing: every
    pass's logits and every appended cache row agree with the torch model."""
    w = oracle_pins.tiny(dtype="bf16", donor=donor, sink=True, window=window)
    m = ModelConfig(d_model=96, d_ff=160, vocab=64, eos=5, rms_eps=1e-2)
    wt = _f64(make_weights(w, m, dtype=torch.float32))
    rng = np.random.default_rng(5)
    for L in wt["layers"]:
        L["norm_1"] = 1.0 + 0.3 * rng.standard_normal(m.d_model)
        L["norm_2"] = 1.0 + 0.3 * rng.standard_normal(m.d_model)
    wt["norm_f"] = 1.0 + 0.3 * rng.standard_normal(m.d_model)
    lw = np.array([[0, 0], [1, 1], [2, 0], [0, 2], [1, 0], [2, 2]], dtype=np.int32)
    C = lw.shape[0]
    prompts = []
    for l in range(w.n_layers):
        a = oracle_pins.layer_arrays(w, l)
        prompts.append({k: a[k] for k in ("clean_k", "clean_v", "donor_k", "donor_v")})
    dec = ref.ReferenceDecoder(w, m, wt, prompts, lw)
    shp = (C, w.n_kv_heads, w.n_steps, w.head_dim)
    gen = [(torch.zeros(shp, dtype=torch.float64), torch.zeros(shp, dtype=torch.float64)) for _ in range(w.n_layers)]
    tokens = np.array([11, 3, 40, 7, 63, 0])
    steps = np.zeros(C, dtype=np.int32)
    for it in range(4):
        if it == 2:
            steps[3] = -1   # a cell that stopped
        got = dec.forward(tokens, steps)
        want = _torch_decode_pass(w, m, wt, prompts, lw, gen, tokens, steps)
        act = steps >= 0
        assert np.allclose(got[act], want[act], rtol=1e-10, atol=1e-10 * np.abs(want[act]).max()), it
        for l in range(w.n_layers):
            assert np.array_equal(ref.from_bf16_bits(dec.gen_k[l]), gen[l][0].numpy()), (it, l)
            assert np.array_equal(ref.from_bf16_bits(dec.gen_v[l]), gen[l][1].numpy()), (it, l)
        tokens = (tokens * 7 + 3) % m.vocab
        steps = np.where(steps >= 0, steps + 1, steps)


MUTANTS = [   # plausible mistakes in the decode loop, planted in a copy of its source
    ("silu sign", "x / (1.0 + np.exp(-x))", "x / (1.0 + np.exp(x))"),
    ("rope direction", "a * c - b * s, b * c + a * s", "a * c + b * s, b * c - a * s"),
    ("rope pairs adjacent", "a, b = x[..., :half], x[..., half:]", "a, b = x[..., 0::2], x[..., 1::2]"),
    ("norm gain dropped", "keepdims=True) + eps) * gain", "keepdims=True) + eps)"),
    ("eps outside the root", "np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)",
     "(np.sqrt(np.mean(x * x, axis=-1, keepdims=True)) + eps)"),
    ("position off by one", "pos = w.prompt_len + np.maximum(steps, 0)",
     "pos = w.prompt_len + np.maximum(steps, 0) + 1"),
    ("attention residual dropped", "x = x + o.reshape(C, Hq * D) @ p[\"w_o\"]", "x = o.reshape(C, Hq * D) @ p[\"w_o\"]"),
    ("gate and up swapped", "_silu(h2 @ p[\"w_gate\"]) * (h2 @ p[\"w_up\"])", "_silu(h2 @ p[\"w_up\"]) * (h2 @ p[\"w_gate\"])"),
    ("second norm reuses the first gain", "h2 = _rms_norm(x, p[\"norm_2\"]", "h2 = _rms_norm(x, p[\"norm_1\"]"),
    ("value row stored as key", "self.gen_v[l][c, :, s] = v[c]", "self.gen_v[l][c, :, s] = k[c]"),
    ("final norm dropped", "return _rms_norm(x, wt[\"norm_f\"], m.rms_eps) @ wt[\"lm_head\"]",
     "return x @ wt[\"lm_head\"]"),
]


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_each_planted_mistake_is_caught(name, old, new, monkeypatch):
    """The torch comparison above fails for every planted mistake (the
    mistake is planted in a copy of the reference's source, on the CPU)."""
    import types
    src = open(ref.__file__).read()
    assert src.count(old) == 1, name
    mod = types.ModuleType("decoder_mutant")
    mod.__dict__["__package__"] = "oracle"
    exec(compile(src.replace(old, new).replace("from . import", "from oracle import"), "decoder_mutant", "exec"),
         mod.__dict__)
    caught = False
    for donor, window in (("blank", 0), ("zero", 5)):
        monkeypatch.setattr(ref, "ReferenceDecoder", mod.ReferenceDecoder)
        try:
            test_decode_passes_match_a_torch_functional_model(donor, window)
        except AssertionError:
            caught = True
        finally:
            monkeypatch.undo()
        if caught:
            break
    assert caught, f"mutant not caught: {name}"
