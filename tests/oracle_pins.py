"""Checks that pin the fp64 oracle to things other than itself.

Each ``pin_*`` function takes a loaded oracle library (the real one, or a
copy compiled with a planted mistake) and raises AssertionError when the
oracle disagrees with:
  * torch's float64 scaled_dot_product_attention and logsumexp on the
    unspliced cache (a library routine for the special case L >= N);
  * a literal simulation of Algorithm 1: the prompt-span cache of every
    layer >= L is overwritten in place once, when decoding reaches step W,
    and stays overwritten; attention then runs through the library routine;
  * the ZERO closed form: zeroed keys score exactly 0 and carry no value, so
    lse_zero = logaddexp(lse_ns, ln n) and out_zero = out_ns * exp(lse_ns -
    lse_zero), where (out_ns, lse_ns) is attention over the non-span keys;
  * invariants: donor == clean is bit-identical to unspliced, a cell with
    L = N or W beyond the last step is unspliced, the splice never reaches
    a window that has slid past the span, and results are equivariant under
    permutations of the cells.
None of them re-types the oracle's own formula.
"""
from __future__ import annotations

import math

import numpy as np
import torch
import torch.nn.functional as F

import oracle
import workloads
from workloads import DONOR_BLANK, DONOR_DIFF, DONOR_ZERO

TOL = 1e-12


def f64(a: np.ndarray) -> np.ndarray:
    """Exact float64 values of stored bits (uint16 = bf16, else float32)."""
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


def tiny(donor=DONOR_ZERO, dtype="f32", window=0, span=None, n_steps=16, sink=False):
    w = workloads.get(0)
    kw = dict(donor=donor, dtype=dtype, n_steps=n_steps, sink=sink)
    if window:
        kw.update(local_window=window, global_period=0)
    if span is not None:
        kw.update(span=span)
    return w.with_(**kw)


def layer_arrays(w, layer, seed=0):
    t = workloads.make_layer(w, layer, seed=seed)
    return {k: workloads.to_numpy(v) for k, v in t.items()}


def q_array(w, layer, step, seed=0):
    return workloads.to_numpy(workloads.make_q(w, layer, step, seed=seed))


def run_attn(lib, w, layer, step, arrs, q, lw, window=None, shape=None):
    shape = shape or oracle.shape_of(w, n_cells=lw.shape[0])
    window = w.window(layer) if window is None else window
    return oracle.attn(shape, layer, step, window, w.scale, lw, q, arrs["clean_k"], arrs["clean_v"],
                       arrs["donor_k"], arrs["donor_v"], arrs["gen_k"], arrs["gen_v"], lib=lib)


def sdpa_row(q_row, keys, vals, scale):
    """Library attention for one query against keys/vals [n][D] (float64)."""
    qt = torch.from_numpy(q_row).reshape(1, 1, 1, -1)
    kt = torch.from_numpy(np.ascontiguousarray(keys)).reshape(1, 1, keys.shape[0], -1)
    vt = torch.from_numpy(np.ascontiguousarray(vals)).reshape(1, 1, vals.shape[0], -1)
    out = F.scaled_dot_product_attention(qt, kt, vt, scale=scale).reshape(-1).numpy()
    lse = torch.logsumexp(scale * (kt.reshape(keys.shape[0], -1) @ qt.reshape(-1)), dim=0).item()
    return out, lse


def sdpa_all(w, q, prompt_k, prompt_v, gen_k, gen_v, step, window):
    """Attention of every (cell, head) over [prompt cache per cell] + gen rows 0..step,
    restricted to positions > p - window when window > 0.
    prompt_k: [C][Hkv][T_p][D] float64 (per-cell prompt cache)."""
    C, Hq, D = q.shape
    G = w.group
    Tp = prompt_k.shape[2]
    p = Tp + step
    out = np.empty((C, Hq, D))
    lse = np.empty((C, Hq))
    for c in range(C):
        for h in range(Hq):
            g = h // G
            ks = np.concatenate([prompt_k[c, g], gen_k[c, g, :step + 1]], axis=0)
            vs = np.concatenate([prompt_v[c, g], gen_v[c, g, :step + 1]], axis=0)
            pos = np.arange(ks.shape[0])
            keep = pos > p - window if window > 0 else np.ones_like(pos, dtype=bool)
            out[c, h], lse[c, h] = sdpa_row(q[c, h], ks[keep], vs[keep], w.scale)
    return out, lse


def assert_close(a, b, tol=TOL, what=""):
    err = np.max(np.abs(np.asarray(a) - np.asarray(b))) if np.size(a) else 0.0
    assert err <= tol, f"{what}: max abs err {err:.3e} > {tol:.1e}"


# --------------------------------------------------------------------------------------
# pins
# --------------------------------------------------------------------------------------

def pin_unspliced_matches_library(lib):
    """L >= N: every cell is unspliced; the oracle equals library attention."""
    for w in (tiny(), tiny(dtype="bf16", donor=DONOR_BLANK, sink=True), tiny(window=12)):
        N = w.n_layers
        lw = np.array([[N, 0], [N + 3, 2], [0, w.n_steps]], dtype=np.int32)
        for layer in range(N):
            arrs = layer_arrays(w, layer)
            C = lw.shape[0]
            pk = np.broadcast_to(f64(arrs["clean_k"])[None], (C,) + arrs["clean_k"].shape)
            pv = np.broadcast_to(f64(arrs["clean_v"])[None], (C,) + arrs["clean_v"].shape)
            gk, gv = f64(arrs["gen_k"])[:C], f64(arrs["gen_v"])[:C]
            arrs = dict(arrs, gen_k=np.ascontiguousarray(arrs["gen_k"][:C]),
                        gen_v=np.ascontiguousarray(arrs["gen_v"][:C]))
            for step in (0, 5, w.n_steps - 1):
                q = q_array(w, layer, step)[:C].copy()
                out, lse = run_attn(lib, w, layer, step, arrs, q, lw)
                ref_o, ref_l = sdpa_all(w, f64(q), pk, pv, gk, gv, step, w.window(layer))
                assert_close(out, ref_o, what=f"out {w.name} l={layer} s={step}")
                assert_close(lse, ref_l, what=f"lse {w.name} l={layer} s={step}")


def simulate_algorithm1(w, arrs_by_layer, cell, n_steps):
    """Literal Algorithm 1 for one cell: returns {(layer, step): prompt cache [Hkv][T_p][D]
    (stored bits)} as seen by the forward pass at that step."""
    L, W = cell
    a, b = w.span
    caches = {l: (arrs_by_layer[l]["clean_k"].copy(), arrs_by_layer[l]["clean_v"].copy())
              for l in range(w.n_layers)}
    seen = {}
    for s in range(n_steps):
        if s == W:                                   # the one in-place replacement
            for l in range(w.n_layers):
                if l >= L:                           # patched layers
                    ck, cv = caches[l]
                    if w.donor == DONOR_ZERO:
                        ck[:, a:b] = 0
                        cv[:, a:b] = 0
                    else:
                        ck[:, a:b] = arrs_by_layer[l]["donor_k"][:, a:b]
                        cv[:, a:b] = arrs_by_layer[l]["donor_v"][:, a:b]
        for l in range(w.n_layers):                  # the forward pass reads the cache
            seen[(l, s)] = (caches[l][0].copy(), caches[l][1].copy())
    return seen


def pin_algorithm1_simulation(lib, steps=None):
    """Gather bits and attention equal a literal in-place simulation of Algorithm 1."""
    variants = [tiny(), tiny(dtype="bf16", donor=DONOR_BLANK, sink=True),
                tiny(dtype="bf16", donor=DONOR_DIFF), tiny(window=12),
                tiny(span=(0, 32))]                   # paper-literal full-prompt splice
    for w in variants:
        N, S = w.n_layers, w.n_steps
        arrs = {l: layer_arrays(w, l) for l in range(N)}
        lw = workloads.cell_lw(w)
        C = lw.shape[0]
        sims = [simulate_algorithm1(w, arrs, tuple(lw[c]), S) for c in range(C)]
        shape = oracle.shape_of(w)
        for l in range(N):
            A = arrs[l]
            for s in (range(S) if steps is None else steps):
                win = w.window(l)
                # gather: compare against the simulated cache, slot by slot
                ok, ov, src = oracle.gather(shape, l, s, win, lw, A["clean_k"], A["clean_v"],
                                            A["donor_k"], A["donor_v"], A["gen_k"], A["gen_v"], lib=lib)
                p = w.prompt_len + s
                for c in range(C):
                    sk, sv = sims[c][(l, s)]
                    fk = np.concatenate([sk, A["gen_k"][c, :, :s + 1]], axis=1)
                    fv = np.concatenate([sv, A["gen_v"][c, :, :s + 1]], axis=1)
                    pos = np.arange(fk.shape[1])
                    keep = pos > p - win if win > 0 else np.ones_like(pos, dtype=bool)
                    assert np.array_equal(ok[c], fk[:, keep]), f"gather K {w.name} c={c} l={l} s={s}"
                    assert np.array_equal(ov[c], fv[:, keep]), f"gather V {w.name} c={c} l={l} s={s}"
                    # source map: a slot is donor/zero exactly where the simulated cache
                    # differs in provenance from clean (in span, after the overwrite)
                    L_c, W_c = lw[c]
                    replaced = (l >= L_c) and (s >= W_c)
                    exp_src = np.zeros(fk.shape[1], dtype=np.uint8)
                    exp_src[w.prompt_len:] = oracle.SRC_GEN
                    if replaced:
                        a, b = w.span
                        exp_src[a:b] = oracle.SRC_ZERO if w.donor == DONOR_ZERO else oracle.SRC_DONOR
                    assert np.array_equal(src[c], exp_src[keep]), f"src {w.name} c={c} l={l} s={s}"
                # attention: library routine over the simulated caches
                q = q_array(w, l, s)
                pk = np.stack([f64(sims[c][(l, s)][0]) for c in range(C)])
                pv = np.stack([f64(sims[c][(l, s)][1]) for c in range(C)])
                out, lse = run_attn(lib, w, l, s, A, q, lw)
                ref_o, ref_l = sdpa_all(w, f64(q), pk, pv, f64(A["gen_k"]), f64(A["gen_v"]), s, win)
                assert_close(out, ref_o, what=f"out {w.name} l={l} s={s}")
                assert_close(lse, ref_l, what=f"lse {w.name} l={l} s={s}")


def pin_zero_closed_form(lib):
    """ZERO slots score 0 and carry no value: compare with attention over the
    non-span keys merged with n keys of score 0."""
    for w in (tiny(), tiny(window=12), tiny(span=(0, 32))):
        a, b = w.span
        Tp = w.prompt_len
        for layer in range(w.n_layers):
            arrs = layer_arrays(w, layer)
            lw = np.array([[0, 0]], dtype=np.int32)   # spliced at every step
            for step in (0, 3, w.n_steps - 1):
                win = w.window(layer)
                q = q_array(w, layer, step)[:1].copy()
                A1 = dict(arrs, gen_k=np.ascontiguousarray(arrs["gen_k"][:1]),
                          gen_v=np.ascontiguousarray(arrs["gen_v"][:1]))
                out_z, lse_z = run_attn(lib, w, layer, step, A1, q, lw, window=win,
                                        shape=oracle.shape_of(w, n_cells=1))
                # visible span slots
                p = Tp + step
                j0 = max(0, p - win + 1) if win > 0 else 0
                n = max(0, b - max(a, j0))
                # non-span keys only: drop the span from the visible list, by the library
                keep = [j for j in range(j0, Tp) if not (a <= j < b)]
                G = w.group
                for h in range(w.n_q_heads):
                    g = h // G
                    ks = [f64(arrs["clean_k"][g, keep])]
                    vs = [f64(arrs["clean_v"][g, keep])]
                    i0 = max(0, j0 - Tp)
                    ks.append(f64(arrs["gen_k"][0, g, i0:step + 1]))
                    vs.append(f64(arrs["gen_v"][0, g, i0:step + 1]))
                    o_ns, l_ns = sdpa_row(f64(q[0, h]), np.concatenate(ks), np.concatenate(vs), w.scale)
                    l_exp = np.logaddexp(l_ns, math.log(n)) if n > 0 else l_ns
                    o_exp = o_ns * math.exp(l_ns - l_exp)
                    assert_close(lse_z[0, h], l_exp, 1e-12, f"ZERO lse l={layer} s={step} h={h}")
                    assert_close(out_z[0, h], o_exp, 1e-12, f"ZERO out l={layer} s={step} h={h}")


def pin_invariants(lib):
    """donor == clean, L = N, W past the end, window past the span, cell permutation."""
    w = tiny(dtype="bf16", donor=DONOR_BLANK, sink=True)
    N, S = w.n_layers, w.n_steps
    for layer in range(N):
        arrs = layer_arrays(w, layer)
        lw = workloads.cell_lw(w)
        C = lw.shape[0]
        never = np.array([[N, 0]] * C, dtype=np.int32)
        same = dict(arrs, donor_k=arrs["clean_k"], donor_v=arrs["clean_v"])
        for step in (0, 4, S - 1):
            q = q_array(w, layer, step)
            o_u, l_u = run_attn(lib, w, layer, step, arrs, q, never)
            o_s, l_s = run_attn(lib, w, layer, step, same, q, lw)
            assert np.array_equal(o_u, o_s) and np.array_equal(l_u, l_s), "donor==clean not bit-identical"
            late = lw.copy()
            late[:, 1] = S + step + 1                  # onset beyond the step
            o_w, l_w = run_attn(lib, w, layer, step, arrs, q, late)
            assert np.array_equal(o_u, o_w) and np.array_equal(l_u, l_w), "W beyond step not unspliced"
            # a spliced cell really differs (guards against a splice that does nothing)
            spliced = [c for c in range(C) if layer >= lw[c, 0] and step >= lw[c, 1]]
            o_d, _ = run_attn(lib, w, layer, step, arrs, q, lw)
            for c in range(C):
                differs = not np.array_equal(o_d[c], o_u[c])
                assert differs == (c in spliced), f"cell {c} spliced={c in spliced} differs={differs}"
            # permutation equivariance
            perm = np.random.default_rng(step + 10 * layer).permutation(C)
            Ap = dict(arrs, gen_k=np.ascontiguousarray(arrs["gen_k"][perm]),
                      gen_v=np.ascontiguousarray(arrs["gen_v"][perm]))
            o_p, l_p = run_attn(lib, w, layer, step, Ap, np.ascontiguousarray(q[perm]), np.ascontiguousarray(lw[perm]))
            assert np.array_equal(o_p, o_d[perm]), "not equivariant under cell permutation"
    # window slid past the span: spliced == unspliced (bit-identical)
    ww = tiny(dtype="bf16", donor=DONOR_BLANK, window=8, n_steps=40, sink=True)
    a, b = ww.span
    arrs = layer_arrays(ww, 0)
    lw = np.array([[0, 0], [0, 0]], dtype=np.int32)
    never = np.array([[9, 0], [9, 0]], dtype=np.int32)
    arrs2 = dict(arrs, gen_k=np.ascontiguousarray(arrs["gen_k"][:2]), gen_v=np.ascontiguousarray(arrs["gen_v"][:2]))
    for step in range(ww.n_steps):
        p = ww.prompt_len + step
        q = q_array(ww, 0, step)[:2].copy()
        o_s, l_s = run_attn(lib, ww, 0, step, arrs2, q, lw, window=8, shape=oracle.shape_of(ww, n_cells=2))
        o_u, l_u = run_attn(lib, ww, 0, step, arrs2, q, never, window=8, shape=oracle.shape_of(ww, n_cells=2))
        span_visible = b > p - 8 + 1
        same_result = np.array_equal(o_s, o_u) and np.array_equal(l_s, l_u)
        assert same_result != span_visible, f"window step={step} span_visible={span_visible}"


def pin_selection_staircase(lib):
    """The splice predicate is the staircase of Section 3: off before the
    cutoff layer or the onset step, on from both onwards, monotone."""
    for L in range(0, 5):
        for W in range(0, 5):
            grid = np.array([[oracle.spliced(l, s, L, W, lib) for s in range(8)] for l in range(8)])
            assert np.all(np.diff(grid.astype(int), axis=0) >= 0)
            assert np.all(np.diff(grid.astype(int), axis=1) >= 0)
            assert grid.sum() == (8 - L) * (8 - W)
            assert not grid[L - 1, W] if L > 0 else True
            assert not grid[L, W - 1] if W > 0 else True
            assert grid[L, W]


ALL_PINS = [pin_selection_staircase, pin_unspliced_matches_library, pin_zero_closed_form,
            pin_invariants, pin_algorithm1_simulation]
