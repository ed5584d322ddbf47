"""The bench's algorithmic bytes per call, pinned to the oracle's gather.

bench.call_bytes, bench.step_bytes and bench.forked_bytes state what a
call must move at the least (each prompt row once however many cells read it, each cell's own
generated rows, q, out and lse).  Here the same total is counted from the
oracle's source map instead: the distinct (cache, prompt slot) pairs that
any computed cell reads (ZERO slots read nothing), plus every computed
cell's visible generated rows, on small versions of every workload's
structure (donor kinds, windows, a full-prompt span, never-spliced cells).
The bench's own arithmetic (window, span clipping, splice predicate) is not
used by the count."""
import numpy as np
import pytest

import bench
import oracle
import workloads

SRC_CLEAN, SRC_DONOR, SRC_ZERO, SRC_GEN = 0, 1, 2, 3


def small_workloads():
    base = workloads.get(1).with_(n_layers=4, prompt_len=96, span=(16, 80), n_steps=24,
                                  cells=((0, 0), (1, 4), (2, 16), (4, 0), (3, 2), (4, 8)))
    return [
        workloads.get(0),                                                  # tiny fp32, ZERO
        base,                                                              # BLANK
        base.with_(donor="zero"),
        base.with_(donor="diff"),
        base.with_(local_window=40, global_period=2),                      # local/global layers
        base.with_(span=(0, 96)),                                          # the whole prompt spliced
        base.with_(cells=((4, 0), (4, 8))),                                # never spliced (L = N)
    ]


def arrays(w, layer):
    t = workloads.make_layer(w, layer, seed=3)
    return {k: workloads.to_numpy(v) for k, v in t.items()}


def counted_bytes(w, A, layer, step, lw, cells):
    """Bytes from the oracle's source map of the cells in `cells` at `step`."""
    e = w.elem_bytes
    row = 2 * w.n_kv_heads * w.head_dim * e
    shape = oracle.shape_of(w)
    _, _, src = oracle.gather(shape, layer, step, w.window(layer), lw, A["clean_k"], A["clean_v"],
                              A["donor_k"], A["donor_v"], A["gen_k"], A["gen_v"])
    n_prompt = int(np.count_nonzero(src[0] != SRC_GEN))
    jp0 = w.prompt_len - n_prompt            # visible prompt slots are jp0 .. Tp - 1, in order
    prompt_rows = set()
    gen_rows = 0
    for c in cells:
        for t in range(src.shape[1]):
            s = int(src[c, t])
            if s in (SRC_CLEAN, SRC_DONOR):
                prompt_rows.add((s, jp0 + t))
            elif s == SRC_GEN:
                gen_rows += 1
    total = (len(prompt_rows) + gen_rows) * row
    total += len(cells) * w.n_q_heads * w.head_dim * e              # q
    total += len(cells) * w.n_q_heads * (4 * w.head_dim + 4)        # out + lse
    return total, gen_rows


@pytest.mark.parametrize("wi", range(7))
def test_call_bytes_match_the_oracle_source_map(wi):
    w = small_workloads()[wi]
    lw = workloads.cell_lw(w)
    cells = list(range(w.n_cells))
    for layer in range(w.n_layers):
        A = arrays(w, layer)
        for step in sorted({0, 1, 2, 4, 5, 8, 16, w.n_steps - 1}):
            want, _ = counted_bytes(w, A, layer, step, lw, cells)
            got = bench.call_bytes(w, layer, step, bench.spliced_flags(w, layer, step))
            assert got == want, (w.name, wi, layer, step, got, want)


@pytest.mark.parametrize("wi", [1, 3, 4])
def test_step_bytes_match_the_oracle_source_map(wi):
    """A decode pass: each cell at its own step (finished cells move nothing);
    the current token's row is read from the input and written to the cache,
    so it counts twice, and is not read back."""
    w = small_workloads()[wi]
    lw = workloads.cell_lw(w)
    e = w.elem_bytes
    row = 2 * w.n_kv_heads * w.head_dim * e
    steps = np.array([0, 7, -1, 23, 5, 12][:w.n_cells], dtype=np.int32)
    for layer in range(w.n_layers):
        A = arrays(w, layer)
        # per active cell: its own gather at its own step; prompt rows pooled
        prompt_rows = set()
        total = 0
        for c, s in enumerate(steps.tolist()):
            if s < 0:
                continue
            shape = oracle.shape_of(w)
            _, _, src = oracle.gather(shape, layer, s, w.window(layer), lw, A["clean_k"], A["clean_v"],
                                      A["donor_k"], A["donor_v"], A["gen_k"], A["gen_v"])
            n_prompt = int(np.count_nonzero(src[c] != SRC_GEN))
            jp0 = w.prompt_len - n_prompt
            for t in range(src.shape[1]):
                k = int(src[c, t])
                if k in (SRC_CLEAN, SRC_DONOR):
                    prompt_rows.add((k, jp0 + t))
            n_gen = int(np.count_nonzero(src[c] == SRC_GEN))
            total += (n_gen - 1) * row + 2 * row
            total += w.n_q_heads * w.head_dim * e + w.n_q_heads * (4 * w.head_dim + 4)
        total += len(prompt_rows) * row
        got = bench.step_bytes(w, layer, steps.tolist(), w.cells)
        assert got == total, (w.name, layer, got, total)


@pytest.mark.parametrize("wi", [1, 3, 4, 6])
def test_forked_bytes_match_the_oracle_source_map(wi):
    """A forked sweep computes the trunk and the cells that have diverged
    (L < N and step >= W); below its onset W a diverged cell's generated
    rows are the trunk's (nothing is spliced before W, so the cell is the
    clean run there), so each (owner, row) pair is read once.  Dormant
    cells read nothing and still receive out and lse."""
    w = small_workloads()[wi].with_(cells=((4, 0), (0, 0), (1, 4), (2, 16), (3, 2), (0, 8)))
    lw = workloads.cell_lw(w)
    N, trunk = w.n_layers, 0
    e = w.elem_bytes
    row = 2 * w.n_kv_heads * w.head_dim * e
    for layer in range(N):
        A = arrays(w, layer)
        for step in (0, 3, 4, 9, 16, w.n_steps - 1):
            div = [c for c, (L, W) in enumerate(w.cells) if c == trunk or (L < N and step >= W)]
            shape = oracle.shape_of(w)
            _, _, src = oracle.gather(shape, layer, step, w.window(layer), lw, A["clean_k"], A["clean_v"],
                                      A["donor_k"], A["donor_v"], A["gen_k"], A["gen_v"])
            n_prompt = int(np.count_nonzero(src[0] != SRC_GEN))
            jp0 = w.prompt_len - n_prompt
            prompt_rows, gen_rows = set(), set()
            for c in div:
                n_gen = int(np.count_nonzero(src[c] == SRC_GEN))
                for t in range(src.shape[1]):
                    k = int(src[c, t])
                    if k in (SRC_CLEAN, SRC_DONOR):
                        prompt_rows.add((k, jp0 + t))
                for r in range(step + 1 - n_gen, step + 1):
                    owner = trunk if (c == trunk or r < w.cells[c][1]) else c
                    gen_rows.add((owner, r))
            want = (len(prompt_rows) + len(gen_rows)) * row
            want += len(div) * w.n_q_heads * w.head_dim * e
            want += w.n_cells * w.n_q_heads * (4 * w.head_dim + 4)
            got = bench.forked_bytes(w, layer, step, list(w.cells), trunk)
            assert got == want, (w.name, layer, step, got, want)
