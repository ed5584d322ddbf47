"""Plant plausible mistakes in a copy of the oracle's C source and check that
at least one pin catches each of them (CPU only; the mistakes live in a
temporary copy, never in the committed oracle)."""
import os
import tempfile

import pytest

import oracle
import oracle_pins as pins
from oracle.build import SRC, build

MUTANTS = {
    "layer_strict": ("return layer >= L && step >= W;", "return layer > L && step >= W;"),
    "onset_strict": ("return layer >= L && step >= W;", "return layer >= L && step > W;"),
    "span_end_inclusive": ("int in_span = j >= sh->span_lo && j < sh->span_hi;",
                           "int in_span = j >= sh->span_lo && j <= sh->span_hi;"),
    "drop_own_gen_row": ("for (i = i0; i <= step; ++i) {", "for (i = i0; i < step; ++i) {"),
    "window_off_by_one": ("return window > 0 ? p - window + 1 : 0;", "return window > 0 ? p - window : 0;"),
    "gqa_modulo": ("int g = h / G;", "int g = h % sh->n_kv_heads;"),
    "drop_scale": ("score[t] = call->scale * dot;", "score[t] = dot;"),
    "zero_masked": ("score[t] = call->scale * dot;", "score[t] = bk ? call->scale * dot : -INFINITY;"),
    "softmax_sign": ("double wgt = exp(score[t] - m);", "double wgt = exp(m - score[t]);"),
    "lse_drop_max": ("lse[r] = m + log(Z);", "lse[r] = log(Z);"),
    "donor_reads_clean": ("return want_v ? donor_v : donor_k;", "return want_v ? clean_v : clean_k;"),
    "value_uses_key": ("const void *bv = row_base(sh, &keys[t], c, g, 1,", "const void *bv = row_base(sh, &keys[t], c, g, 0,"),
    "gen_head_index": ("*off = (((size_t)c * sh->n_kv_heads + g) * sh->gen_capacity + (size_t)kr->row) * D;",
                       "*off = (((size_t)c * sh->n_kv_heads) * sh->gen_capacity + (size_t)kr->row) * D;"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, tmp_path):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) >= 1, f"mutation anchor missing: {old}"
    mutated = src.replace(old, new)
    path = tmp_path / "mutant.c"
    path.write_text(mutated)
    lib_path = str(tmp_path / f"libmutant_{name}.so")
    build(str(path), lib_path)
    lib = oracle.load(lib_path)
    caught = []
    for pin in pins.ALL_PINS:
        try:
            if pin is pins.pin_algorithm1_simulation:
                pin(lib, steps=(0, 1, 4, 5, 15))
            else:
                pin(lib)
        except (AssertionError, RuntimeError, ValueError):
            caught.append(pin.__name__)
            break
    assert caught, f"mutant {name} passed every pin"
