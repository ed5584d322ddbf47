"""The decode-loop GPU test's bars are the ones derived from the attention
bar (tests/decode_bar.py): a bar can only move with its derivation."""
import decode_bar
import test_gpu_decode as t


def test_gpu_decode_bars_are_the_derived_ones():
    got = decode_bar.derive()
    assert (t.LOGIT_REL, t.ROW_REL, t.ROW_FLIP_FRAC) == (got["logit_rel"], got["row_rel"], got["row_flip_frac"]), got


def test_row_deviation_measures_what_it_says():
    import numpy as np
    from oracle import decoder as ref
    want = ref.to_bf16_bits(np.array([[1.0, -2.0, 0.0, 4.0]]))
    got = ref.to_bf16_bits(np.array([[1.0, -2.0, 0.0, 4.5]]))
    dev, flip = decode_bar.row_deviation(want, got)
    rms = np.sqrt((1 + 4 + 16) / 3)          # the written (nonzero) elements
    assert abs(dev - 0.5 / rms) < 1e-12 and abs(flip - 1 / 3) < 1e-12
