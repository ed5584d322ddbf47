"""The fp64 oracle against library routines, a literal Algorithm 1 simulation,
the ZERO closed form and the method's invariants (CPU only)."""
import pytest

import oracle_pins as pins


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda f: f.__name__)
def test_pin(pin, oracle_lib):
    pin(oracle_lib)


def test_visible_len_matches_definition(oracle_lib):
    import oracle
    sh = oracle.make_shape(1, 4, 2, 64, 32, (4, 28), 64, True, 4)
    for step in range(0, 60):
        assert oracle.visible_len(sh, step, 0, oracle_lib) == 32 + step + 1
        # window 10: the 10 positions p-9 .. p
        assert oracle.visible_len(sh, step, 10, oracle_lib) == 10
    sh0 = oracle.make_shape(1, 4, 2, 64, 0, (0, 0), 8, True, 4)   # empty prompt
    assert oracle.visible_len(sh0, 3, 0, oracle_lib) == 4
