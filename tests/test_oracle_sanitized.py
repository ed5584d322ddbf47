"""The C oracle built with AddressSanitizer and UndefinedBehaviorSanitizer
(gcc, host code only): its attention and gather run on the tiny and
bf16 workload shapes -- windows, the ZERO donor, an empty prompt, a span
over the whole prompt, every step -- in a child process with the ASan runtime
preloaded and every report fatal, and give the bits of the normal build."""
import os
import subprocess
import sys
import textwrap

import numpy as np
import pytest

import oracle
from oracle import build as obuild

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

CASES = textwrap.dedent('''
    import sys
    sys.path[:0] = [{root!r}, {tests!r}]
    import numpy as np
    import oracle, oracle_pins, workloads
    from workloads import DONOR_BLANK, DONOR_DIFF, DONOR_ZERO
    lib = oracle.load({lib!r})
    t = oracle_pins.tiny
    cases = [t(), t(donor=DONOR_BLANK, dtype="bf16", sink=True), t(donor=DONOR_ZERO, window=5),
             t(donor=DONOR_DIFF, dtype="bf16", window=40), t(span=(0, 32)), t().with_(prompt_len=0, span=(0, 0))]
    res = {{}}
    for i, w in enumerate(cases):
        lw = workloads.cell_lw(w)
        osh = oracle.shape_of(w)
        for layer in range(w.n_layers):
            arr = oracle_pins.layer_arrays(w, layer)
            for step in range(w.n_steps):
                q = oracle_pins.q_array(w, layer, step)
                o, l = oracle.attn(osh, layer, step, w.window(layer), w.scale, lw, q, arr["clean_k"], arr["clean_v"],
                                   arr["donor_k"], arr["donor_v"], arr["gen_k"], arr["gen_v"], lib=lib)
                k, v, s = oracle.gather(osh, layer, step, w.window(layer), lw, arr["clean_k"], arr["clean_v"],
                                        arr["donor_k"], arr["donor_v"], arr["gen_k"], arr["gen_v"], lib=lib)
                res[f"{{i}}_{{layer}}_{{step}}_o"] = o
                res[f"{{i}}_{{layer}}_{{step}}_l"] = l
                res[f"{{i}}_{{layer}}_{{step}}_k"] = k.view(np.uint8)
                res[f"{{i}}_{{layer}}_{{step}}_v"] = v.view(np.uint8)
                res[f"{{i}}_{{layer}}_{{step}}_s"] = s
    np.savez({out!r}, **res)
''')


def _run(lib, out, env):
    code = CASES.format(root=ROOT, tests=os.path.join(ROOT, "tests"), lib=lib, out=out)
    return subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True, timeout=600)


def test_sanitized_oracle_is_clean_and_gives_the_same_bits(tmp_path):
    asan = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
    if not asan or not os.path.exists(asan):
        pytest.skip("gcc's AddressSanitizer runtime is not installed")
    lib_san = obuild.build(out=str(tmp_path / "liboracle_san.so"),
                           extra=("-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                                  "-fno-omit-frame-pointer", "-g"))
    env = dict(os.environ)
    env.update(LD_PRELOAD=asan, ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1", OMP_NUM_THREADS="4")
    r = _run(lib_san, str(tmp_path / "san.npz"), env)
    assert r.returncode == 0, r.stderr[-4000:]
    assert "ERROR: AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr, r.stderr[-4000:]
    plain = dict(os.environ, OMP_NUM_THREADS="4")
    r = _run(oracle.build.LIB if hasattr(oracle, "build") else obuild.LIB, str(tmp_path / "plain.npz"), plain)
    assert r.returncode == 0, r.stderr[-4000:]
    a, b = np.load(tmp_path / "san.npz"), np.load(tmp_path / "plain.npz")
    assert sorted(a.files) == sorted(b.files) and len(a.files) > 100
    for k in a.files:
        assert np.array_equal(a[k], b[k]), k
