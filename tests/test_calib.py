"""The stream-read calibration library on the CPU: it loads, exports every
symbol its header declares, and rejects bad arguments before launching
anything (no read runs here: there is no GPU)."""
import ctypes
import os
import re

from paper_2605_30574_amd import calib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "splice_calib.h")


def header():
    return open(HEADER).read()


def test_library_exports_every_declared_symbol():
    declared = sorted(set(re.findall(r"SPLICE_CALIB_API\s+[\w\s\*]+?\b(splice_\w+)\s*\(", header())))
    assert declared == ["splice_calib_stream_read"]
    lib = calib.load_library()
    for name in declared:
        assert hasattr(lib, name), name
    m = re.search(r"#define SPLICE_CALIB_MAX_BLOCKS (\d+)", header())
    assert m and int(m.group(1)) == calib.MAX_BLOCKS


def test_bad_arguments_are_rejected_on_the_host():
    lib = calib.load_library()
    fake = ctypes.c_void_p(1 << 20)   # never dereferenced: every case fails its host check
    sink = ctypes.c_void_p(2 << 20)
    cases = [
        (None, 4096, sink, 1),                           # NULL buffer
        (fake, 4096, None, 1),                           # NULL sink
        (ctypes.c_void_p((1 << 20) + 8), 4096, sink, 1),  # misaligned buffer
        (fake, 0, sink, 1),                              # empty
        (fake, 4100, sink, 1),                           # not a multiple of 16
        (fake, 4096, sink, 0),                           # no work group
        (fake, 4096, sink, calib.MAX_BLOCKS + 1),        # too many work groups
    ]
    for buf, n, snk, blocks in cases:
        assert lib.splice_calib_stream_read(buf, n, snk, blocks, None) == -1, (buf, n, snk, blocks)
