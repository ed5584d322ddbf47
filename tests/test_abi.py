"""The C-ABI library on the CPU: it loads, exports every symbol the header
declares, and rejects bad arguments on the host before touching a device
(no compute call runs here: there is no GPU)."""
import ctypes
import os
import re

import pytest

import paper_2605_30574_amd as sp
from paper_2605_30574_amd import splice as S

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "splice_attn.h")


def header_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"SPLICE_API\s+[\w\s\*]+?\b(splice_\w+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    declared = header_functions()
    assert set(declared) == set(S.EXPORTS), declared
    lib = sp.load_library()
    for name in declared:
        assert hasattr(lib, name), name
    assert sp.splice_abi_version() == 6


def test_single_hip_runtime_mapped():
    sp.load_library()
    maps = [ln.split()[-1] for ln in open("/proc/self/maps") if "libamdhip64" in ln]
    assert len(set(maps)) == 1, set(maps)


def test_status_strings():
    for st in (0, -1, -2, -3, -4, -5):
        assert sp.splice_status_str(st) and sp.splice_status_str(st) != "unknown status"
    assert sp.splice_status_str(-99) == "unknown status"


def _shape(**kw):
    base = dict(n_cells=6, n_layers=2, n_q_heads=4, n_kv_heads=2, head_dim=64, prompt_len=32,
                span=(4, 28), gen_capacity=16, donor_zero=True, dtype="f32")
    base.update(kw)
    return sp.make_shape(**base)


def _vis(shape, call):
    lib = sp.load_library()
    return lib.splice_visible_len(ctypes.byref(shape), ctypes.byref(call))


@pytest.mark.parametrize("kw,status", [
    (dict(n_q_heads=3), sp.SPLICE_ESHAPE),              # Hq % Hkv != 0
    (dict(n_q_heads=12, n_kv_heads=4), sp.SPLICE_EUNSUPPORTED),  # G = 3
    (dict(head_dim=96), sp.SPLICE_EUNSUPPORTED),
    (dict(head_dim=0), sp.SPLICE_ESHAPE),
    (dict(span=(5, 4)), sp.SPLICE_ESHAPE),
    (dict(span=(-1, 4)), sp.SPLICE_ESHAPE),
    (dict(span=(4, 33)), sp.SPLICE_ESHAPE),
    (dict(n_cells=-1), sp.SPLICE_ESHAPE),
    (dict(n_cells=257), sp.SPLICE_EUNSUPPORTED),
    (dict(gen_capacity=0), sp.SPLICE_ESHAPE),
    (dict(n_layers=0), sp.SPLICE_ESHAPE),
])
def test_bad_shape(kw, status):
    assert _vis(_shape(**kw), sp.make_call(0, 0, 0, 1.0)) == status


def test_bad_enums():
    sh = _shape()
    sh.donor_kind = 7
    assert _vis(sh, sp.make_call(0, 0, 0, 1.0)) == sp.SPLICE_EINVAL
    sh = _shape()
    sh.dtype = 9
    assert _vis(sh, sp.make_call(0, 0, 0, 1.0)) == sp.SPLICE_EINVAL


@pytest.mark.parametrize("call,status", [
    (sp.make_call(2, 0, 0, 1.0), sp.SPLICE_ESHAPE),        # layer >= N
    (sp.make_call(-1, 0, 0, 1.0), sp.SPLICE_ESHAPE),
    (sp.make_call(0, 16, 0, 1.0), sp.SPLICE_ESHAPE),       # step >= gen_capacity
    (sp.make_call(0, -1, 0, 1.0), sp.SPLICE_ESHAPE),
    (sp.make_call(0, 0, -3, 1.0), sp.SPLICE_ESHAPE),       # negative window
    (sp.make_call(0, 0, 0, float("nan")), sp.SPLICE_EINVAL),
    (sp.make_call(0, 0, 0, float("inf")), sp.SPLICE_EINVAL),
    (sp.make_call(0, 0, 0, 0.0), sp.SPLICE_EINVAL),         # the bf16 kernels need scale > 0
    (sp.make_call(0, 0, 0, -0.125), sp.SPLICE_EINVAL),
    (sp.make_call(0, 0, 0, 1.0, split_keys=100), sp.SPLICE_EINVAL),
    (sp.make_call(0, 0, 0, 1.0, split_keys=32), sp.SPLICE_EINVAL),
])
def test_bad_call(call, status):
    assert _vis(_shape(), call) == status


def test_visible_len_matches_oracle():
    import oracle
    for (Tp, span, cap) in ((32, (4, 28), 16), (0, (0, 0), 8), (4096, (64, 4064), 128)):
        sh = _shape(prompt_len=Tp, span=span, gen_capacity=cap)
        osh = oracle.make_shape(6, 4, 2, 64, Tp, span, cap, True, 4)
        for step in sorted({0, 1, cap // 2, cap - 1}):
            for window in (0, 1, 7, 1024, 5000):
                assert sp.splice_visible_len(sh, sp.make_call(0, step, window, 1.0)) == \
                    oracle.visible_len(osh, step, window)


def test_null_and_workspace_errors_before_device_access():
    lib = sp.load_library()
    sh = _shape()
    call = sp.make_call(1, 5, 0, 0.125)
    lw = (ctypes.c_int32 * 12)(*([0, 0] * 6))
    fake = ctypes.c_void_p(0x1000)   # never dereferenced: validation fails first
    args = [fake] * 10
    # missing cell_LW
    assert lib.splice_decode_attn(ctypes.byref(sh), ctypes.byref(call), None, *args, 0, None) == sp.SPLICE_EINVAL
    # ZERO donor must not get buffers: args[3], args[4] are donor pointers here
    assert lib.splice_decode_attn(ctypes.byref(sh), ctypes.byref(call), lw, *args, 1 << 20, None) == sp.SPLICE_EINVAL
    zargs = [fake, fake, fake, None, None, fake, fake, fake, fake, ctypes.c_void_p(0x2000)]
    need = sp.splice_decode_attn_workspace_bytes(sh, call)
    assert lib.splice_decode_attn(ctypes.byref(sh), ctypes.byref(call), lw, *zargs, need - 4, None) == sp.SPLICE_EWORKSPACE
    misaligned = list(zargs)
    misaligned[9] = ctypes.c_void_p(0x2010)   # workspace must be 256-byte aligned
    assert lib.splice_decode_attn(ctypes.byref(sh), ctypes.byref(call), lw, *misaligned, need, None) == sp.SPLICE_EWORKSPACE
    bad_q = list(zargs)
    bad_q[0] = ctypes.c_void_p(0x1008)        # q not 16-byte aligned
    assert lib.splice_decode_attn(ctypes.byref(sh), ctypes.byref(call), lw, *bad_q, need, None) == sp.SPLICE_EINVAL
    # BUFFER donor without buffers
    shb = _shape(donor_zero=False)
    assert lib.splice_decode_attn(ctypes.byref(shb), ctypes.byref(call), lw, *zargs, need, None) == sp.SPLICE_EINVAL
    # negative L
    lwn = (ctypes.c_int32 * 12)(*([0, 0] * 5 + [-1, 0]))
    assert lib.splice_decode_attn(ctypes.byref(sh), ctypes.byref(call), lwn, *zargs, need, None) == sp.SPLICE_ESHAPE
    # the gather validates the same way
    gargs = [fake, fake, None, None, fake, fake, fake, fake, fake]
    assert lib.splice_kv_build(ctypes.byref(sh), ctypes.byref(call), None, *gargs, None) == sp.SPLICE_EINVAL
    assert lib.splice_kv_build(ctypes.byref(shb), ctypes.byref(call), lw, *gargs, None) == sp.SPLICE_EINVAL
    # zero cells: a valid no-op that touches nothing
    sh0 = _shape(n_cells=0)
    assert lib.splice_decode_attn(ctypes.byref(sh0), ctypes.byref(call), None, *([None] * 10), 0, None) == sp.SPLICE_OK
    assert lib.splice_workspace_init(None, 256, None) == sp.SPLICE_EINVAL


def test_workspace_bound_covers_every_call():
    for (C, Hkv, Tp, cap) in ((6, 2, 32, 16), (80, 8, 256, 512), (128, 8, 8192, 1024), (1, 1, 4096, 4096),
                              (48, 4, 4096, 128), (3, 1, 100000, 70000)):
        sh = _shape(n_cells=C, n_q_heads=Hkv, n_kv_heads=Hkv, prompt_len=Tp, span=(0, Tp // 2),
                    gen_capacity=cap, n_layers=4)
        worst = sp.splice_decode_attn_workspace_bytes(sh)
        for step in sorted({0, 1, cap // 3, cap // 2, cap - 1}):
            for window in (0, 1, 1024):
                need = sp.splice_decode_attn_workspace_bytes(sh, sp.make_call(0, step, window, 1.0))
                assert need <= worst, (C, Hkv, Tp, cap, step, window)


def _bf16_slots(sh, nbytes):
    """Partial-result slots per (cell, KV head) that a bf16 workspace of nbytes
    holds: statistics (256 bytes), int32 counters per pair rounded up to 256
    bytes, then per pair 16-bit prompt slots and one fp32 generated-row slot."""
    G, D = sh.n_q_heads // sh.n_kv_heads, sh.head_dim
    pairs = sh.n_cells * sh.n_kv_heads
    up = lambda x, m: (x + m - 1) // m * m
    pslot, gslot = up(G * D * 2 + 16 * G, 256), up(G * D + 2 * G, 64) * 4
    part = nbytes - 256 - up(pairs * 4, 256)
    assert (part - pairs * gslot) % (pairs * pslot) == 0
    return 1 + (part - pairs * gslot) // (pairs * pslot)


def test_call_workspace_covers_fewer_computed_cells():
    """A forked sweep computes its diverged cells only, and fewer computed
    cells take more prompt chunks by default: the bytes for a call on C
    cells must hold the slots the same call needs with any n <= C computed
    (what the call needs on a shape of n cells)."""
    for (C, Tp, window) in ((25, 1024, 0), (128, 8192, 0), (48, 4096, 1024)):
        for step in (0, 64, 255):
            call = sp.make_call(0, step, window, 0.125)
            sh = _shape(dtype="bf16", n_cells=C, n_q_heads=32, n_kv_heads=8, head_dim=128, prompt_len=Tp,
                        span=(8, Tp - 8), gen_capacity=256, n_layers=4)
            have = _bf16_slots(sh, sp.splice_decode_attn_workspace_bytes(sh, call))
            for n in (1, 2, 4, 9, C // 2, C):
                shn = _shape(dtype="bf16", n_cells=n, n_q_heads=32, n_kv_heads=8, head_dim=128, prompt_len=Tp,
                             span=(8, Tp - 8), gen_capacity=256, n_layers=4)
                need = _bf16_slots(shn, sp.splice_decode_attn_workspace_bytes(shn, call))
                assert need <= have, (C, Tp, window, step, n, need, have)


def test_decode_step_validation_before_device_access():
    lib = sp.load_library()
    sh = _shape(dtype="bf16")
    call = sp.make_call(1, 999, 0, 0.125)   # step is ignored by a decode step
    lw = (ctypes.c_int32 * 12)(*([0, 0] * 6))
    fake = ctypes.c_void_p(0x1000)   # never dereferenced: validation fails first
    ws = ctypes.c_void_p(0x2000)
    need = sp.splice_decode_attn_workspace_bytes(sh)

    def step(shape, steps, kn=fake, vn=fake, wbytes=need):
        st = None if steps is None else (ctypes.c_int32 * len(steps))(*steps)
        return lib.splice_decode_step(ctypes.byref(shape), ctypes.byref(call), lw, st, fake, kn, vn, fake, fake,
                                      None, None, fake, fake, fake, fake, ws, wbytes, None)

    assert step(sh, None) == sp.SPLICE_EINVAL                          # cell_step required
    assert step(sh, [0, 1, 2, 3, 4, 16]) == sp.SPLICE_ESHAPE           # s_c >= gen_capacity
    assert step(sh, [0, 1, 2, 3, 4, 5], kn=None) == sp.SPLICE_EINVAL   # new rows required
    assert step(sh, [0, 1, 2, 3, 4, 5], vn=ctypes.c_void_p(0x1004)) == sp.SPLICE_EINVAL   # misaligned
    assert step(sh, [0, 1, 2, 3, 4, 5], wbytes=16) == sp.SPLICE_EWORKSPACE
    assert step(_shape(dtype="f32"), [0, 1, 2, 3, 4, 5]) == sp.SPLICE_EUNSUPPORTED
    # every cell finished: a valid call with nothing to do (nothing launched)
    assert step(sh, [-1] * 6) == sp.SPLICE_OK
    # the call's own step is not validated, its other fields are
    bad = sp.make_call(2, 0, 0, 0.125)
    st = (ctypes.c_int32 * 6)(*([0] * 6))
    assert lib.splice_decode_step(ctypes.byref(sh), ctypes.byref(bad), lw, st, fake, fake, fake, fake, fake, None,
                                  None, fake, fake, fake, fake, ws, need, None) == sp.SPLICE_ESHAPE


def test_decode_forked_validation_before_device_access():
    lib = sp.load_library()
    sh = _shape(dtype="bf16")            # 6 cells, 2 layers
    call = sp.make_call(1, 5, 0, 0.125)
    fake = ctypes.c_void_p(0x1000)
    ws = ctypes.c_void_p(0x2000)
    need = sp.splice_decode_attn_workspace_bytes(sh)

    def forked(shape, cells, trunk, wbytes=need):
        lw = (ctypes.c_int32 * (2 * len(cells)))(*[x for c in cells for x in c])
        return lib.splice_decode_forked(ctypes.byref(shape), ctypes.byref(call), lw, trunk, fake, fake, fake,
                                        None, None, fake, fake, fake, fake, ws, wbytes, None)

    cells = [(2, 0), (0, 0), (1, 4), (0, 9), (1, 1), (2, 3)]   # cells 0 and 5 are never spliced (L >= 2)
    assert forked(sh, cells, -1) == sp.SPLICE_EINVAL           # a trunk is required
    assert forked(sh, cells, 6) == sp.SPLICE_ESHAPE            # out of range
    assert forked(sh, cells, 1) == sp.SPLICE_ESHAPE            # the trunk would be spliced
    assert forked(sh, cells, 0, wbytes=16) == sp.SPLICE_EWORKSPACE
    assert forked(_shape(dtype="f32"), cells, 0) == sp.SPLICE_EUNSUPPORTED


def test_noalloc_rejects_calls_beyond_its_array_before_device_access():
    """A call whose workspace would exceed the library's per-GPU array is
    refused on the host (no GPU is touched here)."""
    lib = sp.load_library()
    sh = _shape(n_cells=256, n_q_heads=32, n_kv_heads=8, head_dim=128, prompt_len=8192, span=(128, 8128),
                gen_capacity=1024, donor_zero=False, dtype="bf16")
    call = sp.make_call(0, 0, 0, 128 ** -0.5, split_keys=512)   # 16 prompt chunks: 17 slots per pair
    assert sp.splice_decode_attn_workspace_bytes(sh, call) > S.SPLICE_NOALLOC_WORKSPACE_BYTES
    lw = (ctypes.c_int32 * 512)(*([0, 0] * 256))
    fake = ctypes.c_void_p(0x1000)   # never dereferenced
    assert lib.splice_decode_attn_noalloc(ctypes.byref(sh), ctypes.byref(call), lw, *([fake] * 9), None) == \
        sp.SPLICE_EWORKSPACE
    # a bad argument is reported as such before the size is looked at
    bad = sp.make_call(0, 0, 0, float("nan"))
    assert lib.splice_decode_attn_noalloc(ctypes.byref(sh), ctypes.byref(bad), lw, *([fake] * 9), None) == \
        sp.SPLICE_EINVAL
