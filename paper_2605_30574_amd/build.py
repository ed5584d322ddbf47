"""Build the gfx950 libraries in-tree: paper_2605_30574_amd/libsplice_attn.so
(the spliced decode attention) and paper_2605_30574_amd/libsplice_calib.so (a
plain stream-read kernel, the measured read ceiling).

    python -m paper_2605_30574_amd.build

Each translation unit under csrc/ (the host/ABI unit and one unit per
(head_dim, element type) of the attention kernels) is compiled to an object
in parallel, then the objects are linked into one shared library.
"""
from __future__ import annotations

import glob
import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
INCLUDE = os.path.join(ROOT, "include")
CSRC = os.path.join(PKG, "csrc")
OBJDIR = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libsplice_attn.so")
CALIB_SRC = os.path.join(PKG, "calib", "stream_read.hip")
CALIB_LIB = os.path.join(PKG, "libsplice_calib.so")
ARCH = "gfx950"

COMPILE_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-fvisibility=hidden", "-Wall",
    # no packed-FP32 instructions in device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # MFMA sources and results in VGPRs: the accumulators stay where the
    # online-softmax rescale (a vector-ALU multiply) can reach them, with no
    # AGPR copies in the streaming loops
    "-mllvm", "-amdgpu-mfma-vgpr-form",
]
NOISE = "is not a recognized feature for this target"


def sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")))


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found: the splice library needs ROCm's hipcc")


def _run(cmd):
    res = subprocess.run(cmd, capture_output=True, text=True)
    msgs = [ln for ln in (res.stderr or "").splitlines() if NOISE not in ln]
    return res.returncode, msgs


def build(out: str = LIB, extra=(), verbose: bool = False, jobs: int = 0) -> str:
    cc = hipcc()
    os.makedirs(OBJDIR, exist_ok=True)
    srcs = sources()
    objs = [os.path.join(OBJDIR, os.path.basename(s)[:-4] + ".o") for s in srcs]
    cmds = [[cc, *COMPILE_FLAGS, f"-I{INCLUDE}", f"-I{CSRC}", *extra, "-c", "-o", o, s]
            for s, o in zip(srcs, objs)]
    jobs = jobs or min(len(cmds), max(1, min(16, os.cpu_count() or 1)))
    if verbose:
        for c in cmds:
            print(" ".join(c), flush=True)
    with ThreadPoolExecutor(max_workers=jobs) as ex:
        results = list(ex.map(_run, cmds))
    failed = [(c, m) for c, (rc, m) in zip(cmds, results) if rc != 0]
    if failed:
        raise RuntimeError("hipcc failed:\n" + "\n".join(
            " ".join(c[-1:]) + "\n" + "\n".join(m) for c, m in failed))
    if verbose:
        for _, m in results:
            if m:
                print("\n".join(m), file=sys.stderr)
    link = [cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", out + ".tmp", *objs]
    rc, msgs = _run(link)
    if rc != 0:
        raise RuntimeError("link failed:\n" + "\n".join(msgs))
    os.replace(out + ".tmp", out)
    return out


def build_calib(out: str = CALIB_LIB) -> str:
    """Compile and link the stream-read library (one translation unit)."""
    cmd = [hipcc(), *COMPILE_FLAGS, f"-I{INCLUDE}", "-shared", "-o", out + ".tmp", CALIB_SRC]
    rc, msgs = _run(cmd)
    if rc != 0:
        raise RuntimeError("hipcc failed:\n" + "\n".join(msgs))
    os.replace(out + ".tmp", out)
    return out


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
    print(build_calib())
