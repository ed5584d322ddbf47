"""Spliced grouped-query decode attention for MI355X (gfx950).

The hot path of the splice intervention in "Probing the Prompt KV Cache:
Where It Becomes Dispensable": single-query GQA decode attention over a
prompt cache whose span slots are read, per sweep cell (L, W), from a donor
cache.  The work runs in hand-written HIP kernels behind the C ABI declared
in include/splice_attn.h; ``splice`` is its ctypes binding.
"""
from .splice import (EXPORTS, LIB_PATH, SPLICE_BF16, SPLICE_DONOR_BUFFER, SPLICE_DONOR_ZERO,
                     SPLICE_EHIP, SPLICE_EINVAL, SPLICE_ESHAPE, SPLICE_EUNSUPPORTED,
                     SPLICE_EWORKSPACE, SPLICE_F32, SPLICE_MAX_CELLS, SPLICE_OK, SPLICE_SRC_CLEAN,
                     SPLICE_SRC_DONOR, SPLICE_SRC_GEN, SPLICE_SRC_ZERO, SpliceCall, SpliceError,
                     SpliceShape, load_library, make_call, make_shape, new_workspace,
                     splice_abi_version, splice_decode_attn, splice_decode_attn_noalloc,
                     splice_decode_attn_workspace_bytes,
                     splice_decode_forked, splice_decode_step,
                     splice_kv_build, splice_status_str, splice_visible_len, splice_workspace_handovers,
                     splice_workspace_init,
                     status_name)

__all__ = [n for n in dir() if not n.startswith("_")]
