"""MI355X-native replicated-encoder step of the transpose schedule.

The work happens in ``libmpipe.so`` (hand-written gfx950 HIP kernels behind a
C ABI, ``include/mpipe.h``).  This package is the Python binding: it marshals
torch tensors (device memory and streams only) into the C calls.  Nothing here
computes; if the library is missing, every call raises.
"""
from ._binding import (  # noqa: F401
    MpipeError, Encoder, EncoderCfg, load, lib_path, last_error,
    merge_scatter, merge_gather, merge_check_indices,
    op_gemm, op_layernorm_fwd, op_layernorm_bwd, op_rope, op_attention_fwd,
    op_attention_bwd, op_scratch_bytes,
    F32, BF16, OK, NOOP_FROZEN,
    owner_map, OWNER_GREEDY, OWNER_EXACT, OWNER_REFINED,
)
