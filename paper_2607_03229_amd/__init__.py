"""MI355X-native replicated-encoder step of the transpose schedule.

The work happens in ``libmpipe.so`` (hand-written gfx950 HIP kernels behind a
C ABI, ``include/mpipe.h``).  This package is the Python binding: it marshals
torch tensors (device memory and streams only) into the C calls.  Nothing here
computes; if the library is missing, every call raises.
"""
from ._binding import (  # noqa: F401
    MpipeError, Encoder, EncoderCfg, load, lib_path, last_error,
    merge_scatter, merge_gather, merge_check_indices, merge_check_indices_noalloc,
    CHECK_NOALLOC_MAX_ROWS,
    op_gemm, op_layernorm_fwd, op_layernorm_bwd, op_rope, op_attention_fwd,
    op_attention_bwd, op_scratch_bytes, op_splitk_reduce, gemm_split,
    F32, BF16, OK, NOOP_FROZEN,
    owner_map, OWNER_GREEDY, OWNER_EXACT, OWNER_REFINED,
    schedule_valid, Derived, EVENT_FIELDS,
    SK_1F1B, SK_GPIPE, SK_TRANSPOSE, LAYOUT_SHARDED, LAYOUT_REPLICATED,
    COMM_NONE, COMM_GATHER, COMM_SCATTER, COMM_SEND, COMM_RECVGRAD, GROUP_REPLICA, GROUP_DATA,
    EV_FWD, EV_BWD, EV_COLL, EV_DPREDUCE, EV_LOSS, EV_STEP_BARRIER,
    EDGE_ACTIVATION, EDGE_GRADIENT, EDGE_TURNAROUND, EDGE_ACCUMULATE, EDGE_SEQUENCE,
)
