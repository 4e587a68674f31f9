"""ctypes binding of libmpipe (include/mpipe.h, mpipe_ops.h, mpipe_sched.h, mpipe_derive.h).

Argument marshalling only: torch tensors provide device memory and the current
HIP stream; every step of the encoder runs in the library's kernels."""
from __future__ import annotations

import ctypes as C
import os
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libmpipe.so")

F32, BF16 = 0, 1
OK, NOOP_FROZEN = 0, 1
_STATUS = {0: "OK", 1: "NOOP_FROZEN", -1: "INVALID_ARG", -2: "BAD_METADATA", -3: "WORKSPACE",
           -4: "NO_TAPE", -5: "UNSUPPORTED", -6: "HIP"}


class MpipeError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"mpipe status {status} ({_STATUS.get(status, '?')}): {msg}")
        self.status = status


class EncoderCfg(C.Structure):
    _fields_ = [("in_chans", C.c_int32), ("patch", C.c_int32), ("temporal_patch", C.c_int32),
                ("hidden", C.c_int32), ("layers", C.c_int32), ("heads", C.c_int32),
                ("mlp", C.c_int32), ("merge", C.c_int32), ("llm_hidden", C.c_int32),
                ("dtype", C.c_int32), ("ln_eps", C.c_float), ("rope_theta", C.c_float)]

    @classmethod
    def from_config(cls, cfg) -> "EncoderCfg":
        """From any object with the encoder-config attributes (e.g. workload.EncoderConfig)."""
        dt = BF16 if getattr(cfg, "dtype", "bf16") in ("bf16", BF16) else F32
        return cls(cfg.in_chans, cfg.patch, cfg.temporal_patch, cfg.hidden, cfg.layers,
                   cfg.heads, cfg.mlp, cfg.merge, cfg.llm_hidden, dt, float(cfg.ln_eps),
                   float(cfg.rope_theta))


_lib = None


def lib_path() -> str:
    return _LIB_PATH


def load():
    """Load libmpipe.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise MpipeError(-6, f"{_LIB_PATH} is missing: build it with paper_2607_03229_amd/build.py")
    L = C.CDLL(_LIB_PATH)
    P, i32, i64, sz = C.c_void_p, C.c_int32, C.c_int64, C.c_size_t
    st = C.c_int
    sig = {
        "mpipe_encoder_create": (st, [P, P]),
        "mpipe_encoder_destroy": (None, [P]),
        "mpipe_param_count": (i64, [P]),
        "mpipe_param_tensors": (i32, [P]),
        "mpipe_param_info": (st, [P, i32, C.c_char_p, i32, P, P, P]),
        "mpipe_encoder_sizes": (st, [P, P, i32, P, i32, i32, P, P, P, P]),
        "mpipe_encoder_regions": (st, [P, P, i32, P, i32, i32, i32, P, P, i32, P]),
        "mpipe_encoder_fwd": (st, [P, P, P, P, i32, P, i32, i32, P, P, sz, P, sz, P]),
        "mpipe_encoder_bwd": (st, [P, P, P, P, i32, P, i32, i32, P, sz, P, P, P, P, sz, P]),
        "mpipe_merge_scatter": (st, [P, i64, i32, i32, P, P, i64, P]),
        "mpipe_merge_gather": (st, [P, i64, i32, i32, P, i64, P, P]),
        "mpipe_merge_check_indices": (st, [P, i64, i64, P, P, P]),
        "mpipe_merge_check_indices_noalloc": (st, [P, i64, i64, P, P]),
        "mpipe_last_error": (C.c_char_p, []),
        "mpipe_profile_enable": (st, [P, i32]),
        "mpipe_encoder_set_side_stream": (st, [P, i32]),
        "mpipe_profile_read": (i32, [P, P, i32, P, i32, P, P, P]),
        "mpipe_op_gemm": (st, [i32, i32, i32, i32, i32, i32, P, i64, P, i64, P, i64, P, P, i64,
                               P, i64, i32, i32, i64, P]),
        "mpipe_op_splitk_reduce": (st, [P, i32, i64, i64, P, i64, P]),
        "mpipe_op_weight_grad_splits": (i32, [i64, i64, i64]),
        "mpipe_op_layernorm_fwd": (st, [i32, P, i64, i32, P, P, C.c_float, P, P, P, P]),
        "mpipe_op_layernorm_bwd": (st, [i32, P, P, P, P, P, i64, i32, P, P, P, P, P, P, P, sz, P]),
        "mpipe_op_rope": (st, [i32, P, i64, i32, i32, P, i32, C.c_float, i32, P, sz, P]),
        "mpipe_op_attention_fwd": (st, [i32, P, i64, i32, i32, P, i32, P, P, P, sz, P]),
        "mpipe_op_attention_bwd": (st, [i32, P, P, P, P, i64, i32, i32, P, i32, P, P, sz, P]),
        "mpipe_op_scratch_bytes": (sz, [i64, i32, i32, i32]),
        "mpipe_encoder_cost": (st, [P, P, i32, P, i32, i32, C.c_double, C.c_double, P]),
        "mpipe_owner_map": (st, [P, i32, P, i32, i32, P, P, P]),
        "mpipe_schedule_valid": (st, [P, i32, i32, P]),
        "mpipe_derive": (st, [P, i32, i32, P, P, i32, i32, P, P]),
        "mpipe_derived_destroy": (None, [P]),
        "mpipe_derived_shape": (st, [P, P, P, P, P, P]),
        "mpipe_derived_placement": (st, [P, i32, P, P, P, P]),
        "mpipe_derived_owner": (st, [P, P]),
        "mpipe_derived_lists": (st, [P, P, P, P, P, P]),
        "mpipe_derived_nodes": (i32, [P, i32, P, i32]),
        "mpipe_event_costs": (st, [P, P, P, P, P, C.c_double, C.c_double, C.c_double, P]),
        "mpipe_makespan": (st, [P, P, P, P, P, P]),
        "mpipe_memory_peak": (st, [P, P, P]),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    _lib = L
    return L


def last_error() -> str:
    v = load().mpipe_last_error()
    return v.decode() if v else ""


def _check(status: int, allow=(OK,)) -> int:
    if status not in allow:
        raise MpipeError(status, last_error())
    return status


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream=None) -> int:
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def _host_i32(a) -> Tuple[np.ndarray, C.c_void_p]:
    arr = np.ascontiguousarray(np.asarray(a, dtype=np.int32))
    return arr, arr.ctypes.data_as(C.c_void_p)


# --------------------------------------------------------------------------
# Encoder handle
# --------------------------------------------------------------------------

class Encoder:
    """Handle over mpipe_encoder_*; all tensors are torch device tensors."""

    def __init__(self, cfg):
        self.L = load()
        self.ccfg = cfg if isinstance(cfg, EncoderCfg) else EncoderCfg.from_config(cfg)
        h = C.c_void_p()
        _check(self.L.mpipe_encoder_create(C.byref(self.ccfg), C.byref(h)))
        self._h = h

    def close(self):
        if getattr(self, "_h", None) is not None and self._h.value:
            self.L.mpipe_encoder_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # -- parameter table --
    def param_count(self) -> int:
        return int(self.L.mpipe_param_count(C.byref(self.ccfg)))

    def param_table(self) -> List[Tuple[str, int, int, int]]:
        n = self.L.mpipe_param_tensors(C.byref(self.ccfg))
        buf = C.create_string_buffer(128)
        off, r, c = C.c_int64(), C.c_int64(), C.c_int64()
        out = []
        for i in range(n):
            _check(self.L.mpipe_param_info(C.byref(self.ccfg), i, buf, 128, C.byref(off),
                                           C.byref(r), C.byref(c)))
            out.append((buf.value.decode(), off.value, r.value, c.value))
        return out

    # -- sizes --
    def sizes(self, cu_seqlens, grid_thw, trainable: bool) -> Dict[str, int]:
        cu, cup = _host_i32(cu_seqlens)
        g, gp = _host_i32(np.asarray(grid_thw).reshape(-1, 3))
        ws, tp, nm, npch = C.c_size_t(), C.c_size_t(), C.c_int64(), C.c_int64()
        _check(self.L.mpipe_encoder_sizes(self._h, cup, max(len(cu) - 1, 0), gp, g.shape[0],
                                          int(trainable), C.byref(ws), C.byref(tp),
                                          C.byref(nm), C.byref(npch)))
        return {"workspace": ws.value, "tape": tp.value, "n_merged": nm.value,
                "n_patches": npch.value}

    def regions(self, cu_seqlens, grid_thw, trainable, which: int) -> np.ndarray:
        """int64 [n][2] (offset, bytes) of the workspace (which=0) or tape (1) ranges the
        step may write; at least 256 bytes after each range are never written."""
        cu, cup = _host_i32(cu_seqlens)
        g, gp = _host_i32(np.asarray(grid_thw).reshape(-1, 3))
        n = C.c_int32()
        args = (self._h, cup, max(len(cu) - 1, 0), gp, g.shape[0], int(trainable), which)
        _check(self.L.mpipe_encoder_regions(*args, None, None, 0, C.byref(n)))
        off, nb = np.zeros(n.value, np.int64), np.zeros(n.value, np.int64)
        _check(self.L.mpipe_encoder_regions(*args, off.ctypes.data_as(C.c_void_p),
                                            nb.ctypes.data_as(C.c_void_p), n.value, C.byref(n)))
        return np.stack([off, nb], axis=1)

    # -- fwd / bwd --
    def fwd(self, weights, patches, cu_seqlens, grid_thw, trainable: bool, merged, tape,
            workspace, stream=None) -> int:
        cu, cup = _host_i32(cu_seqlens)
        g, gp = _host_i32(np.asarray(grid_thw).reshape(-1, 3))
        tb = 0 if tape is None else tape.numel() * tape.element_size()
        wb = 0 if workspace is None else workspace.numel() * workspace.element_size()
        return _check(self.L.mpipe_encoder_fwd(
            self._h, _ptr(weights), _ptr(patches), cup, max(len(cu) - 1, 0), gp, g.shape[0],
            int(trainable), _ptr(merged), _ptr(tape), tb, _ptr(workspace), wb, _stream(stream)))

    def bwd(self, weights, patches, cu_seqlens, grid_thw, trainable: bool, tape, d_merged,
            d_weights, d_patches, workspace, stream=None) -> int:
        cu, cup = _host_i32(cu_seqlens)
        g, gp = _host_i32(np.asarray(grid_thw).reshape(-1, 3))
        tb = 0 if tape is None else tape.numel() * tape.element_size()
        wb = 0 if workspace is None else workspace.numel() * workspace.element_size()
        return _check(self.L.mpipe_encoder_bwd(
            self._h, _ptr(weights), _ptr(patches), cup, max(len(cu) - 1, 0), gp, g.shape[0],
            int(trainable), _ptr(tape), tb, _ptr(d_merged), _ptr(d_weights), _ptr(d_patches),
            _ptr(workspace), wb, _stream(stream)), allow=(OK, NOOP_FROZEN))

    # -- cost model --
    def cost(self, cu_seqlens, grid_thw, trainable, flops_per_second: float,
             bytes_per_second: float) -> Dict[str, float]:
        """W, D and the roofline seconds of this micro-batch's forward and backward slabs."""
        cu, cup = _host_i32(cu_seqlens)
        g, gp = _host_i32(np.asarray(grid_thw).reshape(-1, 3))
        out = (C.c_double * 6)()
        _check(self.L.mpipe_encoder_cost(self._h, cup, max(len(cu) - 1, 0), gp, g.shape[0],
                                         int(trainable), float(flops_per_second),
                                         float(bytes_per_second), out))
        keys = ("fwd_flops", "fwd_bytes", "fwd_seconds", "bwd_flops", "bwd_bytes", "bwd_seconds")
        return dict(zip(keys, list(out)))

    def set_side_stream(self, enable: bool):
        """Backward weight-gradient work on the handle's internal stream (default) or not."""
        _check(self.L.mpipe_encoder_set_side_stream(self._h, int(enable)))

    # -- kernel timing --
    def profile(self, enable: bool):
        _check(self.L.mpipe_profile_enable(self._h, int(enable)))

    def profile_read(self, stream=None) -> Dict[str, Tuple[int, float, float]]:
        cap, stride = 64, 64
        names = C.create_string_buffer(cap * stride)
        la = (C.c_int64 * cap)()
        ms = (C.c_double * cap)()
        fl = (C.c_double * cap)()
        n = self.L.mpipe_profile_read(self._h, _stream(stream), cap, names, stride, la, ms, fl)
        if n < 0:
            raise MpipeError(-6, "profile read failed")
        out = {}
        for i in range(n):
            nm = names.raw[i * stride:(i + 1) * stride].split(b"\0", 1)[0].decode()
            out[nm] = (int(la[i]), float(ms[i]), float(fl[i]))
        return out


# --------------------------------------------------------------------------
# Seam scatter / gather
# --------------------------------------------------------------------------

def _dt(t) -> int:
    import torch
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.float32:
        return F32
    raise MpipeError(-1, f"unsupported dtype {t.dtype}")


OWNER_GREEDY, OWNER_EXACT, OWNER_REFINED = 0, 1, 2


def owner_map(cost, warmup, method: int = OWNER_GREEDY):
    """ByMicrobatch owner: (owner [n_mb] int32, spill [n_ranks], max spill)."""
    c = np.ascontiguousarray(cost, dtype=np.float64)
    w = np.ascontiguousarray(warmup, dtype=np.float64)
    owner = np.zeros(c.shape[0], np.int32)
    spill = np.zeros(w.shape[0], np.float64)
    worst = C.c_double()
    _check(load().mpipe_owner_map(c.ctypes.data_as(C.c_void_p), c.shape[0],
                                  w.ctypes.data_as(C.c_void_p), w.shape[0], int(method),
                                  owner.ctypes.data_as(C.c_void_p),
                                  spill.ctypes.data_as(C.c_void_p), C.byref(worst)))
    return owner, spill, worst.value


# --------------------------------------------------------------------------
# Schedule algebra (host only)
# --------------------------------------------------------------------------

SK_1F1B, SK_GPIPE, SK_TRANSPOSE = 0, 1, 2
LAYOUT_SHARDED, LAYOUT_REPLICATED = 0, 1
COMM_NONE, COMM_GATHER, COMM_SCATTER, COMM_SEND, COMM_RECVGRAD = -1, 0, 1, 2, 3
GROUP_REPLICA, GROUP_DATA = 0, 1
EV_FWD, EV_BWD, EV_COLL, EV_DPREDUCE, EV_LOSS, EV_STEP_BARRIER = 0, 1, 2, 3, 4, 5
EDGE_ACTIVATION, EDGE_GRADIENT, EDGE_TURNAROUND, EDGE_ACCUMULATE, EDGE_SEQUENCE = 0, 1, 2, 3, 4
EVENT_FIELDS = ("kind", "region", "rank", "mb", "stage", "comm", "seam", "group")


def _vp(a: np.ndarray) -> C.c_void_p:
    return a.ctypes.data_as(C.c_void_p)


def schedule_valid(cut, n_layers: int, schedule) -> Tuple[bool, str]:
    """(valid, reason) for a (cut, schedule) pair."""
    c, cp = _host_i32(cut)
    s, sp = _host_i32(schedule)
    st = load().mpipe_schedule_valid(cp if c.size else None, s.size, int(n_layers), sp)
    return st == OK, ("" if st == OK else last_error())


class Derived:
    """derive(cut, schedule, model) read out into numpy arrays.

    layout, runs_bwd: [k]; slab_lo, slab_hi: [k, P]; owner: [M];
    seams: [k-1, 3] (left, fwd comm, bwd comm); reduces: [n, 2] (region, group);
    events: [n_events, 8] int32 with columns EVENT_FIELDS; edges: [n_edges, 3]
    (from, to, kind); nodes: list of P int32 arrays."""

    def __init__(self, cut, n_layers: int, schedule, trainable, n_ranks: int, n_mb: int,
                 owner=None):
        self.L = load()
        c, cp = _host_i32(cut)
        s, sp = _host_i32(schedule)
        t, tp = _host_i32(trainable)
        if t.size != s.size:
            raise MpipeError(-1, "one trainable bit per region")
        o, op = (None, None) if owner is None else _host_i32(owner)
        if o is not None and o.size != n_mb:
            raise MpipeError(-1, "one owner per micro-batch")
        h = C.c_void_p()
        _check(self.L.mpipe_derive(cp if c.size else None, s.size, int(n_layers), sp, tp,
                                   int(n_ranks), int(n_mb), op, C.byref(h)))
        self._h = h
        self.k, self.P, self.M = s.size, int(n_ranks), int(n_mb)
        ho, ne, nd, ns, nr = (C.c_int32() for _ in range(5))
        _check(self.L.mpipe_derived_shape(h, C.byref(ho), C.byref(ne), C.byref(nd),
                                          C.byref(ns), C.byref(nr)))
        self.has_order = bool(ho.value)
        self.layout = np.zeros(self.k, np.int32)
        self.runs_bwd = np.zeros(self.k, np.int32)
        self.slab_lo = np.zeros((self.k, self.P), np.int32)
        self.slab_hi = np.zeros((self.k, self.P), np.int32)
        for j in range(self.k):
            lay, rb = C.c_int32(), C.c_int32()
            _check(self.L.mpipe_derived_placement(h, j, C.byref(lay), C.byref(rb),
                                                  _vp(self.slab_lo[j]), _vp(self.slab_hi[j])))
            self.layout[j], self.runs_bwd[j] = lay.value, rb.value
        self.owner = np.zeros(self.M, np.int32)
        _check(self.L.mpipe_derived_owner(h, _vp(self.owner)))
        self.events = np.zeros((ne.value, 8), np.int32)
        self.edges = np.zeros((nd.value, 3), np.int32)
        self.seams = np.zeros((ns.value, 3), np.int32)
        red_r = np.zeros(nr.value, np.int32)
        red_g = np.zeros(nr.value, np.int32)
        _check(self.L.mpipe_derived_lists(h, _vp(self.events), _vp(self.edges), _vp(self.seams),
                                          _vp(red_r), _vp(red_g)))
        self.reduces = np.stack([red_r, red_g], axis=1) if nr.value else np.zeros((0, 2), np.int32)
        self.nodes = []
        for r in range(self.P):
            n = self.L.mpipe_derived_nodes(h, r, None, 0)
            if n < 0:
                raise MpipeError(-1, last_error())
            v = np.zeros(n, np.int32)
            self.L.mpipe_derived_nodes(h, r, _vp(v), n)
            self.nodes.append(v)

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value:
            self.L.mpipe_derived_destroy(h)
            self._h = None

    def event_costs(self, fwd_cost, bwd_cost, seam_bytes, reduce_bytes, alpha: float,
                    beta: float, loss_cost: float) -> np.ndarray:
        """Cost of every event (Sec. 4.3); fwd_cost/bwd_cost [k, M] seconds of a whole
        region, seam_bytes [k-1, M], reduce_bytes [k]."""
        f = np.ascontiguousarray(fwd_cost, dtype=np.float64).reshape(-1)
        b = np.ascontiguousarray(bwd_cost, dtype=np.float64).reshape(-1)
        sb = np.ascontiguousarray(seam_bytes, dtype=np.float64).reshape(-1)
        rb = np.ascontiguousarray(reduce_bytes, dtype=np.float64).reshape(-1)
        if f.size != self.k * self.M or b.size != self.k * self.M or rb.size != self.k \
                or sb.size != (self.k - 1) * self.M:
            raise MpipeError(-1, "cost arrays do not match (k, M)")
        out = np.zeros(self.events.shape[0], np.float64)
        _check(self.L.mpipe_event_costs(self._h, _vp(f), _vp(b), _vp(sb) if sb.size else None,
                                        _vp(rb), float(alpha), float(beta), float(loss_cost),
                                        _vp(out)))
        return out

    def makespan(self, cost):
        """(T, bubble [P], start [n_events], finish [n_events])."""
        c = np.ascontiguousarray(cost, dtype=np.float64)
        if c.size != self.events.shape[0]:
            raise MpipeError(-1, "one cost per event")
        T = C.c_double()
        bub = np.zeros(self.P, np.float64)
        st = np.zeros(c.size, np.float64)
        fin = np.zeros(c.size, np.float64)
        _check(self.L.mpipe_makespan(self._h, _vp(c), C.byref(T), _vp(bub), _vp(st), _vp(fin)))
        return T.value, bub, st, fin

    def memory_peak(self, act_bytes) -> np.ndarray:
        a = np.ascontiguousarray(act_bytes, dtype=np.float64)
        if a.size != self.events.shape[0]:
            raise MpipeError(-1, "one byte count per event")
        out = np.zeros(self.P, np.float64)
        _check(self.L.mpipe_memory_peak(self._h, _vp(a), _vp(out)))
        return out


def merge_scatter(merged, placeholder_idx, embeds, stream=None) -> None:
    """embeds.view(-1, H)[idx[j]] = merged[j] (bit-exact, in place)."""
    H = merged.shape[-1]
    n_rows = embeds.numel() // H
    _check(load().mpipe_merge_scatter(_ptr(merged), merged.shape[0], H, _dt(merged),
                                      _ptr(placeholder_idx), _ptr(embeds), n_rows,
                                      _stream(stream)))


def merge_gather(d_embeds, placeholder_idx, d_merged, stream=None) -> None:
    """d_merged[j] = d_embeds.view(-1, H)[idx[j]]."""
    H = d_merged.shape[-1]
    n_rows = d_embeds.numel() // H
    _check(load().mpipe_merge_gather(_ptr(d_embeds), n_rows, H, _dt(d_embeds),
                                     _ptr(placeholder_idx), d_merged.shape[0], _ptr(d_merged),
                                     _stream(stream)))


def merge_check_indices(placeholder_idx, n_rows: int, marks, status, stream=None) -> None:
    _check(load().mpipe_merge_check_indices(_ptr(placeholder_idx), placeholder_idx.numel(),
                                            n_rows, _ptr(marks), _ptr(status), _stream(stream)))


def merge_check_indices_noalloc(placeholder_idx, n_rows: int, status, stream=None) -> None:
    """mpipe_merge_check_indices without a caller buffer (the library's built-in
    counters; n_rows <= CHECK_NOALLOC_MAX_ROWS)."""
    _check(load().mpipe_merge_check_indices_noalloc(_ptr(placeholder_idx),
                                                    placeholder_idx.numel(), n_rows,
                                                    _ptr(status), _stream(stream)))


CHECK_NOALLOC_MAX_ROWS = 1 << 20   # MPIPE_CHECK_NOALLOC_MAX_ROWS of include/mpipe.h


# --------------------------------------------------------------------------
# Kernel-level ops
# --------------------------------------------------------------------------

def op_scratch_bytes(N: int, heads: int, n: int, n_seg: int) -> int:
    return int(load().mpipe_op_scratch_bytes(N, heads, n, n_seg))


def op_gemm(dtype: int, layout: int, epilogue: int, M: int, N: int, K: int, A, lda: int, B,
            ldb: int, Cout, ldc: int, bias=None, aux=None, ld_aux: int = 0, C2=None,
            ldc2: int = 0, beta: int = 0, k_per_split: int = 0, split_stride: int = 0,
            stream=None) -> None:
    _check(load().mpipe_op_gemm(dtype, layout, epilogue, M, N, K, _ptr(A), lda, _ptr(B), ldb,
                                _ptr(Cout), ldc, _ptr(bias), _ptr(aux), ld_aux, _ptr(C2), ldc2,
                                beta, k_per_split, split_stride, _stream(stream)))


def op_splitk_reduce(part, splits: int, M: int, N: int, out, ldo: int, stream=None) -> None:
    _check(load().mpipe_op_splitk_reduce(_ptr(part), splits, M, N, _ptr(out), ldo,
                                         _stream(stream)))


def gemm_split(M: int, N: int, K: int) -> int:
    """K splits of the backward's weight-gradient product dW[M][N] over K tokens."""
    return int(load().mpipe_op_weight_grad_splits(M, N, K))


def op_layernorm_fwd(dtype, X, rows, n, g, b, eps, Y, mean=None, rstd=None, stream=None):
    _check(load().mpipe_op_layernorm_fwd(dtype, _ptr(X), rows, n, _ptr(g), _ptr(b), eps, _ptr(Y),
                                         _ptr(mean), _ptr(rstd), _stream(stream)))


def op_layernorm_bwd(dtype, dY, X, mean, rstd, g, rows, n, dres, dX, dXt, grad_g, grad_b,
                     scratch, stream=None, colsum_dx=None):
    _check(load().mpipe_op_layernorm_bwd(dtype, _ptr(dY), _ptr(X), _ptr(mean), _ptr(rstd), _ptr(g),
                                         rows, n, _ptr(dres), _ptr(dX), _ptr(dXt), _ptr(grad_g),
                                         _ptr(grad_b), _ptr(colsum_dx), _ptr(scratch),
                                         scratch.numel() * scratch.element_size(),
                                         _stream(stream)))


def op_rope(dtype, qkv, rows, heads, head_dim, grid_thw, theta, inverse, scratch, stream=None):
    g, gp = _host_i32(np.asarray(grid_thw).reshape(-1, 3))
    _check(load().mpipe_op_rope(dtype, _ptr(qkv), rows, heads, head_dim, gp, g.shape[0], theta,
                                int(inverse), _ptr(scratch),
                                scratch.numel() * scratch.element_size(), _stream(stream)))


def op_attention_fwd(dtype, qkv, N, heads, head_dim, cu_seqlens, o, lse, scratch, stream=None):
    cu, cup = _host_i32(cu_seqlens)
    _check(load().mpipe_op_attention_fwd(dtype, _ptr(qkv), N, heads, head_dim, cup,
                                         max(len(cu) - 1, 0), _ptr(o), _ptr(lse), _ptr(scratch),
                                         scratch.numel() * scratch.element_size(),
                                         _stream(stream)))


def op_attention_bwd(dtype, qkv, o, d_o, lse, N, heads, head_dim, cu_seqlens, dqkv, scratch,
                     stream=None):
    cu, cup = _host_i32(cu_seqlens)
    _check(load().mpipe_op_attention_bwd(dtype, _ptr(qkv), _ptr(o), _ptr(d_o), _ptr(lse), N,
                                         heads, head_dim, cup, max(len(cu) - 1, 0), _ptr(dqkv),
                                         _ptr(scratch), scratch.numel() * scratch.element_size(),
                                         _stream(stream)))
