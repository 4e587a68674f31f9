"""CPU oracle for the replicated-encoder step -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product path (the HIP library and
its binding) never loads it.

This is a thin ctypes wrapper over ``liboracle.so`` (built with g++ from
``mpipe_ref.cpp``, no HIP).  It takes numpy arrays and returns numpy arrays.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
from typing import Optional, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "mpipe_ref.cpp")
_LIB = os.path.join(_HERE, "liboracle.so")
# A test may point the wrapper at another build of the same source (the
# planted-mistake meta-test does); nothing else sets this.
_LIB_OVERRIDE = os.environ.get("MPIPE_ORACLE_LIB")

OK, NOOP_FROZEN = 0, 1


def build(force: bool = True) -> str:
    """Compile liboracle.so with g++ (OpenMP, plain -O2; no fast-math)."""
    if force or not os.path.exists(_LIB):
        cmd = ["g++", "-O2", "-std=c++17", "-fPIC", "-shared", "-fopenmp",
               "-march=x86-64-v3", "-o", _LIB + ".tmp", _SRC]
        subprocess.run(cmd, check=True)
        os.replace(_LIB + ".tmp", _LIB)
    return _LIB


class _Cfg(C.Structure):
    _fields_ = [("in_chans", C.c_int32), ("patch", C.c_int32), ("temporal_patch", C.c_int32),
                ("hidden", C.c_int32), ("layers", C.c_int32), ("heads", C.c_int32),
                ("mlp", C.c_int32), ("merge", C.c_int32), ("llm_hidden", C.c_int32),
                ("ln_eps", C.c_double), ("rope_theta", C.c_double)]


def make_cfg(cfg) -> _Cfg:
    """From any object with the encoder-config attributes (e.g. workload.EncoderConfig)."""
    return _Cfg(cfg.in_chans, cfg.patch, cfg.temporal_patch, cfg.hidden, cfg.layers, cfg.heads,
                cfg.mlp, cfg.merge, cfg.llm_hidden, float(cfg.ln_eps), float(cfg.rope_theta))


_lib = None


def lib():
    global _lib
    if _lib is None:
        if _LIB_OVERRIDE:
            L = C.CDLL(_LIB_OVERRIDE)
        else:
            if not os.path.exists(_LIB):
                build(force=False)
            L = C.CDLL(_LIB)
        P = C.c_void_p
        i32, i64 = C.c_int32, C.c_int64
        L.ref_param_count.restype = i64
        L.ref_param_count.argtypes = [P]
        L.ref_param_tensors.restype = i32
        L.ref_param_tensors.argtypes = [P]
        L.ref_param_info.restype = C.c_int
        L.ref_param_info.argtypes = [P, i32, C.c_char_p, i32, P, P, P]
        L.ref_positions.restype = C.c_int
        L.ref_positions.argtypes = [P, i32, P, P]
        for n in ("ref_encoder_f64", "ref_encoder_f32"):
            f = getattr(L, n)
            f.restype = C.c_int
            f.argtypes = [P, P, P, P, i32, P, i32, i32, P, P, P, P]
        L.ref_linear_f64.argtypes = [P, P, P, i64, i64, i64, P]
        L.ref_linear_bwd_f64.argtypes = [P, P, P, i64, i64, i64, P, P, P]
        L.ref_layernorm_f64.argtypes = [P, P, P, i64, i64, C.c_double, P, P, P]
        L.ref_layernorm_bwd_f64.argtypes = [P, P, P, P, P, i64, i64, P, P, P]
        L.ref_gelu_f64.argtypes = [P, i64, P]
        L.ref_gelu_grad_f64.argtypes = [P, i64, P]
        L.ref_rope2d_f64.argtypes = [P, i64, i32, i32, i64, P, P, C.c_double, i32]
        L.ref_attention_f64.argtypes = [P, P, P, i64, P, i32, i32, i32, P, i64, P]
        L.ref_attention_bwd_f64.argtypes = [P, P, P, i64, P, P, i64, P, P, i32, i32, i32,
                                            P, P, P, i64]
        L.ref_merge_scatter.restype = C.c_int
        L.ref_merge_scatter.argtypes = [P, i64, i64, P, P, i64]
        L.ref_merge_gather.restype = C.c_int
        L.ref_merge_gather.argtypes = [P, i64, i64, P, i64, P]
        L.ref_num_threads.restype = i32
        _lib = L
    return _lib


def _p(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(C.c_void_p)


def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float64)


def num_threads() -> int:
    return int(lib().ref_num_threads())


# --------------------------------------------------------------------------
# Parameter table
# --------------------------------------------------------------------------

def param_count(cfg) -> int:
    c = make_cfg(cfg)
    return int(lib().ref_param_count(C.byref(c)))


def param_table(cfg):
    c = make_cfg(cfg)
    L = lib()
    out = []
    n = L.ref_param_tensors(C.byref(c))
    buf = C.create_string_buffer(128)
    off, r, cc = C.c_int64(), C.c_int64(), C.c_int64()
    for i in range(n):
        L.ref_param_info(C.byref(c), i, buf, 128, C.byref(off), C.byref(r), C.byref(cc))
        out.append((buf.value.decode(), int(off.value), int(r.value), int(cc.value)))
    return out


def positions(grid_thw: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    g = np.ascontiguousarray(grid_thw, dtype=np.int32).reshape(-1, 3)
    n = int((g[:, 0].astype(np.int64) * g[:, 1] * g[:, 2]).sum())
    py, px = np.zeros(n, np.int32), np.zeros(n, np.int32)
    rc = lib().ref_positions(_p(g), g.shape[0], _p(py), _p(px))
    if rc:
        raise ValueError(f"ref_positions: {rc}")
    return py, px


# --------------------------------------------------------------------------
# Whole encoder
# --------------------------------------------------------------------------

def encoder(cfg, weights, patches, cu_seqlens, grid_thw, trainable,
            d_merged=None, want_d_patches: bool = False, d_w_init=None,
            precision: str = "f64"):
    """Run the oracle encoder.  trainable: False/0 frozen, True/1 every part trainable,
    2 only the merger trainable (its backward stops at the merger's LayerNorm).

    Returns (status, merged, d_w, d_patches); d_w / d_patches are None unless a
    backward ran.  d_w starts from ``d_w_init`` (zeros by default): the oracle
    accumulates into it."""
    dt = np.float64 if precision == "f64" else np.float32
    fn = lib().ref_encoder_f64 if precision == "f64" else lib().ref_encoder_f32
    c = make_cfg(cfg)
    w = np.ascontiguousarray(weights, dtype=dt)
    X = np.ascontiguousarray(patches, dtype=dt)
    cu = np.ascontiguousarray(cu_seqlens, dtype=np.int32)
    g = np.ascontiguousarray(grid_thw, dtype=np.int32).reshape(-1, 3)
    n_merged = int((g[:, 0].astype(np.int64) * (g[:, 1] // 2) * (g[:, 2] // 2)).sum())
    merged = np.zeros((n_merged, cfg.llm_hidden), dt)
    dM = None if d_merged is None else np.ascontiguousarray(d_merged, dtype=dt)
    d_w = None
    d_x = None
    if dM is not None:
        d_w = (np.zeros(w.shape, dt) if d_w_init is None
               else np.array(d_w_init, dtype=dt, copy=True))
        if want_d_patches:
            d_x = np.zeros(X.shape, dt)
    rc = fn(C.byref(c), _p(w), _p(X), _p(cu), len(cu) - 1, _p(g), g.shape[0], int(trainable),
            _p(merged), _p(dM), _p(d_w), _p(d_x))
    if rc < 0:
        raise ValueError(f"oracle encoder rejected the metadata (status {rc})")
    return rc, merged, d_w, d_x


# --------------------------------------------------------------------------
# Building blocks
# --------------------------------------------------------------------------

def linear(X, W, b=None):
    X, W = _f64(X), _f64(W)
    M, K = X.shape
    N = W.shape[0]
    Y = np.zeros((M, N))
    lib().ref_linear_f64(_p(X), _p(W), _p(None if b is None else _f64(b)), M, K, N, _p(Y))
    return Y


def linear_bwd(dY, X, W):
    dY, X, W = _f64(dY), _f64(X), _f64(W)
    M, K = X.shape
    N = W.shape[0]
    dX, dW, db = np.zeros((M, K)), np.zeros((N, K)), np.zeros(N)
    lib().ref_linear_bwd_f64(_p(dY), _p(X), _p(W), M, K, N, _p(dX), _p(dW), _p(db))
    return dX, dW, db


def layernorm(X, g, b, eps):
    X = _f64(X)
    M, n = X.shape
    Y, mu, rs = np.zeros((M, n)), np.zeros(M), np.zeros(M)
    lib().ref_layernorm_f64(_p(X), _p(_f64(g)), _p(_f64(b)), M, n, eps, _p(Y), _p(mu), _p(rs))
    return Y, mu, rs


def layernorm_bwd(dY, X, g, mean, rstd):
    dY, X = _f64(dY), _f64(X)
    M, n = X.shape
    dX, dg, db = np.zeros((M, n)), np.zeros(n), np.zeros(n)
    lib().ref_layernorm_bwd_f64(_p(dY), _p(X), _p(_f64(g)), _p(_f64(mean)), _p(_f64(rstd)),
                                M, n, _p(dX), _p(dg), _p(db))
    return dX, dg, db


def gelu(u):
    u = _f64(u)
    y = np.zeros_like(u)
    lib().ref_gelu_f64(_p(u), u.size, _p(y))
    return y


def gelu_grad(u):
    u = _f64(u)
    y = np.zeros_like(u)
    lib().ref_gelu_grad_f64(_p(u), u.size, _p(y))
    return y


def rope2d(x, heads, d, pos_y, pos_x, theta=10000.0, inverse=False):
    """Rotate every head of x [N, heads*d] (returns a new array)."""
    x = np.array(x, dtype=np.float64, copy=True, order="C")
    py = np.ascontiguousarray(pos_y, dtype=np.int32)
    px = np.ascontiguousarray(pos_x, dtype=np.int32)
    lib().ref_rope2d_f64(_p(x), x.shape[0], heads, d, x.shape[1], _p(py), _p(px), theta,
                         int(inverse))
    return x


def attention(q, k, v, cu_seqlens, heads, d):
    """q, k, v: [N, heads*d].  Returns (o [N, heads*d], lse [N, heads])."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    cu = np.ascontiguousarray(cu_seqlens, dtype=np.int32)
    N = q.shape[0]
    o, lse = np.zeros((N, heads * d)), np.zeros((N, heads))
    lib().ref_attention_f64(_p(q), _p(k), _p(v), heads * d, _p(cu), len(cu) - 1, heads, d,
                            _p(o), heads * d, _p(lse))
    return o, lse


def attention_bwd(q, k, v, o, d_o, lse, cu_seqlens, heads, d):
    q, k, v, o, d_o, lse = map(_f64, (q, k, v, o, d_o, lse))
    cu = np.ascontiguousarray(cu_seqlens, dtype=np.int32)
    N = q.shape[0]
    dq, dk, dv = np.zeros((N, heads * d)), np.zeros((N, heads * d)), np.zeros((N, heads * d))
    lib().ref_attention_bwd_f64(_p(q), _p(k), _p(v), heads * d, _p(o), _p(d_o), heads * d,
                                _p(lse), _p(cu), len(cu) - 1, heads, d, _p(dq), _p(dk), _p(dv),
                                heads * d)
    return dq, dk, dv


def merge_scatter(merged: np.ndarray, idx: np.ndarray, emb: np.ndarray) -> np.ndarray:
    """Returns a copy of emb with emb[idx[j]] = merged[j] (raw bytes)."""
    out = np.array(emb, copy=True, order="C")
    m = np.ascontiguousarray(merged)
    ix = np.ascontiguousarray(idx, dtype=np.int64)
    rb = m.strides[0] if m.shape[0] else out.strides[0]
    rc = lib().ref_merge_scatter(_p(m), m.shape[0], rb, _p(ix), _p(out), out.shape[0])
    if rc:
        raise ValueError("index out of range or repeated")
    return out


def merge_gather(d_emb: np.ndarray, idx: np.ndarray) -> np.ndarray:
    e = np.ascontiguousarray(d_emb)
    ix = np.ascontiguousarray(idx, dtype=np.int64)
    out = np.zeros((ix.shape[0],) + e.shape[1:], e.dtype)
    rc = lib().ref_merge_gather(_p(e), e.shape[0], e.strides[0], _p(ix), ix.shape[0], _p(out))
    if rc:
        raise ValueError("index out of range or repeated")
    return out


# --------------------------------------------------------------------------
# ByMicrobatch owner (cost model, Sec. 4.3) -- plain Python by the definition
# --------------------------------------------------------------------------

def owner_spill(owner, cost, warmup):
    """spill_r = max(0, E_r - w_r) with E_r the summed cost of the micro-batches rank r
    owns (added in index order); returns (per-rank spill list, the step's max_r spill_r)."""
    E = [0.0] * len(warmup)
    for m, r in enumerate(owner):
        E[int(r)] += float(cost[m])
    spill = [max(0.0, E[r] - float(warmup[r])) for r in range(len(warmup))]
    return spill, max(spill, default=0.0)


def owner_bruteforce(cost, warmup):
    """The ByMicrobatch owner by its definition: among all n_ranks ** n_mb assignments,
    one that minimises max_r spill_r (tiny inputs only).  Returns (owner, max spill)."""
    import itertools
    best = None
    for owner in itertools.product(range(len(warmup)), repeat=len(cost)):
        s = owner_spill(owner, cost, warmup)[1]
        if best is None or s < best[1]:
            best = (list(owner), s)
    return best
