"""Helpers for the GPU parity tests (device tensors, error metrics)."""
import sys

import numpy as np

import workload as W


def torch_dev():
    import torch
    return torch, torch.device("cuda:0")


def announce(msg: str):
    """Name the case before its GPU step (so a lost box still tells which one)."""
    print(f"[gpu-case] {msg}", flush=True)
    sys.stdout.flush()


def to_dev(a, dtype_str: str):
    torch, dev = torch_dev()
    t = torch.from_numpy(np.ascontiguousarray(np.asarray(a, np.float32)))
    if dtype_str == "bf16":
        t = t.to(torch.bfloat16)
    return t.to(dev)


def zeros(shape, dtype_str: str):
    torch, dev = torch_dev()
    return torch.zeros(shape, dtype=torch.bfloat16 if dtype_str == "bf16" else torch.float32,
                       device=dev)


def nans(shape, dtype_str: str):
    """An output buffer the library must overwrite: NaN everywhere, so an element that is
    never written fails max_rel (which is NaN-propagating) instead of passing as 0."""
    torch, dev = torch_dev()
    return torch.full(shape, float("nan"),
                      dtype=torch.bfloat16 if dtype_str == "bf16" else torch.float32, device=dev)


def host(t) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def max_rel(x, r) -> float:
    """max |x - r| / max |r|, per tensor; NaN (which fails every bound) when either side
    holds a NaN."""
    x, r = np.asarray(x, np.float64), np.asarray(r, np.float64)
    if np.isnan(x).any() or np.isnan(r).any():
        return float("nan")
    den = np.max(np.abs(r)) if r.size else 0.0
    if den == 0.0:
        return float(np.max(np.abs(x))) if x.size else 0.0
    return float(np.max(np.abs(x - r)) / den)


def rnd(rng, shape, dtype_str, scale=1.0, loc=0.0):
    v = (rng.standard_normal(shape) * scale + loc).astype(np.float32)
    return W.round_bf16(v) if dtype_str == "bf16" else v
