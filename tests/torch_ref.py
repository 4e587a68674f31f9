"""An independent fp64 PyTorch (CPU) formulation of the encoder, used only to pin
the oracle: every block is a library routine (``F.layer_norm``, ``F.gelu``,
``F.scaled_dot_product_attention``, ``F.conv3d`` for the patch embedding,
complex multiplication for the rotary position) and gradients come from
autograd rather than from hand-written adjoints.

It takes a different route from the oracle wherever the route can differ:
patch embedding by convolution on raw pixels, the merge window by the
four-consecutive-rows view, positions from a coordinate image pushed through
the generator's patchify, and RoPE as a complex rotation."""
from __future__ import annotations

import numpy as np
import torch
import torch.nn.functional as F

import workload as W


def split_params(cfg, w: torch.Tensor):
    out = {}
    off = 0
    for name, shape, _ in W.param_table(cfg):
        n = int(np.prod(shape))
        out[name] = w[off:off + n].view(*shape)
        off += n
    return out


def coordinate_positions(cfg, grid_thw):
    """(tau, y, x) of every packed row, by patchifying images whose pixels hold
    their own patch coordinates (independent of the oracle's index arithmetic)."""
    P, T = cfg.patch, cfg.temporal_patch
    ys, xs, ts = [], [], []
    for (t, gh, gw) in np.asarray(grid_thw):
        t, gh, gw = int(t), int(gh), int(gw)
        img = np.zeros((cfg.in_chans, t * T, gh * P, gw * P), np.float32)
        yy = (np.arange(gh * P) // P)[:, None]
        xx = (np.arange(gw * P) // P)[None, :]
        img[0] = yy[None]
        img[1] = xx[None]
        img[2] = (np.arange(t * T) // T)[:, None, None]
        rows = W.patchify(img, P, T)
        k = T * P * P
        ys.append(rows[:, 0].astype(np.int64))
        xs.append(rows[:, k].astype(np.int64))
        ts.append(rows[:, 2 * k].astype(np.int64))
    if not ys:
        z = np.zeros(0, np.int64)
        return z, z, z
    return np.concatenate(ts), np.concatenate(ys), np.concatenate(xs)


def rope_complex(x: torch.Tensor, heads: int, d: int, py, px, theta: float):
    """Rotate pairs (j, j+d/2) as the complex number x_j + i x_{j+d/2} times e^{i a_j}."""
    N = x.shape[0]
    q = x.view(N, heads, d)
    k = torch.arange(d // 4, dtype=torch.float64)
    omega = theta ** (-4.0 * k / d)
    a = torch.cat([torch.as_tensor(py, dtype=torch.float64)[:, None] * omega[None],
                   torch.as_tensor(px, dtype=torch.float64)[:, None] * omega[None]], dim=1)
    z = torch.complex(q[..., : d // 2], q[..., d // 2:])
    z = z * torch.polar(torch.ones_like(a), a)[:, None, :]
    return torch.cat([z.real, z.imag], dim=-1).reshape(N, heads * d)


def patch_embed_conv(cfg, images, w_pe: torch.Tensor, b_pe: torch.Tensor, grid_thw):
    """Patch embedding as a strided conv3d on raw pixels, rows put in packed order."""
    P, T = cfg.patch, cfg.temporal_patch
    kern = w_pe.view(cfg.hidden, cfg.in_chans, T, P, P)
    tau, y, x = coordinate_positions(cfg, grid_thw)
    outs = []
    start = 0
    for img, (t, gh, gw) in zip(images, np.asarray(grid_thw)):
        n = int(t) * int(gh) * int(gw)
        o = F.conv3d(torch.as_tensor(img, dtype=torch.float64)[None], kern, b_pe,
                     stride=(T, P, P))[0]                 # [h, t, gh, gw]
        sl = slice(start, start + n)
        outs.append(o[:, torch.as_tensor(tau[sl]), torch.as_tensor(y[sl]),
                      torch.as_tensor(x[sl])].T)
        start += n
    return torch.cat(outs, 0)


def encoder(cfg, w: torch.Tensor, cu_seqlens, grid_thw, patches: torch.Tensor = None,
            images=None):
    """Merged output [T_m, llm_hidden].  Pass either packed patches or raw images."""
    p = split_params(cfg, w)
    h, nh = cfg.hidden, cfg.heads
    d = h // nh
    _, py, px = coordinate_positions(cfg, grid_thw)
    if images is not None:
        H = patch_embed_conv(cfg, images, p["pe.w"], p["pe.b"], grid_thw)
    else:
        H = patches @ p["pe.w"].T + p["pe.b"]
    cu = [int(v) for v in cu_seqlens]
    for l in range(cfg.layers):
        b = f"blk{l}."
        A = F.layer_norm(H, (h,), p[b + "ln1.g"], p[b + "ln1.b"], cfg.ln_eps)
        qkv = A @ p[b + "qkv.w"].T + p[b + "qkv.b"]
        q, k, v = qkv[:, :h], qkv[:, h:2 * h], qkv[:, 2 * h:]
        q = rope_complex(q, nh, d, py, px, cfg.rope_theta)
        k = rope_complex(k, nh, d, py, px, cfg.rope_theta)
        outs = []
        for s in range(len(cu) - 1):
            sl = slice(cu[s], cu[s + 1])
            qs = q[sl].view(-1, nh, d).transpose(0, 1)
            ks = k[sl].view(-1, nh, d).transpose(0, 1)
            vs = v[sl].reshape(-1, nh, d).transpose(0, 1)
            o = F.scaled_dot_product_attention(qs[None], ks[None], vs[None])[0]
            outs.append(o.transpose(0, 1).reshape(-1, h))
        O = torch.cat(outs, 0)
        H = H + O @ p[b + "proj.w"].T + p[b + "proj.b"]
        B = F.layer_norm(H, (h,), p[b + "ln2.g"], p[b + "ln2.b"], cfg.ln_eps)
        H = H + F.gelu(B @ p[b + "fc1.w"].T + p[b + "fc1.b"]) @ p[b + "fc2.w"].T + p[b + "fc2.b"]
    Z = F.layer_norm(H, (h,), p["merger.ln.g"], p["merger.ln.b"], cfg.ln_eps)
    Zc = Z.reshape(-1, 4 * h)
    U = Zc @ p["merger.fc1.w"].T + p["merger.fc1.b"]
    return F.gelu(U) @ p["merger.fc2.w"].T + p["merger.fc2.b"]
