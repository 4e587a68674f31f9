"""Seeded synthetic workloads for the replicated-encoder hot path.

This module only draws inputs: image/clip sizes, pixels, weights, placeholder
positions and upstream gradients.  It holds none of the encoder's arithmetic,
so both the CPU oracle and the HIP library can be fed from it without sharing
any computation.

The shapes follow the five encoder configurations the build is measured on
(tiny fp32 ViT, ViT-L/14 frozen and trained, the Qwen2-VL-ViT shape, and a
mixed image/video micro-batch).  The paper trains on an internal multimodal
dataset and on CapsFusion and states neither's resolution distribution
(Sec. 5, Experiments A and B); the size distributions below stand in for them.

Layout conventions shared by every consumer (they are interface, not math):

* A packed micro-batch concatenates items in order.  Inside item ``i`` with
  grid ``(t, gh, gw)`` (in patches) the rows are ordered by
  ``(tau, hb, wb, dh, dw)`` with patch position ``y = 2*hb + dh``,
  ``x = 2*wb + dw``: every 2x2 merge window is four consecutive rows.
* A patch vector is flattened in ``(c, tau', py, px)`` order.
* The flat weight buffer holds the tensors of :func:`param_table` back to back,
  each Linear weight stored ``[out, in]``.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional, Tuple

import numpy as np

__all__ = [
    "EncoderConfig", "Workload", "CONFIGS", "param_table", "param_count",
    "make_workload", "round_bf16", "bf16_bits", "bf16_bits_to_f32",
    "patchify", "draw_sizes",
]


# --------------------------------------------------------------------------
# bf16 helpers (round-to-nearest-even, the conversion both sides assume)
# --------------------------------------------------------------------------

def bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 array -> uint16 bf16 bit patterns, round to nearest even."""
    r = np.array(x, dtype=np.float32, copy=True, order="C")
    round_bf16_inplace(r)
    return (r.view(np.uint32) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32)
            << np.uint32(16)).view(np.float32)


def round_bf16_inplace(x: np.ndarray, chunk: int = 1 << 24) -> None:
    """Round a float32 array to the nearest bf16 values in place (RNE)."""
    u = x.reshape(-1).view(np.uint32)
    for i in range(0, u.size, chunk):
        c = u[i:i + chunk]
        c += ((c >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
        c &= np.uint32(0xFFFF0000)


def round_bf16(x: np.ndarray) -> np.ndarray:
    """float32 values rounded to the nearest bf16 (returned as float32)."""
    r = np.array(x, dtype=np.float32, copy=True, order="C")
    round_bf16_inplace(r)
    return r


# --------------------------------------------------------------------------
# Encoder configurations
# --------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class EncoderConfig:
    hidden: int
    layers: int
    heads: int
    mlp: int
    llm_hidden: int
    temporal_patch: int = 1
    patch: int = 14
    in_chans: int = 3
    merge: int = 2
    dtype: str = "bf16"          # activation / weight storage type: "bf16" | "f32"
    ln_eps: float = 1e-6
    rope_theta: float = 10000.0

    @property
    def head_dim(self) -> int:
        return self.hidden // self.heads

    @property
    def k_pe(self) -> int:
        return self.in_chans * self.temporal_patch * self.patch * self.patch


@dataclasses.dataclass(frozen=True)
class WorkloadSpec:
    name: str
    cfg: EncoderConfig
    trainable: int                  # 0 frozen, 1 every part trainable, 2 only the merger
    # image sizes: ("choice", values) | ("uniform28", lo, hi) | ("loguniform28", lo, hi)
    image_sizes: tuple
    n_images: int                   # fixed count, or -1 for budget-driven draws
    emb_seqs: int                   # text sequences in the LLM input buffer
    emb_seq_len: int
    video_frac: Optional[float] = None   # set for the mixed-modality draws: image fraction f
    patch_budget: int = 0
    clip_frames: int = 16
    clip_side: int = 448


_C1 = EncoderConfig(hidden=128, layers=2, heads=4, mlp=512, llm_hidden=256, dtype="f32")
_VITL = EncoderConfig(hidden=1024, layers=24, heads=16, mlp=4096, llm_hidden=4096)
_QWEN = EncoderConfig(hidden=1280, layers=32, heads=16, mlp=5120, llm_hidden=3584,
                      temporal_patch=2)

CONFIGS: Dict[str, WorkloadSpec] = {
    # tiny fp32 ViT, fwd+bwd, trained
    "c1_tiny_fp32": WorkloadSpec("c1_tiny_fp32", _C1, True, ("choice", (56, 84, 112)), 4,
                                 emb_seqs=2, emb_seq_len=256),
    # ViT-L/14 shape, bf16, frozen (forward only)
    "c2_vitl_frozen": WorkloadSpec("c2_vitl_frozen", _VITL, False, ("uniform28", 224, 672), 16,
                                   emb_seqs=4, emb_seq_len=4096),
    # ViT-L/14 shape, bf16, trained
    "c3_vitl_trained": WorkloadSpec("c3_vitl_trained", _VITL, True, ("loguniform28", 224, 1008), 32,
                                    emb_seqs=8, emb_seq_len=8192),
    # Qwen2-VL-ViT shape (~675M), bf16, trained
    "c4_qwen2vl_trained": WorkloadSpec("c4_qwen2vl_trained", _QWEN, True,
                                       ("loguniform28", 224, 1344), 24,
                                       emb_seqs=8, emb_seq_len=8192),
    # the same micro-batch with only the merger (projector) trainable: frozen blocks
    "c4_qwen2vl_merger": WorkloadSpec("c4_qwen2vl_merger", _QWEN, 2,
                                      ("loguniform28", 224, 1344), 24,
                                      emb_seqs=8, emb_seq_len=8192),
}
for _f, _tag in ((0.0, "f0"), (0.5, "f05"), (1.0, "f1")):
    for _tr in (False, True):
        _n = f"c5_mixed_{_tag}_{'trained' if _tr else 'frozen'}"
        CONFIGS[_n] = WorkloadSpec(_n, _QWEN, _tr, ("loguniform28", 224, 1344), -1,
                                   emb_seqs=8, emb_seq_len=8192, video_frac=_f,
                                   patch_budget=65536)


# --------------------------------------------------------------------------
# Parameter table (interface: names, shapes and order of the flat buffer)
# --------------------------------------------------------------------------

def param_table(cfg: EncoderConfig) -> List[Tuple[str, Tuple[int, ...], str]]:
    """(name, shape, init-kind) in flat-buffer order.  kind: w | b | g (LN gain) | beta."""
    h, m, H = cfg.hidden, cfg.mlp, cfg.llm_hidden
    mh = cfg.merge * cfg.merge * h
    t: List[Tuple[str, Tuple[int, ...], str]] = [
        ("pe.w", (h, cfg.k_pe), "w"), ("pe.b", (h,), "b")]
    for l in range(cfg.layers):
        p = f"blk{l}."
        t += [(p + "ln1.g", (h,), "g"), (p + "ln1.b", (h,), "beta"),
              (p + "qkv.w", (3 * h, h), "w"), (p + "qkv.b", (3 * h,), "b"),
              (p + "proj.w", (h, h), "w"), (p + "proj.b", (h,), "b"),
              (p + "ln2.g", (h,), "g"), (p + "ln2.b", (h,), "beta"),
              (p + "fc1.w", (m, h), "w"), (p + "fc1.b", (m,), "b"),
              (p + "fc2.w", (h, m), "w"), (p + "fc2.b", (h,), "b")]
    t += [("merger.ln.g", (h,), "g"), ("merger.ln.b", (h,), "beta"),
          ("merger.fc1.w", (mh, mh), "w"), ("merger.fc1.b", (mh,), "b"),
          ("merger.fc2.w", (H, mh), "w"), ("merger.fc2.b", (H,), "b")]
    return t


def param_count(cfg: EncoderConfig) -> int:
    return int(sum(int(np.prod(s)) for _, s, _ in param_table(cfg)))


# --------------------------------------------------------------------------
# Size draws
# --------------------------------------------------------------------------

def _draw_side(rng: np.random.Generator, dist: tuple) -> int:
    kind = dist[0]
    if kind == "choice":
        return int(rng.choice(np.asarray(dist[1])))
    lo, hi = dist[1], dist[2]
    if kind == "uniform28":
        return int(28 * rng.integers(lo // 28, hi // 28 + 1))
    if kind == "loguniform28":
        v = math.exp(rng.uniform(math.log(lo), math.log(hi)))
        return int(min(hi, max(lo, 28 * round(v / 28))))
    raise ValueError(kind)


def draw_sizes(spec: WorkloadSpec, rng: np.random.Generator) -> List[Tuple[int, int, int, bool]]:
    """Items as (frames, height_px, width_px, is_video), in packing order."""
    items: List[Tuple[int, int, int, bool]] = []
    cfg = spec.cfg
    if spec.video_frac is None:
        for _ in range(spec.n_images):
            items.append((cfg.temporal_patch, _draw_side(rng, spec.image_sizes),
                          _draw_side(rng, spec.image_sizes), False))
        return items
    # mixed modality: n_clips = round((1-f) * budget / clip_patches), then images
    # until the next one would overflow the patch budget.
    p = cfg.patch
    clip_patches = (spec.clip_frames // cfg.temporal_patch) * (spec.clip_side // p) ** 2
    n_clips = int(round((1.0 - spec.video_frac) * spec.patch_budget / clip_patches))
    used = n_clips * clip_patches
    clips = [(spec.clip_frames, spec.clip_side, spec.clip_side, True)] * n_clips
    images = []
    while spec.video_frac > 0:
        hp, wp = _draw_side(rng, spec.image_sizes), _draw_side(rng, spec.image_sizes)
        n = (hp // p) * (wp // p)
        if used + n > spec.patch_budget:
            break
        used += n
        images.append((cfg.temporal_patch, hp, wp, False))
    # interleave clips and images in a seeded order
    items = clips + images
    order = rng.permutation(len(items))
    return [items[i] for i in order]


# --------------------------------------------------------------------------
# Patchify (input layout only)
# --------------------------------------------------------------------------

def patchify(img: np.ndarray, patch: int, temporal_patch: int) -> np.ndarray:
    """[C, F, Hpx, Wpx] -> [t*gh*gw, C*T*P*P] in the window-major row order."""
    C, F, Hp, Wp = img.shape
    T, P = temporal_patch, patch
    t, gh, gw = F // T, Hp // P, Wp // P
    x = img.reshape(C, t, T, gh // 2, 2, P, gw // 2, 2, P)
    # axes: c, tau, tau', hb, dh, py, wb, dw, px  ->  tau, hb, wb, dh, dw, c, tau', py, px
    x = x.transpose(1, 3, 6, 4, 7, 0, 2, 5, 8)
    return np.ascontiguousarray(x.reshape(t * gh * gw, C * T * P * P))


# --------------------------------------------------------------------------
# Workload
# --------------------------------------------------------------------------

@dataclasses.dataclass
class Workload:
    spec: WorkloadSpec
    seed: int
    grid_thw: np.ndarray            # int32 [n_items, 3], in patches
    cu_seqlens: np.ndarray          # int32 [n_items + 1], one attention segment per item
    sharp: bool
    _streams: list

    @property
    def cfg(self) -> EncoderConfig:
        return self.spec.cfg

    @property
    def name(self) -> str:
        return self.spec.name

    @property
    def trainable(self) -> int:
        """Trainability mode: 0 frozen, 1 every part trainable, 2 only the merger."""
        return int(self.spec.trainable)

    @property
    def n_items(self) -> int:
        return int(self.grid_thw.shape[0])

    @property
    def n_patches(self) -> int:
        return int(self.cu_seqlens[-1])

    @property
    def merged_per_item(self) -> np.ndarray:
        t, gh, gw = self.grid_thw[:, 0], self.grid_thw[:, 1], self.grid_thw[:, 2]
        return (t * (gh // 2) * (gw // 2)).astype(np.int64)

    @property
    def n_merged(self) -> int:
        return int(self.merged_per_item.sum())

    @property
    def emb_rows(self) -> int:
        return self.spec.emb_seqs * self.spec.emb_seq_len

    def _rng(self, k: int) -> np.random.Generator:
        return np.random.Generator(np.random.PCG64(self._streams[k]))

    # -- pixels ------------------------------------------------------------
    def images(self) -> List[np.ndarray]:
        """Raw pixel tensors [C, F, Hpx, Wpx], uniform[-1, 1] (bf16-rounded for bf16 configs).

        Images of a temporal-patch-2 encoder are one frame repeated twice."""
        rng = self._rng(1)
        cfg = self.cfg
        out = []
        for (t, gh, gw) in self.grid_thw:
            frames = int(t) * cfg.temporal_patch
            hp, wp = int(gh) * cfg.patch, int(gw) * cfg.patch
            is_image = (int(t) == 1)
            nf = 1 if is_image else frames
            px = rng.uniform(-1.0, 1.0, size=(cfg.in_chans, nf, hp, wp)).astype(np.float32)
            if is_image and frames > 1:
                px = np.repeat(px, frames, axis=1)
            if cfg.dtype == "bf16":
                px = round_bf16(px)
            out.append(px)
        return out

    def patches(self) -> np.ndarray:
        """Packed patch matrix [N, K_pe] (float32, bf16-exact for bf16 configs)."""
        cfg = self.cfg
        parts = [patchify(im, cfg.patch, cfg.temporal_patch) for im in self.images()]
        if not parts:
            return np.zeros((0, cfg.k_pe), np.float32)
        return np.concatenate(parts, axis=0)

    # -- weights -----------------------------------------------------------
    def weights(self) -> np.ndarray:
        """Flat weight buffer (float32; bf16-exact for bf16 configs).

        Linear weights and biases ~ N(0, 0.02); LN gain 1 + N(0, 0.02),
        LN shift N(0, 0.02).  The 'sharp' draw uses std 0.1 for the qkv weights
        so that attention rows are far from uniform."""
        rng = self._rng(2)
        cfg = self.cfg
        w = np.empty(param_count(cfg), np.float32)
        off = 0
        for name, shape, kind in param_table(cfg):
            n = int(np.prod(shape))
            seg = w[off:off + n]
            std = 0.1 if (self.sharp and name.endswith("qkv.w")) else 0.02
            rng.standard_normal(out=seg, dtype=np.float32)
            seg *= np.float32(std)
            if kind == "g":
                seg += np.float32(1.0)
            off += n
        if cfg.dtype == "bf16":
            round_bf16_inplace(w)
        return w

    # -- placeholders ------------------------------------------------------
    def placeholders(self) -> np.ndarray:
        """int64 [n_merged]: flat row of the LLM input buffer for merged row j.

        One contiguous run per item; runs are spread over the text sequences
        in item order, never cross a sequence, and sit at random offsets."""
        rng = self._rng(3)
        B, S = self.spec.emb_seqs, self.spec.emb_seq_len
        runs = self.merged_per_item
        total = int(runs.sum())
        if total == 0:
            return np.zeros(0, np.int64)
        seq_of = np.zeros(len(runs), np.int64)
        fill = np.zeros(B, np.int64)
        s = 0
        cum = 0
        for i, r in enumerate(runs):
            target = min(B - 1, int(B * (cum + r / 2.0) / total))
            s = max(s, target)
            while fill[s] + r > S:
                s += 1
                if s >= B:
                    raise ValueError("placeholder runs do not fit the text sequences")
            seq_of[i] = s
            fill[s] += r
            cum += int(r)
        idx = np.empty(total, np.int64)
        pos = 0
        for sq in range(B):
            members = np.nonzero(seq_of == sq)[0]
            if len(members) == 0:
                continue
            free = S - int(runs[members].sum())
            k = len(members)
            # k+1 non-negative gaps summing to `free`, uniformly (stars and bars)
            bars = np.sort(rng.choice(free + k, size=k, replace=False))
            gaps = np.diff(np.concatenate([[-1], bars])) - 1
            off = 0
            for g, it in zip(gaps, members):
                off += int(g)
                r = int(runs[it])
                idx[pos:pos + r] = sq * S + off + np.arange(r)
                pos += r
                off += r
        return idx

    # -- LLM-side buffers --------------------------------------------------
    def emb_init(self) -> np.ndarray:
        """Text embeddings already in the LLM input buffer, N(0, 1)."""
        rng = self._rng(4)
        v = rng.standard_normal((self.emb_rows, self.cfg.llm_hidden), dtype=np.float32)
        return round_bf16(v) if self.cfg.dtype == "bf16" else v

    def d_emb(self) -> np.ndarray:
        """Upstream gradient of the LLM input buffer, N(0, 1)."""
        rng = self._rng(5)
        v = rng.standard_normal((self.emb_rows, self.cfg.llm_hidden), dtype=np.float32)
        return round_bf16(v) if self.cfg.dtype == "bf16" else v

    def d_merged(self) -> np.ndarray:
        """Upstream gradient of the merged rows (the gather of d_emb at the placeholders)."""
        return np.ascontiguousarray(self.d_emb()[self.placeholders()])


def make_workload(name: str, seed: int = 0, *, sharp: bool = False,
                  grid_thw: Optional[np.ndarray] = None) -> Workload:
    """Draw workload `name` with seed `seed` (5 independent PCG64 streams:
    sizes, pixels, weights, placeholders, LLM-side buffers / upstream grads)."""
    spec = CONFIGS[name]
    ss = np.random.SeedSequence(seed)
    streams = ss.spawn(6)
    if grid_thw is None:
        rng = np.random.Generator(np.random.PCG64(streams[0]))
        items = draw_sizes(spec, rng)
        p, T = spec.cfg.patch, spec.cfg.temporal_patch
        grid = np.array([[f // T, hp // p, wp // p] for (f, hp, wp, _) in items],
                        dtype=np.int32).reshape(-1, 3)
    else:
        grid = np.ascontiguousarray(grid_thw, dtype=np.int32).reshape(-1, 3)
    n = grid[:, 0].astype(np.int64) * grid[:, 1] * grid[:, 2]
    cu = np.concatenate([[0], np.cumsum(n)]).astype(np.int32)
    return Workload(spec=spec, seed=seed, grid_thw=grid, cu_seqlens=cu, sharp=sharp,
                    _streams=streams)


def custom_spec(name: str, cfg: EncoderConfig, trainable: bool = True,
                emb_seqs: int = 2, emb_seq_len: int = 256) -> WorkloadSpec:
    """A spec for hand-built test shapes (sizes come from an explicit grid_thw)."""
    spec = WorkloadSpec(name, cfg, trainable, ("choice", (56,)), 0,
                        emb_seqs=emb_seqs, emb_seq_len=emb_seq_len)
    CONFIGS[name] = spec
    return spec
