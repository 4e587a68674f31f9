"""C-ABI checks that need no GPU: the library loads, exports every symbol the
headers declare, its parameter table agrees with the generator's and the
oracle's, and every metadata check fails on the host before any launch."""
import ctypes as C
import os
import re

import numpy as np
import pytest

import oracle
import workload as W
from paper_2607_03229_amd import _binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    names = set()
    for h in ("mpipe.h", "mpipe_ops.h", "mpipe_sched.h", "mpipe_derive.h"):
        src = open(os.path.join(ROOT, "include", h)).read()
        src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
        names |= set(re.findall(r"\b(mpipe_[a-z0-9_]+)\s*\(", src))
    return sorted(names)


@pytest.fixture(scope="module")
def L():
    return B.load()


def test_exports_every_declared_symbol(L):
    names = _declared_functions()
    assert len(names) >= 20
    for n in names:
        assert hasattr(L, n), f"{n} declared in include/ but not exported"


def test_param_table_agrees_three_ways(L):
    for name in ("c1_tiny_fp32", "c2_vitl_frozen", "c4_qwen2vl_trained"):
        cfg = W.CONFIGS[name].cfg
        enc = B.Encoder(cfg)
        lt = enc.param_table()
        ot = oracle.param_table(cfg)
        gt = W.param_table(cfg)
        assert enc.param_count() == oracle.param_count(cfg) == W.param_count(cfg)
        assert [(n, o, r, c) for n, o, r, c in lt] == ot
        assert [n for n, _, _, _ in lt] == [g[0] for g in gt]
        enc.close()


def test_unsupported_configs_rejected(L):
    good = W.CONFIGS["c4_qwen2vl_trained"].cfg
    import dataclasses
    for bad in (dict(heads=12), dict(hidden=1000), dict(merge=3), dict(mlp=5121),
                dict(llm_hidden=3583)):
        cfg = dataclasses.replace(good, **bad)
        with pytest.raises(B.MpipeError) as e:
            B.Encoder(cfg)
        assert e.value.status == -5


@pytest.mark.parametrize("trainable", [0, 1, 2])
def test_workspace_and_tape_regions(L, trainable):
    """The writable ranges the planner lays out: inside the buffer, in order, and each
    followed by at least 256 unwritten guard bytes (the canary check of the GPU test
    relies on this)."""
    wl = W.make_workload("c4_qwen2vl_trained", 0)
    enc = B.Encoder(wl.cfg)
    s = enc.sizes(wl.cu_seqlens, wl.grid_thw, trainable)
    for which, total in ((0, s["workspace"]), (1, s["tape"])):
        r = enc.regions(wl.cu_seqlens, wl.grid_thw, trainable, which)
        if which == 1 and trainable == 0:
            assert len(r) == 0 and total == 0
            continue
        assert len(r) > 0 and (r[:, 1] > 0).all() and (r[:, 0] % 256 == 0).all()
        ends = r[:, 0] + r[:, 1]
        assert (r[1:, 0] >= ends[:-1] + 256).all()
        assert ends[-1] + 256 <= total
    enc.close()


def test_weight_grad_split_plan(L):
    """The split plan the backward uses (host query): no split below 2,048 tokens, the
    benchmark's weight gradients split, at most four ways, rejected sizes answer -1."""
    import paper_2607_03229_amd as mp
    assert mp.gemm_split(3840, 1280, 656) == 1
    assert mp.gemm_split(3840, 1280, 2047) == 1
    for M, N in ((3840, 1280), (1280, 1280), (5120, 1280), (1280, 5120), (1280, 1176)):
        s = mp.gemm_split(M, N, 42940)
        assert 2 <= s <= 4, (M, N, s)
    assert mp.gemm_split(-1, 8, 8) == -1


def test_sizes_and_metadata_validation(L):
    wl = W.make_workload("c4_qwen2vl_trained", 0)
    enc = B.Encoder(wl.cfg)
    s = enc.sizes(wl.cu_seqlens, wl.grid_thw, True)
    assert s["n_patches"] == wl.n_patches and s["n_merged"] == wl.n_merged
    assert s["tape"] > 0 and s["workspace"] > 0
    sf = enc.sizes(wl.cu_seqlens, wl.grid_thw, False)
    assert sf["tape"] == 0
    cu, g = wl.cu_seqlens, wl.grid_thw
    bad_cases = [
        (cu[:-1], g),                                              # does not reach N
        (np.concatenate([[0], cu[2:]]), g),                        # segment crosses an item
        (cu, np.vstack([[[1, 5, 4]], g[1:]])),                     # odd grid height
        (np.array([0, 5, 3] + list(cu[3:])), g),                   # not increasing
    ]
    for c2, g2 in bad_cases:
        with pytest.raises(B.MpipeError) as e:
            enc.sizes(c2, g2, True)
        assert e.value.status == -2
    # per-temporal-slice segments accepted for a video item
    gv = np.array([[4, 6, 8]], np.int32)
    assert enc.sizes(np.arange(0, 4 * 48 + 1, 48), gv, True)["n_patches"] == 192
    with pytest.raises(B.MpipeError):
        enc.sizes(np.array([0, 30, 192]), gv, True)
    # grid sides: positions are packed y << 16 | x, so a side may be at most 32768 patches
    # (a larger coordinate would reach the sign bit of the packed int32)
    for side, ok in ((32768, True), (32770, False), (65534, False)):
        for gg in (np.array([[1, side, 2]], np.int32), np.array([[1, 2, side]], np.int32)):
            n = int(gg[0].prod())
            if ok:
                assert enc.sizes(np.array([0, n]), gg, False)["n_patches"] == n
            else:
                with pytest.raises(B.MpipeError) as e:
                    enc.sizes(np.array([0, n]), gg, False)
                assert e.value.status == -2
    # empty micro-batch (text only) is a valid no-op
    e0 = enc.sizes(np.array([0]), np.zeros((0, 3), np.int32), True)
    assert e0["n_patches"] == 0 and e0["n_merged"] == 0
    enc.close()


def _call_fwd(L, enc, cu, g, trainable, tape_bytes=0, ws_bytes=0):
    cu = np.ascontiguousarray(cu, np.int32)
    g = np.ascontiguousarray(g, np.int32).reshape(-1, 3)
    fake = C.c_void_p(0x1000)   # never dereferenced: the call must fail on the host first
    return L.mpipe_encoder_fwd(enc._h, fake, fake, cu.ctypes.data_as(C.c_void_p), len(cu) - 1,
                               g.ctypes.data_as(C.c_void_p), g.shape[0], trainable, fake,
                               fake if tape_bytes else None, tape_bytes, fake, ws_bytes, None)


def test_host_errors_before_any_launch(L):
    wl = W.make_workload("c1_tiny_fp32", 0)
    enc = B.Encoder(wl.cfg)
    s = enc.sizes(wl.cu_seqlens, wl.grid_thw, True)
    # workspace too small
    assert _call_fwd(L, enc, wl.cu_seqlens, wl.grid_thw, 1, s["tape"], s["workspace"] - 1) == -3
    # trained forward without a tape
    assert _call_fwd(L, enc, wl.cu_seqlens, wl.grid_thw, 1, 0, s["workspace"]) == -4
    # bad metadata
    assert _call_fwd(L, enc, wl.cu_seqlens[:-1], wl.grid_thw, 0, 0, 1 << 30) == -2
    assert "cu_seqlens" in B.last_error()
    # empty micro-batch: OK without touching any buffer
    assert _call_fwd(L, enc, [0], np.zeros((0, 3)), 1) == 0
    # backward on a frozen encoder: NOOP_FROZEN, nothing written (Lemma 1)
    fake = C.c_void_p(0x1000)
    cu = np.ascontiguousarray(wl.cu_seqlens, np.int32)
    g = np.ascontiguousarray(wl.grid_thw, np.int32)
    rc = L.mpipe_encoder_bwd(enc._h, fake, fake, cu.ctypes.data_as(C.c_void_p), len(cu) - 1,
                             g.ctypes.data_as(C.c_void_p), g.shape[0], 0, None, 0, fake, fake,
                             None, fake, 1, None)
    assert rc == 1
    # backward without a tape
    rc = L.mpipe_encoder_bwd(enc._h, fake, fake, cu.ctypes.data_as(C.c_void_p), len(cu) - 1,
                             g.ctypes.data_as(C.c_void_p), g.shape[0], 1, None, 0, fake, fake,
                             None, fake, s["workspace"], None)
    assert rc == -4
    enc.close()


def test_scatter_argument_checks(L):
    fake = C.c_void_p(0x1000)
    assert L.mpipe_merge_scatter(fake, 4, 16, 7, fake, fake, 10, None) == -1      # bad dtype
    assert L.mpipe_merge_scatter(fake, 4, 0, 1, fake, fake, 10, None) == -1       # bad width
    assert L.mpipe_merge_scatter(None, 4, 16, 1, fake, fake, 10, None) == -1      # null buffer
    assert L.mpipe_merge_scatter(None, 0, 16, 1, None, None, 10, None) == 0       # nothing to do


def test_gemm_op_argument_checks(L):
    fake = C.c_void_p(0x1000)
    # bf16 NT with K not a multiple of 8 is refused before launch
    assert L.mpipe_op_gemm(1, 0, 0, 16, 16, 12, fake, 12, fake, 12, fake, 16, None, None, 0,
                           None, 0, 0, 0, 0, None) == -1
    assert L.mpipe_op_gemm(1, 3, 0, 16, 16, 16, fake, 16, fake, 16, fake, 16, None, None, 0,
                           None, 0, 0, 0, 0, None) == -1


def test_merger_only_mode_host_side(L):
    """Trainability modes on the host: the merger-only tape holds the merger's inputs
    only (far smaller than the full tape, larger than nothing), an unknown mode is
    rejected, and the merger as trainable source refuses to send a patch gradient."""
    wl = W.make_workload("c4_qwen2vl_trained", 0)
    enc = B.Encoder(wl.cfg)
    full = enc.sizes(wl.cu_seqlens, wl.grid_thw, 1)
    part = enc.sizes(wl.cu_seqlens, wl.grid_thw, 2)
    N, h, Tm = wl.n_patches, wl.cfg.hidden, wl.n_merged
    # final residual (fp32), LN output (bf16), LN stats, GELU' and GELU of fc1 (bf16)
    expect = N * h * 4 + N * h * 2 + 2 * N * 4 + 2 * Tm * 4 * h * 2
    # six regions, each padded to 256-byte alignment and followed by a 256-byte guard
    assert expect <= part["tape"] <= expect + 6 * 512
    assert part["tape"] * 20 < full["tape"]
    assert part["n_merged"] == full["n_merged"]
    for bad in (3, -1):
        with pytest.raises(B.MpipeError) as e:
            enc.sizes(wl.cu_seqlens, wl.grid_thw, bad)
        assert e.value.status == -1
    fake = C.c_void_p(0x1000)
    cu = np.ascontiguousarray(wl.cu_seqlens, np.int32)
    g = np.ascontiguousarray(wl.grid_thw, np.int32)
    rc = L.mpipe_encoder_bwd(enc._h, fake, fake, cu.ctypes.data_as(C.c_void_p), len(cu) - 1,
                             g.ctypes.data_as(C.c_void_p), g.shape[0], 2, fake, part["tape"],
                             fake, fake, fake, fake, part["workspace"], None)
    assert rc == -1 and "d_patches" in B.last_error()
    enc.close()
