"""Per-kernel parity on the GPU: each HIP kernel (through the op C-ABI) against
the oracle's building block on the same seeded inputs, at sizes spanning
several tiles with ragged tails."""
import numpy as np
import pytest

import oracle
from tests.gpu_util import announce, host, max_rel, nans, rnd, to_dev, torch_dev, zeros

pytestmark = pytest.mark.gpu

NT, NN, TN = 0, 1, 2
E_STORE, E_GELU, E_RESID, E_GELUBWD, E_F32 = range(5)
TOL = {"bf16": 1e-2, "f32": 2e-5}


def _dt(s):
    return 1 if s == "bf16" else 0


def _ref_product(layout, A, B):
    if layout == NT:
        return oracle.linear(A, B)
    if layout == NN:
        return oracle.linear(A, B.T)
    return oracle.linear(A.T, B.T)


GEMM_SHAPES = {
    # small shapes use the 128x128 kernel; M >= 512 and N >= 256 use the 256x256 kernel
    # (the large kernel's K pipeline: 1 to 3 tiles, ragged last tiles, several passes)
    NT: [(300, 200, 256), (1, 8, 8), (129, 257, 72), (512, 384, 1280), (700, 520, 200),
         (1030, 588, 64), (600, 300, 24), (520, 264, 96), (515, 260, 168), (520, 264, 264),
         (530, 256, 1000)],
    NN: [(300, 200, 256), (129, 264, 72), (77, 8, 520), (600, 264, 136), (777, 1032, 1280),
         (530, 280, 40)],
    TN: [(200, 264, 333), (8, 16, 1), (136, 128, 1000), (520, 264, 1000), (1280, 600, 77),
         (512, 256, 5), (600, 392, 63), (600, 392, 250), (520, 264, 291),
         (1280, 1176, 700)],
}


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("layout", [NT, NN, TN])
def test_gemm_layouts(dtype, layout):
    import paper_2607_03229_amd as mp
    torch, dev = torch_dev()
    rng = np.random.default_rng(10 * layout + len(dtype))
    for (M, N, K) in GEMM_SHAPES[layout]:
        if dtype == "f32" and layout != TN and K % 4:
            continue
        announce(f"gemm {dtype} layout={layout} M={M} N={N} K={K}")
        A = rnd(rng, (K, M) if layout == TN else (M, K), dtype)
        B = rnd(rng, (N, K) if layout == NT else (K, N), dtype)
        ref = _ref_product(layout, A, B)
        C = nans((M, N), "f32")
        mp.op_gemm(_dt(dtype), layout, E_F32, M, N, K, to_dev(A, dtype), A.shape[1],
                   to_dev(B, dtype), B.shape[1], C, N)
        torch.cuda.synchronize()
        err = max_rel(host(C), ref)
        assert err < (2e-5 if dtype == "f32" else 1e-5), (M, N, K, err)


@pytest.mark.parametrize("layout", [NT, NN])
@pytest.mark.parametrize("dtype,M,N,K", [("bf16", 333, 264, 192), ("f32", 333, 264, 192),
                                         ("bf16", 700, 392, 256), ("bf16", 530, 300, 64),
                                         ("bf16", 1100, 520, 360)])
def test_gemm_epilogues(dtype, M, N, K, layout):
    """Fused epilogues; (700, 392) and (1100, 520) run the large-tile kernels (256x256
    tiles for NT, 128x256 for NN); (530, 300) has N % 8 != 0 (rows that break 16-byte
    alignment), which the dispatcher sends to the general kernel.  NN takes the weight
    as [K][N]."""
    import paper_2607_03229_amd as mp
    torch, dev = torch_dev()
    rng = np.random.default_rng(7)
    A, B, bias = rnd(rng, (M, K), dtype), rnd(rng, (N, K), dtype, 0.1), rnd(rng, (N,), dtype)
    dA, db = to_dev(A, dtype), to_dev(bias, dtype)
    if layout == NT:
        dB, ldb = to_dev(B, dtype), K
    else:   # [K][N] in rows padded to a multiple of 8 (a K-major operand's stride rule)
        ldb = (N + 7) // 8 * 8
        BT = np.zeros((K, ldb), np.float32)
        BT[:, :N] = B.T
        dB = to_dev(BT, dtype)
    pre = oracle.linear(A, B, bias)
    # store with bias
    announce(f"gemm epilogue store {dtype} layout={layout}")
    C = nans((M, N), dtype)
    mp.op_gemm(_dt(dtype), layout, E_STORE, M, N, K, dA, K, dB, ldb, C, N, bias=db)
    assert max_rel(host(C), pre) < TOL[dtype]
    # GELU, with GELU' of the pre-activation stored for the backward
    announce(f"gemm epilogue gelu {dtype} layout={layout}")
    C, C2 = nans((M, N), dtype), nans((M, N), dtype)
    mp.op_gemm(_dt(dtype), layout, E_GELU, M, N, K, dA, K, dB, ldb, C, N, bias=db, C2=C2, ldc2=N)
    assert max_rel(host(C2), oracle.gelu_grad(pre)) < TOL[dtype]
    assert max_rel(host(C), oracle.gelu(pre)) < TOL[dtype]
    # residual update in place (aux aliases C)
    announce(f"gemm epilogue resid {dtype} layout={layout}")
    R = rng.standard_normal((M, N)).astype(np.float32)
    C = to_dev(R, "f32")
    mp.op_gemm(_dt(dtype), layout, E_RESID, M, N, K, dA, K, dB, ldb, C, N, bias=db, aux=C, ld_aux=N)
    assert max_rel(host(C), R + pre) < 2e-5
    # GELU backward: acc * aux, aux = GELU'(u) as the forward epilogue stores it
    announce(f"gemm epilogue gelu-bwd {dtype} layout={layout}")
    U = rnd(rng, (M, N), dtype)
    Gd = oracle.gelu_grad(U).astype(np.float32)
    C = nans((M, N), dtype)
    mp.op_gemm(_dt(dtype), layout, E_GELUBWD, M, N, K, dA, K, dB, ldb, C, N, aux=to_dev(Gd, dtype),
               ld_aux=N)
    assert max_rel(host(C), oracle.linear(A, B) * oracle.gelu_grad(U)) < TOL[dtype]
    # fp32 accumulate (beta = 1)
    announce(f"gemm epilogue f32 accumulate {dtype} layout={layout}")
    C = to_dev(R, "f32")
    mp.op_gemm(_dt(dtype), layout, E_F32, M, N, K, dA, K, dB, ldb, C, N, beta=1)
    assert max_rel(host(C), R + oracle.linear(A, B)) < 2e-5


@pytest.mark.parametrize("dtype,M,N,K,kps", [("bf16", 136, 264, 1000, 256),
                                              ("f32", 136, 264, 1000, 256),
                                              ("bf16", 520, 264, 1000, 256),
                                              ("bf16", 1280, 768, 3000, 1024)])
@pytest.mark.parametrize("ldo_pad", [0, 3])
def test_gemm_split_k(dtype, M, N, K, kps, ldo_pad):
    """The weight-gradient route of the backward: the TN GEMM writes one fp32 partial per K
    split, and the split-K reduction adds the partials, in split order, into a d_weights
    block that already holds a value (Accumulate).  Checked against the oracle's Linear
    backward, dW = dY^T X.  ldo_pad = 0 takes the four-column reduction, 3 the
    one-column one (a row stride that is not a multiple of 4)."""
    import paper_2607_03229_amd as mp
    torch, dev = torch_dev()
    rng = np.random.default_rng(3 + M)
    announce(f"gemm split-k {dtype} M={M} N={N} K={K} kps={kps} ldo_pad={ldo_pad}")
    A, B = rnd(rng, (K, M), dtype), rnd(rng, (K, N), dtype)
    splits = (K + kps - 1) // kps
    part = nans((splits, M, N), "f32")
    mp.op_gemm(_dt(dtype), TN, E_F32, M, N, K, to_dev(A, dtype), M, to_dev(B, dtype), N, part, N,
               k_per_split=kps, split_stride=M * N)
    got = host(part)
    for s in range(splits):
        sl = slice(s * kps, min(K, (s + 1) * kps))
        _, ref_s, _ = oracle.linear_bwd(A[sl], B[sl], np.zeros((M, N)))
        assert max_rel(got[s], ref_s) < 2e-5, s
    # reduce into an accumulating target
    ldo = N + ldo_pad
    base = rng.standard_normal((M, ldo)).astype(np.float32)
    out = to_dev(base, "f32")
    mp.op_splitk_reduce(part, splits, M, N, out, ldo)
    res = host(out)
    _, ref, _ = oracle.linear_bwd(A, B, np.zeros((M, N)))
    assert max_rel(res[:, :N], base[:, :N] + ref) < 2e-5
    np.testing.assert_array_equal(res[:, N:], base[:, N:])   # the stride's pad untouched
    # the two reduction paths add in the same order: bitwise the same sums
    if ldo_pad:
        out4 = to_dev(base[:, :N], "f32")
        mp.op_splitk_reduce(part, splits, M, N, out4, N)
        np.testing.assert_array_equal(host(out4), res[:, :N])


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("n", [128, 1024, 1280])
def test_layernorm_fwd_bwd(dtype, n):
    import paper_2607_03229_amd as mp
    torch, dev = torch_dev()
    rng = np.random.default_rng(n)
    rows = 333
    announce(f"layernorm {dtype} n={n}")
    X = (rng.standard_normal((rows, n)) * 3 + 1).astype(np.float32)
    g, b = rnd(rng, (n,), dtype, 0.1, 1.0), rnd(rng, (n,), dtype, 0.1)
    Y = nans((rows, n), dtype)
    mean, rstd = nans((rows,), "f32"), nans((rows,), "f32")
    dX_ = to_dev(X, "f32")
    mp.op_layernorm_fwd(_dt(dtype), dX_, rows, n, to_dev(g, dtype), to_dev(b, dtype), 1e-6, Y,
                        mean, rstd)
    ry, rmu, rrs = oracle.layernorm(X, g, b, 1e-6)
    assert max_rel(host(Y), ry) < TOL[dtype]
    assert max_rel(host(mean), rmu) < 1e-5 and max_rel(host(rstd), rrs) < 1e-5
    dY = rng.standard_normal((rows, n)).astype(np.float32)
    dres = rng.standard_normal((rows, n)).astype(np.float32)
    dX, dXt = nans((rows, n), "f32"), nans((rows, n), dtype)
    gg, gb = to_dev(np.ones(n), "f32"), to_dev(np.zeros(n), "f32")
    gc = to_dev(np.full(n, 2.0), "f32")
    scratch = torch.empty(mp.op_scratch_bytes(rows, 1, n, 0), dtype=torch.uint8, device=dev)
    mp.op_layernorm_bwd(_dt(dtype), to_dev(dY, "f32"), dX_, mean, rstd, to_dev(g, dtype), rows, n,
                        to_dev(dres, "f32"), dX, dXt, gg, gb, scratch, colsum_dx=gc)
    rdx, rdg, rdb = oracle.layernorm_bwd(dY, X, g, rmu, rrs)
    assert max_rel(host(dX), rdx + dres) < 1e-4
    assert max_rel(host(dXt), rdx + dres) < TOL[dtype]
    assert max_rel(host(gg), 1 + rdg) < 1e-4 and max_rel(host(gb), rdb) < 1e-4
    # the fused column sums of dX, accumulated onto 2 (the bias-gradient Accumulate)
    assert max_rel(host(gc), 2.0 + (rdx + dres).sum(axis=0)) < 1e-4
    # without colsum_dx, and without dX (affine gradients only), nothing else changes
    gg2, gb2 = to_dev(np.zeros(n), "f32"), to_dev(np.zeros(n), "f32")
    mp.op_layernorm_bwd(_dt(dtype), to_dev(dY, "f32"), dX_, mean, rstd, to_dev(g, dtype), rows, n,
                        None, None, None, gg2, gb2, scratch)
    assert max_rel(host(gg2), rdg) < 1e-4 and max_rel(host(gb2), rdb) < 1e-4


@pytest.mark.parametrize("dtype,heads,d", [("bf16", 16, 80), ("bf16", 4, 64), ("f32", 4, 32)])
def test_rope(dtype, heads, d):
    import paper_2607_03229_amd as mp
    torch, dev = torch_dev()
    grid = np.array([[1, 6, 8], [2, 4, 4], [1, 96, 2]], np.int32)
    N = int((grid[:, 0] * grid[:, 1] * grid[:, 2]).sum())
    announce(f"rope {dtype} heads={heads} d={d} N={N}")
    rng = np.random.default_rng(d)
    h = heads * d
    qkv = rnd(rng, (N, 3 * h), dtype)
    t = to_dev(qkv, dtype)
    scratch = torch.empty(mp.op_scratch_bytes(N, heads, h, 3), dtype=torch.uint8, device=dev)
    mp.op_rope(_dt(dtype), t, N, heads, d, grid, 10000.0, 0, scratch)
    py, px = oracle.positions(grid)
    got = host(t)
    for part in (0, 1):
        ref = oracle.rope2d(qkv[:, part * h:(part + 1) * h], heads, d, py, px)
        assert max_rel(got[:, part * h:(part + 1) * h], ref) < TOL[dtype]
    np.testing.assert_array_equal(got[:, 2 * h:], qkv[:, 2 * h:])    # v untouched
    mp.op_rope(_dt(dtype), t, N, heads, d, grid, 10000.0, 1, scratch)
    assert max_rel(host(t), qkv) < 2 * TOL[dtype]


# segment lengths: empty-ish, sub-tile, exact tiles, ragged tails, and long segments that
# run the pipelined steady state over several loop passes (1000 = 16 key tiles)
ATTN_LENS = [1, 5, 64, 127, 128, 129, 300, 16, 1000, 705]


def test_attention_longest_segments():
    """The longest segments the workloads hold: a 1344 x 1344 image (9,216 patches) and a
    ragged 8,229-row segment, d = 80, forward and backward against the oracle.  Many key
    tiles per query test the lazily moved softmax offset and the long accumulations."""
    import paper_2607_03229_amd as mp
    torch, dev = torch_dev()
    lens = [9216, 8229]
    heads, d = 2, 80
    h = heads * d
    rng = np.random.default_rng(77)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    N = int(cu[-1])
    announce(f"attention longest segments {lens} heads={heads} d={d}")
    qkv = rnd(rng, (N, 3 * h), "bf16", 1.5)
    q, k, v = qkv[:, :h], qkv[:, h:2 * h], qkv[:, 2 * h:]
    tq = to_dev(qkv, "bf16")
    o, lse = nans((N, h), "bf16"), nans((heads, N), "f32")
    scratch = torch.empty(mp.op_scratch_bytes(N, heads, h, len(lens)), dtype=torch.uint8,
                          device=dev)
    mp.op_attention_fwd(_dt("bf16"), tq, N, heads, d, cu, o, lse, scratch)
    dO = rnd(rng, (N, h), "bf16")
    dqkv = nans((N, 3 * h), "bf16")
    mp.op_attention_bwd(_dt("bf16"), tq, o, to_dev(dO, "bf16"), lse, N, heads, d, cu, dqkv,
                        scratch)
    got_o, got_lse, got = host(o), host(lse), host(dqkv)
    ro, rlse = oracle.attention(q, k, v, cu, heads, d)
    assert max_rel(got_o, ro) < 2e-2
    assert max_rel(got_lse, rlse.T) < 1e-3
    rdq, rdk, rdv = oracle.attention_bwd(q, k, v, ro, dO, rlse, cu, heads, d)
    for name, sl, ref in (("dq", slice(0, h), rdq), ("dk", slice(h, 2 * h), rdk),
                          ("dv", slice(2 * h, 3 * h), rdv)):
        err = max_rel(got[:, sl], ref)
        print(f"longest segments {name}: max-rel {err:.2e}")
        assert err < 2e-2, (name, err)


@pytest.mark.parametrize("dtype,heads,d", [("bf16", 2, 80), ("bf16", 2, 64), ("bf16", 3, 32),
                                           ("f32", 2, 32)])
def test_attention_fwd_bwd(dtype, heads, d):
    import paper_2607_03229_amd as mp
    torch, dev = torch_dev()
    rng = np.random.default_rng(d + heads)
    cu = np.concatenate([[0], np.cumsum(ATTN_LENS)]).astype(np.int32)
    N = int(cu[-1])
    h = heads * d
    announce(f"attention {dtype} heads={heads} d={d} N={N}")
    qkv = rnd(rng, (N, 3 * h), dtype, 1.5)
    q, k, v = qkv[:, :h], qkv[:, h:2 * h], qkv[:, 2 * h:]
    ro, rlse = oracle.attention(q, k, v, cu, heads, d)
    tq = to_dev(qkv, dtype)
    o, lse = nans((N, h), dtype), nans((heads, N), "f32")
    scratch = torch.empty(mp.op_scratch_bytes(N, heads, h, len(ATTN_LENS)), dtype=torch.uint8,
                          device=dev)
    mp.op_attention_fwd(_dt(dtype), tq, N, heads, d, cu, o, lse, scratch)
    tol = 2e-2 if dtype == "bf16" else 1e-5
    assert max_rel(host(o), ro) < tol
    assert max_rel(host(lse), rlse.T) < (1e-3 if dtype == "bf16" else 1e-5)
    announce(f"attention bwd {dtype} heads={heads} d={d} N={N}")
    dO = rnd(rng, (N, h), dtype)
    rdq, rdk, rdv = oracle.attention_bwd(q, k, v, ro, dO, rlse, cu, heads, d)
    dqkv = nans((N, 3 * h), dtype)
    mp.op_attention_bwd(_dt(dtype), tq, o, to_dev(dO, dtype), lse, N, heads, d, cu, dqkv, scratch)
    got = host(dqkv)
    for name, sl, ref in (("dq", slice(0, h), rdq), ("dk", slice(h, 2 * h), rdk),
                          ("dv", slice(2 * h, 3 * h), rdv)):
        err = max_rel(got[:, sl], ref)
        assert err < (2e-2 if dtype == "bf16" else 1e-5), (name, err)
