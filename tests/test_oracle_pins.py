"""Pins for the CPU oracle: each test checks it against something other than
itself -- library routines (torch fp64), autograd, closed forms, invariants the
paper fixes, and brute force on tiny inputs.  No GPU needed."""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
import workload as W
from tests import torch_ref

torch.set_default_dtype(torch.float64)
RNG = np.random.default_rng(1234)


def tiny_cfg(layers=1, hidden=16, heads=2, mlp=32, llm=24, T=1, patch=2, chans=3):
    return W.EncoderConfig(hidden=hidden, layers=layers, heads=heads, mlp=mlp, llm_hidden=llm,
                           temporal_patch=T, patch=patch, in_chans=chans, dtype="f32")


def tiny_problem(cfg, grid, seed=0, std=0.3):
    """Weights with larger spread than the production draw so every term matters."""
    rng = np.random.default_rng(seed)
    grid = np.asarray(grid, np.int32).reshape(-1, 3)
    n = (grid[:, 0] * grid[:, 1] * grid[:, 2]).astype(np.int64)
    cu = np.concatenate([[0], np.cumsum(n)]).astype(np.int32)
    w = []
    for name, shape, kind in W.param_table(cfg):
        v = rng.standard_normal(int(np.prod(shape))) * std
        if kind == "g":
            v += 1.0
        w.append(v)
    w = np.concatenate(w)
    images = [rng.uniform(-1, 1, (cfg.in_chans, int(t) * cfg.temporal_patch, int(gh) * cfg.patch,
                                  int(gw) * cfg.patch)) for t, gh, gw in grid]
    X = np.concatenate([W.patchify(im, cfg.patch, cfg.temporal_patch) for im in images], 0)
    return w, X, cu, grid, images


# ---------------------------------------------------------------------------
# parameter table / closed-form sizes
# ---------------------------------------------------------------------------

def test_param_table_matches_generator(oracle_lib):
    for name in ("c1_tiny_fp32", "c2_vitl_frozen", "c4_qwen2vl_trained"):
        cfg = W.CONFIGS[name].cfg
        ot = oracle.param_table(cfg)
        gt = W.param_table(cfg)
        assert len(ot) == len(gt)
        off = 0
        for (on, oo, orow, ocol), (gn, gs, _) in zip(ot, gt):
            assert on == gn and oo == off
            assert orow * ocol == int(np.prod(gs)) and orow == gs[0]
            off += int(np.prod(gs))


def test_param_count_closed_form(oracle_lib):
    # ~675M for the Qwen2-VL-ViT shape: 2x2 merger = LN -> Linear(4h,4h)+GELU -> Linear(4h,H)
    q = W.CONFIGS["c4_qwen2vl_trained"].cfg
    h, m, H, L = 1280, 5120, 3584, 32
    closed = (1176 * h + h + L * (h * 3 * h + 3 * h + h * h + h + h * m + m + m * h + h + 4 * h)
              + 2 * h + (16 * h * h + 4 * h) + (4 * h * H + H))
    assert oracle.param_count(q) == closed == 675_760_384
    assert abs(closed / 1e6 - 675) < 1.0
    assert oracle.param_count(W.CONFIGS["c2_vitl_frozen"].cfg) == 336_477_184


# ---------------------------------------------------------------------------
# building blocks vs library routines
# ---------------------------------------------------------------------------

def test_linear_vs_matmul(oracle_lib):
    X, Wt, b = RNG.standard_normal((37, 19)), RNG.standard_normal((23, 19)), RNG.standard_normal(23)
    Y = oracle.linear(X, Wt, b)
    ref = (torch.tensor(X) @ torch.tensor(Wt).T + torch.tensor(b)).numpy()
    np.testing.assert_allclose(Y, ref, rtol=1e-13, atol=1e-13)


def test_linear_bwd_vs_autograd(oracle_lib):
    X, Wt = RNG.standard_normal((29, 11)), RNG.standard_normal((13, 11))
    b, dY = RNG.standard_normal(13), RNG.standard_normal((29, 13))
    tX, tW, tb = (torch.tensor(a, requires_grad=True) for a in (X, Wt, b))
    (tX @ tW.T + tb).backward(torch.tensor(dY))
    dX, dW, db = oracle.linear_bwd(dY, X, Wt)
    np.testing.assert_allclose(dX, tX.grad.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dW, tW.grad.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(db, tb.grad.numpy(), rtol=1e-12, atol=1e-12)


def test_layernorm_vs_torch(oracle_lib):
    X = RNG.standard_normal((17, 40)) * 3 + 1.5
    g, b = 1 + RNG.standard_normal(40) * 0.1, RNG.standard_normal(40) * 0.1
    Y, mu, rs = oracle.layernorm(X, g, b, 1e-6)
    ref = F.layer_norm(torch.tensor(X), (40,), torch.tensor(g), torch.tensor(b), 1e-6).numpy()
    np.testing.assert_allclose(Y, ref, rtol=1e-12, atol=1e-12)
    # with unit gain and zero shift every row has mean 0 and (biased) variance 1
    Y1, _, _ = oracle.layernorm(X, np.ones(40), np.zeros(40), 0.0)
    np.testing.assert_allclose(Y1.mean(1), 0, atol=1e-13)
    np.testing.assert_allclose((Y1 ** 2).mean(1), 1, atol=1e-12)


def test_layernorm_bwd_vs_autograd(oracle_lib):
    X = RNG.standard_normal((9, 24)) * 2
    g, b, dY = 1 + RNG.standard_normal(24) * 0.2, RNG.standard_normal(24), RNG.standard_normal((9, 24))
    tX, tg, tb = (torch.tensor(a, requires_grad=True) for a in (X, g, b))
    F.layer_norm(tX, (24,), tg, tb, 1e-6).backward(torch.tensor(dY))
    _, mu, rs = oracle.layernorm(X, g, b, 1e-6)
    dX, dg, db = oracle.layernorm_bwd(dY, X, g, mu, rs)
    np.testing.assert_allclose(dX, tX.grad.numpy(), rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(dg, tg.grad.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(db, tb.grad.numpy(), rtol=1e-12, atol=1e-12)


def test_gelu_vs_torch_erf_form(oracle_lib):
    u = np.concatenate([RNG.standard_normal(200) * 3, [0.0, -8.0, 8.0]])
    np.testing.assert_allclose(oracle.gelu(u), F.gelu(torch.tensor(u)).numpy(), rtol=1e-14,
                               atol=1e-15)
    tu = torch.tensor(u, requires_grad=True)
    F.gelu(tu).sum().backward()
    np.testing.assert_allclose(oracle.gelu_grad(u), tu.grad.numpy(), rtol=1e-13, atol=1e-14)
    # special values: GELU(0) = 0, GELU'(0) = 1/2; tanh form differs by ~1e-3 at u = 1
    assert oracle.gelu(np.array([0.0]))[0] == 0.0
    assert abs(oracle.gelu_grad(np.array([0.0]))[0] - 0.5) < 1e-15
    assert abs(oracle.gelu(np.array([1.0]))[0] - 0.5 * (1 + math.erf(1 / math.sqrt(2)))) < 1e-15


def _rope_inputs(N=23, heads=3, d=8):
    x = RNG.standard_normal((N, heads * d))
    py, px = RNG.integers(0, 50, N).astype(np.int32), RNG.integers(0, 50, N).astype(np.int32)
    return x, py, px, heads, d


def test_rope_complex_closed_form(oracle_lib):
    x, py, px, heads, d = _rope_inputs()
    got = oracle.rope2d(x, heads, d, py, px)
    ref = torch_ref.rope_complex(torch.tensor(x), heads, d, py, px, 10000.0).numpy()
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


def test_rope_identity_norm_inverse_translation(oracle_lib):
    x, py, px, heads, d = _rope_inputs()
    z = np.zeros_like(py)
    np.testing.assert_array_equal(oracle.rope2d(x, heads, d, z, z), x)     # identity at (0, 0)
    r = oracle.rope2d(x, heads, d, py, px)
    n0 = np.linalg.norm(x.reshape(-1, heads, d), axis=2)
    np.testing.assert_allclose(np.linalg.norm(r.reshape(-1, heads, d), axis=2), n0, rtol=1e-13)
    back = oracle.rope2d(r, heads, d, py, px, inverse=True)
    np.testing.assert_allclose(back, x, rtol=1e-12, atol=1e-12)
    # scores depend only on relative position: translate every (y, x) by a constant
    q, k = RNG.standard_normal((5, d)), RNG.standard_normal((5, d))
    p1y, p1x = RNG.integers(0, 30, 5).astype(np.int32), RNG.integers(0, 30, 5).astype(np.int32)
    s1 = oracle.rope2d(q, 1, d, p1y, p1x) @ oracle.rope2d(k, 1, d, p1y, p1x).T
    s2 = oracle.rope2d(q, 1, d, p1y + 7, p1x + 3) @ oracle.rope2d(k, 1, d, p1y + 7, p1x + 3).T
    np.testing.assert_allclose(s1, s2, rtol=1e-10, atol=1e-10)


def test_attention_single_segment_vs_sdpa(oracle_lib):
    heads, d, N = 3, 8, 29
    q, k, v = (RNG.standard_normal((N, heads * d)) * 2 for _ in range(3))
    o, lse = oracle.attention(q, k, v, [0, N], heads, d)
    tq, tk, tv = (torch.tensor(a).view(N, heads, d).transpose(0, 1)[None] for a in (q, k, v))
    ref = F.scaled_dot_product_attention(tq, tk, tv)[0].transpose(0, 1).reshape(N, -1).numpy()
    np.testing.assert_allclose(o, ref, rtol=1e-12, atol=1e-12)
    s = torch.einsum("hqd,hkd->hqk", tq[0], tk[0]) / math.sqrt(d)
    np.testing.assert_allclose(lse, torch.logsumexp(s, -1).T.numpy(), rtol=1e-12, atol=1e-12)


def test_attention_packed_equals_each_alone(oracle_lib):
    heads, d = 2, 8
    lens = [5, 1, 12, 7]
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    N = cu[-1]
    q, k, v = (RNG.standard_normal((N, heads * d)) for _ in range(3))
    o, lse = oracle.attention(q, k, v, cu, heads, d)
    for s in range(len(lens)):
        sl = slice(cu[s], cu[s + 1])
        o1, l1 = oracle.attention(q[sl], k[sl], v[sl], [0, lens[s]], heads, d)
        np.testing.assert_array_equal(o[sl], o1)
        np.testing.assert_array_equal(lse[sl], l1)


def test_attention_bwd_vs_autograd(oracle_lib):
    heads, d = 2, 8
    lens = [6, 9]
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    N = cu[-1]
    q, k, v, dO = (RNG.standard_normal((N, heads * d)) for _ in range(4))
    tq, tk, tv = (torch.tensor(a, requires_grad=True) for a in (q, k, v))
    outs = []
    for s in range(len(lens)):
        sl = slice(int(cu[s]), int(cu[s + 1]))
        f = lambda t: t[sl].view(-1, heads, d).transpose(0, 1)[None]
        outs.append(F.scaled_dot_product_attention(f(tq), f(tk), f(tv))[0].transpose(0, 1)
                    .reshape(-1, heads * d))
    torch.cat(outs).backward(torch.tensor(dO))
    o, lse = oracle.attention(q, k, v, cu, heads, d)
    dq, dk, dv = oracle.attention_bwd(q, k, v, o, dO, lse, cu, heads, d)
    for got, t in ((dq, tq), (dk, tk), (dv, tv)):
        np.testing.assert_allclose(got, t.grad.numpy(), rtol=1e-11, atol=1e-11)


# ---------------------------------------------------------------------------
# layout pins: positions and patch embedding
# ---------------------------------------------------------------------------

def test_positions_vs_coordinate_image(oracle_lib):
    cfg = tiny_cfg(T=2)
    grid = np.array([[1, 4, 6], [3, 2, 2], [2, 6, 4]], np.int32)
    py, px = oracle.positions(grid)
    tau, y, x = torch_ref.coordinate_positions(cfg, grid)
    np.testing.assert_array_equal(py, y)
    np.testing.assert_array_equal(px, x)
    # every 2x2 window is four consecutive rows, ordered (0,0),(0,1),(1,0),(1,1)
    assert np.all(py[0::4] % 2 == 0) and np.all(px[0::4] % 2 == 0)
    np.testing.assert_array_equal(py[1::4], py[0::4])
    np.testing.assert_array_equal(px[1::4], px[0::4] + 1)
    np.testing.assert_array_equal(py[2::4], py[0::4] + 1)
    np.testing.assert_array_equal(px[3::4], px[0::4] + 1)


def test_patch_embed_equals_conv3d(oracle_lib):
    for T in (1, 2):
        cfg = tiny_cfg(T=T, patch=3)
        grid = [[2, 4, 2], [1, 2, 6]]
        w, X, cu, grid, images = tiny_problem(cfg, grid)
        p = torch_ref.split_params(cfg, torch.tensor(w))
        ref = torch_ref.patch_embed_conv(cfg, images, p["pe.w"], p["pe.b"], grid).numpy()
        got = oracle.linear(X, p["pe.w"].numpy(), p["pe.b"].numpy())
        np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


# ---------------------------------------------------------------------------
# whole encoder vs the torch formulation (forward and autograd backward)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("T", [1, 2])
def test_encoder_vs_torch_autograd(oracle_lib, T):
    cfg = tiny_cfg(layers=2, T=T, patch=2)
    grid = [[1, 4, 4], [2, 2, 6], [1, 6, 2]]
    w, X, cu, grid, images = tiny_problem(cfg, grid, seed=3)
    tw = torch.tensor(w, requires_grad=True)
    tX = torch.tensor(X, requires_grad=True)
    M = torch_ref.encoder(cfg, tw, cu, grid, patches=tX)
    # the conv route on raw pixels gives the same output
    Mc = torch_ref.encoder(cfg, torch.tensor(w), cu, grid, images=images)
    np.testing.assert_allclose(M.detach().numpy(), Mc.numpy(), rtol=1e-11, atol=1e-11)
    R = np.random.default_rng(9).standard_normal(M.shape)
    M.backward(torch.tensor(R))
    rc, Mo, dw, dx = oracle.encoder(cfg, w, X, cu, grid, True, d_merged=R, want_d_patches=True)
    assert rc == 0
    np.testing.assert_allclose(Mo, M.detach().numpy(), rtol=1e-10, atol=1e-11)
    np.testing.assert_allclose(dw, tw.grad.numpy(), rtol=1e-9, atol=1e-10)
    np.testing.assert_allclose(dx, tX.grad.numpy(), rtol=1e-9, atol=1e-10)


def test_encoder_finite_differences(oracle_lib):
    cfg = tiny_cfg(layers=1)
    w, X, cu, grid, _ = tiny_problem(cfg, [[1, 4, 4], [1, 4, 6]], seed=5)
    R = np.random.default_rng(11).standard_normal((10, cfg.llm_hidden))
    rc, M, dw, dx = oracle.encoder(cfg, w, X, cu, grid, True, d_merged=R, want_d_patches=True)
    loss = lambda ww, xx: float((oracle.encoder(cfg, ww, xx, cu, grid, False)[1] * R).sum())
    rng = np.random.default_rng(12)
    eps = 1e-6
    for _ in range(3):
        v = rng.standard_normal(w.shape)
        fd = (loss(w + eps * v, X) - loss(w - eps * v, X)) / (2 * eps)
        assert abs(fd - dw @ v) <= 1e-6 * max(1.0, abs(fd))
        u = rng.standard_normal(X.shape)
        fd = (loss(w, X + eps * u) - loss(w, X - eps * u)) / (2 * eps)
        assert abs(fd - (dx * u).sum()) <= 1e-6 * max(1.0, abs(fd))
    # single coordinates in each kind of tensor (a dropped term shows up here)
    for name, (off, n) in _some_offsets(cfg).items():
        i = off + n // 2
        e = np.zeros_like(w)
        e[i] = 1
        fd = (loss(w + eps * e, X) - loss(w - eps * e, X)) / (2 * eps)
        assert abs(fd - dw[i]) <= 1e-6 * max(1.0, abs(fd)), name


def _some_offsets(cfg):
    out, off = {}, 0
    for name, shape, _ in W.param_table(cfg):
        n = int(np.prod(shape))
        out[name] = (off, n)
        off += n
    return out


# ---------------------------------------------------------------------------
# invariants the paper and the spec fix
# ---------------------------------------------------------------------------

def _c1_like():
    cfg = tiny_cfg(layers=2, hidden=16, heads=2, T=2, patch=2)
    grid = [[1, 4, 4], [2, 2, 4], [1, 6, 2], [1, 2, 2]]
    return (cfg,) + tiny_problem(cfg, grid, seed=21, std=0.2)


def test_packed_equals_each_item_alone(oracle_lib):
    cfg, w, X, cu, grid, _ = _c1_like()
    _, M, _, _ = oracle.encoder(cfg, w, X, cu, grid, False)
    mrow = 0
    for i in range(len(grid)):
        sl = slice(int(cu[i]), int(cu[i + 1]))
        n = int(cu[i + 1] - cu[i])
        _, Mi, _, _ = oracle.encoder(cfg, w, X[sl], [0, n], grid[i:i + 1], False)
        np.testing.assert_array_equal(M[mrow:mrow + n // 4], Mi)
        mrow += n // 4


def test_permutation_equivariance(oracle_lib):
    cfg, w, X, cu, grid, _ = _c1_like()
    _, M, _, _ = oracle.encoder(cfg, w, X, cu, grid, False)
    perm = [2, 0, 3, 1]
    Xp = np.concatenate([X[cu[i]:cu[i + 1]] for i in perm])
    gp = grid[perm]
    n = gp[:, 0] * gp[:, 1] * gp[:, 2]
    cup = np.concatenate([[0], np.cumsum(n)]).astype(np.int32)
    _, Mp, _, _ = oracle.encoder(cfg, w, Xp, cup, gp, False)
    mo = np.concatenate([[0], np.cumsum((grid[:, 0] * grid[:, 1] * grid[:, 2]) // 4)])
    expect = np.concatenate([M[mo[i]:mo[i + 1]] for i in perm])
    np.testing.assert_array_equal(Mp, expect)
    # moving the placeholder indices along leaves the LLM buffer bitwise unchanged
    idx = np.random.default_rng(0).permutation(200)[:M.shape[0]]
    idxp = np.concatenate([idx[mo[i]:mo[i + 1]] for i in perm])
    emb = np.zeros((200, M.shape[1]))
    np.testing.assert_array_equal(oracle.merge_scatter(M, idx, emb),
                                  oracle.merge_scatter(Mp, idxp, emb))


def test_frozen_and_trained_forward_identical(oracle_lib):
    # Corollary 1: the footprint changes which backward events fire, never the forward
    cfg, w, X, cu, grid, _ = _c1_like()
    R = np.random.default_rng(2).standard_normal(((X.shape[0]) // 4, cfg.llm_hidden))
    _, Mf, _, _ = oracle.encoder(cfg, w, X, cu, grid, False)
    _, Mt, _, _ = oracle.encoder(cfg, w, X, cu, grid, True, d_merged=R)
    np.testing.assert_array_equal(Mf, Mt)


def test_frozen_has_no_weight_gradients(oracle_lib):
    # Lemma 1 (iii): a frozen region reduces no weight gradients
    cfg, w, X, cu, grid, _ = _c1_like()
    R = np.ones(((X.shape[0]) // 4, cfg.llm_hidden))
    sentinel = np.full(w.shape, 7.25)
    rc, _, dw, dx = oracle.encoder(cfg, w, X, cu, grid, False, d_merged=R, want_d_patches=True,
                                   d_w_init=sentinel)
    assert rc == oracle.NOOP_FROZEN
    np.testing.assert_array_equal(dw, sentinel)
    assert not dx.any()


def test_weight_gradients_accumulate(oracle_lib):
    cfg, w, X, cu, grid, _ = _c1_like()
    R = np.random.default_rng(4).standard_normal(((X.shape[0]) // 4, cfg.llm_hidden))
    _, _, g, _ = oracle.encoder(cfg, w, X, cu, grid, True, d_merged=R)
    base = np.random.default_rng(5).standard_normal(w.shape)
    _, _, g2, _ = oracle.encoder(cfg, w, X, cu, grid, True, d_merged=R, d_w_init=base)
    np.testing.assert_array_equal(g2, base + g)


def test_transpose_relocation_is_loss_preserving(oracle_lib):
    """One-GPU emulation of the ByMicrobatch owner + seam gather: encoding owner
    groups separately and scattering them gives the same LLM input, and the
    per-group weight gradients sum to the all-at-once gradient."""
    cfg, w, X, cu, grid, _ = _c1_like()
    n_m = (X.shape[0]) // 4
    idx = np.random.default_rng(8).permutation(300)[:n_m]
    emb0 = np.random.default_rng(9).standard_normal((300, cfg.llm_hidden))
    demb = np.random.default_rng(10).standard_normal((300, cfg.llm_hidden))
    _, M, g_all, _ = oracle.encoder(cfg, w, X, cu, grid, True, d_merged=oracle.merge_gather(demb, idx))
    emb_all = oracle.merge_scatter(M, idx, emb0)
    groups = [[0, 2], [1, 3]]
    per_item_m = (grid[:, 0] * grid[:, 1] * grid[:, 2]) // 4
    mo = np.concatenate([[0], np.cumsum(per_item_m)])
    emb = emb0.copy()
    g_sum = np.zeros_like(w)
    for grp in groups:
        Xg = np.concatenate([X[cu[i]:cu[i + 1]] for i in grp])
        gg = grid[grp]
        cug = np.concatenate([[0], np.cumsum(gg[:, 0] * gg[:, 1] * gg[:, 2])]).astype(np.int32)
        ig = np.concatenate([idx[mo[i]:mo[i + 1]] for i in grp])
        _, Mg, gw_, _ = oracle.encoder(cfg, w, Xg, cug, gg, True,
                                       d_merged=oracle.merge_gather(demb, ig))
        emb = oracle.merge_scatter(Mg, ig, emb)
        g_sum += gw_
    np.testing.assert_array_equal(emb, emb_all)
    np.testing.assert_allclose(g_sum, g_all, rtol=1e-12, atol=1e-12)


def test_metadata_validation(oracle_lib):
    cfg, w, X, cu, grid, _ = _c1_like()
    bad = [
        (np.array([0, 5, cu[-1]], np.int32), grid),             # segment crosses an item
        (cu[:-1], grid),                                         # does not reach N
        (cu, np.array([[1, 3, 4]] + grid[1:].tolist(), np.int32)),  # odd height
    ]
    for c, g in bad:
        with pytest.raises(ValueError):
            oracle.encoder(cfg, w, X, c, g, False)
    # per-temporal-slice segments are accepted and match attention within slices
    g2 = np.array([[2, 2, 4]], np.int32)
    X2 = X[:16]
    rc, _, _, _ = oracle.encoder(cfg, w, X2, np.array([0, 8, 16], np.int32), g2, False)
    assert rc == 0
    with pytest.raises(ValueError):
        oracle.encoder(cfg, w, X2, np.array([0, 4, 16], np.int32), g2, False)
    # empty micro-batch (pure text) is a valid no-op
    rc, M, _, _ = oracle.encoder(cfg, w, X[:0], np.array([0], np.int32),
                                 np.zeros((0, 3), np.int32), False)
    assert rc == 0 and M.shape == (0, cfg.llm_hidden)


# ---------------------------------------------------------------------------
# scatter / gather
# ---------------------------------------------------------------------------

def test_scatter_gather_adjoint_exact(oracle_lib):
    rng = np.random.default_rng(3)
    n_rows, n_m, H = 97, 40, 8
    idx = rng.permutation(n_rows)[:n_m]
    x = rng.integers(-50, 50, (n_m, H)).astype(np.float64)
    y = rng.integers(-50, 50, (n_rows, H)).astype(np.float64)
    sx = oracle.merge_scatter(x, idx, np.zeros((n_rows, H)))
    assert (sx * y).sum() == (x * oracle.merge_gather(y, idx)).sum()


def test_scatter_copies_bits_and_rejects_bad_indices(oracle_lib):
    rng = np.random.default_rng(4)
    bits = rng.integers(0, 2 ** 16, (10, 6), dtype=np.uint16)    # includes NaN patterns
    emb = rng.integers(0, 2 ** 16, (30, 6), dtype=np.uint16)
    idx = rng.permutation(30)[:10]
    out = oracle.merge_scatter(bits, idx, emb)
    np.testing.assert_array_equal(out[idx], bits)
    keep = np.setdiff1d(np.arange(30), idx)
    np.testing.assert_array_equal(out[keep], emb[keep])
    np.testing.assert_array_equal(oracle.merge_gather(out, idx), bits)
    for bad in (np.array([0, 1, 1]), np.array([0, 30, 2]), np.array([-1, 2, 3])):
        with pytest.raises(ValueError):
            oracle.merge_scatter(bits[:3], bad, emb)
