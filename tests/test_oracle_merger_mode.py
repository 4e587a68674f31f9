"""Pins of the oracle's merger-only trainability mode (trainable = 2).

Lemma 1 read over the encoder's own parts (patch embedding and blocks, then the
merger): with only the merger trainable it is the trainable source, so it
receives the gradient of the merged rows, reduces its own weight gradients and
sends nothing upstream; the frozen parts before it run no backward.  The merger's
gradients are pinned by autograd of the independent torch formulation (only the
merger's parameters require a gradient) and by central finite differences; the
frozen parts' entries must stay bitwise untouched."""
import numpy as np
import pytest
import torch

import oracle
import workload as W
from tests import torch_ref
from tests.test_oracle_pins import tiny_cfg, tiny_problem

MERGER = 2


def _merger_slice(cfg):
    """Flat element range of the merger's tensors (LayerNorm, fc1, fc2)."""
    off, lo = 0, None
    for name, shape, _ in W.param_table(cfg):
        if name.startswith("merger.") and lo is None:
            lo = off
        off += int(np.prod(shape))
    return slice(lo, off)


def _problem(T=1, layers=2, seed=3):
    cfg = tiny_cfg(layers=layers, T=T, patch=2)
    grid = [[1, 4, 4], [2, 2, 6], [1, 6, 2]]
    w, X, cu, grid, _ = tiny_problem(cfg, grid, seed=seed)
    R = np.random.default_rng(seed + 7).standard_normal((X.shape[0] // 4, cfg.llm_hidden))
    return cfg, w, X, cu, grid, R


@pytest.mark.parametrize("T", [1, 2])
def test_merger_only_vs_autograd(oracle_lib, T):
    cfg, w, X, cu, grid, R = _problem(T=T)
    ms = _merger_slice(cfg)
    frozen = torch.tensor(w[:ms.start])
    train = torch.tensor(w[ms], requires_grad=True)
    M = torch_ref.encoder(cfg, torch.cat([frozen, train]), cu, grid, patches=torch.tensor(X))
    M.backward(torch.tensor(R))
    sentinel = np.full(w.shape, -2.5)
    rc, Mo, dw, _ = oracle.encoder(cfg, w, X, cu, grid, MERGER, d_merged=R, d_w_init=sentinel)
    assert rc == 0
    np.testing.assert_allclose(Mo, M.detach().numpy(), rtol=1e-10, atol=1e-11)
    np.testing.assert_allclose(dw[ms] - sentinel[ms], train.grad.numpy(), rtol=1e-9, atol=1e-10)
    # the frozen patch embedding and blocks run no backward: bitwise untouched
    np.testing.assert_array_equal(dw[:ms.start], sentinel[:ms.start])


def test_merger_only_finite_differences(oracle_lib):
    cfg, w, X, cu, grid, R = _problem(layers=1, seed=5)
    ms = _merger_slice(cfg)
    rc, _, dw, _ = oracle.encoder(cfg, w, X, cu, grid, MERGER, d_merged=R)
    assert rc == 0
    loss = lambda ww: float((oracle.encoder(cfg, ww, X, cu, grid, False)[1] * R).sum())
    eps = 1e-6
    rng = np.random.default_rng(13)
    for _ in range(3):
        v = np.zeros_like(w)
        v[ms] = rng.standard_normal(ms.stop - ms.start)
        fd = (loss(w + eps * v) - loss(w - eps * v)) / (2 * eps)
        assert abs(fd - dw @ v) <= 1e-6 * max(1.0, abs(fd))
    # one coordinate of each merger tensor: LayerNorm gain and shift, fc1, fc2 and biases
    off = 0
    for name, shape, _ in W.param_table(cfg):
        n = int(np.prod(shape))
        if name.startswith("merger."):
            i = off + n // 2
            e = np.zeros_like(w)
            e[i] = 1
            fd = (loss(w + eps * e) - loss(w - eps * e)) / (2 * eps)
            assert abs(fd - dw[i]) <= 1e-6 * max(1.0, abs(fd)), name
        off += n


def test_merger_only_matches_full_backward_on_merger(oracle_lib):
    """The merger's gradients do not depend on whether the parts before it train."""
    cfg, w, X, cu, grid, R = _problem(seed=8)
    ms = _merger_slice(cfg)
    _, _, full, _ = oracle.encoder(cfg, w, X, cu, grid, True, d_merged=R)
    _, _, part, _ = oracle.encoder(cfg, w, X, cu, grid, MERGER, d_merged=R)
    np.testing.assert_array_equal(part[ms], full[ms])
    assert not part[:ms.start].any()
    assert full[:ms.start].any()


def test_forward_identical_in_every_mode(oracle_lib):
    # Corollary 1: the mode decides which backward work exists, never the forward
    cfg, w, X, cu, grid, R = _problem(T=2, seed=4)
    outs = [oracle.encoder(cfg, w, X, cu, grid, m, d_merged=None if m == 0 else R)[1]
            for m in (0, 1, MERGER)]
    np.testing.assert_array_equal(outs[0], outs[1])
    np.testing.assert_array_equal(outs[0], outs[2])


def test_merger_only_accumulates(oracle_lib):
    cfg, w, X, cu, grid, R = _problem(seed=6)
    _, _, g, _ = oracle.encoder(cfg, w, X, cu, grid, MERGER, d_merged=R)
    base = np.random.default_rng(5).standard_normal(w.shape)
    _, _, g2, _ = oracle.encoder(cfg, w, X, cu, grid, MERGER, d_merged=R, d_w_init=base)
    np.testing.assert_array_equal(g2, base + g)


def test_merger_only_sends_nothing_upstream(oracle_lib):
    cfg, w, X, cu, grid, R = _problem(seed=2)
    with pytest.raises(ValueError):
        oracle.encoder(cfg, w, X, cu, grid, MERGER, d_merged=R, want_d_patches=True)
    with pytest.raises(ValueError):
        oracle.encoder(cfg, w, X, cu, grid, 3, d_merged=R)
