"""Pins of the oracle's SGD step (W-subproblem of eq. (3) and masked
retraining, Section 4).

  * the penalty term equals the derivative of rho/2 ||W - Z + U||_F^2 (central
    finite differences of that function in binary64);
  * with the quadratic loss f(W) = 1/2 ||W - T||^2 (gradient W - T) and step
    lr = 1/(1 + rho), one step lands on the closed-form minimiser of the
    W-subproblem, (T + rho (Z - U)) / (1 + rho);
  * the mask follows each sparsity set's group map, checked against numpy
    broadcasting of the group mask; pruned entries are exactly +0 and kept
    entries equal the unmasked step.
"""
import numpy as np
import pytest

import oracle
from oracle import CHANNEL, ELEMENT, FILTER, SHAPE

SHAPES = [(6, 4, 3, 3), (5, 3, 1, 1), (4, 7, 2, 3)]


def tensors(shape, seed):
    rng = np.random.default_rng(seed)
    f = lambda s=1.0: (rng.standard_normal(shape) * s).astype(np.float32)
    return f(), f(0.1), f(), f(0.5)  # W, Gf, Z, U


@pytest.mark.parametrize("shape", SHAPES)
def test_penalty_term_is_the_gradient_of_the_quadratic(shape):
    W, _, Z, U = tensors(shape, 1)
    rho = 0.37
    zero = np.zeros(shape, np.float32)
    # with Gf = 0 and lr = -1 the step returns W + t: t = rho ((W - Z) + U)
    t = oracle.sgd_step(W, zero, Z, U, None, FILTER, rho, -1.0).astype(np.float64) - W.astype(np.float64)
    f = lambda X: 0.5 * rho * np.sum((X - Z.astype(np.float64) + U.astype(np.float64)) ** 2)
    rng = np.random.default_rng(2)
    for idx in [tuple(rng.integers(0, s) for s in shape) for _ in range(20)]:
        h = 1e-3
        Xp = W.astype(np.float64).copy()
        Xm = Xp.copy()
        Xp[idx] += h
        Xm[idx] -= h
        fd = (f(Xp) - f(Xm)) / (2 * h)
        assert abs(fd - t[idx]) <= 1e-5 * max(1.0, abs(fd)), (idx, fd, t[idx])


@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("rho", [1.5e-3, 0.3, 4.0])
def test_quadratic_loss_step_is_the_closed_form_minimiser(shape, rho):
    W, _, Z, U = tensors(shape, 3)
    T = np.random.default_rng(4).standard_normal(shape).astype(np.float32)
    Gf = (W - T).astype(np.float32)
    Wn = oracle.sgd_step(W, Gf, Z, U, None, FILTER, rho, 1.0 / (1.0 + rho))
    ref = (T.astype(np.float64) + rho * (Z.astype(np.float64) - U.astype(np.float64))) / (1.0 + rho)
    err = np.abs(Wn - ref).max() / max(1.0, np.abs(ref).max())
    assert err < 1e-5, err


def group_mask_dense(mask, kind, shape):
    A, B, C, D = shape
    m = np.asarray(mask, bool)
    if kind == FILTER:
        return np.broadcast_to(m[:, None, None, None], shape)
    if kind == CHANNEL:
        return np.broadcast_to(m[None, :, None, None], shape)
    if kind == SHAPE:
        return np.broadcast_to(m.reshape(B, C, D)[None], shape)
    return m.reshape(shape)


@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("kind", [FILTER, CHANNEL, SHAPE, ELEMENT])
def test_mask_follows_the_group_map(shape, kind):
    W, Gf, Z, U = tensors(shape, 5)
    G = oracle.n_groups(shape, kind)
    mask = (np.random.default_rng(6).random(G) < 0.5).astype(np.uint8)
    free = oracle.sgd_step(W, Gf, Z, U, None, kind, 0.2, 0.05)
    masked = oracle.sgd_step(W, Gf, Z, U, mask, kind, 0.2, 0.05)
    keep = group_mask_dense(mask, kind, shape)
    assert np.array_equal(masked[keep].view(np.uint32), free[keep].view(np.uint32))
    assert np.all(masked[~keep].view(np.uint32) == 0)  # +0, not -0


def test_all_pruned_and_plain_step():
    W, Gf, Z, U = tensors((3, 2, 2, 2), 7)
    out = oracle.sgd_step(W, Gf, Z, U, np.zeros(3, np.uint8), FILTER, 0.5, 0.1)
    assert np.all(out.view(np.uint32) == 0)
    # without the ADMM term and with lr = 0 the weights are returned unchanged
    assert np.array_equal(oracle.sgd_step(W, Gf, None, None, None, FILTER, 0.5, 0.0), W)
