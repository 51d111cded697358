"""Pins of the oracle's Z-update, dual update and regulariser gradient.

The oracle is checked against what the paper and the mathematics fix, never
against a retyping of its own loops:
  * brute force: the Euclidean projection onto each constraint set of
    Section 3 (at most k nonzero filters / channels / filter-shape vectors /
    elements) is found by enumerating every support in exact rational
    arithmetic, with groups built from the paper's slice notation;
  * invariants of a projection (exact count, order, Pythagoras, no feasible
    point closer, idempotence);
  * the gradient of the quadratic term of eq. (3) by automatic
    differentiation in float64;
  * closed forms at k = 0 and k = n_groups.
"""
import itertools
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
from oracle import CHANNEL, ELEMENT, FILTER, SHAPE

KINDS = (FILTER, CHANNEL, SHAPE, ELEMENT)


def groups_by_definition(shape, kind):
    """Flat element indices of every group, in group order, from the slice
    notation of Section 3: X[a,:,:,:], X[:,b,:,:], X[:,b,c,d], single entries."""
    A, B, C, D = shape
    idx = np.arange(A * B * C * D).reshape(shape)
    if kind == FILTER:
        return [idx[a].ravel() for a in range(A)]
    if kind == CHANNEL:
        return [idx[:, b].ravel() for b in range(B)]
    if kind == SHAPE:
        return [idx[:, b, c, d].ravel() for b in range(B) for c in range(C) for d in range(D)]
    return [np.array([e]) for e in range(A * B * C * D)]


def allowed_by_definition(shape, groups, in_ch_mask):
    A, B, C, D = shape
    ok = np.ones(shape, bool)
    if in_ch_mask is not None:
        Ag = A // groups
        for a in range(A):
            for b in range(B):
                ok[a, b] = bool(in_ch_mask[(a // Ag) * B + b])
    return ok.ravel()


def brute_force(V, kind, k, groups=1, in_ch_mask=None):
    """argmin over supports S (|S| = k) of ||V - V_S||^2 in exact rationals;
    among equal minima the lexicographically smallest sorted support."""
    shape = V.shape
    sq = [Fraction(float(x)) ** 2 for x in V.ravel()]
    allowed = allowed_by_definition(shape, groups, in_ch_mask)
    G = groups_by_definition(shape, kind)
    total = sum(sq[e] for e in range(len(sq)))
    best = None
    for S in itertools.combinations(range(len(G)), k):
        kept = sum(sq[e] for g in S for e in G[g] if allowed[e])
        dist = total - kept
        if best is None or dist < best[0]:
            best = (dist, S)
    dist, S = best
    Z = np.zeros(V.size, np.float32)
    for g in S:
        for e in G[g]:
            if allowed[e]:
                Z[e] = V.ravel()[e]
    return Z.reshape(shape), S, dist


def tiny_cases():
    rng = np.random.default_rng(20240)
    shapes = [(1, 1, 1, 1), (2, 1, 1, 1), (3, 2, 1, 1), (2, 2, 2, 1), (4, 3, 1, 1),
              (2, 3, 2, 1), (3, 1, 2, 2), (1, 4, 1, 3), (2, 2, 1, 3)]
    cases = []
    for shape in shapes:
        for style in ("normal", "ties"):
            if style == "normal":
                W = rng.standard_normal(shape).astype(np.float32)
                U = (0.1 * rng.standard_normal(shape)).astype(np.float32)
            else:  # few distinct magnitudes: many exact ties between groups
                W = (rng.integers(-2, 3, size=shape) * 0.5).astype(np.float32)
                U = np.zeros(shape, np.float32)
            cases.append((shape, style, W, U))
    return cases


@pytest.mark.parametrize("kind", KINDS)
def test_projection_equals_bruteforce(kind):
    checked = 0
    for shape, style, W, U in tiny_cases():
        G = oracle.n_groups(shape, kind)
        if G > 12:
            continue
        V = W + U  # one binary32 add, numpy's IEEE arithmetic
        for k in range(G + 1):
            res = oracle.project(W, U, kind, k)
            Zb, S, dist = brute_force(V, kind, k)
            assert np.array_equal(res["Z"].view(np.uint32), Zb.view(np.uint32)), (shape, style, k)
            assert list(res["kept_idx"]) == list(S), (shape, style, k)
            assert res["mask"].sum() == k
            checked += 1
    assert checked > 20


def test_projection_with_channel_support_equals_bruteforce():
    """Projection onto {<= k nonzero filters} intersected with a fixed
    input-channel support (the filter + channel chain)."""
    rng = np.random.default_rng(7)
    for shape, groups in [((4, 3, 1, 1), 1), ((4, 2, 1, 2), 2), ((6, 2, 1, 1), 2), ((3, 3, 2, 1), 1)]:
        A, B = shape[0], shape[1]
        for trial in range(4):
            W = rng.standard_normal(shape).astype(np.float32)
            if trial == 3:
                W[1] = W[0]  # a tie between two filters after masking
            U = (0.05 * rng.standard_normal(shape)).astype(np.float32)
            m = rng.integers(0, 2, size=groups * B).astype(np.uint8)
            m[0] = 1
            V = W + U
            for k in range(A + 1):
                res = oracle.project(W, U, FILTER, k, groups=groups, in_ch_mask=m)
                Zb, S, _ = brute_force(V, FILTER, k, groups=groups, in_ch_mask=m)
                assert np.array_equal(res["Z"].view(np.uint32), Zb.view(np.uint32))
                assert list(res["kept_idx"]) == list(S)


def test_tie_break_lowest_index():
    # three identical filters, keep 2: filters 0 and 1; keep 1: filter 0
    W = np.ones((3, 2, 1, 1), np.float32)
    U = np.zeros_like(W)
    assert list(oracle.project(W, U, FILTER, 2)["kept_idx"]) == [0, 1]
    assert list(oracle.project(W, U, FILTER, 1)["kept_idx"]) == [0]
    # a larger filter always wins over the tied ones
    W[2] *= 2
    assert list(oracle.project(W, U, FILTER, 2)["kept_idx"]) == [0, 2]
    # elements: |v| ties across signs
    W = np.array([-1, 1, -1, 0.5], np.float32).reshape(4, 1, 1, 1)
    assert list(oracle.project(W, np.zeros_like(W), ELEMENT, 2)["kept_idx"]) == [0, 1]


def independent_keys(V, kind):
    V64 = V.astype(np.float64)
    if kind == FILTER:
        return (V64 ** 2).sum(axis=(1, 2, 3))
    if kind == CHANNEL:
        return (V64 ** 2).sum(axis=(0, 2, 3))
    if kind == SHAPE:
        return (V64 ** 2).sum(axis=0).ravel()
    return np.abs(V64).ravel()


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("shape,groups", [((16, 8, 3, 3), 1), ((24, 6, 5, 5), 2), ((32, 16, 1, 1), 1),
                                          ((12, 3, 11, 11), 1)])
def test_projection_invariants(kind, shape, groups):
    rng = np.random.default_rng(hash((kind, shape)) % 2**32)
    W = (0.05 * rng.standard_normal(shape)).astype(np.float32)
    U = (0.01 * rng.standard_normal(shape)).astype(np.float32)
    V = W + U
    G = oracle.n_groups(shape, kind)
    rho = 1.5e-3
    for k in sorted({0, 1, G // 3, G // 2, G - 1, G}):
        res = oracle.project(W, U, kind, k, groups=groups, rho=rho, fused=True)
        Z, Un, Gr, mask = res["Z"], res["U"], res["G"], res["mask"]
        keys = independent_keys(V, kind)
        # exactly k kept, listed ascending
        assert int(mask.sum()) == k
        assert np.array_equal(np.flatnonzero(mask), res["kept_idx"])
        # every kept key >= every pruned key
        if 0 < k < G:
            assert keys[mask == 1].min() >= keys[mask == 0].max()
        # the returned scores are the group scores
        np.testing.assert_allclose(res["scores"], keys, rtol=1e-12, atol=0)
        # Z + U' == V bitwise (U' is exactly 0 on kept entries and v on pruned ones)
        assert np.array_equal((Z + Un).view(np.uint32), V.view(np.uint32))
        # Pythagoras: ||Z||^2 + ||V - Z||^2 == ||V||^2
        z2 = np.sum(Z.astype(np.float64) ** 2)
        r2 = np.sum((V.astype(np.float64) - Z) ** 2)
        v2 = np.sum(V.astype(np.float64) ** 2)
        assert abs(z2 + r2 - v2) <= 1e-12 * v2
        # feasible: at most k nonzero groups
        Gs = groups_by_definition(shape, kind)
        nz = sum(1 for g in Gs if np.any(Z.ravel()[g] != 0))
        assert nz <= k
        # no random feasible point of the set is closer
        for _ in range(20):
            S = rng.choice(G, size=k, replace=False)
            Zp = np.zeros(V.size)
            for g in S:
                Zp[Gs[g]] = V.ravel()[Gs[g]]
            assert np.sum((V.ravel().astype(np.float64) - Zp) ** 2) >= r2 * (1 - 1e-12)
        # idempotence: projecting Z again returns Z
        again = oracle.project(Z, np.zeros_like(Z), kind, k, groups=groups)
        assert np.array_equal(again["Z"].view(np.uint32), Z.view(np.uint32))
        if k == 0 or keys[mask == 1].min() > 0:
            assert np.array_equal(again["mask"], mask)


def test_gradient_is_derivative_of_quadratic_term():
    """G = d/dW [rho/2 ||W - Z + U||_F^2] (eq. 3), by float64 autograd."""
    rng = np.random.default_rng(3)
    shape = (8, 4, 3, 3)
    W = (0.1 * rng.standard_normal(shape)).astype(np.float32)
    U = (0.02 * rng.standard_normal(shape)).astype(np.float32)
    rho = 0.37
    for kind in KINDS:
        G = oracle.n_groups(shape, kind)
        res = oracle.project(W, U, kind, G // 2, rho=rho, fused=True)
        Wt = torch.tensor(W, dtype=torch.float64, requires_grad=True)
        Zt = torch.tensor(res["Z"], dtype=torch.float64)
        Ut = torch.tensor(res["U"], dtype=torch.float64)
        loss = rho / 2 * torch.sum((Wt - Zt + Ut) ** 2)
        loss.backward()
        ref = Wt.grad.numpy()
        err = np.linalg.norm(res["G"] - ref) / np.linalg.norm(ref)
        assert err < 1e-6, (kind, err)
        # standalone dual update + gradient gives the same bits as the fused step
        U2, G2 = oracle.dual_update(W, res["Z"], U, rho, update_dual=True)
        assert np.array_equal(U2.view(np.uint32), res["U"].view(np.uint32))
        assert np.array_equal(G2.view(np.uint32), res["G"].view(np.uint32))
        # gradient only (U untouched)
        U3, G3 = oracle.dual_update(W, res["Z"], U, rho, update_dual=False)
        assert np.array_equal(U3, U)
        Wt.grad = None
        loss = rho / 2 * torch.sum((Wt - Zt + torch.tensor(U, dtype=torch.float64)) ** 2)
        loss.backward()
        ref = Wt.grad.numpy()
        assert np.linalg.norm(G3 - ref) / np.linalg.norm(ref) < 1e-6


@pytest.mark.parametrize("kind", KINDS)
def test_closed_forms_at_k_extremes(kind):
    rng = np.random.default_rng(11)
    shape = (6, 4, 3, 3)
    W = (0.05 * rng.standard_normal(shape)).astype(np.float32)
    zero = np.zeros_like(W)
    rho = 1e-3
    G = oracle.n_groups(shape, kind)
    # keep everything, U = 0: Z = V = W, U' = 0, G = 0 exactly
    r = oracle.project(W, zero, kind, G, rho=rho, fused=True)
    assert np.array_equal(r["Z"], W) and not np.any(r["U"]) and not np.any(r["G"])
    # keep nothing: Z = 0, U' = V, G = rho * (W + V)
    U = (0.01 * rng.standard_normal(shape)).astype(np.float32)
    r = oracle.project(W, U, kind, 0, rho=rho, fused=True)
    V = W + U
    assert not np.any(r["Z"]) and np.array_equal(r["U"], V)
    np.testing.assert_allclose(r["G"], rho * (W.astype(np.float64) + V), rtol=1e-6, atol=1e-12)


def test_admm_loop_converges_on_quadratic_loss():
    """ADMM of Section 4 on f(W) = 1/2 ||W - T||^2 with T inside the filter set:
    W-step in closed form, Z = projection, dual update; with rho increasing the
    primal residual ||W - Z|| vanishes and Z recovers T's support."""
    rng = np.random.default_rng(5)
    shape = (12, 4, 3, 3)
    T = rng.standard_normal(shape).astype(np.float32)
    support = np.sort(rng.choice(12, size=5, replace=False))
    T[np.setdiff1d(np.arange(12), support)] = 0
    Tn = T + (0.3 * rng.standard_normal(shape)).astype(np.float32)  # target with off-support energy
    W = Tn.copy()
    U = np.zeros_like(W)
    Z = oracle.project(W, U, FILTER, 5)["Z"]
    rho = 1.5e-3
    for it in range(60):
        W = ((Tn + rho * (Z - U)) / (1 + rho)).astype(np.float32)
        r = oracle.project(W, U, FILTER, 5, rho=rho, fused=True)
        Z, U = r["Z"], r["U"]
        rho *= 1.3
    assert np.linalg.norm(W - Z) / np.linalg.norm(Z) < 1e-3
    assert list(r["kept_idx"]) == list(support)


def test_rejects_bad_arguments():
    W = np.zeros((4, 2, 1, 1), np.float32)
    with pytest.raises(ValueError):
        oracle.project(W, W, FILTER, 5)
    with pytest.raises(ValueError):
        oracle.project(W, W, FILTER, -1)
    with pytest.raises(ValueError):
        oracle.project(W, W, FILTER, 1, groups=3)
