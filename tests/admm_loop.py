"""The ADMM outer loop of Section 4 on a synthetic quadratic loss, with the
oracle: f(W) = 1/2 ||W - T||_F^2 (gradient W - T), W-subproblem solved by one
SGD step of size 1/(1 + rho) (which lands on its closed-form minimiser),
Z-subproblem = the projection (fused with the dual update), rho increased by a
constant factor per iteration.  Shared by the oracle pins and the GPU parity
test; not a test module."""
from __future__ import annotations

import numpy as np

import oracle

RHO0 = 1.5e-3   # initial rho of Section 4
GROWTH = 1.5    # per-iteration factor


def target(shape, kind, k, seed, margin=10.0):
    """T ~ N(0, 1) with k random groups scaled by `margin` (a clear top k)."""
    rng = np.random.default_rng(seed)
    T = rng.standard_normal(shape).astype(np.float32)
    G = oracle.n_groups(shape, kind)
    sel = np.zeros(G, bool)
    sel[rng.permutation(G)[:k]] = True
    A, B, C, D = shape
    m = {oracle.FILTER: lambda: sel[:, None, None, None], oracle.CHANNEL: lambda: sel[None, :, None, None],
         oracle.SHAPE: lambda: sel.reshape(B, C, D)[None], oracle.ELEMENT: lambda: sel.reshape(shape)}[kind]()
    return np.where(m, T * np.float32(margin), T).astype(np.float32)


def oracle_loop(T, kind, k, iters):
    """Per iteration (W, Z, U, mask) after the Z-step, starting from W = Z = U = 0."""
    W = np.zeros_like(T)
    Z = np.zeros_like(T)
    U = np.zeros_like(T)
    rho = RHO0
    out = []
    for _ in range(iters):
        Gf = (W - T).astype(np.float32)
        W = oracle.sgd_step(W, Gf, Z, U, None, kind, rho, np.float32(1.0 / (1.0 + rho)))
        r = oracle.project(W, U, kind, k, rho=rho, fused=True)
        Z, U = r["Z"], r["U"]
        out.append((W.copy(), Z.copy(), U.copy(), r["mask"].copy()))
        rho *= GROWTH
    return out
