"""Pins of the ADMM outer loop (Section 4) on a synthetic quadratic loss,
using the oracle's SGD step and projection:

  * every iterate's Z lies in the sparsity set (exactly k groups kept, the
    rest exactly zero), as the method guarantees;
  * with rho growing, W and Z meet: ||W - Z|| / ||Z|| < 1e-4 at the end;
  * when T has a clear top k (k groups scaled by 10), the structured loops end
    on the projection of T itself: the same kept groups, and Z within 1% of it.
"""
import numpy as np
import pytest

import oracle
from admm_loop import oracle_loop, target
from oracle import CHANNEL, ELEMENT, FILTER, SHAPE


@pytest.mark.parametrize("kind", [FILTER, CHANNEL, SHAPE, ELEMENT])
def test_loop_feasibility_and_limit(kind):
    shape = (16, 8, 3, 3)
    G = oracle.n_groups(shape, kind)
    k = G // 3
    T = target(shape, kind, k, seed=kind + 1)
    its = oracle_loop(T, kind, k, 40)
    A, B, C, D = shape
    for W, Z, U, mask in its:
        assert int(mask.sum()) == k
        nz = {FILTER: lambda: np.abs(Z).reshape(A, -1).sum(1), CHANNEL: lambda: np.abs(Z).sum((0, 2, 3)),
              SHAPE: lambda: np.abs(Z).sum(0).ravel(), ELEMENT: lambda: np.abs(Z).ravel()}[kind]()
        assert np.all(nz[mask == 0] == 0)
    W, Z, U, mask = its[-1]
    assert np.linalg.norm(W - Z) / np.linalg.norm(Z) < 1e-4
    if kind != ELEMENT:
        P = oracle.project(T, np.zeros_like(T), kind, k)
        assert np.array_equal(mask, P["mask"])
        assert np.linalg.norm(Z - P["Z"]) / np.linalg.norm(P["Z"]) < 1e-2
