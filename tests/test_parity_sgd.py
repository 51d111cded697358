"""GPU parity of structadmm_sgd_step (the W-subproblem's SGD step of eq. (3)
and masked retraining, Section 4) against the oracle on the same seeded
inputs.  Both sides take the same binary32 operations in the same order, so
the bar is bitwise equality, for every group map, with and without the mask
and the ADMM term, on sizes that are not multiples of 4 (scalar tail) and on
several layers in one call.
"""
import numpy as np
import pytest

import oracle
import paper_1807_11091_amd as sa
from gpu_helpers import bitwise_equal, n_groups, to_dev, torch

pytestmark = pytest.mark.gpu

CASES = [
    ((64, 64, 3, 3), sa.FILTER), ((96, 3, 11, 11), sa.SHAPE), ((48, 24, 5, 5), sa.CHANNEL),
    ((7, 5, 3, 1), sa.ELEMENT), ((33, 17, 1, 1), sa.FILTER), ((256, 192, 3, 3), sa.SHAPE),
]


def inputs(shape, seed):
    rng = np.random.default_rng(seed)
    f = lambda s=1.0: (rng.standard_normal(shape) * s).astype(np.float32)
    return f(0.05), f(1e-3), f(0.05), f(1e-2)  # W, Gf, Z, U


@pytest.mark.parametrize("shape,kind", CASES)
@pytest.mark.parametrize("with_mask", [False, True])
@pytest.mark.parametrize("with_admm", [False, True])
def test_sgd_step_matches_oracle(shape, kind, with_mask, with_admm):
    t = torch()
    W, Gf, Z, U = inputs(shape, sum(shape) + kind)
    mask = (np.random.default_rng(9).random(n_groups(shape, kind)) < 0.4).astype(np.uint8) if with_mask else None
    rho, lr = 1.5e-3, 0.01
    ref = oracle.sgd_step(W, Gf, Z if with_admm else None, U if with_admm else None, mask, kind, rho, lr)
    dW = to_dev(W)
    sa.sgd_step([(dW, to_dev(Gf), to_dev(Z) if with_admm else None, to_dev(U) if with_admm else None,
                  to_dev(mask) if with_mask else None, kind, rho, lr)])
    t.cuda.synchronize()
    assert bitwise_equal(dW.cpu().numpy(), ref)


def test_sgd_step_many_layers_one_call():
    """More layers than one kernel-argument table holds, mixed kinds."""
    t = torch()
    items, refs, devs = [], [], []
    for i in range(37):
        shape, kind = CASES[i % len(CASES)]
        shape = (max(1, shape[0] // 4), shape[1], shape[2], shape[3])
        W, Gf, Z, U = inputs(shape, 100 + i)
        mask = (np.random.default_rng(i).random(n_groups(shape, kind)) < 0.5).astype(np.uint8)
        refs.append(oracle.sgd_step(W, Gf, Z, U, mask, kind, 0.2, 0.05))
        dW = to_dev(W)
        devs.append(dW)
        items.append((dW, to_dev(Gf), to_dev(Z), to_dev(U), to_dev(mask), kind, 0.2, 0.05))
    sa.sgd_step(items)
    t.cuda.synchronize()
    for dW, ref in zip(devs, refs):
        assert bitwise_equal(dW.cpu().numpy(), ref)
