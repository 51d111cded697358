"""structadmm_project_noalloc (the projection for callers that cannot
allocate) against structadmm_project with a caller workspace: the same
layers give the same bits.  Two calls in a row, the second with smaller
layers, so that what the first call left in the library's scratch must not
leak into the second."""
import numpy as np
import pytest

import paper_1807_11091_amd as sa
from gpu_helpers import DEV, GpuLayer, run_project, to_dev, torch

pytestmark = pytest.mark.gpu


def _layers(seed, spec):
    rng = np.random.default_rng(seed)
    out = []
    for shape, kind, frac, groups, fused in spec:
        W = (0.05 * rng.standard_normal(shape)).astype(np.float32)
        U = (0.01 * rng.standard_normal(shape)).astype(np.float32)
        G = {sa.FILTER: shape[0], sa.CHANNEL: shape[1], sa.SHAPE: shape[1] * shape[2] * shape[3],
             sa.ELEMENT: int(np.prod(shape))}[kind]
        out.append((W, U, kind, max(1, int(frac * G)), groups, fused))
    return out


def _gpu(spec_layers):
    return [GpuLayer(W, U, kind, k, groups, rho=1.5e-3 if fused else 0.0, fused=fused)
            for W, U, kind, k, groups, fused in spec_layers]


def _host(layers):
    torch().cuda.synchronize()
    return [l.host() for l in layers]


def _same(a, b):
    assert a.keys() == b.keys()
    for key in a:
        assert np.array_equal(np.ascontiguousarray(a[key]).view(np.uint8),
                              np.ascontiguousarray(b[key]).view(np.uint8)), key


BIG = [((384, 256, 3, 3), sa.FILTER, 0.6, 1, True),     # long rows: per-chunk row partials
       ((256, 48, 5, 5), sa.SHAPE, 0.3, 2, True),       # column partials and column keep bytes
       ((96, 3, 11, 11), sa.CHANNEL, 0.5, 1, False),
       ((128, 64, 3, 3), sa.ELEMENT, 0.25, 1, True)]    # histograms and per-chunk counts
SMALL = [((64, 16, 3, 3), sa.ELEMENT, 0.5, 1, True),
         ((40, 24, 3, 3), sa.SHAPE, 0.4, 1, False),
         ((30, 20, 1, 1), sa.FILTER, 0.5, 2, True)]


def test_noalloc_equals_workspace_call_twice():
    for seed, spec in ((1, BIG), (2, SMALL)):
        host = _layers(seed, spec)
        ref_layers = _gpu(host)
        ref = run_project(ref_layers)
        got_layers = _gpu(host)
        sa.project_noalloc([l.layer for l in got_layers])
        got = _host(got_layers)
        for r, g in zip(ref, got):
            _same(r, g)


def test_noalloc_rejects_layers_beyond_its_scratch():
    # shape-wise over 8192 columns of 8192 filters: 256 bands of 8192 binary64
    # column partials alone fill the 16 MiB
    t = torch()
    W = t.empty((8192, 8192, 1, 1), dtype=t.float32, device=DEV)
    Z = t.empty_like(W)
    mask = t.empty(8192, dtype=t.uint8, device=DEV)
    kept = t.empty(16, dtype=t.int32, device=DEV)
    lay = sa.ProjectLayer(W, W, Z, mask, kept, sa.SHAPE, 16)
    assert sa.project_workspace([lay]) > sa.PROJECT_NOALLOC_BYTES
    with pytest.raises(sa.StructAdmmError, match="SA_E_WORKSPACE"):
        sa.project_noalloc([lay])
