"""GPU parity of structadmm_csr and structadmm_conv_sparse_fwd (the CONV of a
non-structured pruned layer as a sparse product) against the oracle.

Bar: row pointers, columns and bf16 values bit-exact; CONV output (bf16,
binary32 accumulation) within max|dY| / RMS(Y_ref) <= 2e-2 of the oracle's
binary64 CSR CONV over the same bf16 operands, and exactly zero where a row
has no entries.  Small cases span several pixel tiles and filter blocks with
ragged tails; the workload cases run the element-wise densities of the
[256,256,3,3] layer on 14x14 at full batch and compare sampled images.
"""
import numpy as np
import pytest

import oracle
import paper_1807_11091_amd as sa
from gpu_helpers import DEV, GpuLayer, bf16_bits_to_f64, maxabs_over_rms, run_project, to_dev, torch
from workloads import WORKLOADS, input_nchw, layer_tensors

pytestmark = pytest.mark.gpu

TOL = 2e-2


def project_element(W, U, k, groups=1):
    L = GpuLayer(W, U, sa.ELEMENT, k, groups)
    got = run_project([L])[0]
    ref = oracle.project(W, U, sa.ELEMENT, k, groups)
    assert np.array_equal(got["mask"], ref["mask"])
    return L, ref


def gpu_csr(L, k):
    t = torch()
    row_ptr, col, val = sa.csr(L.Z, L.kept, nnz=k)
    t.cuda.synchronize()
    return row_ptr.cpu().numpy(), col.cpu().numpy()[:k], val.cpu().numpy()[:k]


@pytest.mark.parametrize("shape,frac,seed", [
    ((7, 3, 3, 3), 0.3, 1), ((64, 16, 3, 3), 0.1, 2), ((5, 2, 5, 3), 0.6, 3), ((1, 1, 1, 1), 1.0, 4),
    ((33, 4, 2, 2), 0.02, 5), ((96, 3, 11, 11), 0.25, 6), ((16, 8, 1, 1), 0.0, 7), ((9, 4, 3, 3), 1.0, 8),
])
def test_csr_bitwise(shape, frac, seed):
    rng = np.random.default_rng(seed)
    W = rng.standard_normal(shape).astype(np.float32)
    U = (0.1 * rng.standard_normal(shape)).astype(np.float32)
    k = int(round(frac * W.size))
    L, ref = project_element(W, U, k)
    row_ptr, col, val = gpu_csr(L, k)
    r = oracle.csr(ref["Z"], ref["mask"])
    assert np.array_equal(row_ptr, r["row_ptr"])
    assert np.array_equal(col, r["col"])
    assert np.array_equal(val, r["val"])


def sparse_case(N, Cin, H, Wd, A, C, D, stride, pad, groups, frac, seed, empty_rows=0, images=None):
    rng = np.random.default_rng(seed)
    B = Cin // groups
    shape = (A, B, C, D)
    W = (0.05 * rng.standard_normal(shape)).astype(np.float32)
    U = (0.01 * rng.standard_normal(shape)).astype(np.float32)
    # the first empty_rows filters score 0 everywhere: with k below the other
    # weights' count they keep no entry
    W[:empty_rows] = 0
    U[:empty_rows] = 0
    k = int(round(frac * (A - empty_rows) * B * C * D))
    L, ref = project_element(W, U, k, groups)
    row_ptr, col, val = sa.csr(L.Z, L.kept, nnz=k)
    X = rng.standard_normal((N, Cin, H, Wd)).astype(np.float32)
    Xp = sa.pack_nhwc(to_dev(X))
    Y = sa.conv_sparse_fwd(Xp, row_ptr, col, val, shape, groups, stride, pad, k)
    torch().cuda.synchronize()
    imgs = list(range(N)) if images is None else images
    got = bf16_bits_to_f64(Y.cpu().numpy()[imgs])
    rc = oracle.csr(ref["Z"], ref["mask"])
    Yref = oracle.conv_csr(oracle.pack(X[imgs]), rc, shape, groups, stride, pad)
    assert got.shape == Yref.shape
    err = maxabs_over_rms(got, Yref) if np.any(Yref) else float(np.max(np.abs(got)))
    assert err <= TOL, err
    # rows without entries give exact zeros
    empty = np.flatnonzero(np.diff(rc["row_ptr"]) == 0)
    assert not np.any(got[..., empty])
    return got, Yref


@pytest.mark.parametrize("N,Cin,H,Wd,A,C,D,stride,pad,groups,frac,seed", [
    (2, 16, 9, 9, 24, 3, 3, 1, 1, 1, 0.3, 11),     # one filter block of 24 rows, ragged pixel tile
    (3, 32, 13, 13, 130, 3, 3, 1, 1, 1, 0.1, 12),  # three filter blocks, the last of 2 rows
    (2, 48, 11, 10, 40, 5, 3, 2, 2, 2, 0.25, 13),  # groups, stride 2, non-square kernel
    (1, 16, 23, 23, 8, 11, 11, 4, 0, 1, 0.05, 14), # large kernel, stride 4
    (4, 24, 7, 7, 72, 1, 1, 1, 0, 3, 0.5, 15),     # 1x1, three groups of 8 channels
    (2, 8, 6, 6, 9, 3, 3, 1, 1, 1, 1.0, 16),       # every weight kept
    (2, 8, 6, 6, 9, 3, 3, 1, 1, 1, 0.0, 17),       # none kept
    (1, 40, 15, 15, 70, 3, 3, 2, 1, 2, 0.2, 18),   # groups of 20 channels (not 8-aligned)
])
def test_conv_sparse_parity(N, Cin, H, Wd, A, C, D, stride, pad, groups, frac, seed):
    sparse_case(N, Cin, H, Wd, A, C, D, stride, pad, groups, frac, seed)


def test_conv_sparse_empty_rows():
    sparse_case(2, 16, 9, 9, 40, 3, 3, 1, 1, 1, 0.2, 21, empty_rows=11)


def test_conv_sparse_equals_dense_path():
    """The sparse CONV and the dense CONV (structadmm_conv_fwd over the
    uncompacted masked weights) agree to the same bar."""
    rng = np.random.default_rng(30)
    shape, N, H = (64, 32, 3, 3), 4, 12
    W = (0.05 * rng.standard_normal(shape)).astype(np.float32)
    U = np.zeros(shape, np.float32)
    k = W.size // 5
    L, ref = project_element(W, U, k)
    row_ptr, col, val = sa.csr(L.Z, L.kept, nnz=k)
    X = rng.standard_normal((N, 32, H, H)).astype(np.float32)
    Xp = sa.pack_nhwc(to_dev(X))
    Ys = sa.conv_sparse_fwd(Xp, row_ptr, col, val, shape, 1, 1, 1, k)
    Wc, _, cc, ct, sz = sa.compact(L.Z, 1)
    Yd = sa.conv_fwd(Xp, Wc, cc, ct, sz, 3, 3, 1, 1)
    torch().cuda.synchronize()
    a, b = bf16_bits_to_f64(Ys.cpu().numpy()), bf16_bits_to_f64(Yd.cpu().numpy())
    assert maxabs_over_rms(a, b) <= TOL


def test_conv_sparse_reuse_ws():
    """A call that reuses the padded entries of the previous call on another
    input gives the same result as a full call."""
    t = torch()
    rng = np.random.default_rng(50)
    shape = (48, 16, 3, 3)
    W = rng.standard_normal(shape).astype(np.float32)
    k = W.size // 8
    L, ref = project_element(W, np.zeros(shape, np.float32), k)
    rp, col, val = sa.csr(L.Z, L.kept, nnz=k)
    X1 = sa.pack_nhwc(to_dev(rng.standard_normal((2, 16, 11, 11)).astype(np.float32)))
    X2 = sa.pack_nhwc(to_dev(rng.standard_normal((2, 16, 11, 11)).astype(np.float32)))
    ws = t.empty(sa.conv_sparse_workspace(X1, shape, 1, 1, 1, k), dtype=t.uint8, device=DEV)
    sa.conv_sparse_fwd(X1, rp, col, val, shape, 1, 1, 1, k, ws=ws)
    Yr = sa.conv_sparse_fwd(X2, rp, col, val, shape, 1, 1, 1, k, ws=ws, reuse_ws=True)
    Yf = sa.conv_sparse_fwd(X2, rp, col, val, shape, 1, 1, 1, k)
    t.cuda.synchronize()
    assert np.array_equal(Yr.cpu().numpy(), Yf.cpu().numpy())


@pytest.mark.parametrize("batch", [1, 2])
def test_conv_sparse_small_grids(batch):
    """Batch-1 AlexNet conv3 and conv4 shapes at the sparsities of Table 4:
    the launch shapes with one filter row per wavefront."""
    sparse_case(batch, 256, 13, 13, 384, 3, 3, 1, 1, 1, 0.057, 60 + batch)
    sparse_case(batch, 384, 13, 13, 384, 3, 3, 1, 1, 2, 0.064, 70 + batch)


@pytest.mark.parametrize("N,Cin,A", [
    (80, 256, 384),  # 64 pixels per workgroup, 16 wavefronts of 8 rows
    (200, 32, 64),   # 64 pixels, 8 wavefronts of 8 rows
    (8, 256, 384),   # 64 pixels, 16 wavefronts of 1 row
])
def test_conv_sparse_launch_shapes(N, Cin, A):
    """13x13 3x3 layers sized so that each launch shape of the CONV is taken;
    first, middle and last image compared."""
    sparse_case(N, Cin, 13, 13, A, 3, 3, 1, 1, 1, 0.1, 80 + N, images=[0, N // 2, N - 1])


def test_conv_sparse_two_calls_share_scratch():
    """A second call with another pattern on the same scratch (the padded
    entry arrays are rebuilt on every call)."""
    t = torch()
    rng = np.random.default_rng(40)
    shape = (32, 16, 3, 3)
    X = rng.standard_normal((2, 16, 10, 10)).astype(np.float32)
    Xp = sa.pack_nhwc(to_dev(X))
    ws = t.empty(sa.conv_sparse_workspace(Xp, shape, 1, 1, 1, int(np.prod(shape))), dtype=t.uint8, device=DEV)
    for frac in (0.5, 0.05):
        W = rng.standard_normal(shape).astype(np.float32)
        k = int(frac * W.size)
        L, ref = project_element(W, np.zeros(shape, np.float32), k)
        rp, col, val = sa.csr(L.Z, L.kept, nnz=k)
        Y = sa.conv_sparse_fwd(Xp, rp, col, val, shape, 1, 1, 1, k, ws=ws)
        t.cuda.synchronize()
        Yref = oracle.conv_csr(oracle.pack(X), oracle.csr(ref["Z"], ref["mask"]), shape, 1, 1, 1)
        assert maxabs_over_rms(bf16_bits_to_f64(Y.cpu().numpy()), Yref) <= TOL


@pytest.mark.parametrize("pct", [10, 25, 50])
def test_conv_sparse_workload_sampled(pct):
    """[256,256,3,3] on 14x14 at batch 256, element-wise keep pct%: the
    benchmark's launch; three images compared with the oracle."""
    wl = WORKLOADS["resnet50_s3_sweep"]
    Lc = wl.layers[0]
    W, U = layer_tensors(wl, 0)
    k = wl.k_for(0, sa.ELEMENT, pct)
    L = GpuLayer(W, U, sa.ELEMENT, k, Lc.groups, scores=False)
    got = run_project([L])[0]
    rp, col, val = sa.csr(L.Z, L.kept, nnz=k)
    X = input_nchw(wl, 0)
    Xp = sa.pack_nhwc(to_dev(X))
    Y = sa.conv_sparse_fwd(Xp, rp, col, val, W.shape, Lc.groups, Lc.stride, Lc.pad, k)
    torch().cuda.synchronize()
    rc = oracle.csr(got["Z"], got["mask"])
    assert rc["row_ptr"][-1] == k
    assert np.array_equal(rp.cpu().numpy(), rc["row_ptr"])
    imgs = [0, wl.batch // 2 + 1, wl.batch - 1]
    Yref = oracle.conv_csr(oracle.pack(X[imgs]), rc, W.shape, Lc.groups, Lc.stride, Lc.pad)
    out = bf16_bits_to_f64(Y.cpu().numpy()[imgs])
    assert maxabs_over_rms(out, Yref) <= TOL
