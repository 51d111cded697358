"""Pins of the oracle's CSR form of a non-structured pruned layer and of its
CONV as a sparse product (Section 3, non-structured sparsity; Section 5 runs
that CONV with a CSR sparse library).

  * the CSR pattern equals scipy.sparse's canonical CSR of the kept entries
    (a library routine), and the values equal torch's float32 -> bfloat16
    conversion of Z there; kept zeros stay explicit entries;
  * empty and full masks give the obvious row pointers and columns;
  * the CSR of an element-wise projection lists exactly its kept_idx;
  * the CSR CONV equals torch.nn.functional.conv2d in float64 on the same
    bf16-rounded operands (grouped, strided, padded, non-square kernels);
  * the CSR CONV equals, bit for bit in float64, the oracle's CONV over the
    dense (uncompacted) matrix of the masked weights: skipping pruned entries
    drops only products that are exactly zero.
"""
import numpy as np
import pytest
import scipy.sparse
import torch
import torch.nn.functional as F

import oracle
from oracle import ELEMENT


def torch_bf16_bits(x):
    t = torch.from_numpy(np.ascontiguousarray(x, np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


@pytest.mark.parametrize("shape,density,seed", [
    ((7, 3, 3, 3), 0.3, 1), ((16, 8, 1, 1), 0.1, 2), ((5, 2, 5, 3), 0.6, 3), ((1, 1, 1, 1), 1.0, 4),
    ((33, 4, 2, 2), 0.02, 5),
])
def test_csr_matches_scipy(shape, density, seed):
    rng = np.random.default_rng(seed)
    Z = rng.standard_normal(shape).astype(np.float32)
    mask = (rng.random(shape) < density).astype(np.uint8)
    Z[mask == 0] = 0.0
    # a kept weight that is exactly zero stays an entry
    kept = np.flatnonzero(mask)
    if kept.size:
        Z.reshape(-1)[kept[0]] = 0.0
    r = oracle.csr(Z, mask)
    A = shape[0]
    K = int(np.prod(shape[1:]))
    rows, cols = np.nonzero(mask.reshape(A, K))
    ref = scipy.sparse.csr_matrix((np.ones(rows.size), (rows, cols)), shape=(A, K))
    ref.sort_indices()
    assert np.array_equal(r["row_ptr"], ref.indptr)
    assert np.array_equal(r["col"], ref.indices)
    assert np.array_equal(r["val"], torch_bf16_bits(Z.reshape(A, K)[rows, cols]))
    assert r["row_ptr"][-1] == mask.sum()


def test_csr_empty_and_full():
    Z = np.arange(24, dtype=np.float32).reshape(4, 2, 3, 1) - 11.5
    r = oracle.csr(Z, np.zeros(Z.shape, np.uint8))
    assert np.array_equal(r["row_ptr"], np.zeros(5, np.int32)) and r["col"].size == 0
    r = oracle.csr(Z, np.ones(Z.shape, np.uint8))
    assert np.array_equal(r["row_ptr"], np.arange(5) * 6)
    assert np.array_equal(r["col"], np.tile(np.arange(6), 4))
    assert np.array_equal(r["val"], torch_bf16_bits(Z.reshape(-1)))


def test_csr_of_element_projection_lists_kept_idx():
    rng = np.random.default_rng(9)
    shape = (12, 5, 3, 3)
    W = rng.standard_normal(shape).astype(np.float32)
    U = (0.1 * rng.standard_normal(shape)).astype(np.float32)
    k = W.size // 7
    p = oracle.project(W, U, ELEMENT, k)
    r = oracle.csr(p["Z"], p["mask"])
    K = 5 * 3 * 3
    flat = np.repeat(np.arange(12), np.diff(r["row_ptr"])) * K + r["col"]
    assert np.array_equal(flat, p["kept_idx"])
    assert np.array_equal(r["row_ptr"], np.searchsorted(p["kept_idx"], np.arange(13) * K))


def torch_conv_nhwc(Xb, Zbits, groups, stride, pad):
    X64 = torch.from_numpy(oracle.bf16_to_f64(Xb))
    W64 = torch.from_numpy(oracle.bf16_to_f64(Zbits))
    return F.conv2d(X64, W64, stride=stride, padding=pad, groups=groups).permute(0, 2, 3, 1).numpy()


@pytest.mark.parametrize("N,Cin,H,Wd,A,C,D,stride,pad,groups,density", [
    (2, 6, 9, 9, 8, 3, 3, 1, 1, 1, 0.3),
    (1, 8, 11, 10, 6, 5, 3, 2, 2, 2, 0.5),
    (3, 4, 8, 6, 4, 3, 2, 2, 1, 1, 0.1),
    (1, 16, 5, 5, 8, 1, 1, 1, 0, 4, 0.25),
    (2, 3, 23, 23, 5, 11, 11, 4, 0, 1, 0.05),
    (1, 4, 6, 6, 3, 3, 3, 1, 1, 1, 0.0),
])
def test_conv_csr_matches_torch_float64(N, Cin, H, Wd, A, C, D, stride, pad, groups, density):
    rng = np.random.default_rng(N * 100 + Cin + A + C)
    B = Cin // groups
    X = rng.standard_normal((N, Cin, H, Wd)).astype(np.float32)
    Z = rng.standard_normal((A, B, C, D)).astype(np.float32)
    mask = (rng.random(Z.shape) < density).astype(np.uint8)
    Z[mask == 0] = 0.0
    Xb = oracle.pack(X)
    r = oracle.csr(Z, mask)
    Y = oracle.conv_csr(Xb, r, Z.shape, groups, stride, pad)
    ref = torch_conv_nhwc(Xb, oracle.bf16_bits(Z), groups, stride, pad)
    assert Y.shape == ref.shape
    assert np.max(np.abs(Y - ref)) <= 1e-12 * max(np.max(np.abs(ref)), 1e-300)


@pytest.mark.parametrize("groups,stride,pad", [(1, 1, 1), (2, 2, 0), (4, 1, 2)])
def test_conv_csr_equals_dense_masked(groups, stride, pad):
    rng = np.random.default_rng(groups * 10 + stride)
    N, B, A, C, D, H = 2, 4, 8, 3, 3, 9
    W = rng.standard_normal((A, B, C, D)).astype(np.float32)
    U = (0.1 * rng.standard_normal((A, B, C, D))).astype(np.float32)
    p = oracle.project(W, U, ELEMENT, W.size // 4, groups)
    Xb = oracle.pack(rng.standard_normal((N, groups * B, H, H)).astype(np.float32))
    Ys = oracle.conv_csr(Xb, oracle.csr(p["Z"], p["mask"]), W.shape, groups, stride, pad)
    Yd = oracle.conv(Xb, oracle.compact(p["Z"], groups), C, D, stride, pad)
    assert np.array_equal(Ys, Yd)


def test_table4_table5_element_rates_from_kept_counts():
    """The per-layer non-structured sparsities of Tables 4 and 5 give the
    printed conv2-5 pruning rates (16.1x and 40.5x) once turned into kept
    weight counts of AlexNet's conv2-5 tensors."""
    from workloads import PAPER_ELEMENT_SPARSITY, WORKLOADS, kept_from_sparsity
    layers = {L.name: L for L in WORKLOADS["alexnet_shape30"].layers}
    for block, rate in (("table4_16.1x", 16.1), ("table5_40.5x", 40.5)):
        sp = PAPER_ELEMENT_SPARSITY[block]
        n = sum(layers[f"conv{i}"].n for i in range(2, 6))
        kept = sum(kept_from_sparsity(sp[f"conv{i}"], layers[f"conv{i}"].n) for i in range(2, 6))
        assert round(n / kept, 1) == rate
