"""Pins of the oracle's bf16 rounding, compaction and GEMM-lowered CONV.

  * bf16 rounding equals torch's float32 -> bfloat16 conversion (round to
    nearest even), a library routine;
  * the compacted matrix equals torch indexing of Z's GEMM view [A, B*C*D]
    (kept rows, kept columns in ascending column order) converted by torch,
    bit for bit;
  * the input preparation equals torch's channel selection and bf16
    conversion, bit for bit;
  * the CONV oracle equals torch.nn.functional.conv2d in float64 on the same
    bf16-rounded operands (grouped, strided, padded, non-square kernels);
  * CONV over the compacted matrix equals the dense CONV with the masked
    weights on the kept output channels (bit for bit in float64), and the
    pruned output channels of the dense CONV are exactly zero (Section 3:
    row / column pruning leaves a smaller full GEMM with the same result);
  * the pruning rates printed in Table 1 and the row sparsities of Table 2
    follow from the compacted sizes.
"""
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from oracle import FILTER, SHAPE
from workloads import kept_count

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([
        rng.standard_normal(100000).astype(np.float32) * np.float32(10.0) ** rng.integers(-30, 30, 100000).astype(np.float32),
        # exact ties in the 16 dropped bits, even and odd kept lsb
        (np.array([0x3f808000, 0x3f818000, 0xbf808000, 0xbf818000, 0x3f80ffff, 0x3f807fff,
                   0x7f7fffff, 0x00008000, 0x00018000, 0x80000000, 0], np.uint32)).view(np.float32),
    ]).astype(np.float32)
    x = x[np.isfinite(x)]
    ours = oracle.bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)


@pytest.mark.parametrize("shape,groups", [((8, 6, 3, 3), 1), ((12, 4, 5, 5), 2), ((6, 3, 3, 2), 3)])
def test_compact_matches_torch_indexing(shape, groups):
    rng = np.random.default_rng(sum(shape) + groups)
    A, B, C, D = shape
    Z = rng.standard_normal(shape).astype(np.float32)
    row_mask = (rng.random(A) < 0.6).astype(np.uint8)
    col_mask = (rng.random(B * C * D) < 0.5).astype(np.uint8)
    in_mask = (rng.random(groups * B) < 0.7).astype(np.uint8)
    for use in [(True, False, False, False), (False, True, False, False), (True, True, True, False),
                (False, False, True, False),
                (True, False, True, True)]:
        rm = row_mask if use[0] else None
        cm = col_mask if use[1] else None
        im = in_mask if use[2] else None
        comp = oracle.compact(Z, groups, row_mask=rm, col_mask=cm, in_ch_mask=im, in_compacted=use[3])
        Ag = A // groups
        Zt = torch.from_numpy(Z)
        off = roff = coff = 0
        for gc in range(groups):
            rows = [a for a in range(gc * Ag, (gc + 1) * Ag) if rm is None or rm[a]]
            # GEMM column j = (b*C + c)*D + d of the [A, B*C*D] view, ascending
            cols = [j for j in range(B * C * D)
                    if (cm is None or cm[j]) and (im is None or im[gc * B + j // (C * D)])]
            view = Zt.reshape(A, B * C * D)
            if rows and cols:
                ref = view[rows][:, cols]
                ref = ref.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16).ravel()
            else:
                ref = np.zeros(0, np.uint16)
            assert comp["M"][gc] == len(rows) and comp["K"][gc] == len(cols)
            got = comp["Wc"][off: off + len(rows) * len(cols)]
            assert np.array_equal(got, ref)
            assert list(comp["row_idx"][roff: roff + len(rows)]) == rows
            full = [gc * B + j // (C * D) for j in cols]
            if use[3]:
                pos = np.cumsum(im) - 1
                want_ch = [int(pos[c]) for c in full]
            else:
                want_ch = full
            assert list(comp["col_ch"][coff: coff + len(cols)]) == want_ch
            assert list(comp["col_tap"][coff: coff + len(cols)]) == [j % (C * D) for j in cols]
            off += len(rows) * len(cols)
            roff += len(rows)
            coff += len(cols)


@pytest.mark.parametrize("shape,keep_frac", [((3, 16, 5, 7), None), ((2, 24, 4, 4), 0.5), ((1, 5, 3, 2), 0.4)])
def test_pack_matches_torch(shape, keep_frac):
    """The input preparation equals torch's channel selection and
    float32 -> bfloat16 conversion (a library routine), bit for bit, in NCHW."""
    rng = np.random.default_rng(sum(shape))
    X = rng.standard_normal(shape).astype(np.float32) * np.float32(3.0)
    keep = None
    if keep_frac is not None:
        keep = (rng.random(shape[1]) < keep_frac).astype(np.uint8)
        keep[0] = 1
    got = oracle.pack(X, keep=keep)
    Xt = torch.from_numpy(X)
    if keep is not None:
        Xt = Xt[:, torch.from_numpy(keep.astype(bool))]
    ref = Xt.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert got.shape == ref.shape
    assert np.array_equal(got, ref)


def torch_conv_nhwc(Xb, Wbits, groups, stride, pad):
    X64 = torch.from_numpy(oracle.bf16_to_f64(Xb))
    W64 = torch.from_numpy(oracle.bf16_to_f64(Wbits))
    Y = F.conv2d(X64, W64, stride=stride, padding=pad, groups=groups)
    return Y.permute(0, 2, 3, 1).numpy()


@pytest.mark.parametrize("N,Cin,H,Wd,A,C,D,stride,pad,groups", [
    (2, 6, 9, 9, 8, 3, 3, 1, 1, 1),
    (1, 3, 23, 23, 5, 11, 11, 4, 0, 1),
    (2, 8, 7, 7, 6, 5, 5, 1, 2, 2),
    (3, 4, 8, 6, 4, 3, 2, 2, 1, 1),
    (1, 16, 5, 5, 8, 1, 1, 1, 0, 4),
    (2, 4, 9, 9, 4, 1, 1, 2, 0, 1),
])
def test_conv_matches_torch_float64(N, Cin, H, Wd, A, C, D, stride, pad, groups):
    rng = np.random.default_rng(N * 1000 + Cin * 10 + A)
    B = Cin // groups
    X = rng.standard_normal((N, Cin, H, Wd)).astype(np.float32)
    Z = rng.standard_normal((A, B, C, D)).astype(np.float32)
    Xb = oracle.pack(X)
    comp = oracle.compact(Z, groups)
    Y = oracle.conv(Xb, comp, C, D, stride, pad)
    ref = torch_conv_nhwc(Xb, oracle.bf16_bits(Z), groups, stride, pad)
    assert Y.shape == ref.shape
    assert np.max(np.abs(Y - ref)) <= 1e-12 * np.max(np.abs(ref))


@pytest.mark.parametrize("kind", [FILTER, SHAPE])
def test_compacted_conv_equals_dense_masked(kind):
    rng = np.random.default_rng(kind + 40)
    N, groups, B, A, C, D, H = 2, 2, 6, 8, 3, 3, 7
    W = rng.standard_normal((A, B, C, D)).astype(np.float32)
    U = (0.1 * rng.standard_normal((A, B, C, D))).astype(np.float32)
    G = oracle.n_groups(W.shape, kind)
    r = oracle.project(W, U, kind, G // 3)
    X = rng.standard_normal((N, groups * B, H, H)).astype(np.float32)
    Xb = oracle.pack(X)
    rows = r["mask"] if kind == FILTER else None
    cols = r["mask"] if kind == SHAPE else None
    comp = oracle.compact(r["Z"], groups, row_mask=rows, col_mask=cols)
    dense = oracle.compact(r["Z"], groups)
    Yc = oracle.conv(Xb, comp, C, D, 1, 1)
    Yd = oracle.conv(Xb, dense, C, D, 1, 1)
    kept_rows = comp["row_idx"]
    assert np.array_equal(Yc, Yd[..., kept_rows])
    pruned = np.setdiff1d(np.arange(A), kept_rows)
    assert not np.any(Yd[..., pruned])
    flops = 2 * N * Yc.shape[1] * Yc.shape[2] * int(np.sum(comp["M"].astype(np.int64) * comp["K"]))
    dense_flops = 2 * N * Yd.shape[1] * Yd.shape[2] * A * B * C * D
    assert flops < dense_flops


def test_chain_input_compaction_equals_dense():
    """Filter pruning with the input restricted to the previous layer's kept
    filters: the conv over the channel-compacted input equals the dense conv
    over the full input on the kept filters."""
    rng = np.random.default_rng(99)
    N, groups, B, A, C, D, H = 2, 2, 4, 6, 3, 3, 6
    prev_mask = np.zeros(groups * B, np.uint8)
    prev_mask[rng.choice(groups * B, size=groups * B // 2, replace=False)] = 1
    W = rng.standard_normal((A, B, C, D)).astype(np.float32)
    U = np.zeros_like(W)
    r = oracle.project(W, U, FILTER, 3, groups=groups, in_ch_mask=prev_mask)
    X = rng.standard_normal((N, groups * B, H, H)).astype(np.float32)
    Xc = oracle.pack(X, keep=prev_mask)
    Xf = oracle.pack(X)
    comp = oracle.compact(r["Z"], groups, row_mask=r["mask"], in_ch_mask=prev_mask, in_compacted=True)
    dense = oracle.compact(r["Z"], groups)
    Yc = oracle.conv(Xc, comp, C, D, 1, 1)
    Yd = oracle.conv(Xf, dense, C, D, 1, 1)
    assert np.array_equal(Yc, Yd[..., comp["row_idx"]])


def _read_golden(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append(line.split())
    return rows


def test_table1_pruning_rates_from_compaction():
    """Table 1: pruning rate = weights / kept weights after column pruning."""
    rows = _read_golden("table1_column_pruning.txt")
    rng = np.random.default_rng(1)
    tot, kept_tot = 0, 0
    for name, A, K, sparsity, rate in rows:
        if name == "conv2-5":
            assert round(tot / kept_tot, 1) == float(rate)
            # the aggregate sparsity is printed to 0.1% from whole-column counts
            # the table does not give: agree within one printed unit
            assert abs(100 * (1 - kept_tot / tot) - float(sparsity)) <= 0.1
            continue
        A, K = int(A), int(K)
        keep = kept_count(int(round(100 - float(sparsity))), K)
        col_mask = np.zeros(K, np.uint8)
        col_mask[rng.choice(K, size=keep, replace=False)] = 1
        Z = np.ones((A, K, 1, 1), np.float32)  # GEMM view: [A, B*C*D]
        comp = oracle.compact(Z, 1, col_mask=col_mask)
        kept = int(comp["M"][0]) * int(comp["K"][0])
        assert round(A * K / kept, 1) == float(rate), name
        tot += A * K
        kept_tot += kept


def test_table2_row_sparsity_from_compaction():
    rows = _read_golden("table2_row_sparsity.txt")
    rng = np.random.default_rng(2)
    for name, A, sparsity, pruned in rows:
        A, pruned = int(A), int(pruned)
        row_mask = np.ones(A, np.uint8)
        row_mask[rng.choice(A, size=pruned, replace=False)] = 0
        comp = oracle.compact(np.ones((A, 2, 1, 1), np.float32), 1, row_mask=row_mask)
        assert round(100 * (A - int(comp["M"][0])) / A, 1) == float(sparsity), name
