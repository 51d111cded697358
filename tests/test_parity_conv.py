"""GPU parity of structadmm_compact, structadmm_pack_nhwc and
structadmm_conv_fwd against the oracle.

Bar: compacted matrix, row / column tables and packed input bit-exact; CONV
output (bf16, fp32 MFMA accumulation) within max|dY| / RMS(Y_ref) <= 2e-2 of
the oracle's binary64 CONV over the same bf16 operands.  Small cases span
several tiles with ragged tails in every dimension; workload cases run the
benchmark's launch configuration at full batch and compare sampled images.
"""
import numpy as np
import pytest

import oracle
import paper_1807_11091_amd as sa
from gpu_helpers import (DEV, GpuLayer, bf16_bits_to_f64, bitwise_equal, maxabs_over_rms, run_project,
                         to_dev, torch)
from workloads import PAPER_TABLE_SPARSITY, WORKLOADS, input_nchw, kept_from_sparsity, layer_tensors

pytestmark = pytest.mark.gpu

TOL = 2e-2


def gpu_compact(Z, groups, row_mask=None, col_mask=None, in_ch_mask=None, in_compacted=False):
    t = torch()
    Wc, row_idx, col_ch, col_tap, sizes = sa.compact(Z, groups, row_mask=row_mask, col_mask=col_mask,
                                                     in_ch_mask=in_ch_mask, in_compacted=in_compacted)
    t.cuda.synchronize()
    return Wc, row_idx, col_ch, col_tap, sizes


def check_compact(gpu, ref):
    """Sizes, kept rows and the padding must be equal; columns are matched by
    their (input channel, tap) pair, since the library may order a group's
    columns differently from the oracle's ascending GEMM column index (any
    order gives the same GEMM): the kept pairs must be the same set, and every
    GPU column must equal, bit for bit, the oracle's column of its pair.  The
    library's alignment columns (kpad of a group, on a channel-compacted
    input) are further pairs of the group's 8-aligned window whose entries are
    all +0, so that they add nothing to the CONV."""
    Wc, row_idx, col_ch, col_tap, sizes = gpu
    assert list(sizes.M)[: sizes.groups] == list(ref["M"])
    kpad = list(sizes.kpad)[: sizes.groups]
    assert [k - p for k, p in zip(list(sizes.K)[: sizes.groups], kpad)] == list(ref["K"])
    nr = int(ref["M"].sum())
    assert np.array_equal(row_idx.cpu().numpy()[:nr], ref["row_idx"])
    full = Wc.cpu().numpy()
    gch, gtap = col_ch.cpu().numpy(), col_tap.cpu().numpy()
    woff = coff = 0
    for g in range(sizes.groups):
        M, K, ldk, off = sizes.M[g], sizes.K[g], sizes.ldk[g], sizes.wc_offset[g]
        goff, Kr = sizes.col_offset[g], K - kpad[g]
        mat = full[off: off + M * ldk].reshape(M, ldk)
        # padding columns hold +0
        assert not np.any(mat[:, K:])
        rch, rtap = ref["col_ch"][coff: coff + Kr], ref["col_tap"][coff: coff + Kr]
        rkey = {(int(c), int(t)): j for j, (c, t) in enumerate(zip(rch, rtap))}
        assert len(rkey) == Kr
        gkey = [(int(c), int(t)) for c, t in zip(gch[goff: goff + K], gtap[goff: goff + K])]
        assert len(set(gkey)) == K and set(rkey) <= set(gkey)
        kept = np.array([k in rkey for k in gkey], dtype=bool)
        perm = np.array([rkey[k] for k in gkey if k in rkey], dtype=np.int64)
        rmat = ref["Wc"][woff: woff + M * Kr].reshape(M, Kr)
        assert np.array_equal(mat[:, :K][:, kept], rmat[:, perm])
        if kpad[g]:
            lo, run = sizes.run_base[g], sizes.run[g]
            assert lo % 8 == 0 and run % 8 == 0 and K == run * (K // run)
            extra = [k for k in gkey if k not in rkey]
            assert all(lo <= c < lo + run for c, _ in extra)
            assert {(c, t) for c in range(lo, lo + run) for t in range(K // run)} == set(gkey)
            assert not np.any(mat[:, :K][:, ~kept])
        woff += M * Kr
        coff += Kr


def conv_case(N, Cin, H, Wd, A, C, D, stride, pad, groups, kind, keep, seed, dense_too=True, dead_lo=0,
              expect=None):
    rng = np.random.default_rng(seed)
    B = Cin // groups
    shape = (A, B, C, D)
    W = (0.05 * rng.standard_normal(shape)).astype(np.float32)
    U = (0.01 * rng.standard_normal(shape)).astype(np.float32)
    # the first dead_lo input channels of every group score 0 and are pruned
    W[:, :dead_lo] = 0
    U[:, :dead_lo] = 0
    G = {sa.FILTER: A, sa.CHANNEL: B, sa.SHAPE: B * C * D}[kind]
    k = max(1, int(round(keep * G)))
    # projection on both sides (bit-exact parity is checked elsewhere; here it feeds compaction)
    ref = oracle.project(W, U, kind, k, groups)
    L = GpuLayer(W, U, kind, k, groups)
    got = run_project([L])[0]
    assert np.array_equal(got["mask"], ref["mask"]) and bitwise_equal(got["Z"], ref["Z"])
    rows = L.mask if kind == sa.FILTER else None
    cols = L.mask if kind == sa.SHAPE else None
    ch = L.mask if kind == sa.CHANNEL else None
    Wc, row_idx, col_ch, col_tap, sizes = sa.compact(L.Z, groups, row_mask=rows, col_mask=cols, chan_mask=ch)
    r_rows = ref["mask"] if kind == sa.FILTER else None
    r_cols = ref["mask"] if kind == sa.SHAPE else None
    r_ch = ref["mask"] if kind == sa.CHANNEL else None
    rc = oracle.compact(ref["Z"], groups, row_mask=r_rows, col_mask=r_cols, chan_mask=r_ch)
    check_compact((Wc, row_idx, col_ch, col_tap, sizes), rc)
    X = rng.standard_normal((N, Cin, H, Wd)).astype(np.float32)
    dX = to_dev(X)
    Xp = sa.pack_nhwc(dX)
    Xb = oracle.pack(X)
    assert bitwise_equal(Xp.cpu().numpy(), Xb.transpose(0, 2, 3, 1))
    if expect is not None:  # the kernel the case is meant to exercise
        plan = sa.conv_plan(Xp, sizes, C, D, stride, pad)
        for key, want in expect.items():
            got = plan[key] if key != "path" else set(plan["path"]) - {sa.CONV_NONE}
            assert got == want, (key, got, want, plan)
    Y = sa.conv_fwd(Xp, Wc, col_ch, col_tap, sizes, C, D, stride, pad)
    Yr = oracle.conv(Xb, rc, C, D, stride, pad)
    y = bf16_bits_to_f64(Y.cpu().numpy())
    assert y.shape == Yr.shape
    err = maxabs_over_rms(y, Yr)
    assert err <= TOL, err
    if dense_too:
        Wd_, ri, cc, ct, sd = sa.compact(L.Z, groups)
        Yd = sa.conv_fwd(Xp, Wd_, cc, ct, sd, C, D, stride, pad)
        rd = oracle.compact(ref["Z"], groups)
        Ydr = oracle.conv(Xb, rd, C, D, stride, pad)
        yd = bf16_bits_to_f64(Yd.cpu().numpy())
        kept = rc["row_idx"]
        assert dense_masked_error(yd, Ydr, kept) <= TOL
        # compacted and dense agree on the kept output channels
        assert maxabs_over_rms(y, yd[..., kept]) <= TOL
    return err


def dense_masked_error(yd, ref, kept_rows):
    """Dense CONV with masked weights: pruned output channels are exactly zero
    on both sides; the kept ones are held to the tolerance (their RMS, not one
    deflated by the zero channels, sets the scale)."""
    A = ref.shape[-1]
    pruned = np.setdiff1d(np.arange(A), kept_rows)
    assert not np.any(ref[..., pruned]) and not np.any(yd[..., pruned])
    return maxabs_over_rms(yd[..., kept_rows], ref[..., kept_rows])


SMALL = [
    # N, Cin, H,  W, A,  C, D, s, p, g, kind,        keep
    (3, 16, 9, 9, 130, 3, 3, 1, 1, 1, sa.FILTER, 0.6),
    (2, 32, 12, 11, 40, 3, 3, 1, 1, 1, sa.FILTER, 1.0),
    (2, 24, 10, 10, 20, 3, 3, 2, 1, 1, sa.FILTER, 1.0),
    (2, 3, 35, 35, 24, 11, 11, 4, 0, 1, sa.FILTER, 0.5),
    (2, 32, 13, 13, 48, 3, 3, 1, 1, 2, sa.SHAPE, 0.3),
    (2, 64, 7, 7, 96, 1, 1, 1, 0, 1, sa.FILTER, 0.6),
    (2, 64, 14, 14, 64, 1, 1, 2, 0, 1, sa.CHANNEL, 0.5),
    (1, 48, 8, 8, 300, 3, 3, 1, 1, 1, sa.SHAPE, 0.25),
    (5, 8, 7, 9, 16, 3, 2, 1, 0, 1, sa.FILTER, 0.75),
    (1, 256, 6, 6, 40, 3, 3, 1, 1, 2, sa.FILTER, 0.5),
    (2, 20, 15, 13, 70, 3, 3, 2, 1, 1, sa.SHAPE, 0.3),
    (2, 6, 23, 23, 34, 5, 5, 3, 2, 2, sa.SHAPE, 0.4),
    (3, 16, 11, 11, 200, 3, 3, 1, 1, 1, sa.SHAPE, 0.5),
    (2, 16, 17, 15, 40, 3, 3, 2, 1, 1, sa.SHAPE, 0.4),
    (2, 24, 23, 23, 36, 5, 5, 3, 2, 3, sa.SHAPE, 0.4),
    # strided, few channels: space-to-depth image of the input, then the footprint kernel
    (2, 2, 19, 17, 40, 5, 5, 2, 2, 1, sa.SHAPE, 0.4),
    (2, 4, 16, 16, 24, 3, 3, 2, 1, 2, sa.SHAPE, 0.5),
    # space-to-depth channels padded to 8 (ResNet stem shape), and channel padding only
    (2, 3, 30, 28, 20, 7, 7, 2, 3, 1, sa.FILTER, 0.6),
    (2, 3, 12, 11, 16, 3, 3, 1, 1, 1, sa.SHAPE, 0.5),
    # inputs whose byte size is not a multiple of 4: the space-to-depth copy's last chunk
    (1, 3, 13, 13, 16, 3, 3, 2, 1, 1, sa.SHAPE, 0.5),
    (1, 3, 11, 9, 8, 3, 3, 1, 1, 1, sa.FILTER, 0.5),
    # odd numbers of kept filters: output rows not 16-byte aligned
    (2, 16, 9, 9, 38, 1, 1, 1, 0, 1, sa.FILTER, 0.6),
    (2, 32, 8, 8, 50, 3, 3, 1, 1, 2, sa.FILTER, 0.62),
    # input rows too wide for an LDS copy of the footprint: two-phase gather
    (1, 64, 3, 2100, 40, 3, 3, 1, 1, 1, sa.SHAPE, 0.3),
    # six-wavefront tiles: 529 tiles of 128 pixels take two rounds at two
    # workgroups per CU, 353 of 192 pixels one (tiles span image boundaries)
    (400, 16, 13, 13, 128, 3, 3, 1, 1, 1, sa.SHAPE, 0.3),
]


@pytest.mark.parametrize("case", SMALL, ids=[f"c{i}" for i in range(len(SMALL))])
def test_conv_small(case):
    conv_case(*case, seed=hash(case) % 2**31)


# cases pinned to a kernel and tile shape (the plan is asserted before the
# parity check, so a change of the selection cannot silently move them)
PLANNED = [
    # at most 48 kept filters over 384-512 columns and at least 2^16 pixels:
    # the 16-row kernel (ragged pixel tails: 65,856 and 73,728 pixels)
    ((21, 448, 56, 56, 64, 1, 1, 1, 0, 1, sa.FILTER, 0.6), {"path": {sa.CONV_DIRECT_IG}, "ig_tile": (3, 2, 1, 1)}),
    ((21, 448, 56, 56, 64, 1, 1, 1, 0, 1, sa.FILTER, 0.45), {"path": {sa.CONV_DIRECT_IG}, "ig_tile": (2, 2, 1, 1)}),
    ((128, 48, 24, 24, 64, 3, 3, 1, 1, 1, sa.FILTER, 0.6), {"path": {sa.CONV_DIRECT_IG}, "ig_tile": (3, 2, 1, 1)}),
    # more filters, fewer columns or fewer pixels: the LDS-staged kernel
    ((21, 256, 56, 56, 128, 1, 1, 1, 0, 1, sa.FILTER, 0.6), {"path": {sa.CONV_DIRECT}}),
    ((70, 256, 14, 14, 512, 1, 1, 1, 0, 1, sa.FILTER, 0.6), {"path": {sa.CONV_DIRECT}}),
    ((48, 64, 20, 20, 64, 1, 1, 1, 0, 1, sa.FILTER, 0.6), {"path": {sa.CONV_DIRECT}}),
    # every tap of a channel run, aligned or wide: the LDS-staged kernel
    ((114, 64, 12, 12, 128, 3, 3, 1, 1, 1, sa.FILTER, 1.0), {"path": {sa.CONV_DIRECT}}),
    ((114, 64, 12, 12, 96, 3, 3, 1, 1, 1, sa.FILTER, 0.6), {"path": {sa.CONV_DIRECT}}),
    # split over the columns at a small batch: 36 slices of 64 columns per
    # tile, two tiles; 9 slices stay whole
    ((1, 256, 12, 12, 96, 3, 3, 1, 1, 1, sa.FILTER, 0.6), {"path": {sa.CONV_DIRECT}, "ksplit": 8}),
    ((1, 64, 12, 12, 96, 3, 3, 1, 1, 1, sa.FILTER, 0.6), {"path": {sa.CONV_DIRECT}, "ksplit": 1}),
    # gathered im2col rows (input rows too wide for LDS), 27 slices over 50
    # tiles: the split takes 5 chunks (one workgroup per CU)
    ((1, 256, 3, 2100, 40, 3, 3, 1, 1, 1, sa.SHAPE, 0.75), {"path": {sa.CONV_GATHER}, "ksplit": 5}),
    # footprint kernel: six-wavefront tiles of 192 filters (AlexNet conv4 at
    # batch 128: one workgroup per CU, 226 tiles of 192 pixels fill one round
    # where 338 of 128 need two) and four-wavefront tiles (two per CU)
    ((128, 384, 13, 13, 384, 3, 3, 1, 1, 2, sa.SHAPE, 0.3), {"path": {sa.CONV_FOOTPRINT}, "footprint_tile": (6, 1, 6)}),
    ((400, 16, 13, 13, 128, 3, 3, 1, 1, 1, sa.SHAPE, 0.3), {"path": {sa.CONV_FOOTPRINT}, "footprint_tile": (4, 1, 4)}),
    ((2, 32, 13, 13, 48, 3, 3, 1, 1, 2, sa.SHAPE, 0.3), {"path": {sa.CONV_FOOTPRINT}}),
    # stem: space-to-depth image, then the direct kernels over every tap and
    # channel of the image (weights rewritten in that column order)
    ((2, 3, 30, 28, 20, 7, 7, 2, 3, 1, sa.FILTER, 0.6), {"path": {sa.CONV_DIRECT}, "space_to_depth": 2}),
    ((64, 3, 60, 60, 40, 7, 7, 2, 3, 1, sa.FILTER, 0.6), {"path": {sa.CONV_DIRECT}, "space_to_depth": 2, "ksplit": 1}),
    ((8, 3, 67, 67, 96, 11, 11, 4, 0, 1, sa.SHAPE, 0.3), {"space_to_depth": 4}),
    # grouped layer on a space-to-depth image: the footprint kernel
    ((2, 4, 16, 16, 24, 3, 3, 2, 1, 2, sa.SHAPE, 0.5), {"path": {sa.CONV_FOOTPRINT}, "space_to_depth": 2}),
]


@pytest.mark.parametrize("case,expect", PLANNED, ids=[f"p{i}" for i in range(len(PLANNED))])
def test_conv_planned_kernel(case, expect):
    conv_case(*case, seed=sum(case[:9]), dense_too=False, expect=expect)


def test_conv_16row_tile_shapes():
    """1x1 layers of 448 input channels at 65,856 pixels, kept-filter counts
    that take both tile shapes of the 16-row kernel (and the LDS-staged kernel
    above 48), all against the oracle."""
    seen = set()
    rng = np.random.default_rng(448)
    X = rng.standard_normal((21, 448, 56, 56)).astype(np.float32)
    Xp = sa.pack_nhwc(to_dev(X))
    for A, keep in ((64, 0.6), (64, 0.45), (40, 0.5), (128, 0.6), (100, 0.6), (512, 0.6)):
        rng = np.random.default_rng(A + int(100 * keep))
        k = max(1, int(round(keep * A)))
        mask = np.zeros(A, np.uint8)
        mask[rng.choice(A, size=k, replace=False)] = 1
        Z = (0.05 * rng.standard_normal((A, 448, 1, 1))).astype(np.float32)
        Wc, ri, cc, ct, sizes = sa.compact(to_dev(Z), 1, row_mask=to_dev(mask))
        plan = sa.conv_plan(Xp, sizes, 1, 1, 1, 0)
        if plan["path"] == [sa.CONV_DIRECT_IG]:
            seen.add(plan["ig_tile"])
        Y = sa.conv_fwd(Xp, Wc, cc, ct, sizes, 1, 1, 1, 0)
        rc = oracle.compact(Z, 1, row_mask=mask)
        sel = [0, 11, 20]  # three images of the batch
        Yr = oracle.conv(oracle.pack(X[sel]), rc, 1, 1, 1, 0)
        err = maxabs_over_rms(bf16_bits_to_f64(Y.cpu().numpy()[sel]), Yr)
        assert err <= TOL, (A, keep, plan, err)
    assert seen == {(2, 2, 1, 1), (3, 2, 1, 1)}, seen


def test_conv_unaligned_channel_window():
    # kept columns start at channel 3 (of 32 per group): the LDS copy starts at
    # the 8-aligned channel below
    assert conv_case(2, 64, 13, 13, 48, 3, 3, 1, 1, 2, sa.SHAPE, 0.3, seed=7, dead_lo=3) <= TOL


def test_compact_chain_input_positions():
    """Channel-compacted input (the previous layer's kept filters): positions
    in the compacted input, and the CONV over the gathered input."""
    rng = np.random.default_rng(31)
    groups, B, A, C, D = 2, 24, 32, 3, 3
    W = (0.05 * rng.standard_normal((A, B, C, D))).astype(np.float32)
    U = np.zeros_like(W)
    prev = np.zeros(groups * B, np.uint8)
    prev[rng.choice(groups * B, size=groups * B // 2, replace=False)] = 1
    ref = oracle.project(W, U, sa.FILTER, 16, groups, in_ch_mask=prev)
    L = GpuLayer(W, U, sa.FILTER, 16, groups, in_ch_mask=prev)
    got = run_project([L])[0]
    assert np.array_equal(got["mask"], ref["mask"])
    dprev = L.in_ch_mask
    gc = sa.compact(L.Z, groups, row_mask=L.mask, in_ch_mask=dprev, in_compacted=True)
    rc = oracle.compact(ref["Z"], groups, row_mask=ref["mask"], in_ch_mask=prev, in_compacted=True)
    check_compact(gc, rc)
    X = rng.standard_normal((2, groups * B, 9, 9)).astype(np.float32)
    Xp = sa.pack_nhwc(to_dev(X), keep=dprev)
    Xb = oracle.pack(X, keep=prev)
    assert bitwise_equal(Xp.cpu().numpy(), Xb.transpose(0, 2, 3, 1))
    Wc, ri, cc, ct, sizes = gc
    Y = sa.conv_fwd(Xp, Wc, cc, ct, sizes, C, D, 1, 1)
    Yr = oracle.conv(Xb, rc, C, D, 1, 1)
    assert maxabs_over_rms(bf16_bits_to_f64(Y.cpu().numpy()), Yr) <= TOL


@pytest.mark.parametrize("kept, kpad_expect", [
    ((20, 20), (4, 4)),      # both groups widen to 8-aligned windows of 24 positions
    ((20, 3, 17), (4, 0, 7)),  # group 1: a window of 8 over 3 kept is too wide
    ((20, 3, 13), (0, 0, 0)),  # 36 input channels: no direct kernel, no widening
    ((16, 8), (0, 0)),       # already aligned
])
def test_compact_alignment_columns(kept, kpad_expect):
    """Alignment columns on a channel-compacted input: group g keeps the
    channels kept[g] of the previous layer; the library widens unaligned runs
    to 8-aligned windows (+0 columns, kpad_expect[g] positions per tap), and
    the CONV over them is the CONV of the kept columns."""
    rng = np.random.default_rng(sum(kept))
    groups, B, A, C, D = len(kept), 32, 16 * len(kept), 3, 3
    prev = np.zeros(groups * B, np.uint8)
    for g, n in enumerate(kept):
        prev[g * B + rng.choice(B, size=n, replace=False)] = 1
    W = (0.05 * rng.standard_normal((A, B, C, D))).astype(np.float32)
    U = np.zeros_like(W)
    ref = oracle.project(W, U, sa.FILTER, 8 * groups, groups, in_ch_mask=prev)
    L = GpuLayer(W, U, sa.FILTER, 8 * groups, groups, in_ch_mask=prev)
    got = run_project([L])[0]
    assert np.array_equal(got["mask"], ref["mask"])
    gc = sa.compact(L.Z, groups, row_mask=L.mask, in_ch_mask=L.in_ch_mask, in_compacted=True)
    rc = oracle.compact(ref["Z"], groups, row_mask=ref["mask"], in_ch_mask=prev, in_compacted=True)
    check_compact(gc, rc)
    Wc, ri, cc, ct, sizes = gc
    assert [sizes.kpad[g] for g in range(groups)] == [p * C * D for p in kpad_expect]
    X = rng.standard_normal((3, groups * B, 10, 11)).astype(np.float32)
    Xp = sa.pack_nhwc(to_dev(X), keep=L.in_ch_mask)
    plan = sa.conv_plan(Xp, sizes, C, D, 1, 1)
    for g in range(groups):
        aligned = sum(kept) % 8 == 0 and kept[g] % 8 == 0 and sum(kept[:g]) % 8 == 0
        if sizes.M[g] > 0 and (kpad_expect[g] or aligned):
            assert plan["path"][g] in (sa.CONV_DIRECT, sa.CONV_DIRECT_IG), (g, plan)
    Xb = oracle.pack(X, keep=prev)
    Y = sa.conv_fwd(Xp, Wc, cc, ct, sizes, C, D, 1, 1)
    Yr = oracle.conv(Xb, rc, C, D, 1, 1)
    assert maxabs_over_rms(bf16_bits_to_f64(Y.cpu().numpy()), Yr) <= TOL


def test_compact_many_matches_one_by_one():
    """structadmm_compact_many over layers of every kind (filter-pruned,
    shape-pruned with groups, channel-masked, channel-compacted input with
    alignment columns, an empty layer) gives, byte for byte, what one
    structadmm_compact call per layer gives, and the oracle's matrices."""
    t = torch()
    rng = np.random.default_rng(77)
    items, refs = [], []

    def add(A, B, C, D, groups, **masks):
        Z = (0.05 * rng.standard_normal((A, B, C, D))).astype(np.float32)
        dev = {k: (to_dev(v) if isinstance(v, np.ndarray) else v) for k, v in masks.items()}
        items.append(dict(Z=to_dev(Z), groups=groups, **dev))
        refs.append((Z, groups, masks))

    def mask(n, k):
        m = np.zeros(n, np.uint8)
        m[rng.choice(n, size=k, replace=False)] = 1
        return m

    add(96, 64, 3, 3, 1, row_mask=mask(96, 58))
    add(64, 48, 3, 3, 2, col_mask=mask(48 * 9, 130))
    add(32, 40, 1, 1, 1, chan_mask=mask(40, 24))
    prev = np.zeros(64, np.uint8)
    prev[:13] = 1
    prev[32:51] = 1
    add(32, 32, 3, 3, 2, row_mask=mask(32, 20), in_ch_mask=prev, in_compacted=True)
    add(16, 8, 3, 3, 1, row_mask=np.zeros(16, np.uint8))
    many = sa.compact_many(items)
    for it, (Z, groups, masks), got in zip(items, refs, many):
        one = sa.compact(it["Z"], groups, row_mask=it.get("row_mask"), col_mask=it.get("col_mask"),
                         chan_mask=it.get("chan_mask"), in_ch_mask=it.get("in_ch_mask"),
                         in_compacted=bool(it.get("in_compacted")))
        sg, so = got[4], one[4]
        assert bytes(sg) == bytes(so)
        used = [sum(sg.M[g] * sg.ldk[g] for g in range(groups)), sum(sg.M[g] for g in range(groups)),
                sum(sg.K[g] for g in range(groups)), sum(sg.K[g] for g in range(groups))]
        for a, b, n in zip(got[:4], one[:4], used):  # Wc, row_idx, col_ch, col_tap
            assert t.equal(a[:n], b[:n])
        rc = oracle.compact(Z, groups, row_mask=masks.get("row_mask"), col_mask=masks.get("col_mask"),
                            chan_mask=masks.get("chan_mask"), in_ch_mask=masks.get("in_ch_mask"),
                            in_compacted=bool(masks.get("in_compacted")))
        check_compact(got, rc)


def sampled_images(N, count):
    """count images spread over the batch, always the first and the last
    (every image when count >= N)."""
    if count >= N:
        return list(range(N))
    return sorted({int(round(i * (N - 1) / (count - 1))) for i in range(count)})


def workload_conv(name, layer_ids=None, variant=0, chain=False, images=4):
    """Full-batch GPU path of a workload (projection -> compaction -> pack ->
    compacted and dense CONV); the oracle recomputes `images` images of the
    batch (all of them when images >= batch)."""
    t = torch()
    wl = WORKLOADS[name]
    kind, pct = wl.variants[variant]
    ids = range(len(wl.layers)) if layer_ids is None else layer_ids
    prev_gpu, prev_ref = None, None
    worst = 0.0
    for li in ids:
        L = wl.layers[li]
        W, U = layer_tensors(wl, li)
        k = wl.k_for(li, kind, pct)
        inm_gpu = prev_gpu if chain else None
        inm_ref = prev_ref if chain else None
        ref = oracle.project(W, U, kind, k, L.groups, in_ch_mask=inm_ref)
        gl = GpuLayer(W, U, kind, k, L.groups, in_ch_mask=inm_gpu)
        got = run_project([gl])[0]
        assert np.array_equal(got["mask"], ref["mask"]) and bitwise_equal(got["Z"], ref["Z"])
        rows = gl.mask if kind == sa.FILTER else None
        cols = gl.mask if kind == sa.SHAPE else None
        gc = sa.compact(gl.Z, L.groups, row_mask=rows, col_mask=cols, in_ch_mask=inm_gpu,
                        in_compacted=inm_gpu is not None)
        rc = oracle.compact(ref["Z"], L.groups, row_mask=ref["mask"] if kind == sa.FILTER else None,
                            col_mask=ref["mask"] if kind == sa.SHAPE else None, in_ch_mask=inm_ref,
                            in_compacted=inm_ref is not None)
        check_compact(gc, rc)
        X = input_nchw(wl, li)
        dX = to_dev(X)
        Xp = sa.pack_nhwc(dX, keep=inm_gpu)
        Wc, ri, cc, ct, sizes = gc
        Y = sa.conv_fwd(Xp, Wc, cc, ct, sizes, L.C, L.D, L.stride, L.pad)
        Xf = sa.pack_nhwc(dX)
        gd = sa.compact(gl.Z, L.groups)
        Yd = sa.conv_fwd(Xf, gd[0], gd[2], gd[3], gd[4], L.C, L.D, L.stride, L.pad)
        t.cuda.synchronize()
        sel = sampled_images(wl.batch, images)
        Xb = oracle.pack(X[sel], keep=inm_ref)
        Yr = oracle.conv(Xb, rc, L.C, L.D, L.stride, L.pad)
        y = bf16_bits_to_f64(Y.cpu().numpy()[sel])
        err = maxabs_over_rms(y, Yr)
        assert err <= TOL, ("compacted", name, li, err)
        rd = oracle.compact(ref["Z"], L.groups)
        Ydr = oracle.conv(oracle.pack(X[sel]), rd, L.C, L.D, L.stride, L.pad)
        yd = bf16_bits_to_f64(Yd.cpu().numpy()[sel])
        errd = dense_masked_error(yd, Ydr, rc["row_idx"])
        assert errd <= TOL, ("dense", name, li, errd)
        worst = max(worst, err, errd)
        prev_gpu, prev_ref = gl.mask, ref["mask"]
        del dX, Xp, Xf, Y, Yd
    return worst


def test_conv_workload_cifar():
    workload_conv("cifar_conv64", images=8)


def test_conv_workload_alexnet_shape30():
    # the whole batch of 128 images
    workload_conv("alexnet_shape30", images=128)


def test_conv_workload_alexnet_chain():
    workload_conv("alexnet_chain_f50c50", chain=True, images=128)


def _resnet50_stage(prefix):
    wl = WORKLOADS["resnet50_filter60"]
    return [i for i, l in enumerate(wl.layers)
            if l.name.startswith(prefix) or (prefix == "layer1" and l.name == "conv1")]


@pytest.mark.parametrize("stage", ["layer1", "layer2", "layer3", "layer4"])
def test_conv_workload_resnet50(stage):
    """Every one of the 53 CONVs (the stem goes with stage 1), four images of
    the batch of 64 each: the first, the last and two inside."""
    workload_conv("resnet50_filter60", _resnet50_stage(stage), images=4)


def test_conv_workload_resnet50_covers_every_layer():
    ids = sorted(i for st in ("layer1", "layer2", "layer3", "layer4") for i in _resnet50_stage(st))
    assert ids == list(range(len(WORKLOADS["resnet50_filter60"].layers))) and len(ids) == 53


@pytest.mark.parametrize("variant", range(9))
def test_conv_workload_sweep(variant):
    """filter / shape / element-wise at 10, 25 and 50% kept."""
    workload_conv("resnet50_s3_sweep", variant=variant, images=4)


def table_masks(W, U, L, block):
    """Row (filter) and column (filter-shape) masks with the per-layer
    sparsities of the pruned AlexNet models of Tables 1-2, drawn by projecting
    the layer's synthetic V = W + U; GPU and oracle masks must agree."""
    rs, cs = PAPER_TABLE_SPARSITY[block][L.name]
    out = []
    for kind, sp, G in ((sa.FILTER, rs, L.A), (sa.SHAPE, cs, L.K)):
        if sp == 0.0:
            out.append(None)
            continue
        k = kept_from_sparsity(sp, G)
        ref = oracle.project(W, U, kind, k, L.groups)
        got = run_project([GpuLayer(W, U, kind, k, L.groups)])[0]
        assert np.array_equal(got["mask"], ref["mask"])
        out.append(ref["mask"])
    return out


@pytest.mark.parametrize("block", list(PAPER_TABLE_SPARSITY))
def test_conv_table_replay_batch1(block):
    """The batch-1 CONVs of AlexNet conv1-5 pruned to the row / column
    sparsities of Tables 1-2 (rows and columns removed together)."""
    wl = WORKLOADS["alexnet_shape30"]
    for li, L in enumerate(wl.layers):
        W, U = layer_tensors(wl, li)
        rows, cols = table_masks(W, U, L, block)
        dW = to_dev(W)
        got = sa.compact(dW, L.groups, row_mask=None if rows is None else to_dev(rows),
                         col_mask=None if cols is None else to_dev(cols))
        rc = oracle.compact(W, L.groups, row_mask=rows, col_mask=cols)
        check_compact(got, rc)
        X = input_nchw(wl, li, batch=1)
        Xp = sa.pack_nhwc(to_dev(X))
        Y = sa.conv_fwd(Xp, got[0], got[2], got[3], got[4], L.C, L.D, L.stride, L.pad)
        Yr = oracle.conv(oracle.pack(X), rc, L.C, L.D, L.stride, L.pad)
        err = maxabs_over_rms(bf16_bits_to_f64(Y.cpu().numpy()), Yr)
        assert err <= TOL, (block, L.name, err)


def test_conv_dense_batch1():
    """The same-shape dense CONVs of AlexNet conv1-5 at batch 1 (the layers
    split their columns over workgroups and add the binary32 partial sums)."""
    wl = WORKLOADS["alexnet_shape30"]
    for li, L in enumerate(wl.layers):
        W, _ = layer_tensors(wl, li)
        got = sa.compact(to_dev(W), L.groups)
        rc = oracle.compact(W, L.groups)
        X = input_nchw(wl, li, batch=1)
        Y = sa.conv_fwd(sa.pack_nhwc(to_dev(X)), got[0], got[2], got[3], got[4], L.C, L.D, L.stride, L.pad)
        Yr = oracle.conv(oracle.pack(X), rc, L.C, L.D, L.stride, L.pad)
        err = maxabs_over_rms(bf16_bits_to_f64(Y.cpu().numpy()), Yr)
        assert err <= TOL, (L.name, err)


def test_conv_is_deterministic():
    t = torch()
    rng = np.random.default_rng(4)
    X = to_dev(rng.standard_normal((4, 64, 14, 14)).astype(np.float32))
    Z = to_dev((0.05 * rng.standard_normal((96, 64, 3, 3))).astype(np.float32))
    Wc, ri, cc, ct, sizes = sa.compact(Z, 1)
    Xp = sa.pack_nhwc(X)
    Y1 = sa.conv_fwd(Xp, Wc, cc, ct, sizes, 3, 3, 1, 1)
    Y2 = sa.conv_fwd(Xp, Wc, cc, ct, sizes, 3, 3, 1, 1)
    t.cuda.synchronize()
    assert t.equal(Y1, Y2)


def test_conv_on_a_non_current_stream():
    """Compaction, pack and CONV enqueued on a torch stream other than the
    current one, with the binding allocating the outputs and scratch: results
    equal those of the current stream, bit for bit."""
    t = torch()
    rng = np.random.default_rng(12)
    X = to_dev(rng.standard_normal((3, 3, 30, 28)).astype(np.float32))  # stem-like: space-to-depth scratch
    Z = to_dev((0.05 * rng.standard_normal((40, 3, 7, 7))).astype(np.float32))
    ref_c = sa.compact(Z, 1)
    ref = sa.conv_fwd(sa.pack_nhwc(X), ref_c[0], ref_c[2], ref_c[3], ref_c[4], 7, 7, 2, 3)
    t.cuda.synchronize()
    s = t.cuda.Stream()
    s.wait_stream(t.cuda.current_stream())
    got_c = sa.compact(Z, 1, stream=s)
    Xp = sa.pack_nhwc(X, stream=s)
    Y = sa.conv_fwd(Xp, got_c[0], got_c[2], got_c[3], got_c[4], 7, 7, 2, 3, stream=s)
    # unrelated work on the current stream may reuse freed blocks meanwhile
    junk = [t.full((1 << 20,), 7, dtype=t.uint8, device=DEV) for _ in range(4)]
    s.synchronize()
    assert t.equal(Y, ref)
    del junk


# (name, N, Cin, H, W, A, C, D, stride, pad, groups, kind, kept, what the plan must take)
PITCH_CASES = [
    ("direct_whole_rows", 32, 64, 64, 64, 64, 3, 3, 1, 1, 1, sa.FILTER, 38, "k_conv"),
    ("direct_tiles", 32, 64, 64, 64, 256, 3, 3, 1, 1, 1, sa.FILTER, 154, "k_conv"),
    ("ig_1x1", 21, 448, 56, 56, 64, 1, 1, 1, 0, 1, sa.FILTER, 38, "k_ig"),
    ("ig_3x3", 128, 48, 24, 24, 64, 3, 3, 1, 1, 1, sa.FILTER, 38, "k_ig"),
    ("footprint", 4, 64, 20, 20, 96, 3, 3, 1, 1, 1, sa.SHAPE, 173, "footprint"),
    ("space_to_depth", 2, 3, 64, 64, 64, 7, 7, 2, 3, 1, sa.FILTER, 38, "s2d"),
    ("split_k", 1, 512, 7, 7, 512, 3, 3, 1, 1, 1, sa.FILTER, 307, "split"),
    ("grouped", 4, 96, 27, 27, 256, 5, 5, 1, 2, 2, sa.FILTER, 129, None),
]


@pytest.mark.parametrize("case", PITCH_CASES, ids=[c[0] for c in PITCH_CASES])
@pytest.mark.parametrize("pitch", ["pad8", "odd"])
def test_conv_output_pitch(case, pitch):
    """Output rows ldy elements apart (ldy > Cy): every output equals, bit for
    bit, the same CONV with rows of Cy; the row padding [Cy, ldy) is left
    unchanged or +0, and nothing past the last row is written."""
    t = torch()
    name, N, Cin, H, Wd, A, C, D, stride, pad, groups, kind, kept, want = case
    rng = np.random.default_rng(len(name) * 131 + (pitch == "odd"))
    B = Cin // groups
    W = (0.05 * rng.standard_normal((A, B, C, D))).astype(np.float32)
    G = {sa.FILTER: A, sa.SHAPE: B * C * D}[kind]
    mask = np.zeros(G, np.uint8)
    mask[rng.choice(G, size=kept, replace=False)] = 1
    if kind == sa.FILTER:
        W[mask == 0] = 0
        Wc, ri, cc, ct, sizes = sa.compact(to_dev(W), groups, row_mask=to_dev(mask))
    else:
        W.reshape(A, -1)[:, mask == 0] = 0
        Wc, ri, cc, ct, sizes = sa.compact(to_dev(W), groups, col_mask=to_dev(mask))
    Xp = sa.pack_nhwc(to_dev(rng.standard_normal((N, Cin, H, Wd)).astype(np.float32)))
    plan = sa.conv_plan(Xp, sizes, C, D, stride, pad)
    paths = set(plan["path"]) - {sa.CONV_NONE}
    if want == "k_conv":
        assert paths == {sa.CONV_DIRECT} and plan["ksplit"] == 1, plan
    elif want == "k_ig":
        assert paths == {sa.CONV_DIRECT_IG}, plan
    elif want == "footprint":
        assert paths == {sa.CONV_FOOTPRINT}, plan
    elif want == "s2d":
        assert plan["space_to_depth"] > 0, plan
    elif want == "split":
        assert plan["ksplit"] > 1, plan
    Y0 = sa.conv_fwd(Xp, Wc, cc, ct, sizes, C, D, stride, pad)
    Nn, P, Q, Cy = Y0.shape
    ldy = (Cy + 8) // 8 * 8 if pitch == "pad8" else Cy + 5  # a multiple of 8 above Cy, or an odd pitch
    assert ldy > Cy
    SENT = 0x7FC1  # a bf16 NaN that no output takes
    buf = t.full((Nn * P * Q * ldy + 64,), SENT, dtype=t.int32, device=DEV).to(t.uint16)
    Y1 = buf[: Nn * P * Q * ldy].view(Nn, P, Q, ldy)
    got = sa.conv_fwd(Xp, Wc, cc, ct, sizes, C, D, stride, pad, Y=Y1, ldy=ldy)
    assert got.data_ptr() == Y1.data_ptr()
    t.cuda.synchronize()
    y0 = Y0.cpu().numpy()
    y1 = Y1.cpu().numpy()
    assert np.array_equal(y1[..., :Cy], y0), (name, pitch)
    pads = y1[..., Cy:]
    assert np.all((pads == SENT) | (pads == 0)), (name, pitch)
    assert np.all(buf[Nn * P * Q * ldy:].cpu().numpy() == SENT)
