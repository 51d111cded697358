"""CPU checks of the C ABI: the library loads, exports every symbol the
header declares, and rejects invalid arguments on the host with the
documented error codes (no GPU work is enqueued on these paths)."""
import ctypes
import os
import re

import pytest

import paper_1807_11091_amd as sa

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    names = set()
    inc = os.path.join(ROOT, "include")
    for f in os.listdir(inc):
        if f.endswith(".h"):
            text = open(os.path.join(inc, f)).read()
            text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
            names |= set(re.findall(r"\b(structadmm_\w+)\s*\(", text))
    return names


def test_library_exports_every_declared_symbol():
    names = declared_functions()
    assert {"structadmm_project", "structadmm_project_workspace", "structadmm_dual_update",
            "structadmm_compact", "structadmm_compact_many", "structadmm_conv_fwd", "structadmm_pack_nhwc",
            "structadmm_sgd_step",
            "structadmm_csr", "structadmm_conv_sparse_fwd", "structadmm_conv_sparse_workspace",
            "structadmm_last_error", "structadmm_version"} <= names
    L = sa.lib()
    for n in names:
        assert hasattr(L, n), n
    assert sa.version().startswith("structadmm-gfx950")


def _c_layout():
    """sizeof / offsetof of the header's structs as gcc lays them out."""
    import subprocess
    import tempfile
    fields = {
        "sa_project_desc": ("ProjectDesc", ["A", "groups", "kind", "k", "W", "in_ch_mask", "scores", "rho", "G"]),
        "sa_dual_desc": ("DualDesc", ["n", "W", "U", "rho", "G", "update_dual"]),
        "sa_sgd_desc": ("SgdDesc", ["A", "kind", "mask", "W", "Gf", "Z", "U", "rho", "lr"]),
        "sa_compact_desc": ("CompactDesc", ["groups", "Z", "in_compacted", "Wc", "ws"]),
        "sa_compact_sizes": ("CompactSizes", ["M", "K", "ldk", "wc_offset", "row_offset", "run", "run_base",
                                              "ch_lo", "ch_span", "kpad"]),
        "sa_conv_desc": ("ConvDesc", ["N", "pad", "sizes", "X", "Y", "ws", "ws_bytes", "ldy"]),
        "sa_conv_plan_info": ("ConvPlanInfo", ["groups", "path", "ksplit", "space_to_depth", "ig_tile",
                                               "footprint_tile"]),
        "sa_csr_desc": ("CsrDesc", ["A", "D", "nnz", "Z", "kept_idx", "row_ptr", "col", "val"]),
        "sa_sparse_conv_desc": ("SparseConvDesc", ["N", "Cx", "A", "D", "groups", "stride", "pad", "nnz", "X",
                                                   "row_ptr", "col", "val", "Y", "ws", "ws_bytes",
                                                   "reuse_ws"]),
    }
    lines = ["#include <stdio.h>", "#include <stddef.h>", '#include "structadmm.h"', "int main(void){"]
    for st, (_, fs) in fields.items():
        lines.append(f'printf("{st} sizeof %zu\\n", sizeof({st}));')
        for f in fs:
            lines.append(f'printf("{st} {f} %zu\\n", offsetof({st}, {f}));')
    lines.append("return 0;}")
    with tempfile.TemporaryDirectory() as d:
        src, exe = os.path.join(d, "l.c"), os.path.join(d, "l")
        open(src, "w").write("\n".join(lines))
        subprocess.check_call(["gcc", "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"),
                               "-I", "/opt/rocm/include", src, "-o", exe])
        out = subprocess.check_output([exe]).decode().split("\n")
    got = {}
    for line in out:
        if line.strip():
            st, f, v = line.split()
            got[(st, f)] = int(v)
    return fields, got


def test_struct_layouts_match_header():
    fields, got = _c_layout()
    for st, (py, fs) in fields.items():
        cls = getattr(sa, py)
        assert ctypes.sizeof(cls) == got[(st, "sizeof")], st
        for f in fs:
            assert getattr(cls, f).offset == got[(st, f)], (st, f)


FAKE = 0x1000  # a 256-byte aligned non-null address; never dereferenced on these paths


def pdesc(**kw):
    d = dict(A=4, B=2, C=1, D=1, groups=1, kind=sa.FILTER, k=2, W=FAKE, U=FAKE + 256, in_ch_mask=None,
             Z=FAKE + 512, mask=FAKE + 768, kept_idx=FAKE + 1024, scores=None, rho=0.0, G=None)
    d.update(kw)
    return sa.ProjectDesc(**d)


def call_project(d, ws=None, ws_bytes=0):
    arr = (sa.ProjectDesc * 1)(d)
    rc = sa.lib().structadmm_project(arr, 1, ws, ws_bytes, None)
    return rc, sa.lib().structadmm_last_error().decode()


@pytest.mark.parametrize("kw,code", [
    (dict(k=5), -1), (dict(k=-1), -1), (dict(A=0), -1), (dict(groups=3), -1), (dict(groups=0), -1),
    (dict(kind=7), -1), (dict(W=None), -1), (dict(Z=None), -1), (dict(mask=None), -1),
    (dict(kept_idx=None), -1), (dict(W=FAKE + 4), -2), (dict(G=FAKE + 8), -2), (dict(Z=FAKE), -1),
    (dict(G=FAKE + 512), -1), (dict(kind=sa.SHAPE, B=100, C=10, D=10, k=1), -4),
    (dict(A=1 << 16, B=1 << 16), -1),
])
def test_project_validation(kw, code):
    rc, msg = call_project(pdesc(**kw))
    assert rc == code, msg
    assert msg


def test_project_workspace_checks():
    # element-wise needs scratch: missing or short workspace is reported
    d = pdesc(kind=sa.ELEMENT, k=3)
    need = sa.lib().structadmm_project_workspace((sa.ProjectDesc * 1)(d), 1)
    assert need > 0
    assert call_project(d)[0] == -3
    assert call_project(d, FAKE, need - 1)[0] == -3
    assert call_project(d, FAKE + 16, need)[0] == -2
    # invalid descriptors report a zero size
    assert sa.lib().structadmm_project_workspace((sa.ProjectDesc * 1)(pdesc(k=9)), 1) == 0
    # filter-wise without exported scores needs room for them
    assert sa.lib().structadmm_project_workspace((sa.ProjectDesc * 1)(pdesc()), 1) >= 4 * 8


def test_dual_validation():
    L = sa.lib()
    def call(**kw):
        d = dict(n=8, W=FAKE, Z=FAKE + 256, U=FAKE + 512, rho=1.0, G=FAKE + 768, update_dual=1)
        d.update(kw)
        return L.structadmm_dual_update((sa.DualDesc * 1)(sa.DualDesc(**d)), 1, None)
    assert call(n=0) == -1
    assert call(U=None) == -1
    assert call(update_dual=0, G=None) == -1
    assert call(Z=FAKE + 4) == -2
    assert L.structadmm_dual_update(None, 1, None) == -1


def test_sgd_validation():
    L = sa.lib()
    def call(**kw):
        d = dict(A=4, B=2, C=3, D=3, kind=sa.FILTER, mask=None, W=FAKE, Gf=FAKE + 256, Z=None, U=None,
                 rho=0.1, lr=0.01)
        d.update(kw)
        return L.structadmm_sgd_step((sa.SgdDesc * 1)(sa.SgdDesc(**d)), 1, None)
    assert call(A=0) == -1
    assert call(kind=9) == -1
    assert call(W=None) == -1
    assert call(Gf=None) == -1
    assert call(Z=FAKE + 512) == -1          # Z without U
    assert call(Gf=FAKE) == -1               # Gf aliases W
    assert call(W=FAKE + 4) == -2
    assert call(Z=FAKE + 512, U=FAKE + 1024 + 8) == -2
    assert call(A=1 << 16, B=1 << 16) == -1
    assert L.structadmm_sgd_step(None, 1, None) == -1


def test_compact_and_conv_validation():
    L = sa.lib()
    def comp(**kw):
        d = dict(A=4, B=2, C=3, D=3, groups=1, Z=FAKE, row_mask=None, col_mask=None, chan_mask=None,
                 in_ch_mask=None, in_compacted=0, Wc=FAKE + 256, row_idx=FAKE + 512, col_ch=FAKE + 768,
                 col_tap=FAKE + 1024, ws=FAKE + 2048)
        d.update(kw)
        s = sa.CompactSizes()
        return L.structadmm_compact(ctypes.byref(sa.CompactDesc(**d)), ctypes.byref(s), None)
    assert comp(groups=3) == -1
    assert comp(groups=32, A=32) == -1
    assert comp(in_compacted=1) == -1
    assert comp(ws=None) == -1
    assert comp(Wc=FAKE + 8) == -2
    assert comp(C=300) == -4

    # the batched form checks every descriptor (and that no two share
    # scratch) before it enqueues anything: these calls do no GPU work
    def many(*descs, n=None):
        arr = (sa.CompactDesc * max(1, len(descs)))()
        for i, kw in enumerate(descs):
            d = dict(A=4, B=2, C=3, D=3, groups=1, Z=FAKE, row_mask=None, col_mask=None, chan_mask=None,
                     in_ch_mask=None, in_compacted=0, Wc=FAKE + 256, row_idx=FAKE + 512, col_ch=FAKE + 768,
                     col_tap=FAKE + 1024, ws=FAKE + 8192 * (i + 1))
            d.update(kw)
            arr[i] = sa.CompactDesc(**d)
        out = (sa.CompactSizes * max(1, len(descs)))()
        return L.structadmm_compact_many(arr, len(descs) if n is None else n, out, None)
    assert many() == 0
    assert many({}, n=-1) == -1
    assert many({}, {"ws": FAKE + 8192 + 256}) == -1  # scratch ranges overlap
    assert many({}, {"groups": 3}) == -1
    assert many({}, {"Wc": FAKE + 8}) == -2
    assert L.structadmm_compact_many(None, 1, None, None) == -1

    s = sa.CompactSizes()
    s.groups = 1
    s.M[0], s.K[0], s.ldk[0] = 4, 18, 64
    def conv(**kw):
        d = dict(N=1, H=8, W=8, Cx=2, C=3, D=3, stride=1, pad=1, sizes=ctypes.pointer(s), X=FAKE,
                 Wc=FAKE + 256, col_ch=FAKE + 512, col_tap=FAKE + 768, Y=FAKE + 1024)
        d.update(kw)
        return L.structadmm_conv_fwd(ctypes.byref(sa.ConvDesc(**d)), None)
    assert conv(sizes=None) == -1
    assert conv(H=1, pad=0) == -1
    assert conv(stride=0) == -1
    assert conv(X=FAKE + 2) == -2
    assert conv(C=256, H=300) == -4
    s.run[0] = 5  # 5 * 9 != 18
    assert conv() == -1
    s.run[0] = 0
    s.ldk[0] = 18  # not the padded stride that compaction produces
    assert conv() == -1
    # arbitrary columns over 8-aligned channels are gathered from an LDS copy of
    # each tile's input footprint: no scratch
    s.ldk[0] = 64
    s.ch_lo[0], s.ch_span[0] = 0, 2
    desc = lambda **kw: sa.ConvDesc(**{**dict(N=1, H=8, W=8, Cx=2, C=3, D=3, stride=1, pad=1,
                                             sizes=ctypes.pointer(s), X=FAKE, Wc=FAKE, col_ch=FAKE,
                                             col_tap=FAKE, Y=FAKE, ws=None, ws_bytes=0), **kw})
    assert L.structadmm_conv_workspace(ctypes.byref(desc(Cx=8))) == 0
    # channels not 8-aligned: the input's space-to-depth image (here stride 1: the
    # zero border folded in, 2 channels padded to 8) goes to caller scratch, then
    # the 4 kept rows rewritten over the image's taps x channels (3x3 taps of 8
    # channels = 72 columns, rows of 128)
    need = L.structadmm_conv_workspace(ctypes.byref(desc()))
    assert need == (10 * 10 * 8 * 2 + 255) // 256 * 256 + 4 * 128 * 2
    s2 = L.structadmm_conv_workspace(ctypes.byref(desc(stride=2)))
    # 2x2 blocks of 2 channels: 8 channels; 2x2 taps of them: 32 columns, rows of 64
    assert s2 == (5 * 5 * 8 * 2 + 255) // 256 * 256 + 4 * 64 * 2
    assert conv() == -3
    assert conv(ws=FAKE + 2048, ws_bytes=need - 1) == -3
    assert conv(ws=FAKE + 2048 + 16, ws_bytes=need) == -2
    s.ch_span[0] = 3  # channels past the input
    assert conv(ws=FAKE + 2048, ws_bytes=need) == -1
    assert L.structadmm_conv_workspace(ctypes.byref(desc())) == 0
    # so do footprints too wide for LDS
    s.ch_span[0] = 16
    wide = dict(W=4000, Cx=16)
    assert L.structadmm_conv_workspace(ctypes.byref(desc(**wide))) == 8 * 4000 * 64 * 2


def test_conv_plan_host_only():
    """structadmm_conv_plan on the host (no device pointer is read): the
    kernel each kind of layer takes, and the descriptor checks."""
    L = sa.lib()
    s = sa.CompactSizes()
    s.groups = 1

    def plan(N, H, W, Cx, C, D, stride, pad, M, run=None, cols=None):
        K = C * D * (Cx if run is None else run) if cols is None else cols
        s.M[0], s.K[0], s.ldk[0] = M, K, (K + 63) // 64 * 64
        s.run[0], s.run_base[0] = (0, 0) if run is None else (run, 0)
        s.ch_lo[0], s.ch_span[0] = 0, Cx
        d = sa.ConvDesc(N, H, W, Cx, C, D, stride, pad, ctypes.pointer(s), FAKE, FAKE, FAKE, FAKE, FAKE, None, 0)
        info = sa.ConvPlanInfo()
        rc = L.structadmm_conv_plan(ctypes.byref(d), ctypes.byref(info))
        return rc, info

    # 38 kept filters of a 1x1 layer over 448 channels, 56x56 at batch 64: the
    # 16-row kernel (64-filter tiles would pad the filter work by a third)
    rc, info = plan(64, 56, 56, 448, 1, 1, 1, 0, 38, run=448)
    assert rc == 0 and list(info.path)[:1] == [sa.CONV_DIRECT_IG] and info.ksplit == 1
    assert tuple(info.ig_tile) == (3, 2, 1, 1)
    # 77 over 256 channels: the LDS-staged kernel
    rc, info = plan(64, 56, 56, 256, 1, 1, 1, 0, 77, run=256)
    assert rc == 0 and list(info.path)[:1] == [sa.CONV_DIRECT]
    # 38 of 64 over 64 channels: the 128 x 64 tiles of the LDS-staged kernel
    rc, info = plan(64, 56, 56, 64, 1, 1, 1, 0, 38, run=64)
    assert rc == 0 and list(info.path)[:1] == [sa.CONV_DIRECT]
    # 77 over 512 channels at 28x28: the LDS-staged kernel again
    rc, info = plan(64, 28, 28, 512, 1, 1, 1, 0, 77, run=512)
    assert rc == 0 and list(info.path)[:1] == [sa.CONV_DIRECT]
    # 512 filters of a 3x3 layer at 7x7, batch 64: 128 x 64 tiles fill the
    # GPU without splitting the columns
    rc, info = plan(64, 7, 7, 512, 3, 3, 1, 1, 512, run=512)
    assert rc == 0 and list(info.path)[:1] == [sa.CONV_DIRECT] and info.ksplit == 1
    # every filter of a 3x3 layer: the LDS-staged kernel
    rc, info = plan(64, 28, 28, 128, 3, 3, 1, 1, 128, run=128)
    assert rc == 0 and list(info.path)[:1] == [sa.CONV_DIRECT]
    # batch 1: split over the columns
    rc, info = plan(1, 13, 13, 256, 3, 3, 1, 1, 384, run=256)
    assert rc == 0 and info.ksplit > 1
    # 3 input channels: the space-to-depth image, then the direct kernels over
    # its taps x channels
    rc, info = plan(2, 30, 28, 3, 7, 7, 2, 3, 12, cols=147)
    assert rc == 0 and list(info.path)[:1] in ([sa.CONV_DIRECT], [sa.CONV_DIRECT_IG]) and info.space_to_depth == 2
    # the same image under two conv groups: the footprint kernel
    s.groups = 2
    s.M[1], s.K[1], s.ldk[1], s.run[1], s.run_base[1], s.ch_lo[1], s.ch_span[1] = 12, 49, 64, 0, 0, 2, 1
    s.wc_offset[1], s.row_offset[1], s.col_offset[1] = 12 * 64, 12, 49
    d = sa.ConvDesc(2, 30, 28, 3, 7, 7, 2, 3, ctypes.pointer(s), FAKE, FAKE, FAKE, FAKE, FAKE, None, 0)
    s.M[0], s.K[0], s.ldk[0], s.run[0], s.ch_lo[0], s.ch_span[0] = 12, 98, 128, 0, 0, 2
    info = sa.ConvPlanInfo()
    assert L.structadmm_conv_plan(ctypes.byref(d), ctypes.byref(info)) == 0
    assert list(info.path)[:2] == [sa.CONV_FOOTPRINT] * 2 and info.space_to_depth == 2
    s.groups = 1
    # arbitrary columns over 8-aligned channels: the footprint kernel
    rc, info = plan(8, 13, 13, 64, 3, 3, 1, 1, 48, cols=100)
    assert rc == 0 and list(info.path)[:1] == [sa.CONV_FOOTPRINT] and info.space_to_depth == 0
    d = sa.ConvDesc(1, 8, 8, 8, 3, 3, 0, 1, ctypes.pointer(s), FAKE, FAKE, FAKE, FAKE, FAKE, None, 0)
    assert L.structadmm_conv_plan(ctypes.byref(d), ctypes.byref(sa.ConvPlanInfo())) == -1  # stride 0
    assert L.structadmm_conv_plan(ctypes.byref(d), None) == -1


def test_csr_validation():
    L = sa.lib()
    def call(**kw):
        d = dict(A=4, B=2, C=3, D=3, nnz=5, Z=FAKE, kept_idx=FAKE + 256, row_ptr=FAKE + 512, col=FAKE + 768,
                 val=FAKE + 1024)
        d.update(kw)
        return L.structadmm_csr(ctypes.byref(sa.CsrDesc(**d)), None)
    assert call(A=0) == -1
    assert call(nnz=-1) == -1
    assert call(nnz=4 * 18 + 1) == -1
    assert call(Z=None) == -1
    assert call(row_ptr=None) == -1
    assert call(kept_idx=None) == -1
    assert call(col=FAKE + 2) == -2
    assert call(A=1 << 16, B=1 << 16) == -4
    assert L.structadmm_csr(None, None) == -1


def test_conv_sparse_validation():
    L = sa.lib()
    def desc(**kw):
        d = dict(N=2, H=14, W=14, Cx=256, A=256, B=256, C=3, D=3, groups=1, stride=1, pad=1, nnz=1000,
                 X=FAKE, row_ptr=FAKE + 256, col=FAKE + 512, val=FAKE + 768, Y=FAKE + 1024, ws=FAKE + 2048,
                 ws_bytes=1 << 30)
        d.update(kw)
        return sa.SparseConvDesc(**d)
    def call(**kw):
        return L.structadmm_conv_sparse_fwd(ctypes.byref(desc(**kw)), None)
    ws = lambda **kw: L.structadmm_conv_sparse_workspace(ctypes.byref(desc(**kw)))
    # padded row pointers, offsets and values: (A+1)*4, (nnz + 7A rounded to 8)*4, *2, each 256-aligned
    cap = (1000 + 7 * 256 + 7) // 8 * 8
    r = lambda x: (x + 255) // 256 * 256
    assert ws() == r(257 * 4) + r(cap * 4) + r(cap * 2)
    assert call(groups=3) == -1                 # A % groups, Cx != groups * B
    assert call(Cx=128) == -1
    assert call(nnz=256 * 2304 + 1) == -1
    assert call(stride=0) == -1
    assert call(H=1, pad=0) == -1               # empty output
    assert call(Cx=12, B=12) == -4              # channels not a multiple of 8
    assert call(H=1000, W=1000) == -4           # footprint of 64 pixels exceeds LDS
    assert call(X=FAKE + 2) == -2
    assert call(Y=FAKE + 1024 + 8) == -2
    assert call(ws=None) == -3
    assert call(ws_bytes=ws() - 1) == -3
    assert call(ws=FAKE + 2048 + 16) == -2
    assert call(col=None) == -1
    assert ws(Cx=12, B=12) == 0
    assert L.structadmm_conv_sparse_fwd(None, None) == -1


def test_pack_validation():
    L = sa.lib()
    assert L.structadmm_pack_nhwc(None, 1, 3, 4, 4, None, 3, FAKE, None) == -1
    assert L.structadmm_pack_nhwc(FAKE, 1, 3, 4, 4, None, 2, FAKE, None) == -1
    assert L.structadmm_pack_nhwc(FAKE, 1, 3, 4, 4, None, 4, FAKE, None) == -1


def test_product_path_has_no_oracle_dependency():
    """The GPU package neither imports nor links the oracle."""
    pkg = os.path.join(ROOT, "paper_1807_11091_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".cpp", ".h")):
                text = open(os.path.join(dirpath, f)).read()
                assert "import oracle" not in text and "from oracle" not in text, f
                assert "oracle.h" not in text and "liboracle" not in text, f
