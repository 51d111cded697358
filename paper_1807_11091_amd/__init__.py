"""Python binding of libstructadmm (gfx950): the StructADMM hot path.

Thin ctypes marshalling over the C ABI in ``include/structadmm.h``: every
step runs in the library's HIP kernels; torch is used only for device memory
(tensor allocation) and streams.  There is no fallback: if the library is
missing or a call fails, an exception is raised.

Entry points (same names as the C ABI):
  project(layers, ws=None, stream=None)
  project_workspace(layers)
  dual_update(layers, stream=None)
  sgd_step(items, stream=None)
  compact(Z, groups, ..., ws=None, stream=None) -> (Wc, row_idx, col_ch, col_tap, sizes)
  pack_nhwc(X, keep=None, Cx=None, stream=None)
  conv_fwd(X, Wc, col_ch, col_tap, sizes, C, D, stride, pad, Y=None, stream=None, ldy=None)
  csr(Z, kept_idx, row_ptr=None, col=None, val=None, stream=None) -> (row_ptr, col, val)
  conv_sparse_workspace(Xp, shape, groups, stride, pad, nnz)
  conv_sparse_fwd(Xp, row_ptr, col, val, shape, groups, stride, pad, Y=None, ws=None, stream=None)
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import List, Optional, Sequence

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libstructadmm.so")

FILTER, CHANNEL, SHAPE, ELEMENT = 0, 1, 2, 3
MAX_CONV_GROUPS = 16
MAX_STRUCT_GROUPS = 8192
COMPACT_WS_BYTES = 4096
ERRORS = {-1: "SA_E_ARG", -2: "SA_E_ALIGN", -3: "SA_E_WORKSPACE", -4: "SA_E_UNSUPPORTED", -5: "SA_E_HIP"}

_vp = ctypes.c_void_p


class ProjectDesc(ctypes.Structure):
    _fields_ = [("A", ctypes.c_int64), ("B", ctypes.c_int64), ("C", ctypes.c_int64), ("D", ctypes.c_int64),
                ("groups", ctypes.c_int32), ("kind", ctypes.c_int32), ("k", ctypes.c_int64),
                ("W", _vp), ("U", _vp), ("in_ch_mask", _vp), ("Z", _vp), ("mask", _vp),
                ("kept_idx", _vp), ("scores", _vp), ("rho", ctypes.c_float), ("G", _vp)]


class DualDesc(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int64), ("W", _vp), ("Z", _vp), ("U", _vp), ("rho", ctypes.c_float),
                ("G", _vp), ("update_dual", ctypes.c_int32)]


class SgdDesc(ctypes.Structure):
    _fields_ = [("A", ctypes.c_int64), ("B", ctypes.c_int64), ("C", ctypes.c_int64), ("D", ctypes.c_int64),
                ("kind", ctypes.c_int32), ("mask", _vp), ("W", _vp), ("Gf", _vp), ("Z", _vp), ("U", _vp),
                ("rho", ctypes.c_float), ("lr", ctypes.c_float)]


class CompactDesc(ctypes.Structure):
    _fields_ = [("A", ctypes.c_int64), ("B", ctypes.c_int64), ("C", ctypes.c_int64), ("D", ctypes.c_int64),
                ("groups", ctypes.c_int32), ("Z", _vp), ("row_mask", _vp), ("col_mask", _vp),
                ("chan_mask", _vp), ("in_ch_mask", _vp), ("in_compacted", ctypes.c_int32),
                ("Wc", _vp), ("row_idx", _vp), ("col_ch", _vp), ("col_tap", _vp), ("ws", _vp)]


_G = MAX_CONV_GROUPS


class CompactSizes(ctypes.Structure):
    _fields_ = [("groups", ctypes.c_int32), ("M", ctypes.c_int32 * _G), ("K", ctypes.c_int32 * _G),
                ("ldk", ctypes.c_int32 * _G), ("wc_offset", ctypes.c_int64 * _G),
                ("row_offset", ctypes.c_int32 * _G), ("col_offset", ctypes.c_int32 * _G),
                ("run", ctypes.c_int32 * _G), ("run_base", ctypes.c_int32 * _G),
                ("ch_lo", ctypes.c_int32 * _G), ("ch_span", ctypes.c_int32 * _G),
                ("kpad", ctypes.c_int32 * _G)]

    def as_dict(self):
        g = self.groups
        return {k: list(getattr(self, k))[:g] for k in
                ("M", "K", "ldk", "wc_offset", "row_offset", "col_offset", "run", "run_base",
                 "ch_lo", "ch_span", "kpad")}


class ConvDesc(ctypes.Structure):
    _fields_ = [("N", ctypes.c_int32), ("H", ctypes.c_int32), ("W", ctypes.c_int32), ("Cx", ctypes.c_int32),
                ("C", ctypes.c_int32), ("D", ctypes.c_int32), ("stride", ctypes.c_int32), ("pad", ctypes.c_int32),
                ("sizes", ctypes.POINTER(CompactSizes)), ("X", _vp), ("Wc", _vp), ("col_ch", _vp),
                ("col_tap", _vp), ("Y", _vp), ("ws", _vp), ("ws_bytes", ctypes.c_size_t),
                ("ldy", ctypes.c_int32)]


class ConvPlanInfo(ctypes.Structure):
    _fields_ = [("groups", ctypes.c_int32), ("path", ctypes.c_int32 * _G), ("ksplit", ctypes.c_int32),
                ("space_to_depth", ctypes.c_int32), ("ig_tile", ctypes.c_int32 * 4),
                ("footprint_tile", ctypes.c_int32 * 3)]


# kernel paths of structadmm_conv_plan
CONV_NONE, CONV_DIRECT, CONV_DIRECT_IG, CONV_FOOTPRINT, CONV_GATHER = 0, 1, 2, 3, 4


class CsrDesc(ctypes.Structure):
    _fields_ = [("A", ctypes.c_int64), ("B", ctypes.c_int64), ("C", ctypes.c_int64), ("D", ctypes.c_int64),
                ("nnz", ctypes.c_int64), ("Z", _vp), ("kept_idx", _vp), ("row_ptr", _vp), ("col", _vp),
                ("val", _vp)]


class SparseConvDesc(ctypes.Structure):
    _fields_ = [("N", ctypes.c_int32), ("H", ctypes.c_int32), ("W", ctypes.c_int32), ("Cx", ctypes.c_int32),
                ("A", ctypes.c_int32), ("B", ctypes.c_int32), ("C", ctypes.c_int32), ("D", ctypes.c_int32),
                ("groups", ctypes.c_int32), ("stride", ctypes.c_int32), ("pad", ctypes.c_int32),
                ("nnz", ctypes.c_int64), ("X", _vp), ("row_ptr", _vp), ("col", _vp), ("val", _vp),
                ("Y", _vp), ("ws", _vp), ("ws_bytes", ctypes.c_size_t), ("reuse_ws", ctypes.c_int32)]


class StructAdmmError(RuntimeError):
    pass


_lib = None


def lib():
    """Loads libstructadmm.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise StructAdmmError(f"{LIB_PATH} is missing: build it with paper_1807_11091_amd/build.py")
        L = ctypes.CDLL(LIB_PATH)
        L.structadmm_project_workspace.argtypes = [ctypes.POINTER(ProjectDesc), ctypes.c_int]
        L.structadmm_project_workspace.restype = ctypes.c_size_t
        L.structadmm_project.argtypes = [ctypes.POINTER(ProjectDesc), ctypes.c_int, _vp, ctypes.c_size_t, _vp]
        L.structadmm_project.restype = ctypes.c_int
        L.structadmm_project_noalloc.argtypes = [ctypes.POINTER(ProjectDesc), ctypes.c_int, _vp]
        L.structadmm_project_noalloc.restype = ctypes.c_int
        L.structadmm_dual_update.argtypes = [ctypes.POINTER(DualDesc), ctypes.c_int, _vp]
        L.structadmm_dual_update.restype = ctypes.c_int
        L.structadmm_sgd_step.argtypes = [ctypes.POINTER(SgdDesc), ctypes.c_int, _vp]
        L.structadmm_sgd_step.restype = ctypes.c_int
        L.structadmm_compact.argtypes = [ctypes.POINTER(CompactDesc), ctypes.POINTER(CompactSizes), _vp]
        L.structadmm_compact.restype = ctypes.c_int
        L.structadmm_compact_many.argtypes = [ctypes.POINTER(CompactDesc), ctypes.c_int32,
                                              ctypes.POINTER(CompactSizes), _vp]
        L.structadmm_compact_many.restype = ctypes.c_int
        L.structadmm_pack_nhwc.argtypes = [_vp, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                           _vp, ctypes.c_int32, _vp, _vp]
        L.structadmm_pack_nhwc.restype = ctypes.c_int
        L.structadmm_conv_fwd.argtypes = [ctypes.POINTER(ConvDesc), _vp]
        L.structadmm_conv_fwd.restype = ctypes.c_int
        L.structadmm_conv_plan.argtypes = [ctypes.POINTER(ConvDesc), ctypes.POINTER(ConvPlanInfo)]
        L.structadmm_conv_plan.restype = ctypes.c_int
        L.structadmm_conv_workspace.argtypes = [ctypes.POINTER(ConvDesc)]
        L.structadmm_conv_workspace.restype = ctypes.c_size_t
        L.structadmm_csr.argtypes = [ctypes.POINTER(CsrDesc), _vp]
        L.structadmm_csr.restype = ctypes.c_int
        L.structadmm_conv_sparse_workspace.argtypes = [ctypes.POINTER(SparseConvDesc)]
        L.structadmm_conv_sparse_workspace.restype = ctypes.c_size_t
        L.structadmm_conv_sparse_fwd.argtypes = [ctypes.POINTER(SparseConvDesc), _vp]
        L.structadmm_conv_sparse_fwd.restype = ctypes.c_int
        L.structadmm_last_error.argtypes = []
        L.structadmm_last_error.restype = ctypes.c_char_p
        L.structadmm_version.argtypes = []
        L.structadmm_version.restype = ctypes.c_char_p
        _lib = L
    return _lib


def _check(rc: int, what: str):
    if rc != 0:
        msg = lib().structadmm_last_error().decode(errors="replace")
        raise StructAdmmError(f"{what} failed: {ERRORS.get(rc, rc)} ({rc}): {msg}")


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    return stream if isinstance(stream, int) else stream.cuda_stream


def _keep_for_stream(stream, *tensors):
    """Temporaries this module allocates come from torch's caching allocator on
    the current stream; when the launch goes to another torch stream, mark them
    in use there, so their memory is not handed out again before that stream's
    work has finished (a raw stream handle gets no such tracking: the caller
    must keep such calls on the current stream or pass its own buffers)."""
    if stream is None or isinstance(stream, int):
        return
    for t in tensors:
        if t is not None:
            t.record_stream(stream)


@dataclass
class ProjectLayer:
    """One layer of a projection call: tensors are torch device tensors."""
    W: "object"
    U: "object"
    Z: "object"
    mask: "object"
    kept_idx: "object"
    kind: int
    k: int
    groups: int = 1
    in_ch_mask: "object" = None
    scores: "object" = None
    rho: float = 0.0
    G: "object" = None

    def desc(self) -> ProjectDesc:
        A, B, C, D = self.W.shape
        return ProjectDesc(A, B, C, D, self.groups, self.kind, self.k, _ptr(self.W), _ptr(self.U),
                           _ptr(self.in_ch_mask), _ptr(self.Z), _ptr(self.mask), _ptr(self.kept_idx),
                           _ptr(self.scores), self.rho, _ptr(self.G))


def _descs(layers: Sequence[ProjectLayer]):
    arr = (ProjectDesc * len(layers))()
    for i, l in enumerate(layers):
        arr[i] = l.desc()
    return arr


def project_workspace(layers: Sequence[ProjectLayer]) -> int:
    return int(lib().structadmm_project_workspace(_descs(layers), len(layers)))


def project(layers: Sequence[ProjectLayer], ws=None, stream=None, descs=None):
    """structadmm_project over the layers; ``ws`` is a uint8 device tensor."""
    d = descs if descs is not None else _descs(layers)
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check(lib().structadmm_project(d, len(layers), _ptr(ws), nbytes, _stream(stream)), "structadmm_project")


# scratch the library holds per GPU for project_noalloc (bytes)
PROJECT_NOALLOC_BYTES = 16 << 20


def project_noalloc(layers: Sequence[ProjectLayer], stream=None, descs=None):
    """structadmm_project_noalloc: the projection with no workspace argument
    and no device allocation (the library's fixed per-GPU scratch)."""
    d = descs if descs is not None else _descs(layers)
    _check(lib().structadmm_project_noalloc(d, len(d), _stream(stream)), "structadmm_project_noalloc")


def dual_descs(items) -> "ctypes.Array":
    """items: iterable of (W, Z, U, rho, G, update_dual)."""
    items = list(items)
    arr = (DualDesc * len(items))()
    for i, (W, Z, U, rho, G, upd) in enumerate(items):
        arr[i] = DualDesc(W.numel(), _ptr(W), _ptr(Z), _ptr(U), rho, _ptr(G), 1 if upd else 0)
    return arr


def dual_update(items, stream=None, descs=None):
    d = descs if descs is not None else dual_descs(items)
    _check(lib().structadmm_dual_update(d, len(d), _stream(stream)), "structadmm_dual_update")


def sgd_descs(items) -> "ctypes.Array":
    """items: iterable of (W, Gf, Z, U, mask, kind, rho, lr); W is [A,B,C,D];
    Z, U and mask may be None."""
    items = list(items)
    arr = (SgdDesc * len(items))()
    for i, (W, Gf, Z, U, mask, kind, rho, lr) in enumerate(items):
        A, B, C, D = W.shape
        arr[i] = SgdDesc(A, B, C, D, kind, _ptr(mask), _ptr(W), _ptr(Gf), _ptr(Z), _ptr(U), rho, lr)
    return arr


def sgd_step(items, stream=None, descs=None):
    """structadmm_sgd_step: W <- keep ? W - lr * (Gf + rho((W - Z) + U)) : 0, in place."""
    d = descs if descs is not None else sgd_descs(items)
    _check(lib().structadmm_sgd_step(d, len(d), _stream(stream)), "structadmm_sgd_step")


def compact(Z, groups: int = 1, row_mask=None, col_mask=None, chan_mask=None, in_ch_mask=None,
            in_compacted: bool = False, ws=None, stream=None, out=None):
    """structadmm_compact; returns (Wc, row_idx, col_ch, col_tap, sizes)."""
    import torch
    A, B, C, D = Z.shape
    dev = Z.device
    K = B * C * D
    if out is None:
        Wc = torch.empty(A * ((K + 63) // 64 * 64), dtype=torch.uint16, device=dev)
        row_idx = torch.empty(A, dtype=torch.int32, device=dev)
        col_ch = torch.empty(groups * K, dtype=torch.int32, device=dev)
        col_tap = torch.empty(groups * K, dtype=torch.int32, device=dev)
    else:
        Wc, row_idx, col_ch, col_tap = out
    if ws is None:
        ws = torch.empty(COMPACT_WS_BYTES, dtype=torch.uint8, device=dev)
    desc = CompactDesc(A, B, C, D, groups, _ptr(Z), _ptr(row_mask), _ptr(col_mask), _ptr(chan_mask),
                       _ptr(in_ch_mask), 1 if in_compacted else 0, _ptr(Wc), _ptr(row_idx), _ptr(col_ch),
                       _ptr(col_tap), _ptr(ws))
    sizes = CompactSizes()
    _check(lib().structadmm_compact(ctypes.byref(desc), ctypes.byref(sizes), _stream(stream)), "structadmm_compact")
    _keep_for_stream(stream, ws, *(() if out is not None else (Wc, row_idx, col_ch, col_tap)))
    return Wc, row_idx, col_ch, col_tap, sizes


def compact_many(items, ws=None, stream=None):
    """structadmm_compact_many: one call (one wait of the host) for many
    compactions.  items: dicts of compact()'s arguments (Z, groups, row_mask,
    col_mask, chan_mask, in_ch_mask, in_compacted, out); ws: uint8 scratch of
    len(items) * COMPACT_WS_BYTES (allocated here when None).  Returns the
    list of (Wc, row_idx, col_ch, col_tap, sizes), one per item."""
    import torch
    n = len(items)
    if n == 0:
        return []
    dev = items[0]["Z"].device
    if ws is None:
        ws = torch.empty(n * COMPACT_WS_BYTES, dtype=torch.uint8, device=dev)
    elif ws.numel() * ws.element_size() < n * COMPACT_WS_BYTES:
        raise StructAdmmError(f"compact_many: ws must hold {n} x {COMPACT_WS_BYTES} bytes")
    descs = (CompactDesc * n)()
    sizes = (CompactSizes * n)()
    outs, made = [], []
    for i, it in enumerate(items):
        Z = it["Z"]
        A, B, C, D = Z.shape
        groups = it.get("groups", 1)
        K = B * C * D
        if it.get("out") is None:
            o = (torch.empty(A * ((K + 63) // 64 * 64), dtype=torch.uint16, device=dev),
                 torch.empty(A, dtype=torch.int32, device=dev),
                 torch.empty(groups * K, dtype=torch.int32, device=dev),
                 torch.empty(groups * K, dtype=torch.int32, device=dev))
            made.extend(o)
        else:
            o = tuple(it["out"])
        outs.append(o)
        descs[i] = CompactDesc(A, B, C, D, groups, _ptr(Z), _ptr(it.get("row_mask")), _ptr(it.get("col_mask")),
                               _ptr(it.get("chan_mask")), _ptr(it.get("in_ch_mask")),
                               1 if it.get("in_compacted") else 0, _ptr(o[0]), _ptr(o[1]), _ptr(o[2]), _ptr(o[3]),
                               ws.data_ptr() + i * COMPACT_WS_BYTES)
    _check(lib().structadmm_compact_many(descs, n, sizes, _stream(stream)), "structadmm_compact_many")
    _keep_for_stream(stream, ws, *made)
    return [outs[i] + (CompactSizes.from_buffer_copy(sizes[i]),) for i in range(n)]


def pack_nhwc(X, keep=None, Cx: Optional[int] = None, out=None, stream=None):
    """fp32 NCHW -> bf16 NHWC (uint16 bits) with an optional channel keep mask."""
    import torch
    N, Cin, H, W = X.shape
    if Cx is None:
        Cx = Cin if keep is None else int(keep.count_nonzero().item())
    Xp = out if out is not None else torch.empty((N, H, W, Cx), dtype=torch.uint16, device=X.device)
    _check(lib().structadmm_pack_nhwc(_ptr(X), N, Cin, H, W, _ptr(keep), Cx, _ptr(Xp), _stream(stream)),
           "structadmm_pack_nhwc")
    if out is None:
        _keep_for_stream(stream, Xp)
    return Xp


def conv_out_shape(N, H, W, C, D, stride, pad, sizes: CompactSizes):
    P = (H + 2 * pad - C) // stride + 1
    Q = (W + 2 * pad - D) // stride + 1
    return (N, P, Q, int(sum(sizes.M[g] for g in range(sizes.groups))))


def conv_desc(Xp, Wc, col_ch, col_tap, sizes: CompactSizes, C, D, stride, pad, Y, ws=None, ldy=0) -> ConvDesc:
    N, H, W, Cx = Xp.shape
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    return ConvDesc(N, H, W, Cx, C, D, stride, pad, ctypes.pointer(sizes), _ptr(Xp), _ptr(Wc),
                    _ptr(col_ch), _ptr(col_tap), _ptr(Y), _ptr(ws), nbytes, ldy)


def conv_workspace(Xp, sizes: CompactSizes, C: int, D: int, stride: int, pad: int) -> int:
    """Scratch bytes structadmm_conv_fwd needs for this input and compaction."""
    N, H, W, Cx = Xp.shape
    d = ConvDesc(N, H, W, Cx, C, D, stride, pad, ctypes.pointer(sizes), 16, 16, 16, 16, 16, None, 0)
    return int(lib().structadmm_conv_workspace(ctypes.byref(d)))


def conv_plan(Xp, sizes: CompactSizes, C: int, D: int, stride: int, pad: int) -> dict:
    """structadmm_conv_plan: the kernels structadmm_conv_fwd takes (host only)."""
    N, H, W, Cx = Xp.shape if not isinstance(Xp, tuple) else Xp
    d = ConvDesc(N, H, W, Cx, C, D, stride, pad, ctypes.pointer(sizes), 16, 16, 16, 16, 16, None, 0)
    info = ConvPlanInfo()
    _check(lib().structadmm_conv_plan(ctypes.byref(d), ctypes.byref(info)), "structadmm_conv_plan")
    g = info.groups
    return {"path": list(info.path)[:g], "ksplit": info.ksplit, "space_to_depth": info.space_to_depth,
            "ig_tile": tuple(info.ig_tile), "footprint_tile": tuple(info.footprint_tile)}


def conv_fwd(Xp, Wc, col_ch, col_tap, sizes: CompactSizes, C: int, D: int, stride: int, pad: int,
             Y=None, ws=None, stream=None, desc: Optional[ConvDesc] = None, ldy: Optional[int] = None):
    """structadmm_conv_fwd; Xp bf16 NHWC (uint16), returns Y bf16 NHWC (uint16).
    ``ws``: uint8 device scratch of conv_workspace() bytes (allocated here when None).
    ``ldy``: output row pitch in elements (>= the output channels Cy); by default
    the last dimension of a given 4-d Y, else Cy.  Y is then [N, P, Q, ldy] whose
    channels [Cy, ldy) are padding (left unchanged or set to +0)."""
    import torch
    temps = []
    if desc is None:
        N, H, W, Cx = Xp.shape
        shape = conv_out_shape(N, H, W, C, D, stride, pad, sizes)
        Cy = shape[-1]
        if ldy is None:
            ldy = Y.shape[-1] if (Y is not None and Y.dim() == 4) else Cy
        if ldy < Cy:
            raise StructAdmmError(f"conv_fwd: ldy={ldy} is below the {Cy} output channels")
        if Y is None:
            Y = torch.empty(shape[:3] + (ldy,), dtype=torch.uint16, device=Xp.device)
            temps.append(Y)
        elif Y.numel() < shape[0] * shape[1] * shape[2] * ldy or Y.dtype != torch.uint16:
            raise StructAdmmError(f"conv_fwd: Y must be uint16 with room for {shape[:3]} rows of {ldy}")
        if ws is None:
            need = conv_workspace(Xp, sizes, C, D, stride, pad)
            ws = torch.empty(need, dtype=torch.uint8, device=Xp.device) if need else None
            temps.append(ws)
        desc = conv_desc(Xp, Wc, col_ch, col_tap, sizes, C, D, stride, pad, Y, ws, 0 if ldy == Cy else ldy)
    _check(lib().structadmm_conv_fwd(ctypes.byref(desc), _stream(stream)), "structadmm_conv_fwd")
    _keep_for_stream(stream, *temps)
    return Y


def csr(Z, kept_idx, nnz: Optional[int] = None, row_ptr=None, col=None, val=None, stream=None):
    """structadmm_csr: CSR (row_ptr int32 [A+1], col int32 [nnz], val bf16 bits
    uint16 [nnz]) of an element-wise pruned layer from its projection's
    ascending kept indices."""
    import torch
    A, B, C, D = Z.shape
    nnz = int(kept_idx.numel()) if nnz is None else int(nnz)
    dev = Z.device
    if row_ptr is None:
        row_ptr = torch.empty(A + 1, dtype=torch.int32, device=dev)
    if col is None:
        col = torch.empty(max(nnz, 1), dtype=torch.int32, device=dev)
    if val is None:
        val = torch.empty(max(nnz, 1), dtype=torch.uint16, device=dev)
    d = CsrDesc(A, B, C, D, nnz, _ptr(Z), _ptr(kept_idx) if nnz else None, _ptr(row_ptr),
                _ptr(col) if nnz else None, _ptr(val) if nnz else None)
    _check(lib().structadmm_csr(ctypes.byref(d), _stream(stream)), "structadmm_csr")
    _keep_for_stream(stream, row_ptr, col, val)
    return row_ptr, col, val


def sparse_conv_desc(Xp, row_ptr, col, val, shape, groups, stride, pad, nnz, Y, ws=None,
                     reuse_ws: bool = False) -> SparseConvDesc:
    N, H, W, Cx = Xp.shape
    A, B, C, D = shape
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    return SparseConvDesc(N, H, W, Cx, A, B, C, D, groups, stride, pad, nnz, _ptr(Xp), _ptr(row_ptr),
                          _ptr(col) if nnz else None, _ptr(val) if nnz else None, _ptr(Y), _ptr(ws), nbytes,
                          1 if reuse_ws else 0)


def conv_sparse_workspace(Xp, shape, groups: int, stride: int, pad: int, nnz: int) -> int:
    """Scratch bytes structadmm_conv_sparse_fwd needs."""
    d = sparse_conv_desc(Xp, None, None, None, shape, groups, stride, pad, nnz, None)
    return int(lib().structadmm_conv_sparse_workspace(ctypes.byref(d)))


def conv_sparse_fwd(Xp, row_ptr, col, val, shape, groups: int, stride: int, pad: int, nnz: int,
                    Y=None, ws=None, reuse_ws: bool = False, stream=None, desc: Optional[SparseConvDesc] = None):
    """structadmm_conv_sparse_fwd; Xp bf16 NHWC (uint16), returns Y bf16 NHWC
    [N, P, Q, A] (uint16).  reuse_ws: ws holds the padded entries an earlier
    call with the same CSR and geometry built."""
    import torch
    temps = []
    if desc is None:
        N, H, W, Cx = Xp.shape
        A, B, C, D = shape
        if Y is None:
            P = (H + 2 * pad - C) // stride + 1
            Q = (W + 2 * pad - D) // stride + 1
            Y = torch.empty((N, P, Q, A), dtype=torch.uint16, device=Xp.device)
            temps.append(Y)
        if ws is None:
            need = conv_sparse_workspace(Xp, shape, groups, stride, pad, nnz)
            ws = torch.empty(max(need, 256), dtype=torch.uint8, device=Xp.device)
            temps.append(ws)
        desc = sparse_conv_desc(Xp, row_ptr, col, val, shape, groups, stride, pad, nnz, Y, ws, reuse_ws)
    _check(lib().structadmm_conv_sparse_fwd(ctypes.byref(desc), _stream(stream)), "structadmm_conv_sparse_fwd")
    _keep_for_stream(stream, *temps)
    return Y


def version() -> str:
    return lib().structadmm_version().decode()
