"""Python access to the CPU oracle (``oracle.c``) via ctypes and numpy.

TEST INFRASTRUCTURE ONLY: imported by the test suite, the smoke check and the
benchmark's CPU-baseline leg.  The GPU library never imports this package and
shares no code with it.

Every function here only marshals numpy arrays into the C routines, which
state the method (arXiv 1807.11091, Sections 3-4) in plain loops.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

FILTER, CHANNEL, SHAPE, ELEMENT = 0, 1, 2, 3


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (binary32/binary64 as written: no fast-math,
    no FMA contraction)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fopenmp", "-ffp-contract=off",
                               "-fno-fast-math", "-shared", "-fPIC", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build(force=False)
        L = ctypes.CDLL(_LIB)
        i64, i32, f32, vp = ctypes.c_int64, ctypes.c_int32, ctypes.c_float, ctypes.c_void_p
        L.oracle_n_groups.argtypes = [i64, i64, i64, i64, i32]
        L.oracle_n_groups.restype = i64
        L.oracle_scores.argtypes = [i64, i64, i64, i64, i32, i32, vp, vp, vp, vp, vp]
        L.oracle_scores.restype = None
        L.oracle_select.argtypes = [i64, vp, i64, vp, vp]
        L.oracle_select.restype = ctypes.c_int
        L.oracle_project.argtypes = [i64, i64, i64, i64, i32, i32, i64, vp, vp, vp, f32,
                                     vp, vp, vp, vp, vp, vp]
        L.oracle_project.restype = ctypes.c_int
        L.oracle_dual_update.argtypes = [i64, vp, vp, vp, f32, vp, i32]
        L.oracle_dual_update.restype = None
        L.oracle_sgd_step.argtypes = [i64, i64, i64, i64, i32, vp, vp, vp, vp, vp, f32, f32]
        L.oracle_sgd_step.restype = None
        L.oracle_bf16_array.argtypes = [i64, vp, vp]
        L.oracle_bf16_array.restype = None
        L.oracle_compact.argtypes = [i64, i64, i64, i64, i32, vp, vp, vp, vp, vp, i32,
                                     vp, vp, vp, vp, vp, vp]
        L.oracle_compact.restype = ctypes.c_int
        L.oracle_pack.argtypes = [i64, i64, i64, i64, vp, vp, vp]
        L.oracle_pack.restype = None
        L.oracle_conv.argtypes = [i64, i64, i64, i64, vp, i32, i64, i64, i64, i64,
                                  vp, vp, vp, vp, vp, vp]
        L.oracle_conv.restype = None
        L.oracle_csr.argtypes = [i64, i64, i64, i64, vp, vp, vp, vp, vp]
        L.oracle_csr.restype = i64
        L.oracle_conv_csr.argtypes = [i64, i64, i64, vp, i64, i64, i64, i64, i32, i64, i64,
                                      vp, vp, vp, vp]
        L.oracle_conv_csr.restype = None
        _lib = L
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return None if a is None else np.ascontiguousarray(a, dtype=dtype)


def n_groups(shape, kind: int) -> int:
    A, B, C, D = shape
    return int(lib().oracle_n_groups(A, B, C, D, kind))


def project(W, U, kind: int, k: int, groups: int = 1, in_ch_mask=None, rho: float = 0.0,
            fused: bool = False):
    """Z-update of one layer (Section 4): returns dict with Z, mask, kept_idx,
    scores; with ``fused`` also U_new (dual update) and G (regulariser gradient)."""
    W = _c(W, np.float32)
    U = _c(U, np.float32)
    A, B, C, D = W.shape
    G = n_groups(W.shape, kind)
    Z = np.empty_like(W)
    mask = np.empty(G, np.uint8)
    kept = np.empty(max(k, 1), np.int32)
    scores = np.empty(G, np.float64)
    m = _c(in_ch_mask, np.uint8)
    U_new = np.empty_like(W) if fused else None
    Gr = np.empty_like(W) if fused else None
    rc = lib().oracle_project(A, B, C, D, groups, kind, k, _p(W), _p(U), _p(m),
                              ctypes.c_float(rho), _p(Z), _p(mask), _p(kept), _p(scores),
                              _p(U_new), _p(Gr))
    if rc != 0:
        raise ValueError(f"oracle_project failed ({rc})")
    out = {"Z": Z, "mask": mask, "kept_idx": kept[:k].copy(), "scores": scores}
    if fused:
        out["U"] = U_new
        out["G"] = Gr
    return out


def dual_update(W, Z, U, rho: float, update_dual: bool = True, want_grad: bool = True):
    """Dual update and regulariser gradient; returns (U_new, G)."""
    W = _c(W, np.float32)
    Z = _c(Z, np.float32)
    U = np.array(U, dtype=np.float32, copy=True)
    G = np.empty_like(W) if want_grad else None
    lib().oracle_dual_update(W.size, _p(W), _p(Z), _p(U), ctypes.c_float(rho), _p(G),
                             1 if update_dual else 0)
    return U, G


def sgd_step(W, Gf, Z=None, U=None, mask=None, kind: int = FILTER, rho: float = 0.0, lr: float = 0.01):
    """One SGD step of the W-subproblem / masked retraining; returns the new W
    (W [A,B,C,D] is not modified)."""
    W = np.array(W, dtype=np.float32, copy=True)
    A, B, C, D = W.shape
    Gf = _c(Gf, np.float32)
    Z = None if Z is None else _c(Z, np.float32)
    U = None if U is None else _c(U, np.float32)
    mask = None if mask is None else _c(mask, np.uint8)
    lib().oracle_sgd_step(A, B, C, D, kind, _p(mask), _p(W), _p(Gf), _p(Z), _p(U),
                          ctypes.c_float(rho), ctypes.c_float(lr))
    return W


def bf16_bits(x) -> np.ndarray:
    """binary32 -> bfloat16 bit patterns (uint16), round to nearest even."""
    x = _c(x, np.float32)
    out = np.empty(x.shape, np.uint16)
    lib().oracle_bf16_array(x.size, _p(x), _p(out))
    return out


def bf16_to_f64(bits) -> np.ndarray:
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def compact(Z, groups: int = 1, row_mask=None, col_mask=None, chan_mask=None,
            in_ch_mask=None, in_compacted: bool = False):
    """Compacted GEMM matrices of a layer (Section 3): dict with Wc (uint16
    bf16 bits, groups concatenated), row_idx, col_ch, col_tap, M, K."""
    Z = _c(Z, np.float32)
    A, B, C, D = Z.shape
    Wc = np.empty(Z.size, np.uint16)
    row_idx = np.empty(A, np.int32)
    col_ch = np.empty(groups * B * C * D, np.int32)
    col_tap = np.empty(groups * B * C * D, np.int32)
    M = np.empty(groups, np.int32)
    K = np.empty(groups, np.int32)
    rc = lib().oracle_compact(A, B, C, D, groups, _p(Z), _p(_c(row_mask, np.uint8)),
                              _p(_c(col_mask, np.uint8)), _p(_c(chan_mask, np.uint8)),
                              _p(_c(in_ch_mask, np.uint8)), 1 if in_compacted else 0,
                              _p(Wc), _p(row_idx), _p(col_ch), _p(col_tap), _p(M), _p(K))
    if rc != 0:
        raise ValueError(f"oracle_compact failed ({rc})")
    nw = int(np.sum(M.astype(np.int64) * K))
    nr, ncol = int(M.sum()), int(K.sum())
    return {"Wc": Wc[:nw].copy(), "row_idx": row_idx[:nr].copy(), "col_ch": col_ch[:ncol].copy(),
            "col_tap": col_tap[:ncol].copy(), "M": M, "K": K}


def pack(X, keep=None) -> np.ndarray:
    """fp32 NCHW input -> bf16 bits NCHW, keeping channels with keep[ch] set."""
    X = _c(X, np.float32)
    N, Cin, H, W = X.shape
    k = _c(keep, np.uint8)
    Cx = Cin if k is None else int(np.count_nonzero(k))
    out = np.empty((N, Cx, H, W), np.uint16)
    lib().oracle_pack(N, Cin, H, W, _p(X), _p(k), _p(out))
    return out


def conv(Xb, comp, C: int, D: int, stride: int, pad: int) -> np.ndarray:
    """fp64 CONV over compacted matrices; Xb = bf16 bits NCHW. Returns NHWC fp64."""
    Xb = np.ascontiguousarray(Xb, dtype=np.uint16)
    N, Cx, H, W = Xb.shape
    groups = len(comp["M"])
    P = (H + 2 * pad - C) // stride + 1
    Q = (W + 2 * pad - D) // stride + 1
    Cy = int(comp["M"].sum())
    Y = np.empty((N, P, Q, Cy), np.float64)
    lib().oracle_conv(N, Cx, H, W, _p(Xb), groups, C, D, stride, pad,
                      _p(comp["Wc"]), _p(comp["M"]), _p(comp["K"]),
                      _p(comp["col_ch"]), _p(comp["col_tap"]), _p(Y))
    return Y


def csr(Z, mask) -> dict:
    """CSR of a non-structured pruned layer's [A, B*C*D] GEMM matrix (kept
    entries of ``mask``, bf16 values): dict with row_ptr, col, val."""
    Z = _c(Z, np.float32)
    A = Z.shape[0]
    m = _c(mask, np.uint8).reshape(-1)
    assert m.size == Z.size
    nnz = int(np.count_nonzero(m))
    row_ptr = np.empty(A + 1, np.int32)
    col = np.empty(max(nnz, 1), np.int32)
    val = np.empty(max(nnz, 1), np.uint16)
    got = lib().oracle_csr(*Z.shape, _p(Z), _p(m), _p(row_ptr), _p(col), _p(val))
    assert got == nnz
    return {"row_ptr": row_ptr, "col": col[:nnz].copy(), "val": val[:nnz].copy()}


def conv_csr(Xb, csr_, shape, groups: int, stride: int, pad: int) -> np.ndarray:
    """fp64 CONV of a CSR layer of weight shape (A, B, C, D); Xb = bf16 bits
    NCHW with groups*B channels.  Returns NHWC fp64 [N, P, Q, A]."""
    Xb = np.ascontiguousarray(Xb, dtype=np.uint16)
    N, Cx, H, W = Xb.shape
    A, B, C, D = shape
    assert Cx == groups * B and A % groups == 0
    P = (H + 2 * pad - C) // stride + 1
    Q = (W + 2 * pad - D) // stride + 1
    Y = np.empty((N, P, Q, A), np.float64)
    col = csr_["col"] if csr_["col"].size else np.zeros(1, np.int32)
    val = csr_["val"] if csr_["val"].size else np.zeros(1, np.uint16)
    lib().oracle_conv_csr(N, H, W, _p(Xb), A, B, C, D, groups, stride, pad,
                          _p(_c(csr_["row_ptr"], np.int32)), _p(_c(col, np.int32)),
                          _p(_c(val, np.uint16)), _p(Y))
    return Y
