"""Helpers shared by the GPU tests: run the library on host arrays and bring
results back, plus the comparisons used throughout (bitwise, rel-L2,
max-abs / RMS).  Not a test module."""
from __future__ import annotations

import numpy as np

import paper_1807_11091_amd as sa

DEV = "cuda"


def torch():
    import torch as t
    return t


def to_dev(a):
    t = torch()
    return t.from_numpy(np.ascontiguousarray(a)).to(DEV)


def n_groups(shape, kind):
    A, B, C, D = shape
    return {sa.FILTER: A, sa.CHANNEL: B, sa.SHAPE: B * C * D, sa.ELEMENT: A * B * C * D}[kind]


class GpuLayer:
    """Device buffers of one projection layer, built from host W, U."""

    def __init__(self, W, U, kind, k, groups=1, in_ch_mask=None, rho=0.0, fused=False, scores=True):
        t = torch()
        self.shape = W.shape
        self.W = to_dev(W)
        self.U = to_dev(U)
        self.Z = t.full_like(self.W, float("nan"))
        G = n_groups(W.shape, kind)
        self.mask = t.full((G,), 7, dtype=t.uint8, device=DEV)
        self.kept = t.full((max(k, 1),), -1, dtype=t.int32, device=DEV)
        self.scores = t.empty(G, dtype=t.float64, device=DEV) if scores else None
        self.G = t.full_like(self.W, float("nan")) if fused else None
        self.in_ch_mask = in_ch_mask if (in_ch_mask is None or hasattr(in_ch_mask, "data_ptr")) else to_dev(in_ch_mask)
        self.layer = sa.ProjectLayer(self.W, self.U, self.Z, self.mask, self.kept, kind, k, groups,
                                     self.in_ch_mask, self.scores, rho, self.G)
        self.k = k

    def host(self):
        out = {"Z": self.Z.cpu().numpy(), "mask": self.mask.cpu().numpy(),
               "kept_idx": self.kept.cpu().numpy()[: self.k]}
        if self.scores is not None:
            out["scores"] = self.scores.cpu().numpy()
        if self.G is not None:
            out["U"] = self.U.cpu().numpy()
            out["G"] = self.G.cpu().numpy()
        return out


def run_project(layers, stream=None):
    t = torch()
    ls = [l.layer for l in layers]
    nbytes = sa.project_workspace(ls)
    ws = t.empty(max(nbytes, 256), dtype=t.uint8, device=DEV)
    sa.project(ls, ws, stream=stream)
    t.cuda.synchronize()
    return [l.host() for l in layers]


def bitwise_equal(a, b):
    a = np.ascontiguousarray(a)
    b = np.ascontiguousarray(b)
    return a.shape == b.shape and np.array_equal(a.view(np.uint8), b.view(np.uint8))


def rel_l2(a, ref):
    ref = ref.astype(np.float64)
    den = np.linalg.norm(ref)
    num = np.linalg.norm(a.astype(np.float64) - ref)
    return 0.0 if den == 0 and num == 0 else num / max(den, 1e-300)


def maxabs_over_rms(y, ref):
    ref = ref.astype(np.float64)
    rms = np.sqrt(np.mean(ref ** 2))
    return float(np.max(np.abs(y.astype(np.float64) - ref)) / max(rms, 1e-300))


def bf16_bits_to_f64(bits):
    b = np.ascontiguousarray(bits).view(np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def boundary_gap(scores, k):
    """Relative gap between the k-th and (k+1)-th largest score."""
    if k <= 0 or k >= len(scores):
        return np.inf
    s = np.sort(scores)[::-1]
    return (s[k - 1] - s[k]) / s[k - 1] if s[k - 1] > 0 else np.inf
