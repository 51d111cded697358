"""Seeded tensor generators (host, numpy PCG64).

Every tensor is drawn from its own stream,
``PCG64(SeedSequence([1807, 11091, workload_id, layer, tensor]))`` with
tensor 0 = W, 1 = U, 2 = X.  Weights are drawn as float64 standard normals,
scaled by sigma and cast to float32; inputs X ~ N(0, 1) are drawn directly
as float32 (ziggurat) to keep host memory and time low at batch 128.
The same host bits feed the GPU library and the oracle.
"""
from __future__ import annotations

import numpy as np

from .configs import ConvLayer, Workload

W_ID, U_ID, X_ID = 0, 1, 2


def _rng(wid: int, layer: int, tensor: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([1807, 11091, wid, layer, tensor])))


def normal_f32(wid: int, layer: int, tensor: int, shape, sigma: float) -> np.ndarray:
    """float32 array ~ N(0, sigma^2); all zeros when sigma == 0."""
    if sigma == 0.0:
        return np.zeros(shape, dtype=np.float32)
    r = _rng(wid, layer, tensor)
    return (r.standard_normal(shape, dtype=np.float64) * sigma).astype(np.float32)


def layer_tensors(wl: Workload, li: int):
    """(W, U) float32 [A, B, C, D] for layer ``li`` of a workload."""
    L: ConvLayer = wl.layers[li]
    shape = (L.A, L.B, L.C, L.D)
    W = normal_f32(wl.wid, li, W_ID, shape, wl.sigma_w(L))
    U = normal_f32(wl.wid, li, U_ID, shape, wl.u_sigma)
    return W, U


def input_nchw(wl: Workload, li: int, batch: int = None) -> np.ndarray:
    """float32 input X ~ N(0, 1) of shape [N, groups*B, H, W] (NCHW)."""
    L: ConvLayer = wl.layers[li]
    n = wl.batch if batch is None else batch
    r = _rng(wl.wid, li, X_ID)
    return r.standard_normal((n, L.in_channels, L.H, L.W), dtype=np.float32)
