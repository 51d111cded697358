#!/usr/bin/env python3
"""Benchmark of the StructADMM hot path on one MI355X.

Workload: AlexNet conv1-5 at batch 128, filter-shape-wise pruning keeping 30%
of the (c, kh, kw) columns of every layer (synthetic weights and inputs of
the paper's AlexNet shapes; no dataset, no trained weights).

One step = one pass of the whole path over one batch:
  1. structadmm_project     fused Z-update + dual update + regulariser gradient, 5 layers in one call
  2. structadmm_dual_update per-SGD-step gradient rho (W - Z + U) of the 5 layers
  3. per layer: structadmm_compact (pruned and dense matrices), then structadmm_pack_nhwc of
     every layer's input
  4. structadmm_conv_fwd of every layer over its compacted matrix, then over the dense one
Inputs are resident in HBM before the timed region.

Output: one JSON line.  value = compacted-CONV TFLOP/s over the step's five
compacted convolutions (algorithmic flops 2*N*P*Q*sum_g M_g*K_g / their
HIP-event time); speedup_vs_dense = dense CONV time / compacted CONV time;
admm_gbps = algorithmic bytes of steps 1-2 / their time.  Each CONV is bracketed
by HIP events on the stream it runs on; the CONVs are enqueued back to back
(the compactions, which return sizes to the host, come first), so the events
measure the kernels rather than host gaps.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "compacted-conv TFLOP/s & speedup vs dense; ADMM projection+update HBM GB/s"
WORKLOAD = "alexnet_shape30"
HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=3)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-seconds", type=float, default=12.0, help="target CPU time of the oracle sample")
    p.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                   help="only copy MIB MiB device-to-device 5 times (HBM counter calibration) and exit")
    return p.parse_args()


class Layer:
    pass


def setup(torch, sa, wl):
    from workloads import input_nchw, layer_tensors
    dev = "cuda"
    kind, pct = wl.variants[0]
    layers = []
    for li, L in enumerate(wl.layers):
        W, U = layer_tensors(wl, li)
        k = wl.k_for(li, kind, pct)
        o = Layer()
        o.cfg, o.k, o.kind = L, k, kind
        o.W = torch.from_numpy(W).to(dev)
        o.U = torch.from_numpy(U).to(dev)
        o.Z = torch.empty_like(o.W)
        o.G = torch.empty_like(o.W)
        o.G2 = torch.empty_like(o.W)
        G = L.n_groups(kind)
        o.mask = torch.empty(G, dtype=torch.uint8, device=dev)
        o.kept = torch.empty(max(k, 1), dtype=torch.int32, device=dev)
        o.X = torch.from_numpy(input_nchw(wl, li)).to(dev)
        N, Cin, H, Wd = o.X.shape
        o.Xp = torch.empty((N, H, Wd, Cin), dtype=torch.uint16, device=dev)
        Kf = L.K
        o.comp_out = (torch.empty(L.A * ((Kf + 63) // 64 * 64), dtype=torch.uint16, device=dev),
                      torch.empty(L.A, dtype=torch.int32, device=dev),
                      torch.empty(L.groups * Kf, dtype=torch.int32, device=dev),
                      torch.empty(L.groups * Kf, dtype=torch.int32, device=dev))
        o.dense_out = tuple(torch.empty_like(t) for t in o.comp_out)
        o.Yc = None
        o.cvws = None
        o.Yd = torch.empty((N, L.P, L.Q, L.A), dtype=torch.uint16, device=dev)
        o.proj = sa.ProjectLayer(o.W, o.U, o.Z, o.mask, o.kept, kind, k, L.groups, None, None, wl.rho, o.G)
        layers.append(o)
    return layers


def run_step(torch, sa, wl, layers, ws, cws, ev, record):
    """One pass of the hot path; returns per-part event pairs when record."""
    marks = {}

    def mark(name):
        if record:
            e = torch.cuda.Event(enable_timing=True)
            e.record()
            marks.setdefault(name, []).append(e)

    mark("admm0")
    sa.project([o.proj for o in layers], ws, descs=ev["pdescs"])
    sa.dual_update(None, descs=ev["ddescs"])
    mark("admm1")
    # compaction synchronises with the host (it returns the sizes), so every
    # layer is compacted first and the CONVs are then enqueued back to back
    comp = []
    for i, o in enumerate(layers):
        L = o.cfg
        cols = o.mask if o.kind == sa.SHAPE else None
        rows = o.mask if o.kind == sa.FILTER else None
        c = sa.compact(o.Z, L.groups, row_mask=rows, col_mask=cols, ws=cws, out=o.comp_out)
        d = sa.compact(o.Z, L.groups, ws=cws, out=o.dense_out)
        sizes, sized = c[4], d[4]
        if o.Yc is None:
            o.Yc = torch.empty(sa.conv_out_shape(*o.Xp.shape[:3], L.C, L.D, L.stride, L.pad, sizes),
                               dtype=torch.uint16, device="cuda")
            o.flops_c = 2 * wl.batch * L.P * L.Q * sum(sizes.M[g] * sizes.K[g] for g in range(sizes.groups))
            o.flops_d = 2 * wl.batch * L.P * L.Q * sum(sized.M[g] * sized.K[g] for g in range(sized.groups))
        # scratch for groups whose im2col rows are gathered first; the kept
        # columns move between ADMM steps, so it is sized for every step (outside
        # the CONV events) and grown when a step needs more
        need = max(sa.conv_workspace(o.Xp, sizes, L.C, L.D, L.stride, L.pad),
                   sa.conv_workspace(o.Xp, sized, L.C, L.D, L.stride, L.pad), 256)
        if o.cvws is None or o.cvws.numel() < need:
            o.cvws = torch.empty(need, dtype=torch.uint8, device="cuda")
        comp.append((c, d))
    # the packs are enqueued after the last compaction, so the GPU is busy with
    # them while the host enqueues the first CONV
    for o in layers:
        sa.pack_nhwc(o.X, out=o.Xp)
    for i, (o, (c, d)) in enumerate(zip(layers, comp)):
        L = o.cfg
        mark(f"c{i}a")
        sa.conv_fwd(o.Xp, c[0], c[2], c[3], c[4], L.C, L.D, L.stride, L.pad, Y=o.Yc, ws=o.cvws)
        mark(f"c{i}b")
    for i, (o, (c, d)) in enumerate(zip(layers, comp)):
        L = o.cfg
        mark(f"d{i}a")
        sa.conv_fwd(o.Xp, d[0], d[2], d[3], d[4], L.C, L.D, L.stride, L.pad, Y=o.Yd, ws=o.cvws)
        mark(f"d{i}b")
    return marks


def cpu_baseline(wl, seconds):
    """The oracle on the host cores over a bounded sample of the same workload:
    the fused ADMM step of all five layers and the compacted CONV of as many
    images as fit the time budget (binary64 loops, OpenMP over images)."""
    import oracle
    from workloads import input_nchw, layer_tensors
    kind, pct = wl.variants[0]
    prep = []
    t_admm = 0.0
    for li, L in enumerate(wl.layers):
        W, U = layer_tensors(wl, li)
        k = wl.k_for(li, kind, pct)
        t0 = time.perf_counter()
        r = oracle.project(W, U, kind, k, L.groups, rho=wl.rho, fused=True)
        t_admm += time.perf_counter() - t0
        rc = oracle.compact(r["Z"], L.groups, col_mask=r["mask"])
        prep.append((L, rc))
    # one image first, then as many as fit the budget
    def conv_images(nimg):
        flops, t = 0, 0.0
        for li, (L, rc) in enumerate(prep):
            X = input_nchw(wl, li, batch=nimg)
            Xb = oracle.pack(X)
            t0 = time.perf_counter()
            oracle.conv(Xb, rc, L.C, L.D, L.stride, L.pad)
            t += time.perf_counter() - t0
            flops += 2 * nimg * L.P * L.Q * int(np.sum(rc["M"].astype(np.int64) * rc["K"]))
        return flops, t
    threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    # calibrate on one image per thread (the oracle runs images in parallel)
    n0 = min(wl.batch, threads)
    f, t = conv_images(n0)
    nimg = int(min(wl.batch, max(n0, (seconds / max(t, 1e-6)) * n0 // threads * threads)))
    if nimg > n0:
        f, t = conv_images(nimg)
    return {"value": f / t / 1e12, "unit": "TFLOP/s", "cores": min(threads, os.cpu_count() or threads),
            "kind": "oracle",
            "sample": f"compacted CONV of conv1-5 on {nimg} of {wl.batch} images "
                      f"({f / 1e9:.1f} GFLOP in {t:.1f} s); fused ADMM step of all 5 layers took "
                      f"{t_admm * 1e3:.0f} ms on one core"}


def copy_probe(mib):
    """A plain copy of known size: the reference the HBM byte counters
    (FETCH_SIZE, WRITE_SIZE) are scaled by."""
    import torch
    n = mib << 20
    src = torch.ones(n, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes": n, "copies": 5}))


def traffic_per_launch():
    """HBM bytes per k_conv_patch launch from the committed counter summary,
    if it was taken on the current CONV source (else None)."""
    import hashlib
    summ = os.path.join(ROOT, "profiles", "k_conv_patch_alexnet_shape30_traffic.md")
    src = os.path.join(ROOT, "paper_1807_11091_amd", "csrc", "conv.hip")
    if not os.path.exists(summ):
        return None
    fields = {}
    for line in open(summ):
        if line.startswith("- ") and ":" in line:
            k, v = line[2:].split(":", 1)
            fields[k.strip()] = v.strip().strip("`")
    digest = hashlib.sha256(open(src, "rb").read()).hexdigest()
    if fields.get("conv.hip sha256") != digest or "bytes per launch" not in fields:
        return None
    return int(fields["bytes per launch"])


def main():
    args = parse()
    if args.copy_probe:
        copy_probe(args.copy_probe)
        return
    if args.gpus != 1:
        print(json.dumps({"error": "this build measures one GPU only; run with --gpus 1"}))
        sys.exit(2)
    import torch
    import paper_1807_11091_amd as sa
    from workloads import WORKLOADS

    if not torch.cuda.is_available():
        raise SystemExit("bench.py needs a GPU")
    sa.lib()  # fails loudly if the HIP library is missing
    wl = WORKLOADS[WORKLOAD]
    layers = setup(torch, sa, wl)
    ws = torch.empty(max(256, sa.project_workspace([o.proj for o in layers])), dtype=torch.uint8, device="cuda")
    cws = torch.empty(sa.COMPACT_WS_BYTES, dtype=torch.uint8, device="cuda")
    ev = {"pdescs": sa._descs([o.proj for o in layers]),
          "ddescs": sa.dual_descs([(o.W, o.Z, o.U, wl.rho, o.G2, False) for o in layers])}

    # at least one untimed step: it sizes the output and scratch buffers
    for _ in range(max(1, args.warmup)):
        run_step(torch, sa, wl, layers, ws, cws, ev, record=False)
    torch.cuda.synchronize()

    t0 = time.perf_counter()
    all_marks = []
    for _ in range(args.steps):
        all_marks.append(run_step(torch, sa, wl, layers, ws, cws, ev, record=True))
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0

    def span(m, a, b):
        return sum(x.elapsed_time(y) for x, y in zip(m[a], m[b]))  # ms

    t_admm = sum(span(m, "admm0", "admm1") for m in all_marks) / args.steps
    t_c = [sum(span(m, f"c{i}a", f"c{i}b") for m in all_marks) / args.steps for i in range(len(layers))]
    t_d = [sum(span(m, f"d{i}a", f"d{i}b") for m in all_marks) / args.steps for i in range(len(layers))]
    flops_c = sum(o.flops_c for o in layers)
    flops_d = sum(o.flops_d for o in layers)
    n_el = sum(o.cfg.n for o in layers)
    admm_bytes = 20 * n_el + 16 * n_el  # fused step (W,U read; Z,U,G written) + gradient (W,Z,U read; G written)
    tflops_c = flops_c / (sum(t_c) * 1e-3) / 1e12
    tflops_d = flops_d / (sum(t_d) * 1e-3) / 1e12
    # dominant kernel of the compacted path: k_conv_patch, one launch per
    # shape-pruned layer whose input channels are 8-aligned (CONV2-5)
    patch = [i for i, o in enumerate(layers) if o.Xp.shape[3] % 8 == 0]
    patch_ms = sum(t_c[i] for i in patch)
    patch_tflops = sum(layers[i].flops_c for i in patch) / (patch_ms * 1e-3) / 1e12
    out = {
        "metric": METRIC,
        "value": round(tflops_c, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall * 1e3 / args.steps, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": WORKLOAD, "layers": "AlexNet conv1-5", "batch": wl.batch,
                   "sparsity": "filter-shape-wise, keep 30% of columns", "parallelism": "single GPU"},
        "speedup_vs_dense": round(sum(t_d) / sum(t_c), 3),
        "dense_conv_tflops": round(tflops_d, 3),
        "admm_gbps": round(admm_bytes / (t_admm * 1e-3) / 1e9, 1),
        "admm_us": round(t_admm * 1e3, 2),
        "per_layer": [{"layer": o.cfg.name, "compact_us": round(tc * 1e3, 1), "dense_us": round(td * 1e3, 1),
                       "compact_tflops": round(o.flops_c / (tc * 1e-3) / 1e12, 1),
                       "dense_tflops": round(o.flops_d / (td * 1e-3) / 1e12, 1),
                       "speedup": round(td / tc, 2)}
                      for o, tc, td in zip(layers, t_c, t_d)],
        "roofline": {"kernel": "k_conv_patch (compacted " + "/".join(layers[i].cfg.name for i in patch) + ")",
                     "bound": "mfma", "achieved": round(patch_tflops, 2), "peak": BF16_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(patch_tflops / BF16_PEAK_TFLOPS, 4),
                     "avg_launch_us": round(patch_ms * 1e3 / len(patch), 2), "launches_per_step": len(patch),
                     "traffic": traffic_per_launch()},
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl, args.cpu_seconds)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
