#!/usr/bin/env python3
"""Benchmark of the StructADMM hot path on one MI355X.

Workload: the 53 convolutions of ResNet-50 v1.5 at 224x224, batch 64,
filter-wise pruning keeping 60% of the filters of every layer (synthetic
weights and inputs of the paper's ResNet-50 shapes; no dataset, no trained
weights).  The AlexNet conv1-5 workload (batch 128, filter-shape-wise 30%)
is measured in the same run with fewer steps and reported under its own key.

One step = one pass of the whole path over one batch:
  1. structadmm_project     fused Z-update + dual update + regulariser gradient, all layers in one call
  2. structadmm_dual_update per-SGD-step gradient rho (W - Z + U) of all layers
  3. per layer: structadmm_compact (pruned and dense matrices), then structadmm_pack_nhwc of
     every layer's input
  4. structadmm_conv_fwd of every layer over its compacted matrix, then over the dense one
Inputs are resident in HBM before the timed region.

Output: one JSON line.  value = compacted-CONV TFLOP/s over the step's
compacted convolutions (algorithmic flops 2*N*P*Q*sum_g M_g*K_g / their
HIP-event time); speedup_vs_dense = dense CONV time / compacted CONV time;
admm_gbps = algorithmic bytes of steps 1-2 / their time.  HIP events on the
stream the work runs on (recorded without a system-scope fence, which would
write back and invalidate the caches at every event) bracket the ADMM calls,
the packs, the block of 53 compacted CONVs and the block of 53 dense CONVs;
a few extra steps bracket every CONV for the per-layer breakdown (each
event pair adds its own gap, so those spans sum above the block spans).  A
spin kernel ahead of each timed block lets the host enqueue the block before
the GPU reaches it, so the events measure the kernels rather than host
gaps.  ms_per_step is the wall time of a step: the GPU time of its parts,
the host-side synchronisations of the compactions, and the spins (reported
separately as spin_ms_per_step).
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
FILTER_KIND, SHAPE_KIND = 0, 2  # sparsity-set kinds (the C ABI's enum)
WORKLOAD = "resnet50_filter60"
SECOND_WORKLOAD = "alexnet_shape30"
HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0
# spin ahead of the ADMM block of a step; the spin ahead of the pack + CONV
# block is sized from the host's measured enqueue time of that block
LEAD_US = 300
LEAD_CONV_MAX_US = 40000


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=3)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-seconds", type=float, default=12.0, help="target CPU time of the oracle sample")
    p.add_argument("--suite", metavar="JSON", default=None,
                   help="measure every workload (ADMM one-call and replicated, CONV per layer against "
                        "MIOpen, density sweep, achievable peaks) and write the report to JSON")
    p.add_argument("--tables", metavar="JSON", default=None,
                   help="only the batch-1 replay of the pruned AlexNet layers of Tables 1-2 (CONV speedups)")
    p.add_argument("--admm", metavar="WORKLOAD", default=None,
                   help="only the ADMM step (fused projection, gradient, SGD steps) of one workload, "
                        "one call and replicated; prints one JSON line")
    p.add_argument("--sparse", metavar="JSON", default=None,
                   help="only the CSR CONV of non-structured pruning: density sweep of the [256,256,3,3] "
                        "layer and batch-1 AlexNet conv2-5 at the sparsities of Tables 4-5")
    p.add_argument("--conv-only", metavar="WORKLOAD", default=None,
                   help="only the compacted CONVs of one workload, --reps times each, untimed (a short "
                        "program for hardware-counter runs); prints one JSON line per layer")
    p.add_argument("--kernel", default=None,
                   help="with --conv-only: only the layers whose compacted CONV is this one kernel")
    p.add_argument("--layers", default=None, help="with --conv-only: comma-separated layer indices")
    p.add_argument("--dense", action="store_true", help="with --conv-only: the uncompacted matrices instead")
    p.add_argument("--reps", type=int, default=5, help="with --conv-only: launches per layer")
    p.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                   help="only copy MIB MiB device-to-device 5 times (HBM counter calibration) and exit")
    return p.parse_args()


class Layer:
    pass


def pitch8(sizes):
    """Output row pitch of a compacted CONV: its kept filters rounded up to a
    multiple of 8 channels, so that every output row starts on a 16-byte
    boundary (the padding channels are not part of the result)."""
    cy = sum(sizes.M[g] for g in range(sizes.groups))
    return (cy + 7) // 8 * 8


def kept_k(sizes, g):
    """Kept columns of conv group g (the compaction's alignment columns, +0,
    are not algorithmic work)."""
    return sizes.K[g] - sizes.kpad[g]


class TimingEvent:
    """A HIP timing event recorded without the system-scope fence
    (hipEventDisableSystemFence): torch's events write back and invalidate the
    caches when recorded, which costs each bracketed kernel several
    microseconds and starts it with cold caches.  Only timestamps are read, after a
    device-wide synchronisation."""
    _hip = None

    def __init__(self):
        import ctypes
        if TimingEvent._hip is None:
            lib = ctypes.CDLL("libamdhip64.so")  # the HIP runtime torch has loaded
            lib.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
            lib.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
            lib.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
            lib.hipEventDestroy.argtypes = [ctypes.c_void_p]
            TimingEvent._hip = lib
        self._ev = ctypes.c_void_p()
        rc = TimingEvent._hip.hipEventCreateWithFlags(ctypes.byref(self._ev), 0x20000000)
        if rc != 0:
            raise RuntimeError(f"hipEventCreateWithFlags failed ({rc})")

    def record(self, torch):
        rc = TimingEvent._hip.hipEventRecord(self._ev, torch.cuda.current_stream().cuda_stream)
        if rc != 0:
            raise RuntimeError(f"hipEventRecord failed ({rc})")

    def elapsed_time(self, other):
        import ctypes
        ms = ctypes.c_float()
        rc = TimingEvent._hip.hipEventElapsedTime(ctypes.byref(ms), self._ev, other._ev)
        if rc != 0:
            raise RuntimeError(f"hipEventElapsedTime failed ({rc})")
        return ms.value

    def __del__(self):
        if TimingEvent._hip is not None and self._ev:
            TimingEvent._hip.hipEventDestroy(self._ev)


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
        # the filter + channel chain: the input channels are the previous
        # layer's kept filters
        o.in_mask = layers[-1].mask if (wl.chain and layers) else None
        o.proj = sa.ProjectLayer(o.W, o.U, o.Z, o.mask, o.kept, kind, k, L.groups, o.in_mask, None, wl.rho, o.G)
        layers.append(o)
    return layers


def run_step(torch, sa, wl, layers, ws, cws, ev, record):
    """One pass of the hot path; returns event pairs around its parts:
    record = "blocks" brackets the ADMM calls, the packs, all compacted CONVs
    and all dense CONVs (the timed steps); "layers" brackets every CONV
    (the per-layer breakdown); False records nothing."""
    marks = {}

    def mark(name, level="blocks"):
        if record and (level == "blocks" or record == "layers"):
            e = TimingEvent()
            e.record(torch)
            marks.setdefault(name, []).append(e)

    # a short spin kernel ahead of each timed block lets the host enqueue the
    # block before the GPU reaches it, so the event spans hold kernel time, not
    # the host's launch latency
    if ev.get("lead"):
        torch.cuda._sleep(ev["lead"])
    mark("admm0")
    sa.project([o.proj for o in layers], ws, descs=ev["pdescs"])
    sa.dual_update(None, descs=ev["ddescs"])
    mark("admm1")
    if any(o.in_mask is not None for o in layers):
        raise SystemExit("the timed step runs workloads without a filter + channel chain (--suite times the chain)")
    # compaction synchronises with the host (it returns the sizes): every
    # layer's kept and dense matrices in one call (one wait), then the CONVs
    # are enqueued back to back
    items = []
    for o in layers:
        cols = o.mask if o.kind == sa.SHAPE else None
        rows = o.mask if o.kind == sa.FILTER else None
        items.append(dict(Z=o.Z, groups=o.cfg.groups, row_mask=rows, col_mask=cols, out=o.comp_out))
        items.append(dict(Z=o.Z, groups=o.cfg.groups, out=o.dense_out))
    done = sa.compact_many(items, ws=cws)
    comp = []
    for i, o in enumerate(layers):
        L = o.cfg
        c, d = done[2 * i], done[2 * i + 1]
        sizes, sized = c[4], d[4]
        if o.Yc is None:
            shape = sa.conv_out_shape(*o.Xp.shape[:3], L.C, L.D, L.stride, L.pad, sizes)
            o.Yc = torch.empty(shape[:3] + (pitch8(sizes),), dtype=torch.uint16, device="cuda")
            o.flops_c = 2 * wl.batch * L.P * L.Q * sum(sizes.M[g] * kept_k(sizes, g) for g in range(sizes.groups))
            o.flops_d = 2 * wl.batch * L.P * L.Q * sum(sized.M[g] * kept_k(sized, g) for g in range(sized.groups))
            o.sizes_c = sizes
            o.plan_c = sa.conv_plan(o.Xp, sizes, L.C, L.D, L.stride, L.pad)
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
    if ev.get("lead_conv"):
        torch.cuda._sleep(ev["lead_conv"])
    t_enq = time.perf_counter()
    mark("pack0")
    for o in layers:
        sa.pack_nhwc(o.X, out=o.Xp)
    mark("pack1")
    mark("c_all0")
    for i, (o, (c, d)) in enumerate(zip(layers, comp)):
        L = o.cfg
        mark(f"c{i}a", "layers")
        sa.conv_fwd(o.Xp, c[0], c[2], c[3], c[4], L.C, L.D, L.stride, L.pad, Y=o.Yc, ws=o.cvws)
        mark(f"c{i}b", "layers")
    mark("c_all1")
    mark("d_all0")
    for i, (o, (c, d)) in enumerate(zip(layers, comp)):
        L = o.cfg
        mark(f"d{i}a", "layers")
        sa.conv_fwd(o.Xp, d[0], d[2], d[3], d[4], L.C, L.D, L.stride, L.pad, Y=o.Yd, ws=o.cvws)
        mark(f"d{i}b", "layers")
    mark("d_all1")
    ev["enqueue_s"] = time.perf_counter() - t_enq
    return marks


def lead_cycles(torch, us):
    """Cycles of torch's spin kernel that last about `us` microseconds."""
    torch.cuda._sleep(1000)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    torch.cuda._sleep(200000)
    e1.record()
    torch.cuda.synchronize()
    return max(1000, int(200000 * us / (e0.elapsed_time(e1) * 1e3)))


def cpu_baseline(wl, seconds):
    """The oracle on the host cores over a bounded sample of the same workload:
    the fused ADMM step of every layer (one thread) and the compacted CONV of
    as many images as fit the time budget (binary64 loops, OpenMP over
    (image, output row) pairs)."""
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
        rc = oracle.compact(r["Z"], L.groups, row_mask=r["mask"] if kind == FILTER_KIND else None,
                            col_mask=r["mask"] if kind == SHAPE_KIND else None)
        prep.append((L, rc))

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
    # calibrate on one image (the oracle threads over its output rows), then
    # as many images as fit the budget
    f, t = conv_images(1)
    nimg = int(min(wl.batch, max(1, seconds / max(t, 1e-6))))
    if nimg > 1:
        f, t = conv_images(nimg)
    n = sum(L.n for L in wl.layers)
    return {"value": f / t / 1e12, "unit": "TFLOP/s", "cores": min(threads, os.cpu_count() or threads),
            "kind": "oracle",
            "sample": f"compacted CONV of all {len(wl.layers)} layers on {nimg} of {wl.batch} images "
                      f"({f / 1e9:.1f} GFLOP in {t:.1f} s); fused ADMM step of all {len(wl.layers)} layers "
                      f"({n} weights) took {t_admm * 1e3:.0f} ms on one core",
            "admm_fused_GBps_1_core": round(20 * n / t_admm / 1e9, 3)}


def conv_only(args):
    """The compacted (or dense) CONV of the selected layers, args.reps launches
    each, layer after layer, with nothing timed: the program hardware-counter
    runs profile.  Every launch of a layer runs the kernel(s) of its plan."""
    import torch
    import paper_1807_11091_amd as sa
    from workloads import WORKLOADS
    if not torch.cuda.is_available():
        raise SystemExit("bench.py needs a GPU")
    sa.lib()
    wl = WORKLOADS[args.conv_only]
    layers = setup(torch, sa, wl)
    ws = torch.empty(max(256, sa.project_workspace([o.proj for o in layers])), dtype=torch.uint8, device="cuda")
    cws = torch.empty(sa.COMPACT_WS_BYTES, dtype=torch.uint8, device="cuda")
    sa.project([o.proj for o in layers], ws)
    ids = range(len(layers)) if args.layers is None else [int(i) for i in args.layers.split(",")]
    picked = []
    for i in ids:
        o, L = layers[i], layers[i].cfg
        rows = o.mask if (o.kind == sa.FILTER and not args.dense) else None
        cols = o.mask if (o.kind == sa.SHAPE and not args.dense) else None
        inm = None if args.dense else o.in_mask
        c = sa.compact(o.Z, L.groups, row_mask=rows, col_mask=cols, in_ch_mask=inm, in_compacted=inm is not None,
                       ws=cws)
        sizes = o.sizes_c = c[4]
        if inm is not None:  # the input holds the previous layer's kept filters only
            o.Xp = sa.pack_nhwc(o.X, keep=inm)
        else:
            sa.pack_nhwc(o.X, out=o.Xp)
        plan = sa.conv_plan(o.Xp, sizes, L.C, L.D, L.stride, L.pad)
        kern = kernel_of(sa, plan)
        if args.kernel is not None and kern != args.kernel:
            continue
        shape = sa.conv_out_shape(*o.Xp.shape[:3], L.C, L.D, L.stride, L.pad, sizes)
        Y = torch.empty(shape[:3] + (pitch8(sizes),), dtype=torch.uint16, device="cuda")
        cv = torch.empty(max(256, sa.conv_workspace(o.Xp, sizes, L.C, L.D, L.stride, L.pad)),
                         dtype=torch.uint8, device="cuda")
        picked.append((i, o, L, c, Y, cv, plan, kern))
    torch.cuda.synchronize()
    for i, o, L, c, Y, cv, plan, kern in picked:
        for _ in range(args.reps):
            sa.conv_fwd(o.Xp, c[0], c[2], c[3], c[4], L.C, L.D, L.stride, L.pad, Y=Y, ws=cv)
        torch.cuda.synchronize()
        sizes = c[4]
        fl = 2 * wl.batch * L.P * L.Q * sum(sizes.M[g] * kept_k(sizes, g) for g in range(sizes.groups))
        print(json.dumps({"layer": i, "name": L.name, "kernel": kern, "plan": plan, "flops": fl,
                          "bytes": layer_bytes(o), "M": [sizes.M[g] for g in range(sizes.groups)],
                          "K": [kept_k(sizes, g) for g in range(sizes.groups)], "launches": args.reps}), flush=True)


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


def traffic_per_launch(kernel, workload, source="conv.hip", field="bytes per launch"):
    """HBM bytes per launch of `kernel` on `workload` (or another figure of
    its committed counter summary: "kernel µs per launch"), if the summary was
    taken on the current source (else None)."""
    import hashlib
    summ = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_traffic.md")
    src = os.path.join(ROOT, "paper_1807_11091_amd", "csrc", source)
    if not os.path.exists(summ):
        return None
    fields = {}
    for line in open(summ):
        if line.startswith("- ") and ":" in line:
            k, v = line[2:].split(":", 1)
            fields[k.strip()] = v.strip().strip("`")
    digest = hashlib.sha256(open(src, "rb").read()).hexdigest()
    if fields.get(f"{source} sha256") != digest or field not in fields:
        return None
    return float(fields[field]) if "." in fields[field] else int(fields[field])


# ---------------------------------------------------------------- suite
def _time(torch, fn, reps=20, warm=5, trials=5):
    """Per-call time (ms) of reps back-to-back calls between two HIP events on
    the current stream (host enqueue overlaps the GPU work); median, min and
    max over trials."""
    for _ in range(warm):
        fn()
    t = []
    for _ in range(trials):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        torch.cuda.synchronize()
        t.append(a.elapsed_time(b) / reps)
    t.sort()
    return {"median_ms": t[len(t) // 2], "p10_ms": t[0], "p90_ms": t[-1]}


def _time_graph(torch, fn, reps=20, warm=3, trials=5):
    """Per-call GPU time (ms) of fn, from a HIP graph of reps calls replayed
    between two events: no host enqueue gaps (for calls of a few microseconds).
    fn must enqueue on the current stream only; median, min and max over trials."""
    for _ in range(warm):
        fn()
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        fn()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for _ in range(reps):
            fn()
    torch.cuda.synchronize()
    g.replay()
    torch.cuda.synchronize()
    t = []
    for _ in range(trials):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        g.replay()
        b.record()
        torch.cuda.synchronize()
        t.append(a.elapsed_time(b) / reps)
    t.sort()
    del g
    return {"median_ms": t[len(t) // 2], "p10_ms": t[0], "p90_ms": t[-1]}


def suite_tables(torch, sa):
    """Batch-1 CONVs of AlexNet conv1-5 pruned to the per-layer row / column
    sparsities of Tables 1-2 (masks drawn by projecting the synthetic weights),
    against the same-shape dense CONV; GPU times from graph replays."""
    import torch.nn.functional as F
    from workloads import PAPER_TABLE_SPARSITY, WORKLOADS, input_nchw, kept_from_sparsity, layer_tensors
    wl = WORKLOADS["alexnet_shape30"]
    res = {}
    for block, table in PAPER_TABLE_SPARSITY.items():
        rows_out = []
        for li, L in enumerate(wl.layers):
            rs, cs = table[L.name]
            W, U = layer_tensors(wl, li)
            dW, dU = torch.from_numpy(W).cuda(), torch.from_numpy(U).cuda()
            masks = []
            for kind, sp, G in ((sa.FILTER, rs, L.A), (sa.SHAPE, cs, L.K)):
                if sp == 0.0:
                    masks.append(None)
                    continue
                k = kept_from_sparsity(sp, G)
                mask = torch.empty(G, dtype=torch.uint8, device="cuda")
                kept = torch.empty(max(k, 1), dtype=torch.int32, device="cuda")
                lay = sa.ProjectLayer(dW, dU, torch.empty_like(dW), mask, kept, kind, k, L.groups)
                ws = torch.empty(max(256, sa.project_workspace([lay])), dtype=torch.uint8, device="cuda")
                sa.project([lay], ws)
                masks.append(mask)
            Wc, ri, cc, ct, sz = sa.compact(dW, L.groups, row_mask=masks[0], col_mask=masks[1])
            Wd, rid, ccd, ctd, szd = sa.compact(dW, L.groups)
            X = torch.from_numpy(input_nchw(wl, li, batch=1)).cuda()
            Xp = sa.pack_nhwc(X)
            need = max(sa.conv_workspace(Xp, sz, L.C, L.D, L.stride, L.pad),
                       sa.conv_workspace(Xp, szd, L.C, L.D, L.stride, L.pad), 256)
            cws = torch.empty(need, dtype=torch.uint8, device="cuda")
            Yc = sa.conv_fwd(Xp, Wc, cc, ct, sz, L.C, L.D, L.stride, L.pad, ws=cws, ldy=pitch8(sz))
            Yd = sa.conv_fwd(Xp, Wd, ccd, ctd, szd, L.C, L.D, L.stride, L.pad, ws=cws)
            dc = sa.conv_desc(Xp, Wc, cc, ct, sz, L.C, L.D, L.stride, L.pad, Yc, cws, Yc.shape[-1])
            dd = sa.conv_desc(Xp, Wd, ccd, ctd, szd, L.C, L.D, L.stride, L.pad, Yd, cws)
            tc = _time_graph(torch, lambda: sa.conv_fwd(None, None, None, None, sz, 0, 0, 0, 0, desc=dc))
            td = _time_graph(torch, lambda: sa.conv_fwd(None, None, None, None, szd, 0, 0, 0, 0, desc=dd))
            xb, wb = X.to(torch.bfloat16), dW.to(torch.bfloat16)
            conv = lambda: F.conv2d(xb, wb, stride=L.stride, padding=L.pad, groups=L.groups)
            try:
                tm = _time_graph(torch, conv)
            except RuntimeError:  # a library path that cannot be captured: events around eager calls
                torch.cuda.synchronize()
                tm = _time(torch, conv)
            best = min(td["median_ms"], tm["median_ms"])
            fc = 2 * L.P * L.Q * sum(sz.M[g] * kept_k(sz, g) for g in range(sz.groups))
            rows_out.append({"layer": L.name, "row_sparsity_pct": rs, "column_sparsity_pct": cs,
                             "kept_rows": [sz.M[g] for g in range(sz.groups)], "kept_cols": sz.K[0],
                             "compact_us": round(tc["median_ms"] * 1e3, 2), "dense_us": round(td["median_ms"] * 1e3, 2),
                             "miopen_dense_us": round(tm["median_ms"] * 1e3, 2),
                             "speedup_vs_own_dense": round(td["median_ms"] / tc["median_ms"], 3),
                             "speedup_vs_best_dense": round(best / tc["median_ms"], 3),
                             "compact_gflop": round(fc / 1e9, 4)})
        c25 = sum(r["compact_us"] for r in rows_out[1:])
        d25 = sum(r["dense_us"] for r in rows_out[1:])
        b25 = sum(min(r["dense_us"], r["miopen_dense_us"]) for r in rows_out[1:])
        res[block] = {"layers": rows_out, "conv2_5_compact_us": round(c25, 2),
                      "conv2_5_speedup_vs_own_dense": round(d25 / c25, 3),
                      "conv2_5_speedup_vs_best_dense": round(b25 / c25, 3)}
    return res


# LDS gather bound of the sparse CONV: one 2-byte gather per kept weight and
# output pixel; gfx950 serves 32 lanes of a ds_read_u16 per clock per CU
# (measured: a 64-lane u16 read every 2.0 clocks per CU with 16 wavefronts)
LDS_GATHER_PEAK_PRODUCTS = 256 * 32 * 2.4e9


def _element_csr(torch, sa, dW, dU, k, groups):
    """Element-wise projection of (W, U) keeping k weights, then its CSR."""
    Z = torch.empty_like(dW)
    mask = torch.empty(dW.numel(), dtype=torch.uint8, device="cuda")
    kept = torch.empty(max(k, 1), dtype=torch.int32, device="cuda")
    lay = sa.ProjectLayer(dW, dU, Z, mask, kept, sa.ELEMENT, k, groups)
    ws = torch.empty(max(256, sa.project_workspace([lay])), dtype=torch.uint8, device="cuda")
    sa.project([lay], ws)
    return Z, sa.csr(Z, kept, nnz=k)


def _sparse_vs_dense(torch, sa, L, Xp, X, dW, Z, csr, k):
    """Graph-timed sparse CONV of one layer against its own dense CONV (over
    the masked weights) and MIOpen's bf16 conv2d of the same shape."""
    import torch.nn.functional as F
    shape = tuple(dW.shape)
    rp, col, val = csr
    need = max(256, sa.conv_sparse_workspace(Xp, shape, L.groups, L.stride, L.pad, k))
    sws = torch.empty(need, dtype=torch.uint8, device="cuda")
    Ys = sa.conv_sparse_fwd(Xp, rp, col, val, shape, L.groups, L.stride, L.pad, k, ws=sws)
    # the padded entries depend only on the pruned layer and its geometry: built
    # once (first call), reused by the timed CONVs; the full call is timed too
    ds = sa.sparse_conv_desc(Xp, rp, col, val, shape, L.groups, L.stride, L.pad, k, Ys, sws, reuse_ws=True)
    ts = _time_graph(torch, lambda: sa.conv_sparse_fwd(None, None, None, None, shape, 0, 0, 0, k, desc=ds))
    dsf = sa.sparse_conv_desc(Xp, rp, col, val, shape, L.groups, L.stride, L.pad, k, Ys, sws)
    tsf = _time_graph(torch, lambda: sa.conv_sparse_fwd(None, None, None, None, shape, 0, 0, 0, k, desc=dsf))
    Wd, _, ccd, ctd, szd = sa.compact(Z, L.groups)
    cws = torch.empty(max(256, sa.conv_workspace(Xp, szd, L.C, L.D, L.stride, L.pad)), dtype=torch.uint8,
                      device="cuda")
    Yd = sa.conv_fwd(Xp, Wd, ccd, ctd, szd, L.C, L.D, L.stride, L.pad, ws=cws)
    dd = sa.conv_desc(Xp, Wd, ccd, ctd, szd, L.C, L.D, L.stride, L.pad, Yd, cws)
    td = _time_graph(torch, lambda: sa.conv_fwd(None, None, None, None, szd, 0, 0, 0, 0, desc=dd))
    xb, wb = X.to(torch.bfloat16), Z.to(torch.bfloat16)
    conv = lambda: F.conv2d(xb, wb, stride=L.stride, padding=L.pad, groups=L.groups)
    try:
        tm = _time_graph(torch, conv)
    except RuntimeError:  # a library path that cannot be captured: events around eager calls
        torch.cuda.synchronize()
        tm = _time(torch, conv)
    N = X.shape[0]
    products = N * L.P * L.Q * k
    best = min(td["median_ms"], tm["median_ms"])
    return {"kept": k, "density_pct": round(100.0 * k / dW.numel(), 3),
            "sparse_us": round(ts["median_ms"] * 1e3, 2), "sparse_with_prep_us": round(tsf["median_ms"] * 1e3, 2),
            "dense_us": round(td["median_ms"] * 1e3, 2),
            "miopen_dense_us": round(tm["median_ms"] * 1e3, 2),
            "speedup_vs_best_dense": round(best / ts["median_ms"], 3),
            "sparse_useful_tflops": round(2 * products / (ts["median_ms"] * 1e-3) / 1e12, 2),
            "lds_gather_frac": round(products / (ts["median_ms"] * 1e-3) / LDS_GATHER_PEAK_PRODUCTS, 4)}


def suite_sparse(torch, sa):
    """Non-structured pruning through the CSR CONV: (a) the [256,256,3,3] layer
    on 14x14 at batch 256 over a density sweep, with the density where it
    starts to beat the best dense CONV; (b) batch-1 AlexNet conv2-5 pruned to
    the per-layer sparsities of Tables 4 and 5 (Section 5's comparison)."""
    from workloads import PAPER_ELEMENT_SPARSITY, WORKLOADS, input_nchw, kept_count, kept_from_sparsity, layer_tensors
    out = {}
    wl = WORKLOADS["resnet50_s3_sweep"]
    L = wl.layers[0]
    W, U = layer_tensors(wl, 0)
    dW, dU = torch.from_numpy(W).cuda(), torch.from_numpy(U).cuda()
    X = torch.from_numpy(input_nchw(wl, 0)).cuda()
    Xp = sa.pack_nhwc(X)
    sweep = []
    for pct in (50, 25, 10, 6.2, 2.5, 1):
        k = kept_count(pct, W.size) if float(pct).is_integer() else int(pct * W.size / 100 + 0.5)
        Z, csr = _element_csr(torch, sa, dW, dU, k, L.groups)
        r = _sparse_vs_dense(torch, sa, L, Xp, X, dW, Z, csr, k)
        sweep.append(r)
        print("sparse sweep", json.dumps(r), flush=True)
        torch.cuda.empty_cache()
    # density where the speedup crosses 1 (log-linear between neighbours)
    cross = None
    for a, b in zip(sweep, sweep[1:]):
        sa_, sb = a["speedup_vs_best_dense"], b["speedup_vs_best_dense"]
        if (sa_ - 1) * (sb - 1) <= 0 and sa_ != sb:
            la, lb = np.log(a["density_pct"]), np.log(b["density_pct"])
            t = (np.log(sa_) - 0.0) / (np.log(sa_) - np.log(sb))
            cross = round(float(np.exp(la + t * (lb - la))), 3)
            break
    out["layer3_conv2_batch256"] = {"sweep": sweep, "crossover_density_pct": cross}
    del X, Xp
    torch.cuda.empty_cache()
    wa = WORKLOADS["alexnet_shape30"]
    for block, table in PAPER_ELEMENT_SPARSITY.items():
        rows = []
        for li, La in enumerate(wa.layers):
            if table[La.name] == 0.0:
                continue
            Wl, Ul = layer_tensors(wa, li)
            dWl, dUl = torch.from_numpy(Wl).cuda(), torch.from_numpy(Ul).cuda()
            k = kept_from_sparsity(table[La.name], Wl.size)
            Z, csr = _element_csr(torch, sa, dWl, dUl, k, La.groups)
            X1 = torch.from_numpy(input_nchw(wa, li, batch=1)).cuda()
            r = _sparse_vs_dense(torch, sa, La, sa.pack_nhwc(X1), X1, dWl, Z, csr, k)
            r["layer"] = La.name
            r["sparsity_pct"] = table[La.name]
            rows.append(r)
        s25 = sum(r["sparse_us"] for r in rows)
        b25 = sum(min(r["dense_us"], r["miopen_dense_us"]) for r in rows)
        out[block + "_batch1"] = {"layers": rows, "conv2_5_sparse_us": round(s25, 2),
                                  "conv2_5_best_dense_us": round(b25, 2),
                                  "conv2_5_speedup_vs_best_dense": round(b25 / s25, 3)}
        print("sparse", block, json.dumps({k: v for k, v in out[block + "_batch1"].items() if k != "layers"}),
              flush=True)
    return out


def _admm_layers(torch, sa, wl, variant, copies=1):
    """Device tensors of every layer (times copies) for one projection call."""
    from workloads import layer_tensors
    kind, pct = wl.variants[variant]
    layers, grads = [], []
    for _ in range(copies):
        prev = None
        for li, L in enumerate(wl.layers):
            W, U = layer_tensors(wl, li)
            k = wl.k_for(li, kind, pct)
            dW = torch.from_numpy(W).cuda()
            dU = torch.from_numpy(U).cuda()
            dZ, dG, dG2 = torch.empty_like(dW), torch.empty_like(dW), torch.empty_like(dW)
            mask = torch.empty(L.n_groups(kind), dtype=torch.uint8, device="cuda")
            kept = torch.empty(max(k, 1), dtype=torch.int32, device="cuda")
            inm = prev if wl.chain else None
            layers.append(sa.ProjectLayer(dW, dU, dZ, mask, kept, kind, k, L.groups, inm, None, wl.rho, dG))
            grads.append((dW, dZ, dU, wl.rho, dG2, False))
            prev = mask
    return layers, grads


def suite_admm(torch, sa, wl, variant):
    n = sum(L.n for L in wl.layers)
    res = {"n_weights": n, "layers": len(wl.layers)}
    for label, copies in (("one_call", 1), ("replicated", max(1, min(1024, -(-512_000_000 // (20 * n)))))):
        if label == "replicated" and copies == 1:
            res[label] = "one call already moves 512 MB or more"
            continue
        layers, grads = _admm_layers(torch, sa, wl, variant, copies)
        ws = torch.empty(max(256, sa.project_workspace(layers)), dtype=torch.uint8, device="cuda")
        pd, dd = sa._descs(layers), sa.dual_descs(grads)
        tp = _time(torch, lambda: sa.project(layers, ws, descs=pd))
        tg = _time(torch, lambda: sa.dual_update(None, descs=dd))
        # SGD steps on the same layers: the W-subproblem's step (loss gradient
        # plus the ADMM term: read W, Gf, Z, U, write W = 20 B/weight) and the
        # masked-retraining step (read W, Gf, write W = 12 B/weight)
        gfs = [torch.zeros_like(l.W) for l in layers]
        sd_admm = sa.sgd_descs([(l.W, gf, l.Z, l.U, None, l.kind, wl.rho, 1e-3) for l, gf in zip(layers, gfs)])
        sd_mask = sa.sgd_descs([(l.W, gf, None, None, l.mask, l.kind, 0.0, 1e-3) for l, gf in zip(layers, gfs)])
        ts = _time(torch, lambda: sa.sgd_step(None, descs=sd_admm))
        tm = _time(torch, lambda: sa.sgd_step(None, descs=sd_mask))
        nn = n * copies
        step = tp["median_ms"] + tg["median_ms"]
        cold = None
        if label == "one_call":
            # cold: L2 and the 256 MB Infinity Cache flushed (512 MB written) before each call
            flush = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
            def one(fn):
                t = []
                for _ in range(7):
                    flush.fill_(1)
                    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                    a.record()
                    fn()
                    b.record()
                    torch.cuda.synchronize()
                    t.append(a.elapsed_time(b))
                t.sort()
                return t[len(t) // 2]
            cp = one(lambda: sa.project(layers, ws, descs=pd))
            cg = one(lambda: sa.dual_update(None, descs=dd))
            cold = {"project_us": round(cp * 1e3, 2), "gradient_us": round(cg * 1e3, 2),
                    "step_us": round((cp + cg) * 1e3, 2), "step_GBps": round(36 * nn / (cp + cg) / 1e6, 1)}
            del flush
        res[label] = {"copies": copies,
                      "project_us": round(tp["median_ms"] * 1e3, 2), "project_GBps": round(20 * nn / tp["median_ms"] / 1e6, 1),
                      "gradient_us": round(tg["median_ms"] * 1e3, 2), "gradient_GBps": round(16 * nn / tg["median_ms"] / 1e6, 1),
                      "step_us": round(step * 1e3, 2), "step_GBps": round(36 * nn / step / 1e6, 1),
                      "step_frac_of_8TBps": round(36 * nn / step / 1e6 / HBM_PEAK_GBS, 4),
                      "project_min_max_us": [round(tp["p10_ms"] * 1e3, 2), round(tp["p90_ms"] * 1e3, 2)],
                      "sgd_admm_us": round(ts["median_ms"] * 1e3, 2), "sgd_admm_GBps": round(20 * nn / ts["median_ms"] / 1e6, 1),
                      "sgd_masked_us": round(tm["median_ms"] * 1e3, 2), "sgd_masked_GBps": round(12 * nn / tm["median_ms"] / 1e6, 1)}
        if cold is not None:
            res[label]["cold"] = cold
        del layers, grads, ws, gfs
        torch.cuda.empty_cache()
    return res


def suite_conv(torch, sa, wl, variant, layer_ids=None):
    """Per layer: compacted and dense CONV with this library, dense bf16 CONV of MIOpen (torch)."""
    import torch.nn.functional as F
    from workloads import input_nchw, layer_tensors
    kind, pct = wl.variants[variant]
    out, prev = [], None
    ids = range(len(wl.layers)) if layer_ids is None else layer_ids
    for li in ids:
        L = wl.layers[li]
        W, U = layer_tensors(wl, li)
        k = wl.k_for(li, kind, pct)
        dW, dU = torch.from_numpy(W).cuda(), torch.from_numpy(U).cuda()
        dZ = torch.empty_like(dW)
        mask = torch.empty(L.n_groups(kind), dtype=torch.uint8, device="cuda")
        kept = torch.empty(max(k, 1), dtype=torch.int32, device="cuda")
        inm = prev if wl.chain else None
        lay = sa.ProjectLayer(dW, dU, dZ, mask, kept, kind, k, L.groups, inm)
        ws = torch.empty(max(256, sa.project_workspace([lay])), dtype=torch.uint8, device="cuda")
        sa.project([lay], ws)
        rows = mask if kind == sa.FILTER else None
        cols = mask if kind == sa.SHAPE else None
        Wc, ri, cc, ct, sz = sa.compact(dZ, L.groups, row_mask=rows, col_mask=cols, in_ch_mask=inm,
                                        in_compacted=inm is not None)
        Wd, rid, ccd, ctd, szd = sa.compact(dZ, L.groups)
        X = torch.from_numpy(input_nchw(wl, li)).cuda()
        Xc = sa.pack_nhwc(X, keep=inm)
        Xf = sa.pack_nhwc(X)
        need = max(sa.conv_workspace(Xc, sz, L.C, L.D, L.stride, L.pad),
                   sa.conv_workspace(Xf, szd, L.C, L.D, L.stride, L.pad), 256)
        cws = torch.empty(need, dtype=torch.uint8, device="cuda")
        Yc = sa.conv_fwd(Xc, Wc, cc, ct, sz, L.C, L.D, L.stride, L.pad, ws=cws, ldy=pitch8(sz))
        Yd = sa.conv_fwd(Xf, Wd, ccd, ctd, szd, L.C, L.D, L.stride, L.pad, ws=cws)
        dc, dd = sa.conv_desc(Xc, Wc, cc, ct, sz, L.C, L.D, L.stride, L.pad, Yc, cws, Yc.shape[-1]), \
            sa.conv_desc(Xf, Wd, ccd, ctd, szd, L.C, L.D, L.stride, L.pad, Yd, cws)
        tc = _time(torch, lambda: sa.conv_fwd(None, None, None, None, sz, 0, 0, 0, 0, desc=dc), reps=10)
        td = _time(torch, lambda: sa.conv_fwd(None, None, None, None, szd, 0, 0, 0, 0, desc=dd), reps=10)
        xb = X.to(torch.bfloat16)
        wb = dZ.to(torch.bfloat16)
        tm = _time(torch, lambda: F.conv2d(xb, wb, stride=L.stride, padding=L.pad, groups=L.groups), reps=10)
        fc = 2 * wl.batch * L.P * L.Q * sum(sz.M[g] * kept_k(sz, g) for g in range(sz.groups))
        fd = 2 * wl.batch * L.P * L.Q * sum(szd.M[g] * kept_k(szd, g) for g in range(szd.groups))
        best_dense = min(td["median_ms"], tm["median_ms"])
        out.append({"layer": L.name, "compact_us": round(tc["median_ms"] * 1e3, 1),
                    "dense_us": round(td["median_ms"] * 1e3, 1), "miopen_dense_us": round(tm["median_ms"] * 1e3, 1),
                    "compact_tflops": round(fc / tc["median_ms"] / 1e9, 1),
                    "dense_tflops": round(fd / td["median_ms"] / 1e9, 1),
                    "speedup_vs_best_dense": round(best_dense / tc["median_ms"], 3),
                    "compact_gflop": round(fc / 1e9, 3), "dense_gflop": round(fd / 1e9, 3)})
        prev = mask
        del X, Xc, Xf, Yc, Yd, xb, wb, cws
    tot_c = sum(r["compact_us"] for r in out)
    tot_b = sum(min(r["dense_us"], r["miopen_dense_us"]) for r in out)
    gf = sum(r["compact_gflop"] for r in out)
    return {"layers": out, "compact_total_us": round(tot_c, 1), "best_dense_total_us": round(tot_b, 1),
            "compact_tflops": round(gf / tot_c * 1e3, 1), "speedup_vs_best_dense": round(tot_b / tot_c, 3)}


def suite_oracle(wl, variant, images):
    """The oracle on the host: the fused ADMM step of every layer (one thread)
    and the compacted and dense CONV of ``images`` images per layer (OpenMP
    over images)."""
    import oracle
    from workloads import input_nchw, layer_tensors
    kind, pct = wl.variants[variant]
    t_admm, fc, fd, tc, td, prev = 0.0, 0, 0, 0.0, 0.0, None
    for li, L in enumerate(wl.layers):
        W, U = layer_tensors(wl, li)
        k = wl.k_for(li, kind, pct)
        inm = prev if wl.chain else None
        t0 = time.perf_counter()
        r = oracle.project(W, U, kind, k, L.groups, in_ch_mask=inm, rho=wl.rho, fused=True)
        t_admm += time.perf_counter() - t0
        rows = r["mask"] if kind == FILTER_KIND else None
        cols = r["mask"] if kind == SHAPE_KIND else None
        rc = oracle.compact(r["Z"], L.groups, row_mask=rows, col_mask=cols, in_ch_mask=inm,
                            in_compacted=inm is not None)
        rd = oracle.compact(r["Z"], L.groups)
        X = input_nchw(wl, li, batch=images)
        Xc, Xf = oracle.pack(X, keep=inm), oracle.pack(X)
        t0 = time.perf_counter()
        oracle.conv(Xc, rc, L.C, L.D, L.stride, L.pad)
        t1 = time.perf_counter()
        oracle.conv(Xf, rd, L.C, L.D, L.stride, L.pad)
        t2 = time.perf_counter()
        tc += t1 - t0
        td += t2 - t1
        fc += 2 * images * L.P * L.Q * int(np.sum(rc["M"].astype(np.int64) * rc["K"]))
        fd += 2 * images * L.P * L.Q * int(np.sum(rd["M"].astype(np.int64) * rd["K"]))
        prev = r["mask"]
    n = sum(L.n for L in wl.layers)
    threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    return {"fused_step_s_1_thread": round(t_admm, 4), "fused_step_GBps": round(20 * n / t_admm / 1e9, 3),
            "conv_images": images, "conv_threads": min(threads, images),
            "conv_compact_s": round(tc, 3), "conv_compact_GFLOPs": round(fc / tc / 1e9, 2),
            "conv_dense_s": round(td, 3), "conv_dense_GFLOPs": round(fd / td / 1e9, 2)}


def suite(path):
    import torch
    import paper_1807_11091_amd as sa
    from workloads import WORKLOADS
    import dataclasses
    if not torch.cuda.is_available():
        raise SystemExit("bench.py needs a GPU")
    sa.lib()
    prop = torch.cuda.get_device_properties(0)
    rep = {"device": {"name": prop.name, "compute_units": prop.multi_processor_count}}
    # achievable peaks on this machine
    n = 1 << 30
    a = torch.empty(n, dtype=torch.uint8, device="cuda")
    b = torch.empty_like(a)
    t = _time(torch, lambda: b.copy_(a), reps=10)
    rep["achievable"] = {"copy_GBps": round(2 * n / t["median_ms"] / 1e6, 1)}
    del a, b
    m = torch.randn(8192, 8192, device="cuda", dtype=torch.bfloat16)
    t = _time(torch, lambda: torch.matmul(m, m), reps=10)
    rep["achievable"]["bf16_matmul_8192_TFLOPs"] = round(2 * 8192 ** 3 / t["median_ms"] / 1e9, 1)
    del m
    torch.cuda.empty_cache()
    print(json.dumps(rep["achievable"]), flush=True)
    rep["admm"], rep["conv"] = {}, {}
    rep["oracle"] = {}
    for name in ("cifar_conv64", "alexnet_shape30", "alexnet_chain_f50c50", "resnet50_filter60"):
        wl = WORKLOADS[name]
        rep["oracle"][name] = suite_oracle(wl, 0, 4 if name == "resnet50_filter60" else 16)
        print(name, "oracle", json.dumps(rep["oracle"][name]), flush=True)
        rep["admm"][name] = suite_admm(torch, sa, wl, 0)
        print(name, "admm", json.dumps(rep["admm"][name]), flush=True)
        rep["conv"][name] = suite_conv(torch, sa, wl, 0)
        print(name, "conv", json.dumps({k: v for k, v in rep["conv"][name].items() if k != "layers"}), flush=True)
        torch.cuda.empty_cache()
    # ResNet-50 stage-3 layer: every kind at every density, and the extra densities
    wl = WORKLOADS["resnet50_s3_sweep"]
    variants = list(wl.variants) + [(kd, p) for kd in (sa.FILTER, sa.SHAPE) for p in wl.extra_percents]
    rep["sweep"] = []
    for kd, p in variants:
        w = dataclasses.replace(wl, variants=((kd, p),))
        r = {"kind": {0: "filter", 1: "channel", 2: "shape", 3: "element"}[kd], "percent": p,
             "admm": suite_admm(torch, sa, w, 0)["one_call"], "conv": suite_conv(torch, sa, w, 0)["layers"][0]}
        if p in (10, 50):
            r["oracle"] = suite_oracle(w, 0, 8)
        rep["sweep"].append(r)
        print("sweep", json.dumps({"kind": r["kind"], "percent": p, "speedup": r["conv"]["speedup_vs_best_dense"]}),
              flush=True)
        torch.cuda.empty_cache()
    rep["sparse"] = suite_sparse(torch, sa)
    rep["tables_batch1"] = suite_tables(torch, sa)
    print("tables", json.dumps({b: v["conv2_5_speedup_vs_best_dense"] for b, v in rep["tables_batch1"].items()}),
          flush=True)
    with open(path, "w") as f:
        json.dump(rep, f, indent=1)
    print("suite written to", path)


def sparse(path):
    import torch
    import paper_1807_11091_amd as sa
    if not torch.cuda.is_available():
        raise SystemExit("bench.py needs a GPU")
    sa.lib()
    rep = suite_sparse(torch, sa)
    with open(path, "w") as f:
        json.dump(rep, f, indent=1)


def tables(path):
    import torch
    import paper_1807_11091_amd as sa
    if not torch.cuda.is_available():
        raise SystemExit("bench.py needs a GPU")
    sa.lib()
    rep = suite_tables(torch, sa)
    for b, v in rep.items():
        print(b, json.dumps({k: x for k, x in v.items() if k != "layers"}), flush=True)
        for r in v["layers"]:
            print("   ", json.dumps(r), flush=True)
    with open(path, "w") as f:
        json.dump(rep, f, indent=1)


def main():
    args = parse()
    if args.copy_probe:
        copy_probe(args.copy_probe)
        return
    if args.tables:
        tables(args.tables)
        return
    if args.sparse:
        sparse(args.sparse)
        return
    if args.admm:
        import torch
        import paper_1807_11091_amd as sa
        from workloads import WORKLOADS
        if not torch.cuda.is_available():
            raise SystemExit("bench.py needs a GPU")
        sa.lib()
        print(json.dumps({"workload": args.admm, **suite_admm(torch, sa, WORKLOADS[args.admm], 0)}))
        return
    if args.suite:
        suite(args.suite)
        return
    if args.conv_only:
        conv_only(args)
        return
    if args.gpus != 1:
        print(json.dumps({"error": "this build measures one GPU only (one MI355X); "
                                   "multi-GPU runs are not part of it: run with --gpus 1"}))
        sys.exit(2)
    import torch
    import paper_1807_11091_amd as sa
    from workloads import WORKLOADS

    if not torch.cuda.is_available():
        raise SystemExit("bench.py needs a GPU")
    sa.lib()  # fails loudly if the HIP library is missing
    main_res = measure(torch, sa, WORKLOADS[WORKLOAD], args.steps, args.warmup)
    second = measure(torch, sa, WORKLOADS[SECOND_WORKLOAD], max(3, args.steps // 4), max(1, args.warmup))
    warm = admm_warm(torch, sa, WORKLOADS[WORKLOAD])
    progress("library GEMM reference")
    gref = gemm_reference(torch, sa, WORKLOADS[WORKLOAD])
    wl = WORKLOADS[WORKLOAD]
    out = {
        "metric": METRIC,
        "value": main_res["compact_tflops"],
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": main_res["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": WORKLOAD, "layers": "ResNet-50 v1.5, all 53 convolutions, 224x224",
                   "batch": wl.batch, "sparsity": "filter-wise, keep 60% of the filters of every layer",
                   "parallelism": "single GPU"},
        "speedup_vs_dense": main_res["speedup_vs_dense"],
        "dense_conv_tflops": main_res["dense_tflops"],
        "compact_conv_us": main_res["compact_us"],
        "dense_conv_us": main_res["dense_us"],
        "compact_conv_us_layer_events": main_res["compact_us_layer_events"],
        "dense_conv_us_layer_events": main_res["dense_us_layer_events"],
        "admm_gbps": main_res["admm_gbps"],
        "admm_us": main_res["admm_us"],
        "admm_note": "fused projection (20 B/weight) + per-SGD-step gradient (16 B/weight) of all layers, "
                     "one call each, timed inside the step after the previous step's CONVs streamed GBs "
                     "through the caches (cold); admm_warm_* = the same two calls back to back",
        "admm_warm_gbps": warm["step_gbps"],
        "admm_warm_us": warm["step_us"],
        "library_gemm_reference": gref | {"note": "torch.matmul (hipBLASLt) bf16 on each layer's GEMM shape with "
                                                  "the im2col matrix in memory (im2col not timed); context "
                                                  "for the CONV rates, not part of the step"},
        "spin_ms_per_step": main_res["spin_ms_per_step"],
        "gpu_ms_per_step": main_res["gpu_ms_per_step"],
        "per_layer": main_res["per_layer"],
        "compact_by_kernel": main_res["compact_by_kernel"],
        "roofline": main_res["roofline"],
        SECOND_WORKLOAD: {k: second[k] for k in ("compact_tflops", "dense_tflops", "speedup_vs_dense",
                                                 "compact_us", "dense_us", "admm_gbps", "admm_us",
                                                 "ms_per_step", "roofline")},
    }
    if not args.no_cpu_baseline:
        progress("oracle on the host cores")
        out["cpu_baseline"] = cpu_baseline(wl, args.cpu_seconds)
    print(json.dumps(out))


# bytes one launch of the direct / footprint CONV must move at least: the input
# pixels its taps reach (every input channel; a strided kernel narrower than
# its stride skips rows and columns), the compacted weights and the output (bf16)
def layer_bytes(o):
    L = o.cfg
    N, H, W, Cx = o.Xp.shape
    m = sum(o.sizes_c.M[g] for g in range(o.sizes_c.groups))
    kk = sum(o.sizes_c.M[g] * kept_k(o.sizes_c, g) for g in range(o.sizes_c.groups))
    rows, cols = min(H, L.P * L.C), min(W, L.Q * L.D)
    return 2 * N * rows * cols * Cx + 2 * kk + 2 * N * L.P * L.Q * m


def progress(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


# source file of each CONV kernel (its profile summaries hold that file's hash)
KERNEL_SOURCE = {"k_conv": "conv.hip", "k_conv_patch": "conv.hip", "k_ig": "conv_ig.hip"}


def kernel_of(sa, plan):
    """The one kernel a compacted CONV launches, from the library's plan
    (None when it launches more than one: space-to-depth image first, column
    split with a summing pass, gathered im2col rows first, mixed groups)."""
    paths = set(plan["path"]) - {sa.CONV_NONE}
    if len(paths) != 1 or plan["ksplit"] > 1 or plan["space_to_depth"]:
        return None
    p = paths.pop()
    if p == sa.CONV_DIRECT:
        return "k_conv"
    if p == sa.CONV_DIRECT_IG:
        return "k_ig"
    if p == sa.CONV_FOOTPRINT:
        return "k_conv_patch"
    return None


def measure(torch, sa, wl, steps, warmup):
    """Timed steps of one workload; returns the figures of its bench line."""
    progress(f"{wl.name}: generating inputs")
    layers = setup(torch, sa, wl)
    progress(f"{wl.name}: {len(layers)} layers resident, warm-up")
    ws = torch.empty(max(256, sa.project_workspace([o.proj for o in layers])), dtype=torch.uint8, device="cuda")
    # compaction scratch: one range per compacted matrix (kept and dense of every layer)
    cws = torch.empty(2 * len(layers) * sa.COMPACT_WS_BYTES, dtype=torch.uint8, device="cuda")
    ev = {"pdescs": sa._descs([o.proj for o in layers]),
          "ddescs": sa.dual_descs([(o.W, o.Z, o.U, wl.rho, o.G2, False) for o in layers]),
          "lead": lead_cycles(torch, LEAD_US), "lead_conv": 0}
    # untimed steps: size the output and scratch buffers, then the spin ahead
    # of the pack + CONV block from the host's enqueue time of that block
    for _ in range(max(1, warmup)):
        run_step(torch, sa, wl, layers, ws, cws, ev, record="blocks")
        torch.cuda.synchronize()
        lead_us = min(LEAD_CONV_MAX_US, 1.3 * ev["enqueue_s"] * 1e6 + 200)
        ev["lead_conv"] = lead_cycles(torch, lead_us)
    spin_ms = (LEAD_US + lead_us) * 1e-3
    torch.cuda.synchronize()
    progress(f"{wl.name}: timing {steps} steps")

    t0 = time.perf_counter()
    all_marks = []
    for _ in range(steps):
        all_marks.append(run_step(torch, sa, wl, layers, ws, cws, ev, record="blocks"))
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    # the per-layer breakdown: the same steps with every CONV bracketed (each
    # event pair adds its own gap, so these spans sum above the block spans)
    nl = max(2, steps // 4)
    progress(f"{wl.name}: {nl} steps with per-layer events")
    layer_marks = [run_step(torch, sa, wl, layers, ws, cws, ev, record="layers") for _ in range(nl)]
    torch.cuda.synchronize()

    def span(m, a, b):
        return sum(x.elapsed_time(y) for x, y in zip(m[a], m[b]))  # ms

    t_admm = sum(span(m, "admm0", "admm1") for m in all_marks) / steps
    t_pack = sum(span(m, "pack0", "pack1") for m in all_marks) / steps
    t_cblk = sum(span(m, "c_all0", "c_all1") for m in all_marks) / steps
    t_dblk = sum(span(m, "d_all0", "d_all1") for m in all_marks) / steps
    t_c = [sum(span(m, f"c{i}a", f"c{i}b") for m in layer_marks) / nl for i in range(len(layers))]
    t_d = [sum(span(m, f"d{i}a", f"d{i}b") for m in layer_marks) / nl for i in range(len(layers))]
    flops_c = sum(o.flops_c for o in layers)
    flops_d = sum(o.flops_d for o in layers)
    n_el = sum(o.cfg.n for o in layers)
    admm_bytes = 20 * n_el + 16 * n_el  # fused step (W,U read; Z,U,G written) + gradient (W,Z,U read; G written)
    # the dominant kernel of the compacted path: the kernel (from the library's
    # plan of each layer) whose launches take the most time in the step; a
    # layer whose CONV runs more than one kernel is not counted for any
    fam = [kernel_of(sa, o.plan_c) for o in layers]
    by = {}
    for i, f in enumerate(fam):
        if f is not None:
            by.setdefault(f, []).append(i)
    kern = max(by, key=lambda f: sum(t_c[i] for i in by[f]))
    dom = by[kern]
    dom_ms = sum(t_c[i] for i in dom)
    dom_flops = sum(layers[i].flops_c for i in dom)
    dom_tflops = dom_flops / (dom_ms * 1e-3) / 1e12
    dom_bytes = sum(layer_bytes(layers[i]) for i in dom)
    dom_gbps = dom_bytes / (dom_ms * 1e-3) / 1e9
    # the kernel's bound: its launches' algorithmic flops per algorithmic byte
    # against the ridge point of the two peaks (2.5 PFLOP/s / 8 TB/s = 312.5)
    ridge = BF16_PEAK_TFLOPS * 1e12 / (HBM_PEAK_GBS * 1e9)
    hbm_bound = dom_flops / dom_bytes < ridge
    # per-layer roofline min(MFMA, AI * HBM) time over the measured time
    roof_ms = sum(max(layers[i].flops_c / (BF16_PEAK_TFLOPS * 1e12), layer_bytes(layers[i]) / (HBM_PEAK_GBS * 1e9))
                  for i in dom) * 1e3
    by_kernel = {f: {"layers": len(v), "us": round(sum(t_c[i] for i in v) * 1e3, 1),
                     "tflops": round(sum(layers[i].flops_c for i in v) / (sum(t_c[i] for i in v) * 1e-3) / 1e12, 1)}
                 for f, v in by.items()}
    per_layer = [{"layer": o.cfg.name, "compact_us": round(tc * 1e3, 1), "dense_us": round(td * 1e3, 1),
                  "compact_tflops": round(o.flops_c / (tc * 1e-3) / 1e12, 1),
                  "dense_tflops": round(o.flops_d / (td * 1e-3) / 1e12, 1),
                  "speedup": round(td / tc, 2)}
                 for o, tc, td in zip(layers, t_c, t_d)]
    res = {
        "compact_tflops": round(flops_c / (t_cblk * 1e-3) / 1e12, 3),
        "dense_tflops": round(flops_d / (t_dblk * 1e-3) / 1e12, 3),
        "speedup_vs_dense": round(t_dblk / t_cblk, 3),
        "compact_us": round(t_cblk * 1e3, 1),
        "dense_us": round(t_dblk * 1e3, 1),
        "compact_us_layer_events": round(sum(t_c) * 1e3, 1),
        "dense_us_layer_events": round(sum(t_d) * 1e3, 1),
        "admm_gbps": round(admm_bytes / (t_admm * 1e-3) / 1e9, 1),
        "admm_us": round(t_admm * 1e3, 2),
        "pack_us": round(t_pack * 1e3, 1),
        "ms_per_step": round(wall * 1e3 / steps, 4),
        "spin_ms_per_step": round(spin_ms, 3),
        "gpu_ms_per_step": round(t_admm + t_pack + t_cblk + t_dblk, 4),
        "per_layer": per_layer,
        "compact_by_kernel": by_kernel,
        "roofline": {"kernel": f"{kern} (compacted CONVs of {len(dom)} of {len(layers)} layers)",
                     "bound": "hbm" if hbm_bound else "mfma",
                     "achieved": round(dom_gbps, 1) if hbm_bound else round(dom_tflops, 2),
                     "peak": HBM_PEAK_GBS if hbm_bound else BF16_PEAK_TFLOPS,
                     "unit": "GB/s" if hbm_bound else "TFLOP/s",
                     "frac": round(dom_gbps / HBM_PEAK_GBS if hbm_bound else dom_tflops / BF16_PEAK_TFLOPS, 4),
                     "arithmetic_intensity_flop_per_byte": round(dom_flops / dom_bytes, 1),
                     "ridge_flop_per_byte": round(ridge, 1),
                     "achieved_tflops": round(dom_tflops, 2),
                     "frac_of_bf16_peak": round(dom_tflops / BF16_PEAK_TFLOPS, 4),
                     "algorithmic_bytes_per_launch": round(dom_bytes / len(dom)),
                     "avg_launch_us": round(dom_ms * 1e3 / len(dom), 2), "launches_per_step": len(dom),
                     "flops_per_launch": round(dom_flops / len(dom)),
                     "frac_of_layer_roofline": round(roof_ms / dom_ms, 4),
                     "traffic": traffic_per_launch(kern, wl.name, KERNEL_SOURCE[kern]),
                     # the same launches' kernel time alone, from the committed rocprofv3
                     # trace (avg_launch_us holds the gap between launches as well)
                     "profile_kernel_us": traffic_per_launch(kern, wl.name, KERNEL_SOURCE[kern],
                                                             "kernel µs per launch")},
    }
    del layers
    torch.cuda.empty_cache()
    return res


def gemm_reference(torch, sa, wl):
    """Context for the CONV figures: the vendor library's plain bf16 GEMM
    (torch.matmul, i.e. hipBLASLt) on each layer's GEMM shape -- [N*P*Q, K]
    times [K, M] with the im2col matrix already in memory (im2col not timed),
    for the compacted (kept filters) and the dense matrix."""
    kind, pct = wl.variants[0]
    tot = {"compact": [0.0, 0.0], "dense": [0.0, 0.0]}
    for li, L in enumerate(wl.layers):
        npq = wl.batch * L.P * L.Q
        m_c = wl.k_for(li, kind, pct) if kind == sa.FILTER else L.A
        k_c = L.K if kind == sa.FILTER else wl.k_for(li, kind, pct)
        for label, m, k in (("compact", m_c, k_c), ("dense", L.A, L.K)):
            a = torch.randn(npq, k, device="cuda", dtype=torch.bfloat16)
            b = torch.randn(m, k, device="cuda", dtype=torch.bfloat16)
            bt = b.t()
            t = _time(torch, lambda: torch.matmul(a, bt), reps=10, warm=3, trials=3)
            tot[label][0] += 2.0 * npq * m * k
            tot[label][1] += t["median_ms"] * 1e-3
            del a, b, bt
    torch.cuda.empty_cache()
    return {f"{lab}_tflops": round(f / s_ / 1e12, 1) for lab, (f, s_) in tot.items()} | \
        {f"{lab}_us": round(s_ * 1e6, 1) for lab, (f, s_) in tot.items()}


def admm_warm(torch, sa, wl):
    """The two ADMM calls of a step back to back (warm caches)."""
    layers, grads = _admm_layers(torch, sa, wl, 0, 1)
    ws = torch.empty(max(256, sa.project_workspace(layers)), dtype=torch.uint8, device="cuda")
    pd, dd = sa._descs(layers), sa.dual_descs(grads)

    def step():
        sa.project(layers, ws, descs=pd)
        sa.dual_update(None, descs=dd)
    t = _time(torch, step, reps=10)
    n = sum(L.n for L in wl.layers)
    res = {"step_us": round(t["median_ms"] * 1e3, 2), "step_gbps": round(36 * n / t["median_ms"] / 1e6, 1)}
    del layers, grads, ws
    torch.cuda.empty_cache()
    return res


if __name__ == "__main__":
    main()
