"""Throughput of the split-FFT convolution hot path on one MI355X.

Default workload: the 56x56x256 layer with a 5x5 kernel, batch 16,
256 -> 256 channels, stride 1, 'same' padding, fp32, tile T = 28 (FFT size
L = 32), overlap-save; synthetic seeded inputs (ReLU of N(0,1)) and
He-normal weights, resident in device memory before timing starts.

A step is one pass of the hot path over the batch: forward patch
transform -> per-bin contraction -> inverse transform with placement (the
three kernels of fftsplit_conv2d, launched through the stage entry points
so that each can be timed with events on the stream it runs on).  The
filter spectra are computed once, before timing (a once-per-layer cost).

Prints one JSON line (see the fields below).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
FP32_MFMA_PEAK_TFLOPS = 157.3  # MI355X dense fp32 matrix, TFLOP/s

DEFAULT_CONFIG = "c4_56x256_k5"
DEFAULT_TILE = 28
WARMUP_S = 1.0                 # default warm-up: seconds of untimed steps


def warm_up(step, warmup, min_s=WARMUP_S):
    """Untimed steps before timing: `warmup` of them if given, else as many
    as fill `min_s` seconds (at least 10), so that the GPU's clocks have
    settled (a few milliseconds of work measure a GPU still ramping up).
    Returns the number of steps run."""
    import torch
    if warmup is not None:
        for _ in range(warmup):
            step()
        torch.cuda.synchronize()
        return warmup
    n = 0
    t0 = time.perf_counter()
    while True:
        for _ in range(10):
            step()
        n += 10
        torch.cuda.synchronize()
        if time.perf_counter() - t0 >= min_s:
            return n


def algorithmic_counts(layer, info):
    """Algorithmic bytes/flops of each kernel per launch (one batch).

    forward : read x once + write the patch spectra once
    contract: 8 flops per complex multiply-add over the stored complex bins,
              and 2 per real multiply-add for the two slots that each hold
              two real bins, per (patch, input channel, output channel)
    inverse : read the output spectra once + write y once
    """
    F, ntp, coutp = info.bins, info.tiles_padded, info.cout_padded
    nt = info.tiles
    x_bytes = 4 * layer.n * layer.cin * layer.h * layer.w
    y_bytes = 4 * layer.n * layer.cout * layer.h * layer.w
    return {
        "forward_bytes": x_bytes + 8 * F * layer.cin * nt,
        "contract_flops": (8 * (F - 2) + 2 * 2 * 2) * layer.cin * layer.cout * nt,
        "contract_bytes": 8 * F * (layer.cin * nt + layer.cin * layer.cout + layer.cout * nt),
        "inverse_bytes": 8 * F * layer.cout * nt + y_bytes,
    }


def cpu_baseline(layer, x, w, b, tile, budget_s=12.0):
    """Time the CPU oracle's split-FFT convolution on a bounded sample of
    the batch (whole images, until about `budget_s` seconds have passed)."""
    import oracle
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max((p.get("num_threads", 1) for p in threadpool_info()), default=1)
    except Exception:  # pragma: no cover
        blas_threads = 1
    cores = len(os.sched_getaffinity(0))
    done, t_total = 0, 0.0
    while done < layer.n and t_total < budget_s:
        t0 = time.perf_counter()
        oracle.split_conv(x[done:done + 1], w, b, t=tile, mode="os")
        t_total += time.perf_counter() - t0
        done += 1
    per_img = t_total / done
    gflops = layer.direct_flops / layer.n / per_img / 1e9
    # the oracle's direct cross-correlation (eq. 1) on a smaller sample
    d_done, d_total = 0, 0.0
    while d_done < layer.n and d_total < budget_s / 3:
        t0 = time.perf_counter()
        oracle.direct_xcorr2d(x[d_done:d_done + 1], w, b)
        d_total += time.perf_counter() - t0
        d_done += 1
    d_img = d_total / d_done
    return {"value": round(gflops, 3), "unit": "GFLOP/s", "cores": int(min(cores, blas_threads)),
            "kind": "oracle",
            "sample": f"oracle.split_conv (float64 numpy, naive-DFT split, overlap-save) on {done} of "
                      f"{layer.n} images, {t_total:.1f} s; {1.0 / per_img:.3f} images/s; "
                      f"{cores} host cores visible, BLAS threads {blas_threads}",
            "direct_xcorr2d": {"value": round(layer.direct_flops / layer.n / d_img / 1e9, 3), "unit": "GFLOP/s",
                               "sample": f"oracle.direct_xcorr2d (float64 numpy, K*K shifted tensordots) on "
                                         f"{d_done} of {layer.n} images, {d_total:.1f} s; "
                                         f"{1.0 / d_img:.3f} images/s"}}


def load_traffic(kernel, workload_tag):
    """HBM bytes per launch of `kernel` on this workload, from the committed
    rocprofv3 --pmc summary (profiles/traffic.json), if it was taken on the
    kernel's current sources; otherwise None."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    try:
        rec = json.load(open(path)).get(f"{kernel}:{workload_tag}")
        if not rec:
            return None
        from paper_2003_12621_amd.build import source_digest
        if rec.get("source_digest") != source_digest(kernel):
            return None
        return rec.get("bytes_per_launch")
    except Exception:
        return None


def bench_vgg16(args):
    """The 13-layer VGG-16 stack at batch 32 (3x224x224 -> 512x7x7), each
    layer's tile chosen by its plan; a step is one forward of the stack."""
    import torch
    import paper_2003_12621_amd as fs  # noqa: F401
    from paper_2003_12621_amd.vgg import VGG16Stack
    from workloads import VGG16_LAYERS, VGG_BATCH, make_vgg16
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    x, layers = make_vgg16(batch=VGG_BATCH, seed=0)
    stack = VGG16Stack(layers, batch=VGG_BATCH, mode=args.mode)
    xd = torch.from_numpy(x).to(dev)
    args.warmup = warm_up(lambda: stack.forward(xd), args.warmup)
    args.steps = args.steps or 20
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(args.steps):
        stack.forward(xd)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    flops = 0
    for i, (cin, cout, hw) in enumerate(VGG16_LAYERS, start=1):
        flops += 2 * VGG_BATCH * cout * hw * hw * cin * 9
    # per-layer times: further passes with each layer's convolution call
    # timed from its kernels' dispatch timestamps (max-pools included where
    # a layer ends a stage)
    reps = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(13)]
            for _ in range(args.steps)]
    for row in reps:
        for a, b in row:
            a.record()
            b.record()
    torch.cuda.synchronize()
    for row in reps:
        stack.forward(xd, layer_events=row)
    torch.cuda.synchronize()
    per_layer = []
    for i, (cin, cout, hw) in enumerate(VGG16_LAYERS):
        lms = sum(r[i][0].elapsed_time(r[i][1]) for r in reps) / len(reps)
        plan = stack.plans[i]
        per_layer.append({"layer": i + 1, "cin": cin, "cout": cout, "hw": hw, "tile": plan.tile,
                          "pool": bool(plan.pool), "fused_channel_sum": bool(plan.info.fused_channel_sum),
                          "ms": round(lms, 4),
                          "GFLOP/s": round(2 * VGG_BATCH * cout * hw * hw * cin * 9 / (lms * 1e-3) / 1e9, 1)})
    spatial = None
    if not args.no_compare:
        spatial = time_vgg_spatial(args, layers, x, stack)
    out = {"metric": "effective direct-conv GFLOP/s", "value": round(flops / (ms * 1e-3) / 1e9, 1),
           "unit": "GFLOP/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
           "ms_per_step": round(ms, 4), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
           "dtype": "f32", "data": "synthetic",
           "config": {"workload": f"vgg16 conv stack, batch {VGG_BATCH}, 3x224x224, bias+ReLU, 5 max-pools",
                      "tiles": stack.tiles, "mode": args.mode},
           "images_per_s": round(VGG_BATCH / (ms * 1e-3), 1), "layers": per_layer}
    if spatial is not None:
        for v in spatial.values():
            if isinstance(v, dict):
                v["GFLOP/s"] = round(flops / (v["ms"] * 1e-3) / 1e9, 1)
        out["spatial_methods"] = spatial
    print(json.dumps(out), flush=True)


def time_vgg_spatial(args, layers, x, split_stack):
    """The VGG-16 stack by spatial convolution: this library's direct kernel
    (the same stack object, method="direct") and torch's fp32 conv2d +
    max_pool2d (MIOpen).  Returns {name: {"ms": ...}} per forward."""
    import torch
    import torch.nn.functional as F
    from paper_2003_12621_amd.vgg import POOL_AFTER, VGG16Stack
    from workloads import VGG_BATCH

    torch.backends.cudnn.allow_tf32 = False
    dev = split_stack.device
    xd = torch.from_numpy(x).to(dev)
    direct = VGG16Stack(layers, batch=VGG_BATCH, method="direct")
    tw = [(torch.from_numpy(w).to(dev), torch.from_numpy(b).to(dev)) for w, b in layers]

    def torch_stack():
        a = xd
        for i, (w, b) in enumerate(tw, start=1):
            a = F.relu(F.conv2d(a, w, b, padding=1))
            if i in POOL_AFTER:
                a = F.max_pool2d(a, 2)
        return a

    res = {}
    oaa = VGG16Stack(layers, batch=VGG_BATCH, tiles=[3] * 13, mode="oaa")
    for name, fn in (("direct_hip", lambda: direct.forward(xd)), ("torch_conv2d", torch_stack),
                     ("oaaconv", lambda: oaa.forward(xd))):
        warm_up(fn, None, min_s=0.3)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(args.steps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        res[name] = {"ms": round(e0.elapsed_time(e1) / args.steps, 4)}
    ys = split_stack.forward(xd).clone()
    yd = direct.forward(xd).clone()
    yt = torch_stack()
    torch.cuda.synchronize()
    nt = torch.linalg.vector_norm(yt)
    res["direct_hip"]["rel_l2_vs_torch"] = float(torch.linalg.vector_norm(yd - yt) / nt)
    res["split_rel_l2_vs_torch"] = float(torch.linalg.vector_norm(ys - yt) / nt)
    res["oaaconv"]["rel_l2_vs_torch"] = float(torch.linalg.vector_norm(oaa.forward(xd) - yt) / nt)
    return res


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None, help="timed steps (default 100; 20 for vgg16)")
    ap.add_argument("--warmup", type=int, default=None,
                    help=f"untimed steps first (default: as many as fill {WARMUP_S:g} s)")
    ap.add_argument("--config", default=DEFAULT_CONFIG, help="a layer config name, or vgg16")
    ap.add_argument("--shape", default=None,
                    help="any layer instead of a named config: n,cin,h,w,cout,k (ReLU(N(0,1)) inputs, He weights)")
    ap.add_argument("--tile", type=int, default=None)
    ap.add_argument("--mode", default="os", choices=["os", "oaa"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-parity", action="store_true")
    ap.add_argument("--no-cold", action="store_true", help="skip the cold-cache stage timings")
    ap.add_argument("--no-compare", action="store_true",
                    help="skip timing the spatial methods (this library's direct kernel, torch/MIOpen conv2d)")
    ap.add_argument("--copy-probe-mb", type=int, default=0,
                    help="before timing, copy a buffer of this many MiB 3 times (calibrates HBM counters)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py: the library runs on one GPU only (asked for {args.gpus}); the multi-GPU "
              "sharding of the path is a design note, not an implementation.", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2003_12621_amd as fs
    from workloads import CONFIGS, make_config

    if args.config == "vgg16" and not args.shape:
        return bench_vgg16(args)
    if args.shape:
        from workloads import Layer, make_layer
        vals = [int(v) for v in args.shape.split(",")]
        if len(vals) != 6:
            raise SystemExit("--shape takes n,cin,h,w,cout,k")
        layer = Layer(*vals)
        args.config = "shape_" + "x".join(str(v) for v in vals)
        tile = args.tile if args.tile is not None else 0
        make = lambda: make_layer(layer)  # noqa: E731
    else:
        cfg = CONFIGS[args.config]
        layer = cfg["layer"]
        tile = (args.tile if args.tile is not None
                else (DEFAULT_TILE if args.config == DEFAULT_CONFIG else cfg["tiles"][-1]))
        make = lambda: make_config(args.config)  # noqa: E731
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)

    x, w, b = make()
    plan = fs.Plan(layer.n, layer.cin, layer.h, layer.w, layer.cout, layer.k, tile=tile, mode=args.mode,
                   bias=b is not None, device=0)
    info = plan.info
    tile = info.tile
    xd = torch.from_numpy(x).to(dev)
    wd = torch.from_numpy(w).to(dev)
    bd = None if b is None else torch.from_numpy(b).to(dev)
    wspec = plan.transform_weights(wd)
    ws = plan.new_workspace()
    y = plan.new_output()
    if args.copy_probe_mb > 0:
        nbytes = args.copy_probe_mb << 20
        src = torch.ones(nbytes // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    torch.cuda.synchronize()

    def step():
        # one pass of the path: the library's single-call entry point
        plan.conv2d(xd, wspec, bd, out=y, workspace=ws)

    def staged_step(ev):
        # the same pass as three stage calls, each kernel's (start, stop)
        # recorded from its own dispatch timestamps (fftsplit_set_timing_events)
        fs.set_timing_events(ev[0], ev[1])
        plan.forward(xd, ws)
        fs.set_timing_events(ev[2], ev[3])
        plan.contract(wspec, ws)
        fs.set_timing_events(ev[4], ev[5])
        plan.inverse(ws, bias=bd, out=y)
        fs.set_timing_events()

    args.warmup = warm_up(step, args.warmup)
    args.steps = args.steps or 100

    # Timed region: K steps, synchronised on both sides.
    e_start, e_stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_wall = time.perf_counter()
    e_start.record()
    for _ in range(args.steps):
        step()
    e_stop.record()
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_wall
    ms_per_step = e_start.elapsed_time(e_stop) / args.steps

    # Per-kernel durations: K more steps with every kernel timed.  Timing
    # events on every launch lengthen the gaps between kernels (not the
    # kernels), so they are kept out of the region above.
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(6)] for _ in range(args.steps)]
    for row in evs:          # give every event its device handle
        for e in row:
            e.record()
    torch.cuda.synchronize()
    for i in range(args.steps):
        staged_step(evs[i])
    torch.cuda.synchronize()
    fwd = [e[0].elapsed_time(e[1]) for e in evs]
    con = [e[2].elapsed_time(e[3]) for e in evs]
    inv = [e[4].elapsed_time(e[5]) for e in evs]
    ms_per_step_staged = evs[0][0].elapsed_time(evs[-1][5]) / args.steps
    avg = lambda v: sum(v) / len(v)  # noqa: E731

    # Cold-cache stage times: before every stage a 512 MB buffer is read
    # (summed), which fills the 256 MB last-level cache with clean lines, so
    # each stage reads its inputs from HBM (the timings above are warm: a
    # stage may find its input there).
    cold = None
    if not args.no_cold:
        flush = torch.ones(128 << 20, dtype=torch.float32, device=dev)   # 512 MB
        ncold = min(args.steps, 20)
        cev = [[torch.cuda.Event(enable_timing=True) for _ in range(6)] for _ in range(ncold)]
        for row in cev:
            for e in row:
                e.record()
        torch.cuda.synchronize()
        for i in range(ncold):
            ev = cev[i]
            flush.sum()
            fs.set_timing_events(ev[0], ev[1])
            plan.forward(xd, ws)
            fs.set_timing_events()
            flush.sum()
            fs.set_timing_events(ev[2], ev[3])
            plan.contract(wspec, ws)
            fs.set_timing_events()
            flush.sum()
            fs.set_timing_events(ev[4], ev[5])
            plan.inverse(ws, bias=bd, out=y)
            fs.set_timing_events()
        torch.cuda.synchronize()
        cold = [avg([e[2 * j].elapsed_time(e[2 * j + 1]) for e in cev]) for j in range(3)]
        del flush

    counts = algorithmic_counts(layer, info)
    fwd_gbs = counts["forward_bytes"] / (avg(fwd) * 1e-3) / 1e9
    inv_gbs = counts["inverse_bytes"] / (avg(inv) * 1e-3) / 1e9
    con_tfs = counts["contract_flops"] / (avg(con) * 1e-3) / 1e12
    value = layer.direct_flops / (ms_per_step * 1e-3) / 1e9

    # Parity of the timed output against the oracle on sampled output channels.
    parity = None
    if not args.no_parity:
        import oracle
        rng = np.random.default_rng(99)
        sel = np.sort(rng.choice(layer.cout, size=4, replace=False))
        imgs = slice(0, min(layer.n, 4))
        ref = oracle.direct_xcorr2d(x[imgs], w[sel], None if b is None else b[sel])
        got = y.cpu().numpy()[imgs][:, sel].astype(np.float64)
        parity = float(np.linalg.norm(got - ref) / np.linalg.norm(ref))

    wtag = f"{args.config}_T{tile}_{args.mode}"
    traffic = load_traffic("contract", wtag)
    out = {
        "metric": "effective direct-conv GFLOP/s",
        "value": round(value, 1),
        "unit": "GFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": f"{args.config}: n={layer.n} cin={layer.cin} {layer.h}x{layer.w} "
                               f"cout={layer.cout} k={layer.k} stride1 same",
                   "tile": info.tile, "nfft": info.nfft, "mode": args.mode, "tiles": info.tiles,
                   "bins": info.bins,
                   "contract_variant": f"{info.contract_tile_m}x{info.contract_tile_n}x{info.contract_stage_k}"
                                       f"/{info.contract_real_products}M/prefetch{info.contract_prefetch}"},
        "images_per_s": round(layer.n / (ms_per_step * 1e-3), 1),
        "roofline": {"bound": "mfma", "kernel": "contract (per-bin complex Cin->Cout product)",
                     "achieved": round(con_tfs, 2), "peak": FP32_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(con_tfs / FP32_MFMA_PEAK_TFLOPS, 4), "traffic": traffic,
                     "flops_per_complex_mac": 8,
                     "mfma_real_products_per_complex_mac": info.contract_real_products,
                     "mfma_executed_frac": round(con_tfs * info.contract_real_products / 4
                                                 / FP32_MFMA_PEAK_TFLOPS, 4)},
        "stages": {
            "forward": {"ms": round(avg(fwd), 4), "GB/s": round(fwd_gbs, 1),
                        "frac_hbm": round(fwd_gbs / HBM_PEAK_GBS, 4), "bytes": counts["forward_bytes"],
                        "traffic": load_traffic("forward", wtag)},
            "contract": {"ms": round(avg(con), 4), "TFLOP/s": round(con_tfs, 2),
                         "frac_mfma": round(con_tfs / FP32_MFMA_PEAK_TFLOPS, 4),
                         "flops": counts["contract_flops"], "bytes": counts["contract_bytes"]},
            "inverse": {"ms": round(avg(inv), 4), "GB/s": round(inv_gbs, 1),
                        "frac_hbm": round(inv_gbs / HBM_PEAK_GBS, 4), "bytes": counts["inverse_bytes"],
                        "traffic": load_traffic("inverse", wtag)},
        },
        "stages_cold": None if cold is None else {
            "forward": {"ms": round(cold[0], 4), "frac_hbm": round(counts["forward_bytes"] / (cold[0] * 1e-3) / 1e9
                                                                 / HBM_PEAK_GBS, 4)},
            "contract": {"ms": round(cold[1], 4), "frac_mfma": round(counts["contract_flops"] / (cold[1] * 1e-3)
                                                                     / 1e12 / FP32_MFMA_PEAK_TFLOPS, 4)},
            "inverse": {"ms": round(cold[2], 4), "frac_hbm": round(counts["inverse_bytes"] / (cold[2] * 1e-3) / 1e9
                                                                 / HBM_PEAK_GBS, 4)},
            "note": "each stage after a 512 MB read has replaced the last-level cache's contents"},
        "timing": "ms_per_step: K fftsplit_conv2d calls between two events on the launch stream, after "
                  "a warm-up that lets the clocks settle; stage times: K further steps as three stage calls "
                  "with each kernel's start/stop taken from its dispatch timestamps (hipExtLaunchKernel events)",
        "ms_per_step_staged": round(ms_per_step_staged, 4),
        "wall_s_timed": round(t_wall, 4),
        "parity_rel_l2": parity,
    }
    if not args.no_compare:
        out["spatial_methods"] = time_spatial_methods(args, plan, layer, xd, wd, bd)
        out["oaaconv"] = time_oaaconv(args, layer, xd, wd, bd)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(layer, x, w, b, tile)
    print(json.dumps(out), flush=True)


def time_oaaconv(args, layer, xd, wd, bd):
    """The same layer by OaAConv, the paper's comparison method (Section 2,
    Fig. 1): this library's overlap-add pipeline at T = K, L = 2K - 1, timed
    like the split path (K conv2d steps; stage times from a staged pass)."""
    import torch
    import paper_2003_12621_amd as fs
    k = layer.k
    plan = fs.Plan(layer.n, layer.cin, layer.h, layer.w, layer.cout, k, tile=k, mode="oaa", bias=bd is not None,
                   device=0)
    wspec = plan.transform_weights(wd)
    ws = plan.new_workspace()
    y = plan.new_output()
    warm_up(lambda: plan.conv2d(xd, wspec, bd, out=y, workspace=ws), None, min_s=0.3)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(args.steps):
        plan.conv2d(xd, wspec, bd, out=y, workspace=ws)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(6)]
    for e in ev:
        e.record()
    torch.cuda.synchronize()
    fs.set_timing_events(ev[0], ev[1])
    plan.forward(xd, ws)
    fs.set_timing_events(ev[2], ev[3])
    plan.contract(wspec, ws)
    fs.set_timing_events(ev[4], ev[5])
    plan.inverse(ws, bias=bd, out=y)
    fs.set_timing_events()
    torch.cuda.synchronize()
    info = plan.info
    return {"ms": round(ms, 4), "GFLOP/s": round(layer.direct_flops / (ms * 1e-3) / 1e9, 1),
            "tile": info.tile, "nfft": info.nfft, "tiles": info.tiles, "bins": info.bins,
            "contract_flops": (8 * info.bins) * layer.cin * layer.cout * info.tiles,
            "stage_ms": {"forward": round(ev[0].elapsed_time(ev[1]), 4),
                         "contract": round(ev[2].elapsed_time(ev[3]), 4),
                         "inverse_and_seams": round(ev[4].elapsed_time(ev[5]), 4)}}


def time_spatial_methods(args, plan, layer, xd, wd, bd):
    """The same layer by spatial convolution, timed the same way (context for
    the split method's speed, as the paper sets it beside direct convolution):
    this library's direct kernel (fftsplit_direct_conv2d) and torch's fp32
    conv2d (MIOpen), both on torch's current stream."""
    import torch
    import torch.nn.functional as F

    torch.backends.cudnn.allow_tf32 = False
    wdir = plan.direct_transform_weights(wd)
    yd = plan.new_output()
    res = {}
    runs = {"direct_hip": lambda: plan.direct_conv2d(xd, wdir, bd, out=yd),
            "torch_conv2d": lambda: F.conv2d(xd, wd, bd, padding=layer.k // 2)}
    for name, fn in runs.items():
        warm_up(fn, None, min_s=0.3)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(args.steps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / args.steps
        res[name] = {"ms": round(ms, 4), "GFLOP/s": round(layer.direct_flops / (ms * 1e-3) / 1e9, 1)}
    yt = F.conv2d(xd, wd, bd, padding=layer.k // 2)
    torch.cuda.synchronize()
    res["direct_hip"]["rel_l2_vs_torch"] = float(torch.linalg.vector_norm(yd - yt) / torch.linalg.vector_norm(yt))
    return res


if __name__ == "__main__":
    main()
