"""Throughput of the split-FFT convolution hot path on one MI355X.

Default workload: the 56x56x256 layer with a 5x5 kernel, batch 16,
256 -> 256 channels, stride 1, 'same' padding, fp32, tile T = 28 (FFT size
L = 32), overlap-save; synthetic seeded inputs (ReLU of N(0,1)) and
He-normal weights, resident in device memory before timing starts.

A step is one pass of the hot path over the batch: one fftsplit_conv2d call
(forward patch transform -> per-bin contraction -> inverse transform with
placement).  The filter spectra are computed once, before timing (a
once-per-layer cost).

Order of a run: an untimed clock-settle pre-roll (steps for --settle-s
seconds, reported as settle_s / settle_steps: a GPU given only a few
milliseconds of work is still raising its clocks), then --warmup counted
warm-up steps, then exactly --steps timed steps between two events on the
launch stream, synchronised on both sides.  Per-kernel times come from a
separate pass of the same steps made of the three stage calls.

Prints one JSON line.  Besides the headline layer it carries, under
"workloads", settled step times and stage fractions of the other single
layers (1x3x32^2 -> 16 K3; 1x64x224^2 -> 64 K3 at T = 6/14/30;
8x128x112^2 -> 128 K3 at T = 14/30; the headline layer at T = 12) and of
the VGG-16 stack at batch 32.
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
SETTLE_S = 1.0                 # untimed clock-settle pre-roll, seconds
DEFAULT_WARMUP = 10
DEFAULT_STEPS = 100

# the other workloads reported beside the headline layer: (config, tile)
OTHER_LAYERS = [("c1_32x3", 6), ("c2_224x64", 6), ("c2_224x64", 14), ("c2_224x64", 30),
                ("c3_112x128", 14), ("c3_112x128", 30), ("c4_56x256_k5", 12)]


def _sync():
    import torch
    torch.cuda.synchronize()


def settle(step, seconds):
    """Untimed steps until `seconds` have passed (batches of 10), so that the
    GPU's clocks have settled.  Returns (steps run, seconds spent)."""
    if seconds <= 0:
        return 0, 0.0
    n = 0
    t0 = time.perf_counter()
    while True:
        for _ in range(10):
            step()
        n += 10
        _sync()
        el = time.perf_counter() - t0
        if el >= seconds:
            return n, el


def warm_up(step, count):
    for _ in range(count):
        step()
    _sync()


def timed_steps(step, steps):
    """Exactly `steps` calls between two events on the current stream,
    synchronised on both sides; returns (ms per step, wall seconds)."""
    import torch
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    _sync()
    t = time.perf_counter()
    e0.record()
    for _ in range(steps):
        step()
    e1.record()
    _sync()
    return e0.elapsed_time(e1) / steps, time.perf_counter() - t


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def algorithmic_counts(layer, info):
    """Algorithmic bytes/flops of each kernel per launch (one batch).

    forward : read x once + write the patch spectra once
    contract: 8 flops per complex multiply-add over the stored complex bins,
              and 2 per real multiply-add for the two slots that each hold
              two real bins, per (patch, input channel, output channel)
    inverse : read the output spectra once + write y once
    """
    F = info.bins
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
    model = cpu_model()
    return {"value": round(gflops, 3), "unit": "GFLOP/s", "cores": int(min(cores, blas_threads)),
            "kind": "oracle", "cpu_model": model,
            "sample": f"oracle.split_conv (float64 numpy, naive-DFT split, overlap-save) on {done} of "
                      f"{layer.n} images, {t_total:.1f} s; {1.0 / per_img:.3f} images/s; "
                      f"{cores} host cores visible ({model}), BLAS threads {blas_threads}",
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


class LayerRun:
    """One layer's plan, filter spectra, workspace and output, with the
    inputs resident on the device."""

    def __init__(self, layer, x, w, b, tile, mode, dev):
        import torch
        import paper_2003_12621_amd as fs
        self.fs = fs
        self.layer = layer
        self.plan = fs.Plan(layer.n, layer.cin, layer.h, layer.w, layer.cout, layer.k, tile=tile, mode=mode,
                            bias=b is not None, device=dev.index)
        self.info = self.plan.info
        self.xd = torch.from_numpy(x).to(dev)
        self.wd = torch.from_numpy(w).to(dev)
        self.bd = None if b is None else torch.from_numpy(b).to(dev)
        self.wspec = self.plan.transform_weights(self.wd)
        self.ws = self.plan.new_workspace()
        self.y = self.plan.new_output()
        _sync()

    def step(self):
        # one pass of the path: the library's single-call entry point
        self.plan.conv2d(self.xd, self.wspec, self.bd, out=self.y, workspace=self.ws)

    def stage_times(self, steps):
        """Per-kernel durations over `steps` passes made of the three stage
        calls, each kernel's (start, stop) recorded from its own dispatch
        timestamps (fftsplit_set_timing_events).  Timing every launch
        lengthens the gaps between kernels, not the kernels."""
        import torch
        fs, plan = self.fs, self.plan
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(6)] for _ in range(steps)]
        for row in evs:          # give every event its device handle
            for e in row:
                e.record()
        _sync()
        for ev in evs:
            fs.set_timing_events(ev[0], ev[1])
            plan.forward(self.xd, self.ws)
            fs.set_timing_events(ev[2], ev[3])
            plan.contract(self.wspec, self.ws)
            fs.set_timing_events(ev[4], ev[5])
            plan.inverse(self.ws, bias=self.bd, out=self.y)
            fs.set_timing_events()
        _sync()
        fwd = [e[0].elapsed_time(e[1]) for e in evs]
        con = [e[2].elapsed_time(e[3]) for e in evs]
        inv = [e[4].elapsed_time(e[5]) for e in evs]
        staged = evs[0][0].elapsed_time(evs[-1][5]) / steps
        return fwd, con, inv, staged

    def cold_stage_times(self, steps):
        """Stage times with a cold last-level cache: before every stage a
        512 MB buffer is read (summed), which fills the 256 MB cache with
        clean lines, so each stage reads its inputs from HBM."""
        import torch
        fs, plan = self.fs, self.plan
        flush = torch.ones(128 << 20, dtype=torch.float32, device=self.xd.device)   # 512 MB
        cev = [[torch.cuda.Event(enable_timing=True) for _ in range(6)] for _ in range(steps)]
        for row in cev:
            for e in row:
                e.record()
        _sync()
        for ev in cev:
            flush.sum()
            fs.set_timing_events(ev[0], ev[1])
            plan.forward(self.xd, self.ws)
            fs.set_timing_events()
            flush.sum()
            fs.set_timing_events(ev[2], ev[3])
            plan.contract(self.wspec, self.ws)
            fs.set_timing_events()
            flush.sum()
            fs.set_timing_events(ev[4], ev[5])
            plan.inverse(self.ws, bias=self.bd, out=self.y)
            fs.set_timing_events()
        _sync()
        del flush
        return [sum(e[2 * j].elapsed_time(e[2 * j + 1]) for e in cev) / steps for j in range(3)]

    def parity(self, x, w, b, images, channels):
        """rel-L2 of the last output against the oracle on the given images
        and output channels."""
        import oracle
        ref = oracle.direct_xcorr2d(x[images], w[channels], None if b is None else b[channels])
        got = self.y.cpu().numpy()[images][:, channels].astype(np.float64)
        return float(np.linalg.norm(got - ref) / np.linalg.norm(ref))


def _avg(v):
    return sum(v) / len(v)


def dispatch_events(n):
    """n (start, stop) pairs of timing events for fftsplit_set_timing_events
    (each recorded once so that it has a device handle), the way the stage
    times are taken: from the kernels' own dispatch timestamps."""
    import torch
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n)]
    for a, b in ev:
        a.record()
        b.record()
    _sync()
    return ev


def hbm_floor(dev, mixes, steps=20):
    """What HBM sustains for each transform's byte mix on this GPU: the
    library's streaming probe (fftsplit_probe_stream: a plain kernel that
    reads R and writes W bytes from 8192 workgroups) timed like the stages
    (dispatch timestamps), warm (its input just read by the previous run)
    and cold (after a 512 MB read has replaced the last-level cache's
    contents), median of `steps` launches.
    `mixes`: {name: (R, W)}."""
    import torch
    import paper_2003_12621_amd as fs
    r16 = lambda b: (int(b) + 15) // 16 * 16  # noqa: E731
    big = max(max(r16(r), r16(w)) for r, w in mixes.values())
    src = torch.ones(big // 4 + 64, dtype=torch.float32, device=dev)
    dst = torch.empty(big // 4 + 64, dtype=torch.float32, device=dev)
    flush = torch.ones(128 << 20, dtype=torch.float32, device=dev)   # 512 MB

    def timed(r, w, cold):
        ev = dispatch_events(steps)
        fs.probe_stream(src, dst, r, w)
        _sync()
        for a, b in ev:
            if cold:
                flush.sum()
            fs.set_timing_events(a, b)
            fs.probe_stream(src, dst, r, w)
            fs.set_timing_events()
        _sync()
        ts = sorted(a.elapsed_time(b) for a, b in ev)
        return ts[len(ts) // 2] * 1e3   # median, us

    out = {}
    for cold in (False, True):
        tag = "cold" if cold else "warm"
        out[tag] = {}
        for name, (r, w) in mixes.items():
            t = timed(r16(r), r16(w), cold)
            out[tag][f"{name}_floor_us"] = round(t, 2)
            out[tag][f"{name}_floor_frac_hbm"] = round((r + w) / (t * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)
    # the same kernel moving 16 bytes: the fixed cost of one launch, timed this way
    out["launch_us"] = round(timed(16, 16, False), 2)
    del src, dst, flush
    out["note"] = ("fftsplit_probe_stream (plain streaming kernel, 8192 workgroups) moving each transform's read "
                   "and write bytes, timed from its dispatch timestamps like the stages; median of 20 launches; "
                   "cold = after a 512 MB read; launch_us: the same kernel moving 16 bytes")
    return out


def matrix_ceiling(run, con_ms, steps=20):
    """What the fp32 matrix cores sustain for the contraction's launch: the
    library's matrix probe (fftsplit_probe_matrix: the same grid and
    occupancy, the same matrix operations per wave, operands in registers,
    no memory traffic), timed like the stages, median of `steps` launches."""
    import torch
    plan, i = run.plan, run.info
    sink = plan.probe_matrix()
    for _ in range(3):
        plan.probe_matrix(sink)
    _sync()
    ev = dispatch_events(steps)
    for a, b in ev:
        run.fs.set_timing_events(a, b)
        plan.probe_matrix(sink)
        run.fs.set_timing_events()
    _sync()
    ts = sorted(a.elapsed_time(b) for a, b in ev)
    probe_us = ts[len(ts) // 2] * 1e3
    kc = i.contract_stage_k
    executed = 2 * i.contract_real_products * i.bins * i.cout_padded * i.tiles_padded * (-(-run.layer.cin // kc) * kc)
    return {"probe_us": round(probe_us, 2), "contract_us": round(con_ms * 1e3, 2),
            "executed_flops": executed,
            "probe_frac_of_peak": round(executed / (probe_us * 1e-6) / 1e12 / FP32_MFMA_PEAK_TFLOPS, 4),
            "contract_vs_probe": round(probe_us / (con_ms * 1e3), 4),
            "note": "fftsplit_probe_matrix: the contraction's grid, occupancy and matrix operations per wave with "
                    "no memory traffic; contract_vs_probe = probe time / contraction time (warm)"}


def stage_record(counts, fwd, con, inv):
    fwd_gbs = counts["forward_bytes"] / (fwd * 1e-3) / 1e9
    inv_gbs = counts["inverse_bytes"] / (inv * 1e-3) / 1e9
    con_tfs = counts["contract_flops"] / (con * 1e-3) / 1e12
    return {
        "forward": {"ms": round(fwd, 4), "GB/s": round(fwd_gbs, 1), "frac_hbm": round(fwd_gbs / HBM_PEAK_GBS, 4),
                    "bytes": counts["forward_bytes"]},
        "contract": {"ms": round(con, 4), "TFLOP/s": round(con_tfs, 2),
                     "frac_mfma": round(con_tfs / FP32_MFMA_PEAK_TFLOPS, 4), "flops": counts["contract_flops"],
                     "bytes": counts["contract_bytes"]},
        "inverse": {"ms": round(inv, 4), "GB/s": round(inv_gbs, 1), "frac_hbm": round(inv_gbs / HBM_PEAK_GBS, 4),
                    "bytes": counts["inverse_bytes"]},
    }


def other_layer(name, tile, dev, steps=20, settle_s=0.25, oracle_budget_s=0.0):
    """A short settled measurement of another single layer: step time,
    effective GFLOP/s, images/s and stage fractions, and the oracle's
    rel-L2 on a sample of the output."""
    from workloads import CONFIGS, make_config
    layer = CONFIGS[name]["layer"]
    x, w, b = make_config(name)
    run = LayerRun(layer, x, w, b, tile, "os", dev)
    settle(run.step, settle_s)
    warm_up(run.step, 5)
    ms, _ = timed_steps(run.step, steps)
    fwd, con, inv, _ = run.stage_times(steps)
    counts = algorithmic_counts(layer, run.info)
    chans = sorted({0, layer.cout // 2, layer.cout - 1})
    rec = {"workload": f"n={layer.n} cin={layer.cin} {layer.h}x{layer.w} cout={layer.cout} k={layer.k}",
           "tile": run.info.tile, "nfft": run.info.nfft, "steps": steps, "ms_per_step": round(ms, 4),
           "GFLOP/s": round(layer.direct_flops / (ms * 1e-3) / 1e9, 1),
           "images_per_s": round(layer.n / (ms * 1e-3), 1),
           "stages": stage_record(counts, _avg(fwd), _avg(con), _avg(inv)),
           "fused_channel_sum": bool(run.info.fused_channel_sum),
           "parity_rel_l2": run.parity(x, w, b, slice(0, 1), chans)}
    del run
    if oracle_budget_s > 0:
        rec["cpu_oracle"] = cpu_baseline(layer, x, w, b, tile, budget_s=oracle_budget_s)
    return rec


def vgg16_summary(dev, steps=10, settle_s=0.5, oracle_timed=False):
    """The VGG-16 stack at batch 32 (plan-chosen tiles, fused max-pools):
    settled step time, effective GFLOP/s, images/s, per-layer times."""
    import torch
    from paper_2003_12621_amd.vgg import VGG16Stack
    from workloads import VGG16_LAYERS, VGG_BATCH, make_vgg16
    x, layers = make_vgg16(batch=VGG_BATCH, seed=0)
    stack = VGG16Stack(layers, batch=VGG_BATCH)
    xd = torch.from_numpy(x).to(dev)
    fwd = lambda: stack.forward(xd)  # noqa: E731
    settle(fwd, settle_s)
    warm_up(fwd, 3)
    ms, _ = timed_steps(fwd, steps)
    flops = sum(2 * VGG_BATCH * cout * hw * hw * cin * 9 for cin, cout, hw in VGG16_LAYERS)
    reps = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(13)]
            for _ in range(steps)]
    for row in reps:
        for a, b in row:
            a.record()
            b.record()
    _sync()
    for row in reps:
        stack.forward(xd, layer_events=row)
    _sync()
    layer_ms = [round(sum(r[i][0].elapsed_time(r[i][1]) for r in reps) / steps, 4) for i in range(13)]
    # final activation of image 0 against the float64 chain
    import oracle
    got = stack.forward(xd)[:1].cpu().numpy().astype(np.float64)
    t0 = time.perf_counter()
    ref = oracle.vgg16_forward(x[:1], layers)
    t_ref = time.perf_counter() - t0
    rec = {"workload": f"vgg16 conv stack, batch {VGG_BATCH}, 3x224x224, bias+ReLU, 5 max-pools",
            "tiles": stack.tiles, "steps": steps, "ms_per_step": round(ms, 4),
            "GFLOP/s": round(flops / (ms * 1e-3) / 1e9, 1), "images_per_s": round(VGG_BATCH / (ms * 1e-3), 1),
            "layer_ms": layer_ms,
            "parity_rel_l2_image0": float(np.linalg.norm(got - ref) / np.linalg.norm(ref))}
    if oracle_timed:
        rec["cpu_oracle"] = {"value": round(flops / VGG_BATCH / t_ref / 1e9, 3), "unit": "GFLOP/s", "kind": "oracle",
                             "sample": f"oracle.vgg16_forward (float64 numpy, direct cross-correlation per layer) "
                                       f"on 1 of {VGG_BATCH} images, {t_ref:.1f} s; {1.0 / t_ref:.3f} images/s"}
    return rec


def bench_vgg16(args):
    """--config vgg16: the 13-layer VGG-16 stack at batch 32 as the step."""
    import torch
    from paper_2003_12621_amd.vgg import VGG16Stack
    from workloads import VGG16_LAYERS, VGG_BATCH, make_vgg16
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    x, layers = make_vgg16(batch=VGG_BATCH, seed=0)
    stack = VGG16Stack(layers, batch=VGG_BATCH, mode=args.mode)
    xd = torch.from_numpy(x).to(dev)
    step = lambda: stack.forward(xd)  # noqa: E731
    settle_n, settle_s = settle(step, args.settle_s)
    warm_up(step, args.warmup)
    steps = args.steps or 20
    ms, wall = timed_steps(step, steps)
    flops = sum(2 * VGG_BATCH * cout * hw * hw * cin * 9 for cin, cout, hw in VGG16_LAYERS)
    out = {"metric": "effective direct-conv GFLOP/s", "value": round(flops / (ms * 1e-3) / 1e9, 1),
           "unit": "GFLOP/s", "n_gpus": 1, "steps": steps, "warmup": args.warmup,
           "ms_per_step": round(ms, 4), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
           "dtype": "f32", "data": "synthetic",
           "config": {"workload": f"vgg16 conv stack, batch {VGG_BATCH}, 3x224x224, bias+ReLU, 5 max-pools",
                      "tiles": stack.tiles, "mode": args.mode},
           "images_per_s": round(VGG_BATCH / (ms * 1e-3), 1), "settle_s": round(settle_s, 3),
           "settle_steps": settle_n, "wall_s_timed": round(wall, 4)}
    if not args.no_compare:
        spatial = time_vgg_spatial(args, layers, x, stack)
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
    steps = args.steps or 20
    for name, fn in (("direct_hip", lambda: direct.forward(xd)), ("torch_conv2d", torch_stack),
                     ("oaaconv", lambda: oaa.forward(xd))):
        settle(fn, 0.3)
        ms, _ = timed_steps(fn, steps)
        res[name] = {"ms": round(ms, 4)}
    ys = split_stack.forward(xd).clone()
    yd = direct.forward(xd).clone()
    yt = torch_stack()
    _sync()
    nt = torch.linalg.vector_norm(yt)
    res["direct_hip"]["rel_l2_vs_torch"] = float(torch.linalg.vector_norm(yd - yt) / nt)
    res["split_rel_l2_vs_torch"] = float(torch.linalg.vector_norm(ys - yt) / nt)
    res["oaaconv"]["rel_l2_vs_torch"] = float(torch.linalg.vector_norm(oaa.forward(xd) - yt) / nt)
    return res


def time_oaaconv(steps, layer, xd, wd, bd):
    """The same layer by OaAConv, the paper's comparison method (Section 2,
    Fig. 1): this library's overlap-add pipeline at T = K, L = 2K - 1, timed
    like the split path (conv2d steps; stage times from a staged pass)."""
    import torch
    import paper_2003_12621_amd as fs
    k = layer.k
    plan = fs.Plan(layer.n, layer.cin, layer.h, layer.w, layer.cout, k, tile=k, mode="oaa", bias=bd is not None,
                   device=0)
    wspec = plan.transform_weights(wd)
    ws = plan.new_workspace()
    y = plan.new_output()
    step = lambda: plan.conv2d(xd, wspec, bd, out=y, workspace=ws)  # noqa: E731
    settle(step, 0.3)
    ms, _ = timed_steps(step, steps)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(6)]
    for e in ev:
        e.record()
    _sync()
    fs.set_timing_events(ev[0], ev[1])
    plan.forward(xd, ws)
    fs.set_timing_events(ev[2], ev[3])
    plan.contract(wspec, ws)
    fs.set_timing_events(ev[4], ev[5])
    plan.inverse(ws, bias=bd, out=y)
    fs.set_timing_events()
    _sync()
    info = plan.info
    return {"ms": round(ms, 4), "GFLOP/s": round(layer.direct_flops / (ms * 1e-3) / 1e9, 1),
            "tile": info.tile, "nfft": info.nfft, "tiles": info.tiles, "bins": info.bins,
            "contract_flops": (8 * info.bins) * layer.cin * layer.cout * info.tiles,
            "stage_ms": {"forward": round(ev[0].elapsed_time(ev[1]), 4),
                         "contract": round(ev[2].elapsed_time(ev[3]), 4),
                         "inverse_and_seams": round(ev[4].elapsed_time(ev[5]), 4)}}


def time_spatial_methods(steps, run):
    """The same layer by spatial convolution, timed the same way (context for
    the split method's speed, as the paper sets it beside direct convolution):
    this library's direct kernel (fftsplit_direct_conv2d) and torch's fp32
    conv2d (MIOpen), both on torch's current stream."""
    import torch
    import torch.nn.functional as F

    torch.backends.cudnn.allow_tf32 = False
    plan, layer, xd, wd, bd = run.plan, run.layer, run.xd, run.wd, run.bd
    wdir = plan.direct_transform_weights(wd)
    yd = plan.new_output()
    res = {}
    runs = {"direct_hip": lambda: plan.direct_conv2d(xd, wdir, bd, out=yd),
            "torch_conv2d": lambda: F.conv2d(xd, wd, bd, padding=layer.k // 2)}
    for name, fn in runs.items():
        settle(fn, 0.3)
        ms, _ = timed_steps(fn, steps)
        res[name] = {"ms": round(ms, 4), "GFLOP/s": round(layer.direct_flops / (ms * 1e-3) / 1e9, 1)}
    yt = F.conv2d(xd, wd, bd, padding=layer.k // 2)
    _sync()
    res["direct_hip"]["rel_l2_vs_torch"] = float(torch.linalg.vector_norm(yd - yt) / torch.linalg.vector_norm(yt))
    return res


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None, help=f"timed steps (default {DEFAULT_STEPS}; 20 for vgg16)")
    ap.add_argument("--warmup", type=int, default=DEFAULT_WARMUP,
                    help="counted warm-up steps, after the clock-settle pre-roll")
    ap.add_argument("--settle-s", type=float, default=SETTLE_S,
                    help="seconds of untimed steps before the warm-up (0: none)")
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
    ap.add_argument("--no-floor", action="store_true",
                    help="skip the practical ceilings: the streaming probe of the transforms' byte mixes and "
                         "the matrix probe of the contraction's launch")
    ap.add_argument("--no-others", action="store_true",
                    help="skip the other workloads (the other single layers and the VGG-16 stack)")
    ap.add_argument("--oracle-all", action="store_true",
                    help="also time the CPU oracle (split and direct) on a bounded sample of each other workload "
                         "and the VGG-16 stack (about a minute of host time; off by default)")
    ap.add_argument("--copy-probe-mb", type=int, default=0,
                    help="before timing, copy a buffer of this many MiB 3 times (calibrates HBM counters)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py: the library runs on one GPU only (asked for {args.gpus}); the multi-GPU "
              "sharding of the path is a design note, not an implementation.", file=sys.stderr)
        sys.exit(2)

    import torch
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
        x, w, b = make_layer(layer)
    else:
        cfg = CONFIGS[args.config]
        layer = cfg["layer"]
        tile = (args.tile if args.tile is not None
                else (DEFAULT_TILE if args.config == DEFAULT_CONFIG else cfg["tiles"][-1]))
        x, w, b = make_config(args.config)
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)

    run = LayerRun(layer, x, w, b, tile, args.mode, dev)
    info = run.info
    tile = info.tile
    if args.copy_probe_mb > 0:
        nbytes = args.copy_probe_mb << 20
        src = torch.ones(nbytes // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        _sync()
        del src, dst

    settle_n, settle_s = settle(run.step, args.settle_s)
    warm_up(run.step, args.warmup)
    steps = args.steps or DEFAULT_STEPS

    # Timed region: exactly `steps` conv2d calls, synchronised on both sides.
    ms_per_step, t_wall = timed_steps(run.step, steps)

    fwd, con, inv, ms_per_step_staged = run.stage_times(steps)
    cold = None if args.no_cold else run.cold_stage_times(min(steps, 20))

    counts = algorithmic_counts(layer, info)
    stages = stage_record(counts, _avg(fwd), _avg(con), _avg(inv))
    con_tfs = stages["contract"]["TFLOP/s"]
    value = layer.direct_flops / (ms_per_step * 1e-3) / 1e9

    parity = None
    if not args.no_parity:
        rng = np.random.default_rng(99)
        sel = np.sort(rng.choice(layer.cout, size=4, replace=False))
        parity = run.parity(x, w, b, slice(0, min(layer.n, 4)), sel)

    wtag = f"{args.config}_T{tile}_{args.mode}"
    stages["forward"]["traffic"] = load_traffic("forward", wtag)
    stages["inverse"]["traffic"] = load_traffic("inverse", wtag)
    out = {
        "metric": "effective direct-conv GFLOP/s",
        "value": round(value, 1),
        "unit": "GFLOP/s",
        "n_gpus": 1,
        "steps": steps,
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
        "settle_s": round(settle_s, 3),
        "settle_steps": settle_n,
        "roofline": {"bound": "mfma", "kernel": "contract (per-bin complex Cin->Cout product)",
                     "achieved": con_tfs, "peak": FP32_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(con_tfs / FP32_MFMA_PEAK_TFLOPS, 4), "traffic": load_traffic("contract", wtag),
                     "flops_per_complex_mac": 8,
                     "mfma_real_products_per_complex_mac": info.contract_real_products,
                     "mfma_executed_frac": round(con_tfs * info.contract_real_products / 4
                                                 / FP32_MFMA_PEAK_TFLOPS, 4)},
        "stages": stages,
        "stages_cold": None if cold is None else {
            "forward": {"ms": round(cold[0], 4), "frac_hbm": round(counts["forward_bytes"] / (cold[0] * 1e-3) / 1e9
                                                                 / HBM_PEAK_GBS, 4)},
            "contract": {"ms": round(cold[1], 4), "frac_mfma": round(counts["contract_flops"] / (cold[1] * 1e-3)
                                                                     / 1e12 / FP32_MFMA_PEAK_TFLOPS, 4)},
            "inverse": {"ms": round(cold[2], 4), "frac_hbm": round(counts["inverse_bytes"] / (cold[2] * 1e-3) / 1e9
                                                                 / HBM_PEAK_GBS, 4)},
            "note": "each stage after a 512 MB read has replaced the last-level cache's contents"},
        "timing": "clock-settle pre-roll (settle_s, untimed), then `warmup` counted warm-up steps, then "
                  "ms_per_step: exactly `steps` fftsplit_conv2d calls between two events on the launch stream; "
                  "stage times: `steps` further passes as three stage calls with each kernel's start/stop "
                  "taken from its dispatch timestamps (hipExtLaunchKernel events)",
        "ms_per_step_staged": round(ms_per_step_staged, 4),
        "wall_s_timed": round(t_wall, 4),
        "parity_rel_l2": parity,
    }
    if not args.no_floor:
        floor = hbm_floor(dev, {"forward": (4 * layer.n * layer.cin * layer.h * layer.w,
                                            counts["forward_bytes"] - 4 * layer.n * layer.cin * layer.h * layer.w),
                                "inverse": (counts["inverse_bytes"] - 4 * layer.n * layer.cout * layer.h * layer.w,
                                            4 * layer.n * layer.cout * layer.h * layer.w)})
        for st, name in (("forward", "forward"), ("inverse", "inverse")):
            stages[st]["frac_of_floor_warm"] = round(floor["warm"][f"{name}_floor_us"] / (stages[st]["ms"] * 1e3), 4)
            if out["stages_cold"] is not None:
                out["stages_cold"][st]["frac_of_floor_cold"] = round(
                    floor["cold"][f"{name}_floor_us"] / (out["stages_cold"][st]["ms"] * 1e3), 4)
        out["hbm_floor"] = floor
    if not args.no_floor and not info.fused_channel_sum:
        out["matrix_ceiling"] = matrix_ceiling(run, _avg(con))
    if not args.no_compare:
        out["spatial_methods"] = time_spatial_methods(steps, run)
        out["oaaconv"] = time_oaaconv(steps, layer, run.xd, run.wd, run.bd)
    if not args.no_others and not args.shape:
        del run
        others = {}
        for name, t in OTHER_LAYERS:
            if name == args.config and t == tile:
                continue
            others[f"{name}_T{t}"] = other_layer(name, t, dev, oracle_budget_s=6.0 if args.oracle_all else 0.0)
            torch.cuda.empty_cache()
        others["vgg16_b32"] = vgg16_summary(dev, oracle_timed=args.oracle_all)
        out["workloads"] = others
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(layer, x, w, b, tile)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
