"""Throughput of the CNN forward pass on one MI355X.

One step is one cnn_net_fwd over a batch of synthetic images: the whole
network, every layer in the paper's layer-setup order (Sec. 4), parameters
resident in HBM, input already on the device (the paper also excludes
parameter loading from its timings, Sec. 4).  Default workload: the
AlexNet-shaped network at batch 64.

Prints ONE JSON line: images/s (whole job), per-layer times measured with
HIP events that the layers' own kernels record (start of a layer's first
kernel, end of its last: cnn_net_fwd_kernel_timed) over timed steps, the convolution
rate as a fraction of the fp32 matrix-core peak, a roofline entry for the
dominant kernel, and the CPU oracle's rate on a bounded sample of the same
workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "images/sec + conv GFLOP/s (% fp32 MFMA peak), AlexNet-shaped fp32 batch 64"
PEAK_FP32_MFMA_TFLOPS = 157.3   # MI355X dense fp32 matrix peak
PEAK_HBM_GBS = 8000.0           # MI355X HBM3E

# HIP runtime setting for the timed process: kernel arguments in device memory
# rather than host memory, so that each wave's first reads of its parameters
# stay on the GPU.  Measured on one box, three alternations each (ms per
# pass, host -> device arguments): LeNet B16 0.0426 -> 0.0392, CIFAR-10 quick
# B32 0.0756 -> 0.0621, AlexNet B1 0.155 -> 0.135, B16 0.389 -> 0.370, B64
# 0.950 -> 0.929, B256 unchanged within noise.  It must be in the environment
# before the HIP runtime starts; a value the caller set is kept.
RUNTIME_ENV = {"HIP_FORCE_DEV_KERNARG": "1"}


def layer_work(net, batch, cnn):
    """Per layer: (name, kind, flops, bytes) with algorithmic counts.

    conv: 2*N*K*P*Q*(C/G)*R*S flops; fc: 2*N*I*O flops; pool: read input +
    write output (+ int32 index); LRN: read + write; ReLU: read + write.
    Bytes are fp32 tensor sizes; parameters are counted for conv / fc only as
    part of the contraction, not as bandwidth.  An LRN layer followed by a
    pooling layer runs inside the pooling kernel: the LRN gets kind "fused"
    and no bytes, the pooling layer the LRN's read and its own write."""
    c, h, w = net.input_chw
    out = []
    counts = {}
    layers = list(net.layers)
    for li, layer in enumerate(layers):
        counts[layer.kind] = counts.get(layer.kind, 0) + 1
        name = f"{layer.kind}{counts[layer.kind]}"
        if layer.kind == "conv":
            p, q = cnn.cnn_conv2d_out_shape(h, w, *layer.kernel, layer.stride, layer.pad)
            k = layer.out_channels
            flops = 2 * batch * k * p * q * (c // layer.groups) * layer.kernel[0] * layer.kernel[1]
            byts = 4 * batch * (c * h * w + k * p * q)
            out.append((name, "conv", flops, byts))
            c, h, w = k, p, q
        elif layer.kind == "fc":
            i, o = c * h * w, layer.out_features
            out.append((name, "fc", 2 * batch * i * o, 4 * (batch * (i + o) + i * o)))
            c, h, w = o, 1, 1
        elif layer.kind == "pool":
            p, q = cnn.cnn_pool_out_shape(h, w, layer.kernel, layer.stride, layer.pad, layer.ceil)
            byts = 4 * batch * c * (h * w + p * q)
            kind = "lrn+pool" if li > 0 and layers[li - 1].kind == "lrn" else "pool"
            out.append((name, kind, 0, byts))
            h, w = p, q
        elif layer.kind == "lrn":
            fused = li + 1 < len(layers) and layers[li + 1].kind == "pool"
            out.append((name, "fused" if fused else "lrn", 0, 0 if fused else 8 * batch * c * h * w))
        elif layer.kind == "softmax":
            out.append((name, "softmax", 0, 8 * batch * c * h * w))
        else:
            out.append((name, "relu", 0, 8 * batch * c * h * w))
    return out


# Host-only sources (argument checks, tuning table, NetFile parser): they do
# not change what a kernel reads or writes.
HOST_ONLY_SOURCES = ("api.hip", "tuner.hip", "netfile.cpp")


def source_digest():
    """Digest of the kernel sources (and their launchers) under csrc/, without
    their comments and blank lines (a comment edit changes no kernel)."""
    import re
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_1511_07376_amd", "csrc")
    for f in sorted(os.listdir(csrc)):
        if f in HOST_ONLY_SOURCES:
            continue
        with open(os.path.join(csrc, f), encoding="utf-8") as fh:
            text = fh.read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        text = re.sub(r"//[^\n]*", "", text)
        code = "\n".join(l.rstrip() for l in text.splitlines() if l.strip())
        h.update(f.encode() + code.encode())
    return h.hexdigest()[:16]


def conv_configs_of(tuning_text, layer):
    """Tile configurations a tuning table (cnn_tuning_export's text) records
    for a conv layer: its lines with the layer's input and output channels,
    filter, stride and groups, sorted.  Height, width and padding are left out:
    in a network a padded layer may run on a zero-bordered input without
    padding."""
    st = layer.stride if isinstance(layer.stride, (tuple, list)) else (layer.stride, layer.stride)
    want = (layer.in_channels, layer.out_channels, layer.kernel[0], layer.kernel[1], st[0], st[1], layer.groups)
    cfgs = []
    for line in tuning_text.splitlines():
        f = line.split()
        if len(f) != 13:
            continue
        v = [int(t) for t in f]
        if (v[1], v[4], v[5], v[6], v[7], v[8], v[11]) == want:
            cfgs.append(v[12])
    return sorted(cfgs)


def stored_traffic(workload, layer_name, layer=None, tuning_text=None, prof_dir=None):
    """HBM bytes per launch measured by rocprofv3 --pmc (FETCH_SIZE, WRITE_SIZE),
    kept with the digest of the kernel sources and the tuning table they were
    taken with: traffic_<workload>.json in `prof_dir` (profiles/), then
    records taken with other tuning tables (traffic_<workload>_*.json).  The
    first record that applies gives the figure: the sources unchanged since,
    and, for a conv layer (`layer`), the same tile configuration in its tuning
    table as in the current one (`tuning_text`).  None when none applies."""
    prof = prof_dir or os.path.join(ROOT, "profiles")
    if not os.path.isdir(prof):
        return None
    alts = sorted(f for f in os.listdir(prof) if f.startswith(f"traffic_{workload}_") and f.endswith(".json"))
    paths = [os.path.join(prof, f) for f in [f"traffic_{workload}.json"] + alts]
    digest = source_digest()
    for pth in paths:
        if not os.path.exists(pth):
            continue
        with open(pth) as f:
            rec = json.load(f)
        if rec.get("source_digest") != digest:
            continue
        lay = rec.get("layers", {}).get(layer_name)
        if lay is None:
            continue
        if layer is not None and layer.kind == "conv":
            then = conv_configs_of("\n".join(rec.get("tuning", [])), layer)
            if not then or then != conv_configs_of(tuning_text or "", layer):
                continue
        return lay.get("hbm_bytes_per_launch")
    return None


def host_cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(net, x, params, budget_s, y_gpu=None):
    """Times the oracle on a bounded sample of the batch, and checks the GPU
    output of every image the oracle computed against it (the conv / FC
    criterion of the last layer).  Returns (record, parity record)."""
    import oracle
    threads = oracle.get_threads()
    t0 = time.perf_counter()
    ref0 = oracle.net_fwd(net, x[:1], params)
    t1 = time.perf_counter() - t0
    n_more = int(max(0, min(x.shape[0] - 1, (budget_s - t1) / max(t1, 1e-3))))
    t2 = 0.0
    reps = 0
    n = 1
    refs = [ref0]
    if n_more > 0:
        # the same images again while less than ~2/3 of the budget is spent,
        # so that a fast oracle pass is still timed over several seconds
        while reps == 0 or (t1 + t2 < 0.67 * budget_s and reps < 10000):
            t0 = time.perf_counter()
            r = oracle.net_fwd(net, x[1:1 + n_more], params)
            t2 += time.perf_counter() - t0
            if reps == 0:
                refs.append(r)
            reps += 1
        n = 1 + reps * n_more
    # the paper's sequential baseline: one thread, one image, mean of 3 runs
    oracle.set_threads(1)
    t_one = []
    for _ in range(3):
        t0 = time.perf_counter()
        oracle.net_fwd(net, x[:1], params)
        t_one.append(time.perf_counter() - t0)
    oracle.set_threads(threads)
    rec = {"value": n / (t1 + t2), "unit": "images/s", "cores": threads, "kind": "oracle",
           "sample": f"{n} images ({max(reps, 1)} pass(es) over {1 + n_more} of the {x.shape[0]} images of "
                     f"the same batch) through the oracle's layer-by-layer network (double "
                     f"accumulation, OpenMP over images x channels), {t1 + t2:.1f} s",
           "host_cpu": host_cpu_model(), "host_threads_available": os.cpu_count(),
           "value_1_thread": round(1.0 / float(np.mean(t_one)), 3),
           "value_1_thread_runs_s": [round(t, 3) for t in t_one]}
    parity = None
    if y_gpu is not None:
        ref = np.concatenate(refs, axis=0).astype(np.float64)
        got = y_gpu[: ref.shape[0]].reshape(ref.shape).astype(np.float64)
        last = [l for l in net.layers if l.kind in ("conv", "fc")][-1]
        kred = last.in_features if last.kind == "fc" else \
            (last.in_channels // last.groups) * last.kernel[0] * last.kernel[1]
        err = float(np.abs(got - ref).max())
        rel = float(np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-300))
        tol = 1e-4 * np.sqrt(kred)
        parity = {"images_checked": int(ref.shape[0]), "max_abs_err": err, "abs_tol": float(tol),
                  "rel_l2_err": rel, "rel_tol": 1e-4, "ok": bool(err <= tol and rel <= 1e-4)}
    return rec, parity


def conv_sweep(args):
    """Single-layer conv sweep: each case auto-tunes on its first call (unless
    --no-autotune; --tuning-file imports recorded choices), then `--steps`
    launches are timed between two HIP events on the launch stream."""
    import torch
    from paper_1511_07376_amd import cnn
    from paper_1511_07376_amd import workloads as wl

    if args.tuning_file and os.path.exists(args.tuning_file):
        with open(args.tuning_file) as f:
            cnn.cnn_tuning_import(f.read())
    cnn.cnn_set_autotune(args.autotune)
    for shape in wl.SWEEP_SHAPES:
        c, h, w_, k, r, s_, stride, pad = shape
        for n in wl.SWEEP_BATCHES:
            x, w, b = (torch.from_numpy(t).cuda() for t in wl.make_sweep_tensors(shape, n, args.seed))
            p, q = cnn.cnn_conv2d_out_shape(h, w_, r, s_, stride, pad)
            flops = 2.0 * n * k * p * q * c * r * s_

            def timed(fn):
                for _ in range(max(args.warmup, 1)):
                    fn()
                torch.cuda.synchronize()
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                for _ in range(args.steps):
                    fn()
                e1.record()
                torch.cuda.synchronize()
                return e0.elapsed_time(e1) / args.steps

            y = torch.empty(n, k, p, q, device="cuda")
            ms = timed(lambda: cnn.cnn_conv2d_fwd(x, w, b, stride, pad, 1, True, y=y))
            tf = flops / (ms * 1e-3) / 1e12
            rec = {"case": {"C": c, "H": h, "W": w_, "K": k, "R": r, "S": s_, "stride": stride, "pad": pad,
                            "N": n},
                   "us": round(ms * 1e3, 2), "gflop": round(flops / 1e9, 4), "tflops": round(tf, 2),
                   "frac_fp32_mfma": round(tf / PEAK_FP32_MFMA_TFLOPS, 4)}
            if args.sweep_miopen:
                import torch.nn.functional as F
                ms_m = timed(lambda: torch.relu_(F.conv2d(x, w, b, stride, pad)))
                rec["miopen_us"] = round(ms_m * 1e3, 2)
            print(json.dumps(rec), flush=True)
    cnn.cnn_set_autotune(False)
    if args.save_tuning:
        with open(args.save_tuning, "w") as f:
            f.write(cnn.cnn_tuning_export())


def conv_shapes(net, batch, cnn):
    """(name, N, C, H, W, layer) for each conv layer, with the library's shape rules."""
    c, h, w = net.input_chw
    out, nconv = [], 0
    for layer in net.layers:
        if layer.kind == "conv":
            nconv += 1
            out.append((f"conv{nconv}", batch, c, h, w, layer))
            h, w = cnn.cnn_conv2d_out_shape(h, w, *layer.kernel, layer.stride, layer.pad)
            c = layer.out_channels
        elif layer.kind == "pool":
            h, w = cnn.cnn_pool_out_shape(h, w, layer.kernel, layer.stride, layer.pad, layer.ceil)
        elif layer.kind == "fc":
            c, h, w = layer.out_features, 1, 1
    return out


def single_layer(args):
    """One conv or FC layer of the network on its own, as the network runs it
    (a padded conv after an LRN + pooling pair reads bordered planes and runs
    unpadded, as the network executor arranges), called `--steps` times with
    HIP events around each call and, with --flush-mb, a read-only sweep of
    that many MiB before each call, so that no earlier kernel's cached or
    dirty lines are charged to it (counter runs of one kernel).  One JSON
    line."""
    import torch
    from paper_1511_07376_amd import cnn
    from paper_1511_07376_amd import workloads as wl

    net = wl.NETS[args.net]
    batch = args.batch or (64 if args.net == "alexnet" else net.default_batch)
    c, h, w = net.input_chw
    counts, found = {}, None
    layers = list(net.layers)
    for i, layer in enumerate(layers):
        counts[layer.kind] = counts.get(layer.kind, 0) + 1
        name = f"{layer.kind}{counts[layer.kind]}"
        if layer.kind == "conv":
            p_, q_ = cnn.cnn_conv2d_out_shape(h, w, *layer.kernel, layer.stride, layer.pad)
            bordered = (max(layer.pad) > 0 and i >= 2 and layers[i - 1].kind == "pool"
                        and layers[i - 2].kind == "lrn")
            if name == args.single_layer:
                found = (layer, c, h, w, bordered)
            c, h, w = layer.out_channels, p_, q_
        elif layer.kind == "pool":
            h, w = cnn.cnn_pool_out_shape(h, w, layer.kernel, layer.stride, layer.pad, layer.ceil)
        elif layer.kind == "fc":
            if name == args.single_layer:
                found = (layer, c * h * w, 1, 1, False)
            c, h, w = layer.out_features, 1, 1
    if found is None:
        raise SystemExit(f"bench: no conv or fc layer {args.single_layer!r} in {net.name}")
    layer, c, h, w, bordered = found
    if args.tuning_file and os.path.exists(args.tuning_file):
        with open(args.tuning_file) as f:
            cnn.cnn_tuning_import(f.read())
    gen = torch.Generator(device="cuda").manual_seed(args.seed)
    if layer.kind == "conv":
        pad = (0, 0) if bordered else layer.pad
        hh, ww = (h + 2 * layer.pad[0], w + 2 * layer.pad[1]) if bordered else (h, w)
        x = torch.rand((batch, c, hh, ww), device="cuda", generator=gen)
        wt = torch.randn((layer.out_channels, c // layer.groups) + tuple(layer.kernel), device="cuda",
                         generator=gen) * 0.01
        b = torch.randn(layer.out_channels, device="cuda", generator=gen) * 0.01
        p_, q_ = cnn.cnn_conv2d_out_shape(hh, ww, *layer.kernel, layer.stride, pad)
        y = torch.empty((batch, layer.out_channels, p_, q_), device="cuda")
        flops = 2.0 * batch * layer.out_channels * p_ * q_ * (c // layer.groups) * layer.kernel[0] * layer.kernel[1]
        byts = 4.0 * (x.numel() + y.numel())
        shape = {"N": batch, "C": c, "H": hh, "W": ww, "K": layer.out_channels, "R": layer.kernel[0],
                 "S": layer.kernel[1], "stride": list(layer.stride), "pad": list(pad), "groups": layer.groups}
        call = lambda: cnn.cnn_conv2d_fwd(x, wt, b, layer.stride, pad, layer.groups, layer.relu, y=y)  # noqa: E731
    else:
        x = torch.rand((batch, c), device="cuda", generator=gen)
        wt = torch.randn((layer.out_features, c), device="cuda", generator=gen) * 0.01
        b = torch.randn(layer.out_features, device="cuda", generator=gen) * 0.01
        y = torch.empty((batch, layer.out_features), device="cuda")
        flops = 2.0 * batch * c * layer.out_features
        byts = 4.0 * (x.numel() + y.numel() + wt.numel())
        shape = {"N": batch, "I": c, "O": layer.out_features}
        call = lambda: cnn.cnn_fc_fwd(x, wt, b, layer.relu, y=y)  # noqa: E731
    flush = torch.ones(args.flush_mb * (1 << 18), device="cuda") if args.flush_mb else None
    if args.autotune and not args.tuning_file:
        cnn.cnn_set_autotune(True)
    for _ in range(max(args.warmup, 1)):
        call()
    cnn.cnn_set_autotune(False)
    if flush is not None:
        flush.max()
        flush.max()  # a sweep over clean caches: its own traffic, for counter runs
    torch.cuda.synchronize()
    times = []
    for _ in range(args.steps):
        if flush is not None:
            flush.max()  # reads every line of the buffer
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        call()
        e1.record()
        times.append((e0, e1))
    torch.cuda.synchronize()
    us = [a.elapsed_time(b_) * 1e3 for a, b_ in times]
    mean = float(np.mean(us))
    rec = {"single_layer": args.single_layer, "net": net.name, "bordered_input": bordered, "shape": shape,
           "flush_mb": args.flush_mb, "steps": args.steps, "us_mean": round(mean, 2),
           "us_median": round(float(np.median(us)), 2), "gflop": round(flops / 1e9, 4),
           "tflops": round(flops / mean / 1e6, 2), "frac_fp32_mfma": round(flops / mean / 1e6 / PEAK_FP32_MFMA_TFLOPS, 4),
           "algorithmic_mbytes": round(byts / 1e6, 2),
           "tuning": cnn.cnn_tuning_export().strip()}
    print(json.dumps(rec), flush=True)


# Shapes on which the built-in tile heuristic was fitted: AlexNet's five
# conv layers as the network runs them (conv2 and conv3 on bordered input),
# the conv sweep's five shapes, and the conv layers of LeNet and CIFAR-10
# quick past their first; (C, H, W, K, R, stride, pad, groups).
CONFIG_TABLE_SHAPES = [
    (3, 227, 227, 96, 11, 4, 0, 1), (96, 31, 31, 256, 5, 1, 0, 2), (256, 15, 15, 384, 3, 1, 0, 1),
    (384, 13, 13, 384, 3, 1, 1, 2), (384, 13, 13, 256, 3, 1, 1, 2),
    (3, 224, 224, 64, 7, 2, 3, 1), (64, 56, 56, 64, 3, 1, 1, 1), (256, 28, 28, 256, 3, 1, 1, 1),
    (512, 14, 14, 512, 3, 1, 1, 1), (256, 56, 56, 64, 1, 1, 0, 1),
    (20, 12, 12, 50, 5, 1, 0, 1), (32, 16, 16, 32, 5, 1, 2, 1), (32, 8, 8, 64, 5, 1, 2, 1),
]


def config_table(args):
    """Every conv tile configuration, and the built-in heuristic (config -1),
    timed on CONFIG_TABLE_SHAPES at batches 1, 16, 64 and 256 (256 only where
    the input holds at most 100k elements per image): 2 warm-up launches, then
    the mean of 10 between HIP events.  One JSON line per shape, then one
    line with the heuristic's total against always taking the fastest."""
    import torch
    from paper_1511_07376_amd import cnn

    gen = torch.Generator(device="cuda").manual_seed(args.seed)
    tot_h = tot_best = 0.0
    ncfg = cnn.cnn_conv2d_num_configs()
    for n in (1, 16, 64, 256):
        for (c, h, w_, k, r, st, pd, g) in CONFIG_TABLE_SHAPES:
            if n == 256 and h * w_ * c > 100000:
                continue
            x = torch.rand((n, c, h, w_), device="cuda", generator=gen)
            wt = torch.randn((k, c // g, r, r), device="cuda", generator=gen) * 0.05
            b = torch.randn(k, device="cuda", generator=gen)
            p_, q_ = cnn.cnn_conv2d_out_shape(h, w_, r, r, st, pd)
            y = torch.empty((n, k, p_, q_), device="cuda")
            us = {}
            for cfg in range(-1, ncfg):
                for _ in range(2):
                    cnn.cnn_conv2d_fwd(x, wt, b, st, pd, g, True, y=y, config=cfg)
                torch.cuda.synchronize()
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                for _ in range(10):
                    cnn.cnn_conv2d_fwd(x, wt, b, st, pd, g, True, y=y, config=cfg)
                e1.record()
                torch.cuda.synchronize()
                us[cfg] = round(e0.elapsed_time(e1) / 10 * 1000, 2)
            best = min((v, cfg) for cfg, v in us.items() if cfg >= 0)
            tot_h += us[-1]
            tot_best += best[0]
            print(json.dumps({"shape": {"N": n, "C": c, "H": h, "W": w_, "K": k, "R": r, "stride": st, "pad": pd,
                                        "groups": g}, "us": {str(cf): v for cf, v in us.items()},
                              "best_config": best[1], "heuristic_over_best": round(us[-1] / best[0], 4)}), flush=True)
            del x, y
    print(json.dumps({"heuristic_total_us": round(tot_h, 1), "best_total_us": round(tot_best, 1),
                      "heuristic_over_best": round(tot_h / tot_best, 4)}), flush=True)


FC_TABLE_SHAPES = [  # (I, O): AlexNet's fc6-fc8, LeNet's ip1-ip2, CIFAR-10 quick's ip1-ip2
    (9216, 4096), (4096, 4096), (4096, 1000), (800, 500), (500, 10), (1024, 64), (64, 10),
]


def fc_config_table(args):
    """Every FC kernel configuration, and the built-in choice (config -1),
    timed on FC_TABLE_SHAPES at batches 1, 16, 32, 64 and 256 (configurations
    that do not take a shape are left out): fuse_relu on, bias, 2 warm-up
    calls, then the mean of 20 calls between HIP events.  A call whose
    reduction is split also runs the kernels that set the output to the bias
    first and apply the ReLU after (inside a network pass the first runs in a
    pooling kernel and the second in the next layer's reads).  One JSON line
    per shape."""
    import torch
    from paper_1511_07376_amd import cnn

    gen = torch.Generator(device="cuda").manual_seed(args.seed)
    ncfg = cnn.cnn_fc_num_configs()
    for n in (1, 16, 32, 64, 256):
        for (i_, o_) in FC_TABLE_SHAPES:
            x = torch.rand((n, i_), device="cuda", generator=gen)
            wt = torch.randn((o_, i_), device="cuda", generator=gen) * 0.02
            b = torch.randn(o_, device="cuda", generator=gen)
            y = torch.empty((n, o_), device="cuda")
            us = {}
            for cfg in range(-1, ncfg):
                try:
                    for _ in range(2):
                        cnn.cnn_fc_fwd(x, wt, b, True, y=y, config=cfg)
                except cnn.CnnError:
                    continue
                torch.cuda.synchronize()
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                for _ in range(20):
                    cnn.cnn_fc_fwd(x, wt, b, True, y=y, config=cfg)
                e1.record()
                torch.cuda.synchronize()
                us[cfg] = round(e0.elapsed_time(e1) / 20 * 1000, 2)
            best = min((v, cfg) for cfg, v in us.items() if cfg >= 0)
            print(json.dumps({"shape": {"N": n, "I": i_, "O": o_}, "us": {str(cf): v for cf, v in us.items()},
                              "names": {str(cf): cnn.cnn_fc_config_name(cf) for cf in us if cf >= 0},
                              "best_config": best[1], "builtin_over_best": round(us[-1] / best[0], 4)}),
                  flush=True)
            del x, y, wt


def gemm_reference(args):
    """Each conv layer of the network beside torch's fp32 batched GEMM on the
    same contraction with the im2col matrix already unrolled in memory (so the
    library pays no gather): per group, [K/G x (C/G)RS] times [(C/G)RS x NPQ],
    and the pixel-major [NPQ x (C/G)RS] times its transpose.  Context for the
    implicit-GEMM kernels, one JSON line per layer."""
    import torch
    from paper_1511_07376_amd import cnn
    from paper_1511_07376_amd import workloads as wl

    torch.backends.cuda.matmul.allow_tf32 = False
    net = wl.NETS[args.net]
    batch = args.batch or (64 if args.net == "alexnet" else net.default_batch)
    cnn.cnn_set_autotune(True)

    def timed(fn):
        for _ in range(max(args.warmup, 1)):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(args.steps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / args.steps

    for name, n, c, h, w_, layer in conv_shapes(net, batch, cnn):
        g, (r, s_) = layer.groups, layer.kernel
        k = layer.out_channels
        p, q = cnn.cnn_conv2d_out_shape(h, w_, r, s_, layer.stride, layer.pad)
        kg, kr, m = k // g, (c // g) * r * s_, n * p * q
        flops = 2.0 * g * kg * kr * m
        x = torch.rand(n, c, h, w_, device="cuda")
        wt = torch.randn(k, c // g, r, s_, device="cuda") * 0.05
        b = torch.randn(k, device="cuda")
        y = torch.empty(n, k, p, q, device="cuda")
        ms_ours = timed(lambda: cnn.cnn_conv2d_fwd(x, wt, b, layer.stride, layer.pad, g, True, y=y))
        del x, y
        a = torch.randn(g, kg, kr, device="cuda")
        bm = torch.randn(g, kr, m, device="cuda")
        ms_km = timed(lambda: torch.bmm(a, bm))
        del bm
        xm = torch.randn(g, m, kr, device="cuda")
        at = a.transpose(1, 2).contiguous()
        ms_mk = timed(lambda: torch.bmm(xm, at))
        del xm
        rec = {"layer": name, "gemm": {"groups": g, "rows": kg, "reduction": kr, "cols": m},
               "implicit_gemm_us": round(ms_ours * 1e3, 1),
               "library_gemm_us": {"channels_x_pixels": round(ms_km * 1e3, 1),
                                   "pixels_x_channels": round(ms_mk * 1e3, 1)},
               "frac_fp32_mfma": {"implicit_gemm": round(flops / ms_ours / 1e9 / PEAK_FP32_MFMA_TFLOPS, 3),
                                  "library_best": round(flops / min(ms_km, ms_mk) / 1e9
                                                        / PEAK_FP32_MFMA_TFLOPS, 3)}}
        print(json.dumps(rec), flush=True)
        torch.cuda.empty_cache()
    cnn.cnn_set_autotune(False)


def main():
    for k, v in RUNTIME_ENV.items():
        os.environ.setdefault(k, v)
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--net", default="alexnet", choices=["lenet", "cifar_quick", "alexnet"])
    ap.add_argument("--batch", type=int, default=None)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--cpu-budget", type=float, default=15.0,
                    help="seconds of oracle work for the CPU baseline (0 disables it)")
    ap.add_argument("--no-autotune", dest="autotune", action="store_false",
                    help="use the built-in tile heuristic instead of tuning during warm-up")
    ap.add_argument("--tuning-file", default=None,
                    help="import this conv tuning table before warm-up (no tuning runs for its shapes)")
    ap.add_argument("--save-tuning", default=None, help="write the tuning table here afterwards")
    ap.add_argument("--graph", action="store_true",
                    help="time the steps as launches of the network captured as a HIP graph "
                         "(the library's graph execution mode)")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="only run a plain device-to-device copy of MIB MiB (HBM counter calibration)")
    ap.add_argument("--sweep", action="store_true",
                    help="instead of the network: time the single-layer conv sweep (five shapes x "
                         "batches 1, 16, 64, bias + ReLU fused), one JSON line per case")
    ap.add_argument("--sweep-miopen", action="store_true",
                    help="with --sweep: also time torch's own conv2d (MIOpen) on the same tensors, as context")
    ap.add_argument("--streams", type=int, default=1,
                    help="run the timed steps round-robin on this many streams, each with its own replica "
                         "of the network (own workspace), so that consecutive passes overlap: serving "
                         "throughput rather than one pass after another")
    ap.add_argument("--single-layer", default=None, metavar="NAME",
                    help="instead of the network: time one conv or fc layer of it (conv1, fc2, ...) as the "
                         "network runs it, one JSON line")
    ap.add_argument("--flush-mb", type=int, default=0, metavar="MIB",
                    help="read a buffer of MIB MiB before each timed call (--single-layer) or before each "
                         "step of the per-layer event pass, so that caches start cold")
    ap.add_argument("--fc-config-table", action="store_true",
                    help="time every FC configuration on the networks' FC shapes (one JSON line per shape)")
    ap.add_argument("--config-table", action="store_true",
                    help="instead of the network: time every conv tile configuration and the built-in heuristic "
                         "on the shapes the heuristic was fitted to, one JSON line per shape")
    ap.add_argument("--gemm-reference", action="store_true",
                    help="instead of the network: time each conv layer beside torch's fp32 batched GEMM "
                         "on its contraction with the im2col matrix precomputed, one JSON line per layer")
    args = ap.parse_args()
    if args.copy_probe:
        import torch
        a = torch.ones(args.copy_probe * (1 << 20) // 4, device="cuda")
        b = torch.empty_like(a)
        b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes": a.numel() * 4}), flush=True)
        return
    if args.sweep:
        return conv_sweep(args)
    if args.gemm_reference:
        return gemm_reference(args)
    if args.single_layer:
        return single_layer(args)
    if args.config_table:
        return config_table(args)
    if args.fc_config_table:
        return fc_config_table(args)
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported "
              "(the images of a batch are independent: on N GPUs each would run batch/N)",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_1511_07376_amd import cnn
    from paper_1511_07376_amd import workloads as wl

    net = wl.NETS[args.net]
    batch = args.batch or (64 if args.net == "alexnet" else net.default_batch)
    x = wl.make_input(net, batch, args.seed)
    params = wl.make_params(net, args.seed)
    model = cnn.Network(net, params)
    xd = torch.from_numpy(x).cuda()
    yd = torch.empty(model.out_shape(batch), device="cuda")

    nl = len(net.layers)
    # The auto-tuner (the paper's first-launch tuning, Sec. 3.6) picks each conv
    # layer's tile configuration during the first warm-up step; the timed steps
    # use the recorded choices.
    if args.tuning_file and os.path.exists(args.tuning_file):
        with open(args.tuning_file) as f:
            cnn.cnn_tuning_import(f.read())
    if args.autotune:
        cnn.cnn_set_autotune(True)
    for _ in range(max(args.warmup, 1 if args.autotune else 0)):
        model(xd, y=yd)
    cnn.cnn_set_autotune(False)
    if args.save_tuning:
        with open(args.save_tuning, "w") as f:
            f.write(cnn.cnn_tuning_export())
    # torch creates an event at its first record: record each once
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(nl + 1)] for _ in range(args.steps)]
    kstart = [[torch.cuda.Event(enable_timing=True) for _ in range(nl)] for _ in range(args.steps)]
    kstop = [[torch.cuda.Event(enable_timing=True) for _ in range(nl)] for _ in range(args.steps)]
    for evs in events + kstart + kstop:
        for e in evs:
            e.record()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    graph = None
    if args.graph:
        # the library's graph execution mode: one forward pass captured by
        # cnn_net_graph_create, one graph launch per step
        graph = cnn.Network(net, params, execution_mode="graph")
        graph(xd, y=yd)                # eager pass + capture
        graph(xd, y=yd)
        torch.cuda.synchronize()

    # timed region: K steps of cnn_net_fwd (graph launches with --graph)
    if args.streams > 1 and graph is None:
        # round-robin over replicas on their own streams (default priority);
        # the start and end events on the current stream bracket them all
        reps = [model] + [model.replica() for _ in range(args.streams - 1)]
        ys = [yd] + [torch.empty_like(yd) for _ in range(args.streams - 1)]
        streams = [torch.cuda.Stream() for _ in range(args.streams)]
        for _ in range(max(args.warmup, 1)):  # first use of each stream and workspace untimed
            for j in range(args.streams):
                reps[j](xd, y=ys[j], stream=streams[j])
        torch.cuda.synchronize()
        cur = torch.cuda.current_stream()
        start.record(cur)
        for s_ in streams:
            s_.wait_event(start)
        for k in range(args.steps):
            j = k % args.streams
            reps[j](xd, y=ys[j], stream=streams[j])
        for s_ in streams:
            cur.wait_stream(s_)
        end.record(cur)
        torch.cuda.synchronize()
        for j in range(1, args.streams):
            assert torch.allclose(ys[j], yd, rtol=1e-5, atol=1e-6), "replicas disagree"
    else:
        torch.cuda.synchronize()
        start.record()
        for k in range(args.steps):
            if graph is not None:
                graph(xd, y=yd)
            else:
                model(xd, y=yd)
        end.record()
        torch.cuda.synchronize()
    ms_step = start.elapsed_time(end) / args.steps
    # per-layer region: K more steps in which every layer's kernels record
    # their own start and end times into its pair of events
    # (cnn_net_fwd_kernel_timed: no packets of their own between the layers);
    # then K steps with events recorded between the layers
    # (cnn_net_fwd_timed), whose records add a few microseconds to each
    # interval.  Neither region is used for `value`.
    flush = torch.ones(args.flush_mb * (1 << 18), device="cuda") if args.flush_mb else None
    torch.cuda.synchronize()
    start.record()
    for k in range(args.steps):
        if flush is not None:
            flush.max()  # cold caches for this step's layers (outside their events)
        model(xd, y=yd, kernel_events=(kstart[k], kstop[k]))
    end.record()
    torch.cuda.synchronize()
    ms_step_kevents = start.elapsed_time(end) / args.steps
    assert torch.isfinite(yd).all().item(), "non-finite output"
    layer_ms = [float(np.mean([kstart[k][i].elapsed_time(kstop[k][i]) for k in range(args.steps)]))
                for i in range(nl)]

    torch.cuda.synchronize()
    start.record()
    for k in range(args.steps):
        if flush is not None:
            flush.max()
        model(xd, y=yd, events=events[k])
    end.record()
    torch.cuda.synchronize()
    ms_step_events = start.elapsed_time(end) / args.steps
    layer_ms_markers = [float(np.mean([events[k][i].elapsed_time(events[k][i + 1]) for k in range(args.steps)]))
                        for i in range(nl)]
    step_ms_events = [events[k][0].elapsed_time(events[k][nl]) for k in range(args.steps)]
    work = layer_work(net, batch, cnn)
    layers = []
    for (name, kind, flops, byts), ms, ms_m in zip(work, layer_ms, layer_ms_markers):
        ent = {"layer": name, "ms": round(ms, 5), "ms_between_markers": round(ms_m, 5)}
        if kind in ("conv", "fc"):
            tf = flops / (ms * 1e-3) / 1e12 if ms > 0 else 0.0
            ent.update({"gflop": round(flops / 1e9, 4), "tflops": round(tf, 2),
                        "frac_fp32_mfma": round(tf / PEAK_FP32_MFMA_TFLOPS, 4)})
        elif kind == "fused":
            ent["runs_inside_next_layer"] = True  # no kernel of its own
        else:
            gbs = byts / (ms * 1e-3) / 1e9 if ms > 0 else 0.0
            ent.update({"mbytes": round(byts / 1e6, 2), "gbs": round(gbs, 1),
                        "frac_hbm": round(gbs / PEAK_HBM_GBS, 4)})
        layers.append(ent)

    conv_flops = sum(w[2] for w in work if w[1] == "conv")
    conv_ms = sum(ms for w, ms in zip(work, layer_ms) if w[1] == "conv")
    conv_tf = conv_flops / (conv_ms * 1e-3) / 1e12

    dom = int(np.argmax(layer_ms))
    dname, dkind, dflops, dbytes = work[dom]
    workload = f"{net.name}_b{batch}"
    if dkind in ("conv", "fc"):
        ach = dflops / (layer_ms[dom] * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": round(ach, 2), "peak": PEAK_FP32_MFMA_TFLOPS,
                "unit": "TFLOP/s", "frac": round(ach / PEAK_FP32_MFMA_TFLOPS, 4)}
    else:
        ach = dbytes / (layer_ms[dom] * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(ach / PEAK_HBM_GBS, 4)}
    named, counts = {}, {}
    for layer in net.layers:  # the names layer_work gives
        counts[layer.kind] = counts.get(layer.kind, 0) + 1
        named[f"{layer.kind}{counts[layer.kind]}"] = layer
    roof["traffic"] = stored_traffic(workload, dname, named.get(dname), cnn.cnn_tuning_export())
    roof["layer"] = dname
    roof["launch_ms"] = round(layer_ms[dom], 5)

    shape = "x".join(map(str, net.input_chw))
    result = {
        "metric": METRIC,
        "value": round(batch / (ms_step * 1e-3), 1),
        "unit": "images/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded uniform [0,1) images, N(0, std) weights and biases)",
        "runtime_env": {k: os.environ.get(k) for k in RUNTIME_ENV},
        "config": {"workload": f"{net.name}-shaped fp32 forward, batch {batch} x {shape}",
                   "net": net.name, "batch": batch, "layers": nl},
        "conv_gflops": round(conv_tf * 1e3, 1),
        "conv_frac_fp32_mfma_peak": round(conv_tf / PEAK_FP32_MFMA_TFLOPS, 4),
        "conv_ms": round(conv_ms, 5),
        "ms_per_step_with_kernel_events": round(ms_step_kevents, 4),
        "ms_per_step_with_layer_events": round(ms_step_events, 4),
        "ms_per_step_with_layer_events_median": round(float(np.median(step_ms_events)), 4),
        "layer_events_after_flush_mb": args.flush_mb,
        "graph_replay": bool(graph is not None),
        "streams": args.streams if graph is None else 1,
        "autotune": bool(args.autotune),
        "conv_configs": {" ".join(l.split()[:-1]): cnn.cnn_conv2d_config_name(int(l.split()[-1]))
                         for l in cnn.cnn_tuning_export().splitlines()},
        "layers": layers,
        "roofline": roof,
    }
    if args.cpu_budget > 0:
        cb, parity = cpu_baseline(net, x, params, args.cpu_budget, yd.cpu().numpy())
        result["cpu_baseline"] = cb
        # the timed pass's output, checked against the oracle on every image
        # the baseline computed
        result["parity_vs_oracle"] = parity
        # the paper's speedups are GPU vs the sequential CPU implementation
        result["speedup_vs_oracle"] = {"all_cores": round(result["value"] / cb["value"], 1),
                                       "one_thread": round(result["value"] / cb["value_1_thread"], 1)}
    print(json.dumps(result), flush=True)
    if result.get("parity_vs_oracle") and not result["parity_vs_oracle"]["ok"]:
        print(f"bench: the timed output differs from the oracle: {result['parity_vs_oracle']}", file=sys.stderr)
        sys.exit(1)


if __name__ == "__main__":
    main()
