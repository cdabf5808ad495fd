#!/usr/bin/env python3
"""Benchmark of one rank's synchronous data-parallel SGD step on one MI355X.

A step is one mtx_train_step over one batch: forward and backward of every shard, the average
of the R shard gradients and the momentum update.  Inputs are seeded synthetic tensors already
resident in HBM when the timed region starts.

    python bench.py [--steps K] [--warmup W] [--workload alexnet|cifar|resnet|lenet|mlp]
                    [--no-cpu-baseline] [--no-microbench] [--no-extra]

Prints one JSON line.  The default workload is the AlexNet-shaped CNN in bf16 at B = 256 on
R = 8 shards (the paper's AlexNet runs at batch 256, Sec. IV-B, the largest configuration that
one GPU holds).  `value` is samples/s of the whole job (one GPU); `roofline` covers the
kernel that takes the most time in the step, timed in place with HIP events on the step's
stream (its `traffic` comes from a committed rocprofv3 counter summary of the same kernel
sources, else null); `grad_avg_update` is the fused average + momentum kernel at the
61M- and 250M-element, 16-buffer sizes; `other_workloads` are short runs of the other
workloads (MLP, LeNet, CIFAR, the residual network with batch normalisation, the bottleneck
residual network with projection shortcuts); `shard_sweep` is
samples/s of the LeNet workload at the same global batch for shard counts R = 1 .. 16;
`cpu_baseline` is the CPU oracle timed on a bounded sample of the headline workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK = {"hbm_GBps": 8000.0, "f32_TFLOPs": 157.3, "bf16_TFLOPs": 2500.0,
        "f32_vector_TFLOPs": 157.3}
METRIC = "train samples/sec per GPU; grad-avg+update GB/s and conv/GEMM MFMA % of peak"


def geometry(net):
    """Per-layer shapes (the same definitions as the library's plan)."""
    from paper_1704_04560_amd import workloads as wl
    c, h, w = net.in_shape
    out = []
    for l in net.layers:
        if l.kind == wl.CONV:
            oc, oh, ow = l.out, (h + 2 * l.pad - l.k) // l.stride + 1, (w + 2 * l.pad - l.k) // l.stride + 1
        elif l.kind == wl.FC:
            oc, oh, ow = l.out, 1, 1
        elif l.kind in (wl.BN, wl.ADD, wl.ADDP):
            oc, oh, ow = c, h, w
        else:
            oc, oh, ow = c, (h - l.k) // l.stride + 1, (w - l.k) // l.stride + 1
        out.append(dict(layer=l, c=c, h=h, w=w, oc=oc, oh=oh, ow=ow))
        c, h, w = oc, oh, ow
    return out


def site_work(name, layer, geo, wkl, es, fused=()):
    """Algorithmic work of one launch of a step's launch site: ("alu", flops) for the direct
    first-convolution kernels (fp32 vector fused multiply-adds), ("hbm", bytes) for the
    memory-bound ones (each tensor read once and written once), (None, 0) when not modelled.
    A matrix launch is ("mfma", flops) (2 x multiply-adds of the convolution / product) when its
    flops take longer at the MFMA peak than its algorithmic bytes at the HBM peak, else
    ("hbm", bytes): operands read once, the output written once (a data gradient also reads
    the ReLU mask; a weight gradient writes R fp32 gradient rows; a weight gradient fused with
    the average + update, "wgrad_update", also reads w and v and writes the average, v and w).
    "avg_update" is the whole step's stand-alone average + update over the parameters of the
    layers not in `fused`."""
    return _site_work(name, layer, geo, wkl, es, fused)[:2]


def matrix_flops(name, layer, geo, wkl):
    """2 x multiply-adds of a matrix launch site (0 for the others)."""
    from paper_1704_04560_amd import workloads as wl
    if layer < 0 or name not in ("fwd", "dgrad", "wgrad", "wgrad_update"):
        return 0.0
    g = geo[layer]
    l = g["layer"]
    B = wkl.batch
    if l.kind == wl.CONV:
        return 2.0 * B * g["oh"] * g["ow"] * g["oc"] * (g["c"] // l.groups) * l.k * l.k
    if l.kind == wl.ADDP:  # the projection: a 1x1 convolution of the source's output
        return 2.0 * B * g["oh"] * g["ow"] * g["oc"] * geo[l.k]["oc"]
    if l.kind == wl.FC:
        return 2.0 * B * g["c"] * g["h"] * g["w"] * g["oc"]
    return 0.0


def layer_params(geo, layer):
    """Parameters (W and b) of one layer."""
    from paper_1704_04560_amd import workloads as wl
    g = geo[layer]
    l = g["layer"]
    if l.kind == wl.CONV:
        return g["oc"] * (g["c"] // l.groups) * l.k * l.k + g["oc"]
    if l.kind == wl.FC:
        return g["oc"] * g["c"] * g["h"] * g["w"] + g["oc"]
    if l.kind == wl.ADDP:
        return g["oc"] * geo[l.k]["oc"] + g["oc"]
    if l.kind == wl.BN:
        return 2 * g["c"]
    return 0


def _site_work(name, layer, geo, wkl, es, fused=()):
    from paper_1704_04560_amd import workloads as wl
    B, R, Nb = wkl.batch, wkl.shards, wkl.shard_batch
    if layer >= 0:
        g = geo[layer]
        l = g["layer"]
        in_sz = B * g["c"] * g["h"] * g["w"]
        out_sz = B * g["oc"] * g["oh"] * g["ow"]
        if name in ("fwd", "dgrad", "wgrad", "wgrad_update") and l.kind in (wl.CONV, wl.FC, wl.ADDP):
            flops = matrix_flops(name, layer, geo, wkl)
            if l.kind == wl.ADDP:
                src = geo[l.k]
                x_sz, wn = B * src["oc"] * src["oh"] * src["ow"], g["oc"] * src["oc"]
            elif l.kind == wl.CONV:
                x_sz, wn = in_sz, g["oc"] * (g["c"] // l.groups) * l.k * l.k
            else:
                x_sz, wn = in_sz, g["oc"] * g["c"] * g["h"] * g["w"]
            if name == "fwd":
                nbytes = (x_sz + wn + out_sz) * es
            elif name == "dgrad":
                below = l.k if l.kind == wl.ADDP else layer - 1
                mask = below >= 0 and geo[below]["layer"].relu
                nbytes = (out_sz + wn + (2 if mask else 1) * x_sz) * es
            else:
                nbytes = (x_sz + out_sz) * es + R * (wn + g["oc"]) * 4
                if name == "wgrad_update":  # w (and v) read, the average, v and w written
                    nbytes += (wn + g["oc"]) * (20 if wkl.momentum != 0.0 else 12)
            peak = PEAK["bf16_TFLOPs"] if es == 2 else PEAK["f32_TFLOPs"]
            if flops / (peak * 1e12) >= nbytes / (PEAK["hbm_GBps"] * 1e9):
                return "mfma", flops, flops
            return "hbm", float(nbytes), flops
        macs = matrix_flops("fwd", layer, geo, wkl) / 2 if l.kind == wl.CONV else 0.0
        if name in ("fwd_direct", "wgrad_direct"):
            return "alu", 2.0 * macs, 0.0
        if name == "wgrad_direct_reduce":  # per-image fp32 sums read, the shard rows written
            no = g["oc"] * l.k * l.k + g["oc"]
            return "hbm", 4.0 * no * (B + R), 0.0
        if name == "dgrad_col2im":  # fp32 col read once, dx written, mask read
            return "hbm", 4.0 * l.k * l.k * g["c"] * B * g["oh"] * g["ow"] + 2 * es * in_sz, 0.0
        if name == "pool_fwd":
            return "hbm", in_sz * es + out_sz * (es + 1), 0.0
        if name == "pool_bwd":
            return "hbm", out_sz * (es + 1) + in_sz * es * 2, 0.0  # dy + argmax, mask + dx
        if name == "bn_fwd":  # the statistics pass reads x
            return "hbm", in_sz * es, 0.0
        if name == "bn_fwd_apply":  # x read, y written; with the residual addition that
            # follows, computed in the same pass, also its other operand read and its sum written
            nxt = geo[layer + 1]["layer"].kind if layer + 1 < len(geo) else None
            return "hbm", (4 if nxt in (wl.ADD, wl.ADDP) else 2) * in_sz * es, 0.0
        if name == "bn_bwd":  # x and dy read
            return "hbm", 2 * in_sz * es, 0.0
        if name == "bn_bwd_apply":  # x, dy and the mask read, dx written
            return "hbm", 4 * in_sz * es, 0.0
        if name == "add_fwd":  # two read, one written
            return "hbm", 3 * out_sz * es, 0.0
        if name == "skip_add":
            # the source's gradient and the shortcut's share read, the sum written; an identity
            # shortcut's share is the addition's own output gradient, times the source's ReLU mask
            ident = any(h["layer"].kind == wl.ADD and h["layer"].k == layer for h in geo)
            return "hbm", (4 if ident and l.relu else 3) * out_sz * es, 0.0
        if name == "add_bwd":  # dy and the mask read, dx written (runs only where not shared)
            return "hbm", 3 * out_sz * es, 0.0
        return None, 0.0, 0.0
    P = wkl_params(wkl)
    if name == "avg_update":  # the whole step's share (the caller divides by its launches)
        mom = wkl.momentum != 0.0
        P -= sum(layer_params(geo, f) for f in fused)
        return "hbm", (R + (5 if mom else 3)) * 4 * P, 0.0
    if name == "prep_w":
        # every weight tensor is read once (fp32) and written once per layout it is prepared in
        # (convolutions below the first parameter layer need a data-gradient layout too)
        first = min(i for i, g in enumerate(geo) if g["layer"].kind in (wl.CONV, wl.FC))
        tot = 0.0
        for i, g in enumerate(geo):
            l = g["layer"]
            if l.kind == wl.CONV:
                n = g["oc"] * (g["c"] // l.groups) * l.k * l.k
                tot += n * (4 + es) * (2 if i > first else 1)
            elif l.kind == wl.FC:
                tot += g["oc"] * g["c"] * g["h"] * g["w"] * (4 + es)
        return "hbm", tot, 0.0
    if name == "prep_x":
        c, h, w = wkl.net.in_shape
        return "hbm", (4 + es) * B * c * h * w, 0.0
    if name == "softmax_xent":
        nc = wkl.net.num_classes
        return "hbm", B * nc * (4 + es) + B * 4 + 4, 0.0
    return None, 0.0, 0.0


_P = {}


def wkl_params(wkl):
    key = wkl.net.name
    if key not in _P:
        from paper_1704_04560_amd import mtx
        from paper_1704_04560_amd import workloads as wl
        d = mtx.make_desc(wkl.net.in_shape, wl.layer_tuples(wkl.net), wkl.net.dtype)
        _P[key] = mtx.mtx_model_sizes(d, wkl.shards, wkl.shard_batch)[0]
    return _P[key]


def shard_sweep(torch, mtx, wl, name, shard_counts=(1, 2, 4, 8, 16), steps=20, warmup=3):
    """Samples/s of one workload at a fixed global batch over several shard counts R (the
    paper's strong scaling, Sec. IV, with the R replicas on one GPU): each point is a whole
    training step (R shard gradients, their average and the update)."""
    import dataclasses
    base = wl.WORKLOADS[name]
    net = base.net
    layers = wl.layer_tuples(net)
    x, y = wl.make_batch(net, base.batch, seed=0)
    xd, yd = torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda()
    stream = torch.cuda.current_stream()
    points = []
    for R in shard_counts:
        if base.batch % R:
            continue
        wkl = dataclasses.replace(base, shards=R)
        model = mtx.Model(net.in_shape, layers, net.dtype, R, wkl.shard_batch, seed=0)
        for _ in range(warmup):
            model.train_step(xd, yd, wkl.lr, wkl.momentum, None, stream)
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t0.record(stream)
        for _ in range(steps):
            model.train_step(xd, yd, wkl.lr, wkl.momentum, None, stream)
        t1.record(stream)
        torch.cuda.synchronize()
        ms = t0.elapsed_time(t1) / steps
        model.close()
        points.append({"R": R, "shard_batch": wkl.shard_batch, "ms_per_step": round(ms, 5),
                       "samples_per_s": round(base.batch / (ms * 1e-3), 1)})
    return {"workload": base.description.split(",")[0], "global_batch": base.batch,
            "points": points}


def _time_calls(torch, fn, reps):
    for _ in range(3):
        fn()
    torch.cuda.synchronize()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s.record()
    for _ in range(reps):
        fn()
    e.record()
    torch.cuda.synchronize()
    return s.elapsed_time(e) / reps


def _rate(nbytes, ms):
    gbps = nbytes / (ms * 1e-3) / 1e9
    return {"bytes_per_call": nbytes, "ms": round(ms, 4), "GBps": round(gbps, 1),
            "peak_GBps": PEAK["hbm_GBps"], "frac": round(gbps / PEAK["hbm_GBps"], 4)}


def microbench_avg_update(torch, mtx, reps=20):
    """Fused average + update over R=16 flattened fp32 gradient buffers: the momentum update at
    n = 61,000,000 and 250,000,000 elements, and Adam / AdaGrad after the same average at
    n = 61,000,000.  Bytes per element: (R + 5) * 4 for momentum (R grads, w and v read; the
    average, w and v written), (R + 7) * 4 for Adam (m as well), (R + 5) * 4 for AdaGrad (the
    accumulator in place of v)."""
    R = 16
    out = {}
    for n in (61_000_000, 250_000_000):
        gen = torch.Generator(device="cuda").manual_seed(0)
        grads = torch.randn(R * n, device="cuda", generator=gen) * 1e-3
        w = torch.randn(n, device="cuda", generator=gen) * 0.05
        v = torch.randn(n, device="cuda", generator=gen) * 1e-3
        avg = torch.empty(n, device="cuda")
        ms = _time_calls(torch, lambda: mtx.mtx_sgd_update(w, v, grads, R, n, n, 0.01, 0.9, avg),
                         reps if n < 100_000_000 else reps // 2)
        rec = {"R": R, "n": n, **_rate((R + 5) * 4 * n, ms)}
        if n == 61_000_000:
            out.update(rec)
            m2 = (torch.randn(n, device="cuda", generator=gen) * 1e-3) ** 2
            ms = _time_calls(torch, lambda: mtx.mtx_adam_update(
                w, v, m2, grads, R, n, n, 1e-3, 0.9, 0.999, 1e-8, 10, avg), reps)
            out["adam"] = {"R": R, "n": n, **_rate((R + 7) * 4 * n, ms)}
            ms = _time_calls(torch, lambda: mtx.mtx_adagrad_update(
                w, m2, grads, R, n, n, 0.01, 1e-10, avg), reps)
            out["adagrad"] = {"R": R, "n": n, **_rate((R + 5) * 4 * n, ms)}
            del m2
        else:
            out["n250M"] = rec
        del grads, w, v, avg
        torch.cuda.empty_cache()
    return out


def _cpu_model():
    """The host CPU's model name (for the oracle baseline's record)."""
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(wkl, budget_s=12.0):
    """The CPU oracle on a bounded sample of the workload.  AlexNet: one shard of the step (its
    32 samples, R = 1) timed once; a step is R such shards, so samples/s = shard samples / shard
    time (x R extrapolated to the step).  Other workloads: whole steps (R shards of a reduced
    shard batch) repeated until `budget_s` seconds have passed; samples/s over the sample."""
    from oracle import oracle as orc
    from paper_1704_04560_amd import workloads as wl
    net = wkl.net
    layers = wl.layer_tuples(net)
    R = wkl.shards
    prec = "bf16" if net.dtype == wl.BF16 else "f32"
    if net.name == "alexnet":
        nb = wkl.shard_batch
        x, y = wl.make_batch(net, wkl.batch, seed=0)
        w = orc.init_glorot(net.in_shape, layers, 0)
        t0 = time.perf_counter()
        shards = 0
        while shards < R:  # shards 0, 1, ... of the step until the budget is spent
            sl = slice(shards * nb, (shards + 1) * nb)
            orc.train_step(net.in_shape, layers, 1, x[sl], y[sl], w, w * 0, wkl.lr,
                           wkl.momentum, prec=prec, want_grads=False)
            shards += 1
            el = time.perf_counter() - t0
            if el >= budget_s:
                break
        return {"value": round(shards * nb / el, 3), "unit": "samples/s",
                "cores": orc.num_threads(), "cpu": _cpu_model(), "kind": "oracle",
                "sample": f"{shards} shards of the step, each {nb} samples run as R = 1 "
                          f"({prec}), {el:.1f} s; a step is {R} such shards "
                          f"(x{R} extrapolated)"}
    nb = {"mlp": 32, "lenet": 16, "cifar": 1}.get(net.name, 1)
    x, y = wl.make_batch(net, R * nb, seed=0)
    w = orc.init_glorot(net.in_shape, layers, 0)
    v = None if wkl.momentum == 0.0 else w * 0
    t0 = time.perf_counter()
    steps = 0
    while True:
        orc.train_step(net.in_shape, layers, R, x, y, w, v, wkl.lr, wkl.momentum, prec=prec,
                       want_grads=False)
        steps += 1
        el = time.perf_counter() - t0
        if el >= budget_s:
            break
    return {"value": round(steps * R * nb / el, 3), "unit": "samples/s",
            "cores": orc.num_threads(), "cpu": _cpu_model(), "kind": "oracle",
            "sample": f"{steps} oracle steps of {R} shards x {nb} samples ({prec}), {el:.1f} s"}


def source_hash():
    """sha256 over the HIP sources and the C header (identifies the kernels a stored counter
    summary was taken from)."""
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_1704_04560_amd", "csrc")
    for f in sorted(os.listdir(csrc)) + ["../../include/mtx.h"]:
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(f.encode())
            h.update(fh.read())
    return h.hexdigest()


def stored_traffic(workload, site, layer):
    """HBM bytes per launch of a kernel from a committed rocprofv3 counter summary under
    profiles/ (FETCH_SIZE and WRITE_SIZE, scaled by a plain copy of known size), or None when no
    summary covers it or the kernels have changed since it was taken."""
    d = os.path.join(ROOT, "profiles")
    if not os.path.isdir(d):
        return None
    want = source_hash()
    for f in sorted(os.listdir(d)):
        if not f.endswith(".md"):
            continue
        with open(os.path.join(d, f)) as fh:
            for line in fh:
                if not line.startswith("traffic-json: "):
                    continue
                rec = json.loads(line[len("traffic-json: "):])
                if (rec.get("workload") == workload and rec.get("site") == site
                        and rec.get("layer") == layer and rec.get("source_sha256") == want):
                    return rec["bytes_per_launch"]
    return None


def measure(torch, mtx, wl, name, steps, warmup):
    """Timed steps of one workload; returns the bench fields of that workload."""
    wkl = wl.WORKLOADS[name]
    net = wkl.net
    layers = wl.layer_tuples(net)
    model = mtx.Model(net.in_shape, layers, net.dtype, wkl.shards, wkl.shard_batch, seed=0)
    x, y = wl.make_batch(net, wkl.batch, seed=0)
    xd, yd = torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda()
    del x, y
    loss = torch.zeros(1, device="cuda")
    stream = torch.cuda.current_stream()

    for _ in range(warmup):
        model.train_step(xd, yd, wkl.lr, wkl.momentum, loss, stream)
    torch.cuda.synchronize()

    def timed(k):
        t_start = torch.cuda.Event(enable_timing=True)
        t_end = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t_start.record(stream)
        for _ in range(k):
            model.train_step(xd, yd, wkl.lr, wkl.momentum, loss, stream)
        t_end.record(stream)
        torch.cuda.synchronize()
        return t_start.elapsed_time(t_end) / k

    # timed region: K steps as a training loop runs them
    ms = timed(steps)
    assert torch.isfinite(loss).item(), "non-finite loss"
    # the spread of single steps: K more steps, each between its own event pair
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(steps)]
    torch.cuda.synchronize()
    for a, b in evs:
        a.record(stream)
        model.train_step(xd, yd, wkl.lr, wkl.momentum, loss, stream)
        b.record(stream)
    torch.cuda.synchronize()
    single = sorted(a.elapsed_time(b) for a, b in evs)

    def pct(q):
        return round(single[min(len(single) - 1, int(q * (len(single) - 1) + 0.5))], 5)
    # second timed region of K steps with a HIP event pair around every kernel (on the step's
    # stream), for the per-kernel durations behind the roofline figures
    mtx.mtx_set_timing(model.handle, True)
    mtx.mtx_get_timing(model.handle, reset=True)
    ms_events = timed(steps)
    sites = mtx.mtx_get_timing(model.handle)
    mtx.mtx_set_timing(model.handle, False)
    model.close()
    del xd, yd

    es = 2 if net.dtype == wl.BF16 else 4
    geo = geometry(net)
    kernels = []
    fused = sorted({layer for (sname, layer, launches, _) in sites
                    if sname == "wgrad_update" and launches})
    # one entry per (site, layer): the stand-alone average + update can be several launches of
    # a step (one per contiguous range of parameters not updated by a fused launch)
    merged = {}
    for (sname, layer, launches, total) in sites:
        n0, t0 = merged.get((sname, layer), (0, 0.0))
        merged[(sname, layer)] = (n0 + launches, t0 + total)
    sites = [(sname, layer, n, t) for (sname, layer), (n, t) in merged.items()]
    for (sname, layer, launches, total) in sites:
        if launches == 0:
            continue
        bound, work, mm = _site_work(sname, layer, geo, wkl, es, fused)
        per_step = max(1, round(launches / steps))
        if sname == "avg_update":  # launches per step: one per contiguous parameter range
            work /= per_step
        kernels.append(dict(name=sname, layer=layer, avg_ms=total / launches, bound=bound,
                            work=work, mm_flops=mm, per_step=per_step))
    peak_mm = PEAK["bf16_TFLOPs"] if net.dtype == wl.BF16 else PEAK["f32_TFLOPs"]
    # the dominant kernel: the longest one whose algorithmic work is modelled
    dom = max((k for k in kernels if k["bound"]), key=lambda k: k["avg_ms"])
    if dom["bound"] == "mfma":
        ach = dom["work"] / (dom["avg_ms"] * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": round(ach, 3), "peak": peak_mm, "unit": "TFLOP/s"}
        roof["frac"] = round(ach / peak_mm, 4)
    elif dom["bound"] == "alu":
        ach = dom["work"] / (dom["avg_ms"] * 1e-3) / 1e12
        pk = PEAK["f32_vector_TFLOPs"]
        roof = {"bound": "alu", "achieved": round(ach, 3), "peak": pk, "unit": "TFLOP/s",
                "frac": round(ach / pk, 4)}
    else:
        ach = dom["work"] / (dom["avg_ms"] * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(ach, 1), "peak": PEAK["hbm_GBps"],
                "unit": "GB/s"}
        roof["frac"] = round(ach / PEAK["hbm_GBps"], 4)
    roof["traffic"] = stored_traffic(name, dom["name"], dom["layer"])
    roof["kernel"] = f"{dom['name']} (layer {dom['layer']})"
    roof["kernel_ms"] = round(dom["avg_ms"], 5)
    roof["work_per_launch"] = dom["work"]

    mfma_ms = sum(k["avg_ms"] for k in kernels if k["mm_flops"])
    mfma_flops = sum(k["mm_flops"] for k in kernels if k["mm_flops"])
    au = [k for k in kernels if k["name"] == "avg_update"]
    return {
        "wkl": wkl,
        "value": round(wkl.batch / (ms * 1e-3), 1),
        "ms_per_step": round(ms, 5),
        "dtype": "bf16" if net.dtype == wl.BF16 else "f32",
        "roofline": roof,
        "gemm_mfma": {"achieved_TFLOPs": round(mfma_flops / (mfma_ms * 1e-3) / 1e12, 3),
                      "peak_TFLOPs": peak_mm,
                      "frac": round(mfma_flops / (mfma_ms * 1e-3) / 1e12 / peak_mm, 4)},
        # the stand-alone average + update of the step: all its launches together
        "step_avg_update": ({"GBps": round(au[0]["work"] / (au[0]["avg_ms"] * 1e-3) / 1e9, 1),
                             "ms": round(au[0]["avg_ms"] * au[0]["per_step"], 5),
                             "launches": au[0]["per_step"],
                             "params": wkl_params(wkl) - sum(layer_params(geo, f) for f in fused)}
                            if au else None),
        "fused_update_layers": fused,
        "kernel_ms_sum": round(sum(k["avg_ms"] for k in kernels), 5),
        "ms_per_step_with_kernel_events": round(ms_events, 5),
        "step_ms_single": {"median": pct(0.5), "p10": pct(0.1), "p90": pct(0.9),
                           "steps": len(single)},
        "kernels": [{"name": k["name"], "layer": k["layer"], "ms": round(k["avg_ms"], 5)}
                    for k in kernels],
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="alexnet")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-microbench", action="store_true")
    ap.add_argument("--no-extra", action="store_true",
                    help="skip the short runs of the other workloads and the shard sweep")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a plain 512 MiB device copy (torch copy_) so that hardware "
                         "byte counters can be scaled against a kernel of known traffic")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the library has no cross-GPU path (the all-reduce across "
              "GPUs is out of scope); run it with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_1704_04560_amd import mtx
    from paper_1704_04560_amd import workloads as wl

    mtx.lib()  # fails loudly if the HIP library is not built
    if args.copy_calibration:
        src = torch.ones(128 * 1024 * 1024, device="cuda")  # 512 MiB of fp32
        dst = torch.empty_like(src)
        for _ in range(2):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    r = measure(torch, mtx, wl, args.workload, args.steps, args.warmup)
    wkl = r.pop("wkl")
    out = {
        "metric": METRIC,
        "value": r.pop("value"),
        "unit": "samples/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": r.pop("ms_per_step"),
        "higher_is_better": True,
        "scaling": "strong",
        "vs_baseline": None,
        "dtype": r.pop("dtype"),
        "data": "synthetic (seeded; no dataset)",
        "config": {"workload": wkl.description, "global_batch": wkl.batch, "shards": wkl.shards,
                   "shard_batch": wkl.shard_batch, "lr": wkl.lr, "momentum": wkl.momentum,
                   "parallelism": f"{wkl.shards} data-parallel shards on 1 GPU"},
    }
    out.update(r)
    if not args.no_microbench:
        out["grad_avg_update"] = microbench_avg_update(torch, mtx)
    if not args.no_extra:
        extra = {}
        for name in ("mlp", "lenet", "cifar", "alexnet", "resnet", "bottleneck"):
            if name == args.workload:
                continue
            e = measure(torch, mtx, wl, name, 50 if name in ("mlp", "lenet") else 20, 3)
            extra[name] = {"workload": e["wkl"].description, "samples_per_s": e["value"],
                           "ms_per_step": e["ms_per_step"], "dtype": e["dtype"],
                           "roofline": e["roofline"], "gemm_mfma": e["gemm_mfma"],
                           "step_avg_update": e["step_avg_update"],
                           "step_ms_single": e["step_ms_single"]}
            torch.cuda.empty_cache()
        out["other_workloads"] = extra
    if not args.no_extra:
        out["shard_sweep"] = shard_sweep(torch, mtx, wl, "lenet")
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wkl)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
