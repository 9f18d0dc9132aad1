#!/usr/bin/env python3
"""Benchmark: one training step of the CaffeNet conv1-5 stack on one MI355X.

A step is the whole hot path over one batch of 256 synthetic images: the
forward pass of conv1..conv5 (bias + fused ReLU, with 3x3/2 max pooling and
LRN after conv1 and conv2), then the backward pass (ReLU mask, bias
gradient, weight gradient and data gradient of every layer, conv1's data
gradient included, and the glue's backward).  Inputs are resident in HBM
before the timed region starts.

Prints one JSON line.  `value` is the convolution FLOPs of a step (forward +
data gradient + weight gradient, 2 per multiply-add) divided by the wall
time of the whole step, glue included.
"""
import argparse
import json
import os
import platform
import sys
import time

METRIC = ("conv-stack TFLOP/s (% of MFMA peak) + images/sec, CaffeNet conv1-5 fwd+bwd, N=256")
FP32_MFMA_PEAK_TFLOPS = 157.3   # MI355X dense fp32 matrix peak
BF16_MFMA_PEAK_TFLOPS = 2516.6  # MI355X dense bf16 matrix peak (no sparsity)
HBM_PEAK_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--batch", type=int, default=256)
    ap.add_argument("--bf16", action="store_true", help="bfloat16 operands (N=512 workload)")
    ap.add_argument("--cpu-images", type=int, default=192,
                    help="images in the CPU-oracle baseline sample (0 = skip)")
    ap.add_argument("--network-steps", type=int, default=-1,
                    help="steps of the whole-network step (conv1-5, pool5, fc6-fc8) timed "
                         "after the conv stack (-1 = --steps; 0 = skip; fp32 only)")
    ap.add_argument("--network-only", action="store_true",
                    help="time only the whole-network step (profiling); the JSON line then "
                         "carries its images/s as the value")
    ap.add_argument("--calibrate-copy-mb", type=int, default=0,
                    help="first run one plain device copy of this many MiB (a known-size "
                         "reference for the HBM byte counters)")
    return ap.parse_args()


def traffic_record(kernel_source):
    """HBM bytes per launch of the dominant kernel, as measured with the
    FETCH_SIZE / WRITE_SIZE counters and committed under profiles/ -- or None
    when the kernel's source has changed since that measurement."""
    import hashlib
    here = os.path.dirname(os.path.abspath(__file__))
    try:
        rec = json.load(open(os.path.join(here, "profiles", "traffic.json")))
        src = open(os.path.join(here, kernel_source), "rb").read()
    except (OSError, ValueError):
        return None
    if rec.get("source_sha256") != hashlib.sha256(src).hexdigest():
        return None
    return rec


def caffenet_glue(wl):
    return {0: [("pool", wl.CAFFENET_POOL), ("lrn", wl.CAFFENET_LRN)],
            1: [("pool", wl.CAFFENET_POOL), ("lrn", wl.CAFFENET_LRN)]}


def cpu_baseline(inp, wl, n_img):
    """The oracle, as it stands, on the first n_img images of the same batch:
    forward and backward of conv1..5 with the same glue."""
    import numpy as np
    import oracle

    t0 = time.perf_counter()
    x = inp["x"][:n_img]
    acts = []
    for l, L in enumerate(wl.CAFFENET):
        y = oracle.conv_forward(x, inp["W"][l], inp["b"][l], L.s, L.p, L.g, L.relu)
        acts.append((x, y))
        x = y
        if l < 2:
            p, r = wl.CAFFENET_POOL, wl.CAFFENET_LRN
            xp = oracle.maxpool_forward(x, p["kernel"], p["stride"])
            xl = oracle.lrn_forward(xp, r["size"], r["alpha"], r["beta"], r["k"])
            acts[-1] = acts[-1] + (xp,)
            x = xl
    g = inp["top_diff"][:n_img].astype(np.float64)
    for l in range(4, -1, -1):
        L = wl.CAFFENET[l]
        if l < 2:
            p, r = wl.CAFFENET_POOL, wl.CAFFENET_LRN
            xp = acts[l][2]
            g = oracle.lrn_backward(xp, g, r["size"], r["alpha"], r["beta"], r["k"])
            g = oracle.maxpool_backward(acts[l][1], g, p["kernel"], p["stride"])
        dx, _, _ = oracle.conv_backward(acts[l][0], inp["W"][l], g, top=acts[l][1], stride=L.s,
                                        pad=L.p, group=L.g, relu=L.relu)
        g = dx
    dt = time.perf_counter() - t0
    flops = sum(3 * L.flops(n_img) for L in wl.CAFFENET)
    cpu = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                cpu = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": oracle.num_threads(),
            "kind": "oracle", "images_per_s": n_img / dt, "seconds": dt, "cpu": cpu,
            "sample": f"CaffeNet conv1-5 fwd + bwd (with pool/LRN glue) on the first {n_img} "
                      f"of the step's 256 seeded images, plain fp64 loops, OpenMP"}


def network_step(wl, ConvStack, N, steps, warmup, stream):
    """The whole CaffeNet chain -- conv1-5 with their glue, max-pool after
    conv5, the fc6-fc8 inner products -- forward and backward from a
    synthetic fc8 top gradient: images/s and per-layer call times."""
    import numpy as np
    import torch
    print(f"[bench] whole-network step N={N}", file=sys.stderr, flush=True)
    inp = wl.caffenet_net_step(N)
    net = ConvStack(wl.CAFFENET_NET, N, inp["W"], inp["b"], glue=wl.CAFFENET_NET_GLUE)
    x = torch.from_numpy(inp["x"]).cuda()
    g = torch.from_numpy(inp["top_diff"]).cuda()
    for _ in range(warmup):
        net.forward(x, stream)
        net.backward(g, stream)
    torch.cuda.synchronize()
    net.events = []
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    start.record(stream)
    for _ in range(steps):
        net.forward(x, stream)
        net.backward(g, stream)
    end.record(stream)
    torch.cuda.synchronize()
    ms = start.elapsed_time(end) / steps
    acc = {}
    evs, net.events = net.events, None
    for i in range(0, len(evs), 2):
        (tb, eb), (_, ee) = evs[i], evs[i + 1]
        acc.setdefault(tb[:2], []).append(eb.elapsed_time(ee))
    flops = sum(3 * L.flops(N) for L in wl.CAFFENET_NET)
    return {"workload": ("CaffeNet conv1-5 + max-pool + fc6-fc8 (ReLU on fc6, fc7) forward + "
                         "data, weight and bias gradients"),
            "global_batch": N, "ms_per_step": ms, "images_per_s": N / (ms * 1e-3),
            "tflops": flops / (ms * 1e-3) / 1e12, "flops_per_step": flops,
            "breakdown_ms": {f"{k[0]}_{wl.CAFFENET_NET[k[1]].name}": round(float(np.mean(v)), 4)
                             for k, v in sorted(acc.items())}}


def shard_step(wl, ConvStack, steps, warmup, stream, N=32):
    """The conv1-5 step on one GPU's shard of a data-parallel batch (32 of
    8 x 32 images): what each GPU would compute between two gradient
    all-reduces."""
    import torch
    print(f"[bench] conv1-5 step on a shard N={N}", file=sys.stderr, flush=True)
    inp = wl.caffenet_step(N)
    net = ConvStack(wl.CAFFENET, N, inp["W"], inp["b"], glue=caffenet_glue(wl))
    x = torch.from_numpy(inp["x"]).cuda()
    g = torch.from_numpy(inp["top_diff"]).cuda()
    for _ in range(warmup):
        net.forward(x, stream)
        net.backward(g, stream)
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    start.record(stream)
    for _ in range(steps):
        net.forward(x, stream)
        net.backward(g, stream)
    end.record(stream)
    torch.cuda.synchronize()
    ms = start.elapsed_time(end) / steps
    flops = sum(3 * L.flops(N) for L in wl.CAFFENET)
    return {"workload": "CaffeNet conv1-5 training step on a 32-image shard", "global_batch": N,
            "ms_per_step": ms, "images_per_s": N / (ms * 1e-3),
            "tflops": flops / (ms * 1e-3) / 1e12}


def lenet_training(wl, ConvStack, steps, warmup, stream, N=64):
    """LeNet training iterations (forward, softmax loss, backward, SGD update
    of every blob) at N=64 on one resident synthetic batch: images/s."""
    import torch
    from paper_1408_5093_amd.net import SGDTrainer
    print(f"[bench] LeNet training N={N}", file=sys.stderr, flush=True)
    inp = wl.lenet_train(N, 1)
    net = ConvStack(wl.LENET_NET, N, inp["W"], inp["b"], glue=wl.LENET_NET_GLUE)
    sol = dict(wl.LENET_SOLVER)
    tr = SGDTrainer(net, momentum=sol.pop("momentum"), weight_decay=sol.pop("weight_decay"),
                    **sol)
    x = torch.from_numpy(inp["x"][0]).cuda()
    y = torch.from_numpy(inp["labels"][0]).cuda()
    for _ in range(warmup):
        tr.step(x, y, stream)
    torch.cuda.synchronize()

    def timed(fn):
        start = torch.cuda.Event(enable_timing=True)
        end = torch.cuda.Event(enable_timing=True)
        start.record(stream)
        for _ in range(steps):
            fn()
        end.record(stream)
        torch.cuda.synchronize()
        return start.elapsed_time(end) / steps

    ms_eager = timed(lambda: tr.step(x, y, stream))
    # the same iteration captured once as a HIP graph and replayed (the
    # per-launch host cost of ~40 small kernels is what the eager loop pays)
    tr.capture(x, y)
    for _ in range(warmup):
        tr.replay()
    torch.cuda.synchronize()
    ms = timed(tr.replay)
    return {"workload": ("LeNet training iteration: conv1, max-pool, conv2, max-pool, ip1 + ReLU, "
                         "ip2, softmax loss, backward, SGD (momentum 0.9, decay 5e-4, inv "
                         "schedule), replayed as one captured HIP graph"),
            "global_batch": N, "ms_per_step": ms, "images_per_s": N / (ms * 1e-3),
            "ms_per_step_eager": ms_eager, "images_per_s_eager": N / (ms_eager * 1e-3),
            "final_loss": float(tr.loss.item())}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py: measures one GPU only (asked for --gpus {args.gpus}); the library "
              "runs one GPU's share of a data-parallel step and does no collectives",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_1408_5093_amd as cc
    from paper_1408_5093_amd import workloads as wl
    from paper_1408_5093_amd.net import ConvStack

    cc.load()  # fails loudly when the HIP library is missing
    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        sys.exit(3)
    if args.network_only:
        from paper_1408_5093_amd import workloads as wl
        stream = torch.cuda.current_stream()
        r = network_step(wl, ConvStack, args.batch, args.steps, args.warmup, stream)
        print(json.dumps({"metric": "CaffeNet whole-network training images/s", "value":
                          r["images_per_s"], "unit": "images/s", "n_gpus": 1, "steps": args.steps,
                          "warmup": args.warmup, "ms_per_step": r["ms_per_step"],
                          "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
                          "dtype": "f32", "data": "synthetic", "config": {
                              "workload": r["workload"], "global_batch": args.batch},
                          "network": r}), flush=True)
        return
    N = args.batch if not args.bf16 or args.batch != 256 else 512
    workload = wl.CAFFENET_STEP_BF16 if args.bf16 else wl.CAFFENET_STEP
    print(f"[bench] generating seeded inputs N={N}", file=sys.stderr, flush=True)
    inp = wl.caffenet_step(N, workload)
    if args.bf16:
        inp["x"] = wl.round_bf16(inp["x"])
    net = ConvStack(wl.CAFFENET, N, inp["W"], inp["b"], glue=caffenet_glue(wl), bf16=args.bf16)
    x = torch.from_numpy(inp["x"]).cuda()
    g = torch.from_numpy(inp["top_diff"]).cuda()
    stream = torch.cuda.current_stream()
    if args.calibrate_copy_mb > 0:
        n = args.calibrate_copy_mb * (1 << 20) // 4
        src = torch.ones(n, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    def step():
        net.forward(x, stream)
        net.backward(g, stream)

    print(f"[bench] warmup {args.warmup}", file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # timed region: events around every convolution call, on the library's stream
    net.events = []
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    start.record(stream)
    for _ in range(args.steps):
        step()
    end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms_step = start.elapsed_time(end) / args.steps
    print(f"[bench] {args.steps} steps, {ms_step:.3f} ms/step", file=sys.stderr, flush=True)

    # per-call durations (ms), averaged over the timed steps
    # (the weight-gradient calls, "wgt", run on a second stream beside the
    # data gradients: conv_ms is the time covered by at least one call)
    acc = {}
    spans = []
    evs = net.events
    net.events = None
    for i in range(0, len(evs), 2):
        (tag_b, eb), (tag_e, ee) = evs[i], evs[i + 1]
        assert tag_b[:2] == tag_e[:2] and tag_b[2] == "begin" and tag_e[2] == "end"
        acc.setdefault(tag_b[:2], []).append(eb.elapsed_time(ee))
        spans.append((start.elapsed_time(eb), start.elapsed_time(ee)))
    call_ms = {k: float(np.mean(v)) for k, v in acc.items()}
    covered, reach = 0.0, float("-inf")
    for b0, b1 in sorted(spans):
        if b1 > reach:
            covered += b1 - max(b0, reach)
            reach = b1

    flops_step = sum(3 * L.flops(N) for L in wl.CAFFENET)
    conv_ms = covered / args.steps
    peak = BF16_MFMA_PEAK_TFLOPS if args.bf16 else FP32_MFMA_PEAK_TFLOPS
    tflops = flops_step / (ms_step * 1e-3) / 1e12

    # roofline of the dominant single-kernel call: the slowest forward (one
    # implicit-GEMM launch per call)
    fwd = {k: v for k, v in call_ms.items() if k[0] == "fwd"}
    kdom = max(fwd, key=fwd.get)
    Ldom = wl.CAFFENET[kdom[1]]
    ach = Ldom.flops(N) / (fwd[kdom] * 1e-3) / 1e12
    rec = traffic_record("paper_1408_5093_amd/csrc/conv_gemm.hip")
    traffic = None
    if rec and rec.get("layer") == Ldom.name and rec.get("batch") == N and not args.bf16:
        traffic = rec["bytes_per_launch"]
    roofline = {"bound": "mfma", "achieved": ach, "peak": peak, "unit": "TFLOP/s",
                "frac": ach / peak, "traffic": traffic,
                "kernel": f"conv_gemm (forward, {Ldom.name})",
                "kernel_ms": fwd[kdom], "flops_per_launch": Ldom.flops(N)}

    breakdown = {f"{k[0]}_{wl.CAFFENET[k[1]].name}": round(v, 4) for k, v in sorted(call_ms.items())}
    out = {
        "metric": METRIC,
        "value": tflops,
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if args.bf16 else "f32",
        "data": "synthetic (seeded N(0,50) pixels, N(0,0.01) weights, N(0,1e-3) top gradient)",
        "config": {"workload": ("CaffeNet conv1-5 training step: forward (bias+ReLU) + data, "
                                "weight and bias gradients, 3x3/2 max-pool + LRN(5) glue after "
                                "conv1 and conv2"),
                   "global_batch": N, "image": "3x227x227",
                   "operands": "bf16" if args.bf16 else "fp32", "accumulate": "fp32"},
        "images_per_s": N / (ms_step * 1e-3),
        "pct_mfma_peak": 100.0 * tflops / peak,
        "conv_tflops_in_conv_calls": flops_step / (conv_ms * 1e-3) / 1e12,
        "conv_calls_ms_per_step": conv_ms,
        "flops_per_step": flops_step,
        "wall_s": wall,
        "breakdown_ms": breakdown,
        "roofline": roofline,
        "cpu_baseline": None,
    }
    nsteps = args.steps if args.network_steps < 0 else args.network_steps
    if nsteps > 0 and not args.bf16:
        out["network"] = network_step(wl, ConvStack, N, nsteps, args.warmup, stream)
        out["lenet_training"] = lenet_training(wl, ConvStack, 10 * nsteps, args.warmup, stream)
        out["shard_n32"] = shard_step(wl, ConvStack, nsteps, args.warmup, stream)
    if args.cpu_images > 0:
        print(f"[bench] CPU oracle baseline on {args.cpu_images} images", file=sys.stderr,
              flush=True)
        out["cpu_baseline"] = cpu_baseline(inp, wl, args.cpu_images)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
