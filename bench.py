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
time of the whole step, glue included.  The same line carries the other
workloads as objects of their own: the LeNet conv pair (N=64), CaffeNet
conv1's forward pass and conv2-5's forward passes (N=256), and the conv1-5
step at N=512 with bfloat16 operands.
"""
import argparse
import json
import os
import sys
import threading
import time

METRIC = ("conv-stack TFLOP/s (% of MFMA peak) + images/sec, CaffeNet conv1-5 fwd+bwd, N=256")
FP32_MFMA_PEAK_TFLOPS = 157.3   # MI355X dense fp32 matrix peak (256 CUs at 2.4 GHz)
BF16_MFMA_PEAK_TFLOPS = 2516.6  # MI355X dense bf16 matrix peak (no sparsity)
SPEC_SCLK_MHZ = 2400.0
HBM_PEAK_GBS = 8000.0
PAPER_CONTEXT = ("over 40 million images per day, about 2.5 ms per image, on one NVIDIA K40 or "
                 "Titan (whole system; model, batch and pass not stated): context, not a target")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--batch", type=int, default=256)
    ap.add_argument("--bf16", action="store_true",
                    help="time the bfloat16 step (N=512 workload) as the headline (profiling)")
    ap.add_argument("--cpu-images", type=int, default=256,
                    help="images in the CPU-oracle baseline sample (0 = skip)")
    ap.add_argument("--network-steps", type=int, default=-1,
                    help="steps of the whole-network step (conv1-5, pool5, fc6-fc8) timed "
                         "after the conv stack (-1 = --steps; 0 = skip; fp32 only)")
    ap.add_argument("--network-only", action="store_true",
                    help="time only the whole-network step (profiling); the JSON line then "
                         "carries its images/s as the value")
    ap.add_argument("--configs", choices=("all", "none"), default="all",
                    help="also time the LeNet pair, conv1 forward, conv2-5 forward and bf16 "
                         "workloads (none: the headline step only, for profiling)")
    ap.add_argument("--headline-only", action="store_true",
                    help="only the warm-up and timed steps of the headline workload: no "
                         "serialized pass, clock sampling, other workloads or CPU baseline (for "
                         "kernel traces and counter runs, whose per-step figures then cover the "
                         "timed steps alone)")
    ap.add_argument("--one-stream", action="store_true",
                    help="issue the fp32 weight gradients on the caller's stream in the timed "
                         "steps too (measurement of the overlap)")
    ap.add_argument("--calibrate-copy-mb", type=int, default=0,
                    help="first run one plain device copy of this many MiB (a known-size "
                         "reference for the HBM byte counters)")
    return ap.parse_args()


# ------------------------------------------------------------ accounting
def call_flops(kind, L, N):
    """FLOPs of one library call: one pass, or two for a combined backward."""
    return (2 if kind == "both" else 1) * L.flops(N)


def kernel_of(kind, L, bf16):
    """The GEMM kernel(s) a call of this kind runs for layer L."""
    if bf16:
        return {"fwd": "conv_gemm_bf16_kernel (forward)",
                "bwd": "conv_gemm_bf16_kernel (data gradient)",
                "wgt": "conv_wgrad_bf16_kernel",
                "both": "conv_gemm_bf16_kernel (data gradient) + conv_wgrad_bf16_kernel"}[kind]
    if L.H == 1 and L.W == 1 and L.k == 1:
        return "dense_gemm (inner product)"
    # (the quad-order layers run the LDS-DMA variant of the quad kernel)
    quad = (L.C // L.g) % 4 == 0 and L.k in (3, 5)
    wgt = "conv_wgrad_dma_f32_kernel" if quad else "conv_wgrad_f32_kernel"
    return {"fwd": "conv_gemm_f32_kernel (forward)",
            "bwd": "conv_gemm_f32_kernel (data gradient)",
            "wgt": wgt,
            "both": f"conv_gemm_f32_kernel (data gradient) + {wgt}"}[kind]


def timed_steps(step, stream, steps, net=None):
    """Run `steps` steps between two events on `stream`; with `net`, also
    the mean duration of every library call (events around each call, on
    the stream it is issued on) and the time covered by at least one call."""
    import torch
    import numpy as np
    if net is not None:
        net.events = []
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    start.record(stream)
    for _ in range(steps):
        step()
    end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms = start.elapsed_time(end) / steps
    if net is None:
        return ms, wall, None, None
    acc, spans = {}, []
    evs, net.events = net.events, None
    # a call's span runs from its "begin" event to the latest of its "end"
    # events (one per stream its work is ordered on)
    calls, open_ = [], {}
    for tag, ev in evs:
        if tag[2] == "begin":
            open_[tag[:2]] = [tag[:2], ev, []]
            calls.append(open_[tag[:2]])
        else:
            open_[tag[:2]][2].append(ev)
    for key, eb, ends in calls:
        assert ends, key
        d = max(eb.elapsed_time(ee) for ee in ends)
        acc.setdefault(key, []).append(d)
        b0 = start.elapsed_time(eb)
        spans.append((b0, b0 + d))
    covered, reach = 0.0, float("-inf")
    for b0, b1 in sorted(spans):
        if b1 > reach:
            covered += b1 - max(b0, reach)
            reach = b1
    return ms, wall, {k: float(np.mean(v)) for k, v in acc.items()}, covered / steps


def roofline(call_ms, layers, N, peak, bf16, sclk=None):
    """Roofline record of the dominant call: the call with the largest mean
    duration per step in `call_ms` (each runs one GEMM kernel, plus small
    table/reduce kernels counted in its duration)."""
    key = max(call_ms, key=call_ms.get)
    kind, l = key
    L = layers[l]
    flops = call_flops(kind, L, N)
    ach = flops / (call_ms[key] * 1e-3) / 1e12
    rec = {"bound": "mfma", "achieved": ach, "peak": peak, "unit": "TFLOP/s",
           "frac": ach / peak, "traffic": None, "call": f"{kind}_{L.name}",
           "kernel": f"{kernel_of(kind, L, bf16)}, {L.name}",
           "kernel_ms": call_ms[key], "flops_per_launch": flops}
    if sclk:
        p = peak * sclk / SPEC_SCLK_MHZ
        rec["peak_at_observed_sclk"] = p
        rec["frac_at_observed_sclk"] = ach / p
    return rec


def traffic_record(call, batch, bf16):
    """HBM bytes per launch of a call's GEMM kernel, as measured with the
    FETCH_SIZE / WRITE_SIZE counters and committed under profiles/ -- or None
    when none was measured for it or its source has changed since."""
    import hashlib
    here = os.path.dirname(os.path.abspath(__file__))
    try:
        recs = json.load(open(os.path.join(here, "profiles", "traffic.json")))
    except (OSError, ValueError):
        return None
    for rec in recs.get("kernels", []):
        if rec.get("call") != call or rec.get("batch") != batch or rec.get("bf16", False) != bf16:
            continue
        try:
            src = open(os.path.join(here, rec["source"]), "rb").read()
        except (OSError, KeyError):
            return None
        if rec.get("source_sha256") != hashlib.sha256(src).hexdigest():
            return None
        return rec
    return None


def observed_sclk(work, bus_id):
    """Median graphics clock (MHz, mean over the XCDs) that the SMU reports
    while `work` runs and the device is at least 90% busy, sampled every
    20 ms through amdsmi for the device on PCI bus `bus_id`.  The SMU
    refreshes these metrics about once a second, so `work` should run for
    a few seconds.  None when amdsmi or the device cannot be read."""
    try:
        import amdsmi
        amdsmi.amdsmi_init()
    except Exception:
        work()
        return None
    try:
        handle = None
        for h in amdsmi.amdsmi_get_processor_handles():
            bdf = amdsmi.amdsmi_get_gpu_device_bdf(h)
            if int(bdf.split(":")[1], 16) == bus_id:
                handle = h
        if handle is None:
            work()
            return None
        samples, stop = [], threading.Event()

        def poll():
            while not stop.is_set():
                try:
                    m = amdsmi.amdsmi_get_gpu_metrics_info(handle)
                    clks = [float(c) for c in m.get("current_gfxclks", []) if isinstance(c, (int, float))]
                    if clks and float(m.get("average_gfx_activity", 0)) >= 90:
                        samples.append(sum(clks) / len(clks))
                except Exception:
                    pass
                time.sleep(0.02)

        t = threading.Thread(target=poll, daemon=True)
        t.start()
        work()
        stop.set()
        t.join()
        samples.sort()
        return samples[len(samples) // 2] if samples else None
    except Exception:
        return None
    finally:
        try:
            amdsmi.amdsmi_shut_down()
        except Exception:
            pass


def caffenet_glue(wl):
    return {0: [("pool", wl.CAFFENET_POOL), ("lrn", wl.CAFFENET_LRN)],
            1: [("pool", wl.CAFFENET_POOL), ("lrn", wl.CAFFENET_LRN)]}


# ------------------------------------------------------------ CPU baseline
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
    n_all = inp["x"].shape[0]
    which = f"all {n_img}" if n_img >= n_all else f"the first {n_img}"
    return {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": oracle.num_threads(),
            "kind": "oracle", "images_per_s": n_img / dt, "seconds": dt, "cpu": cpu,
            "sample": f"CaffeNet conv1-5 fwd + bwd (with pool/LRN glue) on {which} of the "
                      f"step's {n_all} seeded images (full batch: {n_img >= n_all}), plain fp64 "
                      f"loops, OpenMP"}


# ------------------------------------------------------------ other workloads
def network_step(wl, ConvStack, N, steps, warmup, stream):
    """The whole CaffeNet chain -- conv1-5 with their glue, max-pool after
    conv5, the fc6-fc8 inner products -- forward and backward from a
    synthetic fc8 top gradient: images/s and per-layer call times."""
    import torch
    print(f"[bench] whole-network step N={N}", file=sys.stderr, flush=True)
    inp = wl.caffenet_net_step(N)
    net = ConvStack(wl.CAFFENET_NET, N, inp["W"], inp["b"], glue=wl.CAFFENET_NET_GLUE)
    x = torch.from_numpy(inp["x"]).cuda()
    g = torch.from_numpy(inp["top_diff"]).cuda()

    def step():
        net.forward(x, stream)
        net.backward(g, stream)

    for _ in range(warmup):
        step()
    # per-call events in steps of their own: the timed steps carry none
    _, _, call_ms, _ = timed_steps(step, stream, max(2, min(steps, 5)), net)
    ms, _, _, _ = timed_steps(step, stream, steps)
    flops = sum(3 * L.flops(N) for L in wl.CAFFENET_NET)
    return {"workload": ("CaffeNet conv1-5 + max-pool + fc6-fc8 (ReLU on fc6, fc7) forward + "
                         "data, weight and bias gradients"),
            "global_batch": N, "ms_per_step": ms, "images_per_s": N / (ms * 1e-3),
            "tflops": flops / (ms * 1e-3) / 1e12, "flops_per_step": flops,
            "breakdown_ms": {f"{k[0]}_{wl.CAFFENET_NET[k[1]].name}": round(v, 4)
                             for k, v in sorted(call_ms.items())}}


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

    def step():
        net.forward(x, stream)
        net.backward(g, stream)

    for _ in range(warmup):
        step()
    ms, _, _, _ = timed_steps(step, stream, steps)
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
    ms_eager, _, _, _ = timed_steps(lambda: tr.step(x, y, stream), stream, steps)
    # the same iteration captured once as a HIP graph and replayed (the
    # per-launch host cost of ~40 small kernels is what the eager loop pays)
    tr.capture(x, y)
    for _ in range(warmup):
        tr.replay()
    ms, _, _, _ = timed_steps(tr.replay, stream, steps)
    return {"workload": ("LeNet training iteration: conv1, max-pool, conv2, max-pool, ip1 + ReLU, "
                         "ip2, softmax loss, backward, SGD (momentum 0.9, decay 5e-4, inv "
                         "schedule), replayed as one captured HIP graph"),
            "global_batch": N, "ms_per_step": ms, "images_per_s": N / (ms * 1e-3),
            "ms_per_step_eager": ms_eager, "images_per_s_eager": N / (ms_eager * 1e-3),
            "final_loss": float(tr.loss.item())}


def rate_record(workload, N, ms, flops, peak, dtype, **extra):
    r = {"workload": workload, "global_batch": N, "dtype": dtype, "ms_per_step": ms,
         "tflops": flops / (ms * 1e-3) / 1e12, "flops_per_step": flops,
         "pct_mfma_peak": 100.0 * flops / (ms * 1e-3) / 1e12 / peak,
         "images_per_s": N / (ms * 1e-3)}
    r.update(extra)
    return r


def lenet_pair(wl, ConvStack, steps, warmup, stream, N=64):
    """LeNet conv pair (conv1, 2x2/2 max-pool, conv2), fp32, N=64: forward
    and backward (data, weight and bias gradients of both layers) from an
    N(0, 1) top gradient."""
    import torch
    print(f"[bench] LeNet conv pair N={N}", file=sys.stderr, flush=True)
    inp = wl.lenet_pair(N)
    net = ConvStack(wl.LENET, N, inp["W"], inp["b"], glue={0: [("pool", wl.LENET_POOL)]})
    x = torch.from_numpy(inp["x"]).cuda()
    g = torch.from_numpy(inp["top_diff"]).cuda()

    def step():
        net.forward(x, stream)
        net.backward(g, stream)

    for _ in range(warmup):
        step()
    ms, _, _, _ = timed_steps(step, stream, steps)
    flops = sum(3 * L.flops(N) for L in wl.LENET)
    return rate_record("LeNet conv pair: conv1 20x5x5, 2x2/2 max-pool, conv2 50x5x5, forward + "
                       "data, weight and bias gradients", N, ms, flops, FP32_MFMA_PEAK_TFLOPS,
                       "f32")


def forward_only(cc, layers, inputs, steps, warmup, stream, N):
    """Forward passes of `layers` on their own seeded inputs: per layer and
    in all, each call timed on its own between events."""
    import torch
    per = {}
    total_ms, total_flops = 0.0, 0
    for L, inp in zip(layers, inputs):
        d = cc.conv_desc((N, L.C, L.H, L.W), (L.K, L.C // L.g, L.k, L.k), L.s, L.p, L.g, L.relu)
        Ho, Wo = cc.conv_out_shape(d)
        x = torch.from_numpy(inp["x"]).cuda()
        w = torch.from_numpy(inp["W"]).cuda()
        b = torch.from_numpy(inp["b"]).cuda()
        y = torch.empty((N, L.K, Ho, Wo), device="cuda")
        ws = cc.Workspace().get(cc.conv_workspace_size(d, cc.PASS_FORWARD))

        def call():
            cc.caffe_conv_forward(d, x, w, b, y, ws, stream)

        for _ in range(warmup):
            call()
        ms, _, _, _ = timed_steps(call, stream, steps)
        flops = L.flops(N)
        per[L.name] = {"ms": ms, "tflops": flops / (ms * 1e-3) / 1e12,
                       "pct_mfma_peak": 100.0 * flops / (ms * 1e-3) / 1e12 / FP32_MFMA_PEAK_TFLOPS}
        total_ms += ms
        total_flops += flops
        del x, w, b, y, ws
    return total_ms, total_flops, per


def conv1_forward(cc, wl, steps, warmup, stream, N=256):
    print(f"[bench] CaffeNet conv1 forward N={N}", file=sys.stderr, flush=True)
    ms, flops, _ = forward_only(cc, wl.CAFFENET[:1], [wl.caffenet_conv1_fwd(N)], steps, warmup,
                                stream, N)
    return rate_record("CaffeNet conv1 forward: 3x227x227 -> 96x55x55, 11x11 stride 4, bias + "
                       "fused ReLU", N, ms, flops, FP32_MFMA_PEAK_TFLOPS, "f32")


def conv25_forward(cc, wl, steps, warmup, stream, N=256):
    print(f"[bench] CaffeNet conv2-5 forward N={N}", file=sys.stderr, flush=True)
    ms, flops, per = forward_only(cc, wl.CAFFENET[1:],
                                  [wl.caffenet_conv25_layer(l, N) for l in range(1, 5)], steps,
                                  warmup, stream, N)
    return rate_record("CaffeNet conv2-5 forward, each layer on its own half-normal input, bias "
                       "0.1 + fused ReLU (ms_per_step = the four calls back to back)", N, ms, flops,
                       FP32_MFMA_PEAK_TFLOPS, "f32", per_layer=per)


def conv_step(cc, wl, ConvStack, N, bf16, steps, warmup, stream, one_stream=False,
              serialized=True):
    """The conv1-5 training step: per-step time, per-call durations, the
    roofline of the dominant call, and (fp32) the same calls issued one
    stream (each call alone on the device)."""
    import torch
    workload = wl.CAFFENET_STEP_BF16 if bf16 else wl.CAFFENET_STEP
    print(f"[bench] generating seeded inputs N={N}{' bf16' if bf16 else ''}", file=sys.stderr,
          flush=True)
    inp = wl.caffenet_step(N, workload)
    if bf16:
        inp["x"] = wl.round_bf16(inp["x"])
    net = ConvStack(wl.CAFFENET, N, inp["W"], inp["b"], glue=caffenet_glue(wl), bf16=bf16)
    net.serial = one_stream
    x = torch.from_numpy(inp["x"]).cuda()
    g = torch.from_numpy(inp["top_diff"]).cuda()

    def step():
        net.forward(x, stream)
        net.backward(g, stream)

    print(f"[bench] warmup {warmup}", file=sys.stderr, flush=True)
    for _ in range(warmup):
        step()
    # Every call between events, in steps of their own before the timed
    # region: each event record holds its stream for several microseconds,
    # so the timed steps mark only the dominant call (the one the roofline
    # record is about), measured live on the stream it is issued on.
    _, _, call_ms, covered = timed_steps(step, stream, max(2, min(steps, 5)), net)
    dominant = max(call_ms, key=call_ms.get)
    net.mark_only = {dominant}
    ms, wall, live_ms, _ = timed_steps(step, stream, steps, net)
    net.mark_only = None
    print(f"[bench] {steps} steps, {ms:.3f} ms/step", file=sys.stderr, flush=True)
    out = {"inp": inp, "net": net, "x": x, "g": g, "step": step, "ms": ms, "wall": wall,
           "call_ms": call_ms, "live_ms": live_ms, "covered": covered}
    if serialized and not bf16 and not one_stream:
        net.serial = True
        for _ in range(2):
            step()
        _, _, out["call_ms_serial"], _ = timed_steps(step, stream, steps, net)
        net.serial = False
        print("[bench] serialized calls timed", file=sys.stderr, flush=True)
    return out


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py: measures one GPU only (asked for --gpus {args.gpus}); the library "
              "runs one GPU's share of a data-parallel step and does no collectives",
              file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_1408_5093_amd as cc
    from paper_1408_5093_amd import workloads as wl
    from paper_1408_5093_amd.net import ConvStack

    cc.load()  # fails loudly when the HIP library is missing
    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        sys.exit(3)
    stream = torch.cuda.current_stream()
    if args.network_only:
        r = network_step(wl, ConvStack, args.batch, args.steps, args.warmup, stream)
        print(json.dumps({"metric": "CaffeNet whole-network training images/s", "value":
                          r["images_per_s"], "unit": "images/s", "n_gpus": 1, "steps": args.steps,
                          "warmup": args.warmup, "ms_per_step": r["ms_per_step"],
                          "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
                          "dtype": "f32", "data": "synthetic", "config": {
                              "workload": r["workload"], "global_batch": args.batch},
                          "network": r}), flush=True)
        return
    if args.calibrate_copy_mb > 0:
        n = args.calibrate_copy_mb * (1 << 20) // 4
        src = torch.ones(n, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    bf16 = args.bf16
    N = args.batch if not bf16 or args.batch != 256 else 512
    peak = BF16_MFMA_PEAK_TFLOPS if bf16 else FP32_MFMA_PEAK_TFLOPS
    if args.headline_only:
        args.configs, args.network_steps, args.cpu_images = "none", 0, 0
    run = conv_step(cc, wl, ConvStack, N, bf16, args.steps, args.warmup, stream,
                    one_stream=args.one_stream, serialized=not args.headline_only)
    ms_step, call_ms = run["ms"], run["call_ms"]
    flops_step = sum(3 * L.flops(N) for L in wl.CAFFENET)
    tflops = flops_step / (ms_step * 1e-3) / 1e12

    # graphics clock while the same steps run again (not part of the timed region)
    props = torch.cuda.get_device_properties(0)
    nsclk = max(1, int(2.5 / (ms_step * 1e-3)))

    def clock_work():
        for i in range(nsclk):
            run["step"]()
            if i % 20 == 19:  # keep the host close to the device
                torch.cuda.synchronize()
        torch.cuda.synchronize()

    sclk = None
    if not args.headline_only:
        sclk = observed_sclk(clock_work, getattr(props, "pci_bus_id", -1))
        print(f"[bench] observed sclk {sclk} MHz", file=sys.stderr, flush=True)

    roof = roofline(run["live_ms"], wl.CAFFENET, N, peak, bf16, sclk)
    roof["traffic"] = (traffic_record(roof["call"], N, bf16) or {}).get("bytes_per_launch")
    roof["duration_source"] = ("HIP events around the call on the stream it is issued on, mean "
                               "over the timed steps (the call's small table and reduce kernels "
                               "included); the call is the longest one of breakdown_ms, whose "
                               "steps, before the timed region, put events around every call")
    ser = run.get("call_ms_serial")
    if ser:
        key = next(k for k in ser if f"{k[0]}_{wl.CAFFENET[k[1]].name}" == roof["call"])
        a = call_flops(key[0], wl.CAFFENET[key[1]], N) / (ser[key] * 1e-3) / 1e12
        roof["serialized"] = {"kernel_ms": ser[key], "achieved": a, "frac": a / peak}
        dom = roofline(ser, wl.CAFFENET, N, peak, bf16, sclk)
        roof["dominant_serialized"] = {k: dom[k] for k in ("call", "kernel", "kernel_ms",
                                                           "achieved", "frac")}
        roof["note"] = ("kernel_ms is the call's duration in the timed steps, where the weight "
                        "gradients run on a second stream beside the data gradients and both "
                        "stretch; 'serialized' times the same calls issued one after another on "
                        "one stream")

    def names(d):
        return {f"{k[0]}_{wl.CAFFENET[k[1]].name}": round(v, 4) for k, v in sorted(d.items())}

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
        "dtype": "bf16" if bf16 else "f32",
        "data": "synthetic (seeded N(0,50) pixels, N(0,0.01) weights, N(0,1e-3) top gradient)",
        "config": {"workload": ("CaffeNet conv1-5 training step: forward (bias+ReLU) + data, "
                                "weight and bias gradients, 3x3/2 max-pool + LRN(5) glue after "
                                "conv1 and conv2"),
                   "global_batch": N, "image": "3x227x227",
                   "operands": "bf16" if bf16 else "fp32", "accumulate": "fp32",
                   "weight_gradient_stream": "caller's" if args.one_stream else "second"},
        "images_per_s": N / (ms_step * 1e-3),
        "pct_mfma_peak": 100.0 * tflops / peak,
        "observed_sclk_mhz": sclk,
        "pct_mfma_peak_at_observed_sclk": (100.0 * tflops / (peak * sclk / SPEC_SCLK_MHZ)
                                           if sclk else None),
        "conv_tflops_in_conv_calls": flops_step / (run["covered"] * 1e-3) / 1e12,
        "conv_calls_ms_per_step": run["covered"],
        "flops_per_step": flops_step,
        "wall_s": run["wall"],
        "breakdown_ms": names(call_ms),
        "breakdown_source": ("HIP events around every call, in steps run before the timed "
                             "region (the timed steps mark only the roofline's call)"),
        "roofline": roof,
        "cpu_baseline": None,
        "paper_context": PAPER_CONTEXT,
    }
    if ser:
        out["breakdown_ms_serialized"] = names(ser)
    inp = run["inp"]
    del run
    torch.cuda.empty_cache()

    if args.configs == "all" and not bf16:
        out["lenet_pair"] = lenet_pair(wl, ConvStack, 10 * args.steps, args.warmup, stream)
        out["conv1_forward"] = conv1_forward(cc, wl, 2 * args.steps, args.warmup, stream)
        out["conv2_5_forward"] = conv25_forward(cc, wl, 2 * args.steps, args.warmup, stream)
        torch.cuda.empty_cache()
        b = conv_step(cc, wl, ConvStack, 512, True, args.steps, args.warmup, stream,
                      serialized=False)
        bflops = sum(3 * L.flops(512) for L in wl.CAFFENET)
        br = rate_record("CaffeNet conv1-5 training step with bfloat16 inputs and weights, fp32 "
                         "accumulation and outputs, same glue", 512, b["ms"], bflops,
                         BF16_MFMA_PEAK_TFLOPS, "bf16", breakdown_ms=names(b["call_ms"]))
        br["roofline"] = roofline(b["live_ms"], wl.CAFFENET, 512, BF16_MFMA_PEAK_TFLOPS, True,
                                  sclk)
        br["roofline"]["traffic"] = (traffic_record(br["roofline"]["call"], 512, True)
                                     or {}).get("bytes_per_launch")
        out["bf16_step_n512"] = br
        del b
        torch.cuda.empty_cache()
    nsteps = args.steps if args.network_steps < 0 else args.network_steps
    if nsteps > 0 and not bf16:
        out["network"] = network_step(wl, ConvStack, N, nsteps, args.warmup, stream)
        out["lenet_training"] = lenet_training(wl, ConvStack, 10 * nsteps, args.warmup, stream)
        out["shard_n32"] = shard_step(wl, ConvStack, nsteps, args.warmup, stream)
    if args.cpu_images > 0:
        n = min(args.cpu_images, N)
        print(f"[bench] CPU oracle baseline on {n} images", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(inp, wl, n)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
