"""Benchmark: one all-FP16 training step of the ResNet-50 conv2_x bottleneck
block at batch 32 (56x56, 256->64->64->256 channels) on one MI355X.

A step is the whole hot path over one synthetic batch: three convolution
forwards, three fused BN(0.25)+ReLU forwards (the last with the identity
shortcut), their backwards, three data and three weight gradients, and the
FP16 momentum-SGD update of every parameter.  Inputs are resident in HBM
before timing; the step is captured once in a HIP graph and replayed.

Prints one JSON line: the headline value is the convolution throughput of the
step (fwd + dgrad + wgrad FLOPs / step time, TFLOP/s), with images/s, the
fraction of the FP16 matrix-core peak, a per-call breakdown measured with HIP
events, the roofline of the dominant kernel, and the CPU oracle's rate on a
bounded sample of the same step.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_FP16_TFLOPS = 2516.6   # MI355X dense FP16 matrix cores: 256 CU x 2.4 GHz x 4096 FLOP/clk
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
METRIC = "FP16 conv TFLOP/s (fwd+dgrad+wgrad) as % MFMA peak; ResNet-50 train images/sec"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--batch", type=int, default=32)
    ap.add_argument("--eager", action="store_true", help="no HIP graph")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="target duration of the CPU oracle sample")
    ap.add_argument("--sweep", action="store_true",
                    help="also time all 23 ResNet-50 conv shapes (53 layers) at batch 128")
    ap.add_argument("--no-sweep3x3", action="store_true",
                    help="skip the batch-128 3x3-layer sweep")
    ap.add_argument("--no-resnet50", action="store_true",
                    help="skip the full ResNet-50 training step at batch 128")
    ap.add_argument("--resnet50-steps", type=int, default=10)
    ap.add_argument("--no-f16-arith", action="store_true",
                    help="skip the strict binary16-arithmetic timing leg")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="first run three device-to-device copies of MIB MiB (a plain copy of "
                         "known size, the yardstick for the HBM byte counters)")
    return ap.parse_args()


def call_work(name, s):
    """Algorithmic work of one ABI call of the step: (flops, bytes, bound)."""
    n, hw, c, w = s.n, s.hw, s.c, s.width
    m = n * hw * hw
    convs = {"conv1": (c, w, 1), "conv2": (w, w, 3), "conv3": (w, c, 1)}
    if name.startswith("conv") and "_bn" in name:
        # fused conv -> BN forward: the conv's compulsory bytes, then the BN
        # apply (read y, write z; the statistics come from the conv epilogue)
        ci, co, r = convs[name[:5]]
        flops = 2 * m * co * ci * r * r
        e = m * co
        byts = 2 * (m * ci + m * co + co * ci * r * r) + 4 * e + (2 * e if name.startswith("conv3") else 0)
        return flops, byts, "hbm"
    if name.startswith("conv"):
        ci, co, r = convs[name[:5]]
        flops = 2 * m * co * ci * r * r
        byts = 2 * (m * ci + m * co + co * ci * r * r)
        if name.endswith("dgrad_add"):
            byts += 2 * m * ci  # the shortcut gradient read in the epilogue
        bound = "mfma" if flops / byts >= PEAK_FP16_TFLOPS / PEAK_HBM_GBS * 1e3 else "hbm"
        return flops, byts, bound
    if name.startswith("bn"):
        co = {"bn1": w, "bn2": w, "bn3": c}[name[:3]]
        e = m * co
        if name.endswith("fwd"):
            byts = 6 * e + (2 * e if name == "bn3_fwd" else 0)  # reduce x; apply x (+r) -> y
        else:
            # reduce x, dy (+r); apply x, dy -> dx (+ shortcut gradient); the
            # ReLU mask the reduce recomputes from r is kept at one bit per
            # element, which is not counted
            byts = 10 * e + (4 * e if name == "bn3_bwd" else 0)
        return 0, byts, "hbm"
    if name == "sgd_conv":
        return 0, 10 * sum(co * ci * r * r for ci, co, r in s.conv_shapes), "hbm"
    if name == "sgd_bn":
        return 0, 10 * 2 * (w + w + c), "hbm"
    raise KeyError(name)


KERNELS_OF_CALL = {
    "conv_fwd": ["igemm_kernel"],
    "conv_dgrad": ["dgrad_filter_kernel", "igemm_kernel"],
    "conv_wgrad": ["wgrad_kernel", "wgrad_reduce_kernel"],
    "bn_fwd": ["bn_fwd_reduce_vec", "bn_fwd_finalize", "bn_fwd_apply_vec"],
    "bn_bwd": ["bn_bwd_reduce_vec", "bn_bwd_finalize", "bn_bwd_apply_vec"],
    "sgd": ["sgd_kernel"],
}


def profile_calls(block, reps, torch):
    """Average duration of every ABI call of the step, timed with HIP events
    recorded on the stream the calls are enqueued on."""
    stream = torch.cuda.current_stream()
    calls = block.calls()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in calls]
    tot = [0.0] * len(calls)
    for _ in range(reps):
        # hold the stream with a short device-side spin so the whole step is
        # queued before it starts: calls then run back to back, as in the graph
        torch.cuda._sleep(5_000_000)
        for (name, fn), (a, b) in zip(calls, evs):
            a.record(stream)
            fn()
            b.record(stream)
        torch.cuda.synchronize()
        for i, (a, b) in enumerate(evs):
            tot[i] += a.elapsed_time(b)
    return [(name, tot[i] / reps) for i, (name, _) in enumerate(calls)]


def traffic_for(kernel_src: str, call: str):
    """HBM bytes per call from the committed rocprofv3 counter summary, if it
    was taken on the current source of the kernel (else None)."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        data = json.load(open(path))
    except (OSError, ValueError):
        return None
    src = os.path.join(ROOT, "paper_1911_07384_amd", "csrc", kernel_src)
    try:
        digest = hashlib.sha256(open(src, "rb").read()).hexdigest()[:16]
    except OSError:
        return None
    ent = data.get(call)
    if not ent or ent.get("source_sha256_16") != digest:
        return None
    return ent.get("hbm_bytes")


def resnet50_leg(torch, steps: int, warmup: int = 3, batch: int = 128):
    """The whole ResNet-50 training step (forward, softmax cross-entropy,
    backward, FP16 SGD over every parameter) at batch 128 on 224x224 synthetic
    images, captured once in a HIP graph; images/s over `steps` replays, and
    the time per kind of call from one eager pass timed call by call."""
    from paper_1911_07384_amd.network import ResNet50
    net = ResNet50(n=batch, image=224, seed=0)
    net.load_batch(0)
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        net.step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        net.step()
    torch.cuda.synchronize()
    for _ in range(warmup):
        graph.replay()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(steps):
        graph.replay()
    b.record()
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / steps
    loss = float(net.buffers["loss"].float().mean().item())
    finite = bool(torch.isfinite(net.w_arena.float()).all().item())
    # per-kind time: each call between two events on the launch stream
    stream = torch.cuda.current_stream()
    calls = net.calls()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in calls]
    torch.cuda._sleep(200_000_000)  # covers the host enqueue of all 274 calls
    for (_, fn), (e0, e1) in zip(calls, evs):
        e0.record(stream)
        fn()
        e1.record(stream)
    torch.cuda.synchronize()
    kinds = {}
    for (name, _), (e0, e1) in zip(calls, evs):
        kind = name.split(":")[1]
        kinds[kind] = kinds.get(kind, 0.0) + e0.elapsed_time(e1)
    fl = net.step_flops()
    n_calls = len(net.program())
    del graph, net
    torch.cuda.empty_cache()
    return {"images_per_sec": round(batch / (ms * 1e-3), 1), "ms_per_step": round(ms, 4),
            "batch": batch, "image": 224, "steps": steps, "graph": True,
            "conv_tflop_per_step": round(fl / 1e12, 4),
            "conv_tflops_effective": round(fl / (ms * 1e-3) / 1e12, 2),
            "loss_after": round(loss, 4), "weights_finite": finite,
            "eager_ms_by_kind": {k: round(v, 3) for k, v in sorted(kinds.items(),
                                                                    key=lambda kv: -kv[1])},
            "abi_calls_per_step": n_calls,
            "note": "one HIP graph per step; each conv -> BN pair of the forward is one fused "
                    "call; weight gradients on a second stream; images ~N(0,1), uniform labels"}


def f16_arith_leg(torch, reps: int = 10):
    """Timing of the strict binary16-arithmetic mode next to the default:
    the SGD update over the ResNet-50 parameter count, and the three passes
    of the conv4_x 3x3 layer (256 -> 256, 14x14, batch 128) as chains of
    binary16 fmas (accum = 1) and with float32 accumulators."""
    import paper_1911_07384_amd as F
    gen = torch.Generator(device="cuda")
    gen.manual_seed(5)

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(1_000_000)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps

    out = {}
    n = 25_557_032
    w = (torch.randn(n, generator=gen, device="cuda") * 0.05).half()
    g = (torch.randn(n, generator=gen, device="cuda") * 1e-3).half()
    m = torch.zeros(n, dtype=torch.float16, device="cuda")
    for name, fn in (("sgd_f32_sequence", F.fp16_sgd_step), ("sgd_binary16", F.fp16_sgd_step_f16)):
        ms = timed(lambda: fn(w, g, m, lr=0.1, momentum=0.9, weight_decay=1e-4))
        out[name] = {"ms": round(ms, 5), "gb_per_s": round(10 * n / (ms * 1e-3) / 1e9, 1)}
    del w, g, m
    N, C, H, K = 128, 256, 14, 256
    x = torch.randn((N, H, H, C), generator=gen, device="cuda").half()
    wt = (torch.randn((K, 3, 3, C), generator=gen, device="cuda") * (2.0 / (9 * C)) ** 0.5).half()
    dy = (torch.randn((N, H, H, K), generator=gen, device="cuda") * 1e-3).half()
    y = torch.empty_like(dy)
    dx = torch.empty_like(x)
    dw = torch.empty_like(wt)
    flop = 2.0 * N * H * H * K * C * 9
    for accum in (0, 1):
        d = F.conv_desc(N, C, H, H, K, 3, 3, 1, 1, accum=accum)
        ws = F.workspace(max(F.fp16_conv_workspace_bytes(d, q) for q in (0, 1, 2)))
        row = {}
        for pname, fn in (("fwd", lambda: F.fp16_conv_fwd(d, x, wt, y, ws)),
                          ("dgrad", lambda: F.fp16_conv_dgrad(d, dy, wt, dx, ws)),
                          ("wgrad", lambda: F.fp16_conv_wgrad(d, x, dy, dw, ws))):
            ms = timed(fn)
            row[pname] = {"us": round(ms * 1e3, 2), "tflops": round(flop / (ms * 1e-3) / 1e12, 1)}
        out["conv4x_3x3_b128_" + ("binary16_acc" if accum else "float32_acc")] = row
    out["note"] = ("strict binary16 arithmetic (accum = 1 convolutions: every output a chain of "
                   "binary16 fmas, one rounding per term, on the vector ALUs; fp16_sgd_step_f16: "
                   "three binary16 fmas) next to the default float32 accumulators / float32 "
                   "sequence")
    return out


def cpu_baseline(shape, target_s):
    """The oracle's block step on a batch slice, on this host's cores."""
    import numpy as np
    import oracle
    from oracle.bottleneck import block_step, block_flops
    from paper_1911_07384_amd import synth

    def run(n):
        x = synth.normal_f16((n, shape.hw, shape.hw, shape.c), 1.0, 0, 1)
        W = [synth.normal_f16((co, r, r, ci), synth.he_std(ci * r * r), 0, 10 + i)
             for i, (ci, co, r) in enumerate(shape.conv_shapes)]
        g = [np.ones(co, np.float16) for _, co, _ in shape.conv_shapes]
        b = [np.zeros(co, np.float16) for _, co, _ in shape.conv_shapes]
        dout = synth.normal_f16((n, shape.hw, shape.hw, shape.c), 1e-3, 0, 2)
        t = time.perf_counter()
        block_step(x, W, g, b, dout, shape.post_scale, shape.eps)
        dt = time.perf_counter() - t
        return dt, 3 * block_flops(n, shape.hw, shape.conv_shapes)

    t1, _ = run(1)
    n = max(1, min(shape.n, int(round(target_s / max(t1, 1e-3)))))
    dt, fl = run(n)
    return {"value": fl / dt / 1e12, "unit": "TFLOP/s", "cores": oracle.num_threads(),
            "kind": "oracle",
            "sample": f"the full block step (3 conv fwd/dgrad/wgrad, 3 BN fwd/bwd, SGD) at batch "
                      f"{n} of {shape.n}, float64 direct loops, {dt:.2f} s; TFLOP/s counts the "
                      f"convolution FLOPs like the GPU value",
            "seconds": dt, "batch": n}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported (this build runs "
              f"on a single GPU and has no multi-GPU path)", file=sys.stderr)
        sys.exit(2)
    import torch
    import paper_1911_07384_amd as F
    from paper_1911_07384_amd.bottleneck import Bottleneck, BlockShape

    torch.cuda.set_device(0)
    if args.calibrate_copy:
        src = torch.empty(args.calibrate_copy << 20, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    shape = BlockShape(n=args.batch)
    block = Bottleneck(shape, seed=0)
    torch.cuda.synchronize()

    # capture the step once (every call enqueues on the capture stream)
    graph = None
    if not args.eager:
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            block.step()  # one eager step on the capture stream before capturing
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            block.step()
        torch.cuda.synchronize()
    step = graph.replay if graph is not None else block.step

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    start.record()
    for _ in range(args.steps):
        step()
    end.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = start.elapsed_time(end) / args.steps
    flops = 3 * shape.conv_flops()
    tflops = flops / (ms * 1e-3) / 1e12
    assert torch.isfinite(block.w_arena.float()).all(), "weights left the finite range"

    # per-call durations (eager, HIP events on the launch stream)
    per_call = profile_calls(block, max(5, args.steps // 2), torch)
    kernels = []
    for name, t in per_call:
        fl, by, bound = call_work(name, shape)
        k = {"call": name, "ms": round(t, 5), "bound": bound, "bytes": by, "flops": fl}
        if fl:
            k["tflops"] = round(fl / (t * 1e-3) / 1e12, 2)
            k["pct_mfma_peak"] = round(100 * fl / (t * 1e-3) / 1e12 / PEAK_FP16_TFLOPS, 2)
        k["gbs"] = round(by / (t * 1e-3) / 1e9, 1)
        k["pct_hbm_peak"] = round(100 * by / (t * 1e-3) / 1e9 / PEAK_HBM_GBS, 2)
        kernels.append(k)
    dom = max(kernels, key=lambda k: k["ms"])
    call = dom["call"]
    if call.startswith("conv"):
        src = "conv_wgrad.hip" if call.endswith("wgrad") else "conv_igemm.hip"
    else:
        src = "bn.hip" if call.startswith("bn") else "sgd.hip"
    if dom["bound"] == "mfma":
        roof = {"bound": "mfma", "achieved": dom["tflops"], "peak": PEAK_FP16_TFLOPS,
                "unit": "TFLOP/s", "frac": round(dom["tflops"] / PEAK_FP16_TFLOPS, 4)}
    else:
        roof = {"bound": "hbm", "achieved": dom["gbs"], "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(dom["gbs"] / PEAK_HBM_GBS, 4)}
    roof["traffic"] = traffic_for(src, dom["call"])
    roof["kernel"] = dom["call"]
    roof["ms"] = dom["ms"]

    out = {
        "metric": METRIC,
        "value": round(tflops, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16",
        "data": "synthetic",
        "config": {"workload": "resnet50_conv2x_bottleneck_train_step", "batch": shape.n,
                   "hw": shape.hw, "channels": [shape.c, shape.width, shape.width, shape.c],
                   "post_scale": shape.post_scale, "layout": "NHWC",
                   "graph": graph is not None},
        "images_per_sec": round(shape.n / (ms * 1e-3), 1),
        "pct_mfma_peak": round(100 * tflops / PEAK_FP16_TFLOPS, 3),
        "conv_gflop_per_step": round(flops / 1e9, 3),
        "wall_s_timed": round(wall, 4),
        "roofline": roof,
        "kernels": kernels,
    }
    if args.sweep or not args.no_sweep3x3:
        from paper_1911_07384_amd import resnet50
        layers = resnet50.LAYERS if args.sweep else [l for l in resnet50.LAYERS if l.r == 3]
        del graph
        torch.cuda.empty_cache()
        rows = resnet50.sweep(128, layers)
        summ = resnet50.summarize(rows, PEAK_FP16_TFLOPS)
        out["conv3x3_b128"] = {k: round(v, 4) for k, v in summ["3x3_16"].items()}
        out["conv3x3_b128"]["note"] = ("the 16 ResNet-50 3x3 convolutions at batch 128, fwd + dgrad "
                                       "+ wgrad, each pass timed separately with HIP events")
        if args.sweep:
            out["conv53_b128"] = {k: round(v, 4) for k, v in summ["all_53"].items()}
            out["sweep_layers"] = [{k: (round(v, 3) if isinstance(v, float) else v)
                                    for k, v in r.items()} for r in rows]
    if not args.no_resnet50:
        out["resnet50_train_b128"] = resnet50_leg(torch, args.resnet50_steps)
    if not args.no_f16_arith:
        out["f16_arith"] = f16_arith_leg(torch)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(shape, args.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
