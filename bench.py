"""Benchmark: one all-FP16 ResNet-50 training step at batch 128 on 224x224
images on one MI355X (the paper's network, Section 5.1, trained with every
tensor in binary16 and no master copy, Section 5.2).

A step is the whole hot path over one synthetic batch: the 7x7 stem and 52
other convolutions (forward, data and weight gradients), 53 fused BN(x0.25)
+ ReLU forwards and backwards (Section 4.2), the pools, the classifier and
its softmax cross-entropy, and the FP16 momentum-SGD update of all 25.6 M
parameters.  Inputs are resident in HBM before timing; the step is captured
once in a HIP graph and replayed; K replays are timed between HIP events.

Prints one JSON line.  The headline value is training images/s.  Beside it:
- `roofline`: the step's longest ABI call, its algorithmic bytes or FLOPs
  over its event-timed duration against the MI355X peak of its bound, and the
  HBM bytes it moved from the committed rocprofv3 counter summary;
- `cpu_baseline`: the CPU oracle's own training step on a few images;
- `conv3x3_b128` (the metric's convolution half: the 16 ResNet-50 3x3 layers,
  fwd + dgrad + wgrad, TFLOP/s and % of the FP16 matrix-core peak) with its
  own roofline and oracle baseline, `conv53_b128` (all 53 layers), and the
  3x3 layers in NCHW;
- `cold_hbm`: the HBM-bound kernels timed one call at a time after a 1 GiB
  read that evicts the 256 MB Infinity Cache, beside the same calls timed
  back to back (warm);
- `config1_latency`, `config5_stress`, `block_b32` (the conv2_x bottleneck
  at the paper's per-GPU batch of 32), `f16_arith` (strict binary16 mode).
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
RIDGE = PEAK_FP16_TFLOPS / PEAK_HBM_GBS * 1e3  # FLOP per byte
METRIC = "FP16 conv TFLOP/s (fwd+dgrad+wgrad) as % MFMA peak; ResNet-50 train images/sec"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--batch", type=int, default=128)
    ap.add_argument("--image", type=int, default=224)
    ap.add_argument("--eager", action="store_true", help="time the step without a HIP graph")
    ap.add_argument("--call-passes", type=int, default=3,
                    help="eager passes timing every ABI call of the step")
    ap.add_argument("--calls-only", action="store_true",
                    help="only two eager passes of the step, the second with a marker kernel "
                         "before every call (for counter runs)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=20.0,
                    help="target duration of the CPU oracle sample")
    ap.add_argument("--no-sweep", action="store_true", help="skip the batch-128 layer sweeps")
    ap.add_argument("--no-cold", action="store_true", help="skip the cold-cache HBM leg")
    ap.add_argument("--no-latency", action="store_true", help="skip the config-1 latency leg")
    ap.add_argument("--no-stress", action="store_true", help="skip the config-5 counts")
    ap.add_argument("--no-block", action="store_true", help="skip the conv2_x block at batch 32")
    ap.add_argument("--no-f16-arith", action="store_true",
                    help="skip the strict binary16-arithmetic timing leg")
    ap.add_argument("--sweep-only", action="store_true",
                    help="only the 16 3x3 layers at batch 128 (NHWC), for counter runs: every "
                         "timed batch of calls follows a spin kernel")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="first run three device-to-device copies of MIB MiB (a plain copy of "
                         "known size, the yardstick for the HBM byte counters)")
    return ap.parse_args()


# ---- algorithmic work of one ABI call ------------------------------------------------

def _touched(size, out, k, stride, pad):
    """Input rows (or columns) that some output position reads."""
    return len({o * stride - pad + r for o in range(out) for r in range(k)} & set(range(size)))


def conv_work(d, pass_):
    """(flops, compulsory bytes) of one convolution pass: 2 N P Q K C R S
    FLOPs; every input element a tap touches, the filter and the output, once."""
    p = (d.h + 2 * d.pad_h - d.r) // d.stride_h + 1
    q = (d.w + 2 * d.pad_w - d.s) // d.stride_w + 1
    flops = 2 * d.n * p * q * d.k * d.c * d.r * d.s
    x = d.n * d.c * _touched(d.h, p, d.r, d.stride_h, d.pad_h) * _touched(d.w, q, d.s, d.stride_w,
                                                                        d.pad_w)
    if pass_ == "dgrad":  # dx is written whole
        x = d.n * d.c * d.h * d.w
    y = d.n * d.k * p * q
    w = d.k * d.c * d.r * d.s
    return flops, 2 * (x + y + w)


def bn_elems(d):
    return d.n * d.c * d.h * d.w


def op_work(op, net):
    """(flops, bytes, bound) of one call of the network's program (the
    per-unit figures of the design: BN forward 6 B/element + 2 with the
    shortcut, 4 + 2 when its statistics come from the convolution, + 1/8 for
    a kept ReLU mask; BN backward 10 B/element + 4 with the shortcut
    recomputing the mask, + 2 (the shortcut gradient) + 1/4 (the mask, read
    twice) with a kept mask; a data gradient's addend 2 B/element + 1/8 under
    a mask; the BN fused into the max pool 4 B per input element + 3 per
    pooled element; SGD 10 B/element)."""
    a, k = op.a, op.kind
    if k in ("conv_fwd", "conv_dgrad", "conv_dgrad_add", "conv_wgrad"):
        fl, by = conv_work(a["desc"], {"conv_fwd": "fwd", "conv_wgrad": "wgrad"}.get(k, "dgrad"))
        if k == "conv_dgrad_add":
            d, st = a["desc"], a.get("astride", 1)
            ex = d.n * d.c * (-(-d.h // st)) * (-(-d.w // st))  # the addend's elements
            by += 2 * ex + (ex // 8 if a.get("amask") else 0)
        return fl, by, "mfma" if fl / by >= RIDGE else "hbm"
    if k == "conv_bn_fwd":
        fl, by = conv_work(a["desc"], "fwd")
        e = bn_elems(a["bn"])
        by += 4 * e + (2 * e if a["res"] is not None else 0) + (e // 8 if a["mask"] else 0)
        return fl, by, "mfma" if fl / by >= RIDGE else "hbm"
    if k == "bn_fwd":
        e = bn_elems(a["desc"])
        return 0, 6 * e + (2 * e if a["res"] is not None else 0) + (e // 8 if a["mask"] else 0), "hbm"
    if k == "bn_bwd":
        e = bn_elems(a["desc"])
        if a["mask"]:
            return 0, 10 * e + (2 * e if a["dres"] is not None else 0) + e // 4, "hbm"
        return 0, 10 * e + (4 * e if a["dres"] is not None else 0), "hbm"
    if k == "dgrad_filter":
        d = a["desc"]
        return 0, 4 * d.k * d.c * d.r * d.s, "hbm"
    if k == "dgrad_filters":
        return 0, sum(4 * d.k * d.c * d.r * d.s for d, _, _ in a["items"]), "hbm"
    if k == "maxpool_fwd":
        d = a["desc"]
        p, q = (d.h + 2 * d.pad_h - d.r) // d.stride_h + 1, (d.w + 2 * d.pad_w - d.s) // d.stride_w + 1
        return 0, 2 * d.n * d.c * d.h * d.w + 3 * d.n * d.c * p * q, "hbm"
    if k == "bn_maxpool_fwd":
        d, pd = a["desc"], a["pool"]
        e = bn_elems(d)
        p, q = (pd.h + 2 * pd.pad_h - pd.r) // pd.stride_h + 1, (pd.w + 2 * pd.pad_w - pd.s) // pd.stride_w + 1
        return 0, 4 * e + 3 * pd.n * pd.c * p * q, "hbm"
    if k == "maxpool_bwd":
        d = a["desc"]
        p, q = (d.h + 2 * d.pad_h - d.r) // d.stride_h + 1, (d.w + 2 * d.pad_w - d.s) // d.stride_w + 1
        return 0, 2 * d.n * d.c * d.h * d.w + 3 * d.n * d.c * p * q, "hbm"
    if k in ("avgpool_fwd", "avgpool_bwd"):
        d = a["desc"]
        return 0, 2 * d.n * d.c * d.h * d.w + 2 * d.n * d.c, "hbm"
    if k == "softmax_ce":
        return 0, 4 * a["n"] * a["k"] + 4 * a["k"] + 8 * a["n"], "hbm"
    if k == "sgd":
        return 0, 10 * a["w"].numel(), "hbm"
    raise KeyError(k)


def roofline_of(flops, byts, ms, bound):
    if bound == "mfma":
        ach = flops / (ms * 1e-3) / 1e12
        return {"bound": "mfma", "achieved": round(ach, 2), "peak": PEAK_FP16_TFLOPS,
                "unit": "TFLOP/s", "frac": round(ach / PEAK_FP16_TFLOPS, 4)}
    ach = byts / (ms * 1e-3) / 1e9
    return {"bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
            "frac": round(ach / PEAK_HBM_GBS, 4)}


def traffic_for(call: str):
    """HBM bytes of one call from the committed rocprofv3 counter summary, if
    its counters were taken on the current sources of its kernels."""
    try:
        ent = json.load(open(os.path.join(ROOT, "profiles", "traffic.json"))).get(call)
    except (OSError, ValueError):
        return None
    if not ent:
        return None
    for src, digest in ent.get("sources", {}).items():
        path = os.path.join(ROOT, "paper_1911_07384_amd", "csrc", src)
        try:
            if hashlib.sha256(open(path, "rb").read()).hexdigest()[:16] != digest:
                return None
        except OSError:
            return None
    return ent.get("hbm_bytes")


def time_calls(calls, passes, torch):
    """Average duration of each (name, thunk), timed between two HIP events
    on the launch stream; every pass is queued behind a device-side spin so
    the calls run back to back."""
    stream = torch.cuda.current_stream()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in calls]
    tot = [0.0] * len(calls)
    for _ in range(passes):
        torch.cuda._sleep(300_000_000)  # covers the host enqueue of every call
        for (_, fn), (a, b) in zip(calls, evs):
            a.record(stream)
            fn()
            b.record(stream)
        torch.cuda.synchronize()
        for i, (a, b) in enumerate(evs):
            tot[i] += a.elapsed_time(b)
    return [t / passes for t in tot]


# ---- the headline: the ResNet-50 training step at batch 128 -------------------------

def resnet50_step(args, torch):
    from paper_1911_07384_amd.network import ResNet50
    net = ResNet50(n=args.batch, image=args.image, seed=0)
    net.load_batch(0)
    torch.cuda.synchronize()
    out = {}
    if not args.calls_only:
        step = net.step
        graph = None
        if not args.eager:
            side = torch.cuda.Stream()
            side.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(side):
                net.step()  # one eager step on the capture stream before capturing
            torch.cuda.current_stream().wait_stream(side)
            torch.cuda.synchronize()
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph):
                net.step()
            torch.cuda.synchronize()
            step = graph.replay
        for _ in range(args.warmup):
            step()
        torch.cuda.synchronize()
        start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0 = time.perf_counter()
        start.record()
        for _ in range(args.steps):
            step()
        end.record()
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        ms = start.elapsed_time(end) / args.steps
        fl = net.step_flops()
        out = {"ms": ms, "wall_s_timed": wall, "graph": graph is not None,
               "images_per_sec": args.batch / (ms * 1e-3),
               "conv_tflop_per_step": fl / 1e12, "conv_tflops_effective": fl / (ms * 1e-3) / 1e12,
               "loss_after": float(net.buffers["loss"].float().mean().item()),
               "weights_finite": bool(torch.isfinite(net.w_arena.float()).all().item()),
               "abi_calls_per_step": len(net.program())}
        del graph
    # every ABI call of the step, eager, between HIP events on its stream
    ops = net.program()
    times = time_calls(net.calls(), args.call_passes, torch)
    rows = []
    kinds = {}
    for op, t in zip(ops, times):
        fl, by, bound = op_work(op, net)
        rows.append({"call": f"{op.name}:{op.kind}", "ms": t, "flops": fl, "bytes": by,
                     "bound": bound})
        kinds[op.kind] = kinds.get(op.kind, 0.0) + t
    out["calls"] = rows
    out["ms_by_kind"] = {k: round(v, 3) for k, v in sorted(kinds.items(), key=lambda kv: -kv[1])}
    out["eager_calls_ms"] = sum(times)
    del net
    torch.cuda.empty_cache()
    return out


def calls_only(args, torch):
    """For counter runs: one eager step, then one more with a one-thread spin
    kernel launched before every ABI call, so that each call's dispatches can
    be told apart in a dispatch-ordered counter trace; prints the call names
    in order."""
    from paper_1911_07384_amd.network import ResNet50
    net = ResNet50(n=args.batch, image=args.image, seed=0)
    net.load_batch(0)
    calls = net.calls()
    for _, fn in calls:
        fn()
    torch.cuda.synchronize()
    for _, fn in calls:
        torch.cuda._sleep(100)
        fn()
    torch.cuda.synchronize()
    print(json.dumps({"calls": [n for n, _ in calls]}), flush=True)


# ---- config 3: the per-layer sweep at batch 128 -----------------------------------

def conv_sweep_leg(torch, sweep_all: bool, nchw: bool = True):
    from paper_1911_07384_amd import resnet50
    layers = resnet50.LAYERS if sweep_all else [l for l in resnet50.LAYERS if l.r == 3]
    rows = resnet50.sweep(128, layers)
    summ = resnet50.summarize(rows, PEAK_FP16_TFLOPS)
    leg = {k: round(v, 4) for k, v in summ["3x3_16"].items()}
    # the 3x3 (layer, pass) with the most time in the network: its roofline
    best = None
    for r in rows:
        if r["r"] != 3:
            continue
        for p in ("fwd", "dgrad", "wgrad"):
            t = r[p + "_us"] * r["mult"]
            if best is None or t > best[0]:
                best = (t, r, p)
    _, r, p = best
    L = next(l for l in layers if l.name == r["layer"])
    import paper_1911_07384_amd as F
    d = F.conv_desc(128, L.c, L.hw, L.hw, L.k, L.r, L.r, L.stride, L.pad)
    fl, by = conv_work(d, p)
    bound = "mfma" if fl / by >= RIDGE else "hbm"
    roof = roofline_of(fl, by, r[p + "_us"] * 1e-3, bound)
    roof.update({"traffic": None, "kernel": f"{L.name} {p}", "us": round(r[p + "_us"], 2),
                 "flops": fl, "bytes": by})
    leg["roofline"] = roof
    leg["layers"] = [{k: (round(v, 3) if isinstance(v, float) else v) for k, v in row.items()}
                     for row in rows]
    leg["note"] = ("the 16 ResNet-50 3x3 convolutions at batch 128 (NHWC), fwd + dgrad + wgrad, "
                   "each layer pass timed over 10 back-to-back calls with HIP events, weighted by "
                   "its multiplicity in the network")
    out = {"conv3x3_b128": leg}
    if sweep_all:
        out["conv53_b128"] = {k: round(v, 4) for k, v in summ["all_53"].items()}
    torch.cuda.empty_cache()
    if not nchw:
        return out, rows
    nchw = resnet50.sweep(128, [l for l in resnet50.LAYERS if l.r == 3], layout="NCHW")
    s2 = resnet50.summarize(nchw, PEAK_FP16_TFLOPS)["3x3_16"]
    out["conv3x3_b128_nchw"] = {k: round(v, 4) for k, v in s2.items()}
    out["conv3x3_b128_nchw"]["note"] = ("the same layers with NCHW activations and KCRS filters, "
                                        "converted to the native NHWC through the workspace "
                                        "inside each call")
    torch.cuda.empty_cache()
    return out, rows


def conv3x3_cpu_baseline(target_s):
    """The oracle's full convolutions (float64 direct loops) over the 16
    ResNet-50 3x3 layers, all three passes, on a slice of the batch, in
    GFLOP/s: each distinct layer runs once and counts with its
    multiplicity in the network."""
    import oracle
    from paper_1911_07384_amd import resnet50, synth
    layers = [l for l in resnet50.LAYERS if l.r == 3]

    def run(n):
        flops, dt = 0, 0.0
        for li, L in enumerate(layers):
            p = L.out_hw
            shp = oracle.conv_shape(n, L.c, L.hw, L.hw, L.k, 3, 3, L.stride, 1)
            x = synth.normal_f16((n, L.hw, L.hw, L.c), 1.0, 90 + li, 1)
            w = synth.normal_f16((L.k, 3, 3, L.c), synth.he_std(9 * L.c), 90 + li, 2)
            dy = synth.normal_f16((n, p, p, L.k), 1e-3, 90 + li, 3)
            t = time.perf_counter()
            oracle.conv_fwd(shp, x, w)
            oracle.conv_dgrad(shp, dy, w)
            oracle.conv_wgrad(shp, x, dy)
            dt += (time.perf_counter() - t) * L.mult
            flops += 3 * L.flops(n) * L.mult
        return flops, dt

    fl, dt = run(1)
    n = 1
    if dt < 0.5 * target_s:
        n = int(max(2, min(16, round(target_s / dt))))
        fl, dt = run(n)
    return {"value": round(fl / dt / 1e9, 3), "unit": "GFLOP/s", "cores": oracle.num_threads(),
            "kind": "oracle",
            "sample": f"the 16 3x3 layers (each distinct layer once, counted with its "
                      f"multiplicity), fwd + dgrad + wgrad over every output, at batch {n} of 128, "
                      f"float64 direct loops, {dt:.1f} s",
            "seconds": round(dt, 2), "batch": n}


# ---- HBM-bound kernels with the Infinity Cache cold -------------------------------------

def cold_hbm_leg(torch, reps=5):
    """Each call timed alone after a 1 GiB read (which leaves none of the
    call's inputs in the 256 MB Infinity Cache), median of `reps`; and the
    same call repeated back to back (inputs partly cache-resident: warm)."""
    import paper_1911_07384_amd as F
    from paper_1911_07384_amd import synth
    flush = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    gen = torch.Generator(device="cuda")
    gen.manual_seed(11)

    flush.fill_(1)
    words = flush.view(torch.int64)

    def timed_cold(fn):
        out = []
        for _ in range(reps):
            # read (not write) 1 GiB: the Infinity Cache then holds only clean
            # lines of this buffer, so the timed call neither hits on its own
            # inputs nor pays for writing back someone else's dirty lines
            words.sum()
            torch.cuda.synchronize()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            fn()
            b.record()
            torch.cuda.synchronize()
            out.append(a.elapsed_time(b))
        return sorted(out)[len(out) // 2]

    def timed_warm(fn, n=10):
        fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(1_000_000)
        a.record()
        for _ in range(n):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / n

    res = {}
    # what plain streams reach on this chip with the cache cold: a 1 GiB read
    # (sum), write (fill) and copy, the ceilings the fractions below sit under
    buf = torch.empty(1 << 27, dtype=torch.int64, device="cuda")
    dst = torch.empty(1 << 26, dtype=torch.int64, device="cuda")
    ref = {}
    for name, fn, byts in (("read_1GiB", lambda: buf.sum(), 1 << 30),
                           ("write_1GiB", lambda: buf.fill_(3), 1 << 30),
                           ("copy_512MiB", lambda: dst.copy_(buf[: 1 << 26]), 1 << 30)):
        c = timed_cold(fn)
        ref[name] = {"cold_us": round(c * 1e3, 1), "cold_gbs": round(byts / c / 1e6, 1),
                     "cold_frac": round(byts / c / 1e6 / PEAK_HBM_GBS, 4)}
    res["stream_reference"] = ref
    del buf, dst

    def record(name, fn, byts):
        c, w = timed_cold(fn), timed_warm(fn)
        res[name] = {"bytes": byts, "cold_us": round(c * 1e3, 2), "cold_gbs": round(byts / c / 1e6, 1),
                     "cold_frac": round(byts / c / 1e6 / PEAK_HBM_GBS, 4),
                     "warm_us": round(w * 1e3, 2), "warm_gbs": round(byts / w / 1e6, 1)}

    # SGD over the 25,557,032 ResNet-50 parameters: 10 B/element
    n = 25_557_032
    w = (torch.randn(n, generator=gen, device="cuda") * 0.05).half()
    g = (torch.randn(n, generator=gen, device="cuda") * 1e-3).half()
    m = torch.zeros(n, dtype=torch.float16, device="cuda")
    record("sgd_resnet50_params", lambda: F.fp16_sgd_step(w, g, m, lr=0.1, momentum=0.9,
                                                           weight_decay=1e-4), 10 * n)
    del w, g, m
    # the block-last BN of conv2_x at batch 128: [128, 56, 56, 256] with the shortcut
    N, H, C = 128, 56, 256
    e = N * H * H * C
    x = torch.randn((N, H, H, C), generator=gen, device="cuda").half()
    r = torch.randn((N, H, H, C), generator=gen, device="cuda").half()
    dy = (torch.randn((N, H, H, C), generator=gen, device="cuda") * 1e-3).half()
    y = torch.empty_like(x)
    dx = torch.empty_like(x)
    dr = torch.empty_like(x)
    gamma = torch.ones(C, dtype=torch.float16, device="cuda")
    beta = torch.zeros(C, dtype=torch.float16, device="cuda")
    dg, db = torch.empty_like(gamma), torch.empty_like(beta)
    st = torch.empty(2 * C, dtype=torch.float32, device="cuda")
    d = F.bn_desc(N, C, H, H, post_scale=0.25)
    ws = F.workspace(F.fp16_bn_workspace_bytes(d))
    record("bn_fwd_conv2x_b128", lambda: F.fp16_bn_relu(d, x, gamma, beta, r, y, st, ws), 8 * e)
    record("bn_bwd_conv2x_b128", lambda: F.fp16_bn_relu_bwd(d, x, None, dy, gamma, beta, r, st, dx,
                                                            dg, db, dr, ws), 14 * e)
    # the same pair with the ReLU mask kept by the forward (the network's form)
    mk = torch.empty(F.fp16_bn_mask_bytes(d), dtype=torch.uint8, device="cuda")
    record("bn_fwd_mask_conv2x_b128",
           lambda: F.fp16_bn_relu_m(d, x, gamma, beta, r, y, st, mk, ws), 8 * e + e // 8)
    record("bn_bwd_mask_conv2x_b128",
           lambda: F.fp16_bn_relu_bwd_m(d, x, mk, dy, gamma, beta, st, dx, dg, db, dr, ws),
           12 * e + e // 4)
    del x, r, dy, y, dx, dr, ws, mk
    # the 1x1 64 -> 256 convolution of conv2_x at batch 128 (HBM-bound, AI 51)
    xc = torch.randn((N, H, H, 64), generator=gen, device="cuda").half()
    wc = (torch.randn((256, 1, 1, 64), generator=gen, device="cuda") * 0.17).half()
    yc = torch.empty((N, H, H, 256), dtype=torch.float16, device="cuda")
    dc = F.conv_desc(N, 64, H, H, 256, 1, 1)
    wsc = F.workspace(F.fp16_conv_workspace_bytes(dc, 0))
    record("conv1x1_64_256_fwd_b128", lambda: F.fp16_conv_fwd(dc, xc, wc, yc, wsc),
           conv_work(dc, "fwd")[1])
    del xc, wc, yc, flush
    torch.cuda.empty_cache()
    res["note"] = ("cold: one call after reading a 1 GiB buffer (evicts the 256 MB Infinity Cache), "
                   "median of 5; warm: 10 back-to-back calls; bytes are the algorithmic bytes "
                   "(SGD 10 B/element, BN forward with statistics and shortcut 8 (+1/8 keeping the "
                   "ReLU mask), BN backward with shortcut 14 (12.25 with the kept mask), the "
                   "convolution's compulsory bytes); stream_reference: torch's own sum, fill and "
                   "copy under the same cold protocol")
    return res


# ---- config 1: latency of the small 3x3 layer ----------------------------------------

def latency_leg(torch, reps=200):
    import numpy as np
    import paper_1911_07384_amd as F
    from paper_1911_07384_amd import synth
    N, C, H = 2, 64, 56
    d = F.conv_desc(N, C, H, H, C, 3, 3, 1, 1)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to("cuda")
    x = dev(synth.normal_f16((N, H, H, C), 1.0, 0, 1))
    w = dev(synth.normal_f16((C, 3, 3, C), synth.he_std(9 * C), 0, 2))
    dy = dev(synth.normal_f16((N, H, H, C), 1e-2, 0, 3))
    y, dx, dw = torch.empty_like(dy), torch.empty_like(x), torch.empty_like(w)
    m = torch.zeros_like(w)
    ws = F.workspace(max(F.fp16_conv_workspace_bytes(d, q) for q in (0, 1, 2)))
    calls = {"fwd": lambda: F.fp16_conv_fwd(d, x, w, y, ws),
             "dgrad": lambda: F.fp16_conv_dgrad(d, dy, w, dx, ws),
             "wgrad": lambda: F.fp16_conv_wgrad(d, x, dy, dw, ws),
             "sgd": lambda: F.fp16_sgd_step(w, dw, m, lr=0.1, momentum=0.9, weight_decay=1e-4)}
    out = {}
    for name, fn in calls.items():
        fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(5_000_000)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        torch.cuda.synchronize()
        out[name + "_us_eager"] = round(a.elapsed_time(b) / reps * 1e3, 2)
        # host-to-completion latency of one call on an idle device
        t = []
        for _ in range(20):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            fn()
            torch.cuda.synchronize()
            t.append(time.perf_counter() - t0)
        out[name + "_us_host_sync"] = round(sorted(t)[10] * 1e6, 1)

    def step():
        for fn in calls.values():
            fn()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    g.replay()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        g.replay()
    b.record()
    torch.cuda.synchronize()
    out["step_us_graph"] = round(a.elapsed_time(b) / reps * 1e3, 2)
    out["step_us_eager"] = round(sum(out[k + "_us_eager"] for k in calls), 2)
    out["note"] = ("3x3 conv, N=2, C=K=64, 56x56 (0.462 GFLOP per pass) and the SGD update of its "
                   "36,864 weights: device time per call over 200 back-to-back calls, host time of "
                   "one call to completion on an idle device, and the four calls as one HIP graph")
    del g
    return out


# ---- config 5: the subnormal stress counts ---------------------------------------------

def stress_leg(torch):
    """conv4_x 3x3 256 -> 256 at 14x14, batch 128, |dy| log-uniform in
    [2^-24, 2^-10]: counts of subnormal and zero weight-gradient outputs, and
    of weights left unchanged by two SGD steps (lr 2^-14, momentum 0.9, wd
    1e-4); also with x scaled by 2^-10, where dW itself is mostly subnormal."""
    import numpy as np
    import paper_1911_07384_amd as F
    from paper_1911_07384_amd import synth
    N, C, H = 128, 256, 14
    d = F.conv_desc(N, C, H, H, C, 3, 3, 1, 1)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to("cuda")
    x16 = synth.normal_f16((N, H, H, C), 1.0, 5, 1)
    w = dev(synth.normal_f16((C, 3, 3, C), synth.he_std(9 * C), 5, 2))
    dy16 = synth.loguniform_f16((N, H, H, C), -24, -10, 5, 3)
    dy = dev(dy16)
    ws = F.workspace(F.fp16_conv_workspace_bytes(d, 2))
    out = {"dy_subnormal_frac": round(float(np.mean((dy16 != 0) & (np.abs(dy16.astype(np.float32))
                                                                    < 2.0 ** -14))), 4)}

    def counts(t):
        v = t.float()
        sub = ((v != 0) & (v.abs() < 2.0 ** -14)).sum().item()
        return int(sub), int((v == 0).sum().item())

    for tag, scale in (("x", 1.0), ("x_2^-10", 2.0 ** -10)):
        x = dev((x16.astype(np.float32) * scale).astype(np.float16))
        dw = torch.empty_like(w)
        F.fp16_conv_wgrad(d, x, dy, dw, ws)
        wt = w.clone()
        m = torch.zeros_like(w)
        row = {}
        sub, zero = counts(dw)
        row["dw_subnormal"], row["dw_zero"] = sub, zero
        for stepno in (1, 2):
            before = wt.clone()
            F.fp16_sgd_step(wt, dw, m, lr=2.0 ** -14, momentum=0.9, weight_decay=1e-4)
            torch.cuda.synchronize()
            row[f"step{stepno}_w_unchanged"] = int((wt.view(torch.int16) == before.view(torch.int16))
                                                   .sum().item())
            row[f"step{stepno}_m_subnormal"], row[f"step{stepno}_m_zero"] = counts(m)
        row["n_weights"] = wt.numel()
        out[tag] = row
    out["note"] = ("counts over the 589,824 weights; 'unchanged' = the binary16 weight is bit for "
                   "bit what it was before the update (stagnation, Sections 2 and 4.2)")
    return out


# ---- config 2: the conv2_x bottleneck at the paper's per-GPU batch ---------------------

def block_leg(torch, steps=50, warmup=10):
    from paper_1911_07384_amd.bottleneck import Bottleneck, BlockShape
    shape = BlockShape(n=32)
    block = Bottleneck(shape, seed=0)
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        block.step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        block.step()
    for _ in range(warmup):
        g.replay()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(steps):
        g.replay()
    b.record()
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / steps
    fl = 3 * shape.conv_flops()
    calls = block.calls()
    times = time_calls(calls, 5, torch)
    del g
    return {"ms_per_step": round(ms, 5), "conv_tflops_effective": round(fl / (ms * 1e-3) / 1e12, 2),
            "block_images_per_sec": round(shape.n / (ms * 1e-3), 1),
            "calls_ms": {n: round(t, 5) for (n, _), t in zip(calls, times)},
            "note": "ResNet-50 conv2_x bottleneck (256->64->64->256, 56x56, x0.25, identity "
                    "shortcut) at batch 32, forward + backward + SGD, one HIP graph per step; "
                    "block_images_per_sec is the rate of this one block, not of the network"}


# ---- strict binary16 arithmetic ------------------------------------------------------------

def f16_arith_leg(torch, reps=3):
    """The strict binary16 mode next to the default: the SGD update over the
    ResNet-50 parameter count, and the three passes of the conv4_x 3x3 layer
    (256 -> 256, 14x14, batch 128) as chains of binary16 fmas (accum = 1)
    and with float32 accumulators."""
    import paper_1911_07384_amd as F
    gen = torch.Generator(device="cuda")
    gen.manual_seed(5)

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
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
    y, dx, dw = torch.empty_like(dy), torch.empty_like(x), torch.empty_like(wt)
    flop = 2.0 * N * H * H * K * C * 9
    for accum in (0, 1):
        d = F.conv_desc(N, C, H, H, K, 3, 3, 1, 1, accum=accum)
        ws = F.workspace(max(F.fp16_conv_workspace_bytes(d, q) for q in (0, 1, 2)))
        row = {}
        for pname, fn in (("fwd", lambda: F.fp16_conv_fwd(d, x, wt, y, ws)),
                          ("dgrad", lambda: F.fp16_conv_dgrad(d, dy, wt, dx, ws)),
                          ("wgrad", lambda: F.fp16_conv_wgrad(d, x, dy, dw, ws))):
            ms = timed(fn)
            row[pname] = {"us": round(ms * 1e3, 2), "tflops": round(flop / (ms * 1e-3) / 1e12, 2)}
        out["conv4x_3x3_b128_" + ("binary16_chains" if accum else "float32_acc")] = row
    out["note"] = ("strict binary16 arithmetic (accum = 1 convolutions: every output a chain of "
                   "binary16 fmas, one rounding per term, on the vector ALUs; fp16_sgd_step_f16: "
                   "three binary16 fmas) next to the default float32 accumulators / float32 "
                   "sequence")
    return out


# ---- the oracle's rate on the headline workload -------------------------------------------

def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(target_s, image=224):
    """The oracle's own ResNet-50 training step (forward, loss, backward,
    SGD; oracle/resnet50.py) on a few images, in images/s, on this host's
    cores; and the config-1 3x3 layer's three passes on one core."""
    import numpy as np
    import oracle
    from oracle import resnet50 as onet
    from paper_1911_07384_amd import synth
    P = onet.init_params(seed=0)

    def run(n):
        img = synth.normal_f16((n, image, image, 3), 1.0, 0, 1)
        lab = synth.labels(n, 1000, 0, 2)
        t = time.perf_counter()
        onet.train_step(img, lab, P)
        return time.perf_counter() - t

    t1 = run(1)
    n, dt = 1, t1
    if t1 < 0.5 * target_s:
        n = int(max(2, min(8, round(target_s / t1))))
        dt = run(n)
    threads = oracle.num_threads()
    # config 1 on one core: x [2,56,56,64], 3x3 64 -> 64, three passes
    shp = oracle.conv_shape(2, 64, 56, 56, 64, 3, 3, 1, 1)
    x = synth.normal_f16((2, 56, 56, 64), 1.0, 0, 1)
    w = synth.normal_f16((64, 3, 3, 64), synth.he_std(576), 0, 2)
    dy = synth.normal_f16((2, 56, 56, 64), 1e-2, 0, 3)
    oracle.set_num_threads(1)
    t = time.perf_counter()
    oracle.conv_fwd(shp, x, w)
    oracle.conv_dgrad(shp, dy, w)
    oracle.conv_wgrad(shp, x, dy)
    c1 = time.perf_counter() - t
    oracle.set_num_threads(threads)
    return {"value": round(n / dt, 4), "unit": "images/s", "cores": threads, "kind": "oracle",
            "sample": f"the oracle's whole training step (53 convolutions x 3 passes, 53 BN "
                      f"forward/backward, pools, classifier, softmax cross-entropy, SGD of 25.6 M "
                      f"binary16 parameters) at batch {n} of {image}x{image} images, float64 "
                      f"direct loops, {dt:.1f} s",
            "seconds": round(dt, 2), "batch": n, "cpu_model": cpu_model(),
            "nproc": os.cpu_count(),
            "config1_one_core_s": round(c1, 3),
            "config1_one_core_gflops": round(3 * 0.4624 / c1, 3)}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported: this build runs "
              f"the per-GPU hot path on a single GPU and has no multi-GPU path", file=sys.stderr)
        sys.exit(2)
    import torch
    torch.cuda.set_device(0)
    if args.calibrate_copy:
        src = torch.empty(args.calibrate_copy << 20, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    if args.sweep_only:
        legs, _ = conv_sweep_leg(torch, False, nchw=False)
        print(json.dumps(legs), flush=True)
        return
    if args.calls_only:
        calls_only(args, torch)
        return
    step = resnet50_step(args, torch)
    ms = step["ms"]
    dom = max(step["calls"], key=lambda c: c["ms"])
    roof = roofline_of(dom["flops"], dom["bytes"], dom["ms"], dom["bound"])
    roof.update({"traffic": traffic_for(dom["call"]), "kernel": dom["call"],
                 "ms": round(dom["ms"], 5), "bytes": dom["bytes"], "flops": dom["flops"]})
    out = {
        "metric": METRIC,
        "value": round(step["images_per_sec"], 1),
        "unit": "images/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16",
        "data": "synthetic",
        "config": {"workload": "resnet50_train_step", "batch": args.batch, "image": args.image,
                   "classes": 1000, "post_scale": 0.25, "layout": "NHWC",
                   "graph": step["graph"]},
        "images_per_sec": round(step["images_per_sec"], 1),
        "conv_tflop_per_step": round(step["conv_tflop_per_step"], 4),
        "conv_tflops_effective": round(step["conv_tflops_effective"], 2),
        "loss_after": round(step["loss_after"], 4),
        "weights_finite": step["weights_finite"],
        "wall_s_timed": round(step["wall_s_timed"], 4),
        "roofline": roof,
        "step_ms_by_kind": step["ms_by_kind"],
        "top_calls": [{"call": c["call"], "ms": round(c["ms"], 4), "bound": c["bound"],
                       **roofline_of(c["flops"], c["bytes"], c["ms"], c["bound"])}
                      for c in sorted(step["calls"], key=lambda c: -c["ms"])[:12]],
        "note": "one HIP graph per step; each conv -> BN pair of the forward is one fused call; "
                "weight gradients on a second stream; images ~N(0,1), uniform labels over 1000 "
                "classes stand in for ImageNet; roofline = the step's longest ABI call, timed "
                "eagerly between HIP events",
    }
    if not args.no_sweep:
        legs, _ = conv_sweep_leg(torch, True)
        out.update(legs)
    if not args.no_cold:
        out["cold_hbm"] = cold_hbm_leg(torch)
    if not args.no_latency:
        out["config1_latency"] = latency_leg(torch)
    if not args.no_stress:
        out["config5_stress"] = stress_leg(torch)
    if not args.no_block:
        out["block_b32"] = block_leg(torch)
    if not args.no_f16_arith:
        out["f16_arith"] = f16_arith_leg(torch)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(args.cpu_seconds, args.image)
        if "conv3x3_b128" in out:
            out["conv3x3_b128"]["cpu_baseline"] = conv3x3_cpu_baseline(8.0)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
