"""Conv hot-path benchmark on one MI355X.

A step is one pass of a network's whole conv stack, layer by layer, over one
batch of seeded synthetic input already resident in HBM: every layer's input,
weights and bias are drawn once (their own seeds, the configuration's value
distributions) and every layer writes its own output buffer, so the timed
region holds only conv kernels.  The default workload is the ResNet-50 v1
conv stack at batch 1 in fp32 (53 convs); --config picks another.

The passes run through the library's stack executor: W eager passes, then
the timed region, one HIP graph holding exactly K passes (after one untimed
replay of it), then K eager passes whose kernel launches carry start/end
events that the runtime stamps with each kernel's execution interval.

Prints one JSON line with the conv TFLOP/s of the step (from the timed
region), ms per image, the roofline of the dominant kernel (the kernel with
the largest summed execution time; its traffic comes from the committed
counter summaries profiles/traffic_<workload>.txt when they match the kernel source)
and the CPU oracle timed on a bounded sample of the same stack.  The default
run (ResNet-50 at batch 1) also carries, under "b64", the same record for
ResNet-50 at batch 64 with bf16 inputs (the metric's other half), under
"b64_chained" that network as one pass with bf16 channel-last activations,
under "b1_chained" the batch-1 network as one pass (fp32),
under "single_call" the single-layer configuration timed through each entry
point, and under "vision" the detection post-processing operators (box_nms,
segmented argsort, prefix sum) on their own workloads.
"""
from __future__ import annotations

import argparse
import json
import os
import subprocess
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_FP32_MFMA_TFLOPS = 157.3
PEAK_BF16_MFMA_TFLOPS = 2516.6
PEAK_HBM_GBS = 8000.0


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per launch of `kernel` (read + written, calibrated against a
    plain copy) in `workload`, from the committed counter summary
    profiles/traffic_<workload>.txt, or None when it has no line for this
    kernel or the kernel's source changed since the counters were taken."""
    from paper_1907_02154_amd.traffic import source_sha
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.txt")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            parts = line.rstrip("\n").split("\t")
            if parts[0] == kernel and len(parts) >= 4:
                if parts[1] != source_sha(kernel):
                    return None
                return int(parts[2]) + int(parts[3])
    return None


def gpu_info(torch) -> dict:
    """Device properties, plus clocks and socket power from amd-smi when it answers."""
    p = torch.cuda.get_device_properties(0)
    info = dict(name=p.name, arch=getattr(p, "gcnArchName", "").split(":")[0],
                cus=p.multi_processor_count, hbm_gib=round(p.total_memory / 2 ** 30))
    try:
        r = subprocess.run(["amd-smi", "metric", "-g", "0", "--clock", "--power", "--json"],
                           capture_output=True, text=True, timeout=30)
        d = json.loads(r.stdout)
        d = (d["gpu_data"] if isinstance(d, dict) else d)[0]
        info["gfx_clk_max_mhz"] = d["clock"]["gfx_0"]["max_clk"]["value"]
        info["mem_clk_max_mhz"] = d["clock"]["mem_0"]["max_clk"]["value"]
        info["socket_power_w_after_run"] = d["power"]["socket_power"]["value"]
    except Exception:
        pass
    try:
        r = subprocess.run(["rocm-smi", "--showmaxpower", "--json"], capture_output=True, text=True,
                           timeout=30)
        for card in json.loads(r.stdout).values():
            for k, v in card.items():
                if "Power" in k:
                    info["power_cap_w"] = float(v)
    except Exception:
        pass
    return info


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", type=int, default=2, choices=[1, 2, 3, 4, 5, 6],
                    help="1-5: the evaluation configurations; 6: SqueezeNet 1.0 convs at batch 1")
    ap.add_argument("--batch", type=int, default=None, help="override the config's batch")
    ap.add_argument("--cpu-seconds", type=float, default=20.0,
                    help="budget for the CPU-oracle baseline (0 disables it)")
    ap.add_argument("--layers", action="store_true", help="also print a per-layer table to stderr")
    ap.add_argument("--chain", choices=["resnet50_b64", "resnet50_b1", "mobilenet_b1"], default=None,
                    help="instead: a whole-network pass (layers chained, glue and joins included); "
                         "resnet50_b64 keeps bf16 channel-last activations between layers")
    ap.add_argument("--no-b64", action="store_true",
                    help="with the default --config 2: skip the nested batch-64 bf16 record (config 5)")
    ap.add_argument("--profile-passes", type=int, default=0, metavar="N",
                    help="instead: run N eager passes of the stack and exit (for counter runs)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="instead: 4 device-to-device copies of 256 MiB (counter calibration)")
    ap.add_argument("--dw-sweep", type=int, default=0, metavar="N",
                    help="instead: HBM bandwidth of the depthwise kernel on the 13 MobileNet "
                         "depthwise shapes at batch N (e.g. 256)")
    ap.add_argument("--vision", action="store_true",
                    help="instead: only the vision operators (box_nms, segmented argsort, prefix sum)")
    ap.add_argument("--no-vision", action="store_true",
                    help="skip the nested vision-operator record of the default run")
    ap.add_argument("--residual-join", action="store_true",
                    help="instead: the ResNet-50 join layers (last 1x1 of each bottleneck block) "
                         "with the shortcut add + ReLU fused into the conv epilogue, against the "
                         "same convs followed by a separate add kernel (--config 2 or 5)")
    ap.add_argument("--vendor-gemm", action="store_true",
                    help="instead: the vendor bf16 GEMM (torch.matmul, hipBLASLt) on the ResNet-50 b64 "
                         "layer shapes as plain [M, C*R*S] x [C*R*S, K] products, im2col excluded "
                         "(context for the conv kernels, not part of the library)")
    return ap.parse_args()


def _graph_ms(torch, fn, steps, stream):
    """Mean ms of one call of fn(s) (which enqueues on stream s) over a HIP graph
    of `steps` calls, captured on a side stream and replayed on `stream` once
    untimed and once timed."""
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(stream)
    with torch.cuda.graph(g, stream=side):
        for _ in range(steps):
            fn(side)
    torch.cuda.synchronize()
    g.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    g.replay()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / steps


def vendor_gemm(args):
    """The ResNet-50 batch-64 layer shapes (configuration 5) as plain bf16 GEMMs
    through torch.matmul (hipBLASLt), each distinct shape timed as a HIP graph of
    `steps` products over four rotating input/output sets, fp32 accumulation,
    bf16 output.  The operand of a 3x3 or strided layer is taken as an already
    formed [M, C*R*S] matrix, so this is a lower bound on an im2col + GEMM
    convolution: it skips the im2col, the bias, ReLU and residual join."""
    import torch
    from paper_1907_02154_amd import workloads as wl
    torch.cuda.set_device(0)
    torch.backends.cuda.matmul.allow_bf16_reduced_precision_reduction = False
    stream = torch.cuda.current_stream()
    rows, seen, total = [], {}, 0.0
    for l in wl.workload(5).layers:
        P, Q = (l.H + 2 * l.pad - l.R) // l.stride + 1, (l.W + 2 * l.pad - l.S) // l.stride + 1
        M, Kred = l.N * P * Q, l.C * l.R * l.S
        key = (M, Kred, l.K)
        if key not in seen:
            b = torch.randn(Kred, l.K, device="cuda", dtype=torch.bfloat16)
            sets = [(torch.randn(M, Kred, device="cuda", dtype=torch.bfloat16),
                     torch.empty(M, l.K, device="cuda", dtype=torch.bfloat16)) for _ in range(4)]
            it = [0]

            def one(s, sets=sets, b=b, it=it):
                x, y = sets[it[0] % 4]
                it[0] += 1
                torch.matmul(x, b, out=y)

            with torch.cuda.stream(torch.cuda.Stream()):
                for _ in range(args.warmup):
                    one(None)
            torch.cuda.synchronize()
            seen[key] = _graph_ms(torch, one, args.steps, stream) * 1e3
            del sets
        us = seen[key]
        total += us
        fl = 2.0 * M * Kred * l.K
        rows.append({"layer": l.name, "M": M, "CRS": Kred, "K": l.K, "us": round(us, 2),
                     "mfma_frac": round(fl / us / 1e6 / PEAK_BF16_MFMA_TFLOPS, 4)})
    print(json.dumps({"metric": "vendor GEMM time on the ResNet-50 b64 layer shapes (im2col excluded)",
                      "value": round(total / 1e3, 4), "unit": "ms", "n_gpus": 1, "steps": args.steps,
                      "warmup": args.warmup, "higher_is_better": False, "dtype": "bf16", "data": "synthetic",
                      "config": {"workload": "ResNet-50 v1 b64 layer shapes as plain GEMMs",
                                 "library": "torch.matmul (hipBLASLt)", "device": gpu_info(torch)},
                      "layers": rows}), flush=True)


def residual_join(args):
    """Operator fusion of the residual join (ResNet bottleneck: y = relu(conv +
    bias + shortcut)).  The 16 join layers of ResNet-50 (c3 of every block) run
    as one stack with the shortcut read in the conv epilogue, and as the same
    stack without it followed by one add + ReLU kernel per layer (in place, as
    a framework without fusion runs it).  Both variants are timed as HIP graphs
    of K passes with every tensor resident; inputs are seeded as in the
    configuration (shortcuts normal(0, 1))."""
    import torch
    from paper_1907_02154_amd import miconv
    from paper_1907_02154_amd import workloads as wl

    if args.config not in (2, 5):
        print("--residual-join runs on --config 2 or 5 (ResNet-50)", file=sys.stderr)
        sys.exit(2)
    torch.cuda.set_device(0)
    wk = wl.workload(args.config, args.batch)
    bf16 = wk.dtype == "bf16"
    op = miconv.OP_CONV_BF16 if bf16 else miconv.OP_CONV_F32
    gen = torch.Generator(device="cuda")
    gen.manual_seed(wl.SEED_BASE + 4242)
    fused, plain, adds, elems, conv_flops = [], [], [], 0, 0
    for i, l in enumerate(wk.layers):
        if not l.name.endswith("c3"):
            continue
        x, w, b = wl.layer_tensors(args.config, i, l)
        if bf16:
            tx = torch.from_numpy(wl.to_bf16_bits(x).view(np.int16)).cuda().view(torch.bfloat16)
            tw = torch.from_numpy(wl.to_bf16_bits(w).view(np.int16)).cuda().view(torch.bfloat16)
        else:
            tx, tw = torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda()
        tb = torch.from_numpy(b).cuda()
        P, Q = miconv.out_dims(l.H, l.W, l.R, l.S, l.stride, l.pad)
        res = torch.randn((l.N, l.K, P, Q), device="cuda", generator=gen)
        yf = torch.empty_like(res)
        yp = torch.empty_like(res)
        fused.append((op, tx, tw, tb, yf, l.stride, l.pad, l.groups, True, res))
        plain.append((op, tx, tw, tb, yp, l.stride, l.pad, l.groups, False))
        adds.append((yp, res))
        elems += res.numel()
        conv_flops += wl.flops(l, P, Q)
    sf, sp = miconv.Stack(fused), miconv.Stack(plain)
    sf.overlap(False)   # unrelated layers: timed in order, one at a time
    sp.overlap(False)
    stream = torch.cuda.current_stream()
    for _ in range(max(1, args.warmup)):
        sf.launch(stream)
        sp.launch(stream)
        for y, r in adds:
            miconv.add_act_fwd(y, r, y, True, stream)
    torch.cuda.synchronize()
    # the two variants agree (one fp32 rounding of the conv sum apart at most)
    sf.launch(stream)
    sp.launch(stream)
    for y, r in adds:
        miconv.add_act_fwd(y, r, y, True, stream)
    torch.cuda.synchronize()
    diff = max(float((f[4] - a[0]).abs().max()) / max(float(a[0].abs().max()), 1e-30)
               for f, a in zip(fused, adds))
    K = args.steps
    sf.capture(K, timed=False, stream=stream)
    sp.capture(K, timed=False, stream=stream)
    ms = {}
    for name, st in (("fused", sf), ("conv_only", sp)):
        st.replay(stream)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        st.replay(stream)
        e1.record(stream)
        torch.cuda.synchronize()
        ms[name] = e0.elapsed_time(e1) / K

    def add_pass(strm):
        for y, r in adds:
            miconv.add_act_fwd(y, r, y, True, strm)
    ms["add_kernels"] = _graph_ms(torch, add_pass, K, stream)
    sf.close()
    sp.close()
    unfused = ms["conv_only"] + ms["add_kernels"]
    out = {"metric": "ResNet-50 join layers: conv + residual add + ReLU, ms per pass",
           "value": round(ms["fused"], 4), "unit": "ms", "n_gpus": 1, "steps": K,
           "warmup": args.warmup, "ms_per_step": round(ms["fused"], 4), "higher_is_better": False,
           "scaling": "weak", "vs_baseline": None, "dtype": "bf16" if bf16 else "f32",
           "data": "synthetic",
           "config": {"workload": f"{wk.name}: its 16 bottleneck join layers (c3)",
                      "join_elements": elems, "conv_flops": conv_flops,
                      "device": gpu_info(torch)},
           "unfused_ms": round(unfused, 4), "conv_only_ms": round(ms["conv_only"], 4),
           "add_kernels_ms": round(ms["add_kernels"], 4),
           "fused_join_overhead_ms": round(ms["fused"] - ms["conv_only"], 4),
           "speedup": round(unfused / ms["fused"], 3),
           "algorithmic_join_bytes": {"fused": 4 * elems, "separate": 12 * elems},
           "max_rel_diff_fused_vs_separate": diff}
    print(json.dumps(out), flush=True)


def dw_sweep(args):
    """Depthwise bandwidth sweep: the 13 MobileNet-v1 depthwise layer shapes at
    batch N.  Each layer runs in a native stack of `sets` launches on distinct
    (x, y) buffer pairs -- together more than three times the 256 MB last-level
    cache, so every launch streams from HBM -- captured into a HIP graph with a
    timing event around every launch; the per-layer figure is the median launch
    duration.  Inputs are seeded on the device (uniform [0,1)); values do not
    affect the timing, and parity at these shapes is tested separately.  The
    runtime's own device-to-device copy of 1 GiB is timed for context."""
    import torch
    from paper_1907_02154_amd import miconv
    from paper_1907_02154_amd import workloads as wl

    torch.cuda.set_device(0)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(wl.SEED_BASE + 777)
    rows, tot_bytes, tot_ms = [], 0, 0.0
    for l in [l for l in wl.workload(3).layers if l.kind == "dw"]:
        l = l.with_batch(args.dw_sweep)
        P, Q = miconv.out_dims(l.H, l.W, l.R, l.S, l.stride, l.pad)
        nbytes = 4 * (l.N * l.C * l.H * l.W + l.N * l.C * P * Q + 10 * l.C)
        sets = max(2, -(-(768 << 20) // nbytes))            # > 3x the 256 MB cache
        xs = [torch.rand((l.N, l.C, l.H, l.W), device="cuda", generator=gen) for _ in range(sets)]
        ys = [torch.empty((l.N, l.C, P, Q), device="cuda") for _ in range(sets)]
        w = torch.randn((l.C, 1, 3, 3), device="cuda", generator=gen) * l.he_std
        b = torch.randn((l.C,), device="cuda", generator=gen) * 0.01
        st = miconv.Stack([(miconv.OP_DWCONV_F32, xs[i], w, b, ys[i], l.stride, l.pad, l.C, l.relu)
                           for i in range(sets)])
        st.overlap(False)   # the buffer sets rotate through one layer: one launch at a time
        if args.profile_passes:
            # counter runs: eager launches only (every buffer set, N times)
            for _ in range(args.profile_passes):
                st.launch()
            torch.cuda.synchronize()
            st.close()
            print(f"{l.name}: {args.profile_passes} eager passes over {sets} buffer sets", flush=True)
            del xs, ys
            torch.cuda.empty_cache()
            continue
        for _ in range(max(1, -(-args.warmup // sets))):
            st.launch()
        reps = max(2, -(-args.steps // sets))
        st.capture(reps, True)
        st.replay()
        torch.cuda.synchronize()
        t = st.times()                                      # [reps, sets] ms per launch
        ms = float(np.median(t))
        kernel = st.launch_info(0)[1]
        st.close()
        rows.append(dict(layer=l.name, C=l.C, H=l.H, stride=l.stride, MB=round(nbytes / 1e6, 1),
                         us=round(ms * 1e3, 2), GBs=round(nbytes / ms / 1e6, 1), buffers=sets,
                         kernel=kernel))
        print(json.dumps(rows[-1]), file=sys.stderr, flush=True)
        tot_bytes += nbytes
        tot_ms += ms
        del xs, ys
        torch.cuda.empty_cache()
    if args.profile_passes:
        return
    # For context (not a ceiling): the runtime's own device-to-device copy
    # kernel (torch copy_), 1 GiB each way.
    src = torch.empty(1 << 28, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(10):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    copy_gbs = 2 * src.numel() * 4 * 10 / e0.elapsed_time(e1) / 1e6
    del src, dst
    gbs = tot_bytes / tot_ms / 1e6
    # counted HBM bytes of the sweep (FETCH_SIZE + WRITE_SIZE per launch from
    # the committed counter summary, when it matches every kernel's source)
    counted = [measured_traffic(r["kernel"], f"mobilenet_dw_b{args.dw_sweep}") for r in rows]
    traffic = sum(counted) if all(c is not None for c in counted) else None
    out = {"metric": "depthwise conv HBM bandwidth (MobileNet-v1 dw shapes)", "value": round(gbs, 1),
           "unit": "GB/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
           "ms_per_step": round(tot_ms, 4), "higher_is_better": True, "scaling": "weak",
           "vs_baseline": None, "dtype": "f32", "data": "synthetic (device-seeded uniform)",
           "config": {"workload": f"MobileNet-v1 depthwise layers, batch {args.dw_sweep}",
                      "algorithmic_bytes": tot_bytes, "device": gpu_info(torch)},
           "roofline": {"bound": "hbm", "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                        "frac": round(gbs / PEAK_HBM_GBS, 4), "traffic": traffic,
                        "traffic_over_algorithmic": None if traffic is None else round(traffic / tot_bytes, 4)},
           "runtime_copy_GBs": round(copy_gbs, 1),
           "layers": rows}
    print(json.dumps(out), flush=True)


def stack_record(args, config: int, batch, steps: int, warmup: int, cpu_seconds: float,
                 table: bool) -> dict:
    """Time one configuration's conv stack: resident tensors for every layer,
    `warmup` eager passes, then the timed region (one HIP graph of `steps`
    passes, replayed once untimed and once timed), then `steps` eager passes
    whose kernels carry runtime start/end stamps (per-kernel durations for the
    roofline).  Returns the record printed as JSON."""
    import torch
    from paper_1907_02154_amd import miconv
    from paper_1907_02154_amd import workloads as wl

    wk = wl.workload(config, batch)
    bf16 = wk.dtype == "bf16"

    # Resident inputs, weights, biases and outputs for every layer.
    layers = []
    for i, l in enumerate(wk.layers):
        x, w, b = wl.layer_tensors(config, i, l)
        P, Q = miconv.out_dims(l.H, l.W, l.R, l.S, l.stride, l.pad)
        if bf16:
            tx = torch.from_numpy(wl.to_bf16_bits(x).view(np.int16)).cuda().view(torch.bfloat16)
            tw = torch.from_numpy(wl.to_bf16_bits(w).view(np.int16)).cuda().view(torch.bfloat16)
        else:
            tx = torch.from_numpy(x).cuda()
            tw = torch.from_numpy(w).cuda()
        tb = torch.from_numpy(b).cuda()
        ty = torch.empty((l.N, l.K, P, Q), device="cuda")
        fl = wl.flops(l, P, Q)
        elem_in = 2 if bf16 else 4
        nbytes = (x.size + w.size) * elem_in + (b.size + l.N * l.K * P * Q) * 4
        layers.append(dict(layer=l, idx=i, x=tx, w=tw, b=tb, y=ty, P=P, Q=Q, kernel=None,
                           flops=fl, bytes=nbytes, host=(x, w, b)))
    torch.cuda.synchronize()

    ops = []
    for d in layers:
        l = d["layer"]
        op = miconv.OP_CONV_BF16 if bf16 else (miconv.OP_DWCONV_F32 if l.kind == "dw" else miconv.OP_CONV_F32)
        ops.append((op, d["x"], d["w"], d["b"], d["y"], l.stride, l.pad, l.groups, l.relu))
    stack = miconv.Stack(ops)          # plans every layer; packs filters once
    # each layer has its own input, so none depends on another: they stay in
    # order on one stream (the step is the sum of the layers' latencies, as
    # a network runs them), never overlapped
    stack.overlap(False)
    for j, d in enumerate(layers):
        d["kernel"] = stack.describe(j)
    n_launch = stack.launches
    launch_info = [stack.launch_info(j) for j in range(n_launch)]

    stream = torch.cuda.current_stream()
    if args.profile_passes:
        for _ in range(args.profile_passes):
            stack.launch(stream)
        torch.cuda.synchronize()
        print(f"{args.profile_passes} eager passes of {wk.name}", flush=True)
        sys.exit(0)
    for _ in range(warmup):               # eager passes: caches, instruction caches
        stack.launch(stream)
    torch.cuda.synchronize()

    # The timed region: one HIP graph holding exactly K passes, replayed once
    # untimed (first replay of a fresh graph) and once timed.
    K = steps
    stack.capture(K, timed=False, stream=stream)
    stack.replay(stream)
    torch.cuda.synchronize()
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    wall0 = time.perf_counter()
    t_start.record(stream)
    stack.replay(stream)
    t_end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms_total = t_start.elapsed_time(t_end)
    ms_per_step = ms_total / K

    # Per-kernel durations: K eager passes in which every kernel launch carries
    # a start and an end event that the runtime stamps with the kernel's own
    # execution interval (the figure a kernel-trace profiler reports).
    stack.launch_timed(K, stream)
    torch.cuda.synchronize()
    per_launch_ms = stack.times()
    stack.close()

    launch_ms = per_launch_ms.mean(axis=0)          # mean over the K passes, per kernel launch
    layer_ms = np.zeros(len(layers))
    for j in range(n_launch):
        layer_ms[launch_info[j][0]] += launch_ms[j]
    step_flops = sum(d["flops"] for d in layers)
    tflops = step_flops / (ms_per_step * 1e-3) / 1e12

    # Dominant kernel: the kernel name with the largest summed time.  A conv
    # kernel carries its layers' FLOPs and algorithmic bytes; the helper
    # launches of a layer (split-K reduction, channel-last copy of x, filter
    # packing) carry the bytes they move but no FLOPs.
    groups = {}
    for j in range(n_launch):
        li, name = launch_info[j]
        d = layers[li]
        g = groups.setdefault(name, dict(ms=0.0, flops=0, bytes=0, launches=0, layers=[]))
        g["ms"] += float(launch_ms[j])
        g["launches"] += 1
        main = not name.startswith(("nchw_to_nhwc", "pack_krsc", "splitk_reduce"))
        if main:
            g["flops"] += d["flops"]
            g["bytes"] += d["bytes"]
        else:
            l = d["layer"]
            if name.startswith("splitk_reduce"):
                g["bytes"] += l.N * l.K * d["P"] * d["Q"] * 4
            elif name.startswith("nchw_to_nhwc"):
                # a 1x1 strided layer without padding copies only its sampled pixels
                sub = l.R == 1 and l.S == 1 and l.pad == 0 and l.stride > 1
                px = d["P"] * d["Q"] if sub else l.H * l.W
                g["bytes"] += 2 * l.N * l.C * px * (2 if bf16 else 4)
            else:
                g["bytes"] += 2 * l.K * (l.C // l.groups) * l.R * l.S * (2 if bf16 else 4)
        g["layers"].append(d["layer"].name)
    dom_name, dom = max(groups.items(), key=lambda kv: kv[1]["ms"])
    avg_launch_us = dom["ms"] / dom["launches"] * 1e3
    # The bound is the lower ceiling for the kernel's arithmetic intensity:
    # HBM when its FLOP per algorithmic byte is below the ridge point
    # (MFMA peak / HBM peak), else the MFMA peak of its dtype.
    peak = PEAK_BF16_MFMA_TFLOPS if bf16 else PEAK_FP32_MFMA_TFLOPS
    ridge = peak * 1e12 / (PEAK_HBM_GBS * 1e9)
    if dom_name.startswith("dw") or dom["flops"] < ridge * dom["bytes"]:
        achieved = dom["bytes"] / (dom["ms"] * 1e-3) / 1e9
        roof = dict(bound="hbm", achieved=round(achieved, 2), peak=PEAK_HBM_GBS, unit="GB/s",
                    frac=round(achieved / PEAK_HBM_GBS, 4))
    else:
        achieved = dom["flops"] / (dom["ms"] * 1e-3) / 1e12
        roof = dict(bound="mfma", achieved=round(achieved, 3), peak=peak, unit="TFLOP/s",
                    frac=round(achieved / peak, 4))
    tag = {2: "resnet50_b1", 5: "resnet50_b64", 3: "mobilenet_b1", 4: "vgg16_b8", 6: "squeezenet_b1",
           1: "conv3x3_b1"}[config] if batch is None else f"config{config}_b{batch}"
    roof.update(traffic=measured_traffic(dom_name, tag),
                algorithmic_bytes_per_launch=round(dom["bytes"] / dom["launches"]),
                algorithmic_flops_per_launch=round(dom["flops"] / dom["launches"]),
                kernel=dom_name, launches_per_step=dom["launches"],
                avg_launch_us=round(avg_launch_us, 3),
                share_of_step=round(dom["ms"] / float(launch_ms.sum()), 4))

    # Stack-wide fraction of roofline: sum over layers of the time the layer
    # needs at the binding peak (MFMA or HBM, whichever is slower for it), over
    # the graph-timed step (and, for reference, over the summed kernel stamps).
    t_roof = sum(max(d["flops"] / (peak * 1e12), d["bytes"] / (PEAK_HBM_GBS * 1e9)) for d in layers)
    stack_roof_frac = t_roof / (ms_per_step * 1e-3)
    stack_roof_frac_kernels = t_roof / (float(layer_ms.sum()) * 1e-3)

    if table:
        # per layer: mean over the K passes (the launch parts), and the median,
        # 10th and 90th percentile of the layer's per-pass time
        parts = [[] for _ in layers]
        per_pass = np.zeros((per_launch_ms.shape[0], len(layers)))
        for j in range(n_launch):
            parts[launch_info[j][0]].append(float(launch_ms[j]) * 1e3)
            per_pass[:, launch_info[j][0]] += per_launch_ms[:, j]
        for j, d in enumerate(layers):
            l = d["layer"]
            t = float(layer_ms[j])
            p10, med, p90 = (float(v) * 1e3 for v in np.percentile(per_pass[:, j], [10, 50, 90]))
            split = " [" + " + ".join(f"{u:.2f}" for u in parts[j]) + "]" if len(parts[j]) > 1 else ""
            print(f"{j:3d} {l.name:10s} {d['kernel']:45s} {t * 1e3:9.2f} us "
                  f"{d['flops'] / t / 1e9:8.2f} TFLOP/s {d['bytes'] / t / 1e6:8.1f} GB/s "
                  f"(median {med:.2f}, p10 {p10:.2f}, p90 {p90:.2f} us){split}",
                  file=sys.stderr)

    # CPU baseline: the oracle on a bounded prefix of the same layers.
    cpu = None
    if cpu_seconds > 0:
        import oracle
        done_flops, t_cpu, sample = 0, 0.0, []
        for d in layers:
            l = d["layer"]
            x, w, b = d["host"]
            t0 = time.perf_counter()
            if bf16:
                oracle.conv2d_bf16(wl.to_bf16_bits(x), wl.to_bf16_bits(w), b, l.stride, l.pad,
                                   l.groups, l.relu)
            elif l.kind == "dw":
                oracle.dwconv2d(x, w, b, l.stride, l.pad, l.relu)
            else:
                oracle.conv2d(x, w, b, l.stride, l.pad, l.groups, l.relu)
            t_cpu += time.perf_counter() - t0
            done_flops += d["flops"]
            sample.append(l.name)
            if t_cpu > cpu_seconds:
                break
        cpu = dict(value=round(done_flops / t_cpu / 1e12, 6), unit="TFLOP/s",
                   cores=oracle.num_threads(), cpu=cpu_model(), kind="oracle",
                   sample=f"{len(sample)} of {len(layers)} layers ({sample[0]}..{sample[-1]}), "
                          f"{done_flops / 1e9:.3f} GFLOP in {t_cpu:.2f} s, fp64 accumulation")

    rec = {
        "value": round(tflops, 4),
        "unit": "TFLOP/s",
        "ms_per_step": round(ms_per_step, 5),
        "ms_per_image": round(ms_per_step / wk.layers[0].N, 5),
        "dtype": "bf16-in/f32-acc" if bf16 else "f32",
        "config": {"workload": wk.name, "convs": len(layers), "batch": wk.layers[0].N,
                   "gflop_per_step": round(step_flops / 1e9, 4),
                   "wall_s_timed": round(wall, 4),
                   "timing": "value: one HIP graph of K passes between two events; roofline: kernel "
                             "execution times stamped by the runtime on K eager passes",
                   "launches_per_step": n_launch,
                   "kernel_ms_per_step": round(float(launch_ms.sum()), 5),
                   "stack_roofline_frac": round(stack_roof_frac, 4),
                   "stack_roofline_frac_kernel_stamps": round(stack_roof_frac_kernels, 4)},
        "roofline": roof,
        "cpu_baseline": cpu,
    }
    if bf16 and wk.layers[0].N >= 32:
        # the compute-bound 3x3 layers of stages 3-5: fraction of bf16 MFMA peak
        # per layer, copies and split reductions of the layer included
        per = []
        for j, d in enumerate(layers):
            l = d["layer"]
            if l.R == 3 and l.name[:2] in ("s3", "s4", "s5"):
                t = float(layer_ms[j]) * 1e-3
                per.append(dict(layer=l.name, us=round(t * 1e6, 2),
                                mfma_frac=round(d["flops"] / t / 1e12 / peak, 4)))
        rec["mfma_frac_3x3_s3_s5"] = per
    return rec


def single_call_times(steps: int) -> dict:
    """The single-layer configuration (conv 64 -> 64 3x3 at 56 x 56, batch 1,
    fp32) through each entry point, every variant timed as a HIP graph of
    `steps` calls: conv2d_fwd (no workspace, filters as given),
    conv2d_fwd_ws (caller workspace), conv2d_fwd_packed (filters packed once)
    and a one-layer stack."""
    import torch
    from paper_1907_02154_amd import miconv
    from paper_1907_02154_amd import workloads as wl

    l = wl.workload(1).layers[0]
    x, w, b = wl.layer_tensors(1, 0, l)
    tx, tw, tb = torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda(), torch.from_numpy(b).cuda()
    P, Q = miconv.out_dims(l.H, l.W, l.R, l.S, l.stride, l.pad)
    y = torch.empty((l.N, l.K, P, Q), device="cuda")
    ws = miconv.workspace(miconv.conv2d_workspace_bytes(l.N, l.C, l.H, l.W, l.K, l.R, l.S, l.stride, l.pad))
    pk = miconv.PackedFilters(tw, tuple(tx.shape), l.stride, l.pad)
    st = miconv.Stack([(miconv.OP_CONV_F32, tx, tw, tb, y, l.stride, l.pad, 1, l.relu)])
    stream = torch.cuda.current_stream()
    fns = {
        "conv2d_fwd": lambda s: miconv.conv2d_fwd(tx, tw, tb, y, l.stride, l.pad, 1, l.relu, stream=s),
        "conv2d_fwd_ws": lambda s: miconv.conv2d_fwd_ws(tx, tw, tb, y, l.stride, l.pad, 1, l.relu, ws=ws,
                                                        stream=s),
        "conv2d_fwd_packed": lambda s: pk.forward(tx, tb, y, l.relu, stream=s),
        "stack": lambda s: st.launch(s),
    }
    out = {}
    for name, fn in fns.items():
        for _ in range(5):
            fn(stream)
        torch.cuda.synchronize()
        out[name + "_us"] = round(_graph_ms(torch, fn, steps, stream) * 1e3, 3)
    st.close()
    fl = wl.flops(l, P, Q)
    out["workload"] = "conv 64->64 3x3 @56x56 b1 fp32 (231.2 MFLOP)"
    out["kernels"] = {m: miconv.conv2d_describe(l.N, l.C, l.H, l.W, l.K, l.R, l.S, l.stride, l.pad,
                                                mode=m)[0] for m in ("plain", "ws", "packed", "stack")}
    out["tflops_stack"] = round(fl / (out["stack_us"] * 1e-6) / 1e12, 3)
    return out


def chain_record(args, net: str, layout: str, steps: int, warmup: int, table: bool = False) -> dict:
    """A whole-network pass (paper_1907_02154_amd.networks): every layer reads
    the previous layers' outputs, with the network's glue (ResNet's max-pool)
    in the same stack and the shortcut joins fused into the convs.  Timed like
    stack_record: one HIP graph of K passes; per-kernel durations from K eager
    passes with runtime stamps.  net: "resnet50_b64" (bf16, layout "bf16_cl"
    or fp32 NCHW at batch 64 is not offered), "resnet50_b1" or "mobilenet_b1"
    (fp32)."""
    import torch
    from paper_1907_02154_amd import miconv
    from paper_1907_02154_amd import networks as nets
    from paper_1907_02154_amd import workloads as wl

    config = {"resnet50_b64": 5, "resnet50_b1": 2, "mobilenet_b1": 3}[net]
    graph = nets.mobilenet_graph() if net == "mobilenet_b1" else nets.resnet50_graph(config)
    bf16 = layout == "bf16_cl"
    x0, _, _ = wl.layer_tensors(config, 0, wl.workload(config).layers[0])
    params = {}
    for node in graph:
        if node.kind == "conv":
            _, w, b = wl.layer_tensors(config, node.index, node.layer)
            tw = (torch.from_numpy(wl.to_bf16_bits(w).view(np.int16)).cuda().view(torch.bfloat16) if bf16
                  else torch.from_numpy(w).cuda())
            params[node.name] = (tw, torch.from_numpy(b).cuda())
    tx = (torch.from_numpy(wl.to_bf16_bits(x0).view(np.int16)).cuda().view(torch.bfloat16) if bf16
          else torch.from_numpy(x0).cuda())
    ops, outs = nets.build_stack(graph, tx, params, layout)
    stack = miconv.Stack(ops)
    n_launch = stack.launches
    launch_info = [stack.launch_info(j) for j in range(n_launch)]
    stream = torch.cuda.current_stream()
    if args.profile_passes:
        for _ in range(args.profile_passes):
            stack.launch(stream)
        torch.cuda.synchronize()
        print(f"{args.profile_passes} eager passes of the {net} network", flush=True)
        sys.exit(0)
    for _ in range(warmup):
        stack.launch(stream)
    torch.cuda.synchronize()

    def graph_ms():
        stack.capture(steps, timed=False, stream=stream)
        stack.replay(stream)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        stack.replay(stream)
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / steps

    # the pass in one stream, and, for comparison, with the layers the
    # network's dependencies allow on a second stream
    overlapped = stack.overlap(True)
    ms_two = graph_ms()
    stack.overlap(False)
    ms_per_step = graph_ms()
    stack.launch_timed(steps, stream)
    torch.cuda.synchronize()
    launch_ms = stack.times().mean(axis=0)
    names = [n.name for n in graph]
    flops, nbytes, layer_ms = {}, {}, np.zeros(len(graph))
    elem = 2 if bf16 else 4
    for node in graph:
        if node.kind != "conv":
            continue
        l = node.layer
        P, Q = miconv.out_dims(l.H, l.W, l.R, l.S, l.stride, l.pad)
        flops[node.name] = wl.flops(l, P, Q)
        xin = l.N * l.C * l.H * l.W * (2 if bf16 else 4)
        yout = l.N * l.K * P * Q * elem
        nbytes[node.name] = xin + l.K * (l.C // l.groups) * l.R * l.S * (2 if bf16 else 4) + 4 * l.K + yout + \
            (yout if node.res else 0)
    conv_ms, pool_ms, per_kernel = 0.0, 0.0, {}
    for j in range(n_launch):
        li, kname = launch_info[j]
        layer_ms[li] += launch_ms[j]
        if graph[li].kind == "conv":
            conv_ms += float(launch_ms[j])
        else:
            pool_ms += float(launch_ms[j])
        k = per_kernel.setdefault(kname, [0.0, 0])
        k[0] += float(launch_ms[j])
        k[1] += 1
    if table:
        for i, node in enumerate(graph):
            extra = ""
            if node.kind == "conv":
                t = float(layer_ms[i]) * 1e-3
                extra = (f"{flops[node.name] / t / 1e12:8.2f} TFLOP/s {nbytes[node.name] / t / 1e9:8.1f} GB/s")
            print(f"{i:3d} {node.name:10s} {stack.describe(i):60s} {layer_ms[i] * 1e3:9.2f} us {extra}",
                  file=sys.stderr)
    stack.close()
    total_flops = sum(flops.values())
    peak = PEAK_BF16_MFMA_TFLOPS if bf16 else PEAK_FP32_MFMA_TFLOPS
    t_roof = sum(max(flops[n] / (peak * 1e12), nbytes[n] / (PEAK_HBM_GBS * 1e9)) for n in flops)
    dom = max(per_kernel.items(), key=lambda kv: kv[1][0])
    dom_traffic = measured_traffic(dom[0], f"{net}_chained")
    N = graph[0].layer.N
    return {
        "workload": f"{net} network pass ({layout}): {len(flops)} convs"
                    + (" + max-pool" if len(flops) < len(graph) else "") + ", shortcut joins fused",
        "value": round(total_flops / (ms_per_step * 1e-3) / 1e12, 4), "unit": "TFLOP/s",
        "ms_per_step": round(ms_per_step, 5), "ms_per_image": round(ms_per_step / N, 5),
        "two_streams": {"layers_on_second_stream": overlapped, "ms_per_step": round(ms_two, 5)},
        "gflop_per_step": round(total_flops / 1e9, 4), "launches_per_step": n_launch,
        "conv_kernel_ms": round(conv_ms, 5), "glue_kernel_ms": round(pool_ms, 5),
        "stack_roofline_frac": round(t_roof / (ms_per_step * 1e-3), 4),
        "dominant_kernel": {"kernel": dom[0], "ms_per_step": round(dom[1][0], 5), "launches": dom[1][1],
                            "avg_launch_us": round(dom[1][0] / dom[1][1] * 1e3, 3), "traffic": dom_traffic},
    }


def vision_record(steps: int, cpu_seconds: float) -> dict:
    """The vision operators of Sec. 3.1.1 on their own workloads, each timed
    as a HIP graph of `steps` calls with inputs resident in HBM:
      * box_nms on SSD-style detection rows (24564 anchors per image, 20
        classes, score > 0.01, best 400 compared, IoU 0.45) at batch 1
        (latency) and batch 32 (throughput);
      * segmented argsort of 2^22 normal keys in 4096 segments of varying
        length (keys/s; the merge passes move 12 bytes per key each way);
      * the three-stage prefix sum of one row of 2^26 int32 (the across-
        work-group path), against HBM bandwidth (algorithmic bytes: 4 read
        + 4 written per value);
    plus the oracle timed on a bounded sample of the box_nms workload."""
    import torch
    from paper_1907_02154_amd import detections as det
    from paper_1907_02154_amd import miconv, vision

    stream = torch.cuda.current_stream()
    rec = {"workload": "SSD-style detection rows, 24564 x [class, score, x1, y1, x2, y2], 20 classes; "
                       "valid_thresh 0.01, topk 400, overlap 0.45"}
    for B in (1, 32):
        data = torch.from_numpy(det.detection_rows(B, seed=100 + B)).cuda()
        out = torch.empty_like(data)
        ws = miconv.workspace(vision.box_nms_workspace_bytes(B, data.shape[1], 6, 400))
        fn = lambda s, d=data, o=out, w=ws: vision.box_nms(d, 0.45, 0.01, 400, out=o, ws=w, stream=s)  # noqa: E731
        fn(stream)
        ms = _graph_ms(torch, fn, steps, stream)
        rec[f"box_nms_b{B}_us"] = round(ms * 1e3, 2)
        if B > 1:
            rec[f"box_nms_b{B}_images_per_s"] = round(B / (ms * 1e-3), 1)
    n, S = 1 << 22, 4096
    keys = torch.from_numpy(det.keys(n, seed=5)).cuda()
    off = torch.from_numpy(det.segment_offsets(S, n, seed=5)).cuda()
    idx = torch.empty(n, dtype=torch.int32, device="cuda")
    ws = miconv.workspace(vision.argsort_workspace_bytes(n, S))
    fn = lambda s: vision.segmented_argsort(keys, off, True, out=idx, ws=ws, stream=s)  # noqa: E731
    fn(stream)
    ms = _graph_ms(torch, fn, max(steps // 5, 3), stream)
    passes = 0
    L = 2048
    while L < n:
        passes, L = passes + 1, 2 * L
    rec["argsort"] = {"n": n, "segments": S, "us": round(ms * 1e3, 1), "Mkeys_per_s": round(n / (ms * 1e3), 1),
                      "merge_passes": passes}
    n = 1 << 26
    # two input/output sets in turn, so that a call does not find the previous
    # call's input in the 256 MB last-level cache
    sets = [(torch.ones(n, dtype=torch.int32, device="cuda"), torch.empty(n, dtype=torch.int32, device="cuda"))
            for _ in range(2)]
    ws = miconv.workspace(vision.scan_workspace_bytes(1, n))
    turn = [0]

    def fn(s):
        x, y = sets[turn[0] % 2]
        turn[0] += 1
        vision.scan_i32(x, y, ws=ws, stream=s)

    fn(stream)
    ms = _graph_ms(torch, fn, 2 * max(steps // 10, 2), stream)
    gbs = 8.0 * n / (ms * 1e-3) / 1e9
    rec["scan"] = {"n": n, "us": round(ms * 1e3, 1), "GBs_algorithmic": round(gbs, 1), "buffer_sets": 2}
    rec["roofline"] = {"kernel": "scan (upsweep + tile sums + downsweep)", "bound": "hbm",
                       "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                       "frac": round(gbs / PEAK_HBM_GBS, 4), "traffic": None}
    if cpu_seconds > 0:
        import oracle
        data = det.detection_rows(1, seed=101)
        t0, k = time.perf_counter(), 0
        while k < 200 and time.perf_counter() - t0 < cpu_seconds:
            oracle.box_nms(data, 0.45, 0.01, 400)
            k += 1
        dt = (time.perf_counter() - t0) / k
        rec["cpu_baseline"] = {"value": round(dt * 1e3, 3), "unit": "ms/image", "cores": 1, "kind": "oracle",
                               "sample": f"box_nms oracle on {k} calls of the batch-1 workload"}
    return rec


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: --gpus {args.gpus} is not supported "
              "(there is no multi-GPU path)", file=sys.stderr)
        sys.exit(2)
    if args.dw_sweep:
        dw_sweep(args)
        return
    if args.residual_join:
        residual_join(args)
        return
    if args.vendor_gemm:
        vendor_gemm(args)
        return
    if args.vision:
        import torch
        torch.cuda.set_device(0)
        rec = vision_record(args.steps, min(args.cpu_seconds, 5.0))
        rec.update(metric="vision operator latency", n_gpus=1, steps=args.steps, warmup=args.warmup, data="synthetic")
        print(json.dumps(rec), flush=True)
        return
    if args.chain:
        import torch
        torch.cuda.set_device(0)
        layout = "bf16_cl" if args.chain == "resnet50_b64" else "f32"
        rec = chain_record(args, args.chain, layout, args.steps, args.warmup, args.layers)
        rec.update(metric="network pass TFLOP/s", n_gpus=1, steps=args.steps, warmup=args.warmup,
                   higher_is_better=True, dtype="bf16" if layout == "bf16_cl" else "f32", data="synthetic")
        print(json.dumps(rec), flush=True)
        return
    if args.copy_calibration:
        import torch
        torch.cuda.set_device(0)
        src = torch.zeros(64 << 20, device="cuda")     # 256 MiB of fp32
        dst = torch.empty_like(src)
        for _ in range(4):
            dst.copy_(src)
        torch.cuda.synchronize()
        print("copy calibration: 4 copies of 268435456 bytes", flush=True)
        return

    import torch
    from paper_1907_02154_amd import miconv

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)
    miconv.lib()

    rec = stack_record(args, args.config, args.batch, args.steps, args.warmup, args.cpu_seconds, args.layers)
    out = {
        "metric": "conv TFLOP/s and ms/image (ResNet-50 convs, b=1 & b=64); % MFMA/HBM peak",
        "value": rec["value"],
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": rec["ms_per_step"],
        "ms_per_image": rec["ms_per_image"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": rec["dtype"],
        "data": "synthetic (seeded uniform/He-normal per layer, resident in HBM)",
        "config": dict(rec["config"], device=gpu_info(torch)),
        "roofline": rec["roofline"],
        "cpu_baseline": rec["cpu_baseline"],
    }
    if "mfma_frac_3x3_s3_s5" in rec:
        out["mfma_frac_3x3_s3_s5"] = rec["mfma_frac_3x3_s3_s5"]
    if args.config == 2 and args.batch is None and not args.no_b64:
        # the metric's batch-64 half: ResNet-50 at batch 64, bf16 inputs, fp32
        # accumulation and outputs, timed the same way (its own warm-up, K passes)
        out["b64"] = stack_record(args, 5, None, args.steps, args.warmup, min(args.cpu_seconds, 15.0), False)
        # the same network at batch 64 as one chained pass with bf16
        # channel-last activations between layers (no per-layer copies, bf16
        # outputs, joins fused)
        out["b64_chained"] = chain_record(args, "resnet50_b64", "bf16_cl", args.steps, args.warmup)
    if args.config == 2 and args.batch is None:
        # the batch-1 network as one chained pass (stem, max-pool, blocks with
        # the join fused; projection shortcuts beside the block's first convs)
        out["b1_chained"] = chain_record(args, "resnet50_b1", "f32", args.steps, args.warmup)
    if args.config in (1, 2) and args.batch is None:
        out["single_call"] = single_call_times(args.steps)
    if args.config == 2 and args.batch is None and not args.no_vision:
        # the vision operators of detection post-processing (Sec. 3.1.1)
        out["vision"] = vision_record(args.steps, min(args.cpu_seconds, 5.0))
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
