#!/usr/bin/env python3
"""Throughput of the GBLA forward pass on one MI355X.

A step is one gbla_forward call (Conv1D, key gating, global state, readout
and gated RMSNorm of every head) over one batch of synthetic inputs already
resident in HBM.  Default workload: B=1, H=8, n=32768, d=64, bf16 inputs,
conv width 4.  Several copies of the inputs and outputs (at least 1 GiB in
total) are used round-robin so the 256 MB last-level cache cannot hold a
step's working set.

Prints one JSON line (rank 0) with the metric, the roofline of the dominant
kernel (timed live with HIP events on the launch stream) and the fp64 oracle
timed on the host cores over a bounded sample.
"""
import argparse
import hashlib
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "GBLA fwd tokens/sec at n=32768,H=8,d=64; % of HBM roofline (rocprof)"
HBM_PEAK_GBPS = 8000.0
PROFILES = os.path.join(ROOT, "profiles")


def kernel_source_hash() -> str:
    """Hash of the sources the forward pass is built from (kernels and plan)."""
    h = hashlib.sha256()
    for f in ("gbla_kernels.hip", "gbla_stream.hip", "gbla_state64.hip", "gbla_state128.hip",
              "gbla_device.h", "gbla_plan.cpp", "gbla_plan.h"):
        with open(os.path.join(ROOT, "paper_2606_07317_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def algorithmic_bytes(inp, part: str, gate: bool = True, norm: bool = True) -> int:
    """Bytes each stage must move at least once (inputs read once, y written once).
    Per token and head, with e = element size of the inputs:
      state:   k, v (2 d e) + a (e)          = (2d + 1) e
      readout: q, r (2 d e) + y (4 d)        = 2 d e + 4 d
      forward: (4d + 1) e + 4 d               (770 B at d = 64, bf16)
    Without the key gates a is not read; without the gated norm r is not read."""
    w = inp.workload
    e = 2 if w.dtype == "bf16" else 4
    d = w.head_dim
    th = inp.tokens * w.heads
    a_b = e if gate else 0
    r_b = d * e if norm else 0
    per = {"state": 2 * d * e + a_b, "readout": d * e + r_b + 4 * d,
           "forward": 3 * d * e + a_b + r_b + 4 * d}[part]
    return th * per


# The paper's ablation rows (Section 3, "Ablation", Table 4) as forward-bench options:
# name -> (flags attribute of the binding, gate kept, conv kept, norm kept).
SWITCHES = {"none": (None, True, True, True), "no_gate": ("NO_GATE", False, True, True),
            "no_conv": ("NO_CONV", True, False, True), "no_norm": ("NO_NORM", True, True, False),
            "bla": ("BLA", False, False, False)}


def traffic_from_profiles(kernel: str, workload: str):
    """HBM bytes per launch measured with rocprofv3 counters, if the committed
    measurement was taken on the current kernel sources."""
    path = os.path.join(PROFILES, "traffic.json")
    if not os.path.exists(path):
        return None
    try:
        rec = json.load(open(path)).get("%s/%s" % (kernel, workload))
    except (ValueError, OSError):
        return None
    if not rec or rec.get("source_hash") != kernel_source_hash():
        return None
    return rec.get("bytes_per_launch")


def cpu_baseline(inp, seconds: float, gate: bool = True, conv: bool = True, norm: bool = True):
    import oracle
    orc = oracle.load()
    threads = orc.max_threads()
    units = inp.nseq * inp.workload.heads
    times = []
    t_start = time.perf_counter()
    while True:
        t0 = time.perf_counter()
        orc.forward_inputs(inp, want=("y",), nthreads=threads, gate=gate, conv=conv, norm=norm)
        times.append(time.perf_counter() - t0)
        if len(times) >= 3 and time.perf_counter() - t_start >= seconds:
            break
        if len(times) >= 50:
            break
    med = statistics.median(times)
    return {"value": inp.tokens / med, "unit": "tokens/s", "cores": min(threads, units),
            "kind": "oracle",
            "sample": "the full %s batch (%d tokens x %d heads), fp64, %d runs, median %.3f s"
                      % (inp.workload.name, inp.tokens, inp.workload.heads, len(times), med)}


BWD_METRIC = "GBLA bwd tokens/sec at n=32768,H=8,d=64"


def bench_backward(args, inp, dev):
    """A step is one gbla_backward call (state recompute, query, key and
    Conv1D passes, parameter-gradient sums) on resident inputs and dy."""
    import torch
    from paper_2606_07317_amd import gbla, inputs
    w = inp.workload
    base = inputs.device_tensors(inp, dev)
    dy = torch.from_numpy(inputs.make_cotangent(inp)).to(dev)
    shape = gbla.make_shape(base["q"], base["conv_w"], inp.eps, base["cu_seqlens"], base["max_seqlen"])
    ws = torch.empty(gbla.backward_workspace_bytes(shape), dtype=torch.uint8, device=dev)
    per_set = sum(base[n].numel() * base[n].element_size() for n in ("q", "k", "v", "a", "r"))
    per_set += base["q"].numel() * 4 * 5 + base["a"].numel() * 4
    nsets = args.sets or max(2, -(-(1 << 30) // per_set) + 1)
    sets = []
    for i in range(nsets):
        t = {n: (base[n].clone() if isinstance(base[n], torch.Tensor) else base[n]) for n in base}
        t["dy"] = dy.clone()
        t["grads"] = gbla.backward(t["q"], t["k"], t["v"], t["a"], t["r"], t["conv_w"], t["gamma"],
                                   t["dy"], eps=inp.eps, cu_seqlens=t["cu_seqlens"],
                                   max_seqlen=t["max_seqlen"], workspace=ws)
        sets.append(t)

    def step(i):
        t = sets[i % nsets]
        gbla.backward(t["q"], t["k"], t["v"], t["a"], t["r"], t["conv_w"], t["gamma"], t["dy"],
                      eps=inp.eps, cu_seqlens=t["cu_seqlens"], max_seqlen=t["max_seqlen"],
                      workspace=ws, grads=t["grads"])

    for i in range(args.warmup):
        step(i)
    stream = torch.cuda.current_stream()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record(stream)
    for i in range(args.steps):
        step(i)
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = ev0.elapsed_time(ev1) / args.steps
    e = 2 if w.dtype == "bf16" else 4
    d = w.head_dim
    # inputs q, k, v, a, r and dy read once; dq, dk, dv, dr, da written once
    byt = inp.tokens * w.heads * ((4 * d + 1) * e + 4 * d + 4 * (4 * d + 1))
    gbps = byt / (ms * 1e-3) / 1e9
    metric = (BWD_METRIC if inp.workload.name == inputs.THROUGHPUT_WORKLOAD
              else "GBLA bwd tokens/sec on " + inp.workload.name)
    res = {"metric": metric, "value": inp.tokens / (ms * 1e-3), "unit": "tokens/s",
           "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms,
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
           "dtype": "f32", "data": "synthetic",
           "config": {"workload": w.name, "B": inp.nseq, "H": w.heads, "tokens": inp.tokens,
                      "d": d, "conv_width": w.conv_width, "inputs": w.dtype, "pass": "backward",
                      "rotating_sets": nsets, "algorithmic_bytes": byt,
                      "effective_GBps": round(gbps, 1), "hbm_frac": round(gbps / HBM_PEAK_GBPS, 4),
                      "wall_s": round(wall, 4)}}
    print(json.dumps(res), flush=True)


# Per-layer latency of GBLA on H100 at batch 8 (the paper's Table 5), for context.
PAPER_H100_LAYER_MS = {2048: 0.618, 4096: 1.141, 8192: 2.199, 16384: 4.266, 32768: 8.217}
MFMA_BF16_PEAK_TFLOPS = 2500.0


def bench_layer(args, inp, dev):
    """A step is one gbla_layer_forward: the conv on the embeddings, the
    stacked projections (bf16 MFMA GEMM) and the attention core."""
    import torch
    from paper_2606_07317_amd import gbla, inputs
    w = inp.workload
    base = inputs.layer_device_tensors(inp, dev)
    shape = gbla.layer_shape(base["x"], base["conv_x"], w.heads, w.head_dim, w.eps)
    ws = torch.empty(gbla.layer_workspace_bytes(shape), dtype=torch.uint8, device=dev)
    per_set = base["x"].numel() * 2 + base["x"].shape[0] * w.heads * base["x"].shape[1] * w.head_dim * 4
    nsets = args.sets or max(2, -(-(1 << 30) // per_set) + 1)
    sets = []
    for i in range(nsets):
        x = base["x"].clone() if i else base["x"]
        out = torch.empty((w.batch, w.heads, w.seqlen, w.head_dim), dtype=torch.float32, device=dev)
        sets.append((x, out))

    def step(i):
        x, out = sets[i % nsets]
        gbla.layer_forward(x, base["conv_x"], base["w_proj"], base["gamma"], eps=w.eps,
                           workspace=ws, out=out)

    for i in range(args.warmup):
        step(i)
    stream = torch.cuda.current_stream()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record(stream)
    for i in range(args.steps):
        step(i)
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = ev0.elapsed_time(ev1) / args.steps
    # the conv pass, the projection GEMM and the gate-logit pass, timed live on
    # the same stream
    pairs = []
    for i in range(min(args.steps, 50)):
        x, _ = sets[i % nsets]
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        gbla.layer_project(x, base["conv_x"], base["w_proj"], w.heads, w.head_dim, workspace=ws)
        b.record(stream)
        pairs.append((a, b))
    torch.cuda.synchronize()
    proj_ms = statistics.mean(a.elapsed_time(b) for a, b in pairs)
    tokens = w.batch * w.seqlen
    flops = 2.0 * tokens * w.d_model * w.heads * (4 * w.head_dim + 1)
    tfl = flops / (proj_ms * 1e-3) / 1e12
    res = {"metric": "GBLA layer forward latency from the embeddings (Table 5 shape)",
           "value": ms, "unit": "ms/layer", "n_gpus": 1, "steps": args.steps,
           "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": False,
           "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
           "config": {"workload": w.name, "B": w.batch, "L": w.seqlen, "d_model": w.d_model,
                      "H": w.heads, "d": w.head_dim, "conv_width": w.conv_width,
                      "tokens_per_s": tokens / (ms * 1e-3), "rotating_sets": nsets,
                      "paper_h100_ms": PAPER_H100_LAYER_MS.get(w.seqlen),
                      "wall_s": round(wall, 4)},
           "roofline": {"bound": "mfma", "kernel": "conv_x_kernel+proj_kernel+gate_kernel",
                        "achieved": round(tfl, 1),
                        "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                        "frac": round(tfl / MFMA_BF16_PEAK_TFLOPS, 4), "avg_launch_ms": proj_ms,
                        "traffic": None}}
    print(json.dumps(res), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=400)
    ap.add_argument("--warmup", type=int, default=40)
    ap.add_argument("--workload", default=None)
    ap.add_argument("--sets", type=int, default=0, help="rotated input sets (0: enough for 1 GiB)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--pass", dest="which", choices=("forward", "backward", "layer"),
                    default="forward",
                    help="forward (the headline metric), the backward pass (gbla_backward) or "
                         "the full layer from the embeddings (gbla_layer_forward; --workload "
                         "layer_b8_n2048 or layer_b8_n32768)")
    ap.add_argument("--switches", choices=tuple(SWITCHES), default="none",
                    help="forward pass only: the ablation switches of the timed forward "
                         "(removed inputs are not passed)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only copy 256 MiB device-to-device --steps times (reference for "
                         "rocprofv3 FETCH_SIZE / WRITE_SIZE scaling)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2606_07317_amd import gbla, inputs

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    dev = torch.device("cuda:0")
    if args.calibrate_copy:
        n = 1 << 26  # 64 Mi floats = 256 MiB each way
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(args.steps):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibrate_copy_bytes_each_way": 4 * n, "copies": args.steps}))
        return
    if args.which == "layer":
        return bench_layer(args, inputs.make_layer_inputs(
            inputs.LAYER_WORKLOADS[args.workload or "layer_b8_n32768"]), dev)
    wname = args.workload or inputs.THROUGHPUT_WORKLOAD
    if args.which == "backward":
        return bench_backward(args, inputs.make_inputs(wname), dev)
    inp = inputs.make_inputs(wname)
    w = inp.workload
    base = inputs.device_tensors(inp, dev)
    per_set = sum(base[n].numel() * base[n].element_size() for n in ("q", "k", "v", "a", "r"))
    per_set += base["q"].numel() * 4
    nsets = args.sets or max(2, -(-(1 << 30) // per_set) + 1)
    sets = []
    for i in range(nsets):
        t = {n: (base[n].clone() if isinstance(base[n], torch.Tensor) else base[n]) for n in base}
        t["out"] = torch.empty(base["q"].shape, dtype=torch.float32, device=dev)
        sets.append(t)
    shape = gbla.make_shape(base["q"], base["conv_w"], inp.eps, base["cu_seqlens"], base["max_seqlen"])
    ws = gbla.alloc_workspace(shape, dev)
    flag_name, keep_gate, keep_conv, keep_norm = SWITCHES[args.switches]
    flags = getattr(gbla, flag_name) if flag_name else 0

    def used(t):
        """a, r, taps, gamma of a set, None where a switch removes them."""
        return (t["a"] if keep_gate else None, t["r"] if keep_norm else None,
                t["conv_w"] if keep_conv else None, t["gamma"] if keep_norm else None)

    def step(i):
        t = sets[i % nsets]
        a, r, cw, gm = used(t)
        gbla.forward(t["q"], t["k"], t["v"], a, r, cw, gm, eps=inp.eps,
                     cu_seqlens=t["cu_seqlens"], max_seqlen=t["max_seqlen"], workspace=ws,
                     out=t["out"], flags=flags)

    # The side measurements run first, so that the GPU has left its idle
    # clocks before the timed loop starts.
    stream = torch.cuda.current_stream()
    # Distribution of single forwards (events around each call, same rotation)
    n_meas = min(max(args.steps, 100), 200)
    fwd_ev = []
    for i in range(n_meas):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        step(i)
        b.record(stream)
        fwd_ev.append((a, b))
    torch.cuda.synchronize()
    fwd_us = sorted(1e3 * a.elapsed_time(b) for a, b in fwd_ev)
    pct = {"p10": fwd_us[len(fwd_us) // 10], "p50": statistics.median(fwd_us),
           "p90": fwd_us[(9 * len(fwd_us)) // 10]}

    # Practical ceiling: a device-to-device copy moving the forward's
    # algorithmic bytes (half read, half written), over as many rotating
    # buffers as the forward uses, timed the same way.
    half = algorithmic_bytes(inp, "forward", keep_gate, keep_norm) // 2 // 4
    bufs = [torch.empty(half, dtype=torch.float32, device=dev) for _ in range(nsets + 1)]
    for b in bufs:
        b.fill_(1.0)
    cp = []
    for i in range(n_meas):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        bufs[(i + 1) % len(bufs)].copy_(bufs[i % len(bufs)])
        b.record(stream)
        cp.append((a, b))
    torch.cuda.synchronize()
    copy_us = statistics.median(1e3 * a.elapsed_time(b) for a, b in cp)
    copy_gbps = 8 * half / (copy_us * 1e-6) / 1e9
    del bufs

    # The stream ceiling: gbla_stream_ceiling moves exactly the forward's
    # bytes (q, k, v, r and one logit per token read, y written) in one
    # launch with none of its arithmetic, over the same rotating sets; the
    # median of single calls, compared with the forward's (bf16 inputs only).
    ceiling_us = None
    if w.dtype == "bf16" and keep_gate and keep_norm:
        def ceil_step(i):
            t = sets[i % nsets]
            gbla.stream_ceiling(t["q"], t["k"], t["v"], t["a"], t["r"], out=t["out"])
        for i in range(args.warmup):
            ceil_step(i)
        torch.cuda.synchronize()
        ce = []
        for i in range(n_meas):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            ceil_step(i)
            b.record(stream)
            ce.append((a, b))
        torch.cuda.synchronize()
        ceiling_us = statistics.median(1e3 * a.elapsed_time(b) for a, b in ce)

    # The forward's kernels on the GPU (gbla_forward_timed: events recorded
    # before its first kernel and as its last one ends).
    fk = []
    for i in range(n_meas):
        t = sets[i % nsets]
        a_, r_, cw_, gm_ = used(t)
        ka, kb = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        ka.record(stream)
        kb.record(stream)
        gbla.forward(t["q"], t["k"], t["v"], a_, r_, cw_, gm_, eps=inp.eps,
                     cu_seqlens=t["cu_seqlens"], max_seqlen=t["max_seqlen"], workspace=ws,
                     out=t["out"], flags=flags, kernel_events=(ka, kb))
        fk.append((ka, kb))
    torch.cuda.synchronize()
    forward_gpu_us = statistics.mean(1e3 * a.elapsed_time(b) for a, b in fk)

    for i in range(args.warmup):
        step(i)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record(stream)
    for i in range(args.steps):
        step(i)
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_per_step = ev0.elapsed_time(ev1) / args.steps

    # Live per-kernel timing of the dominant stage (the readout: 2/3 of the
    # algorithmic bytes), in forward order after the state stage.  The kernel's
    # own duration comes from events that the launch itself records as the
    # kernel begins and ends (gbla_readout_timed); events recorded around the
    # call, which add the launch gaps, are reported beside it.
    pairs, calls = [], []
    for i in range(n_meas):
        t = sets[i % nsets]
        a_, r_, cw_, gm_ = used(t)
        gbla.state(t["k"], t["v"], a_, cw_, cu_seqlens=t["cu_seqlens"],
                   max_seqlen=t["max_seqlen"], workspace=ws, flags=flags)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        ka, kb = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        ka.record(stream)
        kb.record(stream)
        a.record(stream)
        gbla.readout(t["q"], r_, cw_, gm_, ws, eps=inp.eps,
                     cu_seqlens=t["cu_seqlens"], max_seqlen=t["max_seqlen"], out=t["out"],
                     kernel_events=(ka, kb), flags=flags)
        b.record(stream)
        pairs.append((ka, kb))
        calls.append((a, b))
    torch.cuda.synchronize()
    readout_ms = statistics.mean(a.elapsed_time(b) for a, b in pairs)
    readout_call_ms = statistics.mean(a.elapsed_time(b) for a, b in calls)
    ach = algorithmic_bytes(inp, "readout", keep_gate, keep_norm) / (readout_ms * 1e-3) / 1e9
    fwd_gbps = algorithmic_bytes(inp, "forward", keep_gate, keep_norm) / (ms_per_step * 1e-3) / 1e9
    # the kernel that ran: the streaming readout for bf16 slices under 2^31
    # bytes of fp32 output, the generic one otherwise
    slice_rows = inp.tokens if w.ragged else w.seqlen
    readout_kernel = ("readout_stream_kernel"
                      if w.dtype == "bf16" and slice_rows * w.head_dim * 4 < (1 << 31)
                      else "readout_kernel")

    res = {
        "metric": METRIC if w.name == inputs.THROUGHPUT_WORKLOAD else "GBLA fwd tokens/sec on " + w.name,
        "value": inp.tokens / (ms_per_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if w.dtype == "bf16" else "f32",
        "data": "synthetic",
        "config": {"workload": w.name, "B": inp.nseq, "H": w.heads, "n": w.seqlen if not w.ragged else None,
                   "tokens": inp.tokens, "d": w.head_dim, "conv_width": w.conv_width,
                   "inputs": w.dtype, "output": "f32", "rotating_sets": nsets,
                   "forward_effective_GBps": round(fwd_gbps, 1),
                   "forward_hbm_frac": round(fwd_gbps / HBM_PEAK_GBPS, 4),
                   "single_forward_us": {k: round(v, 2) for k, v in pct.items()},
                   "forward_gpu_us": round(forward_gpu_us, 2),
                   "stream_ceiling_us": round(ceiling_us, 2) if ceiling_us else None,
                   "stream_ceiling_GBps": (round(algorithmic_bytes(inp, "forward") / (ceiling_us * 1e-6) / 1e9, 1)
                                           if ceiling_us else None),
                   "forward_over_ceiling": (round(ceiling_us / pct["p50"], 4)
                                            if ceiling_us else None),
                   "copy_same_bytes_us": round(copy_us, 2),
                   "copy_same_bytes_GBps": round(copy_gbps, 1),
                   "wall_s": round(wall, 4)},
        "roofline": {"bound": "hbm", "kernel": readout_kernel, "achieved": round(ach, 1),
                     "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": round(ach / HBM_PEAK_GBPS, 4),
                     "avg_launch_ms": readout_ms,
                     "avg_call_ms": readout_call_ms,
                     "forward_achieved": round(fwd_gbps, 1),
                     "forward_frac": round(fwd_gbps / HBM_PEAK_GBPS, 4),
                     "traffic": (traffic_from_profiles(readout_kernel, w.name)
                                 if args.switches == "none" else None)},
    }
    if args.switches != "none":
        res["config"]["switches"] = args.switches
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(inp, args.cpu_seconds, keep_gate, keep_conv, keep_norm)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
