#!/usr/bin/env python3
"""Throughput of 1-bit Adam's compression-stage step on one MI355X.

One step = the whole hot path over one batch of synthetic gradients: the
worker pass of all n simulated workers (momentum, error compensation, sign
packing, per-segment scales), the chunk owners' average + recompression, and
the decompress + preconditioned update.  Inputs are resident in HBM before the
timed region.  The Adam warm-up steps that produce the frozen variance run
(untimed) during set-up.  Prints one JSON line.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0  # MI355X HBM3E, published


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def algorithmic_bytes_per_param(n, grad_bytes=4):
    """Bytes the method must move per parameter in a steady-state step, each
    input read once and each output written once (fp32 state, 1-bit
    messages).  The shared momentum is the previous step's server message
    (Algorithm 1 sets every worker's m to it), so it is read as one sign bit:
      worker pass: m's sign bit read once for all n workers, then per worker
                   g read, error state read and written, one sign bit written;
      server pass: n incoming sign bits, server error state read and written,
                   one sign bit written;
      update     : one sign bit read, x read and written, v read."""
    worker = 1 / 8 + n * (grad_bytes + 4 + 4 + 1 / 8)
    server = n / 8 + 4 + 4 + 1 / 8
    update = 1 / 8 + 4 + 4 + 4
    return worker, server, update


# The sources that decide what the kernels touch: the kernels, the plan (tile)
# construction, the shared constants and the launch shapes.
KERNEL_SOURCES = ("onebit_kernels.hip", "onebit_abi.hip", "onebit_internal.h", "onebit_grid.h")


def code_text(src):
    """C/C++ source without its comments, each run of whitespace one space:
    what the compiler sees, so that editing a comment keeps recorded counters
    valid.  String and character literals are kept as written."""
    out, i, n = [], 0, len(src)
    while i < n:
        c = src[i]
        if src.startswith("//", i):
            j = src.find("\n", i)
            i = n if j < 0 else j
            out.append(" ")
        elif src.startswith("/*", i):
            j = src.find("*/", i + 2)
            i = n if j < 0 else j + 2
            out.append(" ")
        elif c in "\"'":
            j = i + 1
            while j < n and src[j] != c:
                j += 2 if src[j] == "\\" else 1
            out.append(src[i:j + 1])
            i = j + 1
        else:
            out.append(c)
            i += 1
    return " ".join("".join(out).split())


def kernels_source_sha256():
    """Digest of the code of KERNEL_SOURCES (comments and layout aside), in
    that order."""
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2102_02888_amd", "csrc", f)) as fh:
            h.update(code_text(fh.read()).encode())
        h.update(b"\0")
    return h.hexdigest()


def server_kernel(plan):
    """The chunk owners' kernel that a whole-range call on this plan runs, by
    the rule include/onebit.h states for onebit_plan_set_server_tables' AUTO
    mode: the tables come from the workspace when those of all S segments fit
    in 32 MiB (2 KB per segment and group of 8 workers), the segments average
    4 or more tiles and tiles times groups reach 32768."""
    groups = (plan.n + 7) // 8
    tables = (plan.S * groups * 2048 <= (32 << 20) and plan.T >= 4 * plan.S
              and plan.T * groups >= 32768)
    if plan.n > 32:
        return "k_server_subblocks" if tables else "k_server_split"
    return "k_server_shared" if tables else "k_server_pass<%d>" % min(4, groups)


def measured_traffic(workload, kernel):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 counter
    summary (FETCH_SIZE + WRITE_SIZE, each calibrated on a plain device copy),
    or None when there is none for this workload or the kernel source has
    changed since the counters were taken."""
    import hashlib
    import re
    path = os.path.join(ROOT, "profiles", "pmc_traffic_%s.md" % workload)
    if not os.path.exists(path):
        return None
    m = re.search(r"```json\n(.*?)\n```", open(path).read(), re.S)
    if not m:
        return None
    info = json.loads(m.group(1))
    if kernels_source_sha256() != info.get("kernels_source_sha256"):
        return None
    k = info["kernels"].get(kernel)
    return None if k is None else k["traffic_bytes"]


def _host_segment(st, plan, q, b=None, e=None):
    """Host copies of one segment's device state (or of its elements [b, e)),
    as the oracle takes them."""
    import numpy as np
    if b is None:
        b, e = int(plan.seg_begin[q]), int(plan.seg_end[q])
    ln, n = e - b, st.n_local
    nw = (ln + 63) // 64
    return {"len": ln, "m": st.m[b:e].cpu().numpy().copy(), "x": st.x[b:e].cpu().numpy().copy(),
            "v": st.v[b:e].cpu().numpy().copy(), "dbar": st.server_err[b:e].cpu().numpy().copy(),
            "g": st.grads[:, b:e].cpu().numpy().copy(),
            "delta": st.worker_err[:, b:e].cpu().numpy().copy(),
            "wbits": np.zeros((n, nw), np.uint64), "wscales": np.zeros(n, np.float32),
            "sbits": np.zeros(nw, np.uint64), "z": np.zeros(ln, np.float32)}


def _oracle_segment(sd, wl):
    """One compression step of the oracle over one segment: every worker's
    pass, the owner's average and recompression, and the update."""
    import oracle
    ln, n = sd["len"], sd["g"].shape[0]
    nw = sd["sbits"].shape[0]
    for i in range(n):
        sd["wscales"][i] = oracle.worker_segment(0, ln, wl.beta1, sd["m"], sd["g"][i],
                                                 sd["delta"][i], sd["wbits"][i], sd["z"])
    s = oracle.server_segment(0, ln, n, sd["wbits"].reshape(-1), nw, sd["wscales"], 1,
                              sd["dbar"], sd["sbits"], sd["z"])
    oracle.update_segment(0, ln, sd["sbits"], s, wl.lr, wl.eps, sd["x"], sd["m"], sd["v"])


def _cpu_model():
    """The host CPU's model name from /proc/cpuinfo, or None."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def cpu_baseline(st, plan, wl, target_s=10.0, threads=None, threaded_s=6.0):
    """Times the oracle on the host cores over whole segments of the
    workload (each segment: every worker's pass, the owner's average and
    recompression, and the update; host copies of the device state).

    Reported value: `threads` threads (the process's CPU share, at most 16),
    each looping over its own pieces of chunk 0 for about `threaded_s`
    seconds; the oracle releases the GIL, so the threads run in parallel.
    Segments longer than chunk 0's length / (4 threads) are cut into
    64-aligned slices, each run through the oracle's segment step (the same
    per-element work; only the scale is taken over the slice).
    Also reported: one thread over up to three whole segments."""
    import threading

    segs = [q for q in (0, plan.S - 1, plan.S // 2) if plan.seg_end[q] > plan.seg_begin[q]]
    done1, spent1, used = 0, 0.0, []
    for q in segs:
        sd = _host_segment(st, plan, q)
        t0 = time.perf_counter()
        _oracle_segment(sd, wl)
        spent1 += time.perf_counter() - t0
        done1 += sd["len"]
        used.append(q)
        del sd
        if spent1 >= target_s:
            break
    single = {"value": done1 / spent1, "cores": 1,
              "sample": "%d whole segment(s) %s of %d (%d params), %.1f s"
                        % (len(used), used, plan.S, done1, spent1)}

    if threads is None:
        threads = max(1, min(16, len(os.sched_getaffinity(0))))
    chunk0 = [q for q in range(0, plan.S, plan.n) if plan.seg_end[q] > plan.seg_begin[q]]
    total = sum(int(plan.seg_end[q] - plan.seg_begin[q]) for q in chunk0)
    piece = max(64, (total // (4 * threads)) // 64 * 64)
    data = []
    for q in chunk0:
        for b in range(int(plan.seg_begin[q]), int(plan.seg_end[q]), piece):
            data.append(_host_segment(st, plan, q, b, min(b + piece, int(plan.seg_end[q]))))
    data.sort(key=lambda sd: -sd["len"])
    share = [[] for _ in range(threads)]
    load = [0] * threads
    for sd in data:  # largest first onto the least loaded thread
        k = load.index(min(load))
        share[k].append(sd)
        load[k] += sd["len"]
    counts = [0] * threads
    start = threading.Barrier(threads + 1)
    t_end = [0.0]

    def run(k):
        start.wait()
        while share[k] and time.perf_counter() < t_end[0]:
            for sd in share[k]:
                _oracle_segment(sd, wl)
                counts[k] += sd["len"]
                if time.perf_counter() >= t_end[0]:
                    break

    pool = [threading.Thread(target=run, args=(k,)) for k in range(threads)]
    for th in pool:
        th.start()
    t0 = time.perf_counter()
    t_end[0] = t0 + threaded_s
    start.wait()
    for th in pool:
        th.join()
    wall = time.perf_counter() - t0
    return {"value": sum(counts) / wall, "unit": "params/s", "cores": threads, "kind": "oracle",
            "cpu_model": _cpu_model(),
            "sample": "%d threads looping over chunk 0 (%d segment(s), %d params, in %d "
                      "pieces of at most %d; all %d workers' passes, the chunk owner's average "
                      "and recompression, and the update) for %.1f s: %d params"
                      % (threads, len(chunk0), total, len(data), piece, st.n_local, wall,
                         sum(counts)),
            "single_thread": single}


def hbm_probe(dev, nbytes=2 << 30, reps=10):
    """Achievable HBM bandwidth of two plain streaming kernels of torch: a
    device copy (one read stream, one write stream) and an elementwise add
    (two read streams, one write stream: the read/write mix of the worker
    pass), each over `nbytes` per operand."""
    import torch
    out = {}
    a = torch.empty(nbytes // 4, dtype=torch.float32, device=dev)
    b = torch.empty_like(a)
    c = torch.empty_like(a)
    a.normal_()
    b.normal_()
    for name, fn, streams in (("copy_1r1w", lambda: c.copy_(a), 2),
                              ("add_2r1w", lambda: torch.add(a, b, out=c), 3)):
        fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        out[name] = streams * nbytes / (ms * 1e-3) / 1e9
    del a, b, c
    return out


def hbm_ceilings(dev, nbytes=2 << 30):
    """Best rates of the hand-written streaming kernels (the passes' 128-bit
    non-temporal buffer loads and stores, XCD-contiguous grids) over `nbytes`
    per stream: one stream read, a copy, and two streams read with the second
    rewritten in place (the worker pass's mix), each over 1, 2 or 4 KB of
    each stream in flight per wave and 2 to 8 four-wave workgroups per CU.
    None when the probe library is not built."""
    import torch
    try:
        from paper_2102_02888_amd import hbm_probe
        hbm_probe.lib()
    except ImportError as e:
        log("no HBM streaming ceilings: %s" % e)
        return None
    a = torch.zeros(nbytes // 4, dtype=torch.float32, device=dev)
    b = torch.zeros_like(a)
    sink = torch.zeros(1, dtype=torch.float32, device=dev)
    rows = hbm_probe.stream_table(a, b, sink, torch.cuda.current_stream(dev))
    del a, b, sink
    out = hbm_probe.best(rows)
    out["source"] = ("paper_2102_02888_amd/csrc/hbm_probe.hip over %d MiB streams, best of %d "
                     "cases per mix" % (nbytes >> 20, len(hbm_probe.CASES)))
    return out


def bench_variant(args, wl, plan, st, gbytes):
    """Times one of the paper's comparison variants on the same workload."""
    import torch
    n, d = wl.n, plan.d
    if args.variant == "uncompressed":
        step = lambda k: st.step_uncompressed(wl.lr, wl.beta1, wl.eps)
        bytes_pp = n * gbytes + 4 + 4 + 4 + 4 + 4
        name = "1-bit Adam (32-bits) step: momenta averaged uncompressed, variance frozen"
    else:
        t0 = wl.warmup_steps
        step = lambda k: st.step_naive(wl.lr, wl.beta1, wl.beta2, wl.eps, t0 + k + 1)
        bytes_pp = (1 / 8 + n * (gbytes + 8 + 1 / 8)) + (n / 8 + 8 + 1 / 8) + (1 / 8 + 24)
        name = "Adam(1-bit Naive) step: gradient compressed, Adam on the decoded average"
    for k in range(args.warmup):
        step(k)
    torch.cuda.synchronize()
    t0w = time.perf_counter()
    for k in range(args.steps):
        step(args.warmup + k)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0w) * 1e3 / args.steps
    print(json.dumps({
        "metric": "%s params/sec, %s" % (args.variant, wl.name), "value": d / (ms * 1e-3),
        "unit": "params/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32", "data": "synthetic",
        "config": {"workload": wl.name, "d": d, "n_workers": n, "variant": args.variant,
                   "grad_dtype": args.grad_dtype, "description": name},
        "bytes_per_param": bytes_pp,
        "step_hbm_gbps_algorithmic": bytes_pp * d / (ms * 1e-3) / 1e9}), flush=True)


def bench_share(args, wl):
    """One GPU's share of an n-worker step: the local worker's pass over all
    d, the owner of one chunk reducing n incoming packed chunks (synthetic,
    seeded), and the update over all d with the gathered message."""
    import torch

    import paper_2102_02888_amd as ob
    import synth
    dev = torch.device("cuda:0")
    n, j = wl.n, wl.server_chunk
    plan = ob.Plan(wl.numel, n)
    st = ob.State(plan, dev, n_local=wl.n_local)
    scale_vec = torch.from_numpy(synth.grad_scale_per_element(wl, plan.D, plan.tensor_off)).to(dev)
    st.x.copy_(synth.device_params(wl, plan.D, dev))
    for t in range(1, wl.warmup_steps + 1):
        synth.device_grads(wl, plan.D, plan.tensor_off, t, st.grads, scale_vec)
        st.warmup(wl.lr, wl.beta1, wl.beta2, wl.eps, t)
    synth.device_grads(wl, plan.D, plan.tensor_off, wl.warmup_steps + 1, st.grads, scale_vec)
    b0, e0 = int(plan.seg_begin[j]), int(plan.seg_end[j])
    cw0, cw1 = b0 // 64, (e0 + 63) // 64
    recv_bits, recv_scales = synth.device_bits_and_scales(n, cw1 - cw0, wl.seed_incoming, dev)
    gath_bits, gath_scales = synth.device_bits_and_scales(1, plan.W, wl.seed_incoming + 1, dev)
    st.server_bits.copy_(gath_bits[0])
    st.server_scales.fill_(float(gath_scales[0]))
    st.server_scales[j] = 0.0
    torch.cuda.synchronize()

    def one_step(ev=None, first=False):
        if ev:
            ev[0].record()
        if first:
            ob.onebit_worker_compress(plan, st.m, st.grads, st.worker_err, st.worker_bits,
                                      st.worker_scales, wl.beta1, st.workspace)
        else:
            ob.onebit_worker_compress(plan, None, st.grads, st.worker_err, st.worker_bits,
                                      st.worker_scales, wl.beta1, st.workspace,
                                      m_bits=st.server_bits, m_scales=st.server_scales)
        if ev:
            ev[1].record()
        ob.onebit_server_reduce_compress(plan, j, j + 1, recv_bits, recv_scales, st.server_err,
                                         st.server_bits, st.server_scales, st.workspace,
                                         bits_word_base=cw0, scales_seg_base=j, scales_ld=1)
        if ev:
            ev[2].record()
        ob.onebit_decompress_update(plan, st.server_bits, st.server_scales, st.x, None, st.v,
                                    wl.lr, wl.eps)
        if ev:
            ev[3].record()

    one_step(first=True)
    for _ in range(args.warmup):
        one_step()
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        one_step(events[k])
    torch.cuda.synchronize()
    ms_step = (time.perf_counter() - t0) * 1e3 / args.steps
    part_ms = [sum(ev[i].elapsed_time(ev[i + 1]) for ev in events) / args.steps for i in range(3)]
    d = plan.d
    chunk = e0 - b0
    worker_b = d * (1 / 8 + 12.125)
    server_b = chunk * (n / 8 + 8.125)
    update_b = d * 12.125
    step_b = worker_b + server_b + update_b
    result = {
        "metric": "compression-phase step params/sec (one GPU's share of a %d-worker step)" % n,
        "value": d / (ms_step * 1e-3), "unit": "params/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_step, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": wl.name, "d": d, "n_workers": n, "n_local": wl.n_local,
                   "server_chunk": j, "chunk_len": chunk, "description": wl.description},
        "step_hbm_gbps_algorithmic": step_b / (ms_step * 1e-3) / 1e9,
        "step_frac_of_peak": step_b / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBPS,
        "kernel_ms": {"worker_compress": part_ms[0], "server_reduce_compress": part_ms[1],
                      "decompress_update": part_ms[2], "sum": sum(part_ms)},
        "kernel_gbps_algorithmic": {"worker_compress": worker_b / (part_ms[0] * 1e-3) / 1e9,
                                    "server_reduce_compress": server_b / (part_ms[1] * 1e-3) / 1e9,
                                    "decompress_update": update_b / (part_ms[2] * 1e-3) / 1e9},
    }
    print(json.dumps(result), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="bert_large",
                    choices=["tiny", "bert_base", "bert_large", "stress", "share256"])
    ap.add_argument("--grad-dtype", default="f32", choices=["f32", "bf16", "f16"],
                    help="gradient element type (16-bit gradients are widened exactly)")
    ap.add_argument("--variant", default="onebit", choices=["onebit", "uncompressed", "naive"],
                    help="1-bit Adam (default), or one of the paper's comparison variants: "
                         "'1-bit Adam (32-bits)' (uncompressed) or 'Adam(1-bit Naive)'")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-probe", action="store_true")
    ap.add_argument("--graph", action="store_true",
                    help="also time the step replayed from a captured HIP graph")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: the compressed exchange is simulated in one GPU's "
              "HBM and no collective is called, so --gpus %d is not supported (use --gpus 1)"
              % args.gpus, file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2102_02888_amd as ob
    import synth

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    wl = synth.get(args.workload)
    if wl.n_local is not None:
        return bench_share(args, wl)
    n = wl.n
    plan = ob.Plan(wl.numel, n)
    log("workload %s: d=%d D=%d n=%d segments=%d tiles=%d" % (wl.name, plan.d, plan.D, n,
                                                              plan.S, plan.T))
    gdt = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}[args.grad_dtype]
    gbytes = {"f32": 4, "bf16": 2, "f16": 2}[args.grad_dtype]
    st = ob.State(plan, dev, grad_dtype=gdt)
    scale_vec = torch.from_numpy(synth.grad_scale_per_element(wl, plan.D, plan.tensor_off)).to(dev)
    st.x.copy_(synth.device_params(wl, plan.D, dev))

    # Adam warm-up (untimed set-up): produces m and the frozen variance v.
    warm_ms = []
    for t in range(1, wl.warmup_steps + 1):
        synth.device_grads(wl, plan.D, plan.tensor_off, t, st.grads, scale_vec)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        st.warmup(wl.lr, wl.beta1, wl.beta2, wl.eps, t)
        e1.record()
        torch.cuda.synchronize()
        warm_ms.append(e0.elapsed_time(e1))
    synth.device_grads(wl, plan.D, plan.tensor_off, wl.warmup_steps + 1, st.grads, scale_vec)
    torch.cuda.synchronize()

    if args.variant != "onebit":
        return bench_variant(args, wl, plan, st, gbytes)

    # The timed step is State.step: the fused onebit_step (worker pass, its
    # scale finalize, the chunk owners' pass, its finalize, the update), in
    # its events form, which also marks the launch stream before the worker
    # pass, before the owners' pass, before the update and after it.
    st.step(wl.lr, wl.beta1, wl.eps)  # untimed: the step that leaves the warm-up's fp32 m
    assert st.momentum_is_packed()
    for _ in range(args.warmup):
        st.step(wl.lr, wl.beta1, wl.eps)
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    for ev in events:  # creates each HIP event; the step re-records them on its stream
        for e in ev:
            e.record()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        st.step(wl.lr, wl.beta1, wl.eps, events=events[k])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = wall * 1e3 / args.steps
    part_ms = [sum(ev[j].elapsed_time(ev[j + 1]) for ev in events) / args.steps
               for j in range(3)]
    gpu_step_ms = sum(part_ms)
    per_step = sorted(ev[0].elapsed_time(ev[3]) for ev in events)
    graph_ms = None
    if args.graph:
        # the same packed-momentum step captured once and replayed: one launch
        # per step instead of five (worker, scales, owners, scales, update)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            st.step(wl.lr, wl.beta1, wl.eps)
        for _ in range(args.warmup):
            graph.replay()
        gev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(args.steps)]
        torch.cuda.synchronize()
        for k in range(args.steps):
            gev[k][0].record()
            graph.replay()
            gev[k][1].record()
        torch.cuda.synchronize()
        gt = sorted(a.elapsed_time(b) for a, b in gev)
        graph_ms = {"median": gt[len(gt) // 2], "min": gt[0], "max": gt[-1]}

    bw, bs, bu = algorithmic_bytes_per_param(n, gbytes)
    gname = {"f32": "GradF32", "bf16": "GradBF16", "f16": "GradF16"}[args.grad_dtype]
    # the first warm-up step is a cold start; later ones are timed
    warm_avg = sum(warm_ms[1:]) / (len(warm_ms) - 1) if len(warm_ms) > 1 else None
    d = plan.d
    step_bytes = d * (bw + bs + bu)
    worker_bytes = d * bw
    achieved = worker_bytes / (part_ms[0] * 1e-3) / 1e9
    # the same pass counted with m read as an fp32 value (4 B) instead of a bit
    bw_fp32_m = 4 + n * (gbytes + 4 + 4 + 1 / 8)
    result = {
        "metric": ("compression-phase step params/sec and achieved HBM GB/s vs peak, BERT-Large"
                   if wl.name == "bert_large" else
                   "compression-phase step params/sec and achieved HBM GB/s vs peak, %s" % wl.name),
        "value": d / (ms_step * 1e-3),
        "unit": "params/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": wl.name, "d": d, "n_workers": n, "segments": plan.S,
                   "grad_dtype": args.grad_dtype,
                   "tensors_shaped": len(wl.grad_scale_ranges or wl.numel),
                   "adam_warmup_steps": wl.warmup_steps, "description": wl.description},
        "step_hbm_gbps_algorithmic": step_bytes / (ms_step * 1e-3) / 1e9,
        "step_frac_of_peak": step_bytes / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBPS,
        "bytes_per_param": {"worker": bw, "server": bs, "update": bu},
        "timed_call": "State.step -> onebit_step (onebit_step_events: the same launches "
                      "with four event marks)",
        "kernel_ms": {"worker_compress": part_ms[0], "server_reduce_compress": part_ms[1],
                      "decompress_update": part_ms[2], "sum": gpu_step_ms},
        "gpu_step_ms": {"median": per_step[len(per_step) // 2], "min": per_step[0],
                        "max": per_step[-1]},
        "warmup_adam_step_ms": warm_avg,
        "graph_step_ms": graph_ms,
        "warmup_step_ms": ({"median": sorted(warm_ms[1:])[(len(warm_ms) - 1) // 2],
                            "min": min(warm_ms[1:]), "max": max(warm_ms[1:])}
                           if len(warm_ms) > 1 else None),
        "roofline": {"bound": "hbm",
                     "kernel": "worker_compress (k_worker_pass<true, %s>: packed momentum, %s "
                               "gradients)" % (gname, args.grad_dtype),
                     "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBPS,
                     "traffic": measured_traffic(wl.name, "k_worker_pass<true, %s>" % gname),
                     "algorithmic_bytes_per_launch": worker_bytes,
                     "bytes_per_param": bw,
                     "bytes_per_param_rule": "m read as its sign bit (packed momentum): "
                                             "1/8 + n*(%d g + 4 err in + 4 err out + 1/8 bit)"
                                             % gbytes,
                     "bytes_per_param_fp32_m": bw_fp32_m,
                     "frac_fp32_m": (bw_fp32_m * d / (part_ms[0] * 1e-3) / 1e9
                                     / HBM_PEAK_GBPS),
                     "ms": part_ms[0],
                     "timed": "HIP events on the launch stream before and after the worker "
                              "pass (k_worker_pass and its scale finalize) of each timed "
                              "onebit_step, averaged over the timed steps"},
        "kernels": {name: {"ms": ms, "algorithmic_bytes": nbytes,
                           "gbps": nbytes / (ms * 1e-3) / 1e9,
                           "frac": nbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBPS,
                           "traffic": measured_traffic(wl.name, kname)}
                    for name, ms, nbytes, kname in (
                        ("worker_compress", part_ms[0], worker_bytes,
                         "k_worker_pass<true, %s>" % gname),
                        ("server_reduce_compress", part_ms[1], d * bs,
                         server_kernel(plan)),
                        ("decompress_update", part_ms[2], d * bu, "k_update"),
                        ("warmup_adam_step", warm_avg, d * (n * gbytes + 24),
                         "k_warmup<%s>" % gname))
                    if ms},
    }
    if not args.no_probe:
        del events
        result["hbm_probe_gbps"] = hbm_probe(dev)
        ceil = hbm_ceilings(dev)
        result["hbm_ceiling_gbps"] = ceil
        if ceil is not None:
            # the worker pass reads two streams and rewrites the second: the `mix`
            result["roofline"]["measured_mix_ceiling"] = {
                "gbps": ceil["mix"]["gbps"],
                "frac": result["roofline"]["achieved"] / ceil["mix"]["gbps"]}
    if not args.no_cpu_baseline:
        log("timing the oracle on sampled segments ...")
        result["cpu_baseline"] = cpu_baseline(st, plan, wl)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
