#!/usr/bin/env python3
"""Benchmark of the M+Adam optimizer step on one MI355X.

A step is one madd_multi_tensor_step call over the whole parameter list (one
kernel launch for a single-format list): read weight codes, gradients and the
three fp32 moments, update, round the weights back with stochastic rounding,
write back.  Default workload: the Llama-7B-shaped list (291 tensors,
6,738,415,616 parameters, bf16 weights, fp32 gradients and m / v / v_e),
all resident in HBM before timing starts, in flat per-role buffers (weights,
gradients, m, v, v_e each one allocation, tensors as views).  Gradients are
synthetic: for the 7B list the gradient buffer is filled anew on the device
from each step's seeds before the step (outside the timed events; each step
is bracketed by its own pair of events on the launching stream); the smaller
lists cycle through up to eight sets made up front, with the steps queued
back to back behind a short GPU-side delay and timed by one pair of events
around them, so that the events time the GPU alone.

Prints one JSON line with optimizer-step throughput (Gparam/s), the achieved
HBM bandwidth of the step kernel against the 8 TB/s peak, and the CPU oracle
timed on a bounded sample on this host, on all of the process's cores (up
to 16) and on one thread.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "optimizer-step Gparams/s + achieved HBM GB/s (% of peak), 7B-shaped set"
HBM_PEAK_GBS = 8000.0
KERNEL_SRC = os.path.join(ROOT, "paper_2607_10611_amd", "csrc", "madd.hip")
PMC_SUMMARY = os.path.join(ROOT, "profiles", "madd_step_kernel_llama7b_bf16_sr_pmc.md")

WBYTES = {"bf16": 2, "e4m3": 1, "e5m2": 1, "mxfp4": 0.5, "nvfp4": 0.5, "nvfp4_current": 0.5}
# linear-layer storage of the low-precision master settings
LOW_MASTER = {"fp8-master": "e4m3", "fp4-master": "mxfp4", "nvfp4-master": "nvfp4",
              "nvfp4cs-master": "nvfp4_current"}
SBYTES = {"fp32": 4, "bf16": 2, "bf16-sr": 2}


def bytes_per_param(wfmt: str, sfmt: str) -> float:
    """Algorithmic bytes: read w, g (fp32), m, v, v_e; write w, m, v, v_e."""
    return 2 * WBYTES[wfmt] + 4 + 6 * SBYTES[sfmt]


def algorithmic_bytes(sizes, plan, sfmt: str) -> float:
    """Bytes one step over a tensor list must move (the method's bytes):
    every array read and written once, plus per tensor its bf16 compute copy
    (written) and its block scales (read and written: FP16 per 128 elements
    for FP8, E8M0 per 32 for MXFP4, E4M3 per 16 for NVFP4, whose fp32 tensor
    scale is read, and with current scaling also written).
    `plan` holds (weight format, block-scaled, compute copy) per tensor."""
    total = 0.0
    for n, (wf, blk, cp) in zip(sizes, plan):
        total += n * bytes_per_param(wf, sfmt) + (n * 2 if cp else 0)
        if blk:
            total += {"mxfp4": (n // 32) * 2, "nvfp4": (n // 16) * 2 + 4,
                      "nvfp4_current": (n // 16) * 2 + 8}.get(wf, (n // 128) * 4)
    return total


def scratch_bytes(sizes, plan) -> float:
    """Bytes the two-pass NVFP4 current-scaling step moves beyond the
    method's: w' written over the fp32 gradient by pass 1 and read back by
    pass 2 (8 B per element), and per tensor the amax word (cleared, folded
    into, read: 12 B)."""
    return sum(8 * n + 12 for n, (wf, blk, _) in zip(sizes, plan) if wf == "nvfp4_current")

WORKLOAD_NAMES = {
    "c5": "llama-7b-shaped list (32 layers, d=4096, SwiGLU 11008, vocab 32000)",
    "c3": "llama-1.1b-shaped list (22 layers, d=2048, GQA 32/4, SwiGLU 5632, vocab 32000)",
    "c4": "llama-1.1b-shaped list in fp8 e4m3",
    "c2": "gpt2-small-shaped list (12 layers, d=768, vocab 50257)",
    "c1": "one 1024x1024 bf16 tensor (33.6 MB per step: cache-resident, a latency figure)",
}


def log(msg: str):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def kernel_sha() -> str:
    """Hash of the kernel source's code: comments and blank lines stripped, so
    that documentation edits do not invalidate a counter summary."""
    src = open(KERNEL_SRC).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    src = re.sub(r"//[^\n]*", "", src)
    code = "\n".join(line.rstrip() for line in src.splitlines() if line.strip())
    return hashlib.sha256(code.encode()).hexdigest()


def traffic_from_profile():
    """HBM bytes per launch from the committed rocprofv3 counter summary, or
    None when it is missing or was taken on a different kernel source."""
    if not os.path.exists(PMC_SUMMARY):
        return None
    text = open(PMC_SUMMARY).read()
    sha = re.search(r"kernel_code_sha256:\s*([0-9a-f]{64})", text)
    val = re.search(r"traffic_bytes_per_launch:\s*([0-9.eE+]+)", text)
    if not sha or not val or sha.group(1) != kernel_sha():
        return None
    return float(val.group(1))


def cpu_threads() -> int:
    """Host threads for the oracle: this process's CPU set, at most 16 (one
    GPU's share of the host)."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(n, 16))


def cpu_baseline(cfg: str, sample: int, steps: int, sfmt: str = "fp32", threads: int = 1,
                 seconds: float = 10.0) -> dict:
    """The CPU oracle on a bounded sample of the workload: the first `sample`
    elements of the list, stepped until `seconds` have passed (at least two
    steps), cycling through `steps` pre-generated gradient sets.  With several
    threads each runs the unchanged oracle on a contiguous index range (the
    step is elementwise and its draws are keyed by global index, so the split
    changes no result)."""
    from concurrent.futures import ThreadPoolExecutor

    import numpy as np

    import oracle
    from paper_2607_10611_amd import workloads as W

    specs = W.specs(cfg)
    wfmt = W.CONFIGS[cfg]["wfmt"]
    sample = min(sample, W.total_params(cfg))
    xs, gs, left = [], [], sample
    for i, s in enumerate(specs):
        k = min(left, s.numel)
        xs.append(W.init_fp32(cfg, i, k))
        gs.append([W.grad_fp32(cfg, i, t, k) for t in range(1, steps + 1)])
        left -= k
        if left == 0:
            break
    codes = oracle.encode_array(wfmt, np.concatenate(xs))
    grads = [np.concatenate([g[t] for g in gs]) for t in range(steps)]
    if sample >= 1 << 27:
        log(f"oracle inputs ready: {sample:,} parameters, {steps} gradient sets")
    m, v, ve = (np.zeros(sample, np.float32 if sfmt == "fp32" else np.uint16) for _ in range(3))
    bounds = [(sample * k // threads) // 8 * 8 for k in range(threads)] + [sample]

    def part(k, t, h):
        lo, hi = bounds[k], bounds[k + 1]
        oracle.step(wfmt, codes[lo:hi], grads[t - 1][lo:hi], m[lo:hi], v[lo:hi], ve[lo:hi], h,
                    sfmt=sfmt, index_base=lo)

    with ThreadPoolExecutor(threads) as ex:
        t0 = time.perf_counter()
        done, dt = 0, 0.0
        while done < 2 or dt < seconds:
            done += 1
            h = W.hparams(cfg, step=done)
            list(ex.map(lambda k: part(k, (done - 1) % steps + 1, h), range(threads)))
            dt = time.perf_counter() - t0
            if sample >= 1 << 27:
                log(f"oracle step {done} done ({dt:.1f} s)")
    return {"value": sample * done / dt / 1e9, "unit": "Gparam/s", "cores": threads,
            "kind": "oracle",
            "sample": f"first {sample:,} parameters of the list, {done} steps cycling "
                      f"{steps} gradient sets ({dt:.1f} s on {threads} thread(s), scalar C, "
                      "one contiguous index range per thread)",
            "host": host_cpu()}


def cpu_full_configs(threads: int) -> dict:
    """The oracle on whole lists: the 1024x1024 tensor, GPT-2-small and
    Llama-1.1B (every parameter; fp32 moments; two steps with their own
    gradient sets), on one thread and on `threads` threads."""
    from paper_2607_10611_amd import workloads as W

    out = {"kind": "oracle", "unit": "Gparam/s", "host": host_cpu(), "configs": []}
    for cfg in ("c1", "c2", "c3"):
        n = W.total_params(cfg)
        for th in sorted({1, threads}):
            log(f"oracle on the whole {cfg} list ({n:,} parameters), {th} thread(s)")
            r = cpu_baseline(cfg, n, 2, "fp32", th, seconds=0.0)
            out["configs"].append({"config": cfg, "workload": WORKLOAD_NAMES[cfg], "params": n,
                                   "cores": th, "value": r["value"], "sample": r["sample"]})
    return out


def host_cpu() -> str:
    """The host CPU model and how many logical CPUs this process may use."""
    model = "unknown CPU"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return f"{model}, {n} logical CPUs available to the process"


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="c5", choices=sorted(WORKLOAD_NAMES))
    ap.add_argument("--states", default="fp32", choices=["fp32", "bf16", "bf16-sr"],
                    help="storage of m, v, v_e (bf16: the paper's optimizer-state precision, "
                         "rounded to nearest; bf16-sr: rounded stochastically)")
    ap.add_argument("--weights", default="list", choices=["list", *LOW_MASTER],
                    help="list: the configuration's weight format for every tensor; fp8-master: "
                         "linear layers block-scaled E4M3 with bf16 compute copies, embeddings, "
                         "norms and head bf16 (the paper's FP8-master setting); fp4-master: the "
                         "same with MXFP4 linear layers; nvfp4-master: the same with NVFP4 "
                         "linear layers (the paper's 4-bit setting) whose tensor scale the step "
                         "keeps; nvfp4cs-master: NVFP4 with the tensor scale derived anew every "
                         "step (current scaling)")
    ap.add_argument("--cpu-sample", type=int, default=1 << 24)
    ap.add_argument("--cpu-steps", type=int, default=None,
                    help="gradient sets generated for the oracle's sample (default 10; 4 with "
                         "bf16 moments)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="time the oracle steps the sample for (at least two steps)")
    ap.add_argument("--cpu-threads", type=int, default=None,
                    help="host threads for the oracle (default: this process's CPUs, at most 16)")
    ap.add_argument("--grads", default=None, choices=["regen", "cycle"],
                    help="regen: fill the gradients anew on the device before every step "
                         "(default when one gradient set exceeds 8 GiB); cycle: generate up to "
                         "8 sets up front and cycle through them, steps queued back to back "
                         "(default for the smaller lists)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-full", action="store_true",
                    help="instead of timing the GPU, time the oracle on the 1024x1024, GPT-2 "
                         "and Llama-1.1B lists in full (every parameter, two steps each), on "
                         "one thread and on all of the process's cores (up to 16)")
    ap.add_argument("--no-ceiling", action="store_true",
                    help="skip the streaming-ceiling probe (same buffers and bytes, no arithmetic)")
    ap.add_argument("--shard", default=None, metavar="K/P",
                    help="time only rank K's contiguous 1/P of the flat list, index base = its "
                         "first element: one GPU's share under P-way optimizer-state sharding")
    ap.add_argument("--copy-probe-gib", type=float, default=0.0,
                    help="after timing, run one plain device copy of this many GiB (a known "
                         "byte count that calibrates HBM traffic counters in a profiler run)")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures the optimizer step on one GPU only; runs on several GPUs "
              "are not implemented (the step shards by index range without communication: "
              "use --shard K/P to time one GPU's share).", file=sys.stderr)
        sys.exit(2)
    if args.cpu_full:
        print(json.dumps(cpu_full_configs(args.cpu_threads or cpu_threads())), flush=True)
        return

    import torch

    from paper_2607_10611_amd import binding as B
    from paper_2607_10611_amd import workloads as W

    B.lib()
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    shard = None
    if args.shard:
        k, p = (int(x) for x in args.shard.split("/"))
        if not (p >= 1 and 0 <= k < p) or args.weights != "list":
            sys.exit("--shard K/P needs 0 <= K < P and the plain list (--weights list)")
        shard = (k, p)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    cfg = args.config
    wfmt = W.CONFIGS[cfg]["wfmt"]
    specs = W.specs(cfg)
    nparam = W.total_params(cfg)
    code_dt = torch.int16 if wfmt == "bf16" else torch.uint8

    log(f"workload {cfg}: {len(specs)} tensors, {nparam:,} params, {wfmt} weights")
    t0 = time.perf_counter()
    # Flat per-role layout: one allocation each for the weight codes, the two
    # gradient sets and each moment, with the 291 tensors as views in list
    # order (the layout fused optimizers keep their state in).
    sizes = [s.numel for s in specs]

    def flat(dtype):
        buf = torch.empty(nparam, dtype=dtype, device=dev)
        views, off = [], 0
        for n in sizes:
            views.append(buf[off:off + n])
            off += n
        return buf, views

    low = LOW_MASTER.get(args.weights)
    if low:
        plan = W.low_precision_master_plan(cfg, low)
    else:
        plan = [(wfmt, False, False)] * len(specs)

    def flat_subset(dtype, pick, per_elem=1, head=0):
        """One buffer for the tensors selected by pick, views (None elsewhere):
        n // per_elem elements per tensor after `head` leading elements, each
        view starting at a multiple of 4 elements."""
        lens = [head + n // per_elem for n in sizes]
        tot = sum(-(-k // 4) * 4 for k, p in zip(lens, plan) if pick(p))
        buf = torch.empty(max(tot, 1), dtype=dtype, device=dev)
        views, off = [], 0
        for k, p in zip(lens, plan):
            if pick(p):
                views.append(buf[off:off + k])
                off += -(-k // 4) * 4
            else:
                views.append(None)
        return buf, views

    if args.weights == "list":
        wbuf, ws = flat(code_dt)
        scales = copies = None
    else:
        wb16, w16 = flat_subset(torch.int16, lambda p: p[0] == "bf16")
        wb8, w8 = flat_subset(torch.uint8, lambda p: p[0] != "bf16",
                              per_elem=2 if low in ("mxfp4", "nvfp4", "nvfp4_current") else 1)
        ws = [a if a is not None else b for a, b in zip(w16, w8)]
        if low == "mxfp4":
            sbuf, scales = flat_subset(torch.uint8, lambda p: p[1], per_elem=32)
        elif low == "nvfp4":  # fp32 tensor scale, then one E4M3 code per 16
            sbuf, scales = flat_subset(torch.uint8, lambda p: p[1], per_elem=16, head=4)
        elif low == "nvfp4_current":  # tensor scale, amax word, E4M3 codes
            sbuf, scales = flat_subset(torch.uint8, lambda p: p[1], per_elem=16, head=8)
        else:
            sbuf, scales = flat_subset(torch.int16, lambda p: p[1], per_elem=128)
        cbuf, copies = flat_subset(torch.int16, lambda p: p[2])
    # Gradients: regenerated on the device before every step (outside the
    # events) when one set is large enough that its generation keeps the GPU
    # busy while the host queues the next step; otherwise a few sets made up
    # front and cycled, with the steps queued behind a short GPU-side delay so
    # that the events between back-to-back steps time the GPU alone.
    grads = args.grads or ("regen" if nparam * 4 > (8 << 30) else "cycle")
    nsets = 1 if grads == "regen" else max(1, min(8, args.steps))
    gsets = [flat(torch.float32) for _ in range(nsets)]
    st_dt = torch.float32 if args.states == "fp32" else torch.int16
    mbuf, ms = flat(st_dt)
    vbuf, vs = flat(st_dt)
    vebuf, ves = flat(st_dt)
    for i in range(len(specs)):
        x = W.init_fp32_device(cfg, i, dev)
        B.madd_encode_weights(x, ws[i], plan[i][0], scales=scales[i] if scales else None)
        del x
        B.madd_init_state(ms[i], vs[i], ves[i])
        if grads == "cycle":
            for k, (_, gl) in enumerate(gsets):
                W.grad_fp32_device_(cfg, i, k + 1, gl[i])
    torch.cuda.synchronize()
    log(f"resident: {torch.cuda.memory_allocated() / 2**30:.1f} GiB in "
        f"{time.perf_counter() - t0:.1f} s; gradients: {grads}"
        + (f" ({nsets} sets)" if grads == "cycle" else ""))

    sfmt = args.states.replace("-", "_")
    tlists = [B.TensorList(ws, [p[0] for p in plan], gl, ms, vs, ves, scales=scales,
                           copies=copies, sfmt=sfmt) for _, gl in gsets]
    stream = torch.cuda.current_stream()
    step_no = 0
    lo, hi = 0, nparam
    if shard:
        # In the flat layout the global index of an element is its offset, so
        # a contiguous range is one madd_step call with that offset as base.
        per = (nparam // shard[1]) // 128 * 128
        lo = shard[0] * per
        hi = nparam if shard[0] == shard[1] - 1 else lo + per
        log(f"shard {shard[0]}/{shard[1]}: elements [{lo:,}, {hi:,})")

    def new_gradients(t):
        """Step t's gradients, generated on the device (not timed)."""
        if grads == "regen":
            for i in range(len(specs)):
                W.grad_fp32_device_(cfg, i, t, gsets[0][1][i])

    def one_step():
        h = W.hparams(cfg, step=step_no)
        k = (step_no - 1) % nsets
        if shard:
            gb = gsets[k][0]
            B.madd_step(wbuf[lo:hi], wfmt, gb[lo:hi], mbuf[lo:hi], vbuf[lo:hi],
                        vebuf[lo:hi], h, index_base=lo, sfmt=sfmt, stream=stream)
        else:
            B.madd_multi_tensor_step(tlists[k], h, stream=stream)

    for _ in range(args.warmup):
        step_no += 1
        new_gradients(step_no)
        one_step()
    torch.cuda.synchronize()
    log(f"warmup {args.warmup} steps done")

    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    if grads == "regen":
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(args.steps)]
        for k in range(args.steps):
            step_no += 1
            new_gradients(step_no)
            ev[k][0].record(stream)
            one_step()
            ev[k][1].record(stream)
        torch.cuda.synchronize()
        per_launch_ms = [a.elapsed_time(b) for a, b in ev]
    else:
        # one pair of events around the back-to-back steps: an event between
        # two short launches costs the stream a few microseconds of its own
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        gpu_delay(stream, args.steps)
        ev[0].record(stream)
        for k in range(args.steps):
            step_no += 1
            one_step()
        ev[1].record(stream)
        torch.cuda.synchronize()
        per_launch_ms = [ev[0].elapsed_time(ev[1]) / args.steps] * args.steps
    wall = time.perf_counter() - wall0
    ms_per_step = sum(per_launch_ms) / args.steps
    avg_launch_ms = ms_per_step
    median_ms = statistics.median(per_launch_ms)
    log(f"timed {args.steps} steps: {ms_per_step:.4f} ms/step (wall {wall * 1e3 / args.steps:.3f}"
        f"{' with gradient generation' if grads == 'regen' else ''}), launches min "
        f"{min(per_launch_ms):.4f} median {median_ms:.4f} max {max(per_launch_ms):.4f} ms")

    n_step = hi - lo
    if shard:
        alg_bytes = n_step * bytes_per_param(wfmt, args.states)
    else:
        alg_bytes = algorithmic_bytes(sizes, plan, args.states)
    bpp = alg_bytes / n_step
    achieved = alg_bytes / (avg_launch_ms / 1e3) / 1e9

    ceiling = None
    if not args.no_ceiling and args.weights == "list" and wfmt == "bf16":
        ceiling = stream_ceiling(wbuf[lo:hi], [gb[lo:hi] for gb, _ in gsets], mbuf[lo:hi], vbuf[lo:hi],
                                 vebuf[lo:hi], 4 if args.states == "fp32" else 2, args.steps,
                                 stream, alg_bytes, achieved)
        log(f"streaming ceiling: {ceiling['achieved']:.1f} GB/s; the step reaches "
            f"{ceiling['step_frac_of_ceiling'] * 100:.1f}% of it; plain streams: read "
            f"{ceiling['read_only_gbs']:.0f}, write {ceiling['write_only_gbs']:.0f}, copy "
            f"{ceiling['copy_gbs']:.0f} GB/s")

    if args.copy_probe_gib > 0:
        nbytes = int(args.copy_probe_gib * 2**30) // 4 * 4
        src = torch.ones(nbytes // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"copy probe: {nbytes} bytes read + {nbytes} bytes written")
        del src, dst

    traffic = (traffic_from_profile()
               if (cfg == "c5" and args.states == "fp32" and args.weights == "list" and not shard)
               else None)
    if shard:
        kname = (f"madd_step_kernel<{wfmt} weights, fp32 grads, {args.states} moments, "
                 f"{W.CONFIGS[cfg]['rounding'].upper()}> on one shard")
    elif args.weights == "list":
        kname = (f"madd_step_kernel<{wfmt} weights, fp32 grads, {args.states} moments, "
                 f"{W.CONFIGS[cfg]['rounding'].upper()}>")
    else:
        low = LOW_MASTER[args.weights]
        if low == "nvfp4_current":
            kname = ("nvcs_clear_kernel + nvcs_step_kernel (NVFP4 with current scaling: the "
                     "two passes pipelined over groups of tensors) + madd_step_kernel<bf16> "
                     "(timed together)")
        else:
            kname = (f"madd_step_block_kernel<{low}> + madd_step_kernel<bf16> (two launches per "
                     "step; timed together)")
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                "traffic": traffic, "algorithmic_bytes_per_launch": int(round(alg_bytes)),
                "kernel": kname, "avg_launch_ms": round(avg_launch_ms, 4)}
    extra = 0 if shard else scratch_bytes(sizes, plan)
    if extra:
        roofline["scratch_bytes_per_launch"] = int(extra)
        roofline["achieved_with_scratch"] = round((alg_bytes + extra) / (avg_launch_ms / 1e3)
                                                  / 1e9, 1)

    cpu = None
    if not args.no_cpu_baseline:
        threads = args.cpu_threads or cpu_threads()
        log(f"timing the CPU oracle on a sample ({threads} threads)")
        steps = args.cpu_steps or (10 if args.states == "fp32" else 4)
        cpu = cpu_baseline(cfg, args.cpu_sample, steps, sfmt, threads, args.cpu_seconds)
        if threads > 1:
            log("timing the CPU oracle on the same sample, one thread")
            one = cpu_baseline(cfg, args.cpu_sample, steps, sfmt, 1, args.cpu_seconds)
            cpu["one_thread"] = {k: one[k] for k in ("value", "unit", "cores", "sample")}

    workload = WORKLOAD_NAMES[cfg]
    if shard:
        workload = f"rank {shard[0]} of {shard[1]} contiguous shards of the {workload}"
    low = LOW_MASTER.get(args.weights)
    out = {
        "metric": METRIC,
        "value": round(n_step / (ms_per_step / 1e3) / 1e9, 3),
        "unit": "Gparam/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "ms_per_step_median": round(median_ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": workload, "params": n_step, "tensors": len(specs),
                   "weight_format": wfmt if args.weights == "list" else
                   f"{low} block-scaled linear layers + bf16 compute copies; bf16 "
                   "embed/norms/head",
                   "grad_format": "fp32",
                   "state": f"{args.states} m, v, v_e",
                   "rounding": W.CONFIGS[cfg]["rounding"], "bytes_per_param": round(bpp, 4)},
        "hbm_gbps": round(alg_bytes / (ms_per_step / 1e3) / 1e9, 1),
        "roofline": roofline,
        "ceiling": ceiling,
        "cpu_baseline": cpu,
    }
    if shard:
        out["config"]["index_base"] = lo
    print(json.dumps(out), flush=True)


def gpu_delay(stream, steps: int):
    """Queue a bounded GPU-side wait (madd_probe_delay) long enough for the
    host to enqueue `steps` short steps behind it: about 5 ms plus 100 us
    per step."""
    import ctypes

    from paper_2607_10611_amd import _build

    lib = ctypes.CDLL(_build.PROBE_LIB)
    lib.madd_probe_delay.argtypes = [ctypes.c_int32, ctypes.c_void_p]
    lib.madd_probe_delay.restype = ctypes.c_int32
    sleeps = int((5e-3 + 1e-4 * steps) / 3.4e-6)
    assert lib.madd_probe_delay(min(sleeps, 1 << 20), stream.cuda_stream) == 0


def stream_ceiling(w, gs, m, v, ve, state_bytes, steps, stream, alg_bytes, step_gbs) -> dict:
    """Time the streaming-ceiling probe (libmadd_probes.so) on the step's own
    buffers: the same bytes and access pattern without the arithmetic, cycling
    through the gradient sets `gs` in the order the timed steps used them."""
    import ctypes

    import torch

    from paper_2607_10611_amd import _build

    lib = ctypes.CDLL(_build.PROBE_LIB)
    lib.madd_ceiling_stream.argtypes = [ctypes.c_void_p] * 5 + [ctypes.c_int32, ctypes.c_int64,
                                                                ctypes.c_void_p]
    lib.madd_ceiling_stream.restype = ctypes.c_int32
    args = [[t.data_ptr() for t in (w, g, m, v, ve)] + [state_bytes, m.numel(), stream.cuda_stream]
            for g in gs]
    for k in range(2 * len(gs)):
        assert lib.madd_ceiling_stream(*args[k % len(gs)]) == 0
    # one pair of events around launches queued behind a GPU-side delay, as
    # the smaller lists' steps are timed: an event recorded after every launch
    # would add microseconds of stream time to each microsecond-scale probe
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    torch.cuda.synchronize()
    gpu_delay(stream, steps)
    ev[0].record(stream)
    for k in range(steps):
        assert lib.madd_ceiling_stream(*args[k % len(gs)]) == 0
    ev[1].record(stream)
    torch.cuda.synchronize()
    ms = ev[0].elapsed_time(ev[1]) / steps
    gbs = alg_bytes / (ms / 1e3) / 1e9
    out = {"kernel": "madd_ceiling_stream (same buffers and bytes, no arithmetic)",
           "avg_launch_ms": round(ms, 4), "achieved": round(gbs, 1), "unit": "GB/s",
           "frac_of_peak": round(gbs / HBM_PEAK_GBS, 4),
           "step_frac_of_ceiling": round(step_gbs / gbs, 4)}
    out.update(stream_modes(lib, steps, stream))
    return out


def stream_modes(lib, steps, stream, gib: int = 8) -> dict:
    """HBM bandwidth of plain read-only, write-only and copy streams in the
    step's access shape (madd_stream_modes) over two fresh `gib` GiB buffers."""
    import ctypes

    import torch

    lib.madd_stream_modes.argtypes = [ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
                                      ctypes.c_int64, ctypes.c_void_p]
    lib.madd_stream_modes.restype = ctypes.c_int32
    nbytes = gib << 30
    a = torch.ones(nbytes // 4, dtype=torch.int32, device="cuda")
    b = torch.empty_like(a)
    res = {}
    for mode, name, moved in ((0, "read_only_gbs", nbytes), (1, "write_only_gbs", nbytes),
                              (2, "copy_gbs", 2 * nbytes)):
        args = (mode, a.data_ptr(), b.data_ptr(), nbytes, stream.cuda_stream)
        for _ in range(2):
            assert lib.madd_stream_modes(*args) == 0
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        torch.cuda.synchronize()
        ev[0].record(stream)
        for _ in range(steps):
            assert lib.madd_stream_modes(*args) == 0
        ev[1].record(stream)
        torch.cuda.synchronize()
        res[name] = round(moved / (ev[0].elapsed_time(ev[1]) / steps / 1e3) / 1e9, 1)
    del a, b
    return res


if __name__ == "__main__":
    main()
