"""Throughput of the GMC boundary operator on one MI355X.

A step is one gmc_prune call over one batch of synthetic boundary tensors
(every stage: message clients, banks, all selection rounds, assignment,
transport, compaction).  Inputs are resident in HBM before timing starts.
Prints one JSON line:
  value       = visual tokens pruned per second = B (N - K) / seconds per step
  roofline    = dominant kernel's algorithmic bytes (or flops) per launch over
                its average launch time, from hipEvents on the op stream in
                a second pass over the same steps with stage timing on
  cpu_baseline= the fp64 oracle timed on this host on a bounded sample
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

HBM_PEAK_GBS = 8000.0        # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0    # dense bf16 MFMA
FP32_PEAK_TFLOPS = 157.3

METRIC = "visual tokens pruned/sec (GMC op, 1 GPU) at Qwen2.5-VL-7B shape; % roofline"

WORKLOAD_TEXT = {
    "qwen": "Qwen2.5-VL-7B boundary: N=1296 (36x36), T=64, d=3584, 28/4 heads, dh=128, K=256, "
            "bf16 16-component Gaussian mixture",
    "batch16": "16 x Qwen2.5-VL-7B boundary problems in one call (N=1296, T=64, K=256 each)",
    "doc": "high-res document: N=4096 (64x64), T=128, d=3584, 28/4 heads, K=820, bf16",
    "frames": "multi-frame: N=16384 (4x64x64), T=256, d=3584, 28/4 heads, K=2048, bf16, bounded bank",
    "tiny": "tiny: N=256 (16x16), T=16, d=512, 8/2 heads, dh=64, K=64, fp32",
}


# Sources whose change invalidates a stored PMC traffic measurement of the
# selection kernels.
TRAFFIC_SOURCES = ["paper_2608_02134_amd/csrc/k_select.hip", "paper_2608_02134_amd/csrc/gmc_device.h",
                   "paper_2608_02134_amd/csrc/gmc_internal.h", "paper_2608_02134_amd/csrc/gmc_api.hip"]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")


def source_hash(paths=TRAFFIC_SOURCES) -> str:
    h = hashlib.sha256()
    for rel in paths:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def stored_traffic(workload: str, stage: str):
    """HBM bytes per launch of the dominant kernel from the stored rocprofv3
    FETCH_SIZE / WRITE_SIZE passes, scaled by the copy-kernel calibration;
    None when absent or taken on different kernel sources."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None, "no stored counter measurement"
    ent = rec.get("workloads", {}).get(workload)
    if not ent or ent.get("stage") != stage:
        return None, "no stored counter measurement for this kernel"
    if ent.get("source_hash") != source_hash():
        return None, "kernel sources changed since the counters were taken"
    cal = rec["copy_calibration"]
    fetch = ent["fetch_kib_per_launch"] * 1024.0 * cal["fetch_factor"]
    write = ent["write_kib_per_launch"] * 1024.0 * cal["write_factor"]
    return fetch + write, (f"rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE on {ent['kernel']}, "
                           f"scaled by a {cal['bytes'] / 2**20:.0f} MiB copy; see profiles/")


def copy_calibration(mib: int, reps: int = 10):
    """A plain device copy of known size (read `mib` MiB, write `mib` MiB), for
    scaling the FETCH_SIZE / WRITE_SIZE counters to bytes."""
    import torch
    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(reps):
        torch.mul(src, 1.0, out=dst)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": n * 4, "reps": reps,
                      "kernel": "torch elementwise mul by 1 (read + write)"}), flush=True)


def kernel_work(stage: str, w, m_rows: int, kr: int = 0, bsel: int = 16, pool_cap: int = 64):
    """Algorithmic bytes or flops of one launch of a stage's kernel."""
    n, k, b = w.n, w.k, w.batch
    if stage == "gains":      # the token-major client matrix once, row weights, coverage, gains
        return "hbm", b * (4.0 * m_rows * n + 8.0 * m_rows + 4.0 * n)
    if stage == "select":     # every round in one launch: per round the client rows of the
        total, sel = 0.0, 0  # unselected tokens (gains), of the pool (responsibilities) and of
        while sel < kr:      # the batch (coverage), plus row weights and coverage once
            ps, bs = min(pool_cap, n - sel), min(bsel, kr - sel)
            total += 4.0 * m_rows * ((n - sel) + ps + bs) + 8.0 * m_rows + 4.0 * n
            sel += bs
        return "hbm", b * total
    if stage == "appearance":  # N x N x d Gram
        return "mfma", b * 2.0 * n * n * w.d
    if stage == "transport":   # every member row once + the compact output
        esz = 2 if w.dtype == "bf16" else 4
        return "hbm", b * (esz * n * w.d + esz * k * w.d)
    if stage == "logits":      # write the grounded client rows
        return "hbm", b * 4.0 * w.hq * w.t * n
    return None, None


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="qwen", choices=sorted(WORKLOAD_TEXT))
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="time budget of the oracle CPU baseline sample (0 disables)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB (counter calibration) and exit")
    ap.add_argument("--serial", action="store_true",
                    help="every kernel on the caller's stream for the whole run (stage-timing mode), for "
                         "profilers whose counter passes serialize dispatches; not a throughput figure")
    ap.add_argument("--op", default="prune", choices=["prune", "compact"],
                    help="prune: the operator (default line); compact: sequence compaction and "
                         "prefix K/V gather after pruning")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the operator is single-GPU and this build has no "
              "multi-GPU path (see the design notes on sharding by image)", file=sys.stderr)
        sys.exit(2)

    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return
    if args.op == "compact":
        bench_compaction(args)
        return

    import torch
    from paper_2608_02134_amd import binding, synth
    from paper_2608_02134_amd.binding import make_pruner, to_device

    prob = synth.make_problem(args.workload)
    w = prob.workload
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    hid = to_device(prob.hidden, w.dtype, torch)
    q = to_device(prob.text_q, w.dtype, torch)
    kk = to_device(prob.vis_k, w.dtype, torch)
    pos = torch.from_numpy(prob.pos3d).cuda()
    pr = make_pruner(prob, torch, max_k=w.k)
    kr = binding.gmc_realized_k(w.n, w.k)
    out_h = torch.empty((w.batch, kr, w.d), dtype=hid.dtype, device=dev)
    out_p = torch.empty((w.batch, kr, 3), dtype=torch.int32, device=dev)
    out_i = torch.empty((w.batch, kr), dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream(dev)
    binding._check(binding.gmc_set_stream(stream.cuda_stream), "gmc_set_stream")
    ptrs = (hid.data_ptr(), q.data_ptr(), kk.data_ptr(), pos.data_ptr())
    outs = (out_h.data_ptr(), out_p.data_ptr(), out_i.data_ptr())

    def step():
        code = binding.lib().gmc_prune(*ptrs, w.n, w.t, w.k, *outs)
        if code != 0:
            raise binding.GmcError(code, "gmc_prune")

    if args.serial:
        # the bank kernels then run on the caller's stream as well: no kernel
        # waits for another stream's kernel, which a profiler that serializes
        # dispatches would never start
        binding._check(binding.gmc_timing_enable(True), "gmc_timing_enable")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # timed region: K steps between events on the op stream
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record(stream)
    for _ in range(args.steps):
        step()
    t1.record(stream)
    torch.cuda.synchronize()
    ms_total = t0.elapsed_time(t1)
    ms_step = ms_total / args.steps
    # the device status of the timed calls (sticky bits: any timed-out
    # device wait or non-finite value in any of them) invalidates the run
    code, diag = binding.gmc_get_diag(0)
    if code != binding.GMC_OK:
        print(f"timed calls failed on the device: {binding.gmc_last_error()}", file=sys.stderr)
        sys.exit(3)
    pruned = w.batch * (w.n - kr)
    value = pruned / (ms_step / 1e3)

    # stage breakdown: the same K steps again with stage events on the stream
    binding._check(binding.gmc_timing_enable(True), "gmc_timing_enable")
    for _ in range(args.steps):
        step()
    stage_ms, stage_n = binding.gmc_timing_read()
    binding._check(binding.gmc_timing_enable(args.serial), "gmc_timing_enable")
    code, _ = binding.gmc_get_diag(0)
    if code != binding.GMC_OK:
        print(f"stage-timed calls failed on the device: {binding.gmc_last_error()}", file=sys.stderr)
        sys.exit(3)
    stages = {name: {"ms_per_step": stage_ms[i] / args.steps,
                     "launch_avg_us": (1e3 * stage_ms[i] / stage_n[i]) if stage_n[i] else None,
                     "launches_per_step": stage_n[i] / args.steps}
              for i, name in enumerate(binding.STAGE_NAMES)}

    rounds, pool_cap, bcap, m_rows = binding.gmc_trace_dims(w.n, w.t, w.k)
    single_kernel = ["select", "gains", "appearance", "transport", "logits"]
    dom = max(single_kernel, key=lambda s: stages[s]["ms_per_step"])
    bound, work = kernel_work(dom, w, m_rows, kr, bcap, pool_cap)
    avg_s = stages[dom]["launch_avg_us"] / 1e6
    if bound == "hbm":
        achieved, peak, unit = work / avg_s / 1e9, HBM_PEAK_GBS, "GB/s"
    else:
        achieved = work / avg_s / 1e12
        peak = BF16_PEAK_TFLOPS if w.dtype == "bf16" else FP32_PEAK_TFLOPS
        unit = "TFLOP/s"
    traffic, traffic_note = stored_traffic(args.workload, dom)
    roofline = {"bound": bound, "kernel": dom, "achieved": achieved, "peak": peak, "unit": unit,
                "frac": achieved / peak, "traffic": traffic, "traffic_note": traffic_note,
                "work_per_launch": work, "launch_avg_us": stages[dom]["launch_avg_us"],
                "source_hash": source_hash()}
    if bound == "hbm" and traffic:
        # `achieved` counts the algorithmic bytes; the counters give what
        # actually crossed the fabric.  Far fewer measured bytes than
        # algorithmic ones means the kernel's operands stayed in the caches
        # and its time is set by latency, not by HBM bandwidth.
        roofline["traffic_gbs"] = traffic / avg_s / 1e9
        roofline["traffic_over_work"] = traffic / work
        roofline["regime"] = ("latency: operands cache-resident, measured traffic well below the algorithmic bytes"
                              if traffic < 0.5 * work else "bandwidth: operands streamed past the L2 caches every round")

    cpu = None
    if args.cpu_seconds > 0:
        cpu = cpu_baseline(prob, args.cpu_seconds)

    line = {
        "metric": METRIC, "value": value, "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_step, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": w.dtype, "data": "synthetic",
        "config": {"workload": WORKLOAD_TEXT[args.workload], "batch": w.batch, "N": w.n, "T": w.t,
                   "K": kr, "d": w.d, "heads": [w.hq, w.hkv], "head_dim": w.dh,
                   "rounds": rounds, "client_rows": m_rows, **({"serial": True} if args.serial else {})},
        "roofline": roofline, "cpu_baseline": cpu, "stages": stages,
    }
    pr.close()
    print(json.dumps(line), flush=True)


# Sequence compaction after pruning at the Qwen2.5-VL-7B shape: 16 prompts of
# 15 system + 1296 visual + 64 question positions, K = 256 retained, the
# boundary states (d = 3584) and the prompt K/V of 16 prefix layers (token
# major, 4 kv heads x 128, bf16) gathered at the retained positions.
COMPACT = dict(batch=16, before=15, n=1296, after=64, k=256, d=3584, layers=16, hkv=4, dh=128)
COMPACT_METRIC = "bytes moved / s (sequence compaction + prefix K/V gather after pruning, 1 GPU)"


def bench_compaction(args):
    import torch
    from paper_2608_02134_amd import binding, synth
    from paper_2608_02134_amd.binding import make_pruner
    c = COMPACT
    b, n, k = c["batch"], c["n"], c["k"]
    seq = c["before"] + n + c["after"]
    l2 = seq - n + k
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    pr = make_pruner(synth.make_problem("tiny", grid=(1, 8, 8), t=4, k=16), torch)   # a context
    g = torch.Generator(device=dev).manual_seed(7)
    kept = torch.stack([torch.randperm(n, generator=g, device=dev)[:k].sort().values for _ in range(b)])
    kept = kept.to(torch.int32).contiguous()
    rows = torch.randn((b, seq, c["d"]), generator=g, device=dev).to(torch.bfloat16)
    vis = torch.randn((b, k, c["d"]), generator=g, device=dev).to(torch.bfloat16)
    pos = torch.randint(0, 1000, (b, seq, 3), generator=g, device=dev, dtype=torch.int32)
    caches = [torch.randn((b, seq, c["hkv"] * c["dh"]), generator=g, device=dev).to(torch.bfloat16)
              for _ in range(2 * c["layers"])]
    iota = torch.empty((b, seq), dtype=torch.int32, device=dev)
    keep = torch.empty((b, l2), dtype=torch.int32, device=dev)
    out_rows = torch.empty((b, l2, c["d"]), dtype=torch.bfloat16, device=dev)
    out_pos = torch.empty((b, l2, 3), dtype=torch.int32, device=dev)
    outs = [torch.empty((b, l2, c["hkv"] * c["dh"]), dtype=torch.bfloat16, device=dev) for _ in caches]
    row_bytes, kv_bytes = c["d"] * 2, c["hkv"] * c["dh"] * 2
    stream = torch.cuda.current_stream(dev)
    binding._check(binding.gmc_set_stream(stream.cuda_stream), "gmc_set_stream")
    src = [t.data_ptr() for t in caches]
    dst = [t.data_ptr() for t in outs]
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    gather_ms = []

    def step(timed=False):
        binding._check(binding.gmc_compact_sequence(b, seq, c["before"], n, k, kept.data_ptr(), iota.data_ptr(),
                                                    keep.data_ptr(), rows.data_ptr(), vis.data_ptr(),
                                                    out_rows.data_ptr(), row_bytes, pos.data_ptr(),
                                                    out_pos.data_ptr()), "gmc_compact_sequence")
        if timed:
            ev[0].record(stream)
        binding._check(binding.gmc_gather_rows(src, dst, b, 1, seq, l2, kv_bytes, keep.data_ptr()), "gmc_gather_rows")
        if timed:
            ev[1].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record(stream)
    for _ in range(args.steps):
        step()
    t1.record(stream)
    torch.cuda.synchronize()
    ms_step = t0.elapsed_time(t1) / args.steps
    # the gather kernel alone: events around its launch on the op stream
    for _ in range(args.steps):
        step(timed=True)
        torch.cuda.synchronize()
        gather_ms.append(ev[0].elapsed_time(ev[1]))
    gather_s = sum(gather_ms) / len(gather_ms) / 1e3
    gather_work = 2.0 * len(caches) * b * l2 * kv_bytes + 4.0 * b * l2          # rows read + written, keep
    seq_work = 2.0 * b * l2 * (row_bytes + 12) + 4.0 * b * (seq + l2 + k)     # rows, ids, maps, out_idx
    work = gather_work + seq_work
    # CPU baseline: the oracle's gather of the same caches on the host, one
    # prompt at a time until about two seconds are used
    from oracle import gmc_oracle as O
    host = [t[0].view(torch.int16).cpu().numpy() for t in caches]
    hkeep = keep[0].cpu().numpy()
    n_done, tc0 = 0, time.perf_counter()
    while time.perf_counter() - tc0 < 2.0 or n_done == 0:
        for h in host:
            O.gather_cache(h, hkeep)
        n_done += 1
    cpu_s = (time.perf_counter() - tc0) / n_done
    line = {
        "metric": COMPACT_METRIC, "value": work / (ms_step / 1e3) / 1e9, "unit": "GB/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_step, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "sequence compaction after pruning, Qwen2.5-VL-7B shape: 16 prompts of 15 + 1296 "
                               "visual + 64 positions, K = 256, boundary states d = 3584 and prompt K/V of 16 "
                               "prefix layers (token-major, 4 x 128, bf16)",
                   "batch": b, "L": seq, "L2": l2, "N": n, "K": k, "tensors": len(caches)},
        "roofline": {"bound": "hbm", "kernel": "gather_rows_kernel", "achieved": gather_work / gather_s / 1e9,
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": gather_work / gather_s / 1e9 / HBM_PEAK_GBS,
                     "traffic": None, "work_per_launch": gather_work, "launch_avg_us": gather_s * 1e6},
        "cpu_baseline": {"value": 2.0 * len(caches) * l2 * kv_bytes / cpu_s / 1e9, "unit": "GB/s", "cores": 1,
                         "kind": "oracle", "sample": f"the oracle's gather of one prompt's {len(caches)} caches, "
                                                     f"{n_done} times ({cpu_s * 1e3:.1f} ms each)"},
    }
    pr.close()
    print(json.dumps(line), flush=True)


def _cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(prob, budget_s: float):
    """The oracle as it stands, on this host, on whole problems of the same
    workload: three runs with the BLAS pool at its default width (the median
    is `value`) and one single-thread run, each of at least one problem and
    about a fifth of the time budget."""
    from oracle import gmc_oracle as O
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:  # pragma: no cover
        threadpool_limits = None
        cores = os.cpu_count()
    w = prob.workload
    per_problem = w.n - min(w.n, max(w.k, 1))

    def run(seconds):
        done, t0 = 0, time.perf_counter()
        while True:
            b = done % w.batch
            O.gmc_single(prob.hidden[b], prob.text_q[b], prob.vis_k[b], prob.pos3d[b], prob.probe, w.k,
                         app_proj=prob.app_proj)
            done += 1
            if time.perf_counter() - t0 >= seconds:
                break
        el = time.perf_counter() - t0
        return done * per_problem / el, done, el

    part = budget_s / 5.0
    runs = [run(part) for _ in range(3)]
    rates = sorted(r[0] for r in runs)
    single = None
    if threadpool_limits is not None:
        with threadpool_limits(limits=1):
            single = run(part)
    return {"value": rates[1], "unit": "tokens/s", "cores": cores, "kind": "oracle",
            "cpu_model": _cpu_model(), "runs": [r[0] for r in runs],
            "single_thread_value": None if single is None else single[0],
            "sample": (f"median of 3 runs of whole {w.name} problems (N={w.n}, K={w.k}) through the fp64 "
                       f"oracle, {sum(r[1] for r in runs)} problems in {sum(r[2] for r in runs):.1f} s on "
                       f"{cores} BLAS threads" +
                       ("" if single is None else f"; single thread: {single[1]} problem(s) in {single[2]:.1f} s"))}


if __name__ == "__main__":
    main()
