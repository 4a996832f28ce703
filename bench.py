#!/usr/bin/env python3
"""Throughput of GDN prefill on one MI355X: tokens/s, roofline fraction, CPU oracle beside it.

    python bench.py [--gpus 1] [--steps 20] [--warmup 5] [--workload 1] [--no-cpu-baseline]
                    [--segment-chunks L] [--pre] [--decode]

One step = one full gdn_prefill call (chunk index, chunk-local, segment maps,
state propagation with output) over the workload: by default one sequence of 4096
tokens, 16 heads, head dim 128, bf16 q/k/v, fp32 gates and state (seeded
synthetic inputs, see paper_2609_32114_amd/inputs.py).  Inputs are resident in
HBM before timing; the step cycles through several input copies (more bytes
than the 256 MB Infinity Cache) so each step reads its inputs from HBM, not
from cache.  The timed region holds only the K steps; per-kernel times come
from HIP events the library records on the launch stream around each kernel
during a second pass over the same K steps (events inside the timed region
would add their own GPU time, about 3 us each, to every step).

--pre times the same prefill from raw projections with every in-kernel
preprocessing flag (q/k L2 normalisation, softplus gate, sigmoid beta).
--decode times the decode step instead: one token for each of 256 sequences
(H = 16, d = 128, bf16, fp32 state pool updated in place); its metric is
decode tokens/s.

Roofline fields (one JSON line):
  roofline        the dominant kernel (longest HIP-event mean): the whole call's
                  algorithmic bytes (q, k, v, gates, beta, s0 in; o, s_final out:
                  16,512 B per token at the timed workload plus the states) over
                  that kernel's mean duration, against 8 TB/s; traffic = the
                  kernel's rocprofv3 FETCH_SIZE + WRITE_SIZE bytes per launch
                  (copy-calibrated, profiles/traffic.json) while its sources are
                  unchanged, else null
  path_roofline   the same algorithmic bytes and FLOPs over the whole step
  kernels         per kernel: mean ms, compulsory and counter bytes, HBM
                  fractions of both, counter MFMA FLOPs and their fraction of the
                  bf16 peak (counters from profiles/traffic.json, null when stale)
  step_ms         mean of the timed steps, and median / p10 / p90 from a pass
                  with one event between steps
  peaks           published peaks and the ones measured in this run with the
                  library's own streaming copy and bf16 MFMA loop

Prints ONE JSON line.
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

METRIC = "GDN prefill tokens/s at H=16,d=128,T=4096 bf16; % of HBM/MFMA roofline"
DECODE_METRIC = "GDN decode tokens/s (one token per sequence, 256 sequences) at H=16,d=128 bf16"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, published
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 MFMA, published
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")


def kernel_source_hash(name: str) -> str:
    """Hash of the sources a kernel is built from (traffic counters go stale when they change)."""
    csrc = os.path.join(ROOT, "paper_2609_32114_amd", "csrc")
    files = {"chunk_local": ("k1_chunk_local.hip", "state_walk.h"),
             "state_prop": ("k2_state_prop.hip", "state_walk.h", "k2_walk.hip", "k3_segments.hip"),
             "seg_transfer": ("k3_segments.hip", "k2_walk.hip"), "chunk_index": ("k0_chunk_index.hip",),
             "decode": ("k4_decode.hip",),
             "overlap_setup": ("k1_chunk_local.hip",),
             "overlapped": ("k1_chunk_local.hip", "state_walk.h")}
    h = hashlib.sha256()
    for f in files[name] + ("device.h", "prefill.h"):
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def counter_record(kernel: str, workload: str):
    """The committed rocprofv3 counter record of a kernel at a workload, if its
    sources are unchanged since the counters were taken."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f).get(f"{kernel}@{workload}")
    except (OSError, ValueError):
        return None
    if not rec or rec.get("source_hash") != kernel_source_hash(kernel):
        return None
    return rec


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per launch from committed rocprofv3 PMC counts, if still current."""
    rec = counter_record(kernel, workload)
    return None if rec is None else rec.get("bytes_per_launch")


def kernel_table(kernel_ms, workload, compulsory):
    """Per kernel: mean ms, compulsory / counter bytes and their HBM fractions,
    counter MFMA FLOPs and their fraction of the bf16 peak."""
    out = {}
    for k, ms in kernel_ms.items():
        if ms <= 0:
            continue
        rec = counter_record(k, workload) or {}
        cb, fl = rec.get("bytes_per_launch"), rec.get("mfma_flops")
        comp = compulsory(k)
        out[k] = {"ms": ms, "compulsory_bytes": comp,
                  "hbm_frac_compulsory": comp / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
                  "counter_bytes": cb,
                  "hbm_frac_counter": None if cb is None else cb / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
                  "mfma_flops_counter": fl,
                  "mfma_frac_counter": None if fl is None else fl / (ms * 1e-3) / 1e12 / BF16_PEAK_TFLOPS,
                  "mfma_busy_counter": rec.get("mfma_busy")}
    return out


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(inp, budget_s=10.0, max_reps=400, pre=0):
    """The fp64 oracle on the host's cores (all the process may use, at most 16),
    repeated over the full workload for about budget_s; then once on one thread."""
    import oracle
    threads = max(1, min(16, len(os.sched_getaffinity(0))))
    oracle.build(force=False)
    reps, t0 = 0, time.perf_counter()
    while True:
        oracle.run_inputs(inp, nthreads=threads, pre=pre)
        reps += 1
        el = time.perf_counter() - t0
        if el >= budget_s or reps >= max_reps:
            break
    tokens = reps * inp.T
    t1 = time.perf_counter()
    oracle.run_inputs(inp, nthreads=1, pre=pre)
    el1 = time.perf_counter() - t1
    return {"value": tokens / el, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"full workload ({inp.T} tokens x {inp.v.shape[1]} heads) repeated "
                      f"{reps}x, {el:.1f} s, fp64 token recurrence",
            "cpu_model": cpu_model(), "value_1thread": inp.T / el1, "seconds_1thread": el1}


def measured_peaks(P, torch, copy_mib=1024, mfma_iters=20000):
    """HBM bandwidth of the library's streaming copy (read + write bytes / time)
    and the bf16 rate of its MFMA loop, each the best of six event-timed runs."""
    src = torch.empty(copy_mib << 18, dtype=torch.float32, device="cuda:0").fill_(1.0)
    dst = torch.empty_like(src)
    n = src.numel() * 4
    sink = torch.empty(16 * 1024, dtype=torch.float32, device="cuda:0")
    best_copy = best_mfma = 0.0
    for _ in range(6):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        P.measure_copy(src, dst)
        b.record()
        torch.cuda.synchronize()
        best_copy = max(best_copy, 2 * n / (a.elapsed_time(b) * 1e-3) / 1e9)
        a.record()
        flops = P.measure_mfma(mfma_iters, sink)
        b.record()
        torch.cuda.synchronize()
        best_mfma = max(best_mfma, flops / (a.elapsed_time(b) * 1e-3) / 1e12)
    del src, dst
    return {"hbm_gbs": HBM_PEAK_GBS, "bf16_tflops": BF16_PEAK_TFLOPS,
            "measured_copy_gbs": best_copy, "measured_bf16_tflops": best_mfma,
            "copy_bytes": 2 * n, "note": "published peaks are the roofline denominators; the measured "
                                         "ones are this device's own copy and MFMA-loop rates"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", type=int, default=1)
    ap.add_argument("--copies", type=int, default=6)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--segment-chunks", type=int, default=0,
                    help="segment length of the state chain in 64-token chunks (0: automatic)")
    ap.add_argument("--no-overlap", action="store_true",
                    help="run the chunk-local kernel and the state walks one after another even where "
                         "the overlapped launch applies")
    ap.add_argument("--pre", action="store_true",
                    help="prefill from raw projections with every in-kernel preprocessing flag")
    ap.add_argument("--decode", action="store_true", help="time the decode step instead of prefill")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB (10 times): the known-size "
                         "reference that scales rocprofv3 FETCH_SIZE / WRITE_SIZE counts")
    ap.add_argument("--calibrate-mfma", type=int, default=0, metavar="ITERS",
                    help="only run the library's bf16 MFMA loop (ITERS rounds, 3 times): the "
                         "known-FLOP reference for rocprofv3 MFMA counters")
    args = ap.parse_args()
    if args.calibrate_mfma:
        import torch
        import paper_2609_32114_amd as P
        sink = torch.empty(16 * 1024, dtype=torch.float32, device="cuda:0")
        flops = [P.measure_mfma(args.calibrate_mfma, sink) for _ in range(3)]
        torch.cuda.synchronize()
        print(json.dumps({"calibrate_mfma_flops_per_launch": flops[0], "launches": 3}), flush=True)
        return
    if args.calibrate_copy:
        import torch
        n = args.calibrate_copy * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(10):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibrate_copy_bytes": n * 4, "launches": 10}), flush=True)
        return
    if args.gpus != 1:
        print("bench.py measures one GPU only: the method shards by (sequence, head) with no "
              "communication, so a multi-GPU figure would be N independent copies of this run; "
              "run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    if args.decode:
        return bench_decode(args)

    import numpy as np
    import torch

    import paper_2609_32114_amd as P
    from paper_2609_32114_amd import cost
    from paper_2609_32114_amd.inputs import WORKLOADS, make_workload

    P.load_library()
    P.set_segment_chunks(args.segment_chunks)
    P.set_overlap(not args.no_overlap)
    wl = WORKLOADS[args.workload]
    pre = P.PRE_ALL if args.pre else 0
    inp = make_workload(args.workload, raw=bool(pre))
    kda = inp.kind == "kda"
    dev = "cuda:0"
    torch.cuda.set_device(0)
    dt = torch.bfloat16 if inp.dtype == "bf16" else torch.float32
    esz = 2 if inp.dtype == "bf16" else 4
    T, N = inp.T, inp.N
    Hqk, Hv, Dk, Dv = wl.Hqk, wl.Hv, wl.Dk, wl.Dv

    def dev_copy(seed_shift):
        t = lambda x, d=torch.float32: torch.from_numpy(np.ascontiguousarray(x)).to(dev).to(d)
        return dict(q=t(inp.q, dt), k=t(inp.k, dt), v=t(inp.v, dt), g=t(inp.g), beta=t(inp.beta),
                    s0=None if inp.s0 is None else t(inp.s0))

    copies = [dev_copy(i) for i in range(max(1, args.copies))]
    cu = torch.from_numpy(inp.cu_seqlens).to(dev)
    fn = P.gdn_prefill if not kda else P.kda_prefill
    ws = torch.empty(P.workspace_size(inp.kind, N, T, Hqk, Hv, Dk, Dv,
                                      P.HAGDN_BF16 if esz == 2 else P.HAGDN_F32),
                     dtype=torch.uint8, device=dev)
    o = torch.empty((T, Hv, Dv), dtype=dt, device=dev)
    sf = torch.empty((N, Hv, Dk, Dv), dtype=torch.float32, device=dev)

    def step(i):
        c = copies[i % len(copies)]
        fn(c["q"], c["k"], c["v"], c["g"], c["beta"], initial_state=c["s0"], cu_seqlens=cu,
           scale=inp.scale, workspace=ws, out=o, final_out=sf, preprocess=pre)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()

    # timed region: K steps bracketed by events on torch's stream (the library
    # launches on it); no per-kernel events inside, they would add their own
    # GPU time to the step
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for i in range(args.steps):
        step(args.warmup + i)
    end.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(end) / args.steps
    # the same K steps with one event between consecutive steps: the per-step
    # distribution (each event adds a little GPU time; the mean above has none)
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    evs[0].record()
    for i in range(args.steps):
        step(args.warmup + i)
        evs[i + 1].record()
    torch.cuda.synchronize()
    per_step = sorted(evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps))
    pct = lambda p: per_step[min(len(per_step) - 1, int(round(p * (len(per_step) - 1))))]
    # the same K steps again with the library's HIP events around every kernel
    # (on the launch stream): per-kernel durations for the roofline
    P.profile_begin(args.steps)
    for i in range(args.steps):
        step(args.warmup + i)
    kernel_ms, ncalls = P.profile_end()

    value = T / (ms * 1e-3)
    dom = max(kernel_ms, key=kernel_ms.get)
    L = P.segment_chunks(N, T, Hv, Dv, torch.bfloat16 if esz == 2 else torch.float32, kind=inp.kind)
    wname = wl.name + (f"_pre{pre}" if pre else "")
    path_bytes = cost.algorithmic_bytes(T, N, Hqk, Hv, Dk, Dv, esz, kda, inp.s0 is not None)
    path_flops = cost.flops(T, Hv, 64, Dk, Dv)
    dom_ms = kernel_ms[dom]
    # the contract's roofline: the method's algorithmic bytes per launch over
    # the dominant kernel's mean duration
    achieved = path_bytes / (dom_ms * 1e-3) / 1e9
    traffic = measured_traffic(dom, wname)
    compulsory = lambda k: cost.kernel_bytes(k, T, N, Hqk, Hv, Dk, Dv, esz, kda, inp.s0 is not None,
                                             seg_chunks=L)
    kernels = kernel_table(kernel_ms, wname, compulsory)
    peaks = measured_peaks(P, torch)
    out = {
        "metric": METRIC,
        "value": value,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": inp.dtype,
        "data": "synthetic",
        "config": {"workload": wname, "kind": inp.kind, "sequences": N, "seq_len": T,
                   "q_k_heads": Hqk, "v_heads": Hv, "head_dim_k": Dk, "head_dim_v": Dv,
                   "chunk": 64, "segment_chunks": L, "input_copies": len(copies),
                   "preprocess": pre,
                   "overlapped": P.overlap_for(N, T, Hv, Dk, Dv, P.HAGDN_BF16 if esz == 2 else P.HAGDN_F32,
                                               inp.kind, torch.cuda.get_device_properties(0).multi_processor_count)},
        "roofline": {"bound": "hbm", "kernel": dom, "achieved": achieved, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS, "traffic": traffic,
                     "algorithmic_bytes": path_bytes, "kernel_ms": dom_ms},
        "path_roofline": {"bound": "hbm", "algorithmic_bytes": path_bytes,
                          "achieved": path_bytes / (ms * 1e-3) / 1e9, "peak": HBM_PEAK_GBS,
                          "unit": "GB/s", "frac": path_bytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
                          "flops": path_flops,
                          "mfma_frac": path_flops / (ms * 1e-3) / 1e12 / BF16_PEAK_TFLOPS},
        "step_ms": {"mean": ms, "median": pct(0.5), "p10": pct(0.1), "p90": pct(0.9),
                    "samples": args.steps},
        "kernels": kernels,
        "kernels_ms": kernel_ms,
        "kernel_calls_timed": ncalls,
        "peaks": peaks,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(inp, pre=pre)
    print(json.dumps(out), flush=True)


def bench_decode(args):
    """Decode step: K steps over the 256-sequence batch, then a profiled pass."""
    import numpy as np
    import torch

    import paper_2609_32114_amd as P
    from paper_2609_32114_amd import cost
    from paper_2609_32114_amd.inputs import DECODE_WORKLOAD as W, make_decode_case

    P.load_library()
    torch.cuda.set_device(0)
    dev = "cuda:0"
    di = make_decode_case(kind=W["kind"], N=W["N"], Hqk=W["Hqk"], Hv=W["Hv"], Dk=W["Dk"],
                          Dv=W["Dv"], dtype=W["dtype"], seed=5)
    N, Hqk, Hv, Dk, Dv = W["N"], W["Hqk"], W["Hv"], W["Dk"], W["Dv"]
    dt = torch.bfloat16 if di.dtype == "bf16" else torch.float32
    esz = 2 if di.dtype == "bf16" else 4
    t = lambda x, d=torch.float32: torch.from_numpy(np.ascontiguousarray(x)).to(dev).to(d)
    toks = dict(q=t(di.q, dt), k=t(di.k, dt), v=t(di.v, dt), g=t(di.g), beta=t(di.beta))
    # two state pools (2 x 256 MiB, more than the 256 MB Infinity Cache) in turn
    pools = [t(di.state) for _ in range(2)]
    o = torch.empty((N, Hv, Dv), dtype=dt, device=dev)

    def step(i):
        P.gdn_decode(toks["q"], toks["k"], toks["v"], toks["g"], toks["beta"], pools[i % 2],
                     scale=di.scale, out=o)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for i in range(args.steps):
        step(args.warmup + i)
    end.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(end) / args.steps
    P.profile_begin(args.steps)
    for i in range(args.steps):
        step(args.warmup + i)
    kernel_ms, ncalls = P.profile_end()
    kms = kernel_ms["decode"]
    nbytes = cost.decode_bytes(N, Hqk, Hv, Dk, Dv, esz, False)
    achieved = nbytes / (kms * 1e-3) / 1e9
    out = {
        "metric": DECODE_METRIC, "value": N / (ms * 1e-3), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": di.dtype, "data": "synthetic",
        "config": {"workload": f"decode_N{N}_H{Hv}_d{Dk}_{di.dtype}", "kind": "gdn",
                   "sequences": N, "q_k_heads": Hqk, "v_heads": Hv, "head_dim_k": Dk,
                   "head_dim_v": Dv, "state_pools": len(pools)},
        "roofline": {"bound": "hbm", "kernel": "decode", "achieved": achieved,
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                     "traffic": measured_traffic("decode", f"decode_N{N}_H{Hv}_d{Dk}_{di.dtype}"),
                     "bytes_per_launch": nbytes, "kernel_ms": kms},
        "kernels_ms": {"decode": kms},
        "kernel_calls_timed": ncalls,
    }
    if not args.no_cpu_baseline:
        import oracle
        threads = max(1, min(16, len(os.sched_getaffinity(0))))
        oracle.build(force=False)
        reps, t0 = 0, time.perf_counter()
        while True:
            oracle.decode("gdn", di.q, di.k, di.v, di.g, di.beta, di.state, di.scale,
                          nthreads=threads)
            reps += 1
            el = time.perf_counter() - t0
            if el >= 10.0 or reps >= 400:
                break
        out["cpu_baseline"] = {"value": reps * N / el, "unit": "tokens/s", "cores": threads,
                               "kind": "oracle",
                               "sample": f"the full decode batch ({N} sequences x {Hv} heads) "
                                         f"repeated {reps}x, {el:.1f} s, fp64"}
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
