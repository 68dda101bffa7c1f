"""Throughput of the ADPSGD hot path on one MI355X.

One bench step is one whole ADPSGD run of the 138M-parameter workload
(K = 8 workers, P = 138,000,000 fp32 parameters in 32 tensors, 500 local
steps, adaptive period from p = 4 with C2 sampled over the first 125 steps):
every local step, every fused sync (mean, broadcast, per-tensor variance) and
every controller decision.  The replicas and momentum buffers are reset to
zero at the start of each run; h and x* stay resident in HBM.

Metric: parameter-updates/s = K * P * 500 * steps / time.  The roofline entry
is for the dominant kernel (the plain local step): algorithmic bytes per
launch (16 K P + 8 P) over its mean duration from HIP events recorded on the
library's stream during the timed region, around every 8th launch of each
kernel kind (--timing-every) so that the events barely disturb the job.

Prints one JSON line.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "local_step_k8_p138m_traffic.md")


def code_tokens(text: str) -> str:
    """C++ source with its comments removed and every run of whitespace made one
    space: what the compiler sees, so that edits to comments leave it alone."""
    out, i, n = [], 0, len(text)
    while i < n:
        if text.startswith("//", i):
            j = text.find("\n", i)
            i = n if j < 0 else j
        elif text.startswith("/*", i):
            j = text.find("*/", i + 2)
            i = n if j < 0 else j + 2
            out.append(" ")
        elif text[i] in "\"'":
            j = i + 1
            while j < n and text[j] != text[i]:
                j += 2 if text[j] == "\\" else 1
            out.append(text[i:j + 1])
            i = j + 1
        else:
            out.append(text[i])
            i += 1
    return " ".join("".join(out).split())


# Every source the profiled kernels are compiled from.
KERNEL_SOURCES = ("paper_2007_06134_amd/csrc/kernels.hip", "paper_2007_06134_amd/csrc/rng.hpp",
                  "paper_2007_06134_amd/csrc/kernels.hpp", "paper_2007_06134_amd/csrc/schedule.hpp",
                  "include/adpsgd.h")


def kernel_source_digest() -> str:
    """sha256 (first 16 hex digits) of the device sources' code, comments and
    whitespace left out: profiles taken on the same code stay valid."""
    h = hashlib.sha256()
    for name in KERNEL_SOURCES:
        with open(os.path.join(ROOT, name), encoding="utf-8") as f:
            h.update(code_tokens(f.read()).encode() + b"\0")
    return h.hexdigest()[:16]


def measured_traffic(w, block, lds, row_chunks):
    """HBM bytes per local-step launch from the committed counter summary, if it
    was taken on the current kernel sources, this problem (K = 8, P = 138M) and
    this launch shape (threads per block, LDS reserved per block, chunks per
    row run); else None."""
    if (w.K, w.P) != (8, 138_000_000) or not os.path.exists(TRAFFIC_FILE):
        return None
    txt = open(TRAFFIC_FILE).read()
    m_d = re.search(r"kernel sources digest:\s*`?([0-9a-f]{16})", txt)
    m_b = re.search(rf"HBM bytes per launch \(scaled\), block {block}, LDS {lds}, row chunks {row_chunks}:"
                    r"\s*([0-9.eE+]+)", txt)
    if not (m_d and m_b) or m_d.group(1) != kernel_source_digest():
        return None
    return float(m_b.group(1))


def period_text(w) -> str:
    import workloads as W
    if w.period_mode == W.PERIOD_ADAPTIVE:
        return f"adaptive, p_init {w.p_init}, K_s {w.k_s}, thresholds {w.thr_lo}/{w.thr_hi}"
    kind = "Algorithm 1 offset" if w.period_mode == W.PERIOD_ALG1 else "constant"
    return f"{kind} {w.p_init}"


def copy_context(torch, n_bytes=2 << 30, reps=5):
    """A plain device-to-device copy (torch's kernel) of n_bytes, as the
    attainable-bandwidth context for the step kernels: GB/s counting the read
    and the write."""
    src = torch.ones(n_bytes // 4, device="cuda:0", dtype=torch.float32)
    dst = torch.empty_like(src)
    dst.copy_(src)
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        dst.copy_(src)
    b.record()
    b.synchronize()
    ms = a.elapsed_time(b) / reps
    del src, dst
    return {"kernel": "torch copy_", "bytes_each_way": n_bytes, "avg_launch_ms": ms,
            "achieved_GBs": 2 * n_bytes / (ms * 1e-3) / 1e9}


def cpu_baseline(w, P_sample=16_000_000, steps=80):
    """The oracle, as it stands, on the first P_sample parameters of the same workload."""
    import oracle
    # keep whole tensors that fit, then cut the one that crosses P_sample
    sizes, acc = [], 0
    for s in w.sizes:
        take = min(s, P_sample - acc)
        if take <= 0:
            break
        sizes.append(take)
        acc += take
    ws = w.replace(name=w.name + "_cpu_sample", sizes=tuple(sizes))
    o = oracle.Oracle(ws)
    h, xs = o.problem_data()
    t0 = time.perf_counter()
    o.run(n_steps=steps, h=h, xs=xs)
    dt = time.perf_counter() - t0
    return {
        "value": ws.K * ws.P * steps / dt, "unit": "param-updates/s", "cores": oracle.num_threads(),
        "kind": "oracle",
        "sample": f"first {ws.P:,} of {w.P:,} parameters (K={w.K}), steps 0-{steps - 1} of the same "
                  f"adaptive run, fp64, {dt:.1f} s",
    }


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="vgg16_adaptive")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-timing", action="store_true", help="skip per-kernel HIP events")
    ap.add_argument("--timing-every", type=int, default=8, metavar="N",
                    help="HIP events around every N-th launch of each kernel kind (default 8)")
    ap.add_argument("--traced", action="store_true",
                    help="run the tracing mode (per-step variance and gradient norm) instead")
    ap.add_argument("--step-launch", default=None, metavar="BLOCK,LDS[,ROWCHUNKS]",
                    help="fix the plain local step's launch shape (threads per block, LDS bytes reserved "
                         "per block, chunks of a row an XCD takes in a run; default 1) instead of the one "
                         "timed fastest at init, e.g. so that separate counter passes profile the same kernel")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB (x3), to scale byte counters")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py: the K workers share one GPU's HBM, so the library runs on one GPU; "
              "--gpus must be 1", file=sys.stderr)
        sys.exit(2)

    import torch
    if args.copy_calibration:
        n = args.copy_calibration * (1 << 20) // 4
        src = torch.ones(n, device="cuda:0", dtype=torch.float32)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes_each_way": n * 4, "launches": 3}), flush=True)
        return
    import workloads as W
    import paper_2007_06134_amd as A

    w = W.full_workloads()[args.workload]
    N = w.total_steps
    eng = A.Adpsgd.from_workload(w, device="cuda:0")
    if args.step_launch:
        eng.set_step_launch(*(int(v) for v in args.step_launch.split(",")))
    stream = eng.stream

    def one_run():
        eng.reset()
        if args.traced:
            return eng.run_traced(N, log_cap=N, with_var=False)[:3]
        return eng.run(N, log_cap=N, with_var=False)

    for _ in range(args.warmup):
        one_run()
    torch.cuda.synchronize()
    eng.set_timing(0 if args.no_timing else max(1, args.timing_every))
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    n_syncs = []
    for _ in range(args.steps):
        recs, _, n = one_run()
        n_syncs.append(n)
    stream.synchronize()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    tm = eng.get_timing()
    step_block, step_lds, step_row_chunks = eng.step_launch
    row_stride = eng.row_stride
    sep = None
    if not args.no_timing:
        # context outside the timed region: the separate sync (mean, broadcast and
        # variance of all K rows, no step) that adpsgd_average runs
        eng.set_timing(True)
        for _ in range(5):
            eng.average()
        ta = eng.get_timing()
        if ta.average_launches > 0:
            a_ms = ta.average_ms / ta.average_launches
            sep = {"avg_launch_ms": a_ms, "bytes_per_launch": 8 * w.K * w.P,
                   "achieved_GBs": 8 * w.K * w.P / (a_ms * 1e-3) / 1e9,
                   "segsum_avg_ms": ta.segsum_ms / max(ta.segsum_launches, 1)}
    eng.close()

    updates = w.K * w.P * N * args.steps
    step_bytes = 16 * w.K * w.P + 8 * w.P          # x, m read+write per worker; h, x* once
    out = {
        "metric": "param-updates/s",
        "value": updates / elapsed,
        "unit": "param-updates/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": 1e3 * elapsed / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": w.name, "K": w.K, "P": w.P, "T": w.T, "local_steps_per_run": N,
                   "period": period_text(w),
                   "syncs_per_run": int(n_syncs[-1]),
                   # the periods the controller chose in the last timed run
                   "p_range": [int(recs["p"].min()), int(recs["p"].max())] if len(recs) else None},
    }
    if args.traced:
        out["config"]["mode"] = "traced"
    if tm.trace_launches > 0:
        trace_ms = tm.trace_ms / tm.trace_launches
        out["traced_step"] = {"avg_launch_ms": trace_ms, "achieved_GBs": step_bytes / (trace_ms * 1e-3) / 1e9}
    if tm.step_launches > 0:
        step_ms = tm.step_ms / tm.step_launches
        achieved = step_bytes / (step_ms * 1e-3) / 1e9
        traffic = measured_traffic(w, step_block, step_lds, step_row_chunks)
        out["roofline"] = {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                           "frac": achieved / HBM_PEAK_GBS, "traffic": traffic,
                           # traffic is not measured in this run: it is the copy-scaled
                           # FETCH_SIZE + WRITE_SIZE of a separate rocprofv3 --pmc run,
                           # read from the committed summary when it was taken on these
                           # kernel sources and this launch shape (else null)
                           "traffic_source": {"profile": os.path.relpath(TRAFFIC_FILE, ROOT),
                                              "kernel_sources_digest": kernel_source_digest(),
                                              "matched": traffic is not None},
                           "kernel": f"k_local_step<{step_block}>",
                           "lds_reserved_per_block": step_lds, "row_chunks": step_row_chunks,
                           "row_stride": row_stride,
                           "bytes_per_launch": step_bytes,
                           "avg_launch_ms": step_ms, "timed_launches": tm.step_launches,
                           "timed_every": args.timing_every}
        if tm.fused_launches > 0:
            fused_ms = tm.fused_ms / tm.fused_launches
            out["fused_step_sync"] = {"avg_launch_ms": fused_ms,
                                      "achieved_GBs": step_bytes / (fused_ms * 1e-3) / 1e9,
                                      "segsum_avg_ms": tm.segsum_ms / max(tm.segsum_launches, 1)}
        out["hbm_GBs_whole_run"] = (step_bytes * N * args.steps) / elapsed / 1e9
    if sep:
        out["separate_sync"] = sep
    if not args.no_timing:
        out["copy_context"] = copy_context(torch)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
