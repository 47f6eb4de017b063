"""Throughput of the batched Poseidon DAG-cost evaluation on one MI355X.

One step = one pass of the whole hot path over the workload's candidate
list: decode every (composition rank, assignment) pair, build the stage
weights from the LDS prefix tables, check the memory caps, take the longest
path of the pipeline DAG (1F1B, or Eager 1F1B with --schedule eager),
write every makespan and the packed feasibility bits,
and min-reduce to the best feasible candidate.  Inputs are resident in HBM
before timing starts.

Default workload: L=126 layers, S=16 stages, M=128 micro-batches, T=4
device types, 2^24 sampled compositions (the largest of the five synthetic
workloads).  Prints one JSON line.
"""
import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_INT32_TOPS = 256 * 64 * 2.4e9 / 1e12   # CUs x lanes x clock: one 32-bit op per lane per cycle
N_SIMD, PEAK_CLOCK = 256 * 4, 2.4e9
CSRC = os.path.join(ROOT, "paper_2609_06086_amd", "csrc")
COUNTERS = os.path.join(ROOT, "profiles", "eval_pipeline_counters_L126_S16_M128.json")


def dp_ops(S, M):
    """add/max operations of the DAG recurrence per candidate: three per node
    (edge add, max, node add) minus the missing inputs of the first stage's
    forwards, the last stage's backwards and each stage's first node."""
    return 6 * S * M - 4 * M - S


def kernel_sha():
    """Hash of the device and launch code the counters depend on."""
    h = hashlib.sha256()
    for f in sorted(os.listdir(CSRC)):
        if f.endswith((".hip", ".h", ".cpp")):
            h.update(f.encode())
            h.update(open(os.path.join(CSRC, f), "rb").read())
    return h.hexdigest()


def committed_counters():
    """Per-call HBM bytes and VALU instructions from the committed rocprofv3
    counter summary, or None if the code changed since it was taken."""
    if not os.path.exists(COUNTERS):
        return None
    t = json.load(open(COUNTERS))
    if t.get("source_sha256") != kernel_sha():
        return None
    return t


def cpu_baseline(wl, target_s):
    from oracle import coracle
    coracle.lib()
    threads = coracle.default_threads()
    n = len(wl.cands)
    probe = min(n, 200000)
    t0 = time.perf_counter()
    coracle.evaluate(wl.problem, wl.cands, nthreads=threads, lo=0, hi=probe)
    dt = time.perf_counter() - t0
    m = int(min(n, max(probe, probe * target_s / max(dt, 1e-6))))
    t0 = time.perf_counter()
    coracle.evaluate(wl.problem, wl.cands, nthreads=threads, lo=0, hi=m)
    dt = time.perf_counter() - t0
    return {"value": m / dt, "unit": "candidates/s", "cores": threads, "kind": "oracle",
            "sample": f"first {m} of the {n} candidates of the same workload, C oracle (explicit DAG, "
                      f"Kahn order, topological DP) on {threads} host threads, {dt:.1f} s"}


SEARCH_OPS_PER_TEST = 15   # integer ops of one stage-choice test (memory 2, ridge 2, Eq. 2 11)


def search_bench(args):
    """The pruned configuration search (Sec. 4.2.3) over every assignment row
    and composition of the 8-stage, 3-type workload: one step = one
    poseidon_search call over all 6561 x C(79,7) = 1.9 x 10^13 candidates."""
    import numpy as np
    import torch

    from oracle import coracle
    from paper_2609_06086_amd import poseidon as P
    from paper_2609_06086_amd import workloads as W

    wl = W.workload(4)
    prob = wl.problem
    c = wl.cands
    # warm-up bound (Sec. 4.2.3): the best of the first 500 sampled candidates, evaluated on the GPU
    ctx = P.poseidon_load_costs(prob, 0)
    dev = torch.device("cuda:0")
    warm = P.poseidon_eval_candidates(ctx, comp_rank=torch.from_numpy(c.comp_rank[:500].view(np.int64)).to(dev),
                                      assign_idx=torch.from_numpy(c.assign_idx[:500].view(np.int32)).to(dev))
    bound = warm.makespan
    rpc = args.rows_per_chunk
    ramp = not args.fixed_chunks
    chunking = f"chunks of 1, 2, 4, ... up to {rpc} rows" if ramp else f"{rpc} rows per chunk"
    stream = torch.cuda.current_stream()

    def step():
        return P.poseidon_search(ctx, bound, rows_per_chunk=rpc, ridge=args.ridge, ramp=ramp, stream=stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    t0 = time.perf_counter()
    for e0, e1 in evs:
        e0.record(stream)
        best, st = step()
        e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    call_ms = sum(e0.elapsed_time(e1) for e0, e1 in evs) / len(evs)
    ms = wall * 1e3 / args.steps
    covered = prob.n_candidates
    tested = st.visited + st.pruned_memory + st.pruned_ridge + st.pruned_bound
    ops = tested * SEARCH_OPS_PER_TEST
    achieved = ops / (call_ms * 1e-3) / 1e12
    out = {
        "metric": "pruned search (Sec. 4.2.3): candidate configurations covered per second",
        "value": covered / (ms * 1e-3),
        "unit": "candidates/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "u32",
        "data": "synthetic (seeded per-layer profile tables)",
        "config": {"workload": f"L={prob.L} S={prob.S} M={prob.M} T={prob.T}, all {prob.A} assignment rows x "
                               f"C({prob.L - 1},{prob.S - 1}) compositions, {chunking}, bound = best of "
                               f"the first 500 sampled candidates ({bound} us)" + (", ridge filter" if args.ridge else ""),
                   "parallelism": "single GPU"},
        "search": {"visited": st.visited, "evaluated": st.evaluated, "pruned_memory": st.pruned_memory,
                   "pruned_ridge": st.pruned_ridge, "pruned_bound": st.pruned_bound,
                   "stage_choices_tested_per_s": tested / (call_ms * 1e-3),
                   "best_index": best.index, "best_makespan": best.makespan, "warmup_bound": bound},
        "roofline": {"bound": "alu", "achieved": achieved, "peak": PEAK_INT32_TOPS, "unit": "Top/s",
                     "frac": achieved / PEAK_INT32_TOPS, "traffic": None, "kernel_ms": call_ms,
                     "algorithmic_ops_per_launch": ops,
                     "launch": "one poseidon_search call (count, scan, write, leaf kernels per level)"},
    }
    if not args.no_cpu_baseline:
        coracle.lib()
        rows = 128
        t0 = time.perf_counter()
        r = coracle.search(prob, bound, first_row=0, n_rows=rows, rows_per_chunk=rpc, ridge=args.ridge, ramp=ramp)
        dt = time.perf_counter() - t0
        t_cpu = r["visited"] + r["pruned_memory"] + r["pruned_ridge"] + r["pruned_bound"]
        out["cpu_baseline"] = {"value": rows * prob.n_candidates / prob.A / dt, "unit": "candidates/s",
                               "cores": coracle.default_threads(), "kind": "oracle",
                               "stage_choices_tested_per_s": t_cpu / dt,
                               "sample": f"C oracle search (oracle/oracle.c, rows split over threads) over the first "
                                         f"{rows} assignment rows, same bound and chunking, {dt:.1f} s"}
    ctx.close()
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", type=int, default=5, choices=[3, 4, 5, 6])
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-early-stop", action="store_true")
    ap.add_argument("--schedule", default="1f1b", choices=["1f1b", "eager", "interleaved"],
                    help="pipeline schedule of the DAG (1F1B, Eager 1F1B, or Interleaved 1F1B with "
                         "the stages as virtual stages on S/2 devices; workloads 3 and 5)")
    ap.add_argument("--search", action="store_true",
                    help="time the pruned configuration search over the whole 8-stage workload instead")
    ap.add_argument("--rows-per-chunk", type=int, default=512)
    ap.add_argument("--fixed-chunks", action="store_true",
                    help="with --search: every chunk has --rows-per-chunk rows (default: chunks of 1, 2, 4, ... rows "
                         "up to --rows-per-chunk)")
    ap.add_argument("--ridge", action="store_true", help="with --search: layer-level (ridge) pruning")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="also run one plain device copy of this size (for counter scaling)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported (the evaluation of "
              f"independent candidates would shard by index range)", file=sys.stderr)
        sys.exit(2)

    if args.search:
        search_bench(args)
        return

    import numpy as np
    import torch

    from paper_2609_06086_amd import poseidon as P
    from paper_2609_06086_amd import workloads as W

    dev = torch.device("cuda:0")
    wl = W.workload(args.workload)
    prob = wl.problem
    if args.schedule == "interleaved":
        wl = W.interleaved_variant(wl, 2)
    else:
        prob.schedule = P.SCHEDULE_EAGER_1F1B if args.schedule == "eager" else P.SCHEDULE_1F1B
    n = len(wl.cands)
    ctx = P.poseidon_load_costs(prob, 0)
    if wl.cands.is_list:
        cand = dict(comp_rank=torch.from_numpy(wl.cands.comp_rank.view(np.int64)).to(dev))
        if wl.cands.assign_idx is not None:
            cand["assign_idx"] = torch.from_numpy(wl.cands.assign_idx.view(np.int32)).to(dev)
        in_bytes = 8 + (4 if wl.cands.assign_idx is not None else 0)
    else:
        cand = dict(first=wl.cands.first, count=wl.cands.count)
        in_bytes = 0
    Tout = torch.empty(n, dtype=torch.int32, device=dev)
    bits = torch.empty((n + 31) // 32, dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream()

    if args.copy_calibration_mib:
        a = torch.empty(args.copy_calibration_mib << 18, dtype=torch.int32, device=dev)
        b = torch.empty_like(a)
        b.copy_(a)
        torch.cuda.synchronize()

    def step():
        P.poseidon_eval_candidates(ctx, makespan_out=Tout, feasible_bits_out=bits, want_best=False,
                                   stream=stream, **cand)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for e0, e1 in evs:
        e0.record(stream)
        step()
        e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    best = P.poseidon_last_best(ctx, stream=stream)
    kms = [e0.elapsed_time(e1) for e0, e1 in evs]
    k_avg = sum(kms) / len(kms)
    ms_per_step = wall * 1e3 / args.steps

    S, M = prob.S, prob.M
    ops = n * dp_ops(S, M)
    achieved = ops / (k_avg * 1e-3) / 1e12
    ctr = committed_counters() if args.workload == 5 and args.schedule == "1f1b" else None
    nodes_per_s = n * 2 * S * M / (ms_per_step * 1e-3)
    value = n / (ms_per_step * 1e-3)
    algo_bytes = n * in_bytes + n * 4 + ((n + 31) // 32) * 4

    # early-stop pass (Eq. 2 bound) over the same list, warm-up bound from its first 500 entries
    es = None
    if wl.cands.is_list and not args.no_early_stop and args.schedule != "interleaved":
        warm = {k: v[:500] for k, v in cand.items()}
        wb = P.poseidon_eval_candidates(ctx, **warm)
        bound = wb.makespan if wb.makespan is not None else 2 ** 31
        reps = 10
        # untimed first call: loads the early-stop kernels and sizes the workspace
        P.poseidon_eval_candidates_bounded(ctx, bound, chunk=1 << 22, stream=stream, **cand)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(reps):
            bb, st = P.poseidon_eval_candidates_bounded(ctx, bound, chunk=1 << 22, stream=stream, **cand)
        e1.record(stream)
        torch.cuda.synchronize()
        es_ms = e0.elapsed_time(e1) / reps
        es = {"ms": round(es_ms, 3), "candidates_per_s": n / (es_ms * 1e-3), "warmup_bound": bound,
              "evaluated": st.evaluated, "pruned": st.pruned, "infeasible": st.infeasible,
              "best_index": bb.index, "best_makespan": bb.makespan,
              "same_argmin_as_exhaustive": (bb.index, bb.makespan) == (best.index, best.makespan),
              "chunk": 1 << 22}

    out = {
        "metric": "candidate configs evaluated/sec + DAG nodes/sec (fraction of INT32 VALU peak)",
        "value": value,
        "unit": "candidates/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u32",
        "data": "synthetic (seeded per-layer profile tables and sampled candidates)",
        "config": {"workload": f"L={prob.L} S={S} M={M} T={prob.T}, {n} sampled compositions, fixed 4x4 "
                               f"stage-type permutation" if args.workload == 5 and args.schedule != "interleaved"
                               else wl.description,
                   "schedule": {"eager": "Eager 1F1B", "interleaved": "Interleaved 1F1B (V = 2)"}.get(
                       args.schedule, "1F1B"),
                   "candidates_per_step": n, "dag_nodes_per_candidate": 2 * S * M,
                   "parallelism": "single GPU"},
        "dag_nodes_per_s": nodes_per_s,
        "int32_valu_frac": achieved / PEAK_INT32_TOPS,
        "best": {"index": best.index, "makespan_us": best.makespan},
        "roofline": {"bound": "alu", "achieved": achieved, "peak": PEAK_INT32_TOPS, "unit": "Top/s",
                     "frac": achieved / PEAK_INT32_TOPS,
                     "traffic": None if ctr is None else ctr["hbm_bytes_per_call"],
                     "kernel_ms": k_avg, "algorithmic_ops_per_launch": ops,
                     "algorithmic_bytes_per_launch": algo_bytes,
                     "launch": "one poseidon_eval_candidates call: decode, eval and resume kernels",
                     # hardware side: VALU wave-instructions the call issues (counters) x 4 cycles
                     # over all SIMD cycles at peak clock during the measured call time
                     "valu_issue_frac": None if ctr is None else
                     ctr["valu_wave_insts_per_call"] * 4 / (N_SIMD * PEAK_CLOCK * k_avg * 1e-3),
                     # INT32 lane-ops the call executes (counters: INT32 wave-instructions x
                     # mean active lanes per kernel) over the measured call time, against the peak
                     "valu_int32_lane_frac": None if ctr is None or "valu_int32_lane_ops_per_call" not in ctr else
                     ctr["valu_int32_lane_ops_per_call"] / (k_avg * 1e-3) / 1e12 / PEAK_INT32_TOPS},
        "early_stop": es,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl, args.cpu_seconds)
    ctx.close()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
