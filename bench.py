"""Throughput of the batched Poseidon DAG-cost evaluation on one MI355X.

One step = one pass of the whole hot path over the workload's candidate
list: decode every (composition rank, assignment) pair, build the stage
weights from the LDS prefix tables, check the memory caps, take the longest
path of the pipeline DAG (1F1B, or Eager / Interleaved 1F1B with
--schedule), write every makespan and the packed feasibility bits, and
min-reduce to the best feasible candidate.  Inputs are resident in HBM
before timing starts.

Default run: the headline line is the 16-stage workload (L=126 layers, S=16
stages, M=128 micro-batches, T=4 device types, 2^24 sampled compositions),
with the early-stop pass over the same list.  The same line carries
sub-records for the other workloads: the two small exhaustive ranges (8
layers on 2 stages, 28 candidates; 32 layers on 4 stages, 71,920
candidates), the exhaustive 8-stage 2-type range (C(47,7) = 62,891,499
compositions) and the 8-stage 3-type list of 2^26 sampled (composition,
assignment) pairs, the latter also as an early-stop pass with the
same-argmin check.  Every record has the CPU oracle timed beside it on a
bounded sample, and `oracle_check` compares the timed pass's makespans and
mask bits with the oracle's on that sample (and the argmin, when the sample
is the whole list).  Prints one JSON line.

Roofline fields: the path is 32-bit integer add/max on the vector ALUs.
`roofline.achieved` is the INT32 lane-operations one call executes, counted
by rocprofv3 (INT32 VALU wave-instructions x the mean active lanes of each
kernel's VALU cycles, summed over the call's kernels), divided by the call
time measured here with HIP events; `frac` = achieved / 39.32 Top/s.
`dominant_kernel` gives the same rate for the kernel with the largest share
of the call, over its own time in the committed kernel trace.  The
counts come from the committed summary profiles/<tag>.counters.json and are
used only while its hash of the kernel and launch sources matches the
current ones (else null).  The plain longest-path recurrence's 6SM - 4M - S
operations per candidate, which the kernels reach with far fewer operations,
are reported as `nominal_equiv_rate` / `nominal_equiv_frac`.

--summarize turns the CSV output of the rocprofv3 passes of one profiled
command into profiles/<tag>.md and profiles/<tag>.counters.json.
"""
import argparse
import collections
import csv
import glob
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_INT32_TOPS = 256 * 64 * 2.4e9 / 1e12   # CUs x lanes x clock: one 32-bit op per lane per cycle
N_SIMD, PEAK_CLOCK = 256 * 4, 2.4e9
CSRC = os.path.join(ROOT, "paper_2609_06086_amd", "csrc")
PROFILES = os.path.join(ROOT, "profiles")
ES_CHUNK = 0                # early-stop chunk (0 = one chunk: every candidate is filtered against the
                            # warm-up bound; the survivors are few, so more chunks cost more than they prune)
ES_WARMUP = 500             # warm-up samples that set the first bound (Sec. 4.2.3)


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


def profile_tag(kind, prob, schedule="1f1b"):
    """Name of a profile: pass kind and workload shape (and whether the DAG
    has all-reduce nodes, which other kernel instances evaluate)."""
    sched = {"1f1b": "", "eager": "_eager", "interleaved": f"_interleaved_N{prob.S // 2}"}[schedule]
    ar = "_allreduce" if getattr(prob, "allreduce", None) is not None else ""
    return f"{kind}{sched}{ar}_L{prob.L}_S{prob.S}_M{prob.M}"


def committed_counters(tag, candidates=None):
    """Per-call counter figures of the committed summary for `tag`, or None
    if it is missing, was taken on another number of candidates per call,
    or the kernel / launch code changed since it was taken."""
    path = os.path.join(PROFILES, tag + ".counters.json")
    if not os.path.exists(path):
        return None
    t = json.load(open(path))
    if t.get("source_sha256") != kernel_sha():
        return None
    if candidates is not None and t.get("candidates") != candidates:
        return None
    t["path"] = os.path.relpath(path, ROOT)
    return t


def dominant_kernel(ctr):
    """The kernel with the largest share of a call in the committed trace,
    with its INT32 lane-op rate over its own traced time."""
    if not ctr or not ctr.get("kernels") or not ctr.get("per_kernel"):
        return None
    calls = ctr["calls_profiled"]
    per_call = {k: v["avg_ns"] * v["dispatches"] / calls * 1e-6 for k, v in ctr["kernels"].items()}
    name = max(per_call, key=per_call.get)
    k = ctr["per_kernel"].get(name, {})
    ms = per_call[name]
    ops = k.get("int32_lane_ops")
    achieved = None if ops is None else ops / (ms * 1e-3) / 1e12
    return {"name": name, "ms_per_call": ms, "share": ms / sum(per_call.values()),
            "int32_lane_ops_per_call": ops, "achieved": achieved,
            "frac": None if achieved is None else achieved / PEAK_INT32_TOPS,
            "valu_issue_frac": None if "SQ_INSTS_VALU" not in k else
            k["SQ_INSTS_VALU"] * 4 / (N_SIMD * PEAK_CLOCK * ms * 1e-3)}


def roofline(ctr, call_ms, nominal_ops, algo_bytes, launch):
    """Hardware roofline of one call (see the module docstring)."""
    lane_ops = None if ctr is None else ctr.get("valu_int32_lane_ops_per_call")
    achieved = None if lane_ops is None else lane_ops / (call_ms * 1e-3) / 1e12
    nominal = None if nominal_ops is None else nominal_ops / (call_ms * 1e-3) / 1e12
    return {"bound": "alu", "achieved": achieved, "peak": PEAK_INT32_TOPS, "unit": "Top/s",
            "frac": None if achieved is None else achieved / PEAK_INT32_TOPS,
            "traffic": None if ctr is None else ctr["hbm_bytes_per_call"],
            "kernel_ms": call_ms,
            "executed_int32_lane_ops_per_launch": lane_ops,
            "algorithmic_ops_per_launch": nominal_ops,
            "nominal_equiv_rate": nominal,
            "nominal_equiv_frac": None if nominal is None else nominal / PEAK_INT32_TOPS,
            "algorithmic_bytes_per_launch": algo_bytes,
            "valu_issue_frac": None if ctr is None else
            ctr["valu_wave_insts_per_call"] * 4 / (N_SIMD * PEAK_CLOCK * call_ms * 1e-3),
            "counters": None if ctr is None else ctr["path"],
            "dominant_kernel": dominant_kernel(ctr),
            "launch": launch}


def timed(torch, step, steps, warmup, stream):
    """Run `warmup` untimed and `steps` timed calls; returns (wall ms per
    step, mean HIP-event ms per call on `stream`, last result)."""
    r = None
    for _ in range(warmup):
        r = step()
    torch.cuda.synchronize()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for e0, e1 in evs:
        e0.record(stream)
        r = step()
        e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    return wall * 1e3 / steps, sum(e0.elapsed_time(e1) for e0, e1 in evs) / steps, r


def cpu_baseline(wl, target_s):
    """The C oracle as it stands on all host threads, on a prefix of the same
    candidates sized for about target_s seconds.  Returns the record and the
    oracle's makespans and feasibility of that prefix."""
    from oracle import coracle
    coracle.lib()
    threads = coracle.default_threads()
    n = len(wl.cands)
    probe = min(n, 100000)
    t0 = time.perf_counter()
    coracle.evaluate(wl.problem, wl.cands, nthreads=threads, lo=0, hi=probe)
    dt = time.perf_counter() - t0
    m = int(min(n, max(probe, probe * target_s / max(dt, 1e-6))))
    t0 = time.perf_counter()
    T, feas = coracle.evaluate(wl.problem, wl.cands, nthreads=threads, lo=0, hi=m)
    dt = time.perf_counter() - t0
    S, M = wl.problem.S, wl.problem.M
    return {"value": m / dt, "unit": "candidates/s", "cores": threads, "kind": "oracle",
            "dag_nodes_per_s": m * 2 * S * M / dt,
            "sample": f"first {m} of the {n} candidates of the same workload, C oracle (explicit DAG, "
                      f"Kahn order, topological DP) on {threads} host threads, {dt:.1f} s"}, T, feas


def python_oracle_baseline(wl, target_s):
    """The pure-Python oracle (explicit DAG, Kahn order, one thread) on a
    prefix of the candidates sized for about target_s seconds.  Returns the
    record and its makespans and feasibility."""
    from oracle import dag
    from paper_2609_06086_amd import workloads as W
    c = wl.cands
    n = len(c)

    def prefix(m):
        if c.is_list:
            return W.Candidates(comp_rank=c.comp_rank[:m],
                                assign_idx=None if c.assign_idx is None else c.assign_idx[:m])
        return W.Candidates(first=c.first, count=m)

    probe = min(n, 200)
    t0 = time.perf_counter()
    dag.evaluate(wl.problem, prefix(probe))
    dt = time.perf_counter() - t0
    m = int(min(n, max(probe, probe * target_s / max(dt, 1e-6))))
    t0 = time.perf_counter()
    T, feas = dag.evaluate(wl.problem, prefix(m))
    dt = time.perf_counter() - t0
    return {"value": m / dt, "unit": "candidates/s", "cores": 1, "kind": "oracle",
            "sample": f"first {m} of the {n} candidates, Python oracle (explicit DAG, Kahn order, "
                      f"topological DP) on one thread, {dt:.2f} s"}, T.astype("uint32"), feas


def oracle_check(e, best, T_o, f_o):
    """The timed pass's outputs against the oracle's on its prefix: every
    makespan and mask bit, and (when the prefix is the whole list) the argmin."""
    import numpy as np
    from oracle import coracle
    m = len(T_o)
    Tg = e.T[:m].cpu().numpy().view(np.uint32)
    words = e.bits[:(m + 31) // 32].cpu().numpy().view(np.uint32)
    i = np.arange(m)
    fg = ((words[i >> 5] >> (i & 31).astype(np.uint32)) & 1).astype(bool)
    rec = {"compared": m, "makespan_mismatches": int(np.count_nonzero(Tg != T_o)),
           "mask_mismatches": int(np.count_nonzero(fg != f_o))}
    if m == e.n:
        ob = coracle.argmin(T_o, f_o)
        rec["oracle_best"] = None if ob is None else {"index": ob[0], "makespan_us": ob[1]}
        rec["same_argmin"] = ob == (best.index, best.makespan)
    return rec


class Eval:
    """One workload on the device: context, resident candidates, outputs."""

    def __init__(self, wl, dev):
        import numpy as np
        import torch
        from paper_2609_06086_amd import poseidon as P
        self.P, self.torch, self.wl = P, torch, wl
        self.prob = wl.problem
        self.n = len(wl.cands)
        self.ctx = P.poseidon_load_costs(self.prob, 0)
        if wl.cands.is_list:
            self.cand = dict(comp_rank=torch.from_numpy(wl.cands.comp_rank.view(np.int64)).to(dev))
            if wl.cands.assign_idx is not None:
                self.cand["assign_idx"] = torch.from_numpy(wl.cands.assign_idx.view(np.int32)).to(dev)
            self.in_bytes = 8 + (4 if wl.cands.assign_idx is not None else 0)
        else:
            self.cand = dict(first=wl.cands.first, count=wl.cands.count)
            self.in_bytes = 0
        self.T = torch.empty(self.n, dtype=torch.int32, device=dev)
        self.bits = torch.empty((self.n + 31) // 32, dtype=torch.int32, device=dev)
        self.stream = torch.cuda.current_stream()

    def step(self):
        self.P.poseidon_eval_candidates(self.ctx, makespan_out=self.T, feasible_bits_out=self.bits,
                                        want_best=False, stream=self.stream, **self.cand)

    def warm_bound(self):
        warm = {k: v[:ES_WARMUP] for k, v in self.cand.items()}
        wb = self.P.poseidon_eval_candidates(self.ctx, **warm)
        return wb.makespan if wb.makespan is not None else 2 ** 31

    def bounded(self, bound, chunk=ES_CHUNK, ramp=False):
        return self.P.poseidon_eval_candidates_bounded(self.ctx, bound, chunk=chunk, ramp=ramp, stream=self.stream,
                                                       **self.cand)

    def close(self):
        self.ctx.close()


def eval_record(wl, dev, args, schedule="1f1b", early_stop=True, cpu_s=0.0, py_s=0.0):
    """Exhaustive pass (and early-stop pass) of one workload as a record."""
    import torch
    e = Eval(wl, dev)
    prob, n = e.prob, e.n
    S, M = prob.S, prob.M
    ms_wall, call_ms, _ = timed(torch, e.step, args.steps, args.warmup, e.stream)
    best = e.P.poseidon_last_best(e.ctx, stream=e.stream)
    ops = n * dp_ops(S, M)
    algo_bytes = n * e.in_bytes + n * 4 + ((n + 31) // 32) * 4
    rec = {"workload": wl.description, "schedule": schedule, "candidates": n,
           "dag_nodes_per_candidate": 2 * S * M, "ms": ms_wall, "kernel_ms": call_ms,
           "candidates_per_s": n / (ms_wall * 1e-3), "dag_nodes_per_s": n * 2 * S * M / (ms_wall * 1e-3),
           "best": {"index": best.index, "makespan_us": best.makespan},
           "roofline": roofline(committed_counters(profile_tag("eval_pipeline", prob, schedule), n), call_ms, ops,
                                algo_bytes, "one poseidon_eval_candidates call: decode, eval and resume kernels")}
    if early_stop and wl.cands.is_list and schedule != "interleaved":
        bound = e.warm_bound()
        es_ms_wall, es_ms, (bb, st) = timed(torch, lambda: e.bounded(bound, args.es_chunk, args.es_ramp),
                                            max(1, args.steps // 5), max(1, args.warmup // 5), e.stream)
        chunking = ("one chunk" if args.es_chunk == 0 else
                    f"chunks of {args.es_chunk}, doubling" if args.es_ramp else f"chunks of {args.es_chunk}")
        rec["early_stop"] = {
            "ms": es_ms_wall, "kernel_ms": es_ms, "candidates_per_s": n / (es_ms_wall * 1e-3),
            "speedup_vs_exhaustive": ms_wall / es_ms_wall,
            "warmup_samples": ES_WARMUP, "warmup_bound": bound, "chunk": args.es_chunk, "ramp": args.es_ramp,
            "evaluated": st.evaluated, "pruned": st.pruned, "infeasible": st.infeasible,
            "best_index": bb.index, "best_makespan": bb.makespan,
            "same_argmin_as_exhaustive": (bb.index, bb.makespan) == (best.index, best.makespan),
            "roofline": roofline(committed_counters(profile_tag("early_stop", prob, schedule), n), es_ms, None, None,
                                 "one poseidon_eval_candidates_bounded call: filter and survivor kernels, "
                                 + chunking)}
    if cpu_s > 0:
        rec["cpu_baseline"], T_o, f_o = cpu_baseline(wl, cpu_s)
        rec["oracle_check"] = oracle_check(e, best, T_o, f_o)
    if py_s > 0:
        rec["python_oracle"], T_p, f_p = python_oracle_baseline(wl, py_s)
        rec["python_oracle"]["check"] = oracle_check(e, best, T_p, f_p)
    e.close()
    if "python_oracle" in rec or rec["roofline"]["achieved"] is None and n < (1 << 20):
        rec["note"] = "launch-bound (a few microseconds of kernel work per call): no counter profile"
    return rec


def load_workload(cfg, schedule):
    from paper_2609_06086_amd import poseidon as P
    from paper_2609_06086_amd import workloads as W
    wl = W.workload(cfg)
    if schedule == "interleaved":
        wl = W.interleaved_variant(wl, 2)
    else:
        wl.problem.schedule = P.SCHEDULE_EAGER_1F1B if schedule == "eager" else P.SCHEDULE_1F1B
    return wl


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
    if args.copy_calibration_mib:
        a = torch.empty(args.copy_calibration_mib << 18, dtype=torch.int32, device=dev)
        torch.empty_like(a).copy_(a)
        torch.cuda.synchronize()
    rpc = args.rows_per_chunk
    ramp = not args.fixed_chunks
    chunking = f"chunks of 1, 2, 4, ... up to {rpc} rows" if ramp else f"{rpc} rows per chunk"
    stream = torch.cuda.current_stream()

    def step():
        return P.poseidon_search(ctx, bound, rows_per_chunk=rpc, ridge=args.ridge, ramp=ramp, stream=stream)

    ms, call_ms, (best, st) = timed(torch, step, args.steps, args.warmup, stream)
    covered = prob.n_candidates
    tested = st.visited + st.pruned_memory + st.pruned_ridge + st.pruned_bound
    ops = tested * SEARCH_OPS_PER_TEST
    tag = "search" + ("_ridge" if args.ridge else "") + f"_L{prob.L}_S{prob.S}_M{prob.M}"
    rl = roofline(committed_counters(tag), call_ms, ops, None,
                  "one poseidon_search call (count, scan, write, leaf kernels per level)")
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
        "roofline": rl,
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


def profile_only(args):
    """One pass only (for rocprofv3): W untimed and K timed calls of the
    exhaustive or the early-stop pass of one workload."""
    import torch
    dev = torch.device("cuda:0")
    wl = load_workload(args.workload, args.schedule)
    e = Eval(wl, dev)
    if args.copy_calibration_mib:
        a = torch.empty(args.copy_calibration_mib << 18, dtype=torch.int32, device=dev)
        b = torch.empty_like(a)
        b.copy_(a)
        torch.cuda.synchronize()
    if args.only == "exhaustive":
        ms, call_ms, _ = timed(torch, e.step, args.steps, args.warmup, e.stream)
    else:
        bound = e.warm_bound()
        ms, call_ms, _ = timed(torch, lambda: e.bounded(bound, args.es_chunk, args.es_ramp), args.steps, args.warmup,
                               e.stream)
    e.close()
    print(json.dumps({"pass": args.only, "workload": wl.description, "calls": args.steps + args.warmup,
                      "ms": ms, "kernel_ms": call_ms}), flush=True)


# ------------------------------------------------------------------ summaries

PASS_KERNELS = {
    "exhaustive": r"pk::(decode_kernel|eval_kernel|sched_kernel|resume_kernel|ilv_kernel|ilv_resume_kernel)",
    "early_stop": r"pk::(filter_kernel|surv_kernel|fill_u64)",
    "search": r"pk::(search_|fill_u64)",
}


def _short(name):
    return re.sub(r"\(pk::.*$|\(unsigned.*$", "", name).strip()


def _csv(d, suffix):
    f = glob.glob(os.path.join(d, "*" + suffix))
    return list(csv.DictReader(open(f[0]))) if f else None


def _dispatches(rows):
    """Per-dispatch counter values from a rocprofv3 counter collection."""
    by = collections.OrderedDict()
    for r in rows:
        k = (int(r["Dispatch_Id"]), r["Kernel_Name"])
        by.setdefault(k, {})[r["Counter_Name"]] = float(r["Counter_Value"])
    return [dict(id=k[0], name=k[1], **v) for k, v in sorted(by.items())]


def summarize(args):
    """profiles/<tag>.md and profiles/<tag>.counters.json from the rocprofv3
    output directories <dir>/{kt,fetch,write,valu,lanes,lds} of one profiled
    command that made `calls` calls of the pass (the last `timed` of them
    timed)."""
    d, tag, calls, timed_calls = args.summarize, args.tag, args.calls, args.timed_calls
    pat = re.compile(PASS_KERNELS[args.pass_kind])
    out = {"tag": tag, "pass": args.pass_kind, "source_sha256": kernel_sha(), "calls_profiled": calls,
           "candidates": args.candidates or None, "commands": args.commands}
    md = [f"# {args.title}\n", args.description + "\n" if args.description else ""]
    kt = _csv(os.path.join(d, "kt"), "_kernel_trace.csv")
    if kt:
        kt = sorted((r for r in kt if pat.search(r["Kernel_Name"])), key=lambda r: int(r["Start_Timestamp"]))
        per = len(kt) // calls if calls and len(kt) % calls == 0 else 0
        agg = collections.OrderedDict()
        for r in kt:
            a = agg.setdefault(_short(r["Kernel_Name"]), [0, 0, 1 << 62, 0])
            dur = int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
            a[0] += 1
            a[1] += dur
            a[2] = min(a[2], dur)
            a[3] = max(a[3], dur)
        busy = sum(a[1] for a in agg.values()) / calls / 1e6
        md.append("## Kernel trace (rocprofv3 --kernel-trace --stats)\n")
        md.append("| Kernel | Dispatches | Average (ns) | Min (ns) | Max (ns) | Per call (ms) | Share |\n"
                  "|---|---|---|---|---|---|---|")
        tot = sum(a[1] for a in agg.values())
        for name, a in sorted(agg.items(), key=lambda kv: -kv[1][1]):
            md.append("| `%s` | %d | %.0f | %d | %d | %.4f | %.1f %% |" % (name, a[0], a[1] / a[0], a[2], a[3],
                                                                          a[1] / calls / 1e6, 100 * a[1] / tot))
        out["kernel_busy_ms_per_call"] = busy
        out["kernels"] = {name: {"dispatches": a[0], "avg_ns": a[1] / a[0]} for name, a in agg.items()}
        md.append("")
        md.append(f"{calls} calls of the pass; kernel busy time per call (sum of its kernels' durations): "
                  f"**{busy:.4f} ms**.")
        if per:
            spans = []
            for c in range(calls - timed_calls, calls):
                g = kt[c * per:(c + 1) * per]
                spans.append((int(g[-1]["End_Timestamp"]) - int(g[0]["Start_Timestamp"])) / 1e6)
            out["call_ms_kernel_trace"] = sum(spans) / len(spans)
            md.append(f"Call duration (first kernel start to last kernel end, {per} dispatches per call), mean "
                      f"over the {timed_calls} timed calls: **{out['call_ms_kernel_trace']:.4f} ms**.")
        md.append("")
    ctr = {}
    for sub in ("fetch", "write", "valu", "lanes", "lds"):
        rows = _csv(os.path.join(d, sub), "_counter_collection.csv")
        if rows:
            ctr[sub] = _dispatches(rows)
    scale = {}
    for sub, key in (("fetch", "FETCH_SIZE"), ("write", "WRITE_SIZE")):
        if sub in ctr:
            copies = [x for x in ctr[sub] if not pat.search(x["name"]) and "pk::" not in x["name"]]
            ref = max(copies, key=lambda x: x.get(key, 0)) if copies else None
            # a plain device copy of `copy_mib` MiB reads and writes that many bytes
            scale[key] = (args.copy_mib * 1024.0 / ref[key]) if ref and ref.get(key) else None
    per_kernel = collections.OrderedDict()

    def add(sub, key, alias=None):
        if sub not in ctr:
            return None
        tot = 0.0
        for x in ctr[sub]:
            if pat.search(x["name"]) and key in x:
                per_kernel.setdefault(_short(x["name"]), collections.OrderedDict())
                k = per_kernel[_short(x["name"])]
                k[alias or key] = k.get(alias or key, 0.0) + x[key] / calls
                tot += x[key]
        return tot / calls

    fetch = add("fetch", "FETCH_SIZE")
    write = add("write", "WRITE_SIZE")
    if fetch is not None and write is not None and scale.get("FETCH_SIZE") and scale.get("WRITE_SIZE"):
        out["hbm_read_bytes_per_call"] = fetch * 1024 * scale["FETCH_SIZE"]
        out["hbm_write_bytes_per_call"] = write * 1024 * scale["WRITE_SIZE"]
        out["hbm_bytes_per_call"] = out["hbm_read_bytes_per_call"] + out["hbm_write_bytes_per_call"]
        out["copy_scale_fetch"], out["copy_scale_write"] = scale["FETCH_SIZE"], scale["WRITE_SIZE"]
    for key in ("SQ_INSTS_VALU", "SQ_INSTS_VALU_INT32", "SQ_INSTS_SALU", "SQ_INSTS_LDS", "SQ_WAVES",
                "SQ_ACTIVE_INST_VALU"):
        v = add("valu", key)
        if v is not None:
            out[key.lower() + "_per_call"] = v
    if "valu" in ctr:
        out["valu_wave_insts_per_call"] = out.get("sq_insts_valu_per_call")
    if "lanes" in ctr:
        lane_ops = 0.0
        for x in ctr["lanes"]:
            if pat.search(x["name"]) and x.get("SQ_ACTIVE_INST_VALU"):
                ops = x["SQ_INSTS_VALU_INT32"] * x["SQ_THREAD_CYCLES_VALU"] / x["SQ_ACTIVE_INST_VALU"]
                k = per_kernel.setdefault(_short(x["name"]), collections.OrderedDict())
                k["int32_lane_ops"] = k.get("int32_lane_ops", 0.0) + ops / calls
                lane_ops += ops
        out["valu_int32_lane_ops_per_call"] = lane_ops / calls
    for key in ("SQ_INSTS_LDS", "SQ_WAIT_INST_LDS", "SQ_LDS_BANK_CONFLICT", "SQ_ACTIVE_INST_LDS", "SQ_WAVES",
                "SQ_BUSY_CYCLES", "SQ_WAVE_CYCLES", "SQ_WAIT_INST_ANY"):
        add("lds", key, "lds." + key)
    if per_kernel:
        cols = sorted({c for k in per_kernel.values() for c in k})
        md.append("## Counters per call (rocprofv3 --pmc, one pass per counter group)\n")
        md.append("| Kernel | " + " | ".join(cols) + " |\n|---|" + "---|" * len(cols))
        for name, k in per_kernel.items():
            md.append(f"| `{name}` | " + " | ".join("%.4g" % k.get(c, 0.0) for c in cols) + " |")
        md.append("")
        out["per_kernel"] = per_kernel
    call_ms = args.call_ms or out.get("call_ms_kernel_trace")
    if call_ms:
        md.append("Per call:\n")
        if "hbm_bytes_per_call" in out:
            md.append(f"* HBM read {out['hbm_read_bytes_per_call'] / 1e6:.1f} MB, written "
                      f"{out['hbm_write_bytes_per_call'] / 1e6:.1f} MB (FETCH_SIZE x{scale['FETCH_SIZE']:.4f}, "
                      f"WRITE_SIZE x{scale['WRITE_SIZE']:.4f}: the factors that make a plain {args.copy_mib} MiB "
                      f"device copy in the same run read and write {args.copy_mib} MiB); "
                      f"{out['hbm_bytes_per_call'] / (call_ms * 1e-3) / 1e9:.0f} GB/s of 8000")
        if out.get("valu_wave_insts_per_call"):
            v = out["valu_wave_insts_per_call"]
            md.append(f"* VALU wave-instructions {v:.4g}; issue {100 * v * 4 / (N_SIMD * PEAK_CLOCK * call_ms * 1e-3):.1f} % "
                      f"of 1024 SIMDs x 2.4 GHz over {call_ms:.4f} ms")
        if "valu_int32_lane_ops_per_call" in out:
            lo = out["valu_int32_lane_ops_per_call"]
            md.append(f"* INT32 lane-ops executed (INT32 wave-instructions x mean active lanes, per kernel): {lo:.4g}"
                      + (f", {lo / args.candidates:.0f} per candidate" if args.candidates else "")
                      + f"; {lo / (call_ms * 1e-3) / 1e12:.2f} Top/s = "
                        f"{100 * lo / (call_ms * 1e-3) / 1e12 / PEAK_INT32_TOPS:.1f} % of the 39.32 Top/s INT32 peak")
        md.append("")
    md.append("## Commands (repository root, one MI355X)\n")
    for c in args.commands:
        md.append("    " + c)
    md.append("\nSummary written by:\n\n    python bench.py " + " ".join(a if " " not in a else repr(a)
                                                                      for a in sys.argv[1:]))
    json.dump(out, open(os.path.join(PROFILES, tag + ".counters.json"), "w"), indent=1)
    open(os.path.join(PROFILES, tag + ".md"), "w").write("\n".join(md) + "\n")
    print(json.dumps({k: out[k] for k in out if k not in ("per_kernel", "kernels", "commands")}), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", type=int, default=5, choices=[3, 4, 5, 6])
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-early-stop", action="store_true")
    ap.add_argument("--es-chunk", type=int, default=ES_CHUNK,
                    help="early-stop chunk in candidates (0 = one chunk: every candidate against the warm-up bound)")
    ap.add_argument("--es-ramp", action="store_true", help="early-stop chunks double: es-chunk, 2 es-chunk, ...")
    ap.add_argument("--no-sub", action="store_true", help="headline workload only (no sub-records)")
    ap.add_argument("--schedule", default="1f1b", choices=["1f1b", "eager", "interleaved"],
                    help="pipeline schedule of the DAG (1F1B, Eager 1F1B, or Interleaved 1F1B with "
                         "the stages as virtual stages on S/2 devices; workloads 3 and 5)")
    ap.add_argument("--only", choices=["exhaustive", "early_stop"],
                    help="time one pass of --workload only (for profiling)")
    ap.add_argument("--search", action="store_true",
                    help="time the pruned configuration search over the whole 8-stage workload instead")
    ap.add_argument("--rows-per-chunk", type=int, default=512)
    ap.add_argument("--fixed-chunks", action="store_true",
                    help="with --search: every chunk has --rows-per-chunk rows (default: chunks of 1, 2, 4, ... rows "
                         "up to --rows-per-chunk)")
    ap.add_argument("--ridge", action="store_true", help="with --search: layer-level (ridge) pruning")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="with --only or --search: also run one plain device copy of this size (for counter "
                         "scaling)")
    # summaries of rocprofv3 output
    ap.add_argument("--summarize", metavar="DIR")
    ap.add_argument("--tag")
    ap.add_argument("--pass-kind", choices=sorted(PASS_KERNELS), default="exhaustive")
    ap.add_argument("--calls", type=int, default=0)
    ap.add_argument("--timed-calls", type=int, default=1)
    ap.add_argument("--call-ms", type=float, default=0.0)
    ap.add_argument("--candidates", type=int, default=0)
    ap.add_argument("--copy-mib", type=int, default=1024)
    ap.add_argument("--title", default="")
    ap.add_argument("--description", default="")
    ap.add_argument("--commands", nargs="*", default=[])
    args = ap.parse_args()
    if args.summarize:
        summarize(args)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported (the evaluation of "
              f"independent candidates would shard by index range)", file=sys.stderr)
        sys.exit(2)
    if args.search:
        search_bench(args)
        return
    if args.only:
        profile_only(args)
        return

    import torch
    dev = torch.device("cuda:0")
    wl = load_workload(args.workload, args.schedule)
    rec = eval_record(wl, dev, args, args.schedule, early_stop=not args.no_early_stop,
                      cpu_s=0.0 if args.no_cpu_baseline else args.cpu_seconds)
    prob = wl.problem
    out = {
        "metric": "candidate configs evaluated/sec + DAG nodes/sec (fraction of INT32 VALU peak)",
        "value": rec["candidates_per_s"],
        "unit": "candidates/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": rec["ms"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u32",
        "data": "synthetic (seeded per-layer profile tables and sampled candidates)",
        "config": {"workload": wl.description,
                   "schedule": {"eager": "Eager 1F1B", "interleaved": "Interleaved 1F1B (V = 2)"}.get(
                       args.schedule, "1F1B"),
                   "candidates_per_step": rec["candidates"], "dag_nodes_per_candidate": 2 * prob.S * prob.M,
                   "parallelism": "single GPU"},
        "dag_nodes_per_s": rec["dag_nodes_per_s"],
        "int32_valu_frac": rec["roofline"]["frac"],
        "best": rec["best"],
        "roofline": rec["roofline"],
        "early_stop": rec.get("early_stop"),
    }
    if "cpu_baseline" in rec:
        out["cpu_baseline"] = rec["cpu_baseline"]
        out["oracle_check"] = rec["oracle_check"]
    if not args.no_sub and args.workload == 5 and args.schedule == "1f1b":
        sub_cpu = 0.0 if args.no_cpu_baseline else max(2.0, args.cpu_seconds / 2)
        tiny_cpu = 0.0 if args.no_cpu_baseline else 0.5
        out["workloads"] = {
            "cfg1": eval_record(load_workload(1, "1f1b"), dev, args, early_stop=False, cpu_s=tiny_cpu,
                                py_s=tiny_cpu),
            "cfg2": eval_record(load_workload(2, "1f1b"), dev, args, early_stop=False, cpu_s=tiny_cpu,
                                py_s=tiny_cpu),
            "cfg3": eval_record(load_workload(3, "1f1b"), dev, args, early_stop=False, cpu_s=sub_cpu),
            "cfg4": eval_record(load_workload(4, "1f1b"), dev, args, early_stop=not args.no_early_stop,
                                cpu_s=sub_cpu),
        }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
