"""Write tests/golden/full_workloads.json from the CPU oracle only.

For each large workload (3, 4, 5, 6; 4 and 5 under Eager 1F1B, written "4e"
and "5e"; 5 under Interleaved 1F1B with 8 devices x 2 chunks, "5i") this
records, over every candidate:
the SHA-256 of the makespan array (uint32 little-endian), the SHA-256 of the
feasibility bit array packed as the library's output (bit i % 32 of uint32
word i / 32), the number of feasible candidates and the argmin.  For
workloads 4 and 6 it also records the early-stop pass: the warm-up bound (best of
the first 500 list entries) and, per chunk size, the oracle's
(best, evaluated, pruned, infeasible); likewise for 4e and 5e.
"4s" records the pruned search (Sec. 4.2.3) over every assignment row and
composition of workload 4, against that warm-up bound, in chunks that grow
1, 2, 4, ... rows up to 512: the best (joint index, makespan) and the five
counters, without and with the ridge filter.

Run from the repository root:  python tests/golden/make_golden.py [workload ...]
"""
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle import coracle  # noqa: E402
from paper_2609_06086_amd import workloads as W  # noqa: E402

OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "full_workloads.json")
WARMUP = 500
CHUNKS = (0, 1 << 22)


def pack_bits(f: np.ndarray) -> np.ndarray:
    pad = (-len(f)) % 32
    return np.packbits(np.concatenate([f.astype(bool), np.zeros(pad, bool)]), bitorder="little").view("<u4")


SEARCH_RPC = 512


def search_entry():
    wl = W.workload(4)
    c = wl.cands
    T, f = coracle.evaluate(wl.problem, W.Candidates(comp_rank=c.comp_rank[:WARMUP].copy(),
                                                     assign_idx=c.assign_idx[:WARMUP].copy()))
    bound = coracle.argmin(T, f)[1]
    ent = {"warmup": WARMUP, "bound": bound, "rows_per_chunk": SEARCH_RPC, "ramp": True}
    for name, ridge in (("plain", False), ("ridge", True)):
        t0 = time.time()
        r = coracle.search(wl.problem, bound, rows_per_chunk=SEARCH_RPC, ridge=ridge, ramp=True)
        ent[name] = {"best_index": r["best"][0], "best_makespan": r["best"][1],
                     **{k: r[k] for k in coracle.SEARCH_COUNTERS}, "oracle_seconds": round(time.time() - t0, 1)}
    return ent


def main():
    res = {"note": "written by tests/golden/make_golden.py from the C oracle; see that script"}
    only = sys.argv[1:] or ["3", "4", "5", "6", "4e", "5e", "5i", "4s"]
    if os.path.exists(OUT):
        res.update({k: v for k, v in json.load(open(OUT)).items() if k != "note"})
    for spec in only:
        if spec == "4s":
            res["cfg4_search"] = search_entry()
            print(spec, res["cfg4_search"], flush=True)
            continue
        eager, ilv = spec.endswith("e"), spec.endswith("i")
        cfg = int(spec.rstrip("ei"))
        wl = W.workload(cfg)
        if eager:
            wl.problem.schedule = 1   # Eager 1F1B
        if ilv:
            wl = W.interleaved_variant(wl, 2)
        t0 = time.time()
        T, f = coracle.evaluate(wl.problem, wl.cands)
        best = coracle.argmin(T, f)
        ent = {
            "n": int(len(T)),
            "makespan_sha256": hashlib.sha256(T.astype("<u4").tobytes()).hexdigest(),
            "feasible_bits_sha256": hashlib.sha256(pack_bits(f).astype("<u4").tobytes()).hexdigest(),
            "n_feasible": int(f.sum()),
            "best_index": best[0], "best_makespan": best[1],
            "makespan_min": int(T.min()), "makespan_max": int(T.max()),
        }
        if cfg in (4, 6) or eager:
            wb = coracle.argmin(T[:WARMUP], f[:WARMUP])
            bound = wb[1]
            ent["warmup"] = WARMUP
            ent["warmup_bound"] = bound
            ent["bounded"] = {}
            for ch in CHUNKS:
                b, ev, pr, inf = coracle.bounded(wl.problem, wl.cands, bound, ch)
                ent["bounded"][str(ch)] = {"best_index": b[0], "best_makespan": b[1], "evaluated": ev,
                                           "pruned": pr, "infeasible": inf}
        ent["oracle_seconds"] = round(time.time() - t0, 1)
        res[f"cfg{cfg}_eager" if eager else f"cfg{cfg}_interleaved" if ilv else f"cfg{cfg}"] = ent
        print(spec, ent, flush=True)
    with open(OUT, "w") as fh:
        json.dump(res, fh, indent=1)
        fh.write("\n")


if __name__ == "__main__":
    main()
