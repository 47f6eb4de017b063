/*
 * poseidon.h - batched evaluation of Poseidon's DAG-based training-time
 * model over many pipeline configurations, with a min-reduction to the best
 * one, on one AMD Instinct MI355X (gfx950).
 *
 * Model (Poseidon, arXiv 2609.06086, Sec. 4.1): a configuration places L
 * layers onto S pipeline stages (a composition of L into S positive parts)
 * and gives every stage a device type.  With M micro-batches, the 1F1B
 * schedule is a DAG of forward nodes F_{s,m} and backward nodes B_{s,m}
 * (Sec. 4.1.1), joined by inter-stage edges F_{s,m}->F_{s+1,m} and
 * B_{s+1,m}->B_{s,m} that carry the activation-transfer time, and by
 * zero-weight intra-stage edges along each stage's execution order
 * (Sec. 4.1.2).  A node weighs the stage's summed per-layer compute time on
 * its device type (Sec. 4.1.3).  The estimated iteration time T is the
 * critical path, the heaviest start-to-end path counting node and edge
 * weights (App. B.1).  A configuration is feasible when every stage's summed
 * per-layer memory fits the memory of its device type (Sec. 3.2).  The
 * search keeps the feasible configuration with the smallest T (Sec. 4.2.3);
 * Eq. 2 / Theorem 1 give a per-configuration lower bound used to skip
 * configurations that cannot beat the best one found so far.
 *
 * Under 1F1B, stage s of S runs min(S - s, M) forward passes, then
 * alternates one forward and one backward pass, then drains the remaining
 * backward passes (the common order; the paper does not spell out the
 * warm-up length).  Eager 1F1B (App. B.1) runs 2(S - s) + 1 warm-up
 * forwards and then alternates a backward and a forward pass.  Interleaved
 * 1F1B (Sec. 4.1.4) puts V model chunks on every device; see
 * poseidon_problem.V.  With data-parallel all-reduce times (Sec. 4.1.1,
 * 4.1.3) each stage (device) ends with an all-reduce node and T is the
 * latest of them.
 *
 * All times are integer microseconds and all memory sizes integer MB, held
 * in uint32; every result is exact integer arithmetic.
 *
 * Candidate indexing: compositions are ranked lexicographically by their
 * sorted cut tuple (c_1 < ... < c_{S-1}, stage s holds layers
 * [c_{s-1}, c_s) with c_0 = 0, c_S = L); assignment a is row a of the
 * caller's table, or, without a table, the base-T digits of a with stage 1
 * the most significant digit.  In range mode candidate i of a call is the
 * joint index first + i = comp_rank * A + a; in list mode it is the pair
 * (comp_rank[i], assign_idx[i]).  "index" in results of the evaluation
 * calls is the joint index first + i in range mode and the position i in
 * list mode; either way, among candidates with equal makespans the smallest
 * index wins.  The search (poseidon_search) enumerates in its own order,
 * assignment row first, and reports the first optimum in that order.
 *
 * Errors: 0 = OK, 1 = POSEIDON_NO_FEASIBLE (the call completed but no
 * candidate qualified; best.index = UINT64_MAX), negative = error.  All
 * argument checks happen before any HIP call; nothing aborts or throws
 * across this interface.  A context is not thread-safe: use one per host
 * thread / stream.  Calls enqueue work on `hip_stream` (a hipStream_t; NULL
 * = the default stream); calls given a host result pointer synchronise that
 * stream before returning.
 */
#ifndef POSEIDON_H
#define POSEIDON_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define POSEIDON_S_MAX 16   /* stages */
#define POSEIDON_L_MAX 256  /* layers */
#define POSEIDON_T_MAX 8    /* device types */
#define POSEIDON_M_MAX (1u << 20)   /* micro-batches: the schedule the kernels hard-code is
                                       checked against a simulation for every M up to this */

/* Pipeline schedules (poseidon_problem.schedule). */
enum {
    POSEIDON_SCHEDULE_1F1B = 0,        /* min(S-s, M) warm-up forwards, then (F, B) pairs */
    POSEIDON_SCHEDULE_EAGER_1F1B = 1,  /* min(2(S-s)+1, M) warm-up forwards, then (B, F)
                                          pairs (App. B.1) */
    POSEIDON_SCHEDULE_INTERLEAVED_1F1B = 2  /* V model chunks per device (Sec. 4.1.4); see
                                               poseidon_problem.V */
};

enum {
    POSEIDON_OK = 0,
    POSEIDON_NO_FEASIBLE = 1,
    POSEIDON_E_INVAL = -1,   /* null pointer, bad size, type id >= T, ... */
    POSEIDON_E_RANGE = -2,   /* a makespan could exceed 2^31, or a count 2^64 */
    POSEIDON_E_DEVICE = -3,  /* a HIP call failed */
    POSEIDON_E_NOMEM = -4    /* host or device allocation failed */
};

typedef struct poseidon_ctx poseidon_ctx;

/* Per-layer profile of one model on T device types (Sec. 4.1.3): all
 * HOST pointers, read during poseidon_load_costs only. */
typedef struct {
    uint32_t L, S, M, T;          /* 1 <= S <= min(L, S_MAX), 1 <= M <= M_MAX, 1 <= T <= T_MAX */
    const uint32_t *fwd_us;       /* [T][L] forward time of layer l on type t */
    const uint32_t *bwd_us;       /* [T][L] backward time */
    const uint32_t *comm_fwd_us;  /* [S-1] weight of F_{b,m}->F_{b+1,m} (NULL iff S == 1) */
    const uint32_t *comm_bwd_us;  /* [S-1] weight of B_{b+1,m}->B_{b,m} (NULL iff S == 1) */
    const uint32_t *mem_mb;       /* [L] memory footprint of layer l */
    const uint32_t *cap_mb;       /* [T] memory of one device of type t */
    const uint8_t *assign;        /* [A][S] allowed stage->type rows, or NULL = all T^S */
    uint64_t A;                   /* rows of `assign` (ignored when assign == NULL) */
    const uint32_t *allreduce_us; /* [T][L] data-parallel gradient all-reduce time of layer l on
                                     type t, or NULL = none.  Stage s's all-reduce node R_s
                                     weighs the sum over its layers and follows B_{s,M};
                                     T = max_s(finish(B_{s,M}) + R_s) (Sec. 4.1.1, 4.1.3) */
    uint32_t schedule;            /* POSEIDON_SCHEDULE_*: the intra-stage order of the DAG
                                     (Sec. 4.1.4: other schedules change only the intra-stage
                                     edges) */
    uint32_t V;                   /* Interleaved 1F1B only (ignored otherwise): model chunks per
                                     device, V >= 2.  S then counts virtual stages (the
                                     composition has S parts); the N = S / V >= 2 devices each
                                     hold V of them, virtual stage j (0-based) on device j mod N;
                                     M must be a multiple of N.  Device p (0-based) runs
                                     Megatron-LM's interleaved order: forward step k runs chunk
                                     (k mod VN) div N on micro-batch (k div VN) N + k mod N + 1,
                                     backward step k chunk V-1 - (k mod VN) div N; a warm-up of
                                     min(2(N-p-1) + (V-1)N, VM) forward steps (all if M = N), then
                                     (forward, backward) pairs, then the remaining backwards.
                                     `assign` rows, base-T digits and memory caps are per device
                                     (a device's memory and all-reduce sum over all its chunks);
                                     comm arrays have S-1 entries, one per virtual boundary.
                                     The early-stop pass and the search reject such problems
                                     (Eq. 2 is stated for one stage per device). */
} poseidon_problem;

/* Candidates of one call.  comp_rank == NULL: range mode over joint indices
 * [first, first + count).  Otherwise list mode: `count` DEVICE arrays
 * comp_rank[count] (uint64) and assign_idx[count] (uint32, or NULL meaning
 * assignment 0); `first` is ignored.  count < 2^32 per call. */
typedef struct {
    uint64_t first, count;
    const uint64_t *comp_rank;
    const uint32_t *assign_idx;
} poseidon_cands;

typedef struct {
    uint64_t index;     /* range mode: joint index first + i; list mode: position i;
                           UINT64_MAX if none */
    uint32_t makespan;  /* critical-path length T in microseconds */
    uint32_t feasible;  /* 1 if every stage fits its memory cap */
} poseidon_best;

typedef struct {
    uint64_t evaluated;   /* feasible candidates whose DAG was evaluated */
    uint64_t pruned;      /* feasible candidates skipped by the Eq. 2 bound */
    uint64_t infeasible;  /* candidates over a memory cap (never evaluated) */
} poseidon_prune_stats;

/* Check a problem without touching the GPU and return the number of
 * candidates C(L-1, S-1) * A (Sec. 4.2.3: the search space of layer
 * allocations and device assignments).  Pure host code. */
int poseidon_validate(const poseidon_problem *problem, uint64_t *n_candidates);

/* Copy the profile tables to device `hip_device` and build the lookup
 * tables every candidate evaluation shares: per-type prefix sums of the
 * per-layer costs and memory, the Pascal table used to unrank compositions
 * (with, per column, the row each search starts from for each value range),
 * and the slot schedule of the problem's DAG for (S, M) and its schedule
 * (Sec. 5: the DAG depends only on the pipeline depth, so it is built once
 * and only re-weighted).  For every problem, the slot pattern the kernels
 * hard-code (1F1B with M >= S, Eager 1F1B with M >= 2S-1) is compared slot
 * by slot with a simulation of the unit-weight schedule, and the
 * Interleaved 1F1B program with the problem's own slot table; a mismatch
 * fails with POSEIDON_E_INVAL.  Fails
 * with POSEIDON_E_RANGE if some candidate's makespan could reach 2^31.  The
 * caller may free the host tables after return; the context owns its device
 * memory until poseidon_free. */
int poseidon_load_costs(const poseidon_problem *problem, int hip_device, poseidon_ctx **out);

/* Evaluate every candidate of `cands` (Sec. 4.1: stage weights, longest path
 * of the schedule's DAG; Sec. 3.2 memory feasibility) and reduce to the feasible
 * candidate with the smallest makespan, ties to the smaller index.
 * makespan_out: DEVICE uint32[count] or NULL; gets every candidate's raw T,
 *   feasible or not.
 * feasible_bits_out: DEVICE uint32[ceil(count/32)] or NULL; bit i % 32 of
 *   word i / 32 is candidate i's feasibility.
 * best_out: HOST pointer or NULL.  Non-NULL synchronises the stream and
 *   returns the best; NULL leaves it on the device for
 *   poseidon_last_best.  Returns POSEIDON_NO_FEASIBLE if no candidate fits. */
int poseidon_eval_candidates(poseidon_ctx *ctx, const poseidon_cands *cands,
                             uint32_t *makespan_out, uint32_t *feasible_bits_out,
                             poseidon_best *best_out, void *hip_stream);

/* The same evaluation as poseidon_eval_candidates (same arguments, outputs,
 * index and status semantics), for callers that cannot allocate device
 * memory during the call: code under stream capture, tight serving loops,
 * harnesses that forbid hipMalloc.  It allocates nothing.  Instead of the
 * context's workspace it uses a fixed scratch array of
 * POSEIDON_NOALLOC_SCRATCH_BYTES that the library holds once per GPU (from
 * its first poseidon_load_costs on that GPU until the process ends), and it
 * processes the call in chunks sized so that the cut codes and straggler
 * queues of one chunk fit that array (2^18 candidates per chunk for
 * S = 16 under 1F1B, 2^17 under Eager 1F1B; more chunks mean more launches
 * than poseidon_eval_candidates needs).  Nothing in the scratch needs clearing:
 * every word a kernel reads was written earlier in the same chunk.  All
 * calls on one GPU share its array, so calls of this function that overlap
 * in time on one GPU (other threads, other streams) race and give wrong
 * results; serialise them.  Returns POSEIDON_E_RANGE if even the smallest
 * chunk of the problem does not fit the scratch, POSEIDON_E_DEVICE if the
 * scratch could not be located on the context's GPU. */
#define POSEIDON_NOALLOC_SCRATCH_BYTES (64u << 20)
int poseidon_eval_candidates_noalloc(poseidon_ctx *ctx, const poseidon_cands *cands,
                                     uint32_t *makespan_out, uint32_t *feasible_bits_out,
                                     poseidon_best *best_out, void *hip_stream);

/* Result of the most recent poseidon_eval_candidates (or poseidon_argmin)
 * on this context, with the index as that call reported it (synchronises
 * the stream). */
int poseidon_last_best(poseidon_ctx *ctx, poseidon_best *best_out, void *hip_stream);

/* Early-stop search (Eq. 2, Theorem 1).  The candidates are processed in
 * consecutive chunks of `chunk` entries (0 = one chunk); with flag
 * POSEIDON_BOUNDED_RAMP the chunks grow instead as chunk, 2 chunk, 4 chunk,
 * ... entries, so that an early chunk sets a bound soon and the later ones
 * pay the fixed cost of a chunk (one pass of the filter and survivor kernels)
 * fewer times.  Within a chunk,
 * a feasible candidate whose lower bound max_x g(S_x) exceeds
 * b = min(bound, best makespan found in earlier chunks) is skipped; all
 * other feasible candidates are evaluated exactly.  The reduction is the
 * same as poseidon_eval_candidates', over evaluated candidates; if its
 * makespan is > bound the call returns POSEIDON_NO_FEASIBLE.  The result
 * is deterministic for a given chunk size and flags.  best_out and
 * stats_out are HOST pointers (either may be NULL); the call synchronises
 * the stream.  POSEIDON_E_INVAL for Interleaved 1F1B problems or unknown
 * flags. */
#define POSEIDON_BOUNDED_RAMP 1u
int poseidon_eval_candidates_bounded(poseidon_ctx *ctx, const poseidon_cands *cands,
                                     uint32_t bound, uint64_t chunk, uint32_t flags,
                                     poseidon_best *best_out, poseidon_prune_stats *stats_out,
                                     void *hip_stream);

/* Argmin over arrays a previous evaluation wrote (DEVICE pointers,
 * `count` entries, layouts as for poseidon_eval_candidates; feasible_bits
 * may be NULL = all feasible).  best_out->index = index_base + position.
 * HOST best_out, required; synchronises the stream. */
int poseidon_argmin(poseidon_ctx *ctx, const uint32_t *makespan, const uint32_t *feasible_bits,
                    uint64_t count, uint64_t index_base, poseidon_best *best_out,
                    void *hip_stream);

/* Pruned configuration search (Sec. 4.2.3).  For every assignment row a in
 * [first_row, first_row + n_rows) (rows of the table, or base-T digits), the
 * layers are allocated stage by stage, smaller layer counts first, and a
 * partial configuration S_x (stages 1..x fixed) is discarded with all its
 * extensions when stage x exceeds the memory of its device type, when
 * (flag POSEIDON_SEARCH_RIDGE, layer-level pruning, Theorem 2) the layer
 * counts of the stages of some device type are no longer ridge-like
 * (non-decreasing, then non-increasing), or when g(S_x) of Eq. 2 exceeds the
 * bound (stage-level pruning, Theorem 1; off with
 * POSEIDON_SEARCH_NO_STAGE_PRUNING).  Complete configurations that pass are
 * evaluated on the DAG.
 * The rows are processed in consecutive chunks of rows_per_chunk rows
 * (0 = one chunk), or with POSEIDON_SEARCH_RAMP in chunks that grow 1, 2,
 * 4, ... rows until they reach rows_per_chunk; a chunk prunes against
 * min(bound, best makespan of the earlier chunks), so every counter is
 * deterministic for a given chunking.  Small first chunks tighten the
 * bound early; large later ones need fewer levels of launches per row.
 * Result: among feasible (and, with the ridge flag, ridge-like) candidates
 * of the rows with makespan <= bound, the smallest makespan, ties to the
 * first in search order (row, then composition rank); best_out->index is
 * its joint index rank * A + row.  Theorem 1 makes it the exhaustive
 * optimum of those candidates.  POSEIDON_NO_FEASIBLE if there is none.
 * best_out and stats_out are HOST pointers (either may be NULL); the call
 * synchronises the stream wherever it reads a level's size back (levels
 * that may need more than one frontier piece) and at its end.  The frontier
 * memory, 4 Mi partial configurations per stage of (6 + 4 ceil((S-1)/4))
 * bytes each (1.5 GB at S = 16), is allocated on the first call and kept by
 * the context.  The work grows with the pruned tree, which for many stages
 * and a loose bound can be very large (Sec. 4.2.3). */
enum {
    POSEIDON_SEARCH_RIDGE = 1,               /* layer-level pruning (Theorem 2) */
    POSEIDON_SEARCH_NO_STAGE_PRUNING = 2,    /* no Eq. 2 test on partial configurations */
    POSEIDON_SEARCH_RAMP = 4                 /* chunks of 1, 2, 4, ... rows up to rows_per_chunk */
};

typedef struct {
    uint64_t visited;         /* partial or complete configurations accepted at a stage */
    uint64_t evaluated;       /* complete configurations evaluated on the DAG */
    uint64_t pruned_memory;   /* stage choices cut by a memory cap */
    uint64_t pruned_ridge;    /* stage choices cut by the ridge test */
    uint64_t pruned_bound;    /* stage choices cut by g(S_x) > bound */
} poseidon_search_stats;

int poseidon_search(poseidon_ctx *ctx, uint64_t first_row, uint64_t n_rows, uint32_t bound,
                    uint64_t rows_per_chunk, uint32_t flags, poseidon_best *best_out,
                    poseidon_search_stats *stats_out, void *hip_stream);

/* Release the context's device memory.  NULL is ignored. */
void poseidon_free(poseidon_ctx *ctx);

/* Static text for a status code. */
const char *poseidon_strerror(int status);

#ifdef __cplusplus
}
#endif

#endif /* POSEIDON_H */
