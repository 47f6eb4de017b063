/*
 * CPU oracle for Poseidon's DAG-based training-time model, multithreaded C.
 *
 * TEST INFRASTRUCTURE.  Only the test-suite, the smoke check and the
 * CPU-baseline leg of the benchmark may load this library.  It shares no
 * code, header or table with the HIP library; it is the paper's definition
 * written out plainly so that large workloads can be checked on the host.
 *
 *  - DAG (Poseidon, Sec. 4.1.1-4.1.2): compute nodes F_{s,m}, B_{s,m}; one
 *    all-reduce node R_s per stage (Sec. 4.1.3: per-layer all-reduce time
 *    summed over the stage, or 0 without a table); start node and end node.  Inter-stage edges F_{s,m}->F_{s+1,m} and
 *    B_{s+1,m}->B_{s,m}; intra-stage edges along each stage's 1F1B order;
 *    B_{s,M}->R_s; start->F_{1,1}; R_s->end.  The topology depends only on
 *    (S, M) and is built once (Sec. 5, simulator design), then ordered with
 *    Kahn's algorithm.
 *  - 1F1B order (reading of Sec. 4.1.2; the paper does not state the warm-up
 *    length): stage s runs w = min(S - s, M) forwards, then (F_{w+i}, B_i)
 *    for i = 1..M-w, then the remaining backwards.  Eager 1F1B (App. B.1):
 *    w = min(2(S - s) + 1, M) forwards, then (B_i, F_{w+i}) for
 *    i = 1..M-w, then the remaining backwards.
 *  - Weights (Sec. 4.1.3): F_{s,m} = sum of the stage's per-layer forward
 *    times on its device type, likewise B_{s,m}; inter-stage edges carry the
 *    per-boundary transfer time; all other edges and control nodes weigh 0.
 *  - Makespan = critical path (App. B.1): finish(v) = w(v) + max(0, max over
 *    predecessors u of finish(u) + w(u,v)), T = finish(end).
 *  - Feasibility (reading of Sec. 3.2): every stage's summed layer memory
 *    <= the cap of its device type.
 *  - Candidates: lexicographic rank of the sorted cut tuple (unranked with a
 *    Pascal table), assignment row or base-T digits (stage 1 most
 *    significant); range mode index = rank * A + a.
 *  - Early stop (Eq. 2, Theorem 1): g(S_x) = sum_{i<x} F_i + M (F_x + B_x)
 *    + max_{1<=i<=x} (sum_{j=i}^{x-1} B_j + d_i), d_i = stage all-reduce
 *    time; prune iff max_x g > b.
 *  - Pruned search (Sec. 4.2.3; readings R16-R19 of oracle/search.py): per
 *    assignment row, layers are allocated stage by stage, smaller counts
 *    first; a stage choice is cut (with every larger count) when the stage
 *    exceeds its memory cap, when a type's layer counts stop being
 *    ridge-like (Theorem 2, with layer-level pruning on), or when g(S_x)
 *    exceeds the chunk's bound (Theorem 1).  Rows are processed in chunks
 *    with a fixed bound per chunk; the result is the first candidate in
 *    (row, rank) order with the smallest makespan <= bound.
 *
 * Finish times are held in 64-bit integers, so no intermediate can wrap.
 */
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
    uint32_t L, S, M, T;
    const uint32_t *fwd, *bwd;     /* [T][L] */
    const uint32_t *cf, *cb;       /* [S-1] */
    const uint32_t *mem;           /* [L] */
    const uint32_t *cap;           /* [T] */
    const uint8_t *assign;         /* [A][S] or NULL (all T^S rows) */
    uint64_t A;
    const uint32_t *allreduce;     /* [T][L] or NULL (no DP all-reduce) */
    uint32_t schedule;             /* 0 = 1F1B, 1 = Eager 1F1B, 2 = Interleaved 1F1B */
    uint32_t V;                    /* model chunks per device (Interleaved 1F1B) */
} oc_problem;

enum { K_F = 0, K_B = 1, K_R = 2, K_START = 3, K_END = 4 };
enum { E_ZERO = 0, E_FWD = 1, E_BWD = 2 };

typedef struct {
    int kind, stage;               /* stage 1-based for F/B/R */
    int npred;
    int pred[2];                   /* compute nodes have <= 2 predecessors */
    int ekind[2];
    int eb[2];                     /* boundary index (0-based) of a weighted edge */
    int *xpred;                    /* end node: S predecessors */
} oc_node;

typedef struct {
    int S, M, n;
    int ND;                        /* devices: all-reduce nodes and end-node predecessors */
    oc_node *nodes;
    int *topo;
    int end;
} oc_dag;

static int idF(int M, int s, int m) { return 2 * ((s - 1) * M + (m - 1)); }
static int idB(int M, int s, int m) { return 2 * ((s - 1) * M + (m - 1)) + 1; }

static void add_pred(oc_node *v, int u, int ek, int b) {
    v->pred[v->npred] = u;
    v->ekind[v->npred] = ek;
    v->eb[v->npred] = b;
    v->npred++;
}

static void dag_free(oc_dag *g) {
    if (!g) return;
    if (g->nodes) free(g->nodes[g->end].xpred);
    free(g->nodes);
    free(g->topo);
    free(g);
}

/* Order of stage s as (kind, m) pairs written to ko/mo (2M entries). */
static void stage_order(int S, int M, int s, int schedule, int *ko, int *mo) {
    int w, k = 0;
    if (schedule == 1) w = 2 * (S - s) + 1 < M ? 2 * (S - s) + 1 : M;
    else w = S - s < M ? S - s : M;
    for (int m = 1; m <= w; ++m) { ko[k] = K_F; mo[k] = m; ++k; }
    for (int i = 1; i <= M - w; ++i) {
        if (schedule == 1) {
            ko[k] = K_B; mo[k] = i; ++k;
            ko[k] = K_F; mo[k] = w + i; ++k;
        } else {
            ko[k] = K_F; mo[k] = w + i; ++k;
            ko[k] = K_B; mo[k] = i; ++k;
        }
    }
    for (int m = M - w + 1; m <= M; ++m) { ko[k] = K_B; mo[k] = m; ++k; }
}

/* Interleaved 1F1B order of device p (1-based) of N, V chunks each: (kind,
 * virtual stage, m) triples (2VM entries); see oracle/dag.py, reading R20. */
static void interleaved_order(int N, int V, int M, int p, int *ko, int *jo, int *mo) {
    int q = p - 1, total = V * M, k = 0;
    int w = M == N ? total : (2 * (N - q - 1) + (V - 1) * N < total ? 2 * (N - q - 1) + (V - 1) * N : total);
#define IL_MB(x) (((x) / (N * V)) * N + (x) % N + 1)
#define IL_FC(x) (((x) % (N * V)) / N)
    for (int x = 0; x < w; ++x) { ko[k] = K_F; jo[k] = IL_FC(x) * N + q + 1; mo[k] = IL_MB(x); ++k; }
    for (int i = 0; i < total - w; ++i) {
        int x = w + i;
        ko[k] = K_F; jo[k] = IL_FC(x) * N + q + 1; mo[k] = IL_MB(x); ++k;
        ko[k] = K_B; jo[k] = (V - 1 - IL_FC(i)) * N + q + 1; mo[k] = IL_MB(i); ++k;
    }
    for (int x = total - w; x < total; ++x) {
        ko[k] = K_B; jo[k] = (V - 1 - IL_FC(x)) * N + q + 1; mo[k] = IL_MB(x); ++k;
    }
#undef IL_MB
#undef IL_FC
}

static oc_dag *dag_build(int S, int M, int schedule, int V) {
    oc_dag *g = calloc(1, sizeof(oc_dag));
    if (!g) return NULL;
    int ncomp = 2 * S * M;
    const int interleaved = schedule == 2;
    const int ND = interleaved ? S / V : S;
    g->S = S; g->M = M; g->ND = ND;
    g->n = ncomp + ND + 2;
    int start = ncomp + ND;
    g->end = ncomp + ND + 1;
    g->nodes = calloc((size_t)g->n, sizeof(oc_node));
    g->topo = malloc(sizeof(int) * (size_t)g->n);
    size_t olen = 2 * (size_t)M * (size_t)(interleaved ? V : 1);
    int *ko = malloc(sizeof(int) * olen), *mo = malloc(sizeof(int) * olen), *jo = malloc(sizeof(int) * olen);
    int *indeg = calloc((size_t)g->n, sizeof(int));
    int *queue = malloc(sizeof(int) * (size_t)g->n);
    if (!g->nodes || !g->topo || !ko || !mo || !jo || !indeg || !queue) {
        free(ko); free(mo); free(jo); free(indeg); free(queue); dag_free(g); return NULL;
    }
    for (int s = 1; s <= S; ++s)
        for (int m = 1; m <= M; ++m) {
            g->nodes[idF(M, s, m)].kind = K_F; g->nodes[idF(M, s, m)].stage = s;
            g->nodes[idB(M, s, m)].kind = K_B; g->nodes[idB(M, s, m)].stage = s;
        }
    for (int s = 1; s <= ND; ++s) { g->nodes[ncomp + s - 1].kind = K_R; g->nodes[ncomp + s - 1].stage = s; }
    g->nodes[start].kind = K_START;
    g->nodes[g->end].kind = K_END;
    /* inter-stage edges */
    for (int m = 1; m <= M; ++m)
        for (int s = 1; s < S; ++s) {
            add_pred(&g->nodes[idF(M, s + 1, m)], idF(M, s, m), E_FWD, s - 1);
            add_pred(&g->nodes[idB(M, s, m)], idB(M, s + 1, m), E_BWD, s - 1);
        }
    /* intra-stage edges along each device's order; the device's all-reduce
     * node follows its last node */
    for (int p = 1; p <= ND; ++p) {
        int len;
        if (interleaved) {
            interleaved_order(ND, V, M, p, ko, jo, mo);
            len = 2 * V * M;
        } else {
            stage_order(S, M, p, schedule, ko, mo);
            for (int k = 0; k < 2 * M; ++k) jo[k] = p;
            len = 2 * M;
        }
        for (int k = 1; k < len; ++k) {
            int u = ko[k - 1] == K_F ? idF(M, jo[k - 1], mo[k - 1]) : idB(M, jo[k - 1], mo[k - 1]);
            int v = ko[k] == K_F ? idF(M, jo[k], mo[k]) : idB(M, jo[k], mo[k]);
            add_pred(&g->nodes[v], u, E_ZERO, 0);
        }
        int last = ko[len - 1] == K_F ? idF(M, jo[len - 1], mo[len - 1]) : idB(M, jo[len - 1], mo[len - 1]);
        add_pred(&g->nodes[ncomp + p - 1], last, E_ZERO, 0);
    }
    add_pred(&g->nodes[idF(M, 1, 1)], start, E_ZERO, 0);
    g->nodes[g->end].xpred = malloc(sizeof(int) * (size_t)ND);
    for (int s = 1; s <= ND; ++s) g->nodes[g->end].xpred[s - 1] = ncomp + s - 1;
    /* Kahn */
    for (int v = 0; v < g->n; ++v) {
        oc_node *nv = &g->nodes[v];
        indeg[v] = nv->kind == K_END ? ND : nv->npred;
    }
    int head = 0, tail = 0, cnt = 0;
    for (int v = 0; v < g->n; ++v) if (indeg[v] == 0) queue[tail++] = v;
    /* successor scan: simple O(n^2)-free approach via reverse lists */
    int *succ_cnt = calloc((size_t)g->n, sizeof(int));
    for (int v = 0; v < g->n; ++v) {
        oc_node *nv = &g->nodes[v];
        int np = nv->kind == K_END ? ND : nv->npred;
        for (int i = 0; i < np; ++i) succ_cnt[nv->kind == K_END ? nv->xpred[i] : nv->pred[i]]++;
    }
    int *succ_off = malloc(sizeof(int) * ((size_t)g->n + 1));
    succ_off[0] = 0;
    for (int v = 0; v < g->n; ++v) succ_off[v + 1] = succ_off[v] + succ_cnt[v];
    int *succ = malloc(sizeof(int) * (size_t)(succ_off[g->n] + 1));
    memset(succ_cnt, 0, sizeof(int) * (size_t)g->n);
    for (int v = 0; v < g->n; ++v) {
        oc_node *nv = &g->nodes[v];
        int np = nv->kind == K_END ? ND : nv->npred;
        for (int i = 0; i < np; ++i) {
            int u = nv->kind == K_END ? nv->xpred[i] : nv->pred[i];
            succ[succ_off[u] + succ_cnt[u]++] = v;
        }
    }
    while (head < tail) {
        int u = queue[head++];
        g->topo[cnt++] = u;
        for (int i = succ_off[u]; i < succ_off[u + 1]; ++i)
            if (--indeg[succ[i]] == 0) queue[tail++] = succ[i];
    }
    free(succ_cnt); free(succ_off); free(succ);
    free(ko); free(mo); free(jo); free(indeg); free(queue);
    if (cnt != g->n) { dag_free(g); return NULL; }
    return g;
}

/* finish times: caller-provided scratch of g->n uint64 */
static uint64_t dag_longest(const oc_dag *g, const uint64_t *F, const uint64_t *B, const uint64_t *D,
                            const uint32_t *cf, const uint32_t *cb, uint64_t *fin) {
    for (int i = 0; i < g->n; ++i) {
        int v = g->topo[i];
        const oc_node *nv = &g->nodes[v];
        uint64_t best = 0, w = 0;
        if (nv->kind == K_END) {
            for (int j = 0; j < g->ND; ++j) if (fin[nv->xpred[j]] > best) best = fin[nv->xpred[j]];
        } else {
            for (int j = 0; j < nv->npred; ++j) {
                uint64_t c = fin[nv->pred[j]];
                if (nv->ekind[j] == E_FWD) c += cf[nv->eb[j]];
                else if (nv->ekind[j] == E_BWD) c += cb[nv->eb[j]];
                if (c > best) best = c;
            }
        }
        if (nv->kind == K_F) w = F[nv->stage - 1];
        else if (nv->kind == K_B) w = B[nv->stage - 1];
        else if (nv->kind == K_R) w = D[nv->stage - 1];
        fin[v] = w + best;
    }
    return fin[g->end];
}

/* Pascal table C(n, k), n <= L-1, k <= S-1, saturating at UINT64_MAX */
static uint64_t *pascal(int nmax, int kmax) {
    uint64_t *c = calloc((size_t)(nmax + 1) * (size_t)(kmax + 1), sizeof(uint64_t));
    if (!c) return NULL;
    for (int n = 0; n <= nmax; ++n)
        for (int k = 0; k <= kmax; ++k) {
            uint64_t v;
            if (k == 0) v = 1;
            else if (n == 0) v = 0;
            else {
                uint64_t a = c[(size_t)(n - 1) * (kmax + 1) + k - 1], b = c[(size_t)(n - 1) * (kmax + 1) + k];
                v = a + b;
                if (v < a) v = UINT64_MAX;
            }
            c[(size_t)n * (kmax + 1) + k] = v;
        }
    return c;
}

typedef struct {
    const oc_problem *p;
    const oc_dag *g;
    const uint64_t *binom;
    uint64_t first, count;
    const uint64_t *rank;
    const uint32_t *aidx;
    uint32_t *out_T;
    uint8_t *out_feas;
    uint64_t lo, hi;          /* slice of [0, count) */
    /* bounded mode */
    int bounded;
    uint64_t bound;
    uint64_t best_key_T, best_idx;
    uint64_t evaluated, pruned, infeasible;
    int err;
} oc_job;

/* decode candidate i: cut points (c_0 = 0 ... c_S = L) and stage types */
static int decode(const oc_job *j, uint64_t i, int *cuts, int *types) {
    const oc_problem *p = j->p;
    uint64_t r, a;
    if (j->rank) {
        r = j->rank[i];
        a = j->aidx ? j->aidx[i] : 0;
    } else {
        uint64_t idx = j->first + i;
        r = idx / p->A;
        a = idx % p->A;
    }
    if (a >= p->A) return -1;
    int S = (int)p->S, L = (int)p->L, k = S - 1;
    if (r >= j->binom[(size_t)(L - 1) * (k + 1) + k]) return -1;
    cuts[0] = 0;
    int v = 0;
    for (int jj = 1; jj <= k; ++jj) {
        ++v;
        for (;;) {
            uint64_t cnt = j->binom[(size_t)(L - 1 - v) * (k + 1) + (k - jj)];
            if (r < cnt) { cuts[jj] = v; break; }
            r -= cnt;
            ++v;
        }
    }
    cuts[S] = L;
    int ND = p->schedule == 2 ? S / (int)p->V : S;   /* one type per device */
    if (p->assign) {
        for (int s = 0; s < ND; ++s) types[s] = p->assign[a * ND + s];
    } else {
        for (int s = ND - 1; s >= 0; --s) { types[s] = (int)(a % p->T); a /= p->T; }
    }
    for (int s = 0; s < ND; ++s) if (types[s] >= (int)p->T) return -1;
    return 0;
}

static void *worker(void *arg) {
    oc_job *j = arg;
    const oc_problem *p = j->p;
    int S = (int)p->S;
    int cuts[65], types[64];
    uint64_t F[64], B[64], D[64];
    uint64_t *fin = malloc(sizeof(uint64_t) * (size_t)j->g->n);
    if (!fin) { j->err = -3; return NULL; }
    j->best_key_T = UINT64_MAX; j->best_idx = UINT64_MAX;
    for (uint64_t i = j->lo; i < j->hi; ++i) {
        if (decode(j, i, cuts, types)) { j->err = -1; break; }
        int feasible = 1;
        /* Interleaved 1F1B: virtual stage s runs on device s mod ND; memory
         * and all-reduce are summed per device (reading R20) */
        int ND = p->schedule == 2 ? S / (int)p->V : S;
        uint64_t MM[64];
        for (int q = 0; q < ND; ++q) { D[q] = 0; MM[q] = 0; }
        for (int s = 0; s < S; ++s) {
            int q = s % ND, t = types[q];
            uint64_t f = 0, b = 0, mm = 0, d = 0;
            for (int l = cuts[s]; l < cuts[s + 1]; ++l) {
                f += p->fwd[(size_t)t * p->L + l];
                b += p->bwd[(size_t)t * p->L + l];
                mm += p->mem[l];
                if (p->allreduce) d += p->allreduce[(size_t)t * p->L + l];
            }
            F[s] = f; B[s] = b; D[q] += d; MM[q] += mm;
        }
        for (int q = 0; q < ND; ++q) if (MM[q] > p->cap[types[q]]) feasible = 0;
        if (j->bounded) {
            /* reading R10: stage by stage in pipeline order, the first stage
             * over its device's memory (infeasible) or with g(S_x) of Eq. 2
             * above the bound (pruned) decides; memory first (one stage per
             * device here: no early stop under Interleaved 1F1B) */
            int cls = 0;
            for (int x = 1; x <= S && !cls; ++x) {
                if (MM[x - 1] > p->cap[types[x - 1]]) { cls = 1; break; }
                uint64_t g = 0, inner = 0;
                for (int i2 = 1; i2 < x; ++i2) g += F[i2 - 1];
                g += (uint64_t)p->M * (F[x - 1] + B[x - 1]);
                for (int i2 = 1; i2 <= x; ++i2) {
                    uint64_t sb = D[i2 - 1];
                    for (int jj = i2; jj <= x - 1; ++jj) sb += B[jj - 1];
                    if (sb > inner) inner = sb;
                }
                if (g + inner > j->bound) cls = 2;
            }
            if (cls == 1) { j->infeasible++; continue; }
            if (cls == 2) { j->pruned++; continue; }
            j->evaluated++;
        }
        uint64_t T = dag_longest(j->g, F, B, D, p->cf, p->cb, fin);
        if (T > UINT32_MAX) { j->err = -2; break; }
        if (j->out_T) j->out_T[i] = (uint32_t)T;
        if (j->out_feas) j->out_feas[i] = (uint8_t)feasible;
        if (j->bounded && (T < j->best_key_T || (T == j->best_key_T && i < j->best_idx))) {
            j->best_key_T = T; j->best_idx = i;
        }
    }
    free(fin);
    return NULL;
}

static int run_jobs(oc_job *proto, uint64_t lo, uint64_t hi, int nthreads, oc_job *jobs) {
    pthread_t th[256];
    if (nthreads < 1) nthreads = 1;
    if (nthreads > 256) nthreads = 256;
    uint64_t n = hi - lo;
    if ((uint64_t)nthreads > n) nthreads = n ? (int)n : 1;
    for (int t = 0; t < nthreads; ++t) {
        jobs[t] = *proto;
        jobs[t].lo = lo + n * (uint64_t)t / (uint64_t)nthreads;
        jobs[t].hi = lo + n * (uint64_t)(t + 1) / (uint64_t)nthreads;
        jobs[t].evaluated = jobs[t].pruned = jobs[t].infeasible = 0;
        jobs[t].err = 0;
    }
    for (int t = 1; t < nthreads; ++t) pthread_create(&th[t], NULL, worker, &jobs[t]);
    worker(&jobs[0]);
    for (int t = 1; t < nthreads; ++t) pthread_join(th[t], NULL);
    return nthreads;
}

static int check(const oc_problem *p) {
    if (!p || p->S < 1 || p->S > 64 || p->L < p->S || p->M < 1 || p->T < 1 || p->A < 1) return -1;
    if (p->schedule > 2) return -1;
    if (p->schedule == 2 && (p->V < 2 || p->S % p->V || p->M % (p->S / p->V))) return -1;
    if (!p->fwd || !p->bwd || !p->mem || !p->cap) return -1;
    if (p->S > 1 && (!p->cf || !p->cb)) return -1;
    return 0;
}

/* Evaluate `count` candidates: range mode if rank == NULL (index first + i),
 * else list mode.  Writes makespans and feasibility.  Returns 0, or <0. */
int oc_eval(const oc_problem *p, uint64_t first, uint64_t count, const uint64_t *rank,
            const uint32_t *aidx, uint32_t *out_T, uint8_t *out_feas, int nthreads) {
    if (check(p)) return -1;
    oc_dag *g = dag_build((int)p->S, (int)p->M, (int)p->schedule, (int)p->V);
    uint64_t *binom = pascal((int)p->L - 1, (int)p->S - 1);
    if (!g || !binom) { dag_free(g); free(binom); return -3; }
    oc_job proto = {0};
    proto.p = p; proto.g = g; proto.binom = binom; proto.first = first; proto.count = count;
    proto.rank = rank; proto.aidx = aidx; proto.out_T = out_T; proto.out_feas = out_feas;
    oc_job jobs[256];
    int nt = run_jobs(&proto, 0, count, nthreads, jobs);
    int err = 0;
    for (int t = 0; t < nt; ++t) if (jobs[t].err) err = jobs[t].err;
    dag_free(g); free(binom);
    return err;
}

/* Early-stop pass in chunks (0 = one chunk); see header comment.  Returns 0
 * with *best_idx = UINT64_MAX if nothing evaluated has makespan <= bound. */
int oc_bounded(const oc_problem *p, uint64_t first, uint64_t count, const uint64_t *rank,
               const uint32_t *aidx, uint32_t bound, uint64_t chunk, int ramp, uint64_t *best_idx,
               uint32_t *best_T, uint64_t *evaluated, uint64_t *pruned, uint64_t *infeasible,
               int nthreads) {
    if (check(p) || p->schedule == 2) return -1;   /* Eq. 2 is stated for one stage per device */
    oc_dag *g = dag_build((int)p->S, (int)p->M, (int)p->schedule, (int)p->V);
    uint64_t *binom = pascal((int)p->L - 1, (int)p->S - 1);
    if (!g || !binom) { dag_free(g); free(binom); return -3; }
    if (chunk == 0) chunk = count ? count : 1;
    oc_job proto = {0};
    proto.p = p; proto.g = g; proto.binom = binom; proto.first = first; proto.count = count;
    proto.rank = rank; proto.aidx = aidx; proto.bounded = 1;
    uint64_t bT = UINT64_MAX, bI = UINT64_MAX, ev = 0, pr = 0, inf = 0;
    int err = 0;
    oc_job jobs[256];
    /* chunks of `chunk` candidates, or (ramp) chunk, 2 chunk, 4 chunk, ... */
    uint64_t size = chunk;
    for (uint64_t c0 = 0, c1; c0 < count && !err; c0 = c1) {
        c1 = count - c0 > size ? c0 + size : count;
        if (ramp && size < count) size *= 2;
        proto.bound = bT < bound ? bT : bound;
        int nt = run_jobs(&proto, c0, c1, nthreads, jobs);
        for (int t = 0; t < nt; ++t) {
            if (jobs[t].err) err = jobs[t].err;
            ev += jobs[t].evaluated; pr += jobs[t].pruned; inf += jobs[t].infeasible;
            if (jobs[t].best_key_T < bT || (jobs[t].best_key_T == bT && jobs[t].best_idx < bI)) {
                bT = jobs[t].best_key_T; bI = jobs[t].best_idx;
            }
        }
    }
    dag_free(g); free(binom);
    if (err) return err;
    if (bT > bound) { bT = UINT32_MAX; bI = UINT64_MAX; }
    *best_idx = bI; *best_T = (uint32_t)bT;
    *evaluated = ev; *pruned = pr; *infeasible = inf;
    return 0;
}

/* DAG shape for pins: compute nodes, edges by kind. */
/* Finish time of every compute node of one pipeline under the given stage
 * weights (Sec. 4.1, App. B.1): fin_F[(s-1) M + m-1] = finish(F_{s,m}),
 * likewise fin_B; D (stage or device all-reduce weights) may be NULL.
 * Returns T = finish(end), or -1 on a bad shape or allocation failure. */
int64_t oc_finish_times(int S, int M, int schedule, int V, const uint64_t *F, const uint64_t *B,
                        const uint64_t *D, const uint32_t *cf, const uint32_t *cb,
                        uint64_t *fin_F, uint64_t *fin_B) {
    if (S < 1 || S > 64 || M < 1 || schedule < 0 || schedule > 2) return -1;
    if (schedule == 2 && (V < 2 || S % V || M % (S / V))) return -1;
    oc_dag *g = dag_build(S, M, schedule, V);
    if (!g) return -1;
    uint64_t zero[64] = {0};
    uint64_t *fin = malloc(sizeof(uint64_t) * (size_t)g->n);
    if (!fin) { dag_free(g); return -1; }
    uint64_t T = dag_longest(g, F, B, D ? D : zero, cf, cb, fin);
    for (int s = 1; s <= S; ++s)
        for (int m = 1; m <= M; ++m) {
            fin_F[(size_t)(s - 1) * M + (m - 1)] = fin[idF(M, s, m)];
            fin_B[(size_t)(s - 1) * M + (m - 1)] = fin[idB(M, s, m)];
        }
    free(fin);
    dag_free(g);
    return (int64_t)T;
}

int oc_dag_counts(int S, int M, int *n_nodes, int *n_fwd, int *n_bwd, int *n_intra, int *n_other) {
    oc_dag *g = dag_build(S, M, 0, 1);
    if (!g) return -1;
    int f = 0, b = 0, in = 0, o = 0;
    for (int v = 0; v < g->n; ++v) {
        const oc_node *nv = &g->nodes[v];
        if (nv->kind == K_END) { o += S; continue; }
        for (int j = 0; j < nv->npred; ++j) {
            if (nv->ekind[j] == E_FWD) ++f;
            else if (nv->ekind[j] == E_BWD) ++b;
            else if ((nv->kind == K_F || nv->kind == K_B) && g->nodes[nv->pred[j]].kind <= K_B) ++in;
            else ++o;
        }
    }
    *n_nodes = g->n; *n_fwd = f; *n_bwd = b; *n_intra = in; *n_other = o;
    dag_free(g);
    return 0;
}

/* ---------------------------------------------------------------------- */
/* Pruned search over assignment rows (see header).                        */

typedef struct {
    const oc_problem *p;
    const oc_dag *g;
    const uint64_t *binom;
    uint64_t row_lo, row_hi;
    uint64_t bound;
    int ridge, stage_pruning;
    /* results */
    uint64_t best_T, best_row, best_rank;
    uint64_t visited, evaluated, pr_mem, pr_ridge, pr_bound;
    int err;
    /* per-row DFS state */
    int types[64];
    int last[64], falling[64];     /* ridge state per type (last = -1: none yet) */
    uint64_t F[64], B[64], D[64];
    uint64_t *fin;
    uint64_t row;
} oc_sjob;

static void s_stage(oc_sjob *j, int x, int lo, uint64_t pre_f, uint64_t inner, uint64_t rank) {
    const oc_problem *p = j->p;
    int S = (int)p->S, L = (int)p->L, k = S - 1;
    int t = j->types[x - 1];
    int last_stage = x == S;
    int hi_min = last_stage ? L : lo + 1, hi_max = last_stage ? L : L - (S - x);
    uint64_t f = 0, b = 0, mm = 0, d = 0, acc = 0;
    for (int l = lo; l < hi_min - 1; ++l) {
        f += p->fwd[(size_t)t * L + l]; b += p->bwd[(size_t)t * L + l]; mm += p->mem[l];
        if (p->allreduce) d += p->allreduce[(size_t)t * L + l];
    }
    for (int hi = hi_min; hi <= hi_max; ++hi) {
        int l = hi - 1;   /* add layer hi-1 */
        f += p->fwd[(size_t)t * L + l]; b += p->bwd[(size_t)t * L + l]; mm += p->mem[l];
        if (p->allreduce) d += p->allreduce[(size_t)t * L + l];
        if (mm > p->cap[t]) { j->pr_mem++; break; }
        int cnt = hi - lo;
        if (j->ridge && j->last[t] >= 0 && j->falling[t] && cnt > j->last[t]) { j->pr_ridge++; break; }
        uint64_t inn = x == 1 ? d : (inner + j->B[x - 2] > d ? inner + j->B[x - 2] : d);
        uint64_t gx = pre_f + (uint64_t)p->M * (f + b) + inn;
        if (j->stage_pruning && gx > j->bound) { j->pr_bound++; break; }
        j->visited++;
        int sv_last = j->last[t], sv_fall = j->falling[t];
        if (j->last[t] >= 0 && cnt < j->last[t]) j->falling[t] = 1;
        j->last[t] = cnt;
        j->F[x - 1] = f; j->B[x - 1] = b; j->D[x - 1] = d;
        uint64_t r = rank + acc;
        if (last_stage) {
            j->evaluated++;
            uint64_t T = dag_longest(j->g, j->F, j->B, j->D, p->cf, p->cb, j->fin);
            if (T <= j->bound && (T < j->best_T || (T == j->best_T && (j->row < j->best_row ||
                                   (j->row == j->best_row && r < j->best_rank))))) {
                j->best_T = T; j->best_row = j->row; j->best_rank = r;
            }
        } else {
            s_stage(j, x + 1, hi, pre_f + f, inn, r);
            /* the next value of cut x skips the tuples whose cut x is hi */
            acc += j->binom[(size_t)(L - 1 - hi) * (k + 1) + (k - x)];
        }
        j->last[t] = sv_last; j->falling[t] = sv_fall;
    }
}

static void *s_worker(void *arg) {
    oc_sjob *j = arg;
    const oc_problem *p = j->p;
    int S = (int)p->S;
    j->fin = malloc(sizeof(uint64_t) * (size_t)j->g->n);
    if (!j->fin) { j->err = -3; return NULL; }
    for (uint64_t a = j->row_lo; a < j->row_hi; ++a) {
        uint64_t aa = a;
        if (p->assign) {
            for (int s = 0; s < S; ++s) j->types[s] = p->assign[a * S + s];
        } else {
            for (int s = S - 1; s >= 0; --s) { j->types[s] = (int)(aa % p->T); aa /= p->T; }
        }
        for (int t = 0; t < 64; ++t) { j->last[t] = -1; j->falling[t] = 0; }
        j->row = a;
        s_stage(j, 1, 0, 0, 0, 0);
    }
    free(j->fin);
    return NULL;
}

/* Pruned search over rows [first_row, first_row + n_rows), chunks of
 * rows_per_chunk rows (0 = one chunk).  flags: bit 0 = layer-level (ridge)
 * pruning, bit 1 = no stage-level pruning, bit 2 = growing chunks (chunk k
 * holds min(2^k, rows_per_chunk) rows).  Outputs the joint index
 * rank * A + row and the makespan (UINT64_MAX / UINT32_MAX if nothing
 * qualifies) and the counters visited, evaluated, pruned by memory, by the
 * ridge test and by the bound. */
int oc_search(const oc_problem *p, uint64_t first_row, uint64_t n_rows, uint32_t bound, uint64_t rows_per_chunk,
              uint32_t flags, uint64_t *best_idx, uint32_t *best_T, uint64_t *counters, int nthreads) {
    if (check(p) || p->schedule == 2 || first_row + n_rows > p->A || p->S > 64 || p->T > 64) return -1;
    oc_dag *g = dag_build((int)p->S, (int)p->M, (int)p->schedule, (int)p->V);
    uint64_t *binom = pascal((int)p->L - 1, (int)p->S - 1);
    if (!g || !binom) { dag_free(g); free(binom); return -3; }
    if (rows_per_chunk == 0) rows_per_chunk = n_rows ? n_rows : 1;
    if (nthreads < 1) nthreads = 1;
    if (nthreads > 256) nthreads = 256;
    oc_sjob *jobs = calloc((size_t)nthreads, sizeof(oc_sjob));
    pthread_t th[256];
    if (!jobs) { dag_free(g); free(binom); return -3; }
    uint64_t bT = UINT64_MAX, bR = UINT64_MAX, bK = UINT64_MAX;
    uint64_t cnt[5] = {0, 0, 0, 0, 0};
    int err = 0;
    uint64_t size = 1;
    for (uint64_t c0 = 0, c1; c0 < n_rows && !err; c0 = c1) {
        uint64_t step = (flags & 4u) && size < rows_per_chunk ? size : rows_per_chunk;
        c1 = step < n_rows - c0 ? c0 + step : n_rows;
        if (size < rows_per_chunk) size *= 2;
        uint64_t n = c1 - c0;
        int nt = (uint64_t)nthreads > n ? (int)n : nthreads;
        for (int t = 0; t < nt; ++t) {
            oc_sjob *j = &jobs[t];
            memset(j, 0, sizeof(*j));
            j->p = p; j->g = g; j->binom = binom;
            j->row_lo = first_row + c0 + n * (uint64_t)t / (uint64_t)nt;
            j->row_hi = first_row + c0 + n * (uint64_t)(t + 1) / (uint64_t)nt;
            j->bound = bT < bound ? bT : bound;
            j->ridge = (int)(flags & 1u);
            j->stage_pruning = !(flags & 2u);
            j->best_T = j->best_row = j->best_rank = UINT64_MAX;
        }
        for (int t = 1; t < nt; ++t) pthread_create(&th[t], NULL, s_worker, &jobs[t]);
        s_worker(&jobs[0]);
        for (int t = 1; t < nt; ++t) pthread_join(th[t], NULL);
        /* the chunk's best, then strictly better than the earlier chunks' */
        uint64_t cT = UINT64_MAX, cR = UINT64_MAX, cK = UINT64_MAX;
        for (int t = 0; t < nt; ++t) {
            oc_sjob *j = &jobs[t];
            if (j->err) err = j->err;
            cnt[0] += j->visited; cnt[1] += j->evaluated; cnt[2] += j->pr_mem;
            cnt[3] += j->pr_ridge; cnt[4] += j->pr_bound;
            if (j->best_T < cT || (j->best_T == cT && (j->best_row < cR ||
                                   (j->best_row == cR && j->best_rank < cK)))) {
                cT = j->best_T; cR = j->best_row; cK = j->best_rank;
            }
        }
        if (cT < bT) { bT = cT; bR = cR; bK = cK; }
    }
    dag_free(g); free(binom); free(jobs);
    if (err) return err;
    if (bT > bound) { *best_idx = UINT64_MAX; *best_T = UINT32_MAX; }
    else { *best_idx = bK * p->A + bR; *best_T = (uint32_t)bT; }
    for (int i = 0; i < 5; ++i) counters[i] = cnt[i];
    return 0;
}
