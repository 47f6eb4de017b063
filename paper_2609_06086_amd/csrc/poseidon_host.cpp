// C-ABI of the batched Poseidon DAG-cost evaluator (declared in poseidon.h).
//
// Host side: argument validation (no HIP call before it completes), the
// lookup tables shared by every evaluation, launch sizing, and the chunk
// loop of the early-stop search.
#include <hip/hip_runtime.h>

#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <array>
#include <new>
#include <vector>

#include "../../include/poseidon.h"
#include "poseidon_internal.h"

#ifndef PK_CASCADE_K0
#define PK_CASCADE_K0 S   // first checkpoint of the steady-state cascade (1F1B)
#endif
#ifndef PK_EAGER_K0
#define PK_EAGER_K0 (2 * S)   // the same for Eager 1F1B, whose steady state settles later
#endif
#ifndef PK_ILV_K0
#define PK_ILV_K0 2   // the same for Interleaved 1F1B, in periods of 2S slots
#endif

namespace {

// device state words of a context (one u64 each)
enum { W_ACC = 0, W_RESULT, W_RUN, W_STAT_EVAL, W_STAT_PRUNED, W_STAT_INFEAS, W_ERR, W_DONE, W_SNAP, W_COUNT };

uint64_t binom_sat(uint64_t n, uint64_t k) {
    // exact C(n, k) for small k, saturating at UINT64_MAX
    if (k > n) return 0;
    k = std::min(k, n - k);
    unsigned __int128 c = 1;
    for (uint64_t i = 1; i <= k; ++i) {
        c = c * (n - k + i) / i;
        if (c > (unsigned __int128)UINT64_MAX) return UINT64_MAX;
    }
    return (uint64_t)c;
}

bool pow_fits(uint64_t base, uint64_t e, uint64_t limit, uint64_t *out) {
    unsigned __int128 v = 1;
    for (uint64_t i = 0; i < e; ++i) {
        v *= base;
        if (v > limit) return false;
    }
    *out = (uint64_t)v;
    return true;
}

// Order of stage s (1-based) under a schedule; kind 0 = F, 1 = B.
//   1F1B:       min(S-s, M) forwards, then (F, B) pairs, then the remaining backwards.
//   Eager 1F1B: min(2(S-s)+1, M) forwards, then (B, F) pairs, then the remaining backwards.
// Node at position `pos` (0-based) of stage s's order, as (kind, m) with
// kind 0 = forward, 1 = backward: w warm-up forwards, then M - w pairs
// (F_{w+i}, B_i) under 1F1B or (B_i, F_{w+i}) under Eager 1F1B, then the
// remaining backwards.
std::pair<int, int> stage_node(int S, int M, int s, int schedule, int pos) {
    const bool eager = schedule == POSEIDON_SCHEDULE_EAGER_1F1B;
    const int w = eager ? std::min(2 * (S - s) + 1, M) : std::min(S - s, M);
    if (pos < w) return {0, pos + 1};
    const int q = pos - w;
    if (q < 2 * (M - w)) {
        const int i = q / 2 + 1;
        const bool first_of_pair = (q & 1) == 0;
        if (eager) return first_of_pair ? std::make_pair(1, i) : std::make_pair(0, w + i);
        return first_of_pair ? std::make_pair(0, w + i) : std::make_pair(1, i);
    }
    return {1, M - w + 1 + (q - 2 * (M - w))};
}

void stage_order(int S, int M, int s, int schedule, std::vector<std::pair<int, int>> &o) {
    o.clear();
    for (int pos = 0; pos < 2 * M; ++pos) o.push_back(stage_node(S, M, s, schedule, pos));
}

// Unit-weight as-soon-as-possible slots of every node of the DAG; fills
// three stage masks per slot (forward, forward whose input is the upstream
// stage's second-newest forward, backward) and checks what the register
// stencil relies on: at most one node per stage per slot, every input
// finished in an earlier slot, a backward input still the newest backward
// of its stage, and a forward input the newest or second-newest forward.
// With `newest_only` (the single-register path) every input must still be
// the newest node of its stage of either kind.
bool build_slots(int S, int M, int schedule, bool newest_only, std::vector<uint32_t> *masks, uint32_t *nslots) {
    std::vector<std::vector<std::pair<int, int>>> ord(S + 1);
    for (int s = 1; s <= S; ++s) stage_order(S, M, s, schedule, ord[s]);
    // finish slot of F_{s,m} / B_{s,m}
    std::vector<int> finF((size_t)(S + 2) * (M + 1), -1), finB((size_t)(S + 2) * (M + 1), -1);
    auto at = [M](int s, int m) { return (size_t)s * (M + 1) + m; };
    std::vector<int> pos(S + 1, 0), slot_of_last(S + 1, 0);
    std::vector<int> startF(finF.size(), -1), startB(finB.size(), -1);
    int placed = 0, total = 2 * S * M, n = 0;
    while (placed < total) {
        bool progress = false;
        for (int s = 1; s <= S; ++s) {
            while (pos[s] < 2 * M) {
                const int kind = ord[s][pos[s]].first, m = ord[s][pos[s]].second;
                int ready = pos[s] ? slot_of_last[s] : 0;
                int dep = 0;
                if (kind == 0 && s > 1) dep = finF[at(s - 1, m)];
                if (kind == 1 && s < S) dep = finB[at(s + 1, m)];
                if (dep < 0) break;
                const int st = std::max(ready, dep);
                if (kind == 0) { startF[at(s, m)] = st; finF[at(s, m)] = st + 1; }
                else { startB[at(s, m)] = st; finB[at(s, m)] = st + 1; }
                slot_of_last[s] = st + 1;
                n = std::max(n, st + 1);
                ++pos[s];
                ++placed;
                progress = true;
            }
        }
        if (!progress) return false;
    }
    std::vector<uint32_t> fm(n, 0), fd(n, 0), bm(n, 0);
    for (int s = 1; s <= S; ++s)
        for (int m = 1; m <= M; ++m) {
            const int a = startF[at(s, m)], b = startB[at(s, m)];
            if (a < 0 || b < 0 || a >= n || b >= n) return false;
            if ((fm[a] | bm[a]) >> (s - 1) & 1u) return false;
            fm[a] |= 1u << (s - 1);
            if ((fm[b] | bm[b]) >> (s - 1) & 1u) return false;
            bm[b] |= 1u << (s - 1);
        }
    // inputs: F_{s,m} reads F_{s-1,m}; B_{s,m} reads B_{s+1,m}
    for (int s = 1; s <= S; ++s) {
        for (const auto &node : ord[s]) {
            const int kind = node.first, m = node.second;
            const int st = kind == 0 ? startF[at(s, m)] : startB[at(s, m)];
            const int u = kind == 0 ? s - 1 : s + 1;
            if (u < 1 || u > S) continue;
            const int ust = kind == 0 ? startF[at(u, m)] : startB[at(u, m)];
            if (ust >= st) return false;
            int newer_same = 0, newer_any = 0;
            for (int q = ust + 1; q < st; ++q) {
                const bool f = (fm[q] >> (u - 1)) & 1u, b = (bm[q] >> (u - 1)) & 1u;
                newer_any += f || b;
                newer_same += kind == 0 ? f : b;
            }
            if (newest_only && newer_any) return false;
            if (kind == 1 && newer_same) return false;
            if (kind == 0 && newer_same > 1) return false;
            if (kind == 0 && newer_same == 1) fd[st] |= 1u << (s - 1);
        }
    }
    if (masks) {
        masks->assign(3 * (size_t)n, 0);
        for (int k = 0; k < n; ++k) {
            (*masks)[3 * k] = fm[k];
            (*masks)[3 * k + 1] = fd[k];
            (*masks)[3 * k + 2] = bm[k];
        }
    }
    *nslots = (uint32_t)n;
    return true;
}

// Interleaved 1F1B (Sec. 4.1.4): device p (0-based) of N, V chunks each,
// Megatron-LM's order: forward step k runs chunk (k mod VN) div N on
// micro-batch (k div VN) N + k mod N + 1, backward step k chunk
// V-1 - (k mod VN) div N on the same micro-batch; a warm-up of
// min(2(N-p-1) + (V-1) N, VM) forward steps (all of them if M = N), then
// (forward, backward) pairs, then the remaining backward steps.  Entries are
// (kind, virtual stage 0-based, micro-batch 1-based).
void interleaved_order(int N, int V, int M, int p, std::vector<std::array<int, 3>> &o) {
    o.clear();
    const int total = V * M;
    const int w = M == N ? total : std::min(2 * (N - p - 1) + (V - 1) * N, total);
    auto mb = [&](int k) { return (k / (N * V)) * N + k % N + 1; };
    auto fwd = [&](int k) { return std::array<int, 3>{0, ((k % (N * V)) / N) * N + p, mb(k)}; };
    auto bwd = [&](int k) { return std::array<int, 3>{1, (V - 1 - (k % (N * V)) / N) * N + p, mb(k)}; };
    for (int k = 0; k < w; ++k) o.push_back(fwd(k));
    for (int i = 0; i < total - w; ++i) {
        o.push_back(fwd(w + i));
        o.push_back(bwd(i));
    }
    for (int k = total - w; k < total; ++k) o.push_back(bwd(k));
}

// Unit-weight as-soon-as-possible slots of the Interleaved 1F1B DAG.  A
// device runs at most one node per slot (its nodes are sequential).  Four
// words per slot: forward, forward-of-depth-2, backward stage masks and a
// 2-bit backward input depth per stage.  A forward must read the upstream
// stage's newest or second-newest forward, a backward one of the downstream
// stage's `max_db` newest backwards; otherwise the stencil does not apply.
bool build_interleaved_slots(int N, int V, int M, int max_db, std::vector<uint32_t> *masks, uint32_t *nslots) {
    const int S = N * V;
    std::vector<std::vector<std::array<int, 3>>> ord(N);
    for (int p = 0; p < N; ++p) interleaved_order(N, V, M, p, ord[p]);
    auto at = [M](int j, int m) { return (size_t)j * (M + 1) + m; };
    std::vector<int> stF((size_t)S * (M + 1), -1), stB((size_t)S * (M + 1), -1);
    std::vector<int> pos(N, 0), free_at(N, 0);
    const int total = 2 * S * M;
    int placed = 0, n = 0;
    while (placed < total) {
        bool progress = false;
        for (int p = 0; p < N; ++p) {
            while (pos[p] < (int)ord[p].size()) {
                const int kind = ord[p][pos[p]][0], j = ord[p][pos[p]][1], m = ord[p][pos[p]][2];
                int dep = 0;
                if (kind == 0 && j > 0) dep = stF[at(j - 1, m)] < 0 ? -1 : stF[at(j - 1, m)] + 1;
                if (kind == 1 && j < S - 1) dep = stB[at(j + 1, m)] < 0 ? -1 : stB[at(j + 1, m)] + 1;
                if (dep < 0) break;
                const int st = std::max(free_at[p], dep);
                (kind == 0 ? stF : stB)[at(j, m)] = st;
                free_at[p] = st + 1;
                n = std::max(n, st + 1);
                ++pos[p];
                ++placed;
                progress = true;
            }
        }
        if (!progress) return false;
    }
    for (int j = 0; j < S; ++j)
        for (int m = 2; m <= M; ++m)
            if (stF[at(j, m)] <= stF[at(j, m - 1)] || stB[at(j, m)] <= stB[at(j, m - 1)]) return false;
    std::vector<uint32_t> fm(n, 0), fd(n, 0), bm(n, 0), bd(n, 0);
    for (int j = 0; j < S; ++j)
        for (int m = 1; m <= M; ++m) {
            const int a = stF[at(j, m)], b = stB[at(j, m)];
            fm[a] |= 1u << j;
            bm[b] |= 1u << j;
            // a stage runs its forwards, and its backwards, in micro-batch
            // order (checked below), so the nodes newer than micro-batch m's
            // are those of the following micro-batches that started earlier
            if (j > 0) {
                // forwards of stage j-1 started after F_{j-1,m} and before slot a
                int newer = 0;
                for (int mm = m + 1; mm <= M && stF[at(j - 1, mm)] < a; ++mm) ++newer;
                if (newer > 1) return false;
                if (newer == 1) fd[a] |= 1u << j;
            }
            if (j < S - 1) {
                int newer = 0;
                for (int mm = m + 1; mm <= M && stB[at(j + 1, mm)] < b; ++mm) ++newer;
                if (newer >= max_db) return false;
                bd[b] |= (uint32_t)newer << (2 * j);
            }
        }
    masks->assign(4 * (size_t)n, 0);
    for (int k = 0; k < n; ++k) {
        (*masks)[4 * k] = fm[k];
        (*masks)[4 * k + 1] = fd[k];
        (*masks)[4 * k + 2] = bm[k];
        (*masks)[4 * k + 3] = bd[k];
    }
    *nslots = (uint32_t)n;
    return true;
}

// The closed-form slot pattern the kernels hard-code (1F1B with M >= S,
// Eager 1F1B with M >= 2S-1), checked slot by slot against the unit-weight
// as-soon-as-possible schedule, simulated here with O(S) state so that any
// M is checked.  In slot k every stage whose next node's input finished in
// an earlier slot runs that node.  The simulation also checks what the
// stencil relies on: under 1F1B every input is still the newest node of its
// stage (either kind); under Eager 1F1B a backward reads the newest backward
// of the stage below and a forward the newest or second-newest forward of
// the stage above (op 3 marks the second-newest).  Ops: 0 idle, 1 forward,
// 2 backward, 3 forward reading the upstream's previous forward.
bool closed_form_check(int S, int M, int schedule) {
    const bool eager = schedule == POSEIDON_SCHEDULE_EAGER_1F1B;
    // per stage: next position in its order, forwards / backwards done,
    // kind of the newest node (-1 none); index 0 and S+1 are sentinels
    std::vector<int> pos(S + 2, 0), nf(S + 2, 0), nb(S + 2, 0), last(S + 2, -1), op(S + 2, 0);
    const int64_t n = 2 * ((int64_t)M + S - 1);
    for (int64_t k = 0; k < n; ++k) {
        for (int s = 1; s <= S; ++s) {
            op[s] = 0;
            if (pos[s] >= 2 * M) continue;
            const std::pair<int, int> v = stage_node(S, M, s, schedule, pos[s]);
            const int m = v.second;
            if (v.first == 0) {
                if (s == 1) { op[s] = 1; continue; }
                if (nf[s - 1] < m) continue;                     // input not finished
                if (eager) {
                    if (nf[s - 1] > m + 1) return false;          // more than one newer forward
                    op[s] = nf[s - 1] == m + 1 ? 3 : 1;
                } else {
                    if (nf[s - 1] != m || last[s - 1] != 0) return false;
                    op[s] = 1;
                }
            } else {
                if (s == S) { op[s] = 2; continue; }
                if (nb[s + 1] < m) continue;
                if (nb[s + 1] != m || (!eager && last[s + 1] != 1)) return false;
                op[s] = 2;
            }
        }
        for (int s = 1; s <= S; ++s) {
            int want;
            if (eager) want = pk::eager_op(S, M, s, (int)k);
            else if (k < 2 * S - 1) want = pk::prologue_op(S, s, (int)k);
            else if (k <= 2 * (int64_t)M - 1) want = ((k - s - 1) & 1) == 0 ? 1 : 2;
            else want = pk::epilogue_op(S, s, (int)(k - 2 * (int64_t)M));
            if (op[s] != want) return false;
            if (op[s]) {
                ++pos[s];
                if (op[s] == 2) ++nb[s];
                else ++nf[s];
                last[s] = op[s] == 2 ? 1 : 0;
            }
        }
    }
    for (int s = 1; s <= S; ++s)
        if (pos[s] != 2 * M) return false;
    return true;
}

}  // namespace

struct poseidon_ctx;
namespace {
uint64_t noalloc_chunk_for(const poseidon_ctx *ctx);
}  // namespace

static_assert(pk::kEntRow >= POSEIDON_L_MAX + 1, "an entry field row holds every end point");
static_assert(pk::kTypesMax >= POSEIDON_T_MAX, "per-type device arrays hold every type");

struct poseidon_ctx {
    int device;
    uint32_t L, S, M, T;
    uint64_t A, n_comp;
    bool wide;
    uint32_t NB;
    pk::KParams base;      // table pointers and problem constants
    void *dmem;
    unsigned long long *state;
    size_t lds_bytes;      // cost, pm, cap (and pd): search and Interleaved 1F1B kernels
    size_t ent_lds_bytes;  // stage entries (and pdx): evaluation and early-stop kernels
    uint32_t filter_grid;  // blocks of the early-stop filter that are resident at once
    uint32_t grid_max;
    void *ws;              // cut codes + straggler queues of the steady-state cascade
    uint64_t ws_cap;       // candidates per chunk the workspace holds
    void *sws;             // search frontiers (allocated on the first poseidon_search)
    unsigned long long *shost;   // pinned host words for the search's read-backs (level totals
                                 // and block offsets), allocated with sws
    uint64_t result_base = 0;    // added to the position the last evaluation or argmin published:
                                 // `first` in range mode (the joint index), else 0 or index_base
    void *scratch;               // the library's fixed scratch on this device (allocation-free calls)
    uint64_t noalloc_chunk;      // candidates per chunk whose workspace fits that scratch (0: none)
};

extern "C" {

const char *poseidon_strerror(int status) {
    switch (status) {
    case POSEIDON_OK: return "ok";
    case POSEIDON_NO_FEASIBLE: return "no candidate satisfies the memory caps (or the bound)";
    case POSEIDON_E_INVAL: return "invalid argument";
    case POSEIDON_E_RANGE: return "value out of range (makespan could reach 2^31, or count overflow)";
    case POSEIDON_E_DEVICE: return "HIP device error";
    case POSEIDON_E_NOMEM: return "out of memory";
    default: return "unknown status";
    }
}

int poseidon_validate(const poseidon_problem *p, uint64_t *n_candidates) {
    if (!p) return POSEIDON_E_INVAL;
    if (p->S < 1 || p->S > POSEIDON_S_MAX || p->L < p->S || p->L > POSEIDON_L_MAX || p->M < 1 ||
        p->M > POSEIDON_M_MAX || p->T < 1 ||
        p->T > POSEIDON_T_MAX)
        return POSEIDON_E_INVAL;
    if (!p->fwd_us || !p->bwd_us || !p->mem_mb || !p->cap_mb) return POSEIDON_E_INVAL;
    if (p->S > 1 && (!p->comm_fwd_us || !p->comm_bwd_us)) return POSEIDON_E_INVAL;
    if (p->schedule > POSEIDON_SCHEDULE_INTERLEAVED_1F1B) return POSEIDON_E_INVAL;
    // Interleaved 1F1B: S virtual stages on N = S / V >= 2 devices, M a multiple of N
    const bool ilv = p->schedule == POSEIDON_SCHEDULE_INTERLEAVED_1F1B;
    if (ilv && (p->V < 2 || p->S % p->V || p->S / p->V < 2 || p->M % (p->S / p->V))) return POSEIDON_E_INVAL;
    const uint32_t ndev = ilv ? p->S / p->V : p->S;
    uint64_t A;
    if (p->assign) {
        if (p->A < 1 || p->A > (1ull << 32)) return p->A < 1 ? POSEIDON_E_INVAL : POSEIDON_E_RANGE;
        for (uint64_t i = 0; i < p->A * ndev; ++i)
            if (p->assign[i] >= p->T) return POSEIDON_E_INVAL;
        A = p->A;
    } else if (!pow_fits(p->T, ndev, 1ull << 32, &A)) {
        return POSEIDON_E_RANGE;
    }
    const uint64_t nc = binom_sat(p->L - 1, p->S - 1);
    if (nc == UINT64_MAX) return POSEIDON_E_RANGE;
    unsigned __int128 tot = (unsigned __int128)nc * A;
    if (tot > (unsigned __int128)UINT64_MAX - 1) return POSEIDON_E_RANGE;
    // Every path weight is at most the sum of all node and edge weights:
    // M * (sum over layers of the slowest type's fwd + bwd + all transfers).
    unsigned __int128 w = 0;
    for (uint32_t l = 0; l < p->L; ++l) {
        uint64_t mx = 0;
        for (uint32_t t = 0; t < p->T; ++t)
            mx = std::max<uint64_t>(mx, (uint64_t)p->fwd_us[(size_t)t * p->L + l] + p->bwd_us[(size_t)t * p->L + l]);
        w += mx;
    }
    for (uint32_t b = 0; b + 1 < p->S; ++b) w += (uint64_t)p->comm_fwd_us[b] + p->comm_bwd_us[b];
    w *= p->M;
    if (p->allreduce_us) {
        // the end node adds at most one stage's all-reduce, which is at most
        // the sum over all layers of the slowest type's all-reduce
        for (uint32_t l = 0; l < p->L; ++l) {
            uint64_t mx = 0;
            for (uint32_t t = 0; t < p->T; ++t) mx = std::max<uint64_t>(mx, p->allreduce_us[(size_t)t * p->L + l]);
            w += mx;
        }
    }
    if (w >= ((unsigned __int128)1 << 31)) return POSEIDON_E_RANGE;
    unsigned __int128 mem = 0;
    for (uint32_t l = 0; l < p->L; ++l) mem += p->mem_mb[l];
    if (mem >= ((unsigned __int128)1 << 32)) return POSEIDON_E_RANGE;
    if (n_candidates) *n_candidates = (uint64_t)tot;
    return POSEIDON_OK;
}

int poseidon_load_costs(const poseidon_problem *p, int hip_device, poseidon_ctx **out) {
    if (!out) return POSEIDON_E_INVAL;
    *out = nullptr;
    uint64_t ncand = 0;
    int rc = poseidon_validate(p, &ncand);
    if (rc != POSEIDON_OK) return rc;
    const uint32_t L = p->L, S = p->S, M = p->M, T = p->T;
    const uint64_t n_comp = binom_sat(L - 1, S - 1);
    const uint64_t A = n_comp ? ncand / n_comp : 0;
    const bool wide = n_comp > 0xFFFFFFFFull;
    const uint32_t NB = pk::kNB;   // Pascal-table column length (L <= kNB)

    // schedule of the DAG: 1F1B with M >= S and Eager 1F1B with M >= 2S-1
    // run the closed forms the kernels hard-code (self-checked against the
    // simulated schedule here); other cases run a slot table
    std::vector<uint32_t> masks;
    uint32_t nslots = 0;
    const uint32_t sched = p->schedule;
    const bool eager = sched == POSEIDON_SCHEDULE_EAGER_1F1B;
    const bool ilv = sched == POSEIDON_SCHEDULE_INTERLEAVED_1F1B;
    const uint32_t ndev = ilv ? S / p->V : S;
    const bool table_path = ilv || (eager ? M + 1 < 2 * S : M < S);
    if (ilv) {
        if (!build_interleaved_slots((int)ndev, (int)p->V, (int)M, pk::ilv_max_db((int)ndev), &masks, &nslots))
            return POSEIDON_E_INVAL;
    } else if (table_path) {
        if (!build_slots((int)S, (int)M, (int)sched, !eager, &masks, &nslots)) return POSEIDON_E_INVAL;
    } else if (!closed_form_check((int)S, (int)M, (int)sched)) {
        return POSEIDON_E_INVAL;
    }

    // host images of the device tables
    std::vector<uint64_t> cost((size_t)T * (L + 1));
    for (uint32_t t = 0; t < T; ++t) {
        uint64_t f = 0, b = 0;
        cost[(size_t)t * (L + 1)] = 0;
        for (uint32_t l = 0; l < L; ++l) {
            f += p->fwd_us[(size_t)t * L + l];
            b += p->bwd_us[(size_t)t * L + l];
            cost[(size_t)t * (L + 1) + l + 1] = (b << 32) | f;
        }
    }
    std::vector<uint32_t> pm(L + 1, 0);
    for (uint32_t l = 0; l < L; ++l) pm[l + 1] = pm[l] + p->mem_mb[l];
    const bool has_ar = p->allreduce_us != nullptr;
    std::vector<uint32_t> pd(has_ar ? (size_t)T * (L + 1) : 0, 0);
    for (uint32_t t = 0; has_ar && t < T; ++t)
        for (uint32_t l = 0; l < L; ++l)
            pd[(size_t)t * (L + 1) + l + 1] = pd[(size_t)t * (L + 1) + l] + p->allreduce_us[(size_t)t * L + l];
    // stage entries (the evaluation and early-stop kernels' table): per type
    // t the field rows Pf, Pb, hm (and Pd) over end points j,
    // where hm_t[j] is the largest end point h >= j whose stage [j, h) fits
    // type t's memory (Pm only grows, so the stages that fit are those
    // ending at or before hm_t[j])
    const uint32_t nfield = pk::entry_fields(has_ar);
    std::vector<uint32_t> ent((size_t)T * nfield * pk::kEntRow, 0);
    for (uint32_t t = 0; t < T; ++t)
        for (uint32_t j = 0; j <= L; ++j) {
            const uint64_t c = cost[(size_t)t * (L + 1) + j];
            uint32_t *e = &ent[(size_t)t * nfield * pk::kEntRow + j];
            const uint32_t f = (uint32_t)c, b = (uint32_t)(c >> 32);
            e[pk::kEPf * pk::kEntRow] = f;
            e[pk::kEPb * pk::kEntRow] = b;
            uint32_t h = j;
            while (h < L && pm[h + 1] - pm[j] <= p->cap_mb[t]) ++h;
            e[pk::kEHm * pk::kEntRow] = h;
            if (has_ar) e[pk::kEPd * pk::kEntRow] = pd[(size_t)t * (L + 1) + j];
        }
    const size_t rsz = wide ? 8 : 4;
    std::vector<unsigned char> binom((size_t)S * NB * rsz);
    for (uint32_t k = 0; k < S; ++k)
        for (uint32_t n = 0; n < NB; ++n) {
            uint64_t v = binom_sat(n, k);
            if (wide) memcpy(&binom[((size_t)k * NB + n) * 8], &v, 8);
            else {
                uint32_t v32 = v > 0xFFFFFFFFull ? 0xFFFFFFFFu : (uint32_t)v;
                memcpy(&binom[((size_t)k * NB + n) * 4], &v32, 4);
            }
        }

    // bucket tables of the unranking searches: per column k, per key, the
    // first row n < 2^H whose (stored) entry reaches the bucket's smallest
    // value (at most 2^H - 1: no search sees a larger value); 64-bit keys for
    // the wide columns of 64-bit ranks, 32-bit keys for the others
    const uint32_t NHd = 1u << pk::decode_levels(L);
    const uint32_t n_narrow = wide ? std::min<uint32_t>(S, 5) : 0;
    std::vector<uint8_t> btab((size_t)S * pk::kBucketTab, 0);
    for (uint32_t k = 0; k < S; ++k) {
        const int w = (wide && k >= n_narrow) ? 64 : 32;
        const unsigned __int128 vmax = w == 64 ? (unsigned __int128)UINT64_MAX : (unsigned __int128)0xFFFFFFFFu;
        std::vector<unsigned __int128> col(NHd);
        for (uint32_t n = 0; n < NHd; ++n) col[n] = std::min<unsigned __int128>(binom_sat(n, k), vmax);
        for (int z = 0; z < w; ++z)
            for (int m = 0; m < 16; ++m) {
                const unsigned __int128 lo = pk::bucket_lo(w, z, m);
                const uint32_t n = (uint32_t)(std::lower_bound(col.begin(), col.end(), lo) - col.begin());
                btab[(size_t)k * pk::kBucketTab + 16 * z + m] = (uint8_t)std::min(n, NHd - 1);
            }
    }

    pk::KParams kp;
    memset(&kp, 0, sizeof(kp));
    kp.A = A;
    kp.n_comp = n_comp;
    kp.L = L; kp.S = S; kp.M = M; kp.T = T; kp.NB = NB;
    kp.wide = wide;
    for (uint32_t b = 0; b + 1 < S; ++b) { kp.cf[b] = p->comm_fwd_us[b]; kp.cb[b] = p->comm_bwd_us[b]; }
    kp.has_ar = has_ar;
    kp.sched = sched;
    kp.ndev = ndev;
    // a last stage [c, L) fits type t iff c >= last_lo[t] (its memory only shrinks with c)
    for (uint32_t t = 0; t < T; ++t) {
        uint32_t c = 0;
        while (c < L && pm[L] - pm[c] > p->cap_mb[t]) ++c;
        kp.last_lo[t] = c;
    }
    // type pairs (t, u) whose every layer has fwd + bwd on t at most M times
    // that on u: the search's last-stage Eq. 2 then falls as the last cut grows
    for (uint32_t t = 0; t < T; ++t)
        for (uint32_t u = 0; u < T; ++u) {
            bool mono = true;
            for (uint32_t l = 0; l < L && mono; ++l)
                mono = (uint64_t)p->fwd_us[(size_t)t * L + l] + p->bwd_us[(size_t)t * L + l] <=
                       (uint64_t)M * ((uint64_t)p->fwd_us[(size_t)u * L + l] + p->bwd_us[(size_t)u * L + l]);
            if (mono) kp.g_mono |= 1ull << (8 * t + u);
        }
    kp.g_mono_all = 1;
    for (uint32_t t = 0; t < T; ++t)
        for (uint32_t u = 0; u < T; ++u)
            if (!((kp.g_mono >> (8 * t + u)) & 1ull)) kp.g_mono_all = 0;
    if (ilv) {
        // the compiled schedule (prologue, `trips` periods, cool-down) is used
        // only if it equals this problem's own slot table word for word
        const uint32_t P = 2 * S;
        std::vector<uint32_t> pro(4 * 4 * (size_t)S), per(4 * (size_t)P), cool(4 * 4 * (size_t)S);
        int a = 0, e = 0;
        if (pk::ilv_program_words(S, ndev, &a, &e, pro.data(), per.data(), cool.data()) &&
            nslots >= (uint32_t)(a + e) && (nslots - a - e) % P == 0) {
            const uint32_t trips = (nslots - a - e) / P;
            bool same = std::equal(pro.begin(), pro.begin() + 4 * (size_t)a, masks.begin()) &&
                        std::equal(cool.begin(), cool.begin() + 4 * (size_t)e, masks.begin() + 4 * ((size_t)nslots - e));
            for (uint32_t t = 0; same && t < trips; ++t)
                same = std::equal(per.begin(), per.end(), masks.begin() + 4 * ((size_t)a + (size_t)t * P));
            kp.ilv_compiled = same;
            kp.ilv_trips = same ? trips : 0;
        }
    }
    for (uint32_t s = 1; s < S; ++s) kp.psi[s] = kp.psi[s - 1] + kp.cf[s - 1];
    // cascade checkpoints of the steady loop: K0, 2 K0, 4 K0, ... below M - S
    // (steady iterations: 1F1B slot pairs after its prologue, Eager 1F1B
    // slot pairs between its prologue and epilogue)
    if (!table_path) {   // (no cascade for the slot-table paths)
        const uint32_t nit = eager ? M + 1 - 2 * S : M - S;
        uint32_t k = std::max<uint32_t>(2, eager ? PK_EAGER_K0 : PK_CASCADE_K0);
        while (k < nit && kp.nlevels < (uint32_t)pk::kMaxLevels) {
            kp.lvl_k[kp.nlevels++] = k;
            k *= 2;
        }
    } else if (ilv && kp.ilv_compiled) {   // Interleaved 1F1B: checkpoints in periods
        uint32_t k = std::max<uint32_t>(1, PK_ILV_K0);
        while (k < kp.ilv_trips && kp.nlevels < (uint32_t)pk::kMaxLevels) {
            kp.lvl_k[kp.nlevels++] = k;
            k *= 2;
        }
    }
    const bool has_table = p->assign && A > 1;
    if (A == 1) {
        kp.assign_mode = pk::kAssignFixed;
        for (uint32_t s = 0; s < ndev; ++s) kp.fixed_types[s] = p->assign ? p->assign[s] : 0;
    } else if (has_table) {
        kp.assign_mode = pk::kAssignTable;
    } else {
        kp.assign_mode = pk::kAssignDigits;
        kp.magicT = (uint32_t)((1ull << 32) / T + 1);
        // T^(ndev-1) <= A / T < 2^32, and it is at least 2 here (T >= 2, ndev >= 2)
        uint64_t d = 1;
        for (uint32_t s = 1; s < ndev; ++s) d *= T;
        kp.s1_div = (uint32_t)d;
        kp.s1_magic = d > 1 ? (uint32_t)((1ull << 32) / d + 1) : 0u;
    }
    // the evaluation kernels' digit table (base-T digits, T <= 4, one stage
    // per device): for r < T^4 the entry-block offsets of r's four digits,
    // most significant first, in 16-bit fields
    const uint32_t erow = nfield * pk::kEntField;
    const uint32_t ent_bytes = (uint32_t)(ent.size() * 4);
    if (kp.assign_mode == pk::kAssignDigits && T <= 4 && !ilv) {
        const uint32_t tg = T * T * T * T;
        for (uint32_t r = 0; r < tg; ++r) {
            uint64_t w = 0;
            for (uint32_t i = 0, x = r, div = T * T * T; i < 4; ++i, div = div > 1 ? div / T : 1) {
                const uint32_t d = x / div;
                x -= d * div;
                w |= (uint64_t)(d * erow) << (16 * i);
            }
            ent.push_back((uint32_t)w);
            ent.push_back((uint32_t)(w >> 32));
        }
        kp.dig_tg = tg;
        kp.dig_magic = (uint32_t)((1ull << 32) / tg + 1);
    }
    // a stage's F + B is at most its type's total over all layers
    kp.g24 = M < (1u << 24);
    for (uint32_t t = 0; t < T; ++t)
        if ((cost[(size_t)t * (L + 1) + L] & 0xFFFFFFFFull) + (cost[(size_t)t * (L + 1) + L] >> 32) >= (1ull << 24))
            kp.g24 = 0;
    static_assert(7 * 4 * pk::kEntField < 65536, "entry-block offsets fit 16 bits");

    // one device block: state words | cost | pm | cap | binom | assign | slots
    auto al = [](size_t x) { return (x + 255) & ~(size_t)255; };
    size_t off = 0;
    const size_t o_state = off; off = al(off + W_COUNT * 8);
    const size_t o_cost = off; off = al(off + cost.size() * 8);
    const size_t o_pm = off; off = al(off + pm.size() * 4);
    const size_t o_cap = off; off = al(off + (size_t)T * 4);
    const size_t o_binom = off; off = al(off + binom.size());
    const size_t o_btab = off; off = al(off + btab.size());
    const size_t o_assign = off; off = al(off + (has_table ? (size_t)A * ndev : 0));
    const size_t o_slots = off; off = al(off + (table_path ? masks.size() * 4 : 0));
    const size_t o_pd = off; off = al(off + pd.size() * 4);
    const size_t o_ent = off; off = al(off + ent.size() * 4);
    const size_t total = off;

    poseidon_ctx *ctx = new (std::nothrow) poseidon_ctx;
    if (!ctx) return POSEIDON_E_NOMEM;
    memset(ctx, 0, sizeof(*ctx));
    int prev = 0;
    if (hipGetDevice(&prev) != hipSuccess || hipSetDevice(hip_device) != hipSuccess) {
        delete ctx;
        return POSEIDON_E_DEVICE;
    }
    int status = POSEIDON_OK;
    void *d = nullptr;
    do {
        if (hipMalloc(&d, total) != hipSuccess) { status = POSEIDON_E_NOMEM; break; }
        unsigned char *b = (unsigned char *)d;
        std::vector<unsigned long long> st(W_COUNT, 0);
        st[W_ACC] = ~0ull; st[W_RESULT] = ~0ull; st[W_RUN] = ~0ull; st[W_SNAP] = ~0ull;
        bool ok = hipMemcpy(b + o_state, st.data(), W_COUNT * 8, hipMemcpyHostToDevice) == hipSuccess &&
                  hipMemcpy(b + o_cost, cost.data(), cost.size() * 8, hipMemcpyHostToDevice) == hipSuccess &&
                  hipMemcpy(b + o_pm, pm.data(), pm.size() * 4, hipMemcpyHostToDevice) == hipSuccess &&
                  hipMemcpy(b + o_cap, p->cap_mb, (size_t)T * 4, hipMemcpyHostToDevice) == hipSuccess &&
                  hipMemcpy(b + o_binom, binom.data(), binom.size(), hipMemcpyHostToDevice) == hipSuccess &&
                  hipMemcpy(b + o_btab, btab.data(), btab.size(), hipMemcpyHostToDevice) == hipSuccess;
        if (ok && has_table)
            ok = hipMemcpy(b + o_assign, p->assign, (size_t)A * ndev, hipMemcpyHostToDevice) == hipSuccess;
        if (ok && table_path)
            ok = hipMemcpy(b + o_slots, masks.data(), masks.size() * 4, hipMemcpyHostToDevice) == hipSuccess;
        if (ok && has_ar) ok = hipMemcpy(b + o_pd, pd.data(), pd.size() * 4, hipMemcpyHostToDevice) == hipSuccess;
        if (ok) ok = hipMemcpy(b + o_ent, ent.data(), ent.size() * 4, hipMemcpyHostToDevice) == hipSuccess;
        if (!ok) { status = POSEIDON_E_DEVICE; break; }
        kp.cost = (const uint64_t *)(b + o_cost);
        kp.pm = (const uint32_t *)(b + o_pm);
        kp.cap = (const uint32_t *)(b + o_cap);
        kp.binom = b + o_binom;
        kp.btab = (const uint8_t *)(b + o_btab);
        kp.assign = has_table ? (const uint8_t *)(b + o_assign) : nullptr;
        kp.slot_mask = table_path ? (const uint32_t *)(b + o_slots) : nullptr;
        kp.pd = has_ar ? (const uint32_t *)(b + o_pd) : nullptr;
        kp.ent = (const uint32_t *)(b + o_ent);
        kp.erow = erow;
        kp.ent_bytes = ent_bytes;
        kp.ent_lds = (uint32_t)((ent.size() * 4 + 15) & ~(size_t)15);
        kp.nslots = table_path ? nslots : 0;
        ctx->state = (unsigned long long *)(b + o_state);
        kp.acc = ctx->state + W_ACC;
        kp.result = ctx->state + W_RESULT;
        kp.run_best = ctx->state + W_RUN;
        kp.snap = ctx->state + W_SNAP;
        kp.stats = ctx->state + W_STAT_EVAL;
        kp.err = (unsigned int *)(ctx->state + W_ERR);
        kp.done = (unsigned int *)(ctx->state + W_DONE);
        const size_t lds = ((cost.size() * 8 + pm.size() * 4 + (size_t)T * 4 + pd.size() * 4) + 15) & ~(size_t)15;
        const size_t elds = kp.ent_lds;
        if (lds > 64 * 1024 || elds > 64 * 1024) { status = POSEIDON_E_RANGE; break; }
        int occ = 0;
        hipDeviceProp_t prop;
        if (pk::eval_occupancy(kp, ilv ? lds : elds, &occ) != hipSuccess ||
            hipGetDeviceProperties(&prop, hip_device) != hipSuccess) {
            status = POSEIDON_E_DEVICE;
            break;
        }
        ctx->lds_bytes = lds;
        ctx->ent_lds_bytes = elds;
        // the early-stop filter's grid: one block per resident slot, each
        // block looping over its share of a piece (a larger grid leaves a
        // partial second wave of blocks, each paying for its LDS tables)
        int focc = 0;
        if (!ilv && pk::filter_occupancy(kp, elds, &focc) != hipSuccess) {
            status = POSEIDON_E_DEVICE;
            break;
        }
        ctx->grid_max = (uint32_t)std::max(1, occ) * (uint32_t)std::max(1, prop.multiProcessorCount);
        // (at most grid_max: the survivor segments are sized for that many blocks)
        ctx->filter_grid = std::min(ctx->grid_max,
                                    (uint32_t)std::max(1, focc) * (uint32_t)std::max(1, prop.multiProcessorCount));
    } while (0);
    (void)hipSetDevice(prev);
    if (status != POSEIDON_OK) {
        if (d) (void)hipFree(d);
        delete ctx;
        return status;
    }
    ctx->device = hip_device;
    ctx->L = L; ctx->S = S; ctx->M = M; ctx->T = T;
    ctx->A = A; ctx->n_comp = n_comp; ctx->wide = wide; ctx->NB = NB;
    ctx->base = kp;
    ctx->dmem = d;
    // the allocation-free evaluation's scratch on this device (looked up once
    // per device) and the chunk size whose workspace fits it
    ctx->scratch = pk::noalloc_scratch(hip_device);
    ctx->noalloc_chunk = noalloc_chunk_for(ctx);
    *out = ctx;
    return POSEIDON_OK;
}

void poseidon_free(poseidon_ctx *ctx) {
    if (!ctx) return;
    int prev = 0;
    if (hipGetDevice(&prev) == hipSuccess && hipSetDevice(ctx->device) == hipSuccess) {
        if (ctx->ws) (void)hipFree(ctx->ws);
        if (ctx->sws) (void)hipFree(ctx->sws);
        if (ctx->shost) (void)hipHostFree(ctx->shost);
        (void)hipFree(ctx->dmem);
        (void)hipSetDevice(prev);
    }
    delete ctx;
}

}  // extern "C"

namespace {

int check_cands(const poseidon_ctx *ctx, const poseidon_cands *c) {
    if (!ctx || !c) return POSEIDON_E_INVAL;
    if (c->count >= (1ull << 32)) return POSEIDON_E_RANGE;
    if (!c->comp_rank) {
        if (c->assign_idx) return POSEIDON_E_INVAL;
        const unsigned __int128 tot = (unsigned __int128)ctx->n_comp * ctx->A;
        if ((unsigned __int128)c->first + c->count > tot) return POSEIDON_E_INVAL;
    }
    return POSEIDON_OK;
}

struct DeviceGuard {
    int prev = -1;
    bool ok = false;
    explicit DeviceGuard(int dev) {
        ok = hipGetDevice(&prev) == hipSuccess && hipSetDevice(dev) == hipSuccess;
    }
    ~DeviceGuard() {
        if (prev >= 0) (void)hipSetDevice(prev);
    }
};

// The device word holds (T << 32 | position within the call); the index
// returned is base + position.
int read_best(poseidon_ctx *ctx, hipStream_t st, unsigned long long word_index, uint64_t base,
              poseidon_best *best) {
    unsigned long long w[W_COUNT];
    if (hipMemcpyAsync(w, ctx->state, sizeof(w), hipMemcpyDeviceToHost, st) != hipSuccess ||
        hipStreamSynchronize(st) != hipSuccess)
        return POSEIDON_E_DEVICE;
    if (w[W_ERR] & 0xFFFFFFFFull) {
        const unsigned long long zero = 0;
        (void)hipMemcpy(ctx->state + W_ERR, &zero, 8, hipMemcpyHostToDevice);
        return POSEIDON_E_INVAL;
    }
    const unsigned long long k = w[word_index];
    if (k == ~0ull || (k >> 32) == 0xFFFFFFFFull) {
        best->index = UINT64_MAX;
        best->makespan = 0xFFFFFFFFu;
        best->feasible = 0;
        return POSEIDON_NO_FEASIBLE;
    }
    best->index = base + (k & 0xFFFFFFFFull);
    best->makespan = (uint32_t)(k >> 32);
    best->feasible = 1;
    return POSEIDON_OK;
}

// Largest number of candidates one launch sequence handles; longer calls
// are processed in chunks of this size.
constexpr uint64_t kChunk = 1ull << 26;

// Workspace for chunks of up to `n` candidates: the cut codes [words][cap],
// the early-stop survivor indices [cap] and per-block survivor counts
// [grid_max] (cap = n plus one decode batch per block of slack, so the
// per-block survivor segments fit) and, with a cascade, two straggler
// queues of qcap entries of queue_entry_words uint32
// (qcap = n plus one block of slack per segment) and the per-block queue
// counts [levels][grid_max].  Grown on demand; the old buffer is released
// only after the stream has drained.
uint64_t queue_cap(const poseidon_ctx *ctx, uint64_t n) { return n + (uint64_t)ctx->grid_max * 256; }

// DP state words per queue entry: S registers for 1F1B, 2S for Eager 1F1B,
// the live registers at a period boundary for Interleaved 1F1B
uint64_t queue_state_words(const poseidon_ctx *ctx) {
    if (ctx->base.sched == POSEIDON_SCHEDULE_INTERLEAVED_1F1B)
        return (uint64_t)pk::ilv_state_words(ctx->S, ctx->base.ndev);
    return ctx->base.sched ? 2ull * ctx->S : ctx->S;
}

// Words of one queue entry: candidate index, cut codes, the assignment
// index (room for it whenever the problem has more than one assignment;
// used by calls with a list of assignment indices) and the DP state.
uint64_t queue_entry_words(const poseidon_ctx *ctx) {
    return 1 + (uint64_t)pk::code_words((int)ctx->S) + (ctx->A > 1 ? 1 : 0) + queue_state_words(ctx);
}

int ensure_workspace(poseidon_ctx *ctx, uint64_t n, hipStream_t st) {
    if (ctx->ws_cap >= n) return POSEIDON_OK;
    if (ctx->ws) {
        if (hipStreamSynchronize(st) != hipSuccess) return POSEIDON_E_DEVICE;
        (void)hipFree(ctx->ws);
        ctx->ws = nullptr;
        ctx->ws_cap = 0;
    }
    // (a multiple of 4 words: the range-mode decode stores four code words at once)
    const uint64_t cap = (std::max<uint64_t>(n, 1024) + (uint64_t)ctx->grid_max * pk::kDecodeIlp * 256 + 3) & ~3ull;
    const uint64_t words = (uint64_t)pk::code_words((int)ctx->S);
    // cut codes, the early stop's survivor and first-stage lists and their counts
    uint64_t elems = (words + 1 + pk::kAListWords) * cap + 2ull * ctx->grid_max;
    if (ctx->base.nlevels)
        elems += 2 * queue_entry_words(ctx) * queue_cap(ctx, cap) +
                 (uint64_t)pk::kMaxLevels * ctx->grid_max;
    // the kernels address the code words, each list and each queue with
    // 32-bit word offsets (n is at most kChunk, so this always holds)
    if ((words + pk::kAListWords) * cap >= (1ull << 32) || queue_entry_words(ctx) * queue_cap(ctx, cap) >= (1ull << 32))
        return POSEIDON_E_RANGE;
    void *q = nullptr;
    if (hipMalloc(&q, elems * 4) != hipSuccess) {
        (void)hipGetLastError();
        return POSEIDON_E_NOMEM;
    }
    ctx->ws = q;
    ctx->ws_cap = cap;
    return POSEIDON_OK;
}

// After a failed launch: re-arm the reduction words and queue counters.
int rearm(poseidon_ctx *ctx, hipStream_t st) {
    (void)pk::launch_fill(ctx->state + W_ACC, 1, ~0ull, st);
    (void)pk::launch_fill(ctx->state + W_DONE, 1, 0ull, st);
    return POSEIDON_E_DEVICE;
}

// Grid of the evaluation kernels for a chunk of n candidates, and the queue
// slots its blocks own: block b of every level holds seg_cap entries, so a
// chunk's queues need grid * seg_cap slots (non-decreasing in n).
struct ChunkGrid {
    uint32_t grid;
    uint64_t seg_cap;
};
ChunkGrid chunk_grid(const poseidon_ctx *ctx, uint64_t n) {
    ChunkGrid g;
    g.grid = (uint32_t)std::min<uint64_t>((n + 255) / 256, ctx->grid_max);
    const uint64_t stride = (uint64_t)g.grid * 256;
    g.seg_cap = (n + stride - 1) / stride * 256;
    return g;
}

// Largest power-of-two chunk (at least one wave) whose cut codes, straggler
// queues and queue counts fit the allocation-free scratch; 0 if none does.
uint64_t noalloc_chunk_for(const poseidon_ctx *ctx) {
    const uint64_t words = (uint64_t)pk::code_words((int)ctx->S), ent = queue_entry_words(ctx);
    const uint64_t cap_words = pk::noalloc_scratch_bytes() / 4;
    for (uint64_t n = kChunk; n >= 64; n >>= 1) {
        const ChunkGrid g = chunk_grid(ctx, n);
        uint64_t need = words * n;
        if (ctx->base.nlevels) need += 2 * ent * g.grid * g.seg_cap + (uint64_t)pk::kMaxLevels * g.grid;
        if (need <= cap_words) return n;
    }
    return 0;
}

// One evaluation call in chunks of at most `chunk` candidates on a
// workspace: cut codes [words][ccap] at `codes`; with a cascade, two
// straggler queues of qcap entries of queue_entry_words at `queues`,
// followed by the per-block queue counts [levels][grid].
int eval_chunks(poseidon_ctx *ctx, const poseidon_cands *cands, uint32_t *makespan_out,
                uint32_t *feasible_bits_out, poseidon_best *best_out, hipStream_t st, uint64_t chunk,
                uint32_t *codes, uint64_t ccap, uint32_t *queues, uint64_t qcap) {
    pk::KParams kp = ctx->base;
    kp.first = cands->first;
    kp.count = cands->count;
    kp.comp_rank = cands->comp_rank;
    kp.assign_idx = cands->assign_idx;
    // queue entries have room for the assignment index only when A > 1
    kp.qasg = cands->comp_rank && cands->assign_idx && ctx->A > 1 ? 1u : 0u;
    kp.makespan_out = makespan_out;
    kp.feas_bits_out = feasible_bits_out;
    kp.nwords = (cands->count + 31) / 32;
    kp.codes = codes;
    kp.ccap = ccap;
    if (kp.nlevels) {
        kp.qcap = qcap;
        kp.queue[0] = queues;
        kp.queue[1] = kp.queue[0] + queue_entry_words(ctx) * kp.qcap;
        kp.qcount = kp.queue[1] + queue_entry_words(ctx) * kp.qcap;
    }
    for (uint64_t c0 = 0; c0 < cands->count; c0 += chunk) {
        kp.first_i = c0;
        kp.n_i = std::min(chunk, cands->count - c0);
        kp.accumulate = c0 > 0;
        const ChunkGrid g = chunk_grid(ctx, kp.n_i);
        pk::LaunchCfg lc;
        lc.lds_bytes = ctx->base.sched == POSEIDON_SCHEDULE_INTERLEAVED_1F1B ? ctx->lds_bytes : ctx->ent_lds_bytes;
        lc.grid = g.grid;
        // queue segments: block b of every level owns seg_cap slots
        kp.nseg = lc.grid;
        kp.seg_cap = g.seg_cap;
        pk::LaunchCfg ld = lc;
        ld.grid = (uint32_t)std::min<uint64_t>((kp.n_i + 4 * 256 - 1) / (4 * 256), ctx->grid_max);
        if (pk::launch_decode(kp, ld, st) != hipSuccess) return rearm(ctx, st);
        if (pk::launch_eval(kp, lc, st) != hipSuccess) return rearm(ctx, st);
        for (uint32_t l = 1; l <= kp.nlevels; ++l)
            if (pk::launch_resume(kp, lc, st, l) != hipSuccess) return rearm(ctx, st);
    }
    if (best_out) return read_best(ctx, st, W_RESULT, ctx->result_base, best_out);
    return POSEIDON_OK;
}

}  // namespace

extern "C" {

int poseidon_eval_candidates(poseidon_ctx *ctx, const poseidon_cands *cands, uint32_t *makespan_out,
                             uint32_t *feasible_bits_out, poseidon_best *best_out, void *hip_stream) {
    int rc = check_cands(ctx, cands);
    if (rc != POSEIDON_OK) return rc;
    hipStream_t st = (hipStream_t)hip_stream;
    DeviceGuard g(ctx->device);
    if (!g.ok) return POSEIDON_E_DEVICE;
    ctx->result_base = cands->comp_rank ? 0 : cands->first;
    if (cands->count == 0) {
        // nothing to evaluate: publish an empty result
        if (pk::launch_fill(ctx->base.result, 1, ~0ull, st) != hipSuccess) return POSEIDON_E_DEVICE;
        if (best_out) return read_best(ctx, st, W_RESULT, ctx->result_base, best_out);
        return POSEIDON_OK;
    }
    const uint64_t chunk = std::min<uint64_t>(cands->count, kChunk);
    rc = ensure_workspace(ctx, chunk, st);
    if (rc != POSEIDON_OK) return rc;
    // workspace: cut codes [words][cap]; the early stop's survivor indices
    // [cap], their counts [grid_max], its first-stage list [kAListWords][cap]
    // and counts [grid_max]; then the straggler queues
    uint32_t *ws = (uint32_t *)ctx->ws;
    const uint64_t words = (uint64_t)pk::code_words((int)ctx->S);
    return eval_chunks(ctx, cands, makespan_out, feasible_bits_out, best_out, st, chunk, ws, ctx->ws_cap,
                       ws + (words + 1 + pk::kAListWords) * ctx->ws_cap + 2ull * ctx->grid_max,
                       queue_cap(ctx, ctx->ws_cap));
}

int poseidon_eval_candidates_noalloc(poseidon_ctx *ctx, const poseidon_cands *cands, uint32_t *makespan_out,
                                     uint32_t *feasible_bits_out, poseidon_best *best_out, void *hip_stream) {
    int rc = check_cands(ctx, cands);
    if (rc != POSEIDON_OK) return rc;
    if (!ctx->scratch) return POSEIDON_E_DEVICE;
    if (ctx->noalloc_chunk == 0) return POSEIDON_E_RANGE;
    hipStream_t st = (hipStream_t)hip_stream;
    DeviceGuard g(ctx->device);
    if (!g.ok) return POSEIDON_E_DEVICE;
    ctx->result_base = cands->comp_rank ? 0 : cands->first;
    if (cands->count == 0) {
        if (pk::launch_fill(ctx->base.result, 1, ~0ull, st) != hipSuccess) return POSEIDON_E_DEVICE;
        if (best_out) return read_best(ctx, st, W_RESULT, ctx->result_base, best_out);
        return POSEIDON_OK;
    }
    // scratch: cut codes [words][chunk], then the straggler queues
    const uint64_t chunk = ctx->noalloc_chunk;
    const ChunkGrid cg = chunk_grid(ctx, chunk);
    uint32_t *scr = (uint32_t *)ctx->scratch;
    const uint64_t words = (uint64_t)pk::code_words((int)ctx->S);
    return eval_chunks(ctx, cands, makespan_out, feasible_bits_out, best_out, st, chunk, scr, chunk,
                       scr + words * chunk, (uint64_t)cg.grid * cg.seg_cap);
}

int poseidon_last_best(poseidon_ctx *ctx, poseidon_best *best_out, void *hip_stream) {
    if (!ctx || !best_out) return POSEIDON_E_INVAL;
    DeviceGuard g(ctx->device);
    if (!g.ok) return POSEIDON_E_DEVICE;
    return read_best(ctx, (hipStream_t)hip_stream, W_RESULT, ctx->result_base, best_out);
}

int poseidon_eval_candidates_bounded(poseidon_ctx *ctx, const poseidon_cands *cands, uint32_t bound,
                                     uint64_t chunk, uint32_t flags, poseidon_best *best_out,
                                     poseidon_prune_stats *stats_out, void *hip_stream) {
    int rc = check_cands(ctx, cands);
    if (rc != POSEIDON_OK) return rc;
    if (ctx->base.sched == POSEIDON_SCHEDULE_INTERLEAVED_1F1B) return POSEIDON_E_INVAL;
    if (flags & ~POSEIDON_BOUNDED_RAMP) return POSEIDON_E_INVAL;
    const bool ramp = flags & POSEIDON_BOUNDED_RAMP;
    hipStream_t st = (hipStream_t)hip_stream;
    DeviceGuard g(ctx->device);
    if (!g.ok) return POSEIDON_E_DEVICE;
    // re-arm the running best, its snapshot and the counters (one fill
    // kernel, not memsets)
    pk::FillRanges fr;
    fr.n = 3;
    fr.ptr[0] = ctx->state + W_RUN; fr.count[0] = 1; fr.value[0] = ~0ull;
    fr.ptr[1] = ctx->state + W_SNAP; fr.count[1] = 1; fr.value[1] = ~0ull;
    fr.ptr[2] = ctx->state + W_STAT_EVAL; fr.count[2] = 3; fr.value[2] = 0ull;
    if (pk::launch_fills(fr, st) != hipSuccess) return POSEIDON_E_DEVICE;
    pk::KParams kp = ctx->base;
    kp.first = cands->first;
    kp.count = cands->count;
    kp.comp_rank = cands->comp_rank;
    kp.assign_idx = cands->assign_idx;
    const uint64_t n = cands->count;
    if (chunk == 0 || chunk > n) chunk = n;
    // the survivor list has room for the survivors of kChunk candidates; a
    // longer chunk is filtered in pieces that all see the bound in force at
    // the chunk's start (the snapshot moves only at chunk ends)
    rc = ensure_workspace(ctx, std::min<uint64_t>(ramp ? n : chunk, kChunk), st);
    if (rc != POSEIDON_OK) return rc;
    kp.codes = (uint32_t *)ctx->ws;
    kp.ccap = ctx->ws_cap;
    kp.sidx = (uint32_t *)ctx->ws + (uint64_t)pk::code_words((int)ctx->S) * ctx->ws_cap;
    kp.scount = (unsigned int *)(kp.sidx + ctx->ws_cap);
    kp.alist = (uint32_t *)(kp.scount + ctx->grid_max);
    kp.acount = (unsigned int *)(kp.alist + (uint64_t)pk::kAListWords * ctx->ws_cap);
    kp.es_bound = bound;
    pk::LaunchCfg lc;
    lc.lds_bytes = ctx->ent_lds_bytes;
    // survivor kernel: as many blocks as the evaluation kernel keeps resident
    // (those the survivors need run, the others leave at once)
    lc.grid2 = ctx->grid_max;
    uint64_t size = chunk;
    for (uint64_t lo = 0, hi; lo < n; lo = hi) {
        hi = n - lo > size ? lo + size : n;
        if (ramp && size < n) size *= 2;
        for (uint64_t s0 = lo; s0 < hi; s0 += kChunk) {
            const uint64_t s1 = std::min(hi, s0 + kChunk);
            kp.first_i = s0;
            kp.n_i = s1 - s0;
            pk::LaunchCfg ld = lc;
            const uint64_t batch = (uint64_t)pk::kDecodeIlp * 256;
            ld.grid = (uint32_t)std::min<uint64_t>((kp.n_i + batch - 1) / batch, ctx->filter_grid);
            // block b filters kDecodeIlp candidates per lane per pass, ceil(n / (grid * batch)) passes
            kp.seg_cap = (kp.n_i + ld.grid * batch - 1) / (ld.grid * batch) * batch;
            if (pk::launch_bounded(kp, ld, st, s1 == hi) != hipSuccess) return rearm(ctx, st);
        }
    }
    unsigned long long w[W_COUNT];
    if (hipMemcpyAsync(w, ctx->state, sizeof(w), hipMemcpyDeviceToHost, st) != hipSuccess ||
        hipStreamSynchronize(st) != hipSuccess)
        return POSEIDON_E_DEVICE;
    if (stats_out) {
        stats_out->evaluated = w[W_STAT_EVAL];
        stats_out->pruned = w[W_STAT_PRUNED];
        stats_out->infeasible = w[W_STAT_INFEAS];
    }
    if (w[W_ERR] & 0xFFFFFFFFull) {
        const unsigned long long zero = 0;
        (void)hipMemcpy(ctx->state + W_ERR, &zero, 8, hipMemcpyHostToDevice);
        return POSEIDON_E_INVAL;
    }
    const unsigned long long k = w[W_RUN];
    poseidon_best b;
    int out;
    if (k == ~0ull || (uint32_t)(k >> 32) > bound) {
        b.index = UINT64_MAX; b.makespan = 0xFFFFFFFFu; b.feasible = 0;
        out = POSEIDON_NO_FEASIBLE;
    } else {
        b.index = (cands->comp_rank ? 0 : cands->first) + (k & 0xFFFFFFFFull);
        b.makespan = (uint32_t)(k >> 32); b.feasible = 1;
        out = POSEIDON_OK;
    }
    if (best_out) *best_out = b;
    return out;
}

int poseidon_argmin(poseidon_ctx *ctx, const uint32_t *makespan, const uint32_t *feasible_bits, uint64_t count,
                    uint64_t index_base, poseidon_best *best_out, void *hip_stream) {
    if (!ctx || !makespan || !best_out) return POSEIDON_E_INVAL;
    if (count >= (1ull << 32)) return POSEIDON_E_RANGE;
    hipStream_t st = (hipStream_t)hip_stream;
    DeviceGuard g(ctx->device);
    if (!g.ok) return POSEIDON_E_DEVICE;
    if (count == 0) {
        if (pk::launch_fill(ctx->base.result, 1, ~0ull, st) != hipSuccess) return POSEIDON_E_DEVICE;
    } else {
        const uint32_t grid = (uint32_t)std::min<uint64_t>((count + 255) / 256, 1024);
        if (pk::launch_argmin(makespan, feasible_bits, count, grid, ctx->base.acc, ctx->base.done, ctx->base.result,
                              st) != hipSuccess)
            return POSEIDON_E_DEVICE;
    }
    ctx->result_base = index_base;
    return read_best(ctx, st, W_RESULT, index_base, best_out);
}

}  // extern "C"

// ---------------------------------------------------------------------------
// Pruned search (Sec. 4.2.3)
// ---------------------------------------------------------------------------
namespace {

constexpr uint64_t kSearchCap = 1ull << 22;            // nodes per frontier piece
constexpr uint32_t kSearchBlk = kSearchCap / 256;      // blocks per piece
static_assert(kSearchBlk <= pk::kSearchScanMax, "a level piece must fit the scan kernel");

// state words: counters, leaf key, best, bound, one child total per level,
// then the count kernels' counter slots
enum {
    SW_STATS = 0, SW_ACC = 5, SW_BEST = 6, SW_BOUND = 9, SW_TOTAL = 10, SW_PART = SW_TOTAL + pk::kSMax,
    SW_COUNT = SW_PART + 5 * pk::kStatSlots
};

struct SearchWs {
    uint32_t *row[pk::kSMax], *codes[pk::kSMax];
    unsigned int *tot[pk::kSMax];
    unsigned long long *off[pk::kSMax];
    uint16_t *node[pk::kSMax];
    unsigned long long *words;
};

// Per level: rows, cut codes, block counts and offsets; then the state words.
SearchWs search_layout(poseidon_ctx *ctx, size_t *bytes) {
    SearchWs w;
    memset(&w, 0, sizeof(w));
    const uint64_t words = (uint64_t)pk::code_words((int)ctx->S);
    unsigned char *b = (unsigned char *)ctx->sws;
    size_t o = 0;
    for (uint32_t l = 0; l < ctx->S; ++l) {
        w.row[l] = (uint32_t *)(b + o); o += kSearchCap * 4;
        w.codes[l] = (uint32_t *)(b + o); o += words * kSearchCap * 4;
        w.tot[l] = (unsigned int *)(b + o); o += (size_t)kSearchBlk * 4;
        w.node[l] = (uint16_t *)(b + o); o += kSearchCap * 2;
        w.off[l] = (unsigned long long *)(b + o); o += ((size_t)kSearchBlk + 1) * 8;
    }
    w.words = (unsigned long long *)(b + o); o += SW_COUNT * 8;
    if (bytes) *bytes = o;
    return w;
}

struct SearchRun {
    poseidon_ctx *ctx;
    pk::KParams kp;
    pk::SearchParams q;
    SearchWs w;
    hipStream_t st;
    std::vector<unsigned long long> off;
};

int search_read_total(SearchRun &r, uint32_t x, unsigned long long *total) {
    if (hipMemcpyAsync(r.ctx->shost, r.w.words + SW_TOTAL + x, 8, hipMemcpyDeviceToHost, r.st) != hipSuccess ||
        hipStreamSynchronize(r.st) != hipSuccess)
        return POSEIDON_E_DEVICE;
    *total = r.ctx->shost[0];
    return POSEIDON_OK;
}

// The level before the one that fixes the last cut (x = S - 3) is expanded
// together with it when one block's grandchildren, at most 256 (L - 1)^2,
// always fit a frontier piece.
bool search_fused(const poseidon_ctx *ctx, uint32_t x) {
    const uint64_t L = ctx->L;
    return ctx->S >= 3 && x + 3 == ctx->S && 256 * (L - 1) * (L - 1) <= kSearchCap;
}

// Expand the nodes at level x (stored in the level's arrays) depth first:
// n of them, or, with n_dev, at most n, their number being on the device.
// When every child of the level fits one frontier piece (n times the most
// children a node can have), the next level is launched on that bound
// without reading the total back; otherwise the host reads it and splits the
// level into pieces.
int search_expand(SearchRun &r, uint32_t x, uint64_t n, const unsigned long long *n_dev) {
    const uint32_t S = r.ctx->S;
    pk::SearchParams q = r.q;
    q.in_row = r.w.row[x];
    q.in_codes = r.w.codes[x];
    q.in_cap = kSearchCap;
    q.n_in = (uint32_t)n;
    q.n_dev = n_dev;
    q.level = x;
    const uint32_t grid = (uint32_t)((n + 255) / 256);
    const size_t lds = r.ctx->lds_bytes;
    // the count and write kernels add three per-type tables (fb, mfb, hm)
    const size_t lds_cw = lds + 3 * (size_t)r.ctx->T * (r.ctx->L + 1) * 4;
    if (x + 1 == S) {
        if (pk::launch_search(pk::kSearchOpLeaf, r.kp, q, grid, lds, r.st) != hipSuccess ||
            pk::launch_search(pk::kSearchOpMerge, r.kp, q, 1, 0, r.st) != hipSuccess)
            return POSEIDON_E_DEVICE;
        return POSEIDON_OK;
    }
    q.blk_tot = r.w.tot[x];
    q.blk_off = r.w.off[x];
    q.node_cnt = r.w.node[x];
    // a fused step writes level x + 2 (complete configurations when x = S - 3)
    const uint32_t step = search_fused(r.ctx, x) ? 2 : 1;
    q.fused = step == 2;
    q.out_row = r.w.row[x + step];
    q.out_codes = r.w.codes[x + step];
    q.out_cap = kSearchCap;
    q.total = r.w.words + SW_TOTAL + x;
    if (pk::launch_search(pk::kSearchOpCount, r.kp, q, grid, lds_cw, r.st) != hipSuccess ||
        pk::launch_search_scan(q, grid, r.st) != hipSuccess)
        return POSEIDON_E_DEVICE;
    const uint64_t most = step == 2 ? (uint64_t)(r.ctx->L - 1) * (r.ctx->L - 1) : r.ctx->L - 1;
    if (n * most <= kSearchCap) {
        q.blk_base = 0;
        if (pk::launch_search(pk::kSearchOpWrite, r.kp, q, grid, lds_cw, r.st) != hipSuccess) return POSEIDON_E_DEVICE;
        return search_expand(r, x + step, n * most, q.total);
    }
    unsigned long long total = 0;
    int rc = search_read_total(r, x, &total);
    if (rc != POSEIDON_OK) return rc;
    if (total == 0) return POSEIDON_OK;
    if (total <= kSearchCap) {
        q.blk_base = 0;
        if (pk::launch_search(pk::kSearchOpWrite, r.kp, q, grid, lds_cw, r.st) != hipSuccess) return POSEIDON_E_DEVICE;
        return search_expand(r, x + step, total, nullptr);
    }
    // more children than a level holds: write and expand them in pieces of
    // whole blocks (one block has at most 256 (L - 1) < kSearchCap children,
    // or 256 (L - 1)^2 <= kSearchCap when fused)
    // (into the pinned words, grid + 1 <= kSearchBlk + 1 of them; the pieces'
    // own expansions reuse those words, so the offsets are copied out first)
    if (hipMemcpyAsync(r.ctx->shost, q.blk_off, (grid + 1) * 8, hipMemcpyDeviceToHost, r.st) != hipSuccess ||
        hipStreamSynchronize(r.st) != hipSuccess)
        return POSEIDON_E_DEVICE;
    const std::vector<unsigned long long> off(r.ctx->shost, r.ctx->shost + grid + 1);
    uint32_t b0 = 0;
    while (b0 < grid) {
        uint32_t b1 = b0 + 1;
        while (b1 < grid && off[b1 + 1] - off[b0] <= kSearchCap) ++b1;
        q.blk_base = b0;
        if (pk::launch_search(pk::kSearchOpWrite, r.kp, q, b1 - b0, lds_cw, r.st) != hipSuccess) return POSEIDON_E_DEVICE;
        if (off[b1] > off[b0]) {
            rc = search_expand(r, x + step, off[b1] - off[b0], nullptr);
            if (rc != POSEIDON_OK) return rc;
        }
        b0 = b1;
    }
    return POSEIDON_OK;
}

}  // namespace

extern "C" int poseidon_search(poseidon_ctx *ctx, uint64_t first_row, uint64_t n_rows, uint32_t bound,
                               uint64_t rows_per_chunk, uint32_t flags, poseidon_best *best_out,
                               poseidon_search_stats *stats_out, void *hip_stream) {
    if (!ctx || (flags & ~(uint32_t)(POSEIDON_SEARCH_RIDGE | POSEIDON_SEARCH_NO_STAGE_PRUNING | POSEIDON_SEARCH_RAMP)))
        return POSEIDON_E_INVAL;
    if (ctx->base.sched == POSEIDON_SCHEDULE_INTERLEAVED_1F1B) return POSEIDON_E_INVAL;
    if (first_row > ctx->A || n_rows > ctx->A - first_row) return POSEIDON_E_INVAL;
    hipStream_t st = (hipStream_t)hip_stream;
    DeviceGuard g(ctx->device);
    if (!g.ok) return POSEIDON_E_DEVICE;
    if (!ctx->sws) {
        size_t bytes = 0;
        search_layout(ctx, &bytes);
        if (hipMalloc(&ctx->sws, bytes) != hipSuccess) {
            (void)hipGetLastError();
            ctx->sws = nullptr;
            return POSEIDON_E_NOMEM;
        }
    }
    if (!ctx->shost) {
        if (hipHostMalloc((void **)&ctx->shost, ((size_t)kSearchBlk + 2) * 8, hipHostMallocDefault) != hipSuccess) {
            (void)hipGetLastError();
            ctx->shost = nullptr;
            return POSEIDON_E_NOMEM;
        }
    }
    SearchRun r;
    r.ctx = ctx;
    r.kp = ctx->base;
    r.st = st;
    r.w = search_layout(ctx, nullptr);
    memset(&r.q, 0, sizeof(r.q));
    r.q.flags = flags;
    r.q.stats = r.w.words + SW_STATS;
    r.q.stats_part = r.w.words + SW_PART;
    r.q.acc = r.w.words + SW_ACC;
    r.q.best = r.w.words + SW_BEST;
    r.q.bound = (uint32_t *)(r.w.words + SW_BOUND);
    if (pk::launch_fill(r.q.stats, 5, 0ull, st) != hipSuccess ||
        pk::launch_fill(r.q.stats_part, 5 * pk::kStatSlots, 0ull, st) != hipSuccess ||
        pk::launch_fill(r.q.acc, 4, ~0ull, st) != hipSuccess)
        return POSEIDON_E_DEVICE;
    const uint64_t chunk = rows_per_chunk ? rows_per_chunk : (n_rows ? n_rows : 1);
    const bool ramp = (flags & POSEIDON_SEARCH_RAMP) != 0;
    int rc = POSEIDON_OK;
    uint64_t size = 1;   // with ramp: the next chunk's rows, doubling up to chunk
    for (uint64_t c0 = 0, c1; c0 < n_rows && rc == POSEIDON_OK; c0 = c1) {
        c1 = c0 + std::min(n_rows - c0, ramp ? std::min(size, chunk) : chunk);
        if (size < chunk) size *= 2;
        // the chunk prunes against min(bound, best of the earlier chunks)
        if (pk::launch_search_bound(r.q, bound, st) != hipSuccess) return POSEIDON_E_DEVICE;
        for (uint64_t r0 = c0; r0 < c1 && rc == POSEIDON_OK; r0 += kSearchCap) {
            const uint32_t n = (uint32_t)std::min<uint64_t>(kSearchCap, c1 - r0);
            pk::SearchParams q = r.q;
            q.out_row = r.w.row[0];
            q.out_codes = r.w.codes[0];
            q.out_cap = kSearchCap;
            q.n_in = n;
            q.root_first = (uint32_t)(first_row + r0);
            if (pk::launch_search(pk::kSearchOpRoot, r.kp, q, (n + 255) / 256, 0, st) != hipSuccess)
                return POSEIDON_E_DEVICE;
            rc = search_expand(r, 0, n, nullptr);
        }
    }
    if (rc != POSEIDON_OK) return rc;
    unsigned long long w[SW_COUNT];
    if (hipMemcpyAsync(w, r.w.words, sizeof(w), hipMemcpyDeviceToHost, st) != hipSuccess ||
        hipStreamSynchronize(st) != hipSuccess)
        return POSEIDON_E_DEVICE;
    for (uint32_t k = 0; k < 5; ++k)
        for (uint32_t j = 0; j < pk::kStatSlots; ++j) w[SW_STATS + k] += w[SW_PART + k * pk::kStatSlots + j];
    if (stats_out) {
        stats_out->visited = w[SW_STATS];
        stats_out->evaluated = w[SW_STATS + 1];
        stats_out->pruned_memory = w[SW_STATS + 2];
        stats_out->pruned_ridge = w[SW_STATS + 3];
        stats_out->pruned_bound = w[SW_STATS + 4];
    }
    const bool found = w[SW_BEST] != ~0ull;
    if (best_out) {
        best_out->index = found ? w[SW_BEST + 2] * ctx->A + w[SW_BEST + 1] : UINT64_MAX;
        best_out->makespan = found ? (uint32_t)w[SW_BEST] : 0xFFFFFFFFu;
        best_out->feasible = found ? 1u : 0u;
    }
    return found ? POSEIDON_OK : POSEIDON_NO_FEASIBLE;
}
