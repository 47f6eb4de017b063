#pragma once
// Device code (templates) for batched evaluation of Poseidon's 1F1B-DAG training-time
// model on gfx950 (CDNA4), one candidate configuration per lane.
//
// Per lane the path is:
//   (a1) decode: index -> (composition rank, assignment) -> cut points, types
//   (a2) stage weights from per-type prefix sums held in LDS, memory check
//   (a3) the longest path of the 1F1B DAG as a register stencil
//   (a4) a wave / block / grid min-reduction of (makespan, index) keys
// and, for the early-stop variant, (a5) the Eq. 2 lower bound with
// block-local compaction of the surviving candidates.
//
// The DAG's longest path is integer add/max work with no contraction, so
// it runs on the VALU; there is nothing here for the matrix cores.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>
#include <utility>

#include "poseidon_internal.h"

namespace pk {

constexpr int kBlock = 256;            // 4 waves of 64
constexpr int kWaves = kBlock / 64;

// ---------------------------------------------------------------------------
// LDS image of the context's tables (one copy per block)
// ---------------------------------------------------------------------------
struct Lds {
    const uint64_t *cost;   // [T][L+1]  (prefix bwd << 32) | prefix fwd
    const uint32_t *pm;     // [L+1]     prefix memory
    const uint32_t *cap;    // [T]
    const uint32_t *pd;     // [T][L+1]  prefix all-reduce time (when the problem has one)
};

// Layout: cost (8-byte entries) | pm | cap | pd.
__device__ __forceinline__ Lds stage_tables(const KParams &p, unsigned char *smem) {
    uint64_t *cost = reinterpret_cast<uint64_t *>(smem);
    const uint32_t ncost = p.T * (p.L + 1);
    uint32_t *pm = reinterpret_cast<uint32_t *>(cost + ncost);
    uint32_t *cap = pm + (p.L + 1);
    for (uint32_t i = threadIdx.x; i < ncost; i += kBlock) cost[i] = p.cost[i];
    for (uint32_t i = threadIdx.x; i <= p.L; i += kBlock) pm[i] = p.pm[i];
    for (uint32_t i = threadIdx.x; i < p.T; i += kBlock) cap[i] = p.cap[i];
    uint32_t *pd = cap + p.T;
    if (p.has_ar)
        for (uint32_t i = threadIdx.x; i < ncost; i += kBlock) pd[i] = p.pd[i];
    __syncthreads();
    return Lds{cost, pm, cap, pd};
}

// Stage entries of the evaluation and early-stop kernels.  For device type
// t and end point j = 0..L the fields
//   Pf_t[j], Pb_t[j]   prefix forward and backward time,
//   hm_t[j]            the largest end point h >= j with Pm[h] - Pm[j] <= cap[t],
//   Pd_t[j]            prefix all-reduce time (with all-reduce times only)
// are uint32 at byte t * erow + field * kEntField + 4 j.  A stage [c0, c1) on
// type t then has F = Pf(c1) - Pf(c0), B = Pb(c1) - Pb(c0) and fits its
// memory iff c1 <= hm_t[c0].  Every load is 4 bytes wide at a per-lane
// address and the fields of one end point are a constant distance apart
// (the load's immediate offset): wider loads at per-lane addresses
// serialise on the LDS banks.
//
// With base-T assignment digits and T <= 4, the digit table follows: for
// every r < T^4 the entry-block offsets of the four digits of r (most
// significant first) as 16-bit fields of a uint64, so the types of four
// stages cost one division by T^4 and one load.
struct Ent {
    const unsigned char *e;    // entry blocks (byte addressed)
    const uint64_t *dig;       // [T^4] packed offsets of four digits (dig_tg > 0)
};

__device__ __forceinline__ Ent entry_tables(const KParams &p, unsigned char *smem) {
    uint4 *e = reinterpret_cast<uint4 *>(smem);
    const uint4 *g = reinterpret_cast<const uint4 *>(p.ent);
    const uint32_t n = (p.ent_bytes + 8 * p.dig_tg) / 16;
    for (uint32_t i = threadIdx.x; i < n; i += kBlock) e[i] = g[i];
    if (threadIdx.x == 0 && (p.dig_tg & 1u))   // an odd number of 8-byte digit entries
        reinterpret_cast<uint64_t *>(smem + p.ent_bytes)[p.dig_tg - 1] =
            reinterpret_cast<const uint64_t *>(reinterpret_cast<const unsigned char *>(p.ent) + p.ent_bytes)[p.dig_tg - 1];
    __syncthreads();
    return Ent{smem, reinterpret_cast<const uint64_t *>(smem + p.ent_bytes)};
}

__device__ __forceinline__ Ent entry_global(const KParams &p) {
    const unsigned char *e = reinterpret_cast<const unsigned char *>(p.ent);
    return Ent{e, reinterpret_cast<const uint64_t *>(e + p.ent_bytes)};
}

// field F of end point c in the type block at byte offset `to` (= t * erow)
template <uint32_t F>
__device__ __forceinline__ uint32_t ent(const Ent &t, uint32_t c, uint32_t to) {
    return *reinterpret_cast<const uint32_t *>(t.e + ((c << 2) + to) + F * kEntField);
}

// ---------------------------------------------------------------------------
// (a1) decode
// ---------------------------------------------------------------------------

// Cut points of the composition with lexicographic rank r (sorted cut
// tuples c_1 < ... < c_{S-1} in 1 .. L-1).  The complements y_j = L - 1 - c_j
// run the other way, and lexicographic order of the cuts is the reverse of
// the co-lexicographic order of the complements, whose rank is
// sum_j C(y_j, S - j) (combinatorial number system).  So R = C(L-1, S-1) - 1
// - r is that rank, and the cuts follow greedily: y_j is the largest y with
// C(y, S - j) <= R, then R <- R - C(y_j, S - j); the last (S - j = 1) is
// y = R.  The kernels carry q = R + 1 and find n = y_j + 1 as the smallest n
// with C(n, S - j) >= q, by a search over column S - j of the Pascal table.
// Cut points in compact form: cut j (1-based) is byte (j-1) % 4 of word
// (j-1) / 4; a valid composition has c_1 >= 1, so an all-zero first byte
// marks an invalid candidate (for S = 1 the single byte is 1 when valid).
template <int S>
struct Codes {
    static constexpr int kWords = S > 1 ? (S - 1 + 3) / 4 : 1;
};

template <int S>
__device__ __forceinline__ void pack_cuts(const uint32_t (&cut)[S + 1], bool ok, uint32_t (&w)[Codes<S>::kWords]) {
#pragma unroll
    for (int k = 0; k < Codes<S>::kWords; ++k) w[k] = 0;
    if (S == 1) {
        w[0] = ok ? 1u : 0u;
        return;
    }
#pragma unroll
    for (int j = 1; j <= S - 1; ++j) w[(j - 1) / 4] |= (ok ? cut[j] : 0u) << (8 * ((j - 1) % 4));
}

template <int S>
__device__ __forceinline__ bool unpack_cuts(const uint32_t (&w)[Codes<S>::kWords], uint32_t L,
                                            uint32_t (&cut)[S + 1]) {
    cut[0] = 0;
    cut[S] = L;
#pragma unroll
    for (int j = 1; j <= S - 1; ++j) cut[j] = (w[(j - 1) / 4] >> (8 * ((j - 1) % 4))) & 0xFFu;
    const bool ok = (w[0] & 0xFFu) != 0u;
    if (!ok) {
#pragma unroll
        for (int j = 1; j <= S - 1; ++j) cut[j] = 0;
    }
    return ok;
}

template <int S>
__device__ __forceinline__ void decode_types(const KParams &p, uint32_t a, uint32_t (&ty)[S]) {
    if (p.assign_mode == kAssignFixed) {
#pragma unroll
        for (int s = 0; s < S; ++s) ty[s] = p.fixed_types[s];
    } else if (p.assign_mode == kAssignTable) {
        const uint8_t *row = p.assign + (uint64_t)a * S;
#pragma unroll
        for (int s = 0; s < S; ++s) ty[s] = row[s];
    } else {
        // base-T digits, stage 1 most significant.  q = umulhi(a, m) with
        // m = floor(2^32 / T) + 1 is floor(a / T) or one more; one
        // correction makes it exact for every 32-bit a.
#pragma unroll
        for (int s = S - 1; s >= 0; --s) {
            uint32_t q = __umulhi(a, p.magicT);
            int32_t rem = (int32_t)(a - q * p.T);
            if (rem < 0) { q -= 1; rem += (int32_t)p.T; }
            ty[s] = (uint32_t)rem;
            a = q;
        }
    }
}

// Stage types as byte offsets of their entry blocks (t * erow; both factors
// fit 24 bits, so this is the full-rate 24-bit multiply).  Base-T digits
// with T <= 4 go four stages at a time through the digit table: the stages
// S-4..S-1 are the digits of a mod T^4, the four before them those of
// (a div T^4) mod T^4, and so on (stage 1 most significant).
template <int S>
__device__ __forceinline__ void decode_toff(const KParams &p, const Ent &t, uint32_t a, uint32_t (&to)[S]) {
    if (p.assign_mode == kAssignDigits && p.dig_tg) {
        constexpr int NG = (S + 3) / 4;
        uint32_t q = a;
#pragma unroll
        for (int k = 0; k < NG; ++k) {
            uint32_t r = q;
            if (k + 1 < NG) {
                uint32_t d = __umulhi(q, p.dig_magic);   // floor(q / T^4) or one more
                int32_t rem = (int32_t)(q - d * p.dig_tg);
                if (rem < 0) { d -= 1; rem += (int32_t)p.dig_tg; }
                r = (uint32_t)rem;
                q = d;
            }
            const uint64_t w = t.dig[r];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int s = S - 4 * k - 4 + i;   // digit i (most significant first) of group k
                if (s >= 0) to[s] = (uint32_t)(w >> (16 * i)) & 0xFFFFu;
            }
        }
        return;
    }
    if (p.assign_mode == kAssignFixed) {
        // the same offsets for every candidate: four stage types a word, each
        // word passed through an empty asm so that the offsets are unpacked
        // (scalar instructions) where they are used instead of S loop-
        // invariant values holding scalar registers through the whole kernel
#pragma unroll
        for (int g = 0; g < (S + 3) / 4; ++g) {
            uint32_t wd = (uint32_t)p.fixed_types[4 * g] | (uint32_t)p.fixed_types[4 * g + 1] << 8 |
                          (uint32_t)p.fixed_types[4 * g + 2] << 16 | (uint32_t)p.fixed_types[4 * g + 3] << 24;
            asm volatile("" : "+s"(wd));
#pragma unroll
            for (int i = 0; i < 4; ++i)
                if (4 * g + i < S) to[4 * g + i < S ? 4 * g + i : 0] = ((wd >> (8 * i)) & 0xFFu) * p.erow;
        }
        return;
    }
    uint32_t ty[S];
    decode_types<S>(p, a, ty);
#pragma unroll
    for (int s = 0; s < S; ++s) to[s] = __umul24(ty[s], p.erow);
}

// Candidate i of the call -> (rank, assignment); false if out of range.
template <typename R>
__device__ __forceinline__ bool candidate(const KParams &p, uint64_t i, R &r, uint32_t &a) {
    uint64_t rank, asg;
    if (p.comp_rank) {
        rank = p.comp_rank[i];
        asg = p.assign_idx ? p.assign_idx[i] : 0u;
    } else {
        const uint64_t idx = p.first + i;
        if (p.A == 1) { rank = idx; asg = 0; }
        else { rank = idx / p.A; asg = idx - rank * p.A; }
    }
    const bool ok = rank < p.n_comp && asg < p.A;
    r = ok ? (R)rank : (R)0;
    a = ok ? (uint32_t)asg : 0u;
    return ok;
}

// Assignment index of candidate i (valid candidates only).
__device__ __forceinline__ uint32_t assign_of(const KParams &p, uint64_t i) {
    if (p.comp_rank) return p.assign_idx ? p.assign_idx[i] : 0u;
    if (p.A == 1) return 0u;
    return (uint32_t)((p.first + i) % p.A);
}

// ---------------------------------------------------------------------------
// (a2) stage weights and memory feasibility
// ---------------------------------------------------------------------------
template <int S>
__device__ __forceinline__ bool stage_weights(const KParams &p, const Lds &t,
                                              const uint32_t (&cut)[S + 1], const uint32_t (&ty)[S],
                                              uint32_t (&F)[S], uint32_t (&B)[S]) {
    bool feas = true;
    const uint32_t row = p.L + 1;
#pragma unroll
    for (int s = 0; s < S; ++s) {
        const uint64_t *c = t.cost + ty[s] * row;
        const uint64_t hi = c[cut[s + 1]], lo = c[cut[s]];
        F[s] = (uint32_t)hi - (uint32_t)lo;
        B[s] = (uint32_t)(hi >> 32) - (uint32_t)(lo >> 32);
        const uint32_t mem = t.pm[cut[s + 1]] - t.pm[cut[s]];
        feas &= mem <= t.cap[ty[s]];   // (no short circuit: no branch per stage)
    }
    return feas;
}

// The same from the stage entries: no multiply, one address per end point.
template <int S>
__device__ __forceinline__ bool stage_weights(const KParams &p, const Ent &t, const uint32_t (&cut)[S + 1],
                                              const uint32_t (&to)[S], uint32_t (&F)[S], uint32_t (&B)[S]) {
    bool feas = true;
#pragma unroll
    for (int s = 0; s < S; ++s) {
        F[s] = ent<kEPf>(t, cut[s + 1], to[s]) - ent<kEPf>(t, cut[s], to[s]);
        B[s] = ent<kEPb>(t, cut[s + 1], to[s]) - ent<kEPb>(t, cut[s], to[s]);
        feas &= cut[s + 1] <= ent<kEHm>(t, cut[s], to[s]);   // (no short circuit: no branch per stage)
    }
    return feas;
}

// ---------------------------------------------------------------------------
// (a3) longest path of the 1F1B DAG
// ---------------------------------------------------------------------------
// With unit node weights the as-soon-as-possible start slot of every node
// puts at most one node per stage in a slot, and each cross-stage
// predecessor is still the newest node of its stage one slot later.  One
// register per stage, X[s] = finish time of stage s's newest node, therefore
// suffices: slot by slot every active stage updates from the previous
// slot's values,
//   forward : X[s] <- F_s + max(X[s], X[s-1] + cf_{s-1})
//   backward: X[s] <- B_s + max(X[s], X[s+1] + cb_s)
// and T = X[1] after the last slot (B_{1,M} is the DAG's only sink).
//
// The registers hold Y[s] = X[s] + phi_s with phi_s = cf_s + ... + cf_{S-1}
// (the transfer times of the boundaries below stage s).  A constant shift
// per stage does not change any max, and with this one the forward input
// Y[s-1] already contains cf_{s-1}, so the updates become
//   forward : Y[s] <- F_s + max(Y[s], Y[s-1])
//   backward: Y[s] <- B_s + max(Y[s], Y[s+1] + (cf_s + cb_s))
// which saves one add per forward node that has an upstream stage; the
// result is T = Y[1] - phi_1.
//
// For M >= S the 2(M+S-1) slots are a prologue of 2S-1 slots, a steady part
// in which stage s (1-based) runs a forward pass in slots k = s+1 (mod 2)
// and a backward pass in the others, and an epilogue of 2S-2 slots.

constexpr int kIdle = 0, kFwd = 1, kBwd = 2;

// slot k < 2S-1 (prologue), 1-based stage s
__host__ __device__ constexpr int pro_op(int S, int s, int k) {
    return (k >= s - 1 && k <= S - 1) ? kFwd
         : (k >= 2 * S - s + 1 && ((k - s - 1) & 1) == 0) ? kFwd
         : (k >= 2 * S - s && ((k - s) & 1) == 0) ? kBwd
         : kIdle;
}
// slot 2M + j, j < 2S-2 (epilogue)
__host__ __device__ constexpr int epi_op(int S, int s, int j) {
    return (((j - s - 1) & 1) == 0 && j <= s - 3) ? kFwd
         : (((j - s) & 1) == 0 && j <= 2 * S - s - 2) ? kBwd
         : kIdle;
}

// wave-uniform transfer weights after the shift (SGPRs)
template <int S>
struct Comm {
    uint32_t e[S > 1 ? S - 1 : 1];   // cf_s + cb_s, 0-based boundary s
    uint32_t phi0;                   // cf_0 + ... + cf_{S-2}
};

template <int S>
__device__ __forceinline__ uint32_t node(int op, int s, const uint32_t (&Y)[S], const uint32_t (&F)[S],
                                         const uint32_t (&B)[S], const Comm<S> &c) {
    // s is 0-based here
    if (op == kFwd) return F[s] + (s > 0 ? max(Y[s], Y[s > 0 ? s - 1 : 0]) : Y[s]);
    if (op == kBwd)
        return B[s] + (s < S - 1 ? max(Y[s], Y[s < S - 1 ? s + 1 : 0] + c.e[s < S - 1 ? s : 0]) : Y[s]);
    return Y[s];
}

// Registers before the first slot: stage 1 starts at phi_1 (its X is 0);
// every other stage's first node is a forward pass whose upstream input is
// at least phi_s, so 0 there leaves every max unchanged.
template <int S>
__device__ __forceinline__ void dp_init(uint32_t (&Y)[S], const Comm<S> &c) {
#pragma unroll
    for (int s = 0; s < S; ++s) Y[s] = 0;
    Y[0] = c.phi0;
}

template <int S>
__device__ __forceinline__ void steady_slot(int parity, uint32_t (&Y)[S], const uint32_t (&F)[S],
                                            const uint32_t (&B)[S], const Comm<S> &c) {
    uint32_t N[S];
#pragma unroll
    for (int s = 0; s < S; ++s) {
        // 1-based stage s+1 runs forward when k = s+2 (mod 2), i.e. k = s (mod 2)
        const int op = (((s & 1) == parity) ? kFwd : kBwd);
        N[s] = node<S>(op, s, Y, F, B, c);
    }
#pragma unroll
    for (int s = 0; s < S; ++s) Y[s] = N[s];
}

// k * x for a small k; U24: the full-rate 24-bit multiply (the problem's
// stage weights fit 24 bits).  The callers take U24 as a template argument
// and branch once on it, so that no select merges the two products into one
// slow 32-bit multiply.
template <bool U24>
__device__ __forceinline__ uint32_t mul_small(uint32_t x, uint32_t k) {
    return U24 ? __umul24(x, k) : x * k;
}

// Prologue (slots 0 .. 2S-2) with its warm-up forwards in closed form.
// Stage s (0-based) first runs S - s forwards F_{s,1..S-s} in slots
// s .. S-1; each reads only its own stage's previous forward and the same
// micro-batch's forward upstream, and with the potential shift every
// forward edge weighs 0.  So the longest path to F_{s,m} is the heaviest
// monotone path through a grid whose row i carries the constant weight F_i:
// it visits rows 0..s once each and spends its other m - 1 steps on the
// heaviest of them,
//     Y[s] = phi_0 + (F_0 + ... + F_s) + (m - 1) max(F_0, ..., F_s),  m = S - s.
// Slots S .. 2S-2 (the first backwards and the forwards between them) run
// on the stencil.  U24: every stage weight is below 2^24.
template <int S, bool U24>
__device__ __forceinline__ void dp_prologue_t(uint32_t (&Y)[S], const uint32_t (&F)[S], const uint32_t (&B)[S],
                                              const Comm<S> &c) {
    uint32_t pre = c.phi0, mx = 0;
#pragma unroll
    for (int s = 0; s < S; ++s) {
        pre += F[s];
        mx = max(mx, F[s]);
        Y[s] = pre + mul_small<U24>(mx, S - 1 - s);
    }
#pragma unroll
    for (int k = S; k < 2 * S - 1; ++k) {
        uint32_t N[S];
#pragma unroll
        for (int s = 0; s < S; ++s) N[s] = node<S>(pro_op(S, s + 1, k), s, Y, F, B, c);
#pragma unroll
        for (int s = 0; s < S; ++s) Y[s] = N[s];
    }
}

template <int S>
__device__ __forceinline__ void dp_prologue(uint32_t (&Y)[S], const uint32_t (&F)[S], const uint32_t (&B)[S],
                                            const Comm<S> &c, bool u24) {
    if (u24) dp_prologue_t<S, true>(Y, F, B, c);
    else dp_prologue_t<S, false>(Y, F, B, c);
}

// one steady iteration: an odd slot then an even slot (slots 2S-1+2i, 2S+2i)
template <int S>
__device__ __forceinline__ void dp_iter(uint32_t (&Y)[S], const uint32_t (&F)[S], const uint32_t (&B)[S],
                                        const Comm<S> &c) {
    steady_slot<S>(1, Y, F, B, c);
    steady_slot<S>(0, Y, F, B, c);
}

// the last steady slot (2M-1) and the epilogue; afterwards Y[s] holds the
// (shifted) finish of B_{s,M}, the last node of every stage
template <int S>
__device__ __forceinline__ void dp_finish(uint32_t (&Y)[S], const uint32_t (&F)[S], const uint32_t (&B)[S],
                                          const Comm<S> &c) {
    steady_slot<S>(1, Y, F, B, c);
#pragma unroll
    for (int j = 0; j < 2 * S - 2; ++j) {
        uint32_t N[S];
#pragma unroll
        for (int s = 0; s < S; ++s) N[s] = node<S>(epi_op(S, s + 1, j), s, Y, F, B, c);
#pragma unroll
        for (int s = 0; s < S; ++s) Y[s] = N[s];
    }
}

// The last steady slot and the epilogue with the drain in closed form, for
// the DAG without all-reduce nodes; returns T = finish(B_{1,M}).
// Stage s (0-based) ends with its last forward F_{s,M} and then its drain,
// the S - s backwards B_{s,m}, m = M-S+s+1 .. M.  Each drain node's
// predecessors are drain nodes, except at the drain's first node: its own
// stage's F_{s,M} and the stage below's last backward before its drain,
// B_{s+1,M-S+s+1} (edge cb_s); and no node outside the drains reads a drain
// node.  Inside the drains a path from stage s to B_{1,M} runs down the
// stages s, s-1, .., 0 (edges cb_i) and takes S - 1 - s more steps along
// its stages, best spent on the heaviest backward, so
//   T = max_s [ max(fin F_{s,M}, fin B_{s+1,M-S+s+1} + cb_s)
//              + (B_0 + .. + B_s) + (cb_0 + .. + cb_{s-1}) + (S-1-s) max(B_0 .. B_s) ].
// The stencil below computes only the nodes outside the drains and keeps,
// per stage, its register just before (Yb) and after (Yf) its last forward:
// the backward before F_{s,M} is B_{s,M-S+s}, the one stage s-1's drain
// starts from.  In shifted registers the bracket is
//   max(Yf[s], Yb[s+1] + cf_s + cb_s) - phi_s, and the constant
//   cb_0 + .. + cb_{s-1} - phi_s is -phi_0 + (cf_0 + cb_0) + .. + (cf_{s-1} + cb_{s-1})
// (modulo 2^32: every sum that reaches T is a path length below 2^31).
template <int S, bool U24>
__device__ __forceinline__ uint32_t dp_finish_t(const KParams &p, uint32_t (&Y)[S], const uint32_t (&F)[S],
                                                const uint32_t (&B)[S], const Comm<S> &c) {
    uint32_t Yf[S], Yb[S];
    Yf[0] = Y[0];                         // stage 0's last forward ran in slot 2M-2
    Yb[S > 1 ? 1 : 0] = Y[S > 1 ? 1 : 0];  // stage 1's runs in slot 2M-1
    {
        // slot 2M-1 without stage 0's backward (the first of its drain)
        uint32_t N[S];
#pragma unroll
        for (int s = 0; s < S; ++s) N[s] = node<S>(s == 0 ? kIdle : ((s & 1) ? kFwd : kBwd), s, Y, F, B, c);
#pragma unroll
        for (int s = 0; s < S; ++s) Y[s] = N[s];
    }
    if (S > 1) Yf[1] = Y[1];
    // epilogue slots 2M + j: stage s >= 2 runs its last forward at j = s - 2;
    // its backwards from j = s - 1 on are drain nodes
#pragma unroll
    for (int j = 0; j + 2 < S; ++j) {
        uint32_t N[S];
#pragma unroll
        for (int s = 0; s < S; ++s) {
            int op = epi_op(S, s + 1, j);
            if (op == kBwd && j >= s - 1) op = kIdle;
            if (op == kFwd && j == s - 2) Yb[s] = Y[s];
            N[s] = node<S>(op, s, Y, F, B, c);
        }
#pragma unroll
        for (int s = 0; s < S; ++s) {
            if (epi_op(S, s + 1, j) == kFwd && j == s - 2) Yf[s] = N[s];
            Y[s] = N[s];
        }
    }
    // ek = cb_0 + .. + cb_{s-1} - phi_s = -phi_0 + e_0 + .. + e_{s-1} (mod 2^32)
    uint32_t T = 0, pb = 0, mxb = 0, ek = 0u - c.phi0;
#pragma unroll
    for (int s = 0; s < S; ++s) {
        pb += B[s];
        mxb = max(mxb, B[s]);
        const uint32_t a = s + 1 < S ? max(Yf[s], Yb[s + 1 < S ? s + 1 : 0] + c.e[s + 1 < S ? s : 0]) : Yf[s];
        T = max(T, a + pb + mul_small<U24>(mxb, S - 1 - s) + ek);
        if (s + 1 < S) ek += c.e[s + 1 < S ? s : 0];
    }
    return T;
}

template <int S>
__device__ __forceinline__ void dp_1f1b(uint32_t M, bool u24, const uint32_t (&F)[S], const uint32_t (&B)[S],
                                        const Comm<S> &c, uint32_t (&Y)[S]) {
    dp_prologue<S>(Y, F, B, c, u24);
    for (uint32_t it = S; it < M; ++it) dp_iter<S>(Y, F, B, c);
    dp_finish<S>(Y, F, B, c);
}

// The steady iteration is one fixed map Y -> A(Y) built from max and +
// only, so A(Y + c) = A(Y) + c for every constant c.  Once one iteration
// raises every stage by the same amount d, every later iteration does the
// same: after n more iterations the state is exactly Y + n d.  The kernels
// check this at a few iteration counts; a lane that passes jumps to the end
// of the steady part, the others are queued and resumed by the next level.
template <int S>
__device__ __forceinline__ bool dp_settled(const uint32_t (&Y)[S], const uint32_t (&Yp)[S], uint32_t &d) {
    d = Y[0] - Yp[0];
    bool same = true;
#pragma unroll
    for (int s = 1; s < S; ++s) same = same && (Y[s] - Yp[s] == d);
    return same;
}

// run iterations k0+1 .. k1 (k0 <= k1 <= nit); returns whether the state
// settled by iteration k1 and, if so, moves it to iteration `nit` (the end).
// With k1 = nit it simply runs to the end.
template <int S>
__device__ __forceinline__ bool dp_advance(uint32_t (&Y)[S], const uint32_t (&F)[S], const uint32_t (&B)[S],
                                           const Comm<S> &c, uint32_t k0, uint32_t k1, uint32_t nit) {
    if (k1 >= nit) {
        for (uint32_t it = k0; it < nit; ++it) dp_iter<S>(Y, F, B, c);
        return true;
    }
    for (uint32_t it = k0 + 1; it < k1; ++it) dp_iter<S>(Y, F, B, c);
    uint32_t Yp[S];
#pragma unroll
    for (int s = 0; s < S; ++s) Yp[s] = Y[s];
    dp_iter<S>(Y, F, B, c);
    uint32_t d;
    const bool ok = dp_settled<S>(Y, Yp, d);
    const uint32_t jump = ok ? (nit - k1) * d : 0u;
#pragma unroll
    for (int s = 0; s < S; ++s) Y[s] += jump;
    return ok;
}

// 1F1B with M < S: the slot schedule comes from a table of per-slot
// forward / backward stage masks built on the host (the host checks that
// every input is still its stage's newest node, so one register suffices).
template <int S>
__device__ __forceinline__ void dp_table(const KParams &p, const uint32_t (&F)[S], const uint32_t (&B)[S],
                                         const Comm<S> &c, uint32_t (&Y)[S]) {
    dp_init<S>(Y, c);
    for (uint32_t k = 0; k < p.nslots; ++k) {
        const uint32_t fm = p.slot_mask[3 * k], bm = p.slot_mask[3 * k + 2];
        uint32_t N[S];
#pragma unroll
        for (int s = 0; s < S; ++s) {
            const int op = ((fm >> s) & 1u) ? kFwd : (((bm >> s) & 1u) ? kBwd : kIdle);
            N[s] = node<S>(op, s, Y, F, B, c);
        }
#pragma unroll
        for (int s = 0; s < S; ++s) Y[s] = N[s];
    }
}

// Any schedule table (Eager 1F1B, Sec. 4.1.4 / App. B.1).  A stage can
// run ahead of its downstream neighbour by more than one forward pass, so
// a forward node may need the upstream stage's second-newest forward; the
// host marks those nodes in a third mask.  Per stage the registers are the
// newest node of either kind (Y), the newest and previous forward (Fn, Fp)
// and the newest backward (Bn), all shifted by the stage's potential.
template <int S>
__device__ __forceinline__ void dp_sched(const KParams &p, const uint32_t (&F)[S], const uint32_t (&B)[S],
                                         const Comm<S> &c, uint32_t (&Y)[S]) {
    uint32_t Fn[S], Fp[S], Bn[S];
    dp_init<S>(Y, c);
#pragma unroll
    for (int s = 0; s < S; ++s) { Fn[s] = 0; Fp[s] = 0; Bn[s] = 0; }
    for (uint32_t k = 0; k < p.nslots; ++k) {
        const uint32_t fm = p.slot_mask[3 * k], fd = p.slot_mask[3 * k + 1], bm = p.slot_mask[3 * k + 2];
        uint32_t N[S];
#pragma unroll
        for (int s = 0; s < S; ++s) {
            if ((fm >> s) & 1u) {
                const uint32_t in = s == 0 ? 0u : (((fd >> s) & 1u) ? Fp[s > 0 ? s - 1 : 0] : Fn[s > 0 ? s - 1 : 0]);
                N[s] = F[s] + max(Y[s], in);
            } else if ((bm >> s) & 1u) {
                N[s] = B[s] + (s < S - 1 ? max(Y[s], Bn[s < S - 1 ? s + 1 : 0] + c.e[s < S - 1 ? s : 0]) : Y[s]);
            } else {
                N[s] = Y[s];
            }
        }
#pragma unroll
        for (int s = 0; s < S; ++s) {
            if ((fm >> s) & 1u) { Fp[s] = Fn[s]; Fn[s] = N[s]; }
            if ((bm >> s) & 1u) Bn[s] = N[s];
            Y[s] = N[s];
        }
    }
}

// ---------------------------------------------------------------------------
// Eager 1F1B in closed form (M >= 2S-1).  Under unit weights, stage s
// (1-based) runs its 2(S-s)+1 warm-up forwards in slots s-1 .. 2S-s-1;
// from slot 2S-s on it runs a backward in every slot with k + s even and a
// forward in the others, up to its last forward in slot 2M-2S+3s-3; then
// backwards in the slots with k + s even up to 2M+2S-s-2.  That is
// 2(M+S-1) slots: a prologue of 2S-1 slots, M-2S+1 steady pairs of slots
// (2S-1+2i, 2S+2i) and an epilogue of 4S-3 slots.  A forward in the
// alternating part reads the upstream stage's previous forward (kFwdDeep),
// except the stage's last one, which reads the upstream's newest; a
// backward always reads the downstream stage's newest node.
// ---------------------------------------------------------------------------
constexpr int kFwdDeep = 3;

// prologue slot k (0 .. 2S-2), 1-based stage s
__host__ __device__ constexpr int eager_pro_op(int S, int s, int k) {
    return k < s - 1 ? kIdle : k <= 2 * S - s - 1 ? kFwd : (((k + s) & 1) == 0 ? kBwd : kFwdDeep);
}
// steady slot of parity `odd` (slot 2S-1+2i is odd)
__host__ __device__ constexpr int eager_steady_op(int s, int odd) {
    return odd ? ((s & 1) ? kBwd : kFwdDeep) : ((s & 1) ? (s == 1 ? kFwd : kFwdDeep) : kBwd);
}
// epilogue slot 2M-2S+1+j (j = 0 .. 4S-4)
__host__ __device__ constexpr int eager_epi_op(int S, int s, int j) {
    return j <= 3 * s - 4 ? (((j + 1 + s) & 1) == 0 ? kBwd : (j < 3 * s - 4 ? kFwdDeep : kFwd))
         : (j <= 4 * S - s - 3 && ((j + 1 + s) & 1) == 0) ? kBwd
         : kIdle;
}

// phase of a slot: prologue slot K, steady odd / even slot, epilogue slot K
enum EagerPhase { kPro = 0, kOdd = 1, kEven = 2, kEpi = 3 };

template <int S, int PH, int K>
__host__ __device__ constexpr int eager_op_at(int s) {
    return PH == kPro ? eager_pro_op(S, s, K)
         : PH == kOdd ? eager_steady_op(s, 1)
         : PH == kEven ? eager_steady_op(s, 0)
         : eager_epi_op(S, s, K);
}

// node of 0-based stage s with a compile-time op
template <int S, int OP, int s>
__device__ __forceinline__ uint32_t eager_node(const uint32_t (&Y)[S], const uint32_t (&Fn)[S],
                                               const uint32_t (&Fp)[S], const uint32_t (&F)[S],
                                               const uint32_t (&B)[S], const Comm<S> &c) {
    constexpr int u = s > 0 ? s - 1 : 0, d = s < S - 1 ? s + 1 : 0;
    if constexpr (OP == kFwd) return F[s] + (s > 0 ? max(Y[s], Fn[u]) : Y[s]);
    else if constexpr (OP == kFwdDeep) return F[s] + (s > 0 ? max(Y[s], Fp[u]) : Y[s]);
    else if constexpr (OP == kBwd) return B[s] + (s < S - 1 ? max(Y[s], Y[d] + c.e[d > 0 ? d - 1 : 0]) : Y[s]);
    else return Y[s];
}

template <int OP>
__device__ __forceinline__ void eager_store(uint32_t n, uint32_t &y, uint32_t &fn, uint32_t &fp) {
    if constexpr (OP == kFwd || OP == kFwdDeep) { fp = fn; fn = n; }
    y = n;
}

// one slot, every stage's op fixed at compile time (synchronous update)
template <int S, int PH, int K, int... I>
__device__ __forceinline__ void eager_slot(std::integer_sequence<int, I...>, uint32_t (&Y)[S], uint32_t (&Fn)[S],
                                           uint32_t (&Fp)[S], const uint32_t (&F)[S], const uint32_t (&B)[S],
                                           const Comm<S> &c) {
    uint32_t N[S];
    ((N[I] = eager_node<S, eager_op_at<S, PH, K>(I + 1), I>(Y, Fn, Fp, F, B, c)), ...);
    (eager_store<eager_op_at<S, PH, K>(I + 1)>(N[I], Y[I], Fn[I], Fp[I]), ...);
}

// the slots K... of a phase, in order
template <int S, int PH, int... K>
__device__ __forceinline__ void eager_run(std::integer_sequence<int, K...>, uint32_t (&Y)[S], uint32_t (&Fn)[S],
                                          uint32_t (&Fp)[S], const uint32_t (&F)[S], const uint32_t (&B)[S],
                                          const Comm<S> &c) {
    (eager_slot<S, PH, K>(std::make_integer_sequence<int, S>{}, Y, Fn, Fp, F, B, c), ...);
}

template <int S>
__device__ __forceinline__ void eager_pair(uint32_t (&Y)[S], uint32_t (&Fn)[S], uint32_t (&Fp)[S],
                                           const uint32_t (&F)[S], const uint32_t (&B)[S], const Comm<S> &c) {
    eager_slot<S, kOdd, 0>(std::make_integer_sequence<int, S>{}, Y, Fn, Fp, F, B, c);
    eager_slot<S, kEven, 0>(std::make_integer_sequence<int, S>{}, Y, Fn, Fp, F, B, c);
}

// n steady pairs, two per trip so that the forward registers come back to
// the same roles at the loop edge
template <int S>
__device__ __forceinline__ void eager_pairs(uint32_t n, uint32_t (&Y)[S], uint32_t (&Fn)[S], uint32_t (&Fp)[S],
                                            const uint32_t (&F)[S], const uint32_t (&B)[S], const Comm<S> &c) {
    for (uint32_t i = 1; i < n; i += 2) {
        eager_pair<S>(Y, Fn, Fp, F, B, c);
        eager_pair<S>(Y, Fn, Fp, F, B, c);
    }
    if (n & 1u) eager_pair<S>(Y, Fn, Fp, F, B, c);
}

template <int S>
__device__ __forceinline__ void eager_prologue(uint32_t (&Y)[S], uint32_t (&Fn)[S], uint32_t (&Fp)[S],
                                               const uint32_t (&F)[S], const uint32_t (&B)[S], const Comm<S> &c) {
    dp_init<S>(Y, c);
#pragma unroll
    for (int s = 0; s < S; ++s) { Fn[s] = 0; Fp[s] = 0; }
    eager_run<S, kPro>(std::make_integer_sequence<int, 2 * S - 1>{}, Y, Fn, Fp, F, B, c);
}

template <int S>
__device__ __forceinline__ void eager_epilogue(uint32_t (&Y)[S], uint32_t (&Fn)[S], uint32_t (&Fp)[S],
                                               const uint32_t (&F)[S], const uint32_t (&B)[S], const Comm<S> &c) {
    eager_run<S, kEpi>(std::make_integer_sequence<int, 4 * S - 3>{}, Y, Fn, Fp, F, B, c);
}

template <int S>
__device__ __forceinline__ void dp_eager(uint32_t M, const uint32_t (&F)[S], const uint32_t (&B)[S],
                                         const Comm<S> &c, uint32_t (&Y)[S]) {
    uint32_t Fn[S], Fp[S];
    eager_prologue<S>(Y, Fn, Fp, F, B, c);
    eager_pairs<S>(M - 2 * S + 1, Y, Fn, Fp, F, B, c);
    eager_epilogue<S>(Y, Fn, Fp, F, B, c);
}

// Between steady pairs the state that the rest of the DP reads is, per
// stage, the newest forward Fn and, for a stage with odd 1-based index (its
// newest node is that forward), the previous forward Fp, else the newest
// node Y (a backward; its Fp is rewritten before any read).  The pair map is
// built from max and + only, so once one pair raises all 2S values by the
// same d, every later pair does the same (as for 1F1B).  Checking it needs
// one saved value per stage: a pair moves the old Fn into Fp, so
// Fn - Fp is the forward's increment.
template <int S>
__device__ __forceinline__ bool eager_advance(uint32_t (&Y)[S], uint32_t (&Fn)[S], uint32_t (&Fp)[S],
                                              const uint32_t (&F)[S], const uint32_t (&B)[S], const Comm<S> &c,
                                              uint32_t k0, uint32_t k1, uint32_t npairs) {
    const bool last = k1 >= npairs;
    eager_pairs<S>(last ? npairs - k0 : k1 - k0 - 1, Y, Fn, Fp, F, B, c);
    if (last) return true;
    uint32_t Z[S];
#pragma unroll
    for (int s = 0; s < S; ++s) Z[s] = (s & 1) == 0 ? Fp[s] : Y[s];
    eager_pair<S>(Y, Fn, Fp, F, B, c);
    const uint32_t d = Fn[0] - Fp[0];
    bool ok = true;
#pragma unroll
    for (int s = 0; s < S; ++s)
        ok = ok && Fn[s] - Fp[s] == d && ((s & 1) == 0 ? Fp[s] : Y[s]) - Z[s] == d;
    const uint32_t jump = ok ? (npairs - k1) * d : 0u;
#pragma unroll
    for (int s = 0; s < S; ++s) { Y[s] += jump; Fn[s] += jump; Fp[s] += jump; }
    return ok;
}

// queue image of the state between pairs (2S words) and back
template <int S>
__device__ __forceinline__ void eager_pack(const uint32_t (&Y)[S], const uint32_t (&Fn)[S], const uint32_t (&Fp)[S],
                                           uint32_t (&X)[2 * S]) {
#pragma unroll
    for (int s = 0; s < S; ++s) { X[s] = Fn[s]; X[S + s] = (s & 1) == 0 ? Fp[s] : Y[s]; }
}

template <int S>
__device__ __forceinline__ void eager_unpack(const uint32_t (&X)[2 * S], uint32_t (&Y)[S], uint32_t (&Fn)[S],
                                             uint32_t (&Fp)[S]) {
#pragma unroll
    for (int s = 0; s < S; ++s) {
        Fn[s] = X[s];
        Y[s] = (s & 1) == 0 ? X[s] : X[S + s];
        Fp[s] = (s & 1) == 0 ? X[S + s] : 0u;
    }
}

// schedules other than 1F1B: the slot table (TAB) or the closed form
template <int S, bool TAB>
__device__ __forceinline__ void dp_other(const KParams &p, const uint32_t (&F)[S], const uint32_t (&B)[S],
                                         const Comm<S> &c, uint32_t (&Y)[S]) {
    if (TAB) dp_sched<S>(p, F, B, c, Y);
    else dp_eager<S>(p.M, F, B, c, Y);
}

// registers after the whole DP (any M); SCH = the problem is not 1F1B
template <int S, bool SCH>
__device__ __forceinline__ void dp_full(const KParams &p, const uint32_t (&F)[S], const uint32_t (&B)[S],
                                        const Comm<S> &c, uint32_t (&Y)[S]) {
    if (SCH && p.nslots) dp_sched<S>(p, F, B, c, Y);
    else if (SCH) dp_eager<S>(p.M, F, B, c, Y);
    else if (p.M >= (uint32_t)S) dp_1f1b<S>(p.M, p.g24 != 0, F, B, c, Y);
    else dp_table<S>(p, F, B, c, Y);
}

// The whole DP for the few lanes of a wave that survive the early-stop test:
// the closed forms take the steady-state check every kSurvStep iterations,
// and the wave leaves the steady loop as soon as all its active lanes have
// settled (jumped to its end) or reached it.
constexpr uint32_t kSurvStep = 8;


template <int S>
__device__ __forceinline__ Comm<S> load_comm(const KParams &p) {
    Comm<S> c;
    uint32_t phi = 0;
#pragma unroll
    for (int s = 0; s < (S > 1 ? S - 1 : 1); ++s) {
        c.e[s] = p.cf[s] + p.cb[s];
        phi += p.cf[s];
    }
    c.phi0 = phi;
    return c;
}

// ---------------------------------------------------------------------------
// (a5) Eq. 2: g(S_x) = sum_{i<x} F_i + M (F_x + B_x) + max_{i<=x}(sum_{j=i}^{x-1} B_j + d_i)
// ---------------------------------------------------------------------------
// Classification of a candidate against the bound b over its stages
// 0 .. X-1 in pipeline order, as the search of Sec. 4.2.3 discards a
// partial configuration: 0 if no stage fails; 1 if the first failing stage
// exceeds its device's memory (tested first at a stage); 2 if its g(S_x)
// exceeds b.  The stage weights come from the stage entries.
template <int S, bool AR, int X, bool G24>
__device__ __forceinline__ uint32_t classify_g(const KParams &p, const Ent &t, const uint32_t (&cut)[S + 1],
                                               const uint32_t (&to)[S], uint32_t b) {
    uint32_t pre = 0, inner = 0, bprev = 0, mm = 0, gm = 0;
#pragma unroll
    for (int x = 0; x < X; ++x) {
        const uint32_t F = ent<kEPf>(t, cut[x + 1], to[x]) - ent<kEPf>(t, cut[x], to[x]);
        const uint32_t B = ent<kEPb>(t, cut[x + 1], to[x]) - ent<kEPb>(t, cut[x], to[x]);
        const uint32_t D = AR ? ent<kEPd>(t, cut[x + 1], to[x]) - ent<kEPd>(t, cut[x], to[x]) : 0u;
        if (cut[x + 1] > ent<kEHm>(t, cut[x], to[x])) mm |= 1u << x;
        inner = x == 0 ? D : max(inner + bprev, D);
        // M (F + B) is below 2^31 like every path weight: a full-rate 24-bit
        // multiply when both factors fit
        const uint32_t G = G24 ? __umul24(p.M, F + B) : p.M * (F + B);
        if (pre + G + inner > b) gm |= 1u << x;
        pre += F;
        bprev = B;
    }
    const uint32_t f = mm | gm;
    return f == 0u ? 0u : (mm & f & (0u - f)) ? 1u : 2u;
}

template <int S, bool AR, int X>
__device__ __forceinline__ uint32_t classify(const KParams &p, const Ent &t, const uint32_t (&cut)[S + 1],
                                             const uint32_t (&to)[S], uint32_t b) {
    return p.g24 ? classify_g<S, AR, X, true>(p, t, cut, to, b) : classify_g<S, AR, X, false>(p, t, cut, to, b);
}

// ---------------------------------------------------------------------------
// end of the iteration: the end node E follows every R_s (Sec. 4.1.1), and
// R_s follows B_{s,M} with the stage's summed per-layer all-reduce time
// (Sec. 4.1.3).  Without all-reduce times T = finish(B_{1,M}).
// ---------------------------------------------------------------------------
template <int S>
__device__ __forceinline__ void stage_allreduce(const KParams &p, const Lds &t, const uint32_t (&cut)[S + 1],
                                                const uint32_t (&ty)[S], uint32_t (&D)[S]) {
    const uint32_t row = p.L + 1;
#pragma unroll
    for (int s = 0; s < S; ++s) D[s] = t.pd[ty[s] * row + cut[s + 1]] - t.pd[ty[s] * row + cut[s]];
}

template <int S>
__device__ __forceinline__ void stage_allreduce(const KParams &p, const Ent &t, const uint32_t (&cut)[S + 1],
                                                const uint32_t (&to)[S], uint32_t (&D)[S]) {
#pragma unroll
    for (int s = 0; s < S; ++s) D[s] = ent<kEPd>(t, cut[s + 1], to[s]) - ent<kEPd>(t, cut[s], to[s]);
}

// T from the registers after the epilogue; with all-reduce times the
// stage's cut codes `w` and assignment `a` give R_s
template <int S, bool AR>
__device__ __forceinline__ uint32_t end_time(const KParams &p, const Lds &t, const uint32_t (&Y)[S],
                                             const Comm<S> &c, const uint32_t (&w)[Codes<S>::kWords], uint32_t a) {
    if (!AR) return Y[0] - c.phi0;
    uint32_t cut[S + 1], ty[S], D[S];
    unpack_cuts<S>(w, p.L, cut);
    decode_types<S>(p, a, ty);
    stage_allreduce<S>(p, t, cut, ty, D);
    // Y[s] - phi_s = finish(B_{s,M}); phi_0 - phi_s = psi_s
    uint32_t e = 0;
#pragma unroll
    for (int s = 0; s < S; ++s) e = max(e, Y[s] + p.psi[s] + D[s]);
    return e - c.phi0;
}

template <int S, bool AR>
__device__ __forceinline__ uint32_t end_time(const KParams &p, const Ent &t, const uint32_t (&Y)[S],
                                             const Comm<S> &c, const uint32_t (&w)[Codes<S>::kWords], uint32_t a) {
    if (!AR) return Y[0] - c.phi0;
    uint32_t cut[S + 1], to[S], D[S];
    unpack_cuts<S>(w, p.L, cut);
    decode_toff<S>(p, t, a, to);
    stage_allreduce<S>(p, t, cut, to, D);
    uint32_t e = 0;
#pragma unroll
    for (int s = 0; s < S; ++s) e = max(e, Y[s] + p.psi[s] + D[s]);
    return e - c.phi0;
}

// After the steady part: T from the last steady slot, the epilogue and the
// end node (1F1B; closed-form drain without all-reduce times).
template <int S, bool AR, typename TAB>
__device__ __forceinline__ uint32_t dp_end(const KParams &p, const TAB &t, uint32_t (&Y)[S], const uint32_t (&F)[S],
                                           const uint32_t (&B)[S], const Comm<S> &c,
                                           const uint32_t (&w)[Codes<S>::kWords], uint32_t a) {
    if constexpr (AR) {
        dp_finish<S>(Y, F, B, c);
        return end_time<S, true>(p, t, Y, c, w, a);
    } else {
        if (p.g24) return dp_finish_t<S, true>(p, Y, F, B, c);
        return dp_finish_t<S, false>(p, Y, F, B, c);
    }
}

// The whole DP of one candidate with a settle check every kSurvStep steady
// iterations (the wave leaves the steady loop once all its lanes settled),
// ending in T (the end node: closed-form drain for 1F1B without all-reduce
// times, else the full epilogue and the all-reduce nodes).
template <int S, bool SCH, bool AR, typename TAB>
__device__ __forceinline__ uint32_t dp_full_settle(const KParams &p, const TAB &t, const uint32_t (&F)[S],
                                                   const uint32_t (&B)[S], const Comm<S> &c,
                                                   const uint32_t (&w)[Codes<S>::kWords], uint32_t a) {
    const unsigned long long act = __ballot(true);
    uint32_t Y[S];
    if (SCH && !p.nslots) {
        uint32_t Fn[S], Fp[S];
        eager_prologue<S>(Y, Fn, Fp, F, B, c);
        const uint32_t np = p.M - 2 * S + 1;
        bool done = false;
        for (uint32_t k = 0; k < np;) {
            const uint32_t k1 = min(k + kSurvStep, np);
            if (!done) done = eager_advance<S>(Y, Fn, Fp, F, B, c, k, k1, np);
            k = k1;
            if (__ballot(done) == act) break;
        }
        eager_epilogue<S>(Y, Fn, Fp, F, B, c);
    } else if (!SCH && p.M >= (uint32_t)S) {
        dp_prologue<S>(Y, F, B, c, p.g24 != 0);
        const uint32_t nit = p.M - S;
        bool done = false;
        for (uint32_t k = 0; k < nit;) {
            const uint32_t k1 = min(k + kSurvStep, nit);
            if (!done) done = dp_advance<S>(Y, F, B, c, k, k1, nit);
            k = k1;
            if (__ballot(done) == act) break;
        }
        return dp_end<S, AR>(p, t, Y, F, B, c, w, a);
    } else {
        dp_full<S, SCH>(p, F, B, c, Y);
    }
    return end_time<S, AR>(p, t, Y, c, w, a);
}

// ---------------------------------------------------------------------------
// (a4) reductions
// ---------------------------------------------------------------------------
__device__ __forceinline__ unsigned long long wave_min(unsigned long long v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        const unsigned long long w = __shfl_xor(v, o, 64);
        v = w < v ? w : v;
    }
    return v;
}

// Block min of `v`, folded into *acc.  When `finalize` is set (the last
// kernel of an evaluation chunk), the last block of the grid also moves *acc
// to *result (or folds it in, for the second and later chunks of a call,
// and/or into *run_best) and re-arms *acc, *done and the straggler-queue
// counters.
__device__ __forceinline__ void block_min_and_finish(unsigned long long v, unsigned long long *acc,
                                                     unsigned int *done, unsigned long long *result,
                                                     unsigned long long *run_best, bool finalize,
                                                     bool accumulate = false,
                                                     unsigned long long *snap = nullptr,
                                                     uint32_t nblocks = 0) {
    __shared__ unsigned long long part[kWaves];
    v = wave_min(v);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    if (lane == 0) part[wave] = v;
    __syncthreads();
    if (threadIdx.x == 0) {
        unsigned long long m = part[0];
#pragma unroll
        for (int w = 1; w < kWaves; ++w) m = part[w] < m ? part[w] : m;
        if (m != ~0ull) atomicMin(acc, m);
        if (finalize) {
            __threadfence();
            const unsigned int ticket = atomicAdd(done, 1u);
            if (ticket == (nblocks ? nblocks : gridDim.x) - 1) {
                __threadfence();
                const unsigned long long k = atomicExch(acc, ~0ull);
                if (result) {
                    if (accumulate) atomicMin(result, k);
                    else atomicExch(result, k);
                }
                if (run_best) {
                    const unsigned long long old = atomicMin(run_best, k);
                    if (snap) atomicExch(snap, old < k ? old : k);
                }
                atomicExch(done, 0u);
            }
        }
    }
}

__device__ __forceinline__ unsigned long long wave_sum_u32(uint32_t v) {
    unsigned long long s = v;
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) s += __shfl_xor(s, o, 64);
    return s;
}

// Exclusive prefix sum over the block's threads in thread order; every
// thread gets its offset and the block total.  All threads must call it.
__device__ __forceinline__ unsigned long long block_exclusive_scan_u64(unsigned long long v,
                                                                       unsigned long long &total) {
    __shared__ unsigned long long wtot[kWaves];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    unsigned long long inc = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const unsigned long long u = __shfl_up(inc, o, 64);
        if (lane >= o) inc += u;
    }
    if (lane == 63) wtot[wave] = inc;
    __syncthreads();
    unsigned long long before = 0, all = 0;
#pragma unroll
    for (int k = 0; k < kWaves; ++k) {
        before += k < wave ? wtot[k] : 0ull;
        all += wtot[k];
    }
    __syncthreads();
    total = all;
    return before + inc - v;
}

__device__ __forceinline__ unsigned long long make_key(bool feasible, uint32_t T, uint32_t i) {
    return ((unsigned long long)(feasible ? T : 0xFFFFFFFFu) << 32) | i;
}

// ---------------------------------------------------------------------------
// kernels
// ---------------------------------------------------------------------------

// Layout of one straggler queue: idx[cap] | codes[kWords][cap] | asg[cap]
// (calls with a list of assignment indices) | Y[NX][cap].  The entry holds
// the assignment index rather than the next level re-reading it from the
// caller's list: a 4-byte read at a scattered index costs a whole memory
// sector.
template <int S>
struct QueueView {
    uint32_t *idx, *codes, *asg, *Y;
    __device__ __forceinline__ QueueView(const KParams &p, int which) {
        idx = p.queue[which];
        codes = idx + p.qcap;
        asg = codes + (uint64_t)Codes<S>::kWords * p.qcap;
        Y = asg + (p.qasg ? p.qcap : 0ull);
    }
};

// Queue a wave's unsettled lanes (candidate index, cut codes, assignment
// index, registers) for the next level.  Block b owns slots
// [b * seg_cap, (b + 1) * seg_cap) of the queue and counts its entries in
// LDS (*nq), so no global atomic is involved; every lane of the wave must
// call this.  The assignment index (list mode with assignment indices only)
// is `a`, or with a < 0 read again from the caller's list for candidate idx
// of the call: the evaluation kernels would otherwise keep it in a register
// through the DP, which costs them more than the reload of the few lanes
// that are queued.
template <int S, int NX>
__device__ __forceinline__ void enqueue(const KParams &p, int which, unsigned int *nq, bool want, uint32_t idx,
                                        const uint32_t (&w)[Codes<S>::kWords], int64_t a,
                                        const uint32_t (&Y)[NX]) {
    const unsigned long long m = __ballot(want);
    if (m == 0) return;
    const unsigned int lane = threadIdx.x & 63;
    unsigned int base = 0;
    if (lane == 0) base = atomicAdd(nq, (unsigned int)__popcll(m));
    base = __shfl(base, 0, 64);
    if (want) {
        const unsigned long long below = lane ? (m & ((1ull << lane) - 1ull)) : 0ull;
        // 32-bit word offsets: a queue holds fewer than 2^32 words
        const uint32_t slot = blockIdx.x * (uint32_t)p.seg_cap + base + __popcll(below), qcap = (uint32_t)p.qcap;
        const QueueView<S> q(p, which);
        q.idx[slot] = idx;
#pragma unroll
        for (int k = 0; k < Codes<S>::kWords; ++k) q.codes[k * qcap + slot] = w[k];
        if (p.qasg) q.asg[slot] = a >= 0 ? (uint32_t)a : __builtin_nontemporal_load(p.assign_idx + idx);
#pragma unroll
        for (int s = 0; s < NX; ++s) q.Y[s * qcap + slot] = Y[s];
    }
}

// (a1) Unrank every candidate of the chunk [p.first_i, p.first_i + p.n_i)
// into compact cut codes.  Each lane walks kIlp candidates through their
// searches together so that the dependent LDS reads of one overlap those of
// the others.  Invalid (rank, assignment) pairs get the invalid code and
// raise the error flag.
constexpr int kIlp = kDecodeIlp;

// kIlp candidates per lane.  A kernel holds the Pascal columns it searches
// in LDS, each sorted (2^H rows, then kBucketPad rows of the type's largest
// value) and with the host's bucket table (per bucket key, the first row
// whose entry reaches the bucket; the keys are defined with bucket_lo).  The
// search for the smallest n with C(n, c) >= Q starts at the row Q's bucket
// names and halves bucket_steps(w, H, c) times over the 2^steps rows after
// it, which hold every row a value of that bucket can land on.  The last cut
// needs no search (decode_range).
// One halving: t <- 2 t + (probe < Q), as a compare into VCC and an add with
// carry-in (the compiler's select and shift-or take one VALU operation more).
__device__ __forceinline__ uint32_t tree_step(uint32_t t, uint64_t probe, uint64_t q) {
    asm("v_cmp_lt_u64_e32 vcc, %1, %2\n\tv_addc_co_u32_e32 %0, vcc, %0, %0, vcc"
                 : "+v"(t) : "v"(probe), "v"(q) : "vcc");
    return t;
}
__device__ __forceinline__ uint32_t tree_step(uint32_t t, uint32_t probe, uint32_t q) {
    asm("v_cmp_lt_u32_e32 vcc, %1, %2\n\tv_addc_co_u32_e32 %0, vcc, %0, %0, vcc"
                 : "+v"(t) : "v"(probe), "v"(q) : "vcc");
    return t;
}

// Bucket key of Q >= 1 (its leading zeros, then the 4 bits after its leading one).
__device__ __forceinline__ uint32_t bucket_key(uint64_t q) {
    const uint32_t z = (uint32_t)__clzll(q);
    return 16u * z + ((uint32_t)((q << z) >> 59) & 15u);
}
__device__ __forceinline__ uint32_t bucket_key(uint32_t q) {
    const uint32_t z = (uint32_t)__clz(q);
    return 16u * z + (((q << z) >> 27) & 15u);
}

constexpr uint32_t kBucketPad = 8;   // rows past 2^H: a search reads at most 2^3 - 2 past its start
constexpr int kBucketStepsMax = 3;

// Halvings a search over column c needs after its bucket's start row: the
// most rows the values of one bucket can land on (2^H rows of C(n, c),
// w-bit entries saturated at the type's largest value, values up to the
// column's last entry), as a power of two.  Evaluated at compile time.
__host__ __device__ constexpr int bucket_steps(int w, int H, int c) {
    const int NH = 1 << H;
    const unsigned __int128 vmax = w == 64 ? (unsigned __int128)~0ull : (unsigned __int128)0xFFFFFFFFu;
    unsigned __int128 col[256] = {};
    unsigned __int128 v = c == 0 ? 1 : 0;   // C(n, c): 0 below n = c, then C(n-1, c) n / (n - c)
    for (int n = 0; n < NH; ++n) {
        if (n == c) v = 1;
        else if (n > c) v = v * (unsigned)n / (unsigned)(n - c);
        col[n] = v < vmax ? v : vmax;
    }
    const unsigned __int128 top = col[NH - 1];
    int most = 1;
    for (int z = 0; z < w; ++z)
        for (int m = 0; m < 16; ++m) {
            const unsigned __int128 lo = bucket_lo(w, z, m);
            const unsigned __int128 nx = m < 15 ? bucket_lo(w, z, m + 1) : z > 0 ? bucket_lo(w, z - 1, 0) : vmax + 1;
            const unsigned __int128 hi = nx < top + 1 ? nx : top + 1;   // the bucket's values a search sees: [lo, hi)
            if (lo >= hi) continue;
            int a = 0, b = 0;
            for (int x = 0; x < 2; ++x) {   // first rows reaching lo and hi - 1
                const unsigned __int128 t = x == 0 ? lo : hi - 1;
                int l = 0, r = NH;
                while (l < r) {
                    const int mid = (l + r) / 2;
                    if (col[mid] < t) l = mid + 1;
                    else r = mid;
                }
                (x == 0 ? a : b) = l;
            }
            most = b - a + 1 > most ? b - a + 1 : most;
        }
    int h = 0;
    while ((1 << h) < most) ++h;
    return h;
}
static_assert(bucket_steps(64, 7, 2) == 2 && bucket_steps(64, 7, 15) == 1 && bucket_steps(32, 7, 3) == 2,
              "bucket steps of the 7-level columns");

// With 64-bit ranks the searches over columns 0 .. kNarrow-1 run in 32 bits:
// C(n, k) < 2^32 for every n <= 255 and k <= 4, and at the search over
// column k the state q is at most C(y, k) for the previous cut's complement
// y <= 254 (or C(L-1, k) at the first cut), so q, every probe and the rank
// left fit 32 bits there.  Those columns are kept in LDS as uint32 (half the
// bytes per probe); the others as R.
template <int S, typename R>
__host__ __device__ constexpr int narrow_cols() {
    return sizeof(R) == 8 ? (S < 5 ? S : 5) : 0;
}

// One cut's search for NI candidates over column c of type V (R or uint32)
// with its bucket table.  q is the decode state (see decode_start): the cut's
// complement y = L - 1 - cut is the largest y with C(y, c) <= q - 1, so
// n = y + 1 is the smallest n with C(n, c) >= q; then q <- q - C(n - 1, c)
// and the cut is L - n.
template <typename V, typename R, int HS, int NI>
__device__ __forceinline__ void search_cut(const KParams &p, const V *col, const uint8_t *tab, R (&q)[NI],
                                           uint32_t (&cut)[NI]) {
    static_assert(HS <= kBucketStepsMax, "a bucket spans at most 2^3 rows (the padding)");
    V Q[NI];
    uint32_t n0[NI], t[NI];
#pragma unroll
    for (int u = 0; u < NI; ++u) Q[u] = (V)q[u];
#pragma unroll
    for (int u = 0; u < NI; ++u) {
        n0[u] = tab[bucket_key(Q[u])];
        t[u] = 0;
    }
    // halving d probes the last row of the left half of rows
    // [n0 + t 2^(HS-d), n0 + (t + 1) 2^(HS-d))
#pragma unroll
    for (int d = 0; d < HS; ++d) {
#pragma unroll
        for (int u = 0; u < NI; ++u)
            t[u] = tree_step(t[u], col[n0[u] + (t[u] << (HS - d)) + (1u << (HS - 1 - d)) - 1u], Q[u]);
    }
#pragma unroll
    for (int u = 0; u < NI; ++u) {
        const uint32_t n = n0[u] + t[u];   // at least 1: C(0, c) = 0 < q
        q[u] = (R)(Q[u] - col[n - 1]);
        cut[u] = p.L - n;
    }
}

// LDS image of Pascal columns C0 .. C1, the ones a kernel searches (cut j
// searches column S - j, so no search reads columns 0 and 1): the wide
// columns among them (NN and up, NN = narrow_cols) as R, then the narrow ones
// as uint32, NP rows each, then their bucket tables in column order.
template <int S, typename R, int H, int C0 = 2, int C1 = S - 1>
struct Pascal {
    static constexpr uint32_t NH = 1u << H, NP = NH + kBucketPad;
    static constexpr int NN = narrow_cols<S, R>();
    static constexpr int WL = C0 > NN ? C0 : NN;              // first wide column held
    static constexpr int NWC = C1 >= WL ? C1 - WL + 1 : 0;   // wide columns held
    static constexpr int NHI = C1 < NN - 1 ? C1 : NN - 1;    // last narrow column held
    static constexpr int NNC = NHI >= C0 ? NHI - C0 + 1 : 0; // narrow columns held
    static constexpr size_t kWideBytes = (size_t)NWC * NP * sizeof(R), kNarrowBytes = (size_t)NNC * NP * 4;
    static constexpr size_t bytes() { return kWideBytes + kNarrowBytes + (size_t)(NWC + NNC) * kBucketTab; }
    const unsigned char *base;
    __device__ __forceinline__ explicit Pascal(const void *b) : base(reinterpret_cast<const unsigned char *>(b)) {}
    template <int c>
    __device__ __forceinline__ const auto *col() const {
        if constexpr (c >= NN) return reinterpret_cast<const R *>(base + (size_t)(c - WL) * NP * sizeof(R));
        else return reinterpret_cast<const uint32_t *>(base + kWideBytes + (size_t)(c - C0) * NP * 4);
    }
    template <int c>
    __device__ __forceinline__ const uint8_t *tab() const {
        return base + kWideBytes + kNarrowBytes + (size_t)(c - C0) * kBucketTab;
    }
    // the search of a cut over column c, for NI candidates
    template <int c, int NI>
    __device__ __forceinline__ void search(const KParams &p, R (&q)[NI], uint32_t (&cut)[NI]) const {
        static_assert(c >= C0 && c <= C1, "column outside the window");
        using V = typename std::conditional<(c >= NN), R, uint32_t>::type;
        search_cut<V, R, bucket_steps(8 * (int)sizeof(V), H, c)>(p, col<c>(), tab<c>(), q, cut);
    }
};

// f(integral_constant<int, i>) for i = A .. B-1 (a loop whose index is a
// constant expression)
template <int A, int B, typename F>
__device__ __forceinline__ void static_for(F &&f) {
    if constexpr (A < B) {
        f(std::integral_constant<int, A>{});
        static_for<A + 1, B>(f);
    }
}

// The decode state of lexicographic rank r: q = C(L-1, S-1) - r, which is
// one more than the co-lexicographic rank of the cut complements
// y_j = L - 1 - c_j (so q >= 1 for every valid rank).
template <typename R>
__device__ __forceinline__ R decode_start(const KParams &p, R r) {
    return (R)(p.n_comp - (uint64_t)r);
}

template <int S, typename R, int H, typename PC>
__device__ __forceinline__ void decode_ilp(const KParams &p, const PC &pc, uint32_t base,
                                           uint32_t stride, bool (&act)[kIlp], bool (&ok)[kIlp],
                                           uint32_t (&asg)[kIlp], uint32_t (&w)[kIlp][Codes<S>::kWords]) {
    constexpr int NW = Codes<S>::kWords;
    R q[kIlp];
#pragma unroll
    for (int u = 0; u < kIlp; ++u) {
        const uint32_t i = base + u * stride;
        act[u] = i < (uint32_t)p.n_i;
        ok[u] = candidate<R>(p, (uint32_t)p.first_i + (act[u] ? i : 0u), q[u], asg[u]) && act[u];
        q[u] = decode_start<R>(p, q[u]);
#pragma unroll
        for (int k = 0; k < NW; ++k) w[u][k] = 0;
    }
    // the searches, cut by cut, interleaved over the kIlp candidates; each
    // cut goes straight into its byte of the code words (cut j searches
    // column S - j)
    static_for<1, S - 1>([&](auto jc) {
        constexpr int j = decltype(jc)::value;
        uint32_t cut[kIlp];
        pc.template search<S - j>(p, q, cut);
#pragma unroll
        for (int u = 0; u < kIlp; ++u) w[u][(j - 1) / 4] |= cut[u] << (8 * ((j - 1) % 4));
    });
    if (S >= 2) {
#pragma unroll
        for (int u = 0; u < kIlp; ++u) w[u][(S - 2) / 4] |= (p.L - (uint32_t)q[u]) << (8 * ((S - 2) % 4));
    }
#pragma unroll
    for (int u = 0; u < kIlp; ++u) {
        if (S == 1) w[u][0] = 1u;
        if (!ok[u]) {
#pragma unroll
            for (int k = 0; k < NW; ++k) w[u][k] = 0u;
        }
    }
}

// Searches of cuts J0+1 .. J1 (J1 <= S - 1) of kIlp candidates from the
// decode state q after cut J0; cut S - 1, the last, needs no search (with
// one cut left, C(y, 1) = y: its complement is q - 1, so c_{S-1} = L - q).
template <int S, typename R, int H, int J0, int J1, typename PC>
__device__ __forceinline__ void decode_range(const KParams &p, const PC &pc, R (&q)[kIlp],
                                             uint32_t (&cut)[kIlp][S + 1]) {
    constexpr int JS = J1 < S - 2 ? J1 : S - 2;   // cuts found by a search
    static_for<J0 + 1, JS + 1>([&](auto jc) {
        constexpr int j = decltype(jc)::value;
        uint32_t cj[kIlp];
        pc.template search<S - j>(p, q, cj);
#pragma unroll
        for (int u = 0; u < kIlp; ++u) cut[u][j] = cj[u];
    });
    if (J1 == S - 1 && S >= 2) {
#pragma unroll
        for (int u = 0; u < kIlp; ++u) cut[u][S - 1] = p.L - (uint32_t)q[u];
    }
}

// Cuts c_1 .. c_J (J <= S - 1) of kIlp candidates at call positions pos
// (valid positions also for inactive lanes) into cut[u][0 .. J], with
// c_0 = 0 and c_S = L; q is left as decode_range needs it to go on.
// Invalid (rank, assignment) pairs get ok = false.
template <int S, typename R, int H, int J, typename PC>
__device__ __forceinline__ void decode_cuts(const KParams &p, const PC &pc,
                                            const uint32_t (&pos)[kIlp], const bool (&act)[kIlp],
                                            bool (&ok)[kIlp], uint32_t (&asg)[kIlp], R (&q)[kIlp],
                                            uint32_t (&cut)[kIlp][S + 1]) {
#pragma unroll
    for (int u = 0; u < kIlp; ++u) {
        ok[u] = candidate<R>(p, pos[u], q[u], asg[u]) && act[u];
        q[u] = decode_start<R>(p, q[u]);
        cut[u][0] = 0;
        cut[u][S] = p.L;
    }
    decode_range<S, R, H, 0, J>(p, pc, q, cut);
}

template <int S, typename R, int H, typename PC>
__device__ __forceinline__ void decode_batch(const KParams &p, const PC &pc, uint32_t base,
                                             uint32_t stride, bool &bad) {
    constexpr int NW = Codes<S>::kWords;
    bool act[kIlp], ok[kIlp];
    uint32_t asg[kIlp], w[kIlp][NW];
    decode_ilp<S, R, H>(p, pc, base, stride, act, ok, asg, w);
#pragma unroll
    for (int u = 0; u < kIlp; ++u) {
        const uint32_t i = base + u * stride;
        bad |= act[u] && !ok[u];
        if (act[u]) {
#pragma unroll
            for (int k = 0; k < NW; ++k) p.codes[k * (uint32_t)p.ccap + i] = w[u][k];
        }
    }
}

// Columns C0 .. C1 of the Pascal table into LDS (layout of
// Pascal<S, R, H, C0, C1>): 2^H rows each, then the padding rows of the
// type's largest value (so that the columns stay sorted), then the host's
// bucket tables of those columns.  Narrow columns saturate at 2^32 - 1 (no
// value of a column below 5 reaches it for n <= 255).
template <int S, typename R, int H, int C0 = 2, int C1 = S - 1>
__device__ __forceinline__ void pascal_tables(const KParams &p, void *lds) {
    using PC = Pascal<S, R, H, C0, C1>;
    constexpr uint32_t NH = PC::NH, NP = PC::NP, NC = C1 >= C0 ? (uint32_t)(C1 - C0 + 1) : 0u;
    unsigned char *b = reinterpret_cast<unsigned char *>(lds);
    R *ws = reinterpret_cast<R *>(b);
    uint32_t *ns = reinterpret_cast<uint32_t *>(b + PC::kWideBytes);
    const R *gb = reinterpret_cast<const R *>(p.binom);
    for (uint32_t e = threadIdx.x; e < NC * NP; e += kBlock) {
        const uint32_t k = C0 + e / NP, i = e % NP;
        const R v = i < NH ? gb[k * kNB + i] : ~(R)0;
        if ((int)k >= PC::NN) ws[(k - PC::WL) * NP + i] = v;
        else ns[(k - C0) * NP + i] = v > (R)0xFFFFFFFFu ? 0xFFFFFFFFu : (uint32_t)v;
    }
    const uint4 *gt = reinterpret_cast<const uint4 *>(p.btab + (size_t)C0 * kBucketTab);
    uint4 *lt = reinterpret_cast<uint4 *>(b + PC::kWideBytes + PC::kNarrowBytes);
    for (uint32_t e = threadIdx.x; e < NC * (kBucketTab / 16); e += kBlock) lt[e] = gt[e];
}

// LDS bytes of Pascal columns C0 .. C1 with their bucket tables
template <int S, typename R, int C0 = 2, int C1 = S - 1>
__host__ __device__ constexpr size_t pascal_bytes(uint32_t L) {
    switch (decode_levels(L)) {
    case 8: return Pascal<S, R, 8, C0, C1>::bytes();
    case 7: return Pascal<S, R, 7, C0, C1>::bytes();
    case 6: return Pascal<S, R, 6, C0, C1>::bytes();
    default: return Pascal<S, R, 5, C0, C1>::bytes();
    }
}

// Range mode with one assignment: candidate i of the chunk is composition
// rank first + first_i + i, so consecutive candidates are consecutive
// ranks.  A lane takes kIlp consecutive candidates: it unranks the first
// (one search per cut) and steps to the others by the lexicographic
// successor, in which the last cut that can still grow (cut j may reach
// L - S + j) grows by one and the cuts after it follow it at distance 1.
// The lane's kIlp code words of one word index are contiguous: one 16-byte
// store (the code rows hold a multiple of 4 words).
template <int S>
__device__ __forceinline__ void next_cuts(uint32_t L, uint32_t (&c)[S + 1]) {
    // js = the last cut that can grow, b = c_js + 1 - js (no register index
    // is dynamic: both are selected in the scan)
    uint32_t js = 0, b = 1;
#pragma unroll
    for (int j = 1; j <= S - 1; ++j) {
        const bool grow = c[j] < L - S + j;
        js = grow ? (uint32_t)j : js;
        b = grow ? c[j] + 1 - j : b;
    }
#pragma unroll
    for (int m = 1; m <= S - 1; ++m) c[m] = (uint32_t)m < js ? c[m] : b + m;
}

template <int S, typename R, int H, typename PC>
__device__ __forceinline__ void decode_succ(const KParams &p, const PC &pc, uint32_t base, bool &bad) {
    static_assert(kIlp == 4, "one 16-byte store per code word");
    constexpr int NW = Codes<S>::kWords;
    const uint64_t rank0 = p.first + (uint32_t)p.first_i + base;
    R q[1] = {decode_start<R>(p, (R)(rank0 < p.n_comp ? rank0 : 0))};
    uint32_t c[S + 1];
    c[0] = 0;
    c[S] = p.L;
    static_for<1, S - 1>([&](auto jc) {
        constexpr int j = decltype(jc)::value;
        uint32_t cj[1];
        pc.template search<S - j>(p, q, cj);
        c[j] = cj[0];
    });
    if (S >= 2) c[S - 1] = p.L - (uint32_t)q[0];
    uint32_t w[kIlp][NW];
#pragma unroll
    for (int u = 0; u < kIlp; ++u) {
        if (u > 0) next_cuts<S>(p.L, c);
        const bool act = base + u < (uint32_t)p.n_i;
        const bool ok = rank0 + u < p.n_comp;
        bad |= act && !ok;
        pack_cuts<S>(c, ok, w[u]);
    }
    const uint32_t ccap = (uint32_t)p.ccap;
#pragma unroll
    for (int k = 0; k < NW; ++k)
        *reinterpret_cast<uint4 *>(p.codes + k * ccap + base) = make_uint4(w[0][k], w[1][k], w[2][k], w[3][k]);
}

template <int S, typename R, int H>
__device__ __forceinline__ void decode_all(const KParams &p, void *lds, bool &bad) {
    pascal_tables<S, R, H>(p, lds);
    __syncthreads();
    const Pascal<S, R, H> pc(lds);
    if (!p.comp_rank && p.A == 1) {
        const uint32_t stride = gridDim.x * kBlock * kIlp, n_i = (uint32_t)p.n_i;
        for (uint32_t base = (blockIdx.x * kBlock + threadIdx.x) * kIlp; base < n_i; base += stride)
            decode_succ<S, R, H>(p, pc, base, bad);
        return;
    }
    // 32-bit positions: a chunk holds at most 2^26 candidates, a call fewer than 2^32
    const uint32_t stride = gridDim.x * kBlock, n_i = (uint32_t)p.n_i;
    for (uint32_t base = blockIdx.x * kBlock + threadIdx.x; base < n_i; base += kIlp * stride)
        decode_batch<S, R, H>(p, pc, base, stride, bad);
}

template <int S, typename R>
__global__ __launch_bounds__(kBlock) void decode_kernel(KParams p) {
    extern __shared__ __align__(16) unsigned char smem[];
    R *lds = reinterpret_cast<R *>(smem);
    bool bad = false;
    switch (decode_levels(p.L)) {
    case 8: decode_all<S, R, 8>(p, lds, bad); break;
    case 7: decode_all<S, R, 7>(p, lds, bad); break;
    case 6: decode_all<S, R, 6>(p, lds, bad); break;
    default: decode_all<S, R, 5>(p, lds, bad); break;
    }
    if (bad) atomicOr(p.err, 1u);
}

// (a2)-(a4), (a6) for the chunk: stage weights from the cut codes, memory
// check, the DP and the reduction.  With a cascade (p.nlevels > 0) a lane
// whose steady state has not settled by iteration p.lvl_k[0] is queued for
// resume_kernel instead of finishing here.
template <int S, bool AR>
__global__ __launch_bounds__(kBlock) void eval_kernel(KParams p) {
    extern __shared__ __align__(16) unsigned char smem[];
    const Ent tab = entry_tables(p, smem);
    const Comm<S> comm = load_comm<S>(p);
    constexpr int NW = Codes<S>::kWords;
    unsigned long long best = ~0ull;
    // 32-bit positions: a chunk holds at most 2^26 candidates, a call fewer
    // than 2^32, and the code buffer fewer than 2^32 words (fewer scalar
    // registers than 64-bit ones, which this kernel is short of)
    const uint32_t stride = gridDim.x * kBlock, n_i = (uint32_t)p.n_i, ccap = (uint32_t)p.ccap;
    const uint32_t first_i = (uint32_t)p.first_i;
    // every wave runs the same trip count so that ballots see whole waves
    const uint32_t span = (n_i + stride - 1) / stride;
    const uint32_t nit = p.M >= (uint32_t)S ? p.M - S : 0u;
    __shared__ unsigned int nq;
    if (threadIdx.x == 0) nq = 0;
    __syncthreads();
    uint32_t i = blockIdx.x * kBlock + threadIdx.x;
    for (uint32_t it = 0; it < span; ++it, i += stride) {
        const bool active = i < n_i;
        const uint32_t gi = first_i + i;   // index within the call
        uint32_t w[NW];
#pragma unroll
        for (int k = 0; k < NW; ++k) w[k] = active ? p.codes[k * ccap + i] : 0u;
        uint32_t cut[S + 1], to[S], F[S], B[S], Y[S];
        const bool ok = unpack_cuts<S>(w, p.L, cut);
        const uint32_t a = ok ? assign_of(p, gi) : 0u;
        decode_toff<S>(p, tab, a, to);
        const bool feas = stage_weights<S>(p, tab, cut, to, F, B) && ok && active;
        bool done_here = true;
        uint32_t T;
        if (p.M < (uint32_t)S) {
            dp_table<S>(p, F, B, comm, Y);
            T = end_time<S, AR>(p, tab, Y, comm, w, a);
        } else {
            dp_prologue<S>(Y, F, B, comm, p.g24 != 0);
            const uint32_t k1 = p.nlevels ? p.lvl_k[0] : nit;
            done_here = dp_advance<S>(Y, F, B, comm, 0, k1, nit);
            if (p.nlevels) enqueue<S, S>(p, 0, &nq, !done_here && active && ok, gi, w, -1, Y);
            T = dp_end<S, AR>(p, tab, Y, F, B, comm, w, a);
        }
        if (!ok) T = 0xFFFFFFFFu;
        const bool write = active && (done_here || !ok);
        // outputs are read back only by the host or the argmin pass: stream them past the caches
        if (write && p.makespan_out) __builtin_nontemporal_store(T, p.makespan_out + gi);
        if (p.feas_bits_out) {
            // chunks start at multiples of 64, so a wave covers 64 aligned candidates
            const unsigned long long bits = __ballot(feas);
            const uint32_t w0 = (gi - (threadIdx.x & 63)) >> 5, nwords = (uint32_t)p.nwords;
            if ((threadIdx.x & 63) == 0 && w0 < nwords) __builtin_nontemporal_store((uint32_t)bits, p.feas_bits_out + w0);
            if ((threadIdx.x & 63) == 32 && w0 + 1 < nwords) __builtin_nontemporal_store((uint32_t)(bits >> 32), p.feas_bits_out + w0 + 1);
        }
        if (write) {
            const unsigned long long key = make_key(feas, T, gi);
            best = key < best ? key : best;
        }
    }
    if (p.nlevels) {
        __syncthreads();
        if (threadIdx.x == 0) p.qcount[blockIdx.x] = nq;   // entries for level 1
    }
    block_min_and_finish(best, p.acc, p.done, p.result, nullptr, p.nlevels == 0, p.accumulate);
}

// Schedules other than 1F1B: the same pass as eval_kernel with the
// schedule-table DP (TAB) or the Eager 1F1B closed form, whose steady part
// takes the same cascade (queue entries carry 2S state words).  Held to 128
// VGPRs (4 waves per SIMD instead of 3 at S = 16, with a few words spilled
// to scratch outside the steady loop): 2 % faster on the 16-stage workload.
template <int S, bool AR, bool TAB>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(4, 8))) void sched_kernel(KParams p) {
    extern __shared__ __align__(16) unsigned char smem[];
    const Ent tab = entry_tables(p, smem);
    const Comm<S> comm = load_comm<S>(p);
    constexpr int NW = Codes<S>::kWords;
    unsigned long long best = ~0ull;
    // 32-bit positions, as in eval_kernel
    const uint32_t stride = gridDim.x * kBlock, n_i = (uint32_t)p.n_i, ccap = (uint32_t)p.ccap;
    const uint32_t first_i = (uint32_t)p.first_i;
    const uint32_t span = (n_i + stride - 1) / stride;
    const uint32_t npairs = TAB ? 0u : p.M - 2 * S + 1;
    __shared__ unsigned int nq;
    if (threadIdx.x == 0) nq = 0;
    __syncthreads();
    uint32_t i = blockIdx.x * kBlock + threadIdx.x;
    for (uint32_t it = 0; it < span; ++it, i += stride) {
        const bool active = i < n_i;
        const uint32_t gi = first_i + i;
        uint32_t w[NW];
#pragma unroll
        for (int k = 0; k < NW; ++k) w[k] = active ? p.codes[k * ccap + i] : 0u;
        uint32_t cut[S + 1], to[S], F[S], B[S], Y[S];
        const bool ok = unpack_cuts<S>(w, p.L, cut);
        const uint32_t a = ok ? assign_of(p, gi) : 0u;
        decode_toff<S>(p, tab, a, to);
        const bool feas = stage_weights<S>(p, tab, cut, to, F, B) && ok && active;
        bool done_here = true;
        if (TAB) {
            dp_sched<S>(p, F, B, comm, Y);
        } else {
            uint32_t Fn[S], Fp[S];
            eager_prologue<S>(Y, Fn, Fp, F, B, comm);
            const uint32_t k1 = p.nlevels ? p.lvl_k[0] : npairs;
            done_here = eager_advance<S>(Y, Fn, Fp, F, B, comm, 0, k1, npairs);
            if (p.nlevels) {
                uint32_t X[2 * S];
                eager_pack<S>(Y, Fn, Fp, X);
                enqueue<S, 2 * S>(p, 0, &nq, !done_here && active && ok, gi, w, -1, X);
            }
            eager_epilogue<S>(Y, Fn, Fp, F, B, comm);
        }
        uint32_t T = end_time<S, AR>(p, tab, Y, comm, w, a);
        if (!ok) T = 0xFFFFFFFFu;
        const bool write = active && (done_here || !ok);
        // outputs are read back only by the host or the argmin pass: stream them past the caches
        if (write && p.makespan_out) __builtin_nontemporal_store(T, p.makespan_out + gi);
        if (p.feas_bits_out) {
            const unsigned long long bits = __ballot(feas);
            const uint32_t w0 = (gi - (threadIdx.x & 63)) >> 5, nwords = (uint32_t)p.nwords;
            if ((threadIdx.x & 63) == 0 && w0 < nwords) __builtin_nontemporal_store((uint32_t)bits, p.feas_bits_out + w0);
            if ((threadIdx.x & 63) == 32 && w0 + 1 < nwords) __builtin_nontemporal_store((uint32_t)(bits >> 32), p.feas_bits_out + w0 + 1);
        }
        if (write) {
            const unsigned long long key = make_key(feas, T, gi);
            best = key < best ? key : best;
        }
    }
    if (!TAB && p.nlevels) {
        __syncthreads();
        if (threadIdx.x == 0) p.qcount[blockIdx.x] = nq;
    }
    block_min_and_finish(best, p.acc, p.done, p.result, nullptr, TAB || p.nlevels == 0, p.accumulate);
}

// Level `lvl` of the cascade: resume the queued lanes from steady
// iteration p.lvl_k[lvl-1] to p.lvl_k[lvl] (the end at the last level).
// SCH: Eager 1F1B (2S state words per entry, steady pairs), else 1F1B.
template <int S, bool AR, bool SCH>
__global__ __launch_bounds__(kBlock) void resume_kernel(KParams p, uint32_t lvl) {
    extern __shared__ __align__(16) unsigned char smem[];
    const Ent tab = entry_tables(p, smem);
    const Comm<S> comm = load_comm<S>(p);
    constexpr int NW = Codes<S>::kWords;
    constexpr int NX = SCH ? 2 * S : S;
    const uint32_t nit = SCH ? p.M - 2 * S + 1 : p.M - S;
    const uint32_t k0 = p.lvl_k[lvl - 1];
    const uint32_t k1 = lvl < p.nlevels ? p.lvl_k[lvl] : nit;
    // this block's segment of the queue written by level lvl - 1
    const uint32_t n = __hip_atomic_load(&p.qcount[(uint64_t)(lvl - 1) * p.nseg + blockIdx.x], __ATOMIC_RELAXED,
                                         __HIP_MEMORY_SCOPE_AGENT);
    const QueueView<S> qin(p, (lvl - 1) & 1);
    __shared__ unsigned int nq;
    if (threadIdx.x == 0) nq = 0;
    __syncthreads();
    unsigned long long best = ~0ull;
    const uint32_t span = (n + kBlock - 1) / kBlock;
    // 32-bit word offsets: a queue holds fewer than 2^32 words
    const uint32_t seg = blockIdx.x * (uint32_t)p.seg_cap, qcap = (uint32_t)p.qcap;
    for (uint32_t it = 0; it < span; ++it) {
        const uint32_t q = seg + it * kBlock + threadIdx.x;
        const bool active = it * kBlock + threadIdx.x < n;
        const uint32_t i = active ? qin.idx[q] : 0u;
        uint32_t w[NW], cut[S + 1], to[S], F[S], B[S], X[NX], Y[S];
#pragma unroll
        for (int k = 0; k < NW; ++k) w[k] = active ? qin.codes[k * qcap + q] : 0u;
#pragma unroll
        for (int s = 0; s < NX; ++s) X[s] = active ? qin.Y[s * qcap + q] : 0u;
        unpack_cuts<S>(w, p.L, cut);   // (a queued entry's codes were valid when it was queued)
        const uint32_t a = !active ? 0u : p.qasg ? qin.asg[q] : assign_of(p, i);
        decode_toff<S>(p, tab, a, to);
        const bool feas = stage_weights<S>(p, tab, cut, to, F, B);
        bool settled;
        uint32_t T;
        if constexpr (SCH) {
            uint32_t Fn[S], Fp[S];
            eager_unpack<S>(X, Y, Fn, Fp);
            settled = eager_advance<S>(Y, Fn, Fp, F, B, comm, k0, k1, nit);
            if (lvl < p.nlevels) {
                eager_pack<S>(Y, Fn, Fp, X);
                enqueue<S, NX>(p, lvl & 1, &nq, active && !settled, i, w, a, X);
            }
            eager_epilogue<S>(Y, Fn, Fp, F, B, comm);
            T = end_time<S, AR>(p, tab, Y, comm, w, a);
        } else {
#pragma unroll
            for (int s = 0; s < S; ++s) Y[s] = X[s];
            settled = dp_advance<S>(Y, F, B, comm, k0, k1, nit);
            if (lvl < p.nlevels) enqueue<S, S>(p, lvl & 1, &nq, active && !settled, i, w, a, Y);
            T = dp_end<S, AR>(p, tab, Y, F, B, comm, w, a);
        }
        if (active && settled) {
            // scattered one-word writes: the nontemporal hint keeps them out of L2 write-allocate
            if (p.makespan_out) __builtin_nontemporal_store(T, p.makespan_out + i);
            const unsigned long long key = make_key(feas, T, i);
            best = key < best ? key : best;
        }
    }
    if (lvl < p.nlevels) {
        __syncthreads();
        if (threadIdx.x == 0) p.qcount[(uint64_t)lvl * p.nseg + blockIdx.x] = nq;
    }
    block_min_and_finish(best, p.acc, p.done, p.result, nullptr, lvl == p.nlevels, p.accumulate);
}

// Early stop (Eq. 2 / Theorem 1) over one piece of a chunk.  Against the
// bound b in force (min of the caller's bound and the best of the earlier
// chunks, fixed within a chunk) every candidate is classified by classify()
// over its stages in pipeline order; the ones no stage discards survive
// and are evaluated exactly.
//
// filter_kernel runs in one of three modes:
//  kFilterFull   decodes every cut (a1), builds the stage weights (a2) and
//                decides all S stages while the cuts are in registers; the
//                survivors go to a list (call position + cut codes), block b
//                filling segment b of seg_cap entries, counted in LDS (no
//                global atomic, whose single address would serialise waves);
//  kFilterPrefix decodes only the first X = filter_prefix<S>() cuts and
//                decides the stages they close; the candidates it keeps go
//                to a list in the same segments (counts in acount) with
//                what the decode needs to go on (AList);
//  kFilterGather takes block b's segment of that list in order (coalesced),
//                decodes the remaining cuts and goes on as kFilterFull.
// For S >= 4 a piece goes through kFilterPrefix, then kFilterGather: most
// candidates are discarded at one of their first stages, and only the rest
// pay for the searches of their later cuts.  surv_kernel evaluates the
// survivor list on the DAG (a3) and folds it into the running best (a4).
enum FilterMode { kFilterFull = 0, kFilterPrefix = 1, kFilterGather = 2 };
template <int S>
__host__ __device__ constexpr int filter_prefix() { return S >= 4 ? S / 2 : 0; }
// Pascal columns a mode searches: the prefix mode cuts 1 .. X (columns
// S-X .. S-1), the gather mode the cuts after them (columns 2 .. S-X-1), the
// full mode every cut (columns 2 .. S-1)
template <int S, int MODE>
__host__ __device__ constexpr int filter_col_lo() { return MODE == kFilterPrefix ? S - filter_prefix<S>() : 2; }
template <int S, int MODE>
__host__ __device__ constexpr int filter_col_hi() { return MODE == kFilterGather ? S - filter_prefix<S>() - 1 : S - 1; }

// The prefix list, arrays of ccap entries: call position, decode state q
// after the first X cuts (low and high words), assignment index, then the
// first X cuts as cut codes.
static_assert(4 + (filter_prefix<kSMax>() + 3) / 4 <= kAListWords, "first-stage list entry too small");
struct AList {
    uint32_t *pos, *rlo, *rhi, *asg, *w;
    __device__ __forceinline__ explicit AList(const KParams &p)
        : pos(p.alist), rlo(p.alist + p.ccap), rhi(p.alist + 2 * p.ccap), asg(p.alist + 3 * p.ccap),
          w(p.alist + 4 * p.ccap) {}
};

// Stage-1 screen of the prefix mode.  Stage 1 = [0, c_1) on type t fits its
// memory iff c_1 <= hm_t(0), and g(S_1) = M (F_1 + B_1) + d_1 only grows
// with c_1, so it passes Eq. 2 iff c_1 <= hb_t, the largest end point with
// g(S_1) <= b.  Ranks are lexicographic with c_1 the most significant cut,
// so the compositions with c_1 <= h hold the ranks below
//   N(h) = C(L-1, S-1) - C(L-1-h, S-1)
// (the others have all S-1 cuts in h+1 .. L-1).  A candidate therefore
// fails stage 1 iff its rank is at least N(min(hm_t, hb_t)), and fails it on
// memory (tested first at a stage) iff its rank is at least N(hm_t): one
// compare decides it before any cut is decoded.  thr[2t], thr[2t+1] = those
// two limits for every type t (threads t < T; the caller's barrier
// publishes them).
template <int S, typename R>
__device__ __forceinline__ void stage1_limits(const KParams &p, const Ent &tab, uint32_t b, unsigned long long *thr) {
    if (threadIdx.x >= p.T) return;
    const uint32_t to = threadIdx.x * p.erow, L = p.L, hmax = L - S + 1;   // hmax: the largest c_1
    const uint32_t pf0 = ent<kEPf>(tab, 0, to), pb0 = ent<kEPb>(tab, 0, to);
    const uint32_t pd0 = p.has_ar ? ent<kEPd>(tab, 0, to) : 0u;
    // g(S_1) is nondecreasing in c_1: the largest passing end point by halving
    // steps (hb = 0: none passes; every c_1 is at least 1)
    uint32_t hb = 0;
    for (uint32_t st = 128; st; st >>= 1) {
        const uint32_t c = hb + st;
        if (c <= hmax) {
            const uint32_t F = ent<kEPf>(tab, c, to) - pf0, B = ent<kEPb>(tab, c, to) - pb0;
            const uint32_t D = p.has_ar ? ent<kEPd>(tab, c, to) - pd0 : 0u;
            // M (F + B) + d_1 is an Eq. 2 value, below 2^31 like every path weight
            if (p.M * (F + B) + D <= b) hb = c;
        }
    }
    const uint32_t hm = min(ent<kEHm>(tab, 0, to), hmax), h1 = min(hb, hm);
    const R *bin = reinterpret_cast<const R *>(p.binom);
    thr[2 * threadIdx.x] = p.n_comp - (uint64_t)bin[(S - 1) * kNB + (L - 1 - h1)];
    thr[2 * threadIdx.x + 1] = p.n_comp - (uint64_t)bin[(S - 1) * kNB + (L - 1 - hm)];
}

// Type of stage 1 of assignment a (valid a).
template <int S>
__device__ __forceinline__ uint32_t first_stage_type(const KParams &p, uint32_t a) {
    if (p.assign_mode == kAssignFixed) return p.fixed_types[0];
    if (p.assign_mode == kAssignTable) return p.assign[(uint64_t)a * S];
    // the top base-T digit: floor(a / T^(S-1)), from a multiply-high that
    // gives it or one more
    uint32_t q = __umulhi(a, p.s1_magic);
    if ((uint64_t)q * p.s1_div > a) q -= 1;
    return q;
}

// LDS words that lanes of one wave wrote are visible to the wave's other
// lanes after this (their writes complete; no code moves across it).
__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Buffered positions of one wave in the screened prefix mode: fewer than one
// batch of kIlp * 64 before a screened tile of as many adds to it.
constexpr uint32_t kScreenBuf = 2 * kIlp * 64;
// The screen costs a second load of every kept candidate and the buffer's
// bookkeeping, and saves the prefix work of the ones it discards.  It pays
// when that work is large: five or more prefix cuts (S >= 10), or stage
// tests with all-reduce terms (measured: 8 % faster at 16 stages, 6 % at 8
// stages with all-reduce times, 3.5 % slower at 8 stages without).
template <int S, bool AR, int MODE>
__host__ __device__ constexpr bool filter_screens() {
    return MODE == kFilterPrefix && (filter_prefix<S>() >= 5 || AR);
}
template <int S, bool AR, int MODE>
__host__ __device__ constexpr size_t filter_static_lds() {
    return filter_screens<S, AR, MODE>() ? (size_t)kScreenBuf * 4 * (kBlock / 64) + 16 * kTypesMax : 0;
}

// The tests of kIlp decoded candidates of one lane (cuts 1 .. X of
// filter_all's mode in cut[u]): classification, counts, and the list entry
// of each candidate kept (the prefix list, or the survivor list).
template <int S, typename R, bool AR, int MODE>
__device__ __forceinline__ void filter_emit(const KParams &p, const Ent &tab, uint32_t b, unsigned int *nq,
                                            const bool (&act)[kIlp], const bool (&ok)[kIlp],
                                            const uint32_t (&pos)[kIlp], const uint32_t (&asg)[kIlp],
                                            const R (&r)[kIlp], const uint32_t (&cut)[kIlp][S + 1],
                                            uint32_t &n_keep, uint32_t &n_pruned, uint32_t &n_infeas, bool &bad) {
    constexpr int X0 = filter_prefix<S>();
    constexpr int X = MODE == kFilterPrefix ? X0 : S;   // stages decided, cuts 1 .. X decoded
    constexpr int NW = Codes<S>::kWords;
    constexpr int AW = (X0 + 3) / 4;                    // code words of the prefix cuts
    const AList al(p);
    const unsigned int lane = threadIdx.x & 63;
    const uint32_t seg = blockIdx.x * (uint32_t)p.seg_cap, ccap = (uint32_t)p.ccap;
#pragma unroll
    for (int u = 0; u < kIlp; ++u) {
        uint32_t to[S];
        decode_toff<S>(p, tab, ok[u] ? asg[u] : 0u, to);
        const uint32_t cls = classify<S, AR, X>(p, tab, cut[u], to, b);
        bool keep = false;
        if (act[u]) {
            if (!ok[u]) bad = true;
            else if (cls == 1) ++n_infeas;
            else if (cls == 2) ++n_pruned;
            else keep = true;
        }
        const unsigned long long m = __ballot(keep);
        if (m) {
            unsigned int slot0 = 0;
            if (lane == 0) slot0 = atomicAdd(nq, (unsigned int)__popcll(m));
            slot0 = __shfl(slot0, 0, 64);
            if (keep) {
                const unsigned long long below = lane ? (m & ((1ull << lane) - 1ull)) : 0ull;
                const uint32_t o = seg + slot0 + (uint32_t)__popcll(below);
                if constexpr (MODE == kFilterPrefix) {
                    uint32_t w[AW];
#pragma unroll
                    for (int k = 0; k < AW; ++k) w[k] = 0;
#pragma unroll
                    for (int j = 1; j <= X0; ++j) w[(j - 1) / 4] |= cut[u][j] << (8 * ((j - 1) % 4));
                    al.pos[o] = pos[u];
                    al.asg[o] = asg[u];
                    al.rlo[o] = (uint32_t)r[u];
                    if (sizeof(R) == 8) al.rhi[o] = (uint32_t)((uint64_t)r[u] >> 32);
#pragma unroll
                    for (int k = 0; k < AW; ++k) al.w[k * ccap + o] = w[k];
                } else {
                    uint32_t w[NW];
                    pack_cuts<S>(cut[u], true, w);
                    p.sidx[o] = pos[u];
#pragma unroll
                    for (int k = 0; k < NW; ++k) p.codes[k * ccap + o] = w[k];
                }
            }
            if (MODE != kFilterPrefix) n_keep += lane == 0 ? (uint32_t)__popcll(m) : 0u;
        }
    }
}

// Prefix mode: each wave screens tiles of kIlp * 64 consecutive candidates
// of the piece (its stream: tiles gw, gw + nwave, ...) on stage 1 alone
// (stage1_limits), keeps the positions of the rest in its LDS buffer buf,
// and decodes and tests them kIlp * 64 at a time, so that the searches of
// the first cuts run only for candidates that pass stage 1 (about two in
// three on the workloads here) and every lane has a candidate to decode.
template <int S, typename R, int H, bool AR, typename PC>
__device__ __forceinline__ void filter_screened(const KParams &p, const PC &pc, const Ent &tab,
                                                uint32_t b, unsigned int *nq, uint32_t *buf,
                                                const unsigned long long *thr, uint32_t &n_keep,
                                                uint32_t &n_pruned, uint32_t &n_infeas, bool &bad) {
    constexpr int X0 = filter_prefix<S>();
    constexpr uint32_t kTile = kIlp * 64;
    const unsigned int lane = threadIdx.x & 63;
    const unsigned long long below = lane ? (~0ull >> (64 - lane)) : 0ull;
    // 32-bit positions: a piece holds at most 2^26 candidates, a call fewer than 2^32
    const uint32_t n = (uint32_t)p.n_i, first_i = (uint32_t)p.first_i;
    const uint32_t nwave = gridDim.x * (kBlock / 64);
    uint32_t tile = blockIdx.x * (kBlock / 64) + (threadIdx.x >> 6);   // next tile of the stream
    uint32_t cnt = 0;                                                  // positions in buf
    for (;;) {
        // screen tiles until a batch is buffered or the stream ends
        while (cnt < kTile && tile * kTile < n) {
            const uint32_t t0 = tile * kTile;
            tile += nwave;
            bool keep[kIlp];
#pragma unroll
            for (int u = 0; u < kIlp; ++u) {
                const uint32_t i = t0 + (uint32_t)u * 64 + lane;
                keep[u] = false;
                if (i < n) {
                    R r;
                    uint32_t a;
                    if (!candidate<R>(p, first_i + i, r, a)) {
                        keep[u] = true;   // out of range: the batch raises the error flag
                    } else {
                        const uint32_t t = first_stage_type<S>(p, a);
                        const uint64_t rk = (uint64_t)r;
                        if (rk < thr[2 * t]) keep[u] = true;
                        else if (rk >= thr[2 * t + 1]) ++n_infeas;
                        else ++n_pruned;
                    }
                }
            }
#pragma unroll
            for (int u = 0; u < kIlp; ++u) {
                const unsigned long long m = __ballot(keep[u]);
                if (keep[u]) buf[cnt + (uint32_t)__popcll(m & below)] = t0 + (uint32_t)u * 64 + lane;
                cnt += (uint32_t)__popcll(m);
            }
        }
        if (cnt == 0) break;
        wave_lds_sync();
        const uint32_t nb = cnt < kTile ? cnt : kTile;
        bool act[kIlp], ok[kIlp];
        uint32_t pos[kIlp], asg[kIlp], cut[kIlp][S + 1];
        R r[kIlp];
#pragma unroll
        for (int u = 0; u < kIlp; ++u) {
            const uint32_t j = (uint32_t)u * 64 + lane;
            act[u] = j < nb;
            pos[u] = first_i + (act[u] ? buf[j] : 0u);   // (position 0 of the piece for idle lanes)
        }
        decode_cuts<S, R, H, X0>(p, pc, pos, act, ok, asg, r, cut);
        filter_emit<S, R, AR, kFilterPrefix>(p, tab, b, nq, act, ok, pos, asg, r, cut, n_keep, n_pruned, n_infeas, bad);
        // the positions past the batch (fewer than kTile) move to the front
        if (cnt > kTile) {
            uint32_t v[kIlp];
#pragma unroll
            for (int u = 0; u < kIlp; ++u) {
                const uint32_t j = kTile + (uint32_t)u * 64 + lane;
                v[u] = j < cnt ? buf[j] : 0u;
            }
            wave_lds_sync();
#pragma unroll
            for (int u = 0; u < kIlp; ++u) {
                const uint32_t j = (uint32_t)u * 64 + lane;
                if (kTile + j < cnt) buf[j] = v[u];
            }
        }
        cnt -= nb;
        wave_lds_sync();
    }
}

template <int S, typename R, int H, bool AR, int MODE>
__device__ __forceinline__ void filter_all(const KParams &p, const R *pas, const Ent &tab, uint32_t b,
                                           unsigned int *nq, uint32_t *buf, const unsigned long long *thr,
                                           uint32_t &n_keep, uint32_t &n_pruned, uint32_t &n_infeas, bool &bad) {
    constexpr int X0 = filter_prefix<S>();
    constexpr int NW = Codes<S>::kWords;
    constexpr int AW = (X0 + 3) / 4;                    // code words of the prefix cuts
    const Pascal<S, R, H, filter_col_lo<S, MODE>(), filter_col_hi<S, MODE>()> pc(pas);
    if constexpr (filter_screens<S, AR, MODE>()) {
        filter_screened<S, R, H, AR>(p, pc, tab, b, nq, buf, thr, n_keep, n_pruned, n_infeas, bad);
        return;
    }
    const AList al(p);
    // 32-bit positions and word offsets: a piece holds at most 2^26
    // candidates, a call fewer than 2^32, and each list fewer than 2^32
    // words (fewer scalar registers than 64-bit ones)
    const uint32_t seg = blockIdx.x * (uint32_t)p.seg_cap, ccap = (uint32_t)p.ccap;
    const uint32_t first_i = (uint32_t)p.first_i;
    // full, prefix: the piece, kIlp candidates a lane, strided over the grid;
    // gather: this block's segment of the list, strided over the block
    const uint32_t n = MODE == kFilterGather ? p.acount[blockIdx.x] : (uint32_t)p.n_i;
    const uint32_t stride = MODE == kFilterGather ? (uint32_t)kBlock : gridDim.x * kBlock;
    const uint32_t start = MODE == kFilterGather ? threadIdx.x : blockIdx.x * kBlock + threadIdx.x;
    for (uint32_t base = start; base < n; base += kIlp * stride) {
        bool act[kIlp], ok[kIlp];
        uint32_t pos[kIlp];
        uint32_t asg[kIlp], cut[kIlp][S + 1];
        R r[kIlp];
        if constexpr (MODE == kFilterGather) {
#pragma unroll
            for (int u = 0; u < kIlp; ++u) {
                const uint32_t i = base + u * stride;
                act[u] = i < n;
                ok[u] = act[u];
                const uint32_t o = seg + (act[u] ? i : 0);
                pos[u] = al.pos[o];
                asg[u] = al.asg[o];
                r[u] = sizeof(R) == 8 ? (R)(((uint64_t)al.rhi[o] << 32) | al.rlo[o]) : (R)al.rlo[o];
                uint32_t w[NW];
#pragma unroll
                for (int k = 0; k < NW; ++k) w[k] = k < AW ? al.w[k * ccap + o] : 0u;
                cut[u][0] = 0;
                cut[u][S] = p.L;
#pragma unroll
                for (int j = 1; j <= X0; ++j) cut[u][j] = (w[(j - 1) / 4] >> (8 * ((j - 1) % 4))) & 0xFFu;
            }
            decode_range<S, R, H, X0, S - 1>(p, pc, r, cut);
        } else {
#pragma unroll
            for (int u = 0; u < kIlp; ++u) {
                const uint32_t i = base + u * stride;
                act[u] = i < n;
                pos[u] = first_i + (act[u] ? i : 0u);
            }
            decode_cuts<S, R, H, MODE == kFilterPrefix ? X0 : S - 1>(p, pc, pos, act, ok, asg, r, cut);
        }
        filter_emit<S, R, AR, MODE>(p, tab, b, nq, act, ok, pos, asg, r, cut, n_keep, n_pruned, n_infeas, bad);
    }
}

// GTAB: the stage entries are read from global memory (L2) instead of LDS,
// when they and the Pascal columns together exceed the 64 KB of LDS one
// block may use (the largest columns: L > 128 with 64-bit ranks).  LDS:
// the stage entries first (unless GTAB), then the Pascal columns.
template <int S, typename R, bool AR, bool GTAB, int MODE>
__global__ __launch_bounds__(kBlock) void filter_kernel(KParams p) {
    extern __shared__ __align__(16) unsigned char smem[];
    const uint32_t H = decode_levels(p.L);
    Ent tab;
    R *pas;
    if constexpr (GTAB) {
        tab = entry_global(p);
        pas = reinterpret_cast<R *>(smem);
    } else {
        pas = reinterpret_cast<R *>(smem + p.ent_lds);
        tab = entry_tables(p, smem);
    }
    // bound in force: min(caller's bound, best of the chunks before this one)
    const unsigned long long rb = __hip_atomic_load(p.snap, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const uint32_t rbT = (uint32_t)(rb >> 32);
    const uint32_t b = rbT < p.es_bound ? rbT : p.es_bound;
    uint32_t n_keep = 0, n_pruned = 0, n_infeas = 0;
    bool bad = false;
    __shared__ unsigned int nq;
    if (threadIdx.x == 0) nq = 0;
    // prefix mode: the waves' position buffers and the stage-1 rank limits
    // (published by the barrier after the Pascal columns)
    uint32_t *buf = nullptr;
    const unsigned long long *thr = nullptr;
    if constexpr (filter_screens<S, AR, MODE>()) {
        __shared__ uint32_t screen_buf[kScreenBuf * (kBlock / 64)];
        __shared__ unsigned long long screen_thr[2 * kTypesMax];
        stage1_limits<S, R>(p, tab, b, screen_thr);
        buf = screen_buf + (threadIdx.x >> 6) * kScreenBuf;
        thr = screen_thr;
    }
    switch (H) {
    case 8: pascal_tables<S, R, 8, filter_col_lo<S, MODE>(), filter_col_hi<S, MODE>()>(p, pas); __syncthreads(); filter_all<S, R, 8, AR, MODE>(p, pas, tab, b, &nq, buf, thr, n_keep, n_pruned, n_infeas, bad); break;
    case 7: pascal_tables<S, R, 7, filter_col_lo<S, MODE>(), filter_col_hi<S, MODE>()>(p, pas); __syncthreads(); filter_all<S, R, 7, AR, MODE>(p, pas, tab, b, &nq, buf, thr, n_keep, n_pruned, n_infeas, bad); break;
    case 6: pascal_tables<S, R, 6, filter_col_lo<S, MODE>(), filter_col_hi<S, MODE>()>(p, pas); __syncthreads(); filter_all<S, R, 6, AR, MODE>(p, pas, tab, b, &nq, buf, thr, n_keep, n_pruned, n_infeas, bad); break;
    default: pascal_tables<S, R, 5, filter_col_lo<S, MODE>(), filter_col_hi<S, MODE>()>(p, pas); __syncthreads(); filter_all<S, R, 5, AR, MODE>(p, pas, tab, b, &nq, buf, thr, n_keep, n_pruned, n_infeas, bad); break;
    }
    // per-block sums, one global atomic per counter and block
    const unsigned long long sk = wave_sum_u32(n_keep), sp = wave_sum_u32(n_pruned), si = wave_sum_u32(n_infeas);
    __shared__ unsigned long long cnt[3];
    if (threadIdx.x < 3) cnt[threadIdx.x] = 0;
    __syncthreads();
    if ((threadIdx.x & 63) == 0) {
        if (sk) atomicAdd(&cnt[0], sk);
        if (sp) atomicAdd(&cnt[1], sp);
        if (si) atomicAdd(&cnt[2], si);
    }
    __syncthreads();
    if (threadIdx.x < 3 && cnt[threadIdx.x]) atomicAdd(&p.stats[threadIdx.x], cnt[threadIdx.x]);
    // (after the barrier above: every wave has added)
    if (threadIdx.x == 0) (MODE == kFilterPrefix ? p.acount : p.scount)[blockIdx.x] = nq;
    if (bad) atomicOr(p.err, 1u);
}

// surv_kernel takes the survivor list as one sequence in segment order
// (segment j: scount[j] entries from j seg_cap).  Every block scans the nseg
// segment counts into LDS, after the stage entries; survivor k then goes to
// thread k mod (grid kBlock), found by a binary search of the scan, so the
// DPs of however many survivors spread over the whole grid, 64 to a wave.
// Only the blocks the list needs (one per kBlock survivors, at least one)
// go on: the others leave before loading the entries and take no ticket on
// the done counter.
template <int S, bool AR, bool SCH>
__global__ __launch_bounds__(kBlock) void surv_kernel(KParams p, uint32_t publish, uint32_t nseg) {
    extern __shared__ __align__(16) unsigned char smem[];
    uint32_t *pre = reinterpret_cast<uint32_t *>(smem + p.ent_lds);   // nseg + 1 entries
    // exclusive scan of the segment counts, kPer consecutive segments a thread
    const uint32_t per = (nseg + kBlock - 1) / kBlock, j0 = threadIdx.x * per;
    uint32_t mine = 0;
    for (uint32_t j = j0; j < j0 + per && j < nseg; ++j)
        mine += __hip_atomic_load(&p.scount[j], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    unsigned long long total;
    uint32_t run = (uint32_t)block_exclusive_scan_u64(mine, total);
    for (uint32_t j = j0; j < j0 + per && j < nseg; ++j) {
        pre[j] = run;
        run += __hip_atomic_load(&p.scount[j], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    const uint32_t n = (uint32_t)total;
    const uint32_t need = n == 0 ? 1u : min(gridDim.x, (n + kBlock - 1) / kBlock);
    if (blockIdx.x >= need) return;   // (block-uniform: every thread has the same n)
    const Ent tab = entry_tables(p, smem);   // (its barrier also publishes pre)
    const Comm<S> comm = load_comm<S>(p);
    constexpr int NW = Codes<S>::kWords;
    unsigned long long best = ~0ull;
    for (uint32_t k = blockIdx.x * kBlock + threadIdx.x; k < n; k += gridDim.x * kBlock) {
        // the last segment j with pre[j] <= k holds survivor k
        uint32_t lo = 0, hi = nseg;
        while (hi - lo > 1) {
            const uint32_t mid = (lo + hi) >> 1;
            if (pre[mid] <= k) lo = mid;
            else hi = mid;
        }
        const uint32_t at = lo * (uint32_t)p.seg_cap + (k - pre[lo]);
        const uint32_t i = p.sidx[at];
        uint32_t w[NW], cut[S + 1], to[S], F[S], B[S];
#pragma unroll
        for (int kk = 0; kk < NW; ++kk) w[kk] = p.codes[kk * (uint32_t)p.ccap + at];
        unpack_cuts<S>(w, p.L, cut);
        const uint32_t a = assign_of(p, i);
        decode_toff<S>(p, tab, a, to);
        stage_weights<S>(p, tab, cut, to, F, B);
        const uint32_t T = dp_full_settle<S, SCH, AR>(p, tab, F, B, comm, w, a);
        const unsigned long long key = make_key(true, T, i);
        best = key < best ? key : best;
    }
    block_min_and_finish(best, p.acc, p.done, nullptr, p.run_best, true, false, publish ? p.snap : nullptr, need);
}

// host-side launchers
// ---------------------------------------------------------------------------
template <int S, typename R>
hipError_t launch_eval_s(const KParams &p, const LaunchCfg &lc, hipStream_t st) {
    if (p.sched) {
        const dim3 g(lc.grid), b(kBlock);
        if (p.has_ar && p.nslots) hipLaunchKernelGGL((sched_kernel<S, true, true>), g, b, lc.lds_bytes, st, p);
        else if (p.has_ar) hipLaunchKernelGGL((sched_kernel<S, true, false>), g, b, lc.lds_bytes, st, p);
        else if (p.nslots) hipLaunchKernelGGL((sched_kernel<S, false, true>), g, b, lc.lds_bytes, st, p);
        else hipLaunchKernelGGL((sched_kernel<S, false, false>), g, b, lc.lds_bytes, st, p);
        return hipGetLastError();
    }
    if (p.has_ar) hipLaunchKernelGGL((eval_kernel<S, true>), dim3(lc.grid), dim3(kBlock), lc.lds_bytes, st, p);
    else hipLaunchKernelGGL((eval_kernel<S, false>), dim3(lc.grid), dim3(kBlock), lc.lds_bytes, st, p);
    return hipGetLastError();
}

template <int S, typename R>
hipError_t launch_decode_s(const KParams &p, const LaunchCfg &lc, hipStream_t st) {
    const size_t lds = pascal_bytes<S, R>(p.L);   // (columns 2 .. S-1)
    hipLaunchKernelGGL((decode_kernel<S, R>), dim3(lc.grid), dim3(kBlock), lds, st, p);
    return hipGetLastError();
}

template <int S, typename R>
hipError_t launch_resume_s(const KParams &p, const LaunchCfg &lc, hipStream_t st, uint32_t lvl) {
    const dim3 g(lc.grid), b(kBlock);
    const bool sch = p.sched != 0;
    if (p.has_ar && sch) hipLaunchKernelGGL((resume_kernel<S, true, true>), g, b, lc.lds_bytes, st, p, lvl);
    else if (p.has_ar) hipLaunchKernelGGL((resume_kernel<S, true, false>), g, b, lc.lds_bytes, st, p, lvl);
    else if (sch) hipLaunchKernelGGL((resume_kernel<S, false, true>), g, b, lc.lds_bytes, st, p, lvl);
    else hipLaunchKernelGGL((resume_kernel<S, false, false>), g, b, lc.lds_bytes, st, p, lvl);
    return hipGetLastError();
}

// One piece of an early-stop chunk: filter_kernel on the grid in lc (LDS:
// Pascal columns, then the stage tables of lc.lds_bytes), in prefix then
// gather mode for S >= 4, else in full mode; then surv_kernel on lc.grid2
// blocks (LDS: the stage entries, then the scan of the lc.grid segment
// counts).
constexpr size_t kLdsBlockMax = 64 * 1024;   // LDS bytes one block of these kernels may use

template <int S, typename R, int MODE>
hipError_t launch_filter_s(const KParams &p, const LaunchCfg &lc, hipStream_t st) {
    const size_t pas = pascal_bytes<S, R, filter_col_lo<S, MODE>(), filter_col_hi<S, MODE>()>(p.L);
    const size_t fixed = p.has_ar ? filter_static_lds<S, true, MODE>() : filter_static_lds<S, false, MODE>();
    const dim3 fg(lc.grid), fb(kBlock);
    if (pas + lc.lds_bytes + fixed > kLdsBlockMax) {
        if (p.has_ar) hipLaunchKernelGGL((filter_kernel<S, R, true, true, MODE>), fg, fb, pas, st, p);
        else hipLaunchKernelGGL((filter_kernel<S, R, false, true, MODE>), fg, fb, pas, st, p);
    } else {
        const size_t lds = pas + lc.lds_bytes;
        if (p.has_ar) hipLaunchKernelGGL((filter_kernel<S, R, true, false, MODE>), fg, fb, lds, st, p);
        else hipLaunchKernelGGL((filter_kernel<S, R, false, false, MODE>), fg, fb, lds, st, p);
    }
    return hipGetLastError();
}

template <int S, typename R>
hipError_t launch_bounded_s(const KParams &p, const LaunchCfg &lc, hipStream_t st, uint32_t publish) {
    hipError_t e;
    if constexpr (filter_prefix<S>() > 0) {
        e = launch_filter_s<S, R, kFilterPrefix>(p, lc, st);
        if (e == hipSuccess) e = launch_filter_s<S, R, kFilterGather>(p, lc, st);
    } else {
        e = launch_filter_s<S, R, kFilterFull>(p, lc, st);
    }
    if (e != hipSuccess) return e;
    const uint32_t nseg = lc.grid;
    const dim3 g(lc.grid2), b(kBlock);
    const size_t sl = (size_t)p.ent_lds + ((size_t)nseg + 1) * 4;
    if (sl > kLdsBlockMax || lc.grid2 == 0) return hipErrorInvalidValue;
    const bool sch = p.sched != 0;
    if (p.has_ar && sch) hipLaunchKernelGGL((surv_kernel<S, true, true>), g, b, sl, st, p, publish, nseg);
    else if (p.has_ar) hipLaunchKernelGGL((surv_kernel<S, true, false>), g, b, sl, st, p, publish, nseg);
    else if (sch) hipLaunchKernelGGL((surv_kernel<S, false, true>), g, b, sl, st, p, publish, nseg);
    else hipLaunchKernelGGL((surv_kernel<S, false, false>), g, b, sl, st, p, publish, nseg);
    return hipGetLastError();
}

// Resident blocks per CU of the early-stop filter instances launch_bounded_s
// picks (their LDS: the Pascal columns plus the stage entries of `ent_lds`);
// with two modes the smaller of their counts, so that the second runs its
// blocks, one per segment of the first's list, in one wave too.
template <int S, typename R, int MODE>
hipError_t filter_occupancy_mode(const KParams &p, size_t ent_lds, int *blocks) {
    const size_t pas = pascal_bytes<S, R, filter_col_lo<S, MODE>(), filter_col_hi<S, MODE>()>(p.L);
    const size_t fixed = p.has_ar ? filter_static_lds<S, true, MODE>() : filter_static_lds<S, false, MODE>();
    if (pas + ent_lds + fixed > kLdsBlockMax) {
        if (p.has_ar) return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks, filter_kernel<S, R, true, true, MODE>, kBlock, pas);
        return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks, filter_kernel<S, R, false, true, MODE>, kBlock, pas);
    }
    if (p.has_ar)
        return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks, filter_kernel<S, R, true, false, MODE>, kBlock, pas + ent_lds);
    return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks, filter_kernel<S, R, false, false, MODE>, kBlock, pas + ent_lds);
}

template <int S, typename R>
hipError_t filter_occupancy_s(const KParams &p, size_t ent_lds, int *blocks) {
    if constexpr (filter_prefix<S>() > 0) {
        int a = 0, b = 0;
        hipError_t e = filter_occupancy_mode<S, R, kFilterPrefix>(p, ent_lds, &a);
        if (e == hipSuccess) e = filter_occupancy_mode<S, R, kFilterGather>(p, ent_lds, &b);
        *blocks = a < b ? a : b;
        return e;
    } else {
        return filter_occupancy_mode<S, R, kFilterFull>(p, ent_lds, blocks);
    }
}

template <int S, typename R>
hipError_t occupancy_s(int *blocks, size_t lds, bool ar, bool sched) {
    // schedules other than 1F1B: the closed-form kernel (the table kernel
    // runs few candidates per call in practice and takes the same grid)
    if (sched && ar) return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks, sched_kernel<S, true, false>, kBlock, lds);
    if (sched) return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks, sched_kernel<S, false, false>, kBlock, lds);
    if (ar) return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks, eval_kernel<S, true>, kBlock, lds);
    return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks, eval_kernel<S, false>, kBlock, lds);
}


}  // namespace pk
