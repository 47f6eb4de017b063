#pragma once
// Device code of the pruned configuration search (Sec. 4.2.3): stage-level
// pruning with Eq. 2 (Theorem 1) and layer-level pruning with the ridge
// pattern (Theorem 2) over partial configurations, level by level.
//
// A frontier node is a partial configuration of one assignment row: the
// row and the cut codes of stages 1..x (one byte per cut).  Every quantity
// the tests need (prefix forward time, the inner max of Eq. 2, the last
// backward time, the ridge state of a type) is recomputed from the cuts and
// the LDS prefix tables, so a node is 4 + 4 * ceil((S-1)/4) bytes.
//
// Level x -> x+1 runs two kernels over the frontier.  The children of a node
// are the end points hi = c_x+1, c_x+2, ... of stage x+1 up to the first
// one that fails a test: the memory sum and g(S_{x+1}) only grow with hi,
// and once a type's counts are falling the ridge test fails for every
// larger count too, so the accepted children form one contiguous range,
// whose length a binary search finds.
// search_count_kernel counts them per block; search_scan_kernel turns the
// block counts into offsets; search_write_kernel writes the children in
// node order (a block-local scan places each node's range), so the next
// frontier is again in search order (row, then composition rank).  The
// level that fixes the last cut (x = S-2) also tests the last stage, which
// that cut determines, and keeps only the children that pass, so the widest
// level is never written in full.  When the children of one block always fit
// a frontier piece, the level before it (x = S-3) is fused with it: the count
// and write kernels expand each accepted child there at once (its prefix
// quantities extended by one stage), so the widest level is not written at
// all.  search_leaf_kernel runs the full DP on the complete configurations.
#include "poseidon_kernels.h"

namespace pk {

constexpr uint32_t kSearchRidge = 1u, kSearchNoStage = 2u;

struct SearchNode {
    uint32_t row, lo, t;          // row, c_x, type of stage x+1
    uint32_t pre_f, inner, last_b;
    int32_t last_l;               // last layer count of type t among stages 1..x (-1: none)
    bool falling;                 // type t's counts have started to fall
    uint32_t tS;                  // type of stage S, with its ridge state over stages 1..x
    int32_t last_lS;
    bool fallingS;
    uint32_t tN;                  // type of stage x+2, with its ridge state over stages 1..x
    int32_t last_lN;              // (what a child's own stage test needs)
    bool fallingN;
};

// Prefix quantities of a node at level x (stages 1..x fixed).
template <int S, bool AR>
__device__ __forceinline__ SearchNode search_node(const KParams &p, const Lds &tab, uint32_t row,
                                                  const uint32_t (&w)[Codes<S>::kWords], uint32_t x,
                                                  uint32_t (&ty)[S], uint32_t (&cut)[S + 1]) {
    decode_types<S>(p, row, ty);
    cut[0] = 0;
#pragma unroll
    for (int s = 1; s < S; ++s) cut[s] = (w[(s - 1) >> 2] >> (8 * ((s - 1) & 3))) & 0xFFu;
    cut[S] = p.L;
    SearchNode n;
    n.row = row;
    n.lo = 0;
    n.t = ty[0];
    n.pre_f = 0;
    n.inner = 0;
    n.last_b = 0;
#pragma unroll
    for (int s = 0; s < S; ++s) {
        if ((uint32_t)s == x) { n.lo = cut[s]; n.t = ty[s]; }
    }
    n.last_l = -1;
    n.falling = false;
    n.tS = ty[S - 1];
    n.last_lS = -1;
    n.fallingS = false;
    n.tN = ty[0];
#pragma unroll
    for (int s = 0; s < S; ++s) {
        if ((uint32_t)s == x + 1) n.tN = ty[s];
    }
    n.last_lN = -1;
    n.fallingN = false;
    const uint32_t row_len = p.L + 1;
#pragma unroll
    for (int s = 0; s < S; ++s) {
        if ((uint32_t)s < x) {
            const uint64_t *c = tab.cost + ty[s] * row_len;
            const uint64_t hi = c[cut[s + 1]], lo = c[cut[s]];
            const uint32_t f = (uint32_t)hi - (uint32_t)lo, b = (uint32_t)(hi >> 32) - (uint32_t)(lo >> 32);
            const uint32_t d = AR ? tab.pd[ty[s] * row_len + cut[s + 1]] - tab.pd[ty[s] * row_len + cut[s]] : 0u;
            n.inner = s == 0 ? d : max(n.inner + n.last_b, d);
            n.pre_f += f;
            n.last_b = b;
            const int32_t l = (int32_t)(cut[s + 1] - cut[s]);
            if (ty[s] == n.t) {
                if (n.last_l >= 0 && l < n.last_l) n.falling = true;
                n.last_l = l;
            }
            if (ty[s] == n.tS) {
                if (n.last_lS >= 0 && l < n.last_lS) n.fallingS = true;
                n.last_lS = l;
            }
            if (ty[s] == n.tN) {
                if (n.last_lN >= 0 && l < n.last_lN) n.fallingN = true;
                n.last_lN = l;
            }
        }
    }
    return n;
}

// The child of a node at level x with stage x+1 = [lo, c): its prefix
// quantities at level x+1, extended by that one stage (the type of its
// stage x+3 is not tracked: used for the level that fixes the last cut,
// whose children are complete).
template <bool AR>
__device__ __forceinline__ SearchNode search_child(const KParams &p, const Lds &tab, const SearchNode &n, uint32_t x,
                                                   uint32_t c) {
    const uint32_t row_len = p.L + 1;
    const uint64_t *ct = tab.cost + n.t * row_len;
    const uint64_t ch = ct[c], cl = ct[n.lo];
    const uint32_t f = (uint32_t)ch - (uint32_t)cl, b = (uint32_t)(ch >> 32) - (uint32_t)(cl >> 32);
    const uint32_t d = AR ? tab.pd[n.t * row_len + c] - tab.pd[n.t * row_len + n.lo] : 0u;
    const int32_t l = (int32_t)(c - n.lo);
    SearchNode m = n;
    m.lo = c;
    m.t = n.tN;
    m.inner = x == 0 ? d : max(n.inner + n.last_b, d);
    m.pre_f = n.pre_f + f;
    m.last_b = b;
    m.last_l = n.last_lN;
    m.falling = n.fallingN;
    if (n.t == n.tN) {
        m.falling = m.falling || (m.last_l >= 0 && l < m.last_l);
        m.last_l = l;
    }
    if (n.t == n.tS) {
        m.fallingS = m.fallingS || (m.last_lS >= 0 && l < m.last_lS);
        m.last_lS = l;
    }
    return m;
}

// Outcome of trying stage x+1 = [lo, hi): 0 accepted, 1 memory, 2 ridge, 3 bound.
template <bool AR>
__device__ __forceinline__ int search_try(const KParams &p, const Lds &tab, const SearchNode &n, uint32_t x,
                                          uint32_t hi, uint32_t flags, uint32_t bound) {
    const uint32_t row_len = p.L + 1;
    if (tab.pm[hi] - tab.pm[n.lo] > tab.cap[n.t]) return 1;
    const int32_t l = (int32_t)(hi - n.lo);
    if ((flags & kSearchRidge) && n.last_l >= 0 && n.falling && l > n.last_l) return 2;
    if (!(flags & kSearchNoStage)) {
        const uint64_t *c = tab.cost + n.t * row_len;
        const uint64_t ch = c[hi], cl = c[n.lo];
        const uint32_t f = (uint32_t)ch - (uint32_t)cl, b = (uint32_t)(ch >> 32) - (uint32_t)(cl >> 32);
        const uint32_t d = AR ? tab.pd[n.t * row_len + hi] - tab.pd[n.t * row_len + n.lo] : 0u;
        const uint32_t inn = x == 0 ? d : max(n.inner + n.last_b, d);
        // Eq. 2: g(S_{x+1}) = sum_{i<=x} F_i + M (F_{x+1} + B_{x+1}) + inner
        if (n.pre_f + p.M * (f + b) + inn > bound) return 3;
    }
    return 0;
}

// Per-type tables of the stage tests, built in LDS behind the stage tables
// by the count and write kernels: fb = prefix fwd + prefix bwd, mfb = M fb
// (below 2^31 like every path weight, checked at load), and hm[t][lo] = the
// largest h with layers [lo, h) within type t's memory cap.  Without
// all-reduce times a stage's Eq. 2 test is then one compare, mfb[h] against
// a per-node threshold, and its memory test a cap on the range.
struct SearchTab {
    const uint32_t *fb, *mfb, *hm;
};

// LDS bytes of the stage tables (the layout of stage_tables), where the
// search tables start; the host sizes the launch the same way.
__device__ __forceinline__ uint32_t search_tab_offset(const KParams &p) {
    const uint32_t n = p.T * (p.L + 1);
    return (n * 8 + (p.L + 1) * 4 + p.T * 4 + (p.has_ar ? n * 4 : 0) + 15) & ~15u;
}

__device__ __forceinline__ SearchTab search_tables(const KParams &p, const Lds &tab, unsigned char *smem) {
    const uint32_t row = p.L + 1, n = p.T * row;
    uint32_t *fb = reinterpret_cast<uint32_t *>(smem + search_tab_offset(p)), *mfb = fb + n, *hm = mfb + n;
    for (uint32_t i = threadIdx.x; i < n; i += kBlock) {
        const uint64_t c = tab.cost[i];
        const uint32_t v = (uint32_t)c + (uint32_t)(c >> 32);
        fb[i] = v;
        mfb[i] = p.M * v;
        const uint32_t t = i / row, lo = i - t * row;
        // pm only grows: the largest h that fits, by halving steps from lo
        uint32_t h = lo;
        for (uint32_t st = 256; st; st >>= 1)
            if (h + st <= p.L && tab.pm[h + st] - tab.pm[lo] <= tab.cap[t]) h += st;
        hm[i] = h;
    }
    __syncthreads();
    return SearchTab{fb, mfb, hm};
}

// The rule that ended a node's accepted range of k end points (0: it ran to
// hmax): the first test end point lo+k+1 fails, in the order memory, ridge,
// bound.  Without all-reduce times the memory and ridge outcomes are range
// limits, and a maximal range that neither ended must have met the bound.
template <bool AR>
__device__ __forceinline__ int search_stop(const KParams &p, const Lds &tab, const SearchTab &sx,
                                           const SearchNode &n, uint32_t x, uint32_t k, uint32_t hmax,
                                           uint32_t flags, uint32_t bound) {
    const uint32_t h = n.lo + k + 1;
    if (h > hmax) return 0;
    if (AR) return search_try<AR>(p, tab, n, x, h, flags, bound);
    if (h > sx.hm[n.t * (p.L + 1) + n.lo]) return 1;
    if ((flags & kSearchRidge) && n.last_l >= 0 && n.falling && (int32_t)(h - n.lo) > n.last_l) return 2;
    return 3;
}

// Outcomes of the last-stage test of the children of one node.
struct LastStage {
    uint32_t pass = 0, mem = 0, ridge = 0, bound = 0;
};

// Number k of accepted choices of stage x+1: the end points lo+1 .. lo+k
// pass the memory, ridge and Eq. 2 tests and lo+k+1 (if <= hmax) fails one.
// Each test, once failed, fails for every larger end point (the memory sum
// and g(S_{x+1}) only grow with it; a falling type's ridge test fails for
// every count above its last one), so k is found by a binary search over
// the end points instead of trying them one by one.
template <bool AR>
__device__ __forceinline__ uint32_t search_accepted(const KParams &p, const Lds &tab, const SearchTab &sx,
                                                    const SearchNode &n, uint32_t x, uint32_t hmax, uint32_t flags,
                                                    uint32_t bound) {
    const uint32_t row_len = p.L + 1;
    uint32_t len = hmax - n.lo;
    if ((flags & kSearchRidge) && n.last_l >= 0 && n.falling) len = min(len, (uint32_t)n.last_l);
    const int H = (int)decode_levels(p.L);   // (uniform: the steps above it are skipped by scalar branches)
    if (!AR) {
        // memory caps the range; Eq. 2, pre_f + M (fb[h] - fb[lo]) + inn <= bound
        // with inn = inner + last_b (0 for the first stage), is mfb[h] <= thr
        const uint32_t *mf = sx.mfb + n.t * row_len;
        len = min(len, sx.hm[n.t * row_len + n.lo] - n.lo);
        if (flags & kSearchNoStage) return len;
        const int64_t thr64 = (int64_t)bound + mf[n.lo] - n.pre_f - (x == 0 ? 0u : n.inner + n.last_b);
        const int32_t thr = thr64 > INT32_MAX ? INT32_MAX : thr64 < 0 ? -1 : (int32_t)thr64;
        // each step loads (an in-range entry) and combines its tests without
        // branches, so the wave never splits over them
        uint32_t k = 0;
#pragma unroll
        for (int b = 7; b >= 0; --b) {
            if (b >= H) continue;
            const uint32_t t = k + (1u << b);
            const int32_t v = (int32_t)mf[n.lo + min(t, len)];
            k = ((t <= len) & (v <= thr)) ? t : k;
        }
        return k;
    }
    const uint64_t *ct = tab.cost + n.t * row_len;
    const uint64_t cl = ct[n.lo];
    const uint32_t pml = tab.pm[n.lo], capt = tab.cap[n.t];
    // with all-reduce times: each probe evaluates the memory and Eq. 2 tests
    const uint32_t *pdt = tab.pd + n.t * row_len;
    const uint32_t dl = pdt[n.lo];
    const bool stage = !(flags & kSearchNoStage);
    const uint32_t carry = n.inner + n.last_b;
    uint32_t k = 0;
#pragma unroll
    for (int b = 7; b >= 0; --b) {
        if (b >= H) continue;
        const uint32_t t = k + (1u << b);
        const uint32_t h = n.lo + min(t, len);
        bool ok = tab.pm[h] - pml <= capt;
        if (stage) {
            const uint64_t ch = ct[h];
            const uint32_t f = (uint32_t)ch - (uint32_t)cl, bw = (uint32_t)(ch >> 32) - (uint32_t)(cl >> 32);
            const uint32_t d = pdt[h] - dl;
            const uint32_t inn = x == 0 ? d : max(carry, d);
            ok = ok && n.pre_f + p.M * (f + bw) + inn <= bound;
        }
        k = (t <= len && ok) ? t : k;
    }
    return k;
}

// Children lo+1 .. lo+k of a node at the level that fixes the last cut
// (x + 2 == S): each fixes every cut, so the last stage [hi, L) is tested
// here (memory in closed form through last_lo, then ridge, then Eq. 2) and
// only children that pass it are kept; lp counts the outcomes.  With WRITE
// the kept children go to positions base, base + 1, ... in order.
//
// Without all-reduce times the last stage's Eq. 2 splits into a per-node
// constant and a function of hi alone:
//   g(S_S) = C + G(hi),  G(hi) = Pf_t[hi] + Pb_t[hi] - M (Pf_tS[hi] + Pb_tS[hi])
// (t, tS the types of stages S-1 and S, Pf / Pb the prefix times).  G falls
// as hi grows when no layer's forward + backward time on t exceeds M times
// that on tS (checked per type pair on the host: bit 8 t + tS of p.g_mono), and the
// last stage's ridge test fails on a prefix of the end points too, so then
// every outcome count is a range length: the ridge prefix in closed form,
// the bound prefix by a binary search.  Otherwise the end points are tried
// one by one.
template <int S>
__device__ __forceinline__ void search_write_child(const SearchParams &q, uint64_t o, uint32_t row, uint32_t x,
                                                   uint32_t hi, const uint32_t (&w)[Codes<S>::kWords]) {
    q.out_row[o] = row;
#pragma unroll
    for (int k = 0; k < Codes<S>::kWords; ++k) {
        const uint32_t v = (uint32_t)k == (x >> 2) ? (w[k] | (hi << (8 * (x & 3)))) : w[k];
        q.out_codes[(uint64_t)k * q.out_cap + o] = v;
    }
}

template <int S, bool AR, bool WRITE, bool MONO>
__device__ __forceinline__ uint32_t search_last_children(const KParams &p, const Lds &tab, const SearchTab &sx,
                                                         const SearchNode &n, uint32_t x, uint32_t k, uint32_t flags,
                                                         uint32_t bound,
                                                         LastStage &lp, const SearchParams &q, uint64_t base,
                                                         const uint32_t (&w)[Codes<S>::kWords]) {
    const uint32_t row_len = p.L + 1;
    // the last stage [hi, L) exceeds its cap exactly for hi < last_lo[type]
    const uint32_t mem_lo = p.last_lo[n.tS];
    const uint32_t h0 = max(n.lo + 1, mem_lo), h1 = n.lo + k;
    lp.mem += (h0 <= h1 ? h0 : h1 + 1) - (n.lo + 1);
    const bool ridge = (flags & kSearchRidge) != 0, stage = !(flags & kSearchNoStage);
    const bool same = n.t == n.tS;
    if (!AR && (MONO || ((p.g_mono >> (8 * n.t + n.tS)) & 1ull))) {
        if (h0 > h1) return 0;
        // ridge: the end points below r0 fail
        uint32_t r0 = h0;
        if (ridge) {
            if (same) {
                // counts of type t fall before lo + last_lS (or throughout), and the
                // last stage is then longer than stage S-1 below ceil((L + lo) / 2)
                const uint32_t e1 = (p.L + n.lo + 1) / 2;
                const uint32_t e2 = n.fallingS ? 0xFFFFFFFFu : (n.last_lS >= 0 ? n.lo + (uint32_t)n.last_lS : 0u);
                r0 = max(h0, min(e1, e2));
            } else if (n.last_lS >= 0 && n.fallingS) {
                r0 = max(h0, p.L - (uint32_t)n.last_lS);
            }
            r0 = min(r0, h1 + 1);
            lp.ridge += r0 - h0;
        }
        // Eq. 2: the end points below g0 fail
        uint32_t g0 = r0;
        if (stage && r0 <= h1) {
            const uint32_t *ft = sx.fb + n.t * row_len, *ms = sx.mfb + n.tS * row_len;
            // g(hi) = C + G(hi), G(hi) = fb_t[hi] - mfb_tS[hi].  g is an Eq. 2
            // value, below 2^31 like every path weight (checked at load), so
            // C + G evaluates exactly in 32-bit modular arithmetic
            const uint32_t C = n.pre_f - ft[n.lo] + (x == 0 ? 0u : n.inner + n.last_b) + ms[p.L];
            const uint32_t len = h1 + 1 - r0;
            // g is smallest at h1: if even that fails, every end point does
            // (the usual case, so the search below mostly runs on no lane)
            uint32_t j = len;
            if (C + ft[h1] - ms[h1] <= bound) {
                const int H = (int)decode_levels(p.L);
                j = 0;
#pragma unroll
                for (int b = 7; b >= 0; --b) {
                    if (b >= H) continue;
                    const uint32_t t = j + (1u << b);
                    const uint32_t h = r0 + min(t, len) - 1;
                    j = ((t <= len) & (C + ft[h] - ms[h] > bound)) ? t : j;
                }
            }
            g0 = r0 + j;
            lp.bound += j;
        }
        lp.pass += h1 + 1 - g0;
        if (WRITE) {
            for (uint32_t hi = g0; hi <= h1; ++hi) search_write_child<S>(q, base + (hi - g0), n.row, x, hi, w);
        }
        return h1 + 1 - g0;
    }
    const uint64_t *ct = tab.cost + n.t * row_len, *cs = tab.cost + n.tS * row_len;
    const uint64_t cl = ct[n.lo], cL = cs[p.L];
    const uint32_t *pdt = tab.pd + n.t * row_len, *pds = tab.pd + n.tS * row_len;
    const uint32_t dl = AR ? pdt[n.lo] : 0u, dL = AR ? pds[p.L] : 0u;
    const uint32_t carry = n.inner + n.last_b;
    uint32_t out = 0;
    for (uint32_t hi = h0; hi <= h1; ++hi) {
        if (ridge) {
            // type tS's counts with stage x+1 appended when it has that type
            const int32_t l = (int32_t)(hi - n.lo);
            int32_t ll = n.last_lS;
            bool fall = n.fallingS;
            if (same) {
                fall = fall || (ll >= 0 && l < ll);
                ll = l;
            }
            if (ll >= 0 && fall && (int32_t)(p.L - hi) > ll) {
                lp.ridge += 1;
                continue;
            }
        }
        if (stage) {
            const uint64_t ch = ct[hi], sh = cs[hi];
            const uint32_t f = (uint32_t)ch - (uint32_t)cl, b = (uint32_t)(ch >> 32) - (uint32_t)(cl >> 32);
            const uint32_t d = AR ? pdt[hi] - dl : 0u;
            const uint32_t inn = x == 0 ? d : max(carry, d);
            const uint32_t fS = (uint32_t)cL - (uint32_t)sh, bS = (uint32_t)(cL >> 32) - (uint32_t)(sh >> 32);
            const uint32_t dS = AR ? dL - pds[hi] : 0u;
            // Eq. 2 for the last stage: g(S_S) = sum_{i<S} F_i + M (F_S + B_S) + max(inner + B_{S-1}, d_S)
            if (n.pre_f + f + p.M * (fS + bS) + max(inn + b, dS) > bound) {
                lp.bound += 1;
                continue;
            }
        }
        lp.pass += 1;
        if (WRITE) search_write_child<S>(q, base + out, n.row, x, hi, w);
        ++out;
    }
    return out;
}

__device__ __forceinline__ void search_flush(const SearchParams &q, unsigned int visited, unsigned int evaluated,
                                             unsigned int mem, unsigned int ridge, unsigned int bound) {
    __shared__ unsigned int c[5];
    if (threadIdx.x < 5) c[threadIdx.x] = 0;
    __syncthreads();
    if (visited) atomicAdd(&c[0], visited);
    if (evaluated) atomicAdd(&c[1], evaluated);
    if (mem) atomicAdd(&c[2], mem);
    if (ridge) atomicAdd(&c[3], ridge);
    if (bound) atomicAdd(&c[4], bound);
    __syncthreads();
    if (threadIdx.x < 5 && c[threadIdx.x]) atomicAdd(&q.stats[threadIdx.x], (unsigned long long)c[threadIdx.x]);
}

// The count kernel's counters: summed over the block in LDS, then one
// atomic per counter into the block's slot of q.stats_part.
__device__ __forceinline__ void search_block_counts(const SearchParams &q, unsigned int visited, unsigned int evaluated,
                                                    unsigned int mem, unsigned int ridge, unsigned int bound) {
    __shared__ unsigned int c[5];
    if (threadIdx.x < 5) c[threadIdx.x] = 0;
    __syncthreads();
    if (visited) atomicAdd(&c[0], visited);
    if (evaluated) atomicAdd(&c[1], evaluated);
    if (mem) atomicAdd(&c[2], mem);
    if (ridge) atomicAdd(&c[3], ridge);
    if (bound) atomicAdd(&c[4], bound);
    __syncthreads();
    if (threadIdx.x < 5 && c[threadIdx.x])
        atomicAdd(&q.stats_part[threadIdx.x * kStatSlots + blockIdx.x % kStatSlots], (unsigned long long)c[threadIdx.x]);
}

template <int S>
__device__ __forceinline__ void search_load(const SearchParams &q, uint32_t i, bool active, uint32_t &row,
                                            uint32_t (&w)[Codes<S>::kWords]) {
    row = active ? q.in_row[i] : 0u;
#pragma unroll
    for (int k = 0; k < Codes<S>::kWords; ++k) w[k] = active ? q.in_codes[(uint64_t)k * q.in_cap + i] : 0u;
}

// Nodes of the level: counted on the device by the previous level's scan
// when the host launched on an upper bound (q.n_dev), else q.n_in.
__device__ __forceinline__ uint32_t search_n_in(const SearchParams &q) {
    return q.n_dev ? (uint32_t)*q.n_dev : q.n_in;
}

// Count the children of every node of the piece; one total per block.  The
// kernel waits on chains of dependent LDS loads (binary searches), so it
// asks for 7 waves per SIMD (72 VGPRs, no spills for any S) rather than the
// compiler's choice of 6.
template <int S, bool AR, bool MONO>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(7, 8))) void search_count_kernel(KParams p, SearchParams q) {
    extern __shared__ __align__(16) unsigned char smem[];
    const uint32_t n_in = search_n_in(q);
    if (blockIdx.x * kBlock >= n_in) {
        // a block past the level's nodes (grid from an upper bound): zero total
        if (threadIdx.x == 0) q.blk_tot[blockIdx.x] = 0;
        return;
    }
    const Lds tab = stage_tables(p, smem);
    const SearchTab sx = search_tables(p, tab, smem);
    const uint32_t i = blockIdx.x * kBlock + threadIdx.x;
    const bool active = i < n_in;
    const uint32_t bound = *q.bound;
    uint32_t row, w[Codes<S>::kWords], ty[S], cut[S + 1];
    search_load<S>(q, i, active, row, w);
    uint32_t cnt = 0, visited = 0;
    LastStage lp;
    uint32_t why_mem = 0, why_ridge = 0, why_bound = 0;
    if (active) {
        const uint32_t x = q.level;
        const SearchNode n = search_node<S, AR>(p, tab, row, w, x, ty, cut);
        const uint32_t hmax = p.L - (S - 1 - x);   // every later stage keeps one layer
        const uint32_t acc = search_accepted<AR>(p, tab, sx, n, x, hmax, q.flags, bound);
        // the rule that stopped the range (0: it ran to its structural end)
        const int why = search_stop<AR>(p, tab, sx, n, x, acc, hmax, q.flags, bound);
        visited = acc;
        why_mem = why == 1;
        why_ridge = why == 2;
        why_bound = why == 3;
        if (q.fused) {
            // x + 3 == S: each child fixes stage S-2 and is expanded here at
            // once; its children fix the last cut, and those that pass the last
            // stage are kept (complete configurations)
            for (uint32_t c = n.lo + 1; c <= n.lo + acc; ++c) {
                const SearchNode m = search_child<AR>(p, tab, n, x, c);
                const uint32_t acc2 = search_accepted<AR>(p, tab, sx, m, x + 1, p.L - 1, q.flags, bound);
                const int why2 = search_stop<AR>(p, tab, sx, m, x + 1, acc2, p.L - 1, q.flags, bound);
                visited += acc2;
                why_mem += why2 == 1;
                why_ridge += why2 == 2;
                why_bound += why2 == 3;
                cnt += search_last_children<S, AR, false, MONO>(p, tab, sx, m, x + 1, acc2, q.flags, bound, lp, q, 0, w);
            }
        } else {
            cnt = x + 2 == (uint32_t)S ? search_last_children<S, AR, false, MONO>(p, tab, sx, n, x, acc, q.flags, bound, lp, q, 0, w)
                                       : acc;
        }
        q.node_cnt[i] = (uint16_t)cnt;   // at most (L - 1)^2 < 2^16 children (fused), else L - 1
    }
    __shared__ unsigned int tot;
    if (threadIdx.x == 0) tot = 0;
    __syncthreads();
    const unsigned int wsum = (unsigned int)wave_sum_u32(cnt);
    if ((threadIdx.x & 63) == 0 && wsum) atomicAdd(&tot, wsum);
    // a child that completes the configuration and passes the last stage
    // counts as visited twice (its stage x+1 and its stage S) and evaluated.
    search_block_counts(q, visited + lp.pass, lp.pass, why_mem + lp.mem, why_ridge + lp.ridge, why_bound + lp.bound);
    if (threadIdx.x == 0) q.blk_tot[blockIdx.x] = tot;
}

// Write the children of blocks [blk_base, blk_base + gridDim.x) in node
// order, the first one at position 0 of the output.
template <int S, bool AR, bool MONO>
__global__ __launch_bounds__(kBlock) void search_write_kernel(KParams p, SearchParams q) {
    extern __shared__ __align__(16) unsigned char smem[];
    const uint32_t blk = q.blk_base + blockIdx.x;
    const uint32_t n_in = search_n_in(q);
    if (blk * kBlock >= n_in) return;   // past the level's nodes
    constexpr int NW = Codes<S>::kWords;
    const uint32_t i = blk * kBlock + threadIdx.x;
    const bool active = i < n_in;
    const uint32_t x = q.level;
    // the count kernel left each node's number of children: nodes without
    // any (most of them at the level that fixes the last cut) do nothing
    const uint32_t cnt = active ? q.node_cnt[i] : 0u;
    unsigned long long total;
    const unsigned long long local = block_exclusive_scan_u64(cnt, total);
    if (total == 0) return;   // no child in the block (most blocks of the last-cut level)
    const uint64_t blk0 = q.blk_off[blk] - q.blk_off[q.blk_base];
    if (!q.fused && x + 2 != (uint32_t)S) {
        // every accepted choice is a child: c_{x+1} = lo+1 .. lo+cnt.  The
        // wave writes the children of its nodes together, 64 consecutive ones
        // per store: lane j takes child o0 + j of the wave's run, and its
        // parent is the first lane whose inclusive count exceeds that
        // (a binary search over the lanes)
        uint32_t row, w[NW];
        search_load<S>(q, i, active, row, w);
        uint32_t lo = 0;
#pragma unroll
        for (int s = 1; s < S; ++s)
            if ((uint32_t)s == x) lo = (w[(s - 1) >> 2] >> (8 * ((s - 1) & 3))) & 0xFFu;
        const uint32_t lane = threadIdx.x & 63;
        const unsigned long long l0 = __shfl(local, 0, 64);
        const uint32_t incl = (uint32_t)(local - l0) + cnt;
        const uint32_t wtot = __shfl(incl, 63, 64);
        for (uint32_t o0 = 0; o0 < wtot; o0 += 64) {
            const uint32_t o = o0 + lane;
            uint32_t pl = 0;
#pragma unroll
            for (uint32_t b = 32; b; b >>= 1) pl = __shfl(incl, (int)(pl + b - 1), 64) <= o ? pl + b : pl;
            const uint32_t first = __shfl(incl - cnt, (int)pl, 64);
            const uint32_t prow = __shfl(row, (int)pl, 64), plo = __shfl(lo, (int)pl, 64);
            uint32_t pw[NW];
#pragma unroll
            for (int k = 0; k < NW; ++k) pw[k] = __shfl(w[k], (int)pl, 64);
            if (o < wtot) search_write_child<S>(q, blk0 + l0 + o, prow, x, plo + 1 + (o - first), pw);
        }
        return;
    }
    const Lds tab = stage_tables(p, smem);
    const SearchTab sx = search_tables(p, tab, smem);
    const uint32_t bound = *q.bound;
    if (cnt) {
        uint32_t row, w[NW], ty[S], cut[S + 1];
        search_load<S>(q, i, true, row, w);
        const uint64_t base = blk0 + local;
        if (q.fused) {
            // the complete configurations under each child, child by child
            LastStage lp;
            const SearchNode n = search_node<S, AR>(p, tab, row, w, x, ty, cut);
            const uint32_t acc = search_accepted<AR>(p, tab, sx, n, x, p.L - (S - 1 - x), q.flags, bound);
            uint64_t o = base;
            for (uint32_t c = n.lo + 1; c <= n.lo + acc; ++c) {
                const SearchNode m = search_child<AR>(p, tab, n, x, c);
                const uint32_t acc2 = search_accepted<AR>(p, tab, sx, m, x + 1, p.L - 1, q.flags, bound);
                uint32_t wc[NW];
#pragma unroll
                for (int k = 0; k < NW; ++k) wc[k] = (uint32_t)k == (x >> 2) ? (w[k] | (c << (8 * (x & 3)))) : w[k];
                o += search_last_children<S, AR, true, MONO>(p, tab, sx, m, x + 1, acc2, q.flags, bound, lp, q, o, wc);
            }
        } else {   // x + 2 == S
            LastStage lp;
            const SearchNode n = search_node<S, AR>(p, tab, row, w, x, ty, cut);
            const uint32_t acc = search_accepted<AR>(p, tab, sx, n, x, p.L - (S - 1 - x), q.flags, bound);
            search_last_children<S, AR, true, MONO>(p, tab, sx, n, x, acc, q.flags, bound, lp, q, base, w);
        }
    }
}

// Level S-1: the last stage is [c_{S-1}, L); test it like any stage, then
// evaluate the complete configuration on the DAG.  Reduces
// (T << 32 | position) over the candidates with T <= bound into *q.acc.
template <int S, bool AR, bool SCH>
__global__ __launch_bounds__(kBlock) void search_leaf_kernel(KParams p, SearchParams q) {
    extern __shared__ __align__(16) unsigned char smem[];
    const uint32_t n_in = search_n_in(q);
    if (blockIdx.x * kBlock >= n_in) return;   // past the level's nodes
    const Lds tab = stage_tables(p, smem);
    const Comm<S> comm = load_comm<S>(p);
    constexpr int NW = Codes<S>::kWords;
    const uint32_t i = blockIdx.x * kBlock + threadIdx.x;
    const bool active = i < n_in;
    const uint32_t bound = *q.bound;
    uint32_t row, w[NW], ty[S], cut[S + 1];
    search_load<S>(q, i, active, row, w);
    int why = 4;
    unsigned long long key = ~0ull;
    if (active) {
        const SearchNode n = search_node<S, AR>(p, tab, row, w, S - 1, ty, cut);
        // for S > 1 the level that fixed the last cut already tested the last stage
        why = S == 1 ? search_try<AR>(p, tab, n, S - 1, p.L, q.flags, bound) : 0;
    }
    const bool leaf = why == 0;
    if (leaf) {
        uint32_t F[S], B[S];
        stage_weights<S>(p, tab, cut, ty, F, B);
        const uint32_t T = dp_full_settle<S, SCH, AR>(p, tab, F, B, comm, w, row);
        if (T <= bound) key = ((unsigned long long)T << 32) | i;
    }
    if (S == 1) search_flush(q, leaf, leaf, why == 1, why == 2, why == 3);
    block_min_and_finish(key, q.acc, nullptr, nullptr, nullptr, false);
}

// After a leaf piece: the piece's best candidate replaces the best so far
// only if strictly better (earlier pieces and chunks come first in search
// order).  best[0..2] = makespan, row, composition rank.
template <typename R>
__global__ void search_merge_kernel(KParams p, SearchParams q) {
    if (threadIdx.x != 0 || blockIdx.x != 0) return;
    const unsigned long long key = *q.acc;
    *q.acc = ~0ull;
    if (key == ~0ull) return;
    const uint64_t T = key >> 32;
    const uint32_t pos = (uint32_t)key;
    if (T >= q.best[0]) return;
    const R *binom = reinterpret_cast<const R *>(p.binom);
    const uint32_t S = p.S, L = p.L;
    // rank = sum_j C(L - 1 - c_{j-1}, S - j) - C(L - c_j, S - j)   (hockey-stick identity)
    uint64_t rank = 0;
    uint32_t prev = 0;
    for (uint32_t j = 1; j < S; ++j) {
        const uint32_t wj = q.in_codes[(uint64_t)((j - 1) >> 2) * q.in_cap + pos];
        const uint32_t c = (wj >> (8 * ((j - 1) & 3))) & 0xFFu;
        const uint32_t k = S - j;
        rank += (uint64_t)binom[k * kNB + (L - 1 - prev)] - (uint64_t)binom[k * kNB + (L - c)];
        prev = c;
    }
    q.best[0] = T;
    q.best[1] = q.in_row[pos];
    q.best[2] = rank;
}

// Roots of a piece of rows: level-0 nodes with no cut.
template <int S>
__global__ __launch_bounds__(kBlock) void search_root_kernel(SearchParams q, uint32_t first_row, uint32_t n) {
    const uint32_t i = blockIdx.x * kBlock + threadIdx.x;
    if (i >= n) return;
    q.out_row[i] = first_row + i;
#pragma unroll
    for (int k = 0; k < Codes<S>::kWords; ++k) q.out_codes[(uint64_t)k * q.out_cap + i] = 0u;
}

// ---------------------------------------------------------------------------
template <int S, typename R>
hipError_t launch_search_s(int op, const KParams &p, const SearchParams &q, uint32_t grid, size_t lds,
                           hipStream_t st) {
    const dim3 g(grid), b(kBlock);
    switch (op) {
    case kSearchOpCount:
        if (p.has_ar) hipLaunchKernelGGL((search_count_kernel<S, true, false>), g, b, lds, st, p, q);
        else if (p.g_mono_all) hipLaunchKernelGGL((search_count_kernel<S, false, true>), g, b, lds, st, p, q);
        else hipLaunchKernelGGL((search_count_kernel<S, false, false>), g, b, lds, st, p, q);
        break;
    case kSearchOpWrite:
        if (p.has_ar) hipLaunchKernelGGL((search_write_kernel<S, true, false>), g, b, lds, st, p, q);
        else if (p.g_mono_all) hipLaunchKernelGGL((search_write_kernel<S, false, true>), g, b, lds, st, p, q);
        else hipLaunchKernelGGL((search_write_kernel<S, false, false>), g, b, lds, st, p, q);
        break;
    case kSearchOpLeaf: {
        const bool sch = p.sched != 0;
        if (p.has_ar && sch) hipLaunchKernelGGL((search_leaf_kernel<S, true, true>), g, b, lds, st, p, q);
        else if (p.has_ar) hipLaunchKernelGGL((search_leaf_kernel<S, true, false>), g, b, lds, st, p, q);
        else if (sch) hipLaunchKernelGGL((search_leaf_kernel<S, false, true>), g, b, lds, st, p, q);
        else hipLaunchKernelGGL((search_leaf_kernel<S, false, false>), g, b, lds, st, p, q);
        break;
    }
    case kSearchOpMerge: hipLaunchKernelGGL((search_merge_kernel<R>), dim3(1), dim3(64), 0, st, p, q); break;
    case kSearchOpRoot: hipLaunchKernelGGL((search_root_kernel<S>), g, b, 0, st, q, q.root_first, q.n_in); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace pk
