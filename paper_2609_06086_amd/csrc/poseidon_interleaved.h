#pragma once
// Interleaved 1F1B (Sec. 4.1.4) as a register stencil.  The S virtual
// stages sit on N devices, V = S / N chunks each; virtual stage j runs on
// device j mod N.  Under unit weights every device runs at most one node
// per slot (its nodes are sequential), so one register per device holds
// its newest node.  A device can run ahead of its neighbours, so a forward
// reads one of the upstream stage's two newest forwards and a backward one
// of the downstream stage's newest backwards, up to ilv_max_db(N) deep
// (checked on the host for every problem): each virtual stage keeps short
// shift registers of its newest forwards and backwards.  The host's slot
// table gives, per slot, the stages that run a forward (and which read the
// second-newest upstream forward), those that run a backward, and each
// backward's input depth (2 bits per stage).  N is a template parameter so
// that the device of every stage, j mod N, is a compile-time register.
#include "poseidon_kernels.h"

namespace pk {

template <int N>
struct IlvDepth {
    static constexpr int kB = N >= 7 ? 4 : (N >= 5 ? 3 : 2);   // backward shift-register depth
};

// ---------------------------------------------------------------------------
// The periodic steady part, at compile time.  After a prologue that depends
// only on (N, V), the slot schedule repeats with period P = 2NV slots
// (every device alternates a forward and a backward; the chunk pattern
// repeats every NV steps) until the cool-down.  ilv_pattern<N, V>()
// simulates the unit-weight schedule for a reference M0 in a constant
// expression and returns one period: for every slot of the period and every
// device, the kind, chunk and input depth of its node, and the slot at which
// the period starts.  The host checks, for the problem's own M, that its
// slot table repeats exactly this period from that slot on, and the kernel
// runs those slots as straight-line code with every register index fixed.
// ---------------------------------------------------------------------------
template <int N, int V>
struct IlvPattern {
    static constexpr int kP = 2 * N * V, kMax = 4 * N * V;
    int start = -1;                 // prologue slots (-1: no compiled form)
    int tail = 0;                   // cool-down slots after the last period
    // section 0 = prologue, 1 = one period, 2 = cool-down; per slot and
    // device: kind (0 forward, 1 backward, 255 idle), chunk, input depth
    // (1 = newest; 0 = no cross-stage input)
    unsigned char kind[3][kMax][N] = {};
    unsigned char chunk[3][kMax][N] = {};
    unsigned char depth[3][kMax][N] = {};
};

template <int N, int V>
constexpr IlvPattern<N, V> ilv_pattern() {
    constexpr int S = N * V, M0 = N * (V + 6), P = 2 * N * V, LEN = 2 * V * M0;
    constexpr int NMAX = 2 * S * M0 + 4 * S + 8;
    int kind[N][LEN] = {}, stg[N][LEN] = {}, mbat[N][LEN] = {};
    for (int q = 0; q < N; ++q) {
        const int total = V * M0;
        int w = 2 * (N - q - 1) + (V - 1) * N;
        w = w < total ? w : total;
        int k = 0;
        for (int x = 0; x < w; ++x, ++k) {
            kind[q][k] = 0; stg[q][k] = ((x % (N * V)) / N) * N + q; mbat[q][k] = (x / (N * V)) * N + x % N + 1;
        }
        for (int i = 0; i < total - w; ++i) {
            const int x = w + i;
            kind[q][k] = 0; stg[q][k] = ((x % (N * V)) / N) * N + q; mbat[q][k] = (x / (N * V)) * N + x % N + 1; ++k;
            kind[q][k] = 1; stg[q][k] = (V - 1 - (i % (N * V)) / N) * N + q; mbat[q][k] = (i / (N * V)) * N + i % N + 1; ++k;
        }
        for (int x = total - w; x < total; ++x, ++k) {
            kind[q][k] = 1; stg[q][k] = (V - 1 - (x % (N * V)) / N) * N + q; mbat[q][k] = (x / (N * V)) * N + x % N + 1;
        }
    }
    // as-soon-as-possible start slots with unit weights
    int st[2][S][M0 + 1] = {};
    for (int a = 0; a < 2; ++a)
        for (int j = 0; j < S; ++j)
            for (int m = 0; m <= M0; ++m) st[a][j][m] = -1;
    int pos[N] = {}, freeat[N] = {};
    int placed = 0, nslot = 0;
    while (placed < 2 * S * M0) {
        bool progress = false;
        for (int q = 0; q < N; ++q) {
            while (pos[q] < LEN) {
                const int kd = kind[q][pos[q]], j = stg[q][pos[q]], m = mbat[q][pos[q]];
                int dep = 0;
                if (kd == 0 && j > 0) dep = st[0][j - 1][m] < 0 ? -1 : st[0][j - 1][m] + 1;
                if (kd == 1 && j < S - 1) dep = st[1][j + 1][m] < 0 ? -1 : st[1][j + 1][m] + 1;
                if (dep < 0) break;
                const int t = freeat[q] > dep ? freeat[q] : dep;
                st[kd][j][m] = t;
                freeat[q] = t + 1;
                nslot = nslot > t + 1 ? nslot : t + 1;
                ++pos[q];
                ++placed;
                progress = true;
            }
        }
        if (!progress) return IlvPattern<N, V>{};
    }
    // per slot and device: kind, chunk, depth (255 = idle)
    unsigned char tk[NMAX][N] = {}, tc[NMAX][N] = {}, td[NMAX][N] = {};
    for (int t = 0; t < NMAX; ++t)
        for (int q = 0; q < N; ++q) tk[t][q] = 255;
    for (int a = 0; a < 2; ++a)
        for (int j = 0; j < S; ++j)
            for (int m = 1; m <= M0; ++m) {
                const int t = st[a][j][m], q = j % N;
                int d = 0;
                const int u = a == 0 ? j - 1 : j + 1;
                if (u >= 0 && u < S) {
                    d = 1;
                    for (int mm = 1; mm <= M0; ++mm)
                        d += st[a][u][mm] > st[a][u][m] && st[a][u][mm] < t;
                }
                tk[t][q] = (unsigned char)a;
                tc[t][q] = (unsigned char)(j / N);
                td[t][q] = (unsigned char)d;
            }
    // the first slot from which two consecutive periods agree, the periods
    // that follow, and the cool-down after the last one
    IlvPattern<N, V> r{};
    for (int a = 0; a + 2 * P <= nslot; ++a) {
        bool same = true;
        for (int t = a; t < a + P && same; ++t)
            for (int q = 0; q < N; ++q)
                same = same && tk[t][q] != 255 && tk[t][q] == tk[t + P][q] && tc[t][q] == tc[t + P][q] &&
                       td[t][q] == td[t + P][q];
        if (!same) continue;
        int trips = 1;
        for (bool more = true; more && a + (trips + 1) * P <= nslot;) {
            for (int t = a; t < a + P && more; ++t)
                for (int q = 0; q < N; ++q)
                    more = more && tk[t][q] == tk[t + trips * P][q] && tc[t][q] == tc[t + trips * P][q] &&
                           td[t][q] == td[t + trips * P][q];
            if (more) ++trips;
        }
        const int tail0 = a + trips * P, E = nslot - tail0;
        if (a > IlvPattern<N, V>::kMax || E > IlvPattern<N, V>::kMax) return r;
        r.start = a;
        r.tail = E;
        for (int q = 0; q < N; ++q) {
            for (int t = 0; t < a; ++t) {
                r.kind[0][t][q] = tk[t][q]; r.chunk[0][t][q] = tc[t][q]; r.depth[0][t][q] = td[t][q];
            }
            for (int t = 0; t < P; ++t) {
                r.kind[1][t][q] = tk[a + t][q]; r.chunk[1][t][q] = tc[a + t][q]; r.depth[1][t][q] = td[a + t][q];
            }
            for (int t = 0; t < E; ++t) {
                r.kind[2][t][q] = tk[tail0 + t][q]; r.chunk[2][t][q] = tc[tail0 + t][q];
                r.depth[2][t][q] = td[tail0 + t][q];
            }
        }
        return r;
    }
    return r;
}

template <int N, int V>
struct IlvConst {
    static constexpr IlvPattern<N, V> kPat = ilv_pattern<N, V>();
};

// Slots [k0, k1) of the host's slot table (prologue and cool-down).
template <int S, int N>
__device__ __forceinline__ void ilv_table_slots(const KParams &p, uint32_t k0, uint32_t k1, const uint32_t (&F)[S],
                                                const uint32_t (&B)[S], uint32_t (&X)[N], uint32_t (&Fq0)[S],
                                                uint32_t (&Fq1)[S], uint32_t (&Bq)[IlvDepth<N>::kB][S]) {
    constexpr int DB = IlvDepth<N>::kB;
    for (uint32_t k = k0; k < k1; ++k) {
        const uint32_t fm = p.slot_mask[4 * k], fd = p.slot_mask[4 * k + 1];
        const uint32_t bm = p.slot_mask[4 * k + 2], bd = p.slot_mask[4 * k + 3];
        uint32_t nv[S];
#pragma unroll
        for (int j = 0; j < S; ++j) {
            const int q = j % N;
            nv[j] = 0;
            if ((fm >> j) & 1u) {
                uint32_t in = 0;
                if (j > 0) in = (((fd >> j) & 1u) ? Fq1[j > 0 ? j - 1 : 0] : Fq0[j > 0 ? j - 1 : 0]) + p.cf[j > 0 ? j - 1 : 0];
                nv[j] = F[j] + max(X[q], in);
            } else if ((bm >> j) & 1u) {
                uint32_t in = 0;
                if (j < S - 1) {
                    const uint32_t d = (bd >> (2 * j)) & 3u;
                    const int u = j < S - 1 ? j + 1 : 0;
                    uint32_t b = Bq[0][u];
#pragma unroll
                    for (int e = 1; e < DB; ++e) b = d == (uint32_t)e ? Bq[e][u] : b;
                    in = b + p.cb[j < S - 1 ? j : 0];
                }
                nv[j] = B[j] + max(X[q], in);
            }
        }
#pragma unroll
        for (int j = 0; j < S; ++j) {
            const int q = j % N;
            if ((fm >> j) & 1u) {
                Fq1[j] = Fq0[j];
                Fq0[j] = nv[j];
                X[q] = nv[j];
            } else if ((bm >> j) & 1u) {
#pragma unroll
                for (int e = DB - 1; e > 0; --e) Bq[e][j] = Bq[e - 1][j];
                Bq[0][j] = nv[j];
                X[q] = nv[j];
            }
        }
    }
}

// Node of device q in slot T of section SEC (every index a constant).
template <int S, int N, int SEC, int T, int q>
__device__ __forceinline__ uint32_t ilv_node_ct(const KParams &p, const uint32_t (&F)[S], const uint32_t (&B)[S],
                                                const uint32_t (&X)[N], const uint32_t (&Fq0)[S],
                                                const uint32_t (&Fq1)[S], const uint32_t (&Bq)[IlvDepth<N>::kB][S]) {
    constexpr int V = S / N;
    constexpr int kd = IlvConst<N, V>::kPat.kind[SEC][T][q];
    constexpr int j = IlvConst<N, V>::kPat.chunk[SEC][T][q] * N + q;
    constexpr int d = IlvConst<N, V>::kPat.depth[SEC][T][q];
    if constexpr (kd == 0) {
        if constexpr (j > 0) return F[j] + max(X[q], (d == 2 ? Fq1[j - 1] : Fq0[j - 1]) + p.cf[j - 1]);
        else return F[j] + X[q];
    } else if constexpr (kd == 1) {
        if constexpr (j < S - 1) return B[j] + max(X[q], Bq[d - 1][j + 1] + p.cb[j]);
        else return B[j] + X[q];
    } else {
        return X[q];
    }
}

template <int S, int N, int SEC, int T, int q>
__device__ __forceinline__ void ilv_commit_ct(uint32_t v, uint32_t (&X)[N], uint32_t (&Fq0)[S], uint32_t (&Fq1)[S],
                                              uint32_t (&Bq)[IlvDepth<N>::kB][S]) {
    constexpr int V = S / N, DB = IlvDepth<N>::kB;
    constexpr int kd = IlvConst<N, V>::kPat.kind[SEC][T][q];
    constexpr int j = IlvConst<N, V>::kPat.chunk[SEC][T][q] * N + q;
    if constexpr (kd == 0) {
        Fq1[j] = Fq0[j];
        Fq0[j] = v;
        X[q] = v;
    } else if constexpr (kd == 1) {
#pragma unroll
        for (int e = DB - 1; e > 0; --e) Bq[e][j] = Bq[e - 1][j];
        Bq[0][j] = v;
        X[q] = v;
    }
}

template <int S, int N, int SEC, int T, int... Q>
__device__ __forceinline__ void ilv_slot_ct(std::integer_sequence<int, Q...>, const KParams &p,
                                            const uint32_t (&F)[S], const uint32_t (&B)[S], uint32_t (&X)[N],
                                            uint32_t (&Fq0)[S], uint32_t (&Fq1)[S],
                                            uint32_t (&Bq)[IlvDepth<N>::kB][S]) {
    const uint32_t nv[N] = {ilv_node_ct<S, N, SEC, T, Q>(p, F, B, X, Fq0, Fq1, Bq)...};
    (ilv_commit_ct<S, N, SEC, T, Q>(nv[Q], X, Fq0, Fq1, Bq), ...);
}

template <int S, int N, int SEC, int... T>
__device__ __forceinline__ void ilv_section_ct(std::integer_sequence<int, T...>, const KParams &p,
                                               const uint32_t (&F)[S], const uint32_t (&B)[S], uint32_t (&X)[N],
                                               uint32_t (&Fq0)[S], uint32_t (&Fq1)[S],
                                               uint32_t (&Bq)[IlvDepth<N>::kB][S]) {
    (ilv_slot_ct<S, N, SEC, T>(std::make_integer_sequence<int, N>{}, p, F, B, X, Fq0, Fq1, Bq), ...);
}

// The whole DP.  Compiled form (p.ilv_trips > 0 or a schedule made only of
// prologue and cool-down, checked by the host against the problem's own
// table): prologue, `trips` periods and the cool-down as straight-line code.
// Otherwise the host's slot table drives the same update.  After it X[q] is
// the finish of device q's last node.
template <int S, int N>
__device__ __forceinline__ void ilv_dp(const KParams &p, const uint32_t (&F)[S], const uint32_t (&B)[S],
                                       uint32_t (&X)[N]) {
    constexpr int DB = IlvDepth<N>::kB, P = 2 * S;
    constexpr IlvPattern<N, S / N> const &pat = IlvConst<N, S / N>::kPat;
    uint32_t Fq0[S], Fq1[S], Bq[DB][S];
#pragma unroll
    for (int q = 0; q < N; ++q) X[q] = 0;
#pragma unroll
    for (int j = 0; j < S; ++j) {
        Fq0[j] = 0;
        Fq1[j] = 0;
#pragma unroll
        for (int d = 0; d < DB; ++d) Bq[d][j] = 0;
    }
    if constexpr (pat.start >= 0) {
        if (p.ilv_compiled) {
            ilv_section_ct<S, N, 0>(std::make_integer_sequence<int, (pat.start > 0 ? pat.start : 0)>{}, p, F, B, X,
                                    Fq0, Fq1, Bq);
            for (uint32_t t = 0; t < p.ilv_trips; ++t)
                ilv_section_ct<S, N, 1>(std::make_integer_sequence<int, P>{}, p, F, B, X, Fq0, Fq1, Bq);
            ilv_section_ct<S, N, 2>(std::make_integer_sequence<int, pat.tail>{}, p, F, B, X, Fq0, Fq1, Bq);
            return;
        }
    }
    ilv_table_slots<S, N>(p, 0, p.nslots, F, B, X, Fq0, Fq1, Bq);
}

template <int S, int N, bool AR>
__global__ __launch_bounds__(kBlock) void ilv_kernel(KParams p) {
    extern __shared__ __align__(16) unsigned char smem[];
    const Lds tab = stage_tables(p, smem);
    constexpr int NW = Codes<S>::kWords;
    constexpr int V = S / N;
    unsigned long long best = ~0ull;
    const uint64_t stride = (uint64_t)gridDim.x * kBlock;
    const uint64_t span = (p.n_i + stride - 1) / stride;
    const uint32_t row = p.L + 1;
    uint64_t i = (uint64_t)blockIdx.x * kBlock + threadIdx.x;
    for (uint64_t it = 0; it < span; ++it, i += stride) {
        const bool active = i < p.n_i;
        const uint64_t gi = p.first_i + i;
        uint32_t w[NW];
#pragma unroll
        for (int k = 0; k < NW; ++k) w[k] = active ? p.codes[(uint64_t)k * p.ccap + i] : 0u;
        uint32_t cut[S + 1], tyd[N], ty[S], F[S], B[S], X[N];
        const bool ok = unpack_cuts<S>(w, p.L, cut);
        const uint32_t a = ok ? assign_of(p, gi) : 0u;
        decode_types<N>(p, a, tyd);
#pragma unroll
        for (int j = 0; j < S; ++j) ty[j] = tyd[j % N];
        stage_weights<S>(p, tab, cut, ty, F, B);
        // a device fits when all its chunks' layers fit its memory
        bool feas = ok && active;
#pragma unroll
        for (int q = 0; q < N; ++q) {
            uint32_t mem = 0;
#pragma unroll
            for (int c = 0; c < V; ++c) mem += tab.pm[cut[c * N + q + 1]] - tab.pm[cut[c * N + q]];
            feas = feas && mem <= tab.cap[tyd[q]];
        }
        ilv_dp<S, N>(p, F, B, X);
        // the end node follows every device's all-reduce node
        uint32_t T = 0;
#pragma unroll
        for (int q = 0; q < N; ++q) {
            uint32_t d = 0;
            if (AR) {
#pragma unroll
                for (int c = 0; c < V; ++c)
                    d += tab.pd[tyd[q] * row + cut[c * N + q + 1]] - tab.pd[tyd[q] * row + cut[c * N + q]];
            }
            T = max(T, X[q] + d);
        }
        if (!ok) T = 0xFFFFFFFFu;
        if (active && p.makespan_out) p.makespan_out[gi] = T;
        if (p.feas_bits_out) {
            const unsigned long long bits = __ballot(feas);
            const uint64_t w0 = (gi - (threadIdx.x & 63)) >> 5;
            if ((threadIdx.x & 63) == 0 && w0 < p.nwords) p.feas_bits_out[w0] = (uint32_t)bits;
            if ((threadIdx.x & 63) == 32 && w0 + 1 < p.nwords) p.feas_bits_out[w0 + 1] = (uint32_t)(bits >> 32);
        }
        if (active) {
            const unsigned long long key = make_key(feas, T, (uint32_t)gi);
            best = key < best ? key : best;
        }
    }
    block_min_and_finish(best, p.acc, p.done, p.result, nullptr, true, p.accumulate);
}

}  // namespace pk
