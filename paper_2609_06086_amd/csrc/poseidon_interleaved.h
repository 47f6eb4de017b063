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

// ---------------------------------------------------------------------------
// Registers live at a period boundary: read by a later node before they are
// written again, in the next period or in the cool-down.  X[q] always is; a
// shift-register entry at position e of stage j is when a node reads depth
// d of that stage's queue after w writes to it with d - 1 - w = e.  The
// live registers, packed in a fixed order (X, then the forward queues
// stage by stage, then the backward queues), are the whole state the rest
// of the DP depends on: the steady-state check compares them between two
// periods and the straggler queue stores them.  Every register is written
// in every period (each stage runs N >= 2 forwards and N >= depth
// backwards per period), so once the live registers rise by the same d
// over one period, every later period does the same.
// ---------------------------------------------------------------------------
template <int N, int V>
struct IlvLive {
    static constexpr int S = N * V, DB = IlvDepth<N>::kB;
    int f[2][S] = {};   // word of Fq0[j] / Fq1[j] in the packed state, or -1
    int b[DB][S] = {};  // word of Bq[e][j], or -1
    int n = 0;          // live words
};

template <int N, int V>
constexpr IlvLive<N, V> ilv_live() {
    constexpr int S = N * V, DB = IlvDepth<N>::kB;
    constexpr const IlvPattern<N, V> &pat = IlvConst<N, V>::kPat;
    bool lf[2][S] = {}, lb[DB][S] = {};
    for (int sec = 1; sec <= 2; ++sec) {
        const int ns = sec == 1 ? 2 * N * V : pat.tail;
        int wf[S] = {}, wb[S] = {};
        for (int t = 0; t < ns; ++t) {
            // a slot reads before it writes (synchronous update)
            for (int q = 0; q < N; ++q) {
                const int kd = pat.kind[sec][t][q], j = pat.chunk[sec][t][q] * N + q, d = pat.depth[sec][t][q];
                if (kd == 0 && j > 0 && d - 1 - wf[j - 1] >= 0) lf[d - 1 - wf[j - 1]][j - 1] = true;
                if (kd == 1 && j < S - 1 && d - 1 - wb[j + 1] >= 0) lb[d - 1 - wb[j + 1]][j + 1] = true;
            }
            for (int q = 0; q < N; ++q) {
                const int kd = pat.kind[sec][t][q], j = pat.chunk[sec][t][q] * N + q;
                if (kd == 0) ++wf[j];
                if (kd == 1) ++wb[j];
            }
        }
    }
    IlvLive<N, V> r{};
    r.n = N;
    for (int j = 0; j < S; ++j)
        for (int e = 0; e < 2; ++e) r.f[e][j] = lf[e][j] ? r.n++ : -1;
    for (int e = 0; e < DB; ++e)
        for (int j = 0; j < S; ++j) r.b[e][j] = lb[e][j] ? r.n++ : -1;
    return r;
}

template <int N, int V>
struct IlvLiveConst {
    static constexpr IlvLive<N, V> kLive = ilv_live<N, V>();
};

// Apply `fn` to every live register with its packed word index W
// (fn.template at<W>(reg); W < 0 marks a dead register).
template <int S, int N, int E, typename Fn, int... J>
__device__ __forceinline__ void ilv_live_bwd(std::integer_sequence<int, J...>, uint32_t (&Bq)[IlvDepth<N>::kB][S],
                                             Fn &fn) {
    constexpr const IlvLive<N, S / N> &lv = IlvLiveConst<N, S / N>::kLive;
    (fn.template at<lv.b[E][J]>(Bq[E][J]), ...);
}

template <int S, int N, typename Fn, int... E>
__device__ __forceinline__ void ilv_live_bwd_all(std::integer_sequence<int, E...>,
                                                 uint32_t (&Bq)[IlvDepth<N>::kB][S], Fn &fn) {
    (ilv_live_bwd<S, N, E>(std::make_integer_sequence<int, S>{}, Bq, fn), ...);
}

template <int S, int N, typename Fn, int... J>
__device__ __forceinline__ void ilv_live_fwd(std::integer_sequence<int, J...>, uint32_t (&Fq0)[S], uint32_t (&Fq1)[S],
                                             Fn &fn) {
    constexpr const IlvLive<N, S / N> &lv = IlvLiveConst<N, S / N>::kLive;
    (fn.template at<lv.f[0][J]>(Fq0[J]), ...);
    (fn.template at<lv.f[1][J]>(Fq1[J]), ...);
}

template <int S, int N, typename Fn, int... Q>
__device__ __forceinline__ void ilv_live_x(std::integer_sequence<int, Q...>, uint32_t (&X)[N], Fn &fn) {
    (fn.template at<Q>(X[Q]), ...);
}

template <int S, int N, typename Fn>
__device__ __forceinline__ void ilv_each_live(uint32_t (&X)[N], uint32_t (&Fq0)[S], uint32_t (&Fq1)[S],
                                              uint32_t (&Bq)[IlvDepth<N>::kB][S], Fn &fn) {
    ilv_live_x<S, N>(std::make_integer_sequence<int, N>{}, X, fn);
    ilv_live_fwd<S, N>(std::make_integer_sequence<int, S>{}, Fq0, Fq1, fn);
    ilv_live_bwd_all<S, N>(std::make_integer_sequence<int, IlvDepth<N>::kB>{}, Bq, fn);
}

template <int NL>
struct IlvPack {      // registers -> packed words
    uint32_t (&w)[NL];
    template <int W> __device__ __forceinline__ void at(uint32_t &r) { if constexpr (W >= 0) w[W] = r; }
};
template <int NL>
struct IlvUnpack {    // packed words -> registers
    const uint32_t (&w)[NL];
    template <int W> __device__ __forceinline__ void at(uint32_t &r) { if constexpr (W >= 0) r = w[W]; }
};
template <int NL>
struct IlvSame {      // does every live register exceed its old value by d?
    const uint32_t (&old)[NL];
    uint32_t d;
    bool ok;
    template <int W> __device__ __forceinline__ void at(uint32_t &r) { if constexpr (W >= 0) ok = ok && r - old[W] == d; }
};
struct IlvShift {     // add a constant to every live register
    uint32_t v;
    template <int W> __device__ __forceinline__ void at(uint32_t &r) { if constexpr (W >= 0) r += v; }
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

template <int S, int N>
__device__ __forceinline__ void ilv_init(uint32_t (&X)[N], uint32_t (&Fq0)[S], uint32_t (&Fq1)[S],
                                         uint32_t (&Bq)[IlvDepth<N>::kB][S]) {
#pragma unroll
    for (int q = 0; q < N; ++q) X[q] = 0;
#pragma unroll
    for (int j = 0; j < S; ++j) {
        Fq0[j] = 0;
        Fq1[j] = 0;
#pragma unroll
        for (int d = 0; d < IlvDepth<N>::kB; ++d) Bq[d][j] = 0;
    }
}

// n steady periods of the compiled schedule
template <int S, int N>
__device__ __forceinline__ void ilv_periods(const KParams &p, uint32_t n, const uint32_t (&F)[S],
                                            const uint32_t (&B)[S], uint32_t (&X)[N], uint32_t (&Fq0)[S],
                                            uint32_t (&Fq1)[S], uint32_t (&Bq)[IlvDepth<N>::kB][S]) {
    for (uint32_t t = 0; t < n; ++t)
        ilv_section_ct<S, N, 1>(std::make_integer_sequence<int, 2 * S>{}, p, F, B, X, Fq0, Fq1, Bq);
}

// Periods k0+1 .. k1 of `trips` (k0 < k1).  With k1 < trips the live
// registers after period k1 are compared with those after period k1 - 1;
// if all rose by the same d, the period map (built from max and + only)
// will raise them by d every time, so they jump to the end of the periods
// at once.  Returns whether the lane is at the end of the periods.
template <int S, int N>
__device__ __forceinline__ bool ilv_advance(const KParams &p, const uint32_t (&F)[S], const uint32_t (&B)[S],
                                            uint32_t (&X)[N], uint32_t (&Fq0)[S], uint32_t (&Fq1)[S],
                                            uint32_t (&Bq)[IlvDepth<N>::kB][S], uint32_t k0, uint32_t k1,
                                            uint32_t trips) {
    if (k1 >= trips) {
        ilv_periods<S, N>(p, trips - k0, F, B, X, Fq0, Fq1, Bq);
        return true;
    }
    ilv_periods<S, N>(p, k1 - k0 - 1, F, B, X, Fq0, Fq1, Bq);
    constexpr int NL = IlvLiveConst<N, S / N>::kLive.n;
    uint32_t old[NL];
    IlvPack<NL> pack{old};
    ilv_each_live<S, N>(X, Fq0, Fq1, Bq, pack);
    ilv_section_ct<S, N, 1>(std::make_integer_sequence<int, 2 * S>{}, p, F, B, X, Fq0, Fq1, Bq);
    IlvSame<NL> same{old, X[0] - old[0], true};
    ilv_each_live<S, N>(X, Fq0, Fq1, Bq, same);
    IlvShift jump{same.ok ? (trips - k1) * same.d : 0u};
    ilv_each_live<S, N>(X, Fq0, Fq1, Bq, jump);
    return same.ok;
}

// Stage types, weights and per-device memory check of one candidate.
template <int S, int N>
__device__ __forceinline__ bool ilv_weights(const KParams &p, const Lds &tab, const uint32_t (&cut)[S + 1],
                                            uint32_t a, uint32_t (&tyd)[N], uint32_t (&F)[S], uint32_t (&B)[S]) {
    constexpr int V = S / N;
    uint32_t ty[S];
    decode_types<N>(p, a, tyd);
#pragma unroll
    for (int j = 0; j < S; ++j) ty[j] = tyd[j % N];
    stage_weights<S>(p, tab, cut, ty, F, B);
    // a device fits when all its chunks' layers fit its memory
    bool feas = true;
#pragma unroll
    for (int q = 0; q < N; ++q) {
        uint32_t mem = 0;
#pragma unroll
        for (int c = 0; c < V; ++c) mem += tab.pm[cut[c * N + q + 1]] - tab.pm[cut[c * N + q]];
        feas = feas && mem <= tab.cap[tyd[q]];
    }
    return feas;
}

// T: the end node follows every device's all-reduce node
template <int S, int N, bool AR>
__device__ __forceinline__ uint32_t ilv_end(const KParams &p, const Lds &tab, const uint32_t (&X)[N],
                                            const uint32_t (&cut)[S + 1], const uint32_t (&tyd)[N]) {
    constexpr int V = S / N;
    const uint32_t row = p.L + 1;
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
    return T;
}

// (a2)-(a4), (a6) under Interleaved 1F1B.  Compiled form (TAB = false, used
// when p.ilv_compiled, which the host sets after checking the compiled
// schedule against the problem's own slot table): prologue, periods and
// cool-down as straight-line code; with a cascade (p.nlevels > 0) a lane
// whose live registers have not settled by period p.lvl_k[0] is queued for
// ilv_resume_kernel.  TAB = true: the host's slot table drives the same
// update (a separate instance, so that its registers do not weigh on the
// compiled one).  X[q] ends as device q's last finish.
template <int S, int N, bool AR, bool TAB>
__global__ __launch_bounds__(kBlock) void ilv_kernel(KParams p) {
    extern __shared__ __align__(16) unsigned char smem[];
    const Lds tab = stage_tables(p, smem);
    constexpr int NW = Codes<S>::kWords, DB = IlvDepth<N>::kB;
    constexpr const IlvPattern<N, S / N> &pat = IlvConst<N, S / N>::kPat;
    unsigned long long best = ~0ull;
    // 32-bit positions: a chunk holds at most 2^26 candidates, a call fewer than 2^32
    const uint32_t stride = gridDim.x * kBlock, n_i = (uint32_t)p.n_i, ccap = (uint32_t)p.ccap;
    const uint32_t first_i = (uint32_t)p.first_i;
    const uint32_t span = (n_i + stride - 1) / stride;
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
        uint32_t cut[S + 1], tyd[N], F[S], B[S], X[N], Fq0[S], Fq1[S], Bq[DB][S];
        const bool ok = unpack_cuts<S>(w, p.L, cut);
        const uint32_t a = ok ? assign_of(p, gi) : 0u;
        const bool feas = ilv_weights<S, N>(p, tab, cut, a, tyd, F, B) && ok && active;
        ilv_init<S, N>(X, Fq0, Fq1, Bq);
        bool done_here = true;
        if constexpr (!TAB && pat.start >= 0) {
            ilv_section_ct<S, N, 0>(std::make_integer_sequence<int, (pat.start > 0 ? pat.start : 0)>{}, p, F, B, X,
                                    Fq0, Fq1, Bq);
            const uint32_t k1 = p.nlevels ? p.lvl_k[0] : p.ilv_trips;
            done_here = ilv_advance<S, N>(p, F, B, X, Fq0, Fq1, Bq, 0, k1, p.ilv_trips);
            if (p.nlevels) {
                constexpr int NL = IlvLiveConst<N, S / N>::kLive.n;
                uint32_t Z[NL];
                IlvPack<NL> pack{Z};
                ilv_each_live<S, N>(X, Fq0, Fq1, Bq, pack);
                enqueue<S, NL>(p, 0, &nq, !done_here && active && ok, gi, w, -1, Z);
            }
            ilv_section_ct<S, N, 2>(std::make_integer_sequence<int, pat.tail>{}, p, F, B, X, Fq0, Fq1, Bq);
        } else {
            ilv_table_slots<S, N>(p, 0, p.nslots, F, B, X, Fq0, Fq1, Bq);
        }
        uint32_t T = ilv_end<S, N, AR>(p, tab, X, cut, tyd);
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
    if (p.nlevels) {
        __syncthreads();
        if (threadIdx.x == 0) p.qcount[blockIdx.x] = nq;   // entries for level 1
    }
    block_min_and_finish(best, p.acc, p.done, p.result, nullptr, p.nlevels == 0, p.accumulate);
}

// Level `lvl` of the Interleaved 1F1B cascade: resume the queued lanes from
// period p.lvl_k[lvl-1] to p.lvl_k[lvl] (the end at the last level), then
// run the cool-down (only compiled schedules have a cascade).
template <int S, int N, bool AR>
__global__ __launch_bounds__(kBlock) void ilv_resume_kernel(KParams p, uint32_t lvl) {
    extern __shared__ __align__(16) unsigned char smem[];
    const Lds tab = stage_tables(p, smem);
    constexpr int NW = Codes<S>::kWords, DB = IlvDepth<N>::kB;
    constexpr const IlvPattern<N, S / N> &pat = IlvConst<N, S / N>::kPat;
    constexpr int NL = IlvLiveConst<N, S / N>::kLive.n;
    const uint32_t trips = p.ilv_trips;
    const uint32_t k0 = p.lvl_k[lvl - 1];
    const uint32_t k1 = lvl < p.nlevels ? p.lvl_k[lvl] : trips;
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
        uint32_t w[NW], Z[NL], cut[S + 1], tyd[N], F[S], B[S], X[N], Fq0[S], Fq1[S], Bq[DB][S];
#pragma unroll
        for (int k = 0; k < NW; ++k) w[k] = active ? qin.codes[k * qcap + q] : 0u;
#pragma unroll
        for (int s = 0; s < NL; ++s) Z[s] = active ? qin.Y[s * qcap + q] : 0u;
        unpack_cuts<S>(w, p.L, cut);   // (a queued entry's codes were valid when it was queued)
        const uint32_t a = !active ? 0u : p.qasg ? qin.asg[q] : assign_of(p, i);
        const bool feas = ilv_weights<S, N>(p, tab, cut, a, tyd, F, B);
        // dead registers are written before any read, so zero is as good as any value
        ilv_init<S, N>(X, Fq0, Fq1, Bq);
        IlvUnpack<NL> unpack{Z};
        ilv_each_live<S, N>(X, Fq0, Fq1, Bq, unpack);
        bool settled = true;
        if constexpr (pat.start >= 0) {
            settled = ilv_advance<S, N>(p, F, B, X, Fq0, Fq1, Bq, k0, k1, trips);
            if (lvl < p.nlevels) {
                IlvPack<NL> pack{Z};
                ilv_each_live<S, N>(X, Fq0, Fq1, Bq, pack);
                enqueue<S, NL>(p, lvl & 1, &nq, active && !settled, i, w, a, Z);
            }
            ilv_section_ct<S, N, 2>(std::make_integer_sequence<int, pat.tail>{}, p, F, B, X, Fq0, Fq1, Bq);
        }
        const uint32_t T = ilv_end<S, N, AR>(p, tab, X, cut, tyd);
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

}  // namespace pk
