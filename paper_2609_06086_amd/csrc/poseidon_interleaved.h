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

template <int S, int N>
__device__ __forceinline__ void ilv_dp(const KParams &p, const uint32_t (&F)[S], const uint32_t (&B)[S],
                                       uint32_t (&X)[N]) {
    constexpr int DB = IlvDepth<N>::kB;
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
    for (uint32_t k = 0; k < p.nslots; ++k) {
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
