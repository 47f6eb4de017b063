// Interleaved 1F1B kernels for every (virtual stages S, devices N) pair
// with V = S / N >= 2 chunks per device and S <= 16, and their dispatch.
#include <hip/hip_runtime.h>

#include "poseidon_interleaved.h"

namespace pk {

#define PK_ILV_PAIRS(X) \
    X(4, 2) X(6, 2) X(6, 3) X(8, 2) X(8, 4) X(9, 3) X(10, 2) X(10, 5) X(12, 2) X(12, 3) X(12, 4) X(12, 6) \
    X(14, 2) X(14, 7) X(15, 3) X(15, 5) X(16, 2) X(16, 4) X(16, 8)

int ilv_max_db(int N) {
    switch (N) {
#define PK_DB_CASE(S_, N_) case N_: return IlvDepth<N_>::kB;
    case 2: return IlvDepth<2>::kB;
    case 3: return IlvDepth<3>::kB;
    case 4: return IlvDepth<4>::kB;
    case 5: return IlvDepth<5>::kB;
    case 6: return IlvDepth<6>::kB;
    case 7: return IlvDepth<7>::kB;
    case 8: return IlvDepth<8>::kB;
#undef PK_DB_CASE
    default: return 0;
    }
}

template <int N, int V>
void section_words(int sec, int n, uint32_t *w) {
    constexpr int S = N * V;
    const IlvPattern<N, V> &pat = IlvConst<N, V>::kPat;
    for (int t = 0; t < n; ++t) {
        uint32_t fm = 0, fd = 0, bm = 0, bd = 0;
        for (int q = 0; q < N; ++q) {
            const int k = pat.kind[sec][t][q], j = pat.chunk[sec][t][q] * N + q, d = pat.depth[sec][t][q];
            if (k == 0) {
                fm |= 1u << j;
                if (d == 2) fd |= 1u << j;
            } else if (k == 1) {
                bm |= 1u << j;
                if (j < S - 1) bd |= (uint32_t)(d - 1) << (2 * j);
            }
        }
        w[4 * t] = fm;
        w[4 * t + 1] = fd;
        w[4 * t + 2] = bm;
        w[4 * t + 3] = bd;
    }
}

template <int N, int V>
bool program_words(int *start, int *tail, uint32_t *pro, uint32_t *period, uint32_t *cool) {
    const IlvPattern<N, V> &pat = IlvConst<N, V>::kPat;
    if (pat.start < 0) return false;
    *start = pat.start;
    *tail = pat.tail;
    section_words<N, V>(0, pat.start, pro);
    section_words<N, V>(1, 2 * N * V, period);
    section_words<N, V>(2, pat.tail, cool);
    return true;
}

bool ilv_program_words(uint32_t S, uint32_t N, int *start, int *tail, uint32_t *pro, uint32_t *period,
                       uint32_t *cool) {
#define PK_ILV_PROG(S_, N_) \
    if (S == S_ && N == N_) return program_words<N_, S_ / N_>(start, tail, pro, period, cool);
    PK_ILV_PAIRS(PK_ILV_PROG)
#undef PK_ILV_PROG
    return false;
}

hipError_t launch_ilv(const KParams &p, const LaunchCfg &lc, hipStream_t st) {
    const dim3 g(lc.grid), b(kBlock);
#define PK_ILV_LAUNCH(S_, N_)                                                                                  \
    if (p.S == S_ && p.ndev == N_) {                                                                       \
        if (p.ilv_compiled) {                                                                              \
            if (p.has_ar) hipLaunchKernelGGL((ilv_kernel<S_, N_, true, false>), g, b, lc.lds_bytes, st, p);  \
            else hipLaunchKernelGGL((ilv_kernel<S_, N_, false, false>), g, b, lc.lds_bytes, st, p);          \
        } else {                                                                                           \
            if (p.has_ar) hipLaunchKernelGGL((ilv_kernel<S_, N_, true, true>), g, b, lc.lds_bytes, st, p);   \
            else hipLaunchKernelGGL((ilv_kernel<S_, N_, false, true>), g, b, lc.lds_bytes, st, p);           \
        }                                                                                                  \
        return hipGetLastError();                                                                          \
    }
    PK_ILV_PAIRS(PK_ILV_LAUNCH)
#undef PK_ILV_LAUNCH
    return hipErrorInvalidValue;
}

hipError_t launch_ilv_resume(const KParams &p, const LaunchCfg &lc, hipStream_t st, uint32_t lvl) {
    const dim3 g(lc.grid), b(kBlock);
#define PK_ILV_RESUME(S_, N_)                                                                                   \
    if (p.S == S_ && p.ndev == N_) {                                                                           \
        if (p.has_ar) hipLaunchKernelGGL((ilv_resume_kernel<S_, N_, true>), g, b, lc.lds_bytes, st, p, lvl);    \
        else hipLaunchKernelGGL((ilv_resume_kernel<S_, N_, false>), g, b, lc.lds_bytes, st, p, lvl);            \
        return hipGetLastError();                                                                              \
    }
    PK_ILV_PAIRS(PK_ILV_RESUME)
#undef PK_ILV_RESUME
    return hipErrorInvalidValue;
}

int ilv_state_words(uint32_t S, uint32_t N) {
#define PK_ILV_WORDS(S_, N_) \
    if (S == S_ && N == N_) return IlvLiveConst<N_, S_ / N_>::kLive.n;
    PK_ILV_PAIRS(PK_ILV_WORDS)
#undef PK_ILV_WORDS
    return 0;
}

hipError_t ilv_occupancy(const KParams &p, size_t lds, int *blocks) {
#define PK_ILV_OCC(S_, N_)                                                                                   \
    if (p.S == S_ && p.ndev == N_) {                                                                    \
        if (p.ilv_compiled)                                                                             \
            return p.has_ar ? hipOccupancyMaxActiveBlocksPerMultiprocessor(                             \
                                  blocks, ilv_kernel<S_, N_, true, false>, kBlock, lds)                 \
                            : hipOccupancyMaxActiveBlocksPerMultiprocessor(                             \
                                  blocks, ilv_kernel<S_, N_, false, false>, kBlock, lds);               \
        return p.has_ar ? hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks, ilv_kernel<S_, N_, true, true>, \
                                                                       kBlock, lds)                     \
                        : hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks, ilv_kernel<S_, N_, false, true>, \
                                                                       kBlock, lds);                    \
    }
    PK_ILV_PAIRS(PK_ILV_OCC)
#undef PK_ILV_OCC
    return hipErrorInvalidValue;
}

}  // namespace pk
