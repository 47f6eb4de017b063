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

hipError_t launch_ilv(const KParams &p, const LaunchCfg &lc, hipStream_t st) {
    const dim3 g(lc.grid), b(kBlock);
#define PK_ILV_LAUNCH(S_, N_)                                                                              \
    if (p.S == S_ && p.ndev == N_) {                                                                   \
        if (p.has_ar) hipLaunchKernelGGL((ilv_kernel<S_, N_, true>), g, b, lc.lds_bytes, st, p);        \
        else hipLaunchKernelGGL((ilv_kernel<S_, N_, false>), g, b, lc.lds_bytes, st, p);                \
        return hipGetLastError();                                                                      \
    }
    PK_ILV_PAIRS(PK_ILV_LAUNCH)
#undef PK_ILV_LAUNCH
    return hipErrorInvalidValue;
}

hipError_t ilv_occupancy(const KParams &p, size_t lds, int *blocks) {
#define PK_ILV_OCC(S_, N_)                                                                                  \
    if (p.S == S_ && p.ndev == N_)                                                                     \
        return p.has_ar ? hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks, ilv_kernel<S_, N_, true>, kBlock, lds) \
                        : hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks, ilv_kernel<S_, N_, false>, kBlock, lds);
    PK_ILV_PAIRS(PK_ILV_OCC)
#undef PK_ILV_OCC
    return hipErrorInvalidValue;
}

}  // namespace pk
