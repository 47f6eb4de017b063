// Kernel instantiations for stage counts 1, 2, 3, 4, 5, 6, 7, 8 (split so that the library
// compiles in parallel).
#include "poseidon_search.h"

namespace pk {

#define PK_INST(S)                                                                                        \
    template hipError_t launch_eval_s<S, uint32_t>(const KParams &, const LaunchCfg &, hipStream_t);           \
    template hipError_t launch_eval_s<S, uint64_t>(const KParams &, const LaunchCfg &, hipStream_t);           \
    template hipError_t launch_decode_s<S, uint32_t>(const KParams &, const LaunchCfg &, hipStream_t);         \
    template hipError_t launch_decode_s<S, uint64_t>(const KParams &, const LaunchCfg &, hipStream_t);         \
    template hipError_t launch_resume_s<S, uint32_t>(const KParams &, const LaunchCfg &, hipStream_t, uint32_t); \
    template hipError_t launch_resume_s<S, uint64_t>(const KParams &, const LaunchCfg &, hipStream_t, uint32_t); \
    template hipError_t launch_bounded_s<S, uint32_t>(const KParams &, const LaunchCfg &, hipStream_t,          \
                                                       uint32_t);                                              \
    template hipError_t launch_bounded_s<S, uint64_t>(const KParams &, const LaunchCfg &, hipStream_t,          \
                                                       uint32_t);                                              \
    template hipError_t occupancy_s<S, uint32_t>(int *, size_t, bool, bool);                                        \
    template hipError_t occupancy_s<S, uint64_t>(int *, size_t, bool, bool);                                        \
    template hipError_t launch_search_s<S, uint32_t>(int, const KParams &, const SearchParams &, uint32_t, size_t,  \
                                                      hipStream_t);                                                 \
    template hipError_t launch_search_s<S, uint64_t>(int, const KParams &, const SearchParams &, uint32_t, size_t,  \
                                                      hipStream_t);

PK_INST(1) PK_INST(2) PK_INST(3) PK_INST(4) PK_INST(5) PK_INST(6) PK_INST(7) PK_INST(8)

}  // namespace pk
