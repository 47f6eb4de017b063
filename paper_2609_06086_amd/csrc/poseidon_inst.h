// Explicit instantiation of the templated kernels for one stage count S:
// every instantiation unit includes this and lists its stage counts, so
// that the library compiles in parallel, one unit per core.
#pragma once
#include "poseidon_search.h"

// (expanded inside namespace pk)
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
    template hipError_t filter_occupancy_s<S, uint32_t>(const KParams &, size_t, int *);                            \
    template hipError_t filter_occupancy_s<S, uint64_t>(const KParams &, size_t, int *);                            \
    template hipError_t launch_search_s<S, uint32_t>(int, const KParams &, const SearchParams &, uint32_t, size_t,  \
                                                      hipStream_t);                                                 \
    template hipError_t launch_search_s<S, uint64_t>(int, const KParams &, const SearchParams &, uint32_t, size_t,  \
                                                      hipStream_t);
