// Launch dispatch over the stage count S and the rank width, plus the
// non-templated kernels.  The templated kernels are instantiated in
// poseidon_inst_*.hip, split by S so that they compile in parallel.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>

#include "../../include/poseidon.h"
#include "poseidon_search.h"

namespace pk {

// Scratch of poseidon_eval_candidates_noalloc: one copy per GPU, resident
// from the code object's load until the process ends.  In host code
// `scratch` names a host-side stand-in, not device memory, so host code
// only ever uses the address hipGetSymbolAddress returns for the current
// device.
static __device__ __align__(256) uint32_t scratch[POSEIDON_NOALLOC_SCRATCH_BYTES / 4];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
bool g_scratch_done[kMaxDevices];
void *g_scratch_ptr[kMaxDevices];
}  // namespace

void *noalloc_scratch(int device) {
    if (device < 0 || device >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_done[device]) {
        g_scratch_done[device] = true;
        int prev = 0;
        void *ptr = nullptr;
        if (hipGetDevice(&prev) == hipSuccess && hipSetDevice(device) == hipSuccess) {
            if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess) {
                (void)hipGetLastError();
                ptr = nullptr;
            }
            (void)hipSetDevice(prev);
        }
        g_scratch_ptr[device] = ptr;
    }
    return g_scratch_ptr[device];
}

size_t noalloc_scratch_bytes() { return sizeof(scratch); }

#define PK_EXTERN(S)                                                                                     \
    extern template hipError_t launch_eval_s<S, uint32_t>(const KParams &, const LaunchCfg &, hipStream_t);    \
    extern template hipError_t launch_eval_s<S, uint64_t>(const KParams &, const LaunchCfg &, hipStream_t);    \
    extern template hipError_t launch_decode_s<S, uint32_t>(const KParams &, const LaunchCfg &, hipStream_t);  \
    extern template hipError_t launch_decode_s<S, uint64_t>(const KParams &, const LaunchCfg &, hipStream_t);  \
    extern template hipError_t launch_resume_s<S, uint32_t>(const KParams &, const LaunchCfg &, hipStream_t,   \
                                                             uint32_t);                                       \
    extern template hipError_t launch_resume_s<S, uint64_t>(const KParams &, const LaunchCfg &, hipStream_t,   \
                                                             uint32_t);                                       \
    extern template hipError_t launch_bounded_s<S, uint32_t>(const KParams &, const LaunchCfg &, hipStream_t,  \
                                                              uint32_t);                                      \
    extern template hipError_t launch_bounded_s<S, uint64_t>(const KParams &, const LaunchCfg &, hipStream_t,  \
                                                              uint32_t);                                      \
    extern template hipError_t occupancy_s<S, uint32_t>(int *, size_t, bool, bool);                                 \
    extern template hipError_t occupancy_s<S, uint64_t>(int *, size_t, bool, bool);                                 \
    extern template hipError_t filter_occupancy_s<S, uint32_t>(const KParams &, size_t, int *);                     \
    extern template hipError_t filter_occupancy_s<S, uint64_t>(const KParams &, size_t, int *);                     \
    extern template hipError_t launch_search_s<S, uint32_t>(int, const KParams &, const SearchParams &, uint32_t,   \
                                                             size_t, hipStream_t);                                  \
    extern template hipError_t launch_search_s<S, uint64_t>(int, const KParams &, const SearchParams &, uint32_t,   \
                                                             size_t, hipStream_t);

PK_EXTERN(1) PK_EXTERN(2) PK_EXTERN(3) PK_EXTERN(4) PK_EXTERN(5) PK_EXTERN(6) PK_EXTERN(7) PK_EXTERN(8)
PK_EXTERN(9) PK_EXTERN(10) PK_EXTERN(11) PK_EXTERN(12) PK_EXTERN(13) PK_EXTERN(14) PK_EXTERN(15) PK_EXTERN(16)

// Argmin over stored makespans / feasibility bits.
__global__ __launch_bounds__(kBlock) void argmin_kernel(const uint32_t *T, const uint32_t *bits, uint64_t count,
                                                        unsigned long long *acc, unsigned int *done,
                                                        unsigned long long *result) {
    unsigned long long best = ~0ull;
    const uint64_t stride = (uint64_t)gridDim.x * kBlock;
    for (uint64_t i = (uint64_t)blockIdx.x * kBlock + threadIdx.x; i < count; i += stride) {
        const bool f = bits ? ((bits[i >> 5] >> (i & 31)) & 1u) : true;
        const unsigned long long key = make_key(f, T[i], (uint32_t)i);
        best = key < best ? key : best;
    }
    block_min_and_finish(best, acc, done, result, nullptr, true);
}

// Exclusive offsets of the block totals (one block); total to q.total.  The
// totals are staged in LDS with coalesced loads (one padding word per 64
// entries, so the per-thread runs of phase 2 start on different banks);
// each thread then scans a contiguous run there, and the offsets go back
// out coalesced.  The kernel sits between the count and write launches of
// every level and its time is the latency of its loads, so it reads nothing
// else (the counters go to slots the host sums).  A block has at most
// 256 (L - 1)^2 < 2^22 children (fused levels, L <= 129) and a run at most
// kSearchScanMax / 256 = 64 blocks, so an offset within its run fits 32 bits
// in LDS; the run's own 64-bit start is kept beside it (a whole piece can
// exceed 2^32 children).

__device__ __forceinline__ uint32_t scan_pad(uint32_t b) { return b + (b >> 6); }

__global__ __launch_bounds__(kBlock) void search_scan_kernel(SearchParams q, uint32_t nblk) {
    __shared__ uint32_t cnt[kSearchScanMax + kSearchScanMax / 64];
    __shared__ unsigned long long run0[kBlock];
#pragma unroll 8
    for (uint32_t b = threadIdx.x; b < nblk; b += kBlock) cnt[scan_pad(b)] = q.blk_tot[b];
    __syncthreads();
    const uint32_t per = (nblk + kBlock - 1) / kBlock;
    const uint32_t b0 = min(nblk, threadIdx.x * per), b1 = min(nblk, b0 + per);
    unsigned long long s = 0;
    for (uint32_t b = b0; b < b1; ++b) s += cnt[scan_pad(b)];
    unsigned long long total;
    run0[threadIdx.x] = block_exclusive_scan_u64(s, total);
    uint32_t rel = 0;
    for (uint32_t b = b0; b < b1; ++b) {
        const uint32_t v = cnt[scan_pad(b)];
        cnt[scan_pad(b)] = rel;
        rel += v;
    }
    __syncthreads();
#pragma unroll 8
    for (uint32_t b = threadIdx.x; b < nblk; b += kBlock) q.blk_off[b] = run0[b / per] + cnt[scan_pad(b)];
    if (threadIdx.x == 0) {
        q.blk_off[nblk] = total;
        *q.total = total;
    }
}

static_assert((uint64_t)(kSearchScanMax / kBlock) * kBlock * 128 * 128 < (1ull << 32),
              "a scan run's offsets must fit 32 bits");

// Start of a chunk: its bound is min(caller's bound, best so far).
__global__ void search_bound_kernel(SearchParams q, uint32_t bound) {
    if (threadIdx.x == 0 && blockIdx.x == 0) {
        const unsigned long long b = q.best[0];
        *const_cast<uint32_t *>(q.bound) = b < bound ? (uint32_t)b : bound;
    }
}

// Small fill kernel used instead of memset so that the calls stay capturable.
__global__ void fill_u64(unsigned long long *p, uint32_t n, unsigned long long v) {
    const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = v;
}

// ---------------------------------------------------------------------------

#define PK_DISPATCH(FN, S_, WIDE_, ...)                                                        \
    switch (S_) {                                                                              \
    case 1: return WIDE_ ? FN<1, uint64_t>(__VA_ARGS__) : FN<1, uint32_t>(__VA_ARGS__);       \
    case 2: return WIDE_ ? FN<2, uint64_t>(__VA_ARGS__) : FN<2, uint32_t>(__VA_ARGS__);       \
    case 3: return WIDE_ ? FN<3, uint64_t>(__VA_ARGS__) : FN<3, uint32_t>(__VA_ARGS__);       \
    case 4: return WIDE_ ? FN<4, uint64_t>(__VA_ARGS__) : FN<4, uint32_t>(__VA_ARGS__);       \
    case 5: return WIDE_ ? FN<5, uint64_t>(__VA_ARGS__) : FN<5, uint32_t>(__VA_ARGS__);       \
    case 6: return WIDE_ ? FN<6, uint64_t>(__VA_ARGS__) : FN<6, uint32_t>(__VA_ARGS__);       \
    case 7: return WIDE_ ? FN<7, uint64_t>(__VA_ARGS__) : FN<7, uint32_t>(__VA_ARGS__);       \
    case 8: return WIDE_ ? FN<8, uint64_t>(__VA_ARGS__) : FN<8, uint32_t>(__VA_ARGS__);       \
    case 9: return WIDE_ ? FN<9, uint64_t>(__VA_ARGS__) : FN<9, uint32_t>(__VA_ARGS__);       \
    case 10: return WIDE_ ? FN<10, uint64_t>(__VA_ARGS__) : FN<10, uint32_t>(__VA_ARGS__);    \
    case 11: return WIDE_ ? FN<11, uint64_t>(__VA_ARGS__) : FN<11, uint32_t>(__VA_ARGS__);    \
    case 12: return WIDE_ ? FN<12, uint64_t>(__VA_ARGS__) : FN<12, uint32_t>(__VA_ARGS__);    \
    case 13: return WIDE_ ? FN<13, uint64_t>(__VA_ARGS__) : FN<13, uint32_t>(__VA_ARGS__);    \
    case 14: return WIDE_ ? FN<14, uint64_t>(__VA_ARGS__) : FN<14, uint32_t>(__VA_ARGS__);    \
    case 15: return WIDE_ ? FN<15, uint64_t>(__VA_ARGS__) : FN<15, uint32_t>(__VA_ARGS__);    \
    case 16: return WIDE_ ? FN<16, uint64_t>(__VA_ARGS__) : FN<16, uint32_t>(__VA_ARGS__);    \
    default: return hipErrorInvalidValue;                                                      \
    }

hipError_t launch_eval(const KParams &p, const LaunchCfg &lc, hipStream_t st) {
    if (p.sched == 2) return launch_ilv(p, lc, st);   // Interleaved 1F1B
    PK_DISPATCH(launch_eval_s, p.S, p.wide, p, lc, st)
}

hipError_t launch_decode(const KParams &p, const LaunchCfg &lc, hipStream_t st) {
    PK_DISPATCH(launch_decode_s, p.S, p.wide, p, lc, st)
}

hipError_t launch_resume(const KParams &p, const LaunchCfg &lc, hipStream_t st, uint32_t lvl) {
    if (p.sched == 2) return launch_ilv_resume(p, lc, st, lvl);   // Interleaved 1F1B
    PK_DISPATCH(launch_resume_s, p.S, p.wide, p, lc, st, lvl)
}

hipError_t launch_bounded(const KParams &p, const LaunchCfg &lc, hipStream_t st, uint32_t publish) {
    PK_DISPATCH(launch_bounded_s, p.S, p.wide, p, lc, st, publish)
}

hipError_t filter_occupancy(const KParams &p, size_t ent_lds, int *blocks) {
    PK_DISPATCH(filter_occupancy_s, p.S, p.wide, p, ent_lds, blocks)
}

hipError_t eval_occupancy(const KParams &p, size_t lds, int *blocks) {
    if (p.sched == 2) return ilv_occupancy(p, lds, blocks);
    PK_DISPATCH(occupancy_s, p.S, p.wide, blocks, lds, p.has_ar != 0, p.sched != 0)
}

hipError_t launch_argmin(const uint32_t *T, const uint32_t *bits, uint64_t count, uint32_t grid,
                         unsigned long long *acc, unsigned int *done, unsigned long long *result, hipStream_t st) {
    hipLaunchKernelGGL(argmin_kernel, dim3(grid), dim3(kBlock), 0, st, T, bits, count, acc, done, result);
    return hipGetLastError();
}

hipError_t launch_search(int op, const KParams &p, const SearchParams &q, uint32_t grid, size_t lds, hipStream_t st) {
    PK_DISPATCH(launch_search_s, p.S, p.wide, op, p, q, grid, lds, st)
}

hipError_t launch_search_scan(const SearchParams &q, uint32_t nblk, hipStream_t st) {
    hipLaunchKernelGGL(search_scan_kernel, dim3(1), dim3(kBlock), 0, st, q, nblk);
    return hipGetLastError();
}

hipError_t launch_search_bound(const SearchParams &q, uint32_t bound, hipStream_t st) {
    hipLaunchKernelGGL(search_bound_kernel, dim3(1), dim3(64), 0, st, q, bound);
    return hipGetLastError();
}

hipError_t launch_fill(unsigned long long *p, uint32_t n, unsigned long long v, hipStream_t st) {
    hipLaunchKernelGGL(fill_u64, dim3((n + 63) / 64), dim3(64), 0, st, p, n, v);
    return hipGetLastError();
}

// Several short fills in one launch (one thread per word).
__global__ void fill_u64_ranges(FillRanges r) {
    uint32_t base = 0;
    for (uint32_t k = 0; k < r.n && k < 4; ++k) {
        if (threadIdx.x >= base && threadIdx.x < base + r.count[k]) r.ptr[k][threadIdx.x - base] = r.value[k];
        base += r.count[k];
    }
}

hipError_t launch_fills(const FillRanges &r, hipStream_t st) {
    hipLaunchKernelGGL(fill_u64_ranges, dim3(1), dim3(64), 0, st, r);
    return hipGetLastError();
}

int code_words(int S) { return S > 1 ? (S - 1 + 3) / 4 : 1; }
int prologue_op(int S, int s, int k) { return pro_op(S, s, k); }
int eager_op(int S, int M, int s, int k) {
    if (k <= 2 * S - 2) return eager_pro_op(S, s, k);
    if (k <= 2 * M - 2 * S) return eager_steady_op(s, k & 1);
    return eager_epi_op(S, s, k - (2 * M - 2 * S + 1));
}
int epilogue_op(int S, int s, int j) { return epi_op(S, s, j); }

}  // namespace pk
