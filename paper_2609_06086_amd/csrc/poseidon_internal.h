// Internal interface between the C-ABI host code and the HIP kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pk {

constexpr int kSMax = 16;
constexpr uint32_t kNB = 256;   // Pascal-table column length (n = 0..255; L <= 256)
constexpr uint32_t kTypesMax = 8;   // device types (the ABI's limit, checked where both are seen)

// Buckets of the unranking searches.  A value Q >= 1 of a w-bit type falls in
// bucket (z, m): z its number of leading zeros in w bits, m the 4 bits after
// its leading one (zero-filled when fewer follow it); key = 16 z + m.  The
// bucket holds [bucket_lo(z, m), bucket_lo of the next key), the next key
// being (z, m + 1), or (z - 1, 0) after m = 15; keys that no value has get
// an empty range.  For each Pascal column the host tabulates, per key, the
// first row whose entry reaches bucket_lo (kBucketTab bytes a column), so a
// search starts there and needs only a few halvings.
// Halvings of one cut search over a whole Pascal column: the smallest H with
// L <= 2^H (at least 5); the columns hold rows n < 2^H.
__host__ __device__ constexpr uint32_t decode_levels(uint32_t L) {
    return L > 128 ? 8u : L > 64 ? 7u : L > 32 ? 6u : 5u;
}

constexpr uint32_t kBucketTab = 1024;   // 64 z values x 16 m values, one byte each
__host__ __device__ constexpr unsigned __int128 bucket_lo(int w, int z, int m) {
    // the smallest value whose leading one is bit e = w - 1 - z and whose next
    // four bits are at least m
    return (w - 1 - z) >= 4 ? (unsigned __int128)(16 + m) << ((w - 1 - z) - 4)
                            : ((unsigned __int128)(16 + m) + ((1u << (4 - (w - 1 - z))) - 1)) >> (4 - (w - 1 - z));
}
constexpr int kMaxLevels = 6;   // cascade checkpoints of the steady loop
constexpr uint32_t kSearchScanMax = 16384;   // blocks of one search level piece (search_scan_kernel's LDS)

enum AssignMode : uint32_t { kAssignFixed = 0, kAssignTable = 1, kAssignDigits = 2 };

// Kernel arguments, passed by value (uniform values land in SGPRs).
struct KParams {
    // device tables owned by the context
    const uint64_t *cost;      // [T][L+1] (prefix bwd << 32) | prefix fwd
    const uint32_t *pm;        // [L+1] prefix memory
    const uint32_t *cap;       // [T]
    const void *binom;         // [S][kNB] C(n, k), uint32 or uint64 (wide)
    const uint8_t *btab;       // [S][kBucketTab] per column: first row reaching each bucket
    const uint8_t *assign;     // [A][S] (table mode)
    const uint32_t *slot_mask; // [nslots][3] forward / deep-forward / backward stage masks
                               // ([nslots][4] under Interleaved 1F1B: + backward depths)
    const uint32_t *pd;        // [T][L+1] prefix all-reduce time (has_ar)
    const uint32_t *ent;       // stage entries of the evaluation kernels: [T][fields][kEntRow], then
                               // (dig_tg > 0) the assignment-digit table [dig_tg] of uint64
    uint32_t erow;             // bytes of one type's block of entry fields
    uint32_t ent_bytes;        // bytes of the entries (the digit table starts there)
    uint32_t ent_lds;          // LDS bytes the entries and the digit table take
    uint32_t dig_tg, dig_magic;   // base-T assignment digits with T <= 4: T^4 and floor(2^32 / T^4) + 1
                                  // (0: no digit table)
    uint32_t g24;                 // every stage's F + B is below 2^24 (and M is), so M (F + B) is a
                                  // 24-bit multiply
    uint64_t A, n_comp;
    uint32_t L, S, M, T, NB, nslots;
    uint32_t magicT, assign_mode;
    uint32_t s1_div, s1_magic;    // base-T assignment digits: T^(S-1) and floor(2^32 / T^(S-1)) + 1,
                                  // so that stage 1's type (the top digit) is one multiply-high
    uint32_t wide;
    uint32_t cf[kSMax], cb[kSMax];
    uint32_t has_ar;              // the problem has DP all-reduce times
    uint32_t sched;               // POSEIDON_SCHEDULE_*
    uint32_t ndev;                // devices: S, or S / V under Interleaved 1F1B
    uint32_t last_lo[kTypesMax];  // per type t: smallest c with pm[L] - pm[c] <= cap[t] (search)
    uint32_t g_mono_all;          // every type pair has its g_mono bit (the search kernels then
                                  // compile the closed-form last stage only)
    uint64_t g_mono;              // bit 8 t + u: every layer's fwd + bwd on t is at most M times
                                  // that on u (the search's last-stage Eq. 2 then falls with the cut)
    uint32_t ilv_compiled, ilv_trips; // Interleaved 1F1B: the schedule runs as compiled code with
                                      // this many steady periods
    uint32_t psi[kSMax];          // cf_0 + ... + cf_{s-1}: undoes the per-stage shift at the end
    uint8_t fixed_types[kSMax];
    // candidates of the call
    uint64_t first, count;
    const uint64_t *comp_rank;
    const uint32_t *assign_idx;
    // outputs
    uint32_t *makespan_out;
    uint32_t *feas_bits_out;
    uint64_t nwords;
    // reduction state (device words owned by the context)
    unsigned long long *acc;
    unsigned int *done;
    unsigned long long *result;
    unsigned long long *run_best;     // early stop: best over the chunks so far
    unsigned long long *snap;         // early stop: run_best as of the previous chunk
    unsigned long long *stats;   // evaluated, pruned, infeasible
    unsigned int *err;
    // early stop: the caller's bound, and the list of the candidates that
    // pass the memory and Eq. 2 tests (call index, cut codes in `codes`), in
    // per-block segments of seg_cap entries with their counts in scount;
    // alist / acount: the same for the candidates that pass the tests of
    // their first stages (kAListWords arrays of ccap words: call index and
    // the state of their decode)
    uint32_t es_bound;
    uint32_t *sidx;
    unsigned int *scount;
    uint32_t *alist;
    unsigned int *acount;
    // steady-state cascade: lanes not settled at iteration (Interleaved
    // 1F1B: period) lvl_k[l-1] are
    // queued (candidate index + registers) and resumed by level l
    uint32_t nlevels;                 // 0 = no cascade
    uint32_t lvl_k[kMaxLevels];
    unsigned int *qcount;             // [level][nseg]: entries block b queued for level + 1
    uint32_t *queue[2];               // ping-pong queues: level l reads queue (l-1) & 1;
                                      // each idx[qcap] | codes[words][qcap] | asg[qcap] (if qasg)
                                      // | Y[NX][qcap] (NX = S for 1F1B, 2S for Eager 1F1B, the
                                      // live registers under Interleaved 1F1B),
                                      // block b owning slots [b * seg_cap, (b+1) * seg_cap)
    uint32_t qasg;                    // queue entries carry the assignment index (calls with a
                                      // list of assignment indices)
    uint64_t qcap, seg_cap;
    uint32_t nseg;                    // blocks of the level-0 grid (= every level's grid)
    // the current chunk of the call: candidates first_i .. first_i + n_i - 1
    uint64_t first_i, n_i;
    uint32_t *codes;                  // [words][ccap] compact cut points of the chunk
    uint64_t ccap;
    uint32_t accumulate;              // fold the chunk's best into *result (not the first chunk)
};

// Pruned search (Sec. 4.2.3): one piece of one frontier level.
// count-kernel blocks spread their counters over this many slots, so that
// no single address takes one atomic per block
constexpr uint32_t kStatSlots = 64;

struct SearchParams {
    const uint32_t *in_row;           // [in_cap] assignment row of each node
    const uint32_t *in_codes;         // [words][in_cap] cut codes, cuts 1..level set
    uint64_t in_cap;
    uint32_t n_in;                    // nodes of this piece (an upper bound when n_dev is set)
    const unsigned long long *n_dev;  // the piece's node count on the device, or null: n_in
    uint32_t level;                   // stages 1..level fixed
    uint32_t *out_row;                // children (or roots)
    uint32_t *out_codes;              // [words][out_cap]
    uint64_t out_cap;
    unsigned int *blk_tot;            // children per block (count kernel)
    unsigned long long *blk_off;      // exclusive offsets, [nblk] = total (scan kernel)
    uint16_t *node_cnt;               // children each node keeps (count kernel -> write kernel)
    uint32_t blk_base;                // first block a write launch covers
    uint32_t flags;                   // kSearchRidge | kSearchNoStage
    uint32_t fused;                   // level S-3 expanded together with the level that fixes the last cut
    uint32_t *bound;                  // the current chunk's bound
    unsigned long long *stats;        // visited, evaluated, pruned by memory / ridge / bound
    unsigned long long *stats_part;   // [5][kStatSlots] the same counters from the count kernels:
                                      // block b adds to slot b % kStatSlots (the host sums them)
    unsigned long long *acc;          // best (T << 32 | position) of a leaf piece
    unsigned long long *best;         // makespan, row, composition rank of the best so far
    unsigned long long *total;        // children of the scanned level piece (one word per level)
    uint32_t root_first;              // first row of a root piece
};

enum SearchOp { kSearchOpCount = 0, kSearchOpWrite = 1, kSearchOpLeaf = 2, kSearchOpMerge = 3, kSearchOpRoot = 4 };

// Stage entries of the evaluation kernels: per device type a block of
// field rows of kEntRow uint32 (end points 0..L <= 256, padded), so that a
// field sits at a compile-time byte offset from its end point's address.
constexpr uint32_t kEntRow = 264;
constexpr uint32_t kEntField = 4 * kEntRow;   // bytes per field row
enum EntField : uint32_t { kEPf = 0, kEPb = 1, kEHm = 2, kEPd = 3 };
__host__ __device__ constexpr uint32_t entry_fields(bool ar) { return ar ? 4u : 3u; }
__host__ __device__ constexpr size_t entry_bytes(uint32_t T, bool ar) {
    return (size_t)T * entry_fields(ar) * kEntField;
}

struct LaunchCfg {
    uint32_t grid = 0;
    uint32_t grid2 = 0;   // early stop: blocks of the survivor kernel
    size_t lds_bytes = 0;     // stage tables: the entries (evaluation, early-stop kernels) or cost, pm,
                          // cap (search and Interleaved 1F1B kernels)
};

hipError_t launch_eval(const KParams &p, const LaunchCfg &lc, hipStream_t st);
hipError_t launch_decode(const KParams &p, const LaunchCfg &lc, hipStream_t st);
hipError_t launch_resume(const KParams &p, const LaunchCfg &lc, hipStream_t st, uint32_t lvl);
hipError_t launch_bounded(const KParams &p, const LaunchCfg &lc, hipStream_t st, uint32_t publish);
constexpr int kAListWords = 6;  // words per entry of the early stop's first-stage list
constexpr int kDecodeIlp = 4;   // candidates per lane of the decode and early-stop filter kernels
hipError_t eval_occupancy(const KParams &p, size_t lds, int *blocks);
hipError_t filter_occupancy(const KParams &p, size_t ent_lds, int *blocks);
hipError_t launch_ilv(const KParams &p, const LaunchCfg &lc, hipStream_t st);
hipError_t ilv_occupancy(const KParams &p, size_t lds, int *blocks);
hipError_t launch_ilv_resume(const KParams &p, const LaunchCfg &lc, hipStream_t st, uint32_t lvl);
int ilv_state_words(uint32_t S, uint32_t N);   // live registers of the Interleaved 1F1B stencil per queue entry
int ilv_max_db(int N);   // backward input depth the Interleaved 1F1B stencil holds for N devices
// The compiled Interleaved 1F1B schedule for (S, N) as slot-table words:
// prologue [start][4], one period [2S][4], cool-down [tail][4].  Returns
// false if (S, N) has no compiled form.
bool ilv_program_words(uint32_t S, uint32_t N, int *start, int *tail, uint32_t *pro, uint32_t *period,
                       uint32_t *cool);
hipError_t launch_argmin(const uint32_t *T, const uint32_t *bits, uint64_t count, uint32_t grid,
                         unsigned long long *acc, unsigned int *done, unsigned long long *result, hipStream_t st);
hipError_t launch_fill(unsigned long long *p, uint32_t n, unsigned long long v, hipStream_t st);
// up to four ranges of words, 64 words in all, filled by one launch
struct FillRanges {
    uint32_t n;
    unsigned long long *ptr[4];
    uint32_t count[4];
    unsigned long long value[4];
};
hipError_t launch_fills(const FillRanges &r, hipStream_t st);
// Scratch of the allocation-free evaluation: the device address of the
// library's fixed scratch array on `device`, looked up once per device
// (with that device current) and kept; null if the lookup failed.
void *noalloc_scratch(int device);
size_t noalloc_scratch_bytes();
hipError_t launch_search(int op, const KParams &p, const SearchParams &q, uint32_t grid, size_t lds, hipStream_t st);
hipError_t launch_search_scan(const SearchParams &q, uint32_t nblk, hipStream_t st);
hipError_t launch_search_bound(const SearchParams &q, uint32_t bound, hipStream_t st);
int code_words(int S);
int prologue_op(int S, int s, int k);
int eager_op(int S, int M, int s, int k);   // Eager 1F1B closed form, M >= 2S-1: 0 idle, 1 F, 2 B, 3 F of depth 2
int epilogue_op(int S, int s, int j);

}  // namespace pk
