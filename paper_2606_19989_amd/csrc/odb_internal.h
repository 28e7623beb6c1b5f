// Internal declarations of the ODB HIP library (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>
#include <vector>

#include "odb.h"

namespace odb {

constexpr int kWave = 64;
constexpr int kBlock = 256;                 // threads per block for most kernels
constexpr int kSortItems = 8;               // keys per thread in a radix tile
constexpr int kSortTile = kBlock * kSortItems;
constexpr int kScanItems = 16;
constexpr int kScanTile = kBlock * kScanItems;
constexpr int kMaxJumpRounds = 40;
// grid cap of the grid-stride kernels of the plan stages, in blocks per compute unit
// (8 measured best: 4 too few loads in flight, 16 to 256 slower as per-block setup and
// same-address atomics grow with the grid)
constexpr int kPlanBlocksPerCU = 8;

// ------------------------------------------------------------------ host error state
int set_error(int code, const char* fmt, ...);
const char* last_error();

#define ODB_TRY_HIP(expr)                                                                   \
    do {                                                                                    \
        hipError_t e_ = (expr);                                                             \
        if (e_ != hipSuccess)                                                               \
            return ::odb::set_error(ODB_E_HIP, "%s failed: %s (%s:%d)", #expr,               \
                                    hipGetErrorString(e_), __FILE__, __LINE__);             \
    } while (0)

#define ODB_TRY(expr)                                                                       \
    do {                                                                                    \
        int s_ = (expr);                                                                    \
        if (s_ != ODB_OK) return s_;                                                        \
    } while (0)

// Launch check: a bad launch configuration shows up as a pending error.
#define ODB_LAUNCHED() ODB_TRY_HIP(hipGetLastError())

// ------------------------------------------------------------------ device status
enum : int32_t {
    kErrLength = 1,      // some l < 1 or l >= 2^31
    kErrOffsets = 2,     // token offsets out of range
    kErrOrder = 4,       // stage-1 order not a valid formation order of the window
    kErrGroupIndex = 8,  // stage-1 group indices inconsistent
    kErrIdentity = 16,   // identity outside [0, num_identities)
    kErrCollate = 32,    // collate met an inconsistent plan
    kErrInternal = 64,
    kErrSortedLen = 128  // a stage-1 sorted length differs from the sample's CSR length
};

struct DevStatus {
    int32_t err;
    int32_t collate_err;
    int64_t first_bad;            // smallest offending sample index (atomicMin)
    int64_t first_bad_len;        // smallest sample with an invalid CSR length found by alignment
    uint32_t min_len;
    uint32_t max_len;
    int32_t jump_changed[kMaxJumpRounds];
    unsigned long long collate_runs;   // runs handed out by the collate beyond its first wave
};

// Per-rank alignment state, kept on the device across rounds.
enum : int32_t { kActInactive = 0, kActKeep = 1, kActSplit = 2, kActOverflow = 3 };

struct RankState {
    int64_t emitted;   // samples emitted so far (all rounds)
    int64_t slots;     // real (non-IDLE) slots so far
    int64_t cnt;       // S_r: samples buffered at the start of this round
    int64_t next_cnt;  // samples back in the buffer after this round
    int64_t G;         // groups formed this round
    int64_t gbase;     // global id of this rank's first group this round
    int64_t X;         // split: positions [0, X) become singletons
    int64_t jstar;     // split: formation group that keeps [X, end)
    int64_t qcut;      // keep/split: first formation position that is emitted
    int64_t ebase;     // samples emitted before this round
    int32_t action;
    int32_t pad;
};

struct RoundState {
    int64_t T;               // alignment target of the current round
    int64_t cut;             // steps of this round that are emitted
    int64_t emitted_total;   // cumulative emitted samples before this round
    int64_t emitted_next;    // the same after this round (current once the round ends)
    int64_t step_max;        // largest global step count so far
    int64_t splits;          // all rounds
    int64_t overflow;        // all rounds
    int64_t quota_hit;       // 1 once the non-join quota was reached
    int64_t active;          // active ranks this round
    int64_t total_groups;    // groups over all ranks this round
    int64_t leftover_total;  // samples back in buffers after this round
    int64_t second_gather;   // rounds in which some active rank had G_r != T (all rounds)
};

// Final summary assembled on the device (mirrors odb_plan_info_t's counters).
struct DevInfo {
    int64_t real_tokens;
    int64_t padded_elems;
    int64_t emitted;
    int64_t bad_views;
    int64_t missing_ids;
    int64_t duplicate_ids;
    int64_t distinct_views;   // views marked at least once (bitset pass)
    double pad_fraction;
};


// ------------------------------------------------------------------ workspace layout
struct Layout {
    size_t status, round, ranks, rank_off, cap, gbase, tile_first, rank_runs;
    size_t len, keys0, keys1, vals0, vals1, counts, partials;
    size_t jmp0, jmp1, marks, incl;
    size_t gstart, gsize, gmax, sadj, cs, ov_slot, ov_lo, kept;
    size_t srows, smax, stok, steps;
    size_t buf_ids0, buf_ids1, buf_len0, buf_len1, gidx, stage, stage_len, cover, row_ts, row_len;
    size_t info, sketch;
    size_t total;
    int64_t num_sort_blocks;
    int64_t partials_len;
};

bool make_layout(const odb_window_t* w, Layout* L);

template <class T>
inline T* ws_at(void* ws, size_t off) {
    return reinterpret_cast<T*>(static_cast<char*>(ws) + off);
}

// Validates the window fields that can be checked on the host.
int check_window(const odb_window_t* w);
int check_workspace(const odb_window_t* w, void* d_ws, size_t ws_bytes, Layout* L);

// Uploads rank offsets (and optionally capacities) and clears the status word.
int upload_small(const odb_window_t* w, const Layout& L, void* d_ws, const int64_t* cap,
                 hipStream_t s);

// Host copy of the status word, round state, summary and per-rank state, read with one
// device-to-host copy (the workspace keeps them next to each other) and one
// synchronisation of the stream.
struct HostState {
    DevStatus st;
    RoundState rs;
    DevInfo info;
    std::vector<RankState> ranks;
    std::vector<char> buf;
};
int read_state(const Layout& L, void* ws, int W, HostState* h, hipStream_t s);

int num_cus();

inline unsigned grid_for(int64_t n, int per_block, int64_t cap = 1 << 20) {
    int64_t g = (n + per_block - 1) / per_block;
    if (g < 1) g = 1;
    if (g > cap) g = cap;
    return (unsigned)g;
}

// ------------------------------------------------------------------ device helpers
// Eq. 1: B(l) = max(floor(L_max / l), 1), integer division, clipped to 2^31 - 1.  A rank
// holds fewer than 2^31 - 1 samples, so a group of B >= 2^31 - 1 takes the rest of its rank
// either way; the clip keeps position + B inside int64 for budgets up to 2^63 - 1.
__device__ __forceinline__ int64_t batch_size(int64_t budget, int32_t l) {
    int64_t b;
    if (budget <= 0xFFFFFFFFll)
        b = (int64_t)((uint32_t)budget / (uint32_t)l);
    else
        b = budget / (int64_t)l;
    b = b < INT32_MAX ? b : INT32_MAX;
    return b > 1 ? b : 1;
}

// Number of ranks r with off[r] <= p, minus one: the rank owning position p
// (off is non-decreasing, p < off[W]).
__device__ __forceinline__ int rank_of(const int64_t* off, int W, int64_t p) {
    int lo = 0, hi = W;  // invariant: off[lo] <= p < off[hi]
    while (hi - lo > 1) {
        int mid = (lo + hi) >> 1;
        if (off[mid] <= p) lo = mid; else hi = mid;
    }
    return lo;
}

// Rank offsets staged in LDS for kernels that look up the rank of many positions;
// windows with more ranks than fit read them from global memory instead.
constexpr int kLdsRanks = 1024;

__device__ __forceinline__ const int64_t* stage_ranks(const int64_t* off, int W, int64_t* s_off) {
    if (W > kLdsRanks) return off;
    for (int i = threadIdx.x; i <= W; i += blockDim.x) s_off[i] = off[i];
    __syncthreads();
    return s_off;
}

// Workgroup barrier ordering LDS only: unlike __syncthreads() it does not wait for the
// wave's outstanding global loads and stores, for loops whose barriers guard LDS tables
// while their global stores are read by nobody in the block before a full barrier.
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

template <typename T>
__device__ __forceinline__ T wave_incl_sum(T v) {
    const int lane = threadIdx.x & (kWave - 1);
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) {
        T o = __shfl_up(v, d, kWave);
        if (lane >= d) v += o;
    }
    return v;
}

template <typename T>
__device__ __forceinline__ T wave_sum(T v) {
#pragma unroll
    for (int d = kWave / 2; d > 0; d >>= 1) v += __shfl_xor(v, d, kWave);
    return v;
}

// DPP lane moves (data-parallel primitives of this ISA): row_shr:n (control 0x110 + n)
// moves a value n lanes up within each row of 16 lanes, row_bcast:15 (0x142) hands the
// last lane of each row to the next row and row_bcast:31 (0x143) lane 31 to rows 2 and 3;
// rows and banks (groups of 4 lanes in a row) left out by the masks, and lanes a shift
// cannot reach, read 0.  A 64-bit value moves as two halves.
template <int CTRL, int ROWS, int BANKS, typename T>
__device__ __forceinline__ T dpp_move(T v) {
    if constexpr (sizeof(T) == 8) {
        const uint64_t u = (uint64_t)v;
        const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)u, CTRL, ROWS, BANKS, true);
        const uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)(u >> 32), CTRL, ROWS, BANKS, true);
        return (T)(((uint64_t)hi << 32) | lo);
    } else {
        return (T)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, ROWS, BANKS, true);
    }
}

struct OpAdd {
    template <typename T>
    __device__ static T apply(T a, T b) { return a + b; }
};
struct OpMax {   // for values >= 0 (a lane that reads nothing reads 0)
    template <typename T>
    __device__ static T apply(T a, T b) { return a > b ? a : b; }
};

// Inclusive scan over the 64 lanes of a wave without LDS: shifts 1-3 give windows of 4
// lanes, shift 4 on banks 1-3 and shift 8 on banks 2-3 complete each row of 16, the two
// broadcasts carry row totals into the rows above.  Every lane of the wave must be active.
template <typename Op, typename T>
__device__ __forceinline__ T wave_scan_dpp(T x) {
    T s = x;
    s = Op::apply(s, dpp_move<0x111, 0xf, 0xf>(x));
    s = Op::apply(s, dpp_move<0x112, 0xf, 0xf>(x));
    s = Op::apply(s, dpp_move<0x113, 0xf, 0xf>(x));
    s = Op::apply(s, dpp_move<0x114, 0xf, 0xe>(s));
    s = Op::apply(s, dpp_move<0x118, 0xf, 0xc>(s));
    s = Op::apply(s, dpp_move<0x142, 0xa, 0xf>(s));
    s = Op::apply(s, dpp_move<0x143, 0xc, 0xf>(s));
    return s;
}

// Value of lane 63 (a wave's inclusive-scan total), uniform over the wave.
template <typename T>
__device__ __forceinline__ T wave_last(T v) {
    if constexpr (sizeof(T) == 8) {
        const uint64_t u = (uint64_t)v;
        const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u, kWave - 1);
        const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), kWave - 1);
        return (T)(((uint64_t)hi << 32) | lo);
    } else {
        return (T)__builtin_amdgcn_readlane((int)v, kWave - 1);
    }
}

// Lanes below this one whose bit is set in a 64-lane mask.
__device__ __forceinline__ int lanes_below(uint64_t m) {
    return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

// Exclusive block scan for blockDim.x == kBlock; *total receives the block sum.
template <typename T>
__device__ __forceinline__ T block_excl_sum(T v, T* total) {
    __shared__ T wtot[kBlock / kWave];
    T inc = wave_incl_sum(v);
    const int w = threadIdx.x / kWave;
    if ((threadIdx.x & (kWave - 1)) == kWave - 1) wtot[w] = inc;
    __syncthreads();
    T pre = 0, tot = 0;
#pragma unroll
    for (int i = 0; i < kBlock / kWave; ++i) {
        T x = wtot[i];
        pre += (i < w) ? x : T(0);
        tot += x;
    }
    __syncthreads();
    *total = tot;
    return pre + inc - v;
}

template <typename T>
__device__ __forceinline__ T block_sum(T v) {
    __shared__ T wtot[kBlock / kWave];
    v = wave_sum(v);
    const int w = threadIdx.x / kWave;
    if ((threadIdx.x & (kWave - 1)) == 0) wtot[w] = v;
    __syncthreads();
    T tot = 0;
#pragma unroll
    for (int i = 0; i < kBlock / kWave; ++i) tot += wtot[i];
    __syncthreads();
    return tot;
}

// ------------------------------------------------------------------ generic device scan
// Exclusive prefix sum out[i] = sum_{k<i} in(k) over i in [0, n), in three launches
// (tile sums, a one-block scan of the tile sums, tile-local scans).  `Load` is a
// functor int64 -> Out, `Store` a functor (int64 i, Out value) -> void.  partials
// needs ceil(n / kScanTile) + 1 entries.  The total is written to partials[tiles].
template <typename Out, typename Load>
__global__ void __launch_bounds__(kBlock) scan_tile_sums(Load load, int64_t n, Out* partials) {
    const int64_t base = (int64_t)blockIdx.x * kScanTile;
    Out s = 0;
#pragma unroll 4
    for (int i = 0; i < kScanItems; ++i) {
        int64_t idx = base + (int64_t)i * kBlock + threadIdx.x;
        if (idx < n) s += load(idx);
    }
    s = block_sum(s);
    if (threadIdx.x == 0) partials[blockIdx.x] = s;
}

// One block of kBlock threads: a 1024-thread block would need a quarter of every SIMD's
// wave slots on one compute unit, which a resident collate grid never leaves free.
template <typename Out>
__global__ void __launch_bounds__(kBlock) scan_partials(Out* partials, int64_t m) {
    __shared__ Out wtot[kBlock / kWave];
    __shared__ Out carry_s;
    if (threadIdx.x == 0) carry_s = 0;
    __syncthreads();
    for (int64_t base = 0; base < m; base += kBlock) {
        int64_t i = base + threadIdx.x;
        Out v = i < m ? partials[i] : Out(0);
        Out inc = wave_incl_sum(v);
        const int w = threadIdx.x / kWave;
        if ((threadIdx.x & (kWave - 1)) == kWave - 1) wtot[w] = inc;
        __syncthreads();
        Out pre = 0, tot = 0;
#pragma unroll
        for (int k = 0; k < kBlock / kWave; ++k) {
            pre += (k < w) ? wtot[k] : Out(0);
            tot += wtot[k];
        }
        Out c = carry_s;
        if (i < m) partials[i] = c + pre + inc - v;
        __syncthreads();
        if (threadIdx.x == 0) carry_s = c + tot;
        __syncthreads();
    }
    if (threadIdx.x == 0) partials[m] = carry_s;
}

template <typename Out, typename Load, typename Store>
__global__ void __launch_bounds__(kBlock) scan_tiles(Load load, Store store, int64_t n,
                                                      const Out* partials) {
    const int64_t base = (int64_t)blockIdx.x * kScanTile;
    Out carry = partials[blockIdx.x];
    for (int i = 0; i < kScanItems; ++i) {
        int64_t idx = base + (int64_t)i * kBlock + threadIdx.x;
        Out v = idx < n ? load(idx) : Out(0);
        Out tot;
        Out ex = block_excl_sum(v, &tot);
        if (idx < n) store(idx, carry + ex);
        carry += tot;
    }
}

// Scans of at most kSmallScan elements run as one launch of one block: 16 consecutive
// elements per thread, one block scan of the thread sums.  The total goes to *total.
constexpr int kSmallScanThreads = 1024;
constexpr int kSmallScanItems = 16;
constexpr int64_t kSmallScan = (int64_t)kSmallScanThreads * kSmallScanItems;

template <typename Out, typename Load, typename Store>
__global__ void __launch_bounds__(kSmallScanThreads) scan_small(Load load, Store store, int64_t n, Out* total) {
    __shared__ Out wtot[kSmallScanThreads / kWave];
    const int t = threadIdx.x, w = t / kWave;
    const int64_t base = (int64_t)t * kSmallScanItems;
    Out v[kSmallScanItems];
    Out sum = 0;
#pragma unroll
    for (int j = 0; j < kSmallScanItems; ++j) {
        v[j] = base + j < n ? load(base + j) : Out(0);
        sum += v[j];
    }
    const Out inc = wave_incl_sum(sum);
    if ((t & (kWave - 1)) == kWave - 1) wtot[w] = inc;
    __syncthreads();
    Out pre = 0, tot = 0;
#pragma unroll
    for (int k = 0; k < kSmallScanThreads / kWave; ++k) {
        pre += k < w ? wtot[k] : Out(0);
        tot += wtot[k];
    }
    Out run = pre + inc - sum;
#pragma unroll
    for (int j = 0; j < kSmallScanItems; ++j) {
        if (base + j < n) store(base + j, run);
        run += v[j];
    }
    if (t == 0) *total = tot;
}

template <typename Out, typename Load, typename Store>
int device_excl_scan(Load load, Store store, int64_t n, Out* partials, hipStream_t s) {
    if (n <= 0) return ODB_OK;
    int64_t tiles = (n + kScanTile - 1) / kScanTile;
    if (n <= kSmallScan) {
        hipLaunchKernelGGL((scan_small<Out, Load, Store>), dim3(1), dim3(kSmallScanThreads), 0, s, load, store, n,
                           partials + tiles);
        ODB_LAUNCHED();
        return ODB_OK;
    }
    hipLaunchKernelGGL((scan_tile_sums<Out, Load>), dim3((unsigned)tiles), dim3(kBlock), 0, s,
                       load, n, partials);
    ODB_LAUNCHED();
    hipLaunchKernelGGL((scan_partials<Out>), dim3(1), dim3(kBlock), 0, s, partials, tiles);
    ODB_LAUNCHED();
    hipLaunchKernelGGL((scan_tiles<Out, Load, Store>), dim3((unsigned)tiles), dim3(kBlock), 0, s,
                       load, store, n, (const Out*)partials);
    ODB_LAUNCHED();
    return ODB_OK;
}

// ------------------------------------------------------------------ cross-file launchers
// Grouping of the per-rank sequences held in `slen` (positions [off[r], off[r] + cnt_r)
// of every rank r, cnt_r = d_ranks[r].cnt): finds the group starts (a walk over the runs of
// equal step, or pointer jumping over the next-group-start links when a rank may hold
// too many runs), then writes the formation group index of every position (d_gidx), the
// global position of every group start (workspace gstart, group ids numbered rank by
// rank), G_r and the first group id of every rank (d_ranks[r].G, .gbase and workspace
// gbase[W+1]), and optionally G_r to d_groups_out.
// len_range = max_len - min_len + 1 of the sequences if known (0 otherwise); it only
// selects between the two equivalent ways of finding the chain (see odb_form.hip).
// tiles_ready: workspace tile_first already holds the sort tiles of d_rank_off.
int group_sequences(const Layout& L, void* ws, int W, int64_t n, int64_t budget,
                    const int64_t* d_rank_off, int64_t max_cnt, int64_t len_range, bool tiles_ready,
                    const int32_t* d_slen, int32_t* d_gidx, int32_t* d_groups_out,
                    RankState* d_ranks, hipStream_t s);

}  // namespace odb
