// Stage 1 of the ODB window pipeline: length-aware grouping (Sec. 2.2, Eq. 1).
//
//   lengths_kernel        l_i = off[i+1] - off[i], validity, window min / max length
//   radix_hist/scatter    segmented stable LSD radix sort of every rank's samples by
//                         (length descending, id ascending): keys are max_l - l, the
//                         segments are the ranks, and stability over the id-ordered input
//                         gives the id tie-break
//   links_kernel          next-group-start links from the batch-size rule
//   jump_kernel           pointer-jumping list ranking that marks every group start
//   gidx / groups         formation group index of every position and G_r
//
// Grouping, restated: visiting a rank's samples longest first with threshold t (1 at
// the start), a group closes once it holds t samples and t becomes B(l) of its last
// (shortest) sample.  So group 0 is position 0 alone and a group starting at position
// p > 0 has B(l[p-1]) members (clipped by the end of the rank): next(0) = 1 and
// next(p) = p + B(l[p-1]).  The group starts are exactly the positions reachable from 0
// along next().
//
// Two equivalent ways to find them.  Lengths are sorted, so the step b(p) = B(l[p-1]) is
// constant on runs of positions, and there are at most ~2 sqrt(budget) distinct values
// of floor(budget / l): inside a run of step b the chain advances by exactly b, so one
// thread per rank can walk the runs (in LDS) and record each run's first chain position,
// and every position then knows whether it is a group start by one modulo.  When the
// number of runs may exceed the LDS table, pointer jumping over the next() links marks
// the chain in O(log G) doubling rounds instead.
#include <climits>
#include <cmath>
#include <vector>

#include "odb_internal.h"

namespace odb {

namespace {

__device__ __forceinline__ uint32_t lanes_below(uint64_t m) {
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

// Lanes of this wave whose `valid` digit equals this lane's (ballot per digit bit).
__device__ __forceinline__ uint64_t match_digit(uint32_t d, bool valid, int dbits) {
    uint64_t peers = __ballot(valid);
    for (int b = 0; b < dbits; ++b) {
        const bool bit = (d >> b) & 1u;
        const uint64_t m = __ballot(bit);
        peers &= bit ? m : ~m;
    }
    return peers;
}

__global__ void __launch_bounds__(kBlock) lengths_kernel(const int64_t* __restrict__ tok_off, int64_t n,
                                                         int32_t* __restrict__ len, DevStatus* st) {
    uint32_t lmin = 0xFFFFFFFFu, lmax = 0;
    int64_t bad = LLONG_MAX;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    auto one = [&](int64_t p, int64_t a, int64_t b) {
        int64_t l = b - a;
        if (l < 1 || l > INT_MAX || a < 0) {
            bad = bad < p ? bad : p;
            l = 1;
        }
        len[p] = (int32_t)l;
        lmin = (uint32_t)l < lmin ? (uint32_t)l : lmin;
        lmax = (uint32_t)l > lmax ? (uint32_t)l : lmax;
    };
    // four grid-stride iterations at a time, their loads issued together: with the grid at
    // full occupancy, one load in flight per lane leaves the kernel latency bound
    int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    for (; p + 3 * stride < n; p += 4 * stride) {
        int64_t a[4], b[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            a[k] = tok_off[p + k * stride];
            b[k] = tok_off[p + k * stride + 1];
        }
#pragma unroll
        for (int k = 0; k < 4; ++k) one(p + k * stride, a[k], b[k]);
    }
    for (; p < n; p += stride) one(p, tok_off[p], tok_off[p + 1]);
    // one pair of atomics per block: lanes -> waves (shuffles) -> block (LDS)
    __shared__ uint32_t s_min[kBlock / kWave], s_max[kBlock / kWave];
#pragma unroll
    for (int d = kWave / 2; d > 0; d >>= 1) {
        uint32_t a = __shfl_xor(lmin, d, kWave), b = __shfl_xor(lmax, d, kWave);
        lmin = a < lmin ? a : lmin;
        lmax = b > lmax ? b : lmax;
    }
    if ((threadIdx.x & (kWave - 1)) == 0) {
        s_min[threadIdx.x / kWave] = lmin;
        s_max[threadIdx.x / kWave] = lmax;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int i = 1; i < kBlock / kWave; ++i) {
            lmin = s_min[i] < lmin ? s_min[i] : lmin;
            lmax = s_max[i] > lmax ? s_max[i] : lmax;
        }
        if (lmax > 0) {
            atomicMin(&st->min_len, lmin);
            atomicMax(&st->max_len, lmax);
        }
    }
    if (bad != LLONG_MAX) {
        atomicOr(&st->err, kErrLength);
        atomicMin((unsigned long long*)&st->first_bad, (unsigned long long)bad);
    }
}

__global__ void rank_counts_kernel(const int64_t* __restrict__ off, int W, RankState* ranks) {
    for (int r = blockIdx.x * blockDim.x + threadIdx.x; r < W; r += gridDim.x * blockDim.x) {
        RankState z = {};
        z.cnt = off[r + 1] - off[r];
        ranks[r] = z;
    }
}

// First radix tile of every rank: tile_first[r] = sum_{r' < r} ceil(n_r' / kSortTile).
// Tiles never straddle ranks.  One block.
__global__ void __launch_bounds__(kBlock) sort_tiles_kernel(const int64_t* __restrict__ off, int W,
                                                            int64_t* __restrict__ tile_first) {
    __shared__ int64_t carry;
    if (threadIdx.x == 0) carry = 0;
    __syncthreads();
    for (int b = 0; b < W; b += kBlock) {
        const int r = b + threadIdx.x;
        const int64_t v = r < W ? (off[r + 1] - off[r] + kSortTile - 1) / kSortTile : 0;
        int64_t tot;
        const int64_t ex = block_excl_sum(v, &tot);
        const int64_t c = carry;
        if (r < W) tile_first[r] = c + ex;
        __syncthreads();
        if (threadIdx.x == 0) carry = c + tot;
        __syncthreads();
    }
    if (threadIdx.x == 0) tile_first[W] = carry;
}

struct SortTile {
    int64_t start;       // first position
    int32_t count;       // keys in this tile (<= kSortTile)
    int32_t seg_tiles;   // tiles of this tile's rank
    int64_t first;       // global index of the rank's first tile
    int32_t j;           // index of this tile within its rank
};

__device__ __forceinline__ SortTile sort_tile(const int64_t* __restrict__ off,
                                              const int64_t* __restrict__ tile_first, int W, int64_t b) {
    const int r = rank_of(tile_first, W, b);
    SortTile t;
    t.first = tile_first[r];
    t.j = (int32_t)(b - t.first);
    t.seg_tiles = (int32_t)(tile_first[r + 1] - t.first);
    t.start = off[r] + (int64_t)t.j * kSortTile;
    const int64_t left = off[r + 1] - t.start;
    t.count = (int32_t)(left < kSortTile ? left : kSortTile);
    return t;
}

// Digit-indexed LDS tables (a row holds 256 digit values): for one wave's access, digits d
// and d + 32 fall in the same bank, so the lanes' accesses by digit conflict when distinct
// digits of a wave share a bank (the first histogram pass, over near-uniform low length
// bits, spends about one conflict cycle per conflict-free LDS cycle).  Splitting each such
// access into four (or eight) masked steps by the digit's high bits, so that a step's
// digits never share a bank, removed every conflict but made the passes slower (measured
// on 16.7 M samples: 44.4 instead of 38.0 us for a histogram pass, 107.6 instead of 89.8
// us for a scatter pass): the steps cost more issue than the conflicts stall.  The
// accesses are therefore made once, and kept few: one LDS add per distinct digit of a
// wave, one slot read per item.

template <bool kFirst>
__global__ void __launch_bounds__(kBlock) radix_hist_kernel(const int64_t* __restrict__ off,
                                                            const int64_t* __restrict__ tile_first, int W,
                                                            const uint32_t* __restrict__ keys_in,
                                                            const int32_t* __restrict__ len_in, uint32_t maxl,
                                                            int shift, int dbits, uint32_t* __restrict__ counts) {
    const SortTile b = sort_tile(off, tile_first, W, blockIdx.x);
    const int radix = 1 << dbits;
    const uint32_t mask = (uint32_t)radix - 1;
    // one count table per wave: each distinct digit of a wave has one leader lane, the only
    // writer of its entry, which adds the digit's count (an LDS add without return: no wait
    // on a read)
    constexpr int kWaves = kBlock / kWave;
    __shared__ uint32_t h[kWaves][256];
    const int w = threadIdx.x / kWave;
    for (int i = threadIdx.x; i < kWaves * 256; i += kBlock) (&h[0][0])[i] = 0;
    __syncthreads();
    for (int it = 0; it < kSortItems; ++it) {
        const int li = it * kBlock + threadIdx.x;
        const bool valid = li < b.count;
        const int64_t p = b.start + li;
        uint32_t key = 0;
        if (valid) key = kFirst ? maxl - (uint32_t)len_in[p] : keys_in[p];
        const uint32_t d = (key >> shift) & mask;
        const uint64_t peers = match_digit(d, valid, dbits);
        const bool lead = valid && lanes_below(peers) == 0;
        const uint32_t c = (uint32_t)__popcll(peers);
        if (lead) atomicAdd(&h[w][d], c);
    }
    __syncthreads();
    const int64_t col = (int64_t)b.first << dbits;
    for (int d = threadIdx.x; d < radix; d += kBlock) {
        uint32_t sum = 0;
#pragma unroll
        for (int k = 0; k < kWaves; ++k) sum += h[k][d];
        counts[col + (int64_t)d * b.seg_tiles + b.j] = sum;
    }
}

// Scatter one tile.  Items are taken in position order (round `it` covers positions
// it*256 .. it*256+255 of the tile, wave w its w-th quarter), so the slot of an item among
// equal digits is: the digit's first slot after earlier rounds (s_run), plus the items of
// earlier waves this round (both folded into s_pre by one thread per digit), plus lower
// lanes with the same digit (ballot match).  That keeps the sort stable.  The items are first
// placed in LDS in digit order (the tile's local digit offsets come from the scanned
// counts: consecutive entries differ by one tile's count of one digit), then written out
// in that order, so each digit's run of the tile goes to consecutive addresses: a round
// holds about two items per digit, and writing those straight from registers cost 4.6 B
// of HBM writes per byte written.
template <bool kFirst, bool kLast>
__global__ void __launch_bounds__(kBlock) radix_scatter_kernel(
    const int64_t* __restrict__ off, const int64_t* __restrict__ tile_first, int W,
    const uint32_t* __restrict__ keys_in,
    const int32_t* __restrict__ len_in, const int32_t* __restrict__ vals_in, uint32_t maxl, int shift,
    int dbits, const uint32_t* __restrict__ offs, uint32_t* __restrict__ keys_out,
    int32_t* __restrict__ vals_out, int32_t* __restrict__ slen_out) {
    const SortTile b = sort_tile(off, tile_first, W, blockIdx.x);
    const int radix = 1 << dbits;
    const uint32_t mask = (uint32_t)radix - 1;
    constexpr int kWaves = kBlock / kWave;
    __shared__ uint32_t s_base[256];   // global position of the tile's first item of digit d
    __shared__ uint32_t s_local[256];  // local position of the same item within the tile
    __shared__ uint32_t s_run[256];    // local slot of the next item of digit d
    __shared__ uint32_t s_w[kWaves][256];    // this round: items of digit d in wave k
    __shared__ uint32_t s_pre[kWaves][256];  // this round: local slot of wave k's first item of digit d
    __shared__ uint32_t s_key[kSortTile];
    __shared__ int32_t s_val[kSortTile];
    const int64_t col = (int64_t)b.first << dbits;
    for (int d = threadIdx.x; d < 256; d += kBlock) {
        uint32_t base = 0, cnt = 0;
        if (d < radix) {
            const int64_t i = col + (int64_t)d * b.seg_tiles + b.j;
            base = offs[i];
            cnt = offs[i + 1] - base;
        }
        s_base[d] = base;
        s_local[d] = cnt;
        s_run[d] = 0;
#pragma unroll
        for (int k = 0; k < kWaves; ++k) s_w[k][d] = 0;
    }
    __syncthreads();
    {
        // exclusive scan of the tile's digit counts (256 entries, one per thread)
        uint32_t tot;
        const uint32_t ex = block_excl_sum(s_local[threadIdx.x], &tot);
        __syncthreads();
        s_local[threadIdx.x] = ex;
        s_run[threadIdx.x] = ex;
    }
    __syncthreads();
    const int w = threadIdx.x / kWave;
    for (int it = 0; it < kSortItems; ++it) {
        const int li = it * kBlock + threadIdx.x;
        const bool valid = li < b.count;
        const int64_t p = b.start + li;
        uint32_t key = 0;
        int32_t val = 0;
        if (valid) {
            key = kFirst ? maxl - (uint32_t)len_in[p] : keys_in[p];
            val = kFirst ? (int32_t)p : vals_in[p];
        }
        const uint32_t d = (key >> shift) & mask;
        const uint64_t peers = match_digit(d, valid, dbits);
        const uint32_t below = lanes_below(peers);
        const bool lead = valid && below == 0;
        const uint32_t c = (uint32_t)__popcll(peers);
        // the wave's count of each digit (leaders), then one thread per digit turns the
        // waves' counts into each wave's first slot, and each item reads its wave's slot
        // for its digit
        if (lead) s_w[w][d] = c;
        __syncthreads();
        for (int dd = threadIdx.x; dd < radix; dd += kBlock) {
            uint32_t at = s_run[dd];
#pragma unroll
            for (int k = 0; k < kWaves; ++k) {
                const uint32_t v = s_w[k][dd];
                s_pre[k][dd] = at;
                s_w[k][dd] = 0;
                at += v;
            }
            s_run[dd] = at;
        }
        __syncthreads();
        uint32_t q = 0;
        if (valid) q = s_pre[w][d] + below;
        if (valid) {
            s_key[q] = key;
            s_val[q] = val;
        }
    }
    __syncthreads();
    for (int q = threadIdx.x; q < b.count; q += kBlock) {
        const uint32_t key = s_key[q];
        const uint32_t d = (key >> shift) & mask;
        const uint32_t pos = s_base[d] + (uint32_t)q - s_local[d];
        vals_out[pos] = s_val[q];
        if (kLast)
            slen_out[pos] = (int32_t)(maxl - key);
        else
            keys_out[pos] = key;
    }
}

__global__ void __launch_bounds__(kBlock) identity_order_kernel(int64_t n, const int32_t* __restrict__ len,
                                                                int32_t* __restrict__ order,
                                                                int32_t* __restrict__ slen) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; p < n; p += stride) {
        order[p] = (int32_t)p;
        slen[p] = len[p];
    }
}

// next-group-start links over the current sequences; positions outside every rank's
// live range [off[r], off[r] + cnt_r) and links leaving a rank point to the sentinel n.
__global__ void __launch_bounds__(kBlock) links_kernel(const int32_t* __restrict__ slen,
                                                       const int64_t* __restrict__ off,
                                                       const RankState* __restrict__ ranks, int W, int64_t n,
                                                       int64_t budget, int32_t* __restrict__ jmp,
                                                       uint8_t* __restrict__ marks) {
    __shared__ int64_t s_off[kLdsRanks + 1];
    off = stage_ranks(off, W, s_off);
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; p <= n; p += stride) {
        if (p == n) {
            jmp[n] = (int32_t)n;
            marks[n] = 0;
            continue;
        }
        const int r = rank_of(off, W, p);
        const int64_t base = off[r];
        const int64_t c = ranks[r].cnt;
        const int64_t q = p - base;
        if (q >= c) {
            jmp[p] = (int32_t)n;
            marks[p] = 0;
            continue;
        }
        const int64_t step = q == 0 ? 1 : batch_size(budget, slen[p - 1]);
        const int64_t t = p + step;
        jmp[p] = (int32_t)(t < base + c ? t : n);
        marks[p] = q == 0 ? 1 : 0;
    }
}

// One doubling round: m <- m U J(m), J <- J o J.  Marks are updated in place (a mark seen
// early only propagates sooner; every marked position is still a chain element), the
// jump table is double-buffered.  A round starts only if the previous one marked
// something new; otherwise the marks are already closed under J and it returns at once.
__global__ void __launch_bounds__(kBlock) jump_kernel(const int32_t* __restrict__ jin,
                                                      int32_t* __restrict__ jout, uint8_t* marks, int64_t n,
                                                      DevStatus* st, int round) {
    if (round > 0 && st->jump_changed[round - 1] == 0) return;
    bool changed = false;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; p <= n; p += stride) {
        const int32_t j = jin[p];
        if (p < n && j < n && marks[p] && !marks[j]) {
            marks[j] = 1;
            changed = true;
        }
        jout[p] = j < n ? jin[j] : (int32_t)n;
    }
    if (__ballot(changed) && (threadIdx.x & (kWave - 1)) == 0) st->jump_changed[round] = 1;
}

// ---- run-table chain walk
// Positions q >= 1 of a rank (q < cnt_r) fall into runs of equal step: q starts a run when
// q = 1 or its step B(l[q - 1]) differs from the step of q - 1.  The chain's group starts
// are q = 0 and, in run k, the positions c_k, c_k + b_k, ... of the run, where b_k is the
// run's step and c_k its first chain position (none if the chain jumps over the run).  The
// group index of a position is the number of group starts at or before it, minus one.
// Rank r's run table (run k: start, step, first chain position, group starts before the
// run) sits at positions off[r] + k of four position-indexed arrays (a rank has fewer runs
// than positions).  Work is split into the sort's tiles (at most kSortTile positions of
// one rank).
constexpr int kRunCap = 4096;   // runs per rank held in LDS by run_chase_kernel

// Whether rank-local position q (global p) starts a run.
__device__ __forceinline__ bool run_start_at(const int32_t* __restrict__ slen, int64_t p, int64_t q, int64_t cnt,
                                             int64_t budget) {
    if (q < 1 || q >= cnt) return false;
    return q == 1 || batch_size(budget, slen[p - 1]) != batch_size(budget, slen[p - 2]);
}

struct RunTile {
    int r;
    int64_t base;    // off[r]
    int64_t start;   // first position of the tile
    int32_t count;   // positions of the tile
    int64_t cnt;     // live positions of the rank
};

__device__ __forceinline__ RunTile run_tile(const int64_t* __restrict__ off, const int64_t* __restrict__ tile_first,
                                            int W, const RankState* __restrict__ ranks, int64_t b) {
    RunTile t;
    t.r = rank_of(tile_first, W, b);
    t.base = off[t.r];
    t.start = t.base + (b - tile_first[t.r]) * kSortTile;
    const int64_t left = off[t.r + 1] - t.start;
    t.count = (int32_t)(left < kSortTile ? left : kSortTile);
    t.cnt = ranks[t.r].cnt;
    return t;
}

// Run starts per tile.
__global__ void __launch_bounds__(kBlock) run_count_kernel(const int64_t* __restrict__ off,
                                                           const int64_t* __restrict__ tile_first, int W,
                                                           const RankState* __restrict__ ranks,
                                                           const int32_t* __restrict__ slen, int64_t budget,
                                                           uint32_t* __restrict__ tile_runs) {
    const RunTile t = run_tile(off, tile_first, W, ranks, blockIdx.x);
    uint32_t c = 0;
    for (int i = threadIdx.x; i < t.count; i += kBlock)
        c += run_start_at(slen, t.start + i, t.start + i - t.base, t.cnt, budget);
    c = block_sum(c);
    if (threadIdx.x == 0) tile_runs[blockIdx.x] = c;
}

// One block per rank: the rank's tile counts become the index of each tile's first run
// (in place), and rank_runs[r] the rank's number of runs.
__global__ void __launch_bounds__(kBlock) run_tile_scan_kernel(const int64_t* __restrict__ tile_first,
                                                               uint32_t* __restrict__ tile_runs,
                                                               uint32_t* __restrict__ rank_runs) {
    const int r = blockIdx.x;
    const int64_t t0 = tile_first[r], t1 = tile_first[r + 1];
    uint32_t carry = 0;
    for (int64_t b = t0; b < t1; b += kBlock) {
        const int64_t t = b + threadIdx.x;
        const uint32_t v = t < t1 ? tile_runs[t] : 0u;
        uint32_t tot;
        const uint32_t ex = block_excl_sum(v, &tot);
        if (t < t1) tile_runs[t] = carry + ex;
        carry += tot;
    }
    if (threadIdx.x == 0) rank_runs[r] = carry;
}

// The run table's starts and steps, written by the tile holding each run start.  A tile's
// positions are taken in rounds of kBlock consecutive positions, so a block scan of the
// round's flags numbers its run starts in position order.
__global__ void __launch_bounds__(kBlock) run_write_kernel(const int64_t* __restrict__ off,
                                                           const int64_t* __restrict__ tile_first, int W,
                                                           const RankState* __restrict__ ranks,
                                                           const int32_t* __restrict__ slen, int64_t budget,
                                                           const uint32_t* __restrict__ tile_runs,
                                                           int32_t* __restrict__ run_start,
                                                           int32_t* __restrict__ run_b) {
    const RunTile t = run_tile(off, tile_first, W, ranks, blockIdx.x);
    uint32_t k0 = tile_runs[blockIdx.x];
    for (int i0 = 0; i0 < t.count; i0 += kBlock) {
        const int i = i0 + threadIdx.x;
        const int64_t p = t.start + i;
        const bool f = i < t.count && run_start_at(slen, p, p - t.base, t.cnt, budget);
        uint32_t tot;
        const uint32_t ex = block_excl_sum((uint32_t)f, &tot);
        if (f) {
            const int64_t k = t.base + k0 + ex;
            const int64_t b = batch_size(budget, slen[p - 1]);
            run_start[k] = (int32_t)(p - t.base);
            run_b[k] = (int32_t)(b < INT32_MAX ? b : INT32_MAX);   // any step >= 2^31 leaves the rank
        }
        k0 += tot;
    }
}

// One block per rank: thread 0 walks the chain run by run and records for every run the
// first chain position (INT32_MAX if the chain skips the run) and the group starts before
// the run; G_r is the rank's number of group starts.  Positions and steps stay below 2^31
// (larger steps are stored as INT32_MAX), so the walk runs in 32-bit integers; the table
// and its results sit in LDS when they fit.
__global__ void __launch_bounds__(kBlock) run_chase_kernel(const int64_t* __restrict__ off, RankState* ranks,
                                                           const uint32_t* __restrict__ rank_runs,
                                                           const int32_t* __restrict__ run_start,
                                                           const int32_t* __restrict__ run_b,
                                                           int32_t* __restrict__ run_c, int32_t* __restrict__ run_g) {
    __shared__ uint32_t ls[kRunCap + 1], lb[kRunCap], lc[kRunCap], lg[kRunCap];
    const int r = blockIdx.x;
    const int64_t base = off[r];
    const int64_t c = ranks[r].cnt;
    if (c < 2) {   // no position >= 1, no run: position 0 (if any) is the only group start
        if (threadIdx.x == 0) ranks[r].G = c;
        return;
    }
    const int64_t R = rank_runs[r];
    if (R <= kRunCap) {
        for (int64_t i = threadIdx.x; i < R; i += blockDim.x) {
            ls[i] = (uint32_t)run_start[base + i];
            lb[i] = (uint32_t)run_b[base + i];
        }
        __syncthreads();
        if (threadIdx.x == 0) {
            ls[R] = (uint32_t)c;
            uint32_t cur = 1;     // next(0) = 1: the second group starts at position 1
            uint32_t marks = 1;   // position 0
#pragma unroll 4
            for (int i = 0; i < (int)R; ++i) {
                const uint32_t e = ls[i + 1], b = lb[i];
                const bool hit = cur < e;
                lc[i] = hit ? cur : (uint32_t)INT32_MAX;
                lg[i] = marks;
                // chain positions cur, cur + b, ... below e; the next one is >= e
                const uint32_t k = hit ? (e - cur + b - 1) / b : 0u;
                cur += k * b;
                marks += k;
            }
            ranks[r].G = marks;
        }
        __syncthreads();
        for (int64_t i = threadIdx.x; i < R; i += blockDim.x) {
            run_c[base + i] = (int32_t)lc[i];
            run_g[base + i] = (int32_t)lg[i];
        }
        return;
    }
    if (threadIdx.x != 0) return;
    uint32_t cur = 1, marks = 1;
    for (int64_t i = 0; i < R; ++i) {
        const uint32_t e = (uint32_t)(i + 1 < R ? run_start[base + i + 1] : c);
        const uint32_t b = (uint32_t)run_b[base + i];
        const bool hit = cur < e;
        run_c[base + i] = hit ? (int32_t)cur : INT32_MAX;
        run_g[base + i] = (int32_t)marks;
        const uint32_t k = hit ? (e - cur + b - 1) / b : 0u;
        cur += k * b;
        marks += k;
    }
    ranks[r].G = marks;
}

// One block: every rank's first global group id (exclusive sum of G_r), the group count
// per rank for the caller, and the total in gbase[W].
__global__ void __launch_bounds__(kBlock) rank_groups_kernel(RankState* ranks, int W, int64_t* __restrict__ gbase,
                                                             int32_t* __restrict__ groups_out) {
    int64_t carry = 0;
    for (int b = 0; b < W; b += kBlock) {
        const int r = b + threadIdx.x;
        const int64_t G = r < W ? ranks[r].G : 0;
        int64_t tot;
        const int64_t ex = block_excl_sum(G, &tot);
        if (r < W) {
            ranks[r].gbase = carry + ex;
            gbase[r] = carry + ex;
            if (groups_out) groups_out[r] = (int32_t)G;
        }
        carry += tot;
    }
    if (threadIdx.x == 0) gbase[W] = carry;
}

// Group index of every live position and the global position of every group start, from
// the run table: position q of run k is in the group that starts at the last chain
// position of the run at or before q, or, before c_k, in the last group started before
// the run.
__global__ void __launch_bounds__(kBlock) run_gidx_kernel(const int64_t* __restrict__ off,
                                                          const int64_t* __restrict__ tile_first, int W,
                                                          const RankState* __restrict__ ranks,
                                                          const int32_t* __restrict__ slen, int64_t budget,
                                                          const uint32_t* __restrict__ tile_runs,
                                                          const int32_t* __restrict__ run_b,
                                                          const int32_t* __restrict__ run_c,
                                                          const int32_t* __restrict__ run_g,
                                                          int32_t* __restrict__ gidx, int32_t* __restrict__ gstart) {
    const RunTile t = run_tile(off, tile_first, W, ranks, blockIdx.x);
    const int64_t gb = ranks[t.r].gbase;
    // run starts before the current position in this rank, the current position included
    uint32_t k0 = tile_runs[blockIdx.x];
    for (int i0 = 0; i0 < t.count; i0 += kBlock) {
        const int i = i0 + threadIdx.x;
        const int64_t p = t.start + i;
        const int64_t q = p - t.base;
        const bool live = i < t.count && q < t.cnt;
        const bool f = live && run_start_at(slen, p, q, t.cnt, budget);
        uint32_t tot;
        const uint32_t ex = block_excl_sum((uint32_t)f, &tot);
        if (live) {
            int64_t g = 0;
            bool mark = true;
            if (q > 0) {
                const int64_t k = t.base + k0 + ex + (f ? 1 : 0) - 1;   // q's run
                const uint32_t c = (uint32_t)run_c[k], b = (uint32_t)run_b[k];
                const int64_t G = run_g[k];
                if ((uint32_t)q >= c) {
                    const uint32_t d = (uint32_t)q - c;
                    const uint32_t m = d / b;
                    g = G + m;
                    mark = d - m * b == 0;
                } else {
                    g = G - 1;
                    mark = false;
                }
            }
            gidx[p] = (int32_t)g;
            if (mark) gstart[gb + g] = (int32_t)p;
        }
        k0 += tot;
    }
}

__global__ void init_jump_flags(DevStatus* st) {
    if (threadIdx.x < kMaxJumpRounds) st->jump_changed[threadIdx.x] = 0;
}

struct CountLoad {
    const uint32_t* c;
    int64_t n;  // entries; the scan runs over n + 1 so that entry n holds the total
    __device__ uint32_t operator()(int64_t i) const { return i < n ? c[i] : 0u; }
};
struct CountStore {
    uint32_t* c;
    __device__ void operator()(int64_t i, uint32_t v) const { c[i] = v; }
};

struct MarkLoad {
    const uint8_t* m;
    __device__ uint32_t operator()(int64_t i) const { return m[i]; }
};
struct InclStore {
    const uint8_t* m;
    int32_t* out;
    __device__ void operator()(int64_t i, uint32_t ex) const { out[i] = (int32_t)(ex + m[i]); }
};

__global__ void __launch_bounds__(kBlock) gidx_kernel(const uint8_t* __restrict__ marks,
                                                      const int32_t* __restrict__ incl,
                                                      const int64_t* __restrict__ off,
                                                      const RankState* __restrict__ ranks, int W, int64_t n,
                                                      int32_t* __restrict__ gidx, int32_t* __restrict__ gstart) {
    __shared__ int64_t s_off[kLdsRanks + 1];
    off = stage_ranks(off, W, s_off);
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; p < n; p += stride) {
        const int r = rank_of(off, W, p);
        const int64_t base = off[r];
        if (p - base >= ranks[r].cnt) continue;
        const int32_t before = base > 0 ? incl[base - 1] : 0;
        gidx[p] = incl[p] - before - 1;
        if (marks[p]) gstart[incl[p] - 1] = (int32_t)p;
    }
}

__global__ void groups_kernel(const int32_t* __restrict__ incl, const int64_t* __restrict__ off, int W,
                              RankState* ranks, int64_t* __restrict__ gbase, int32_t* __restrict__ groups_out) {
    for (int r = blockIdx.x * blockDim.x + threadIdx.x; r < W; r += gridDim.x * blockDim.x) {
        const int64_t base = off[r];
        const int64_t c = ranks[r].cnt;
        const int32_t before = base > 0 ? incl[base - 1] : 0;
        const int64_t G = c > 0 ? incl[base + c - 1] - before : 0;
        ranks[r].G = G;
        ranks[r].gbase = before;
        gbase[r] = before;
        if (r == W - 1) gbase[W] = before + G;
        if (groups_out) groups_out[r] = (int32_t)G;
    }
}

// ---- one block per rank
// When every rank holds at most kRankBlockMax samples, each rank is grouped by one
// 1024-thread block in two launches, with no host synchronisation: rank_sort_kernel (lengths, validity, stable LSD
// radix sort on byte digits of the length) and rank_walk_kernel (the group chain over the
// runs of equal batch size, and the group index of every position in closed form).
constexpr int kRankThreads = 1024;
constexpr int kRankWaves = kRankThreads / kWave;
constexpr int kRankItems = 4;                     // lengths a thread loads at once in the first pass
constexpr int kRankGroup = 4;                     // rounds of a pass whose items are loaded together
constexpr int kRankRunCap = 3840;                 // runs of equal batch size a rank may have
// Samples of the largest rank grouped this way.  A block's pass over its rank is bound by
// the issue rate of its one compute unit (every round of 1024 items costs each of its 16
// waves a few hundred instructions: ~2.7 us per round on MI355X), so larger ranks go to the
// multi-block path, whose launches and one synchronisation cost less than a block's
// rounds from about this size on.
constexpr int64_t kRankBlockMax = 16384;

// Exclusive scan of v over the first 256 threads of a kRankThreads block (4 waves), every
// thread of the block taking part in the barriers; *total receives the sum.
__device__ __forceinline__ uint32_t scan256(uint32_t v, uint32_t* total) {
    __shared__ uint32_t s_w[4];
    const int t = threadIdx.x;
    uint32_t inc = 0;
    if (t < 256) {
        inc = wave_scan_dpp<OpAdd>(v);
        if ((t & (kWave - 1)) == kWave - 1) s_w[t / kWave] = inc;
    }
    __syncthreads();
    uint32_t pre = 0, tot = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const uint32_t x = s_w[i];
        pre += (t < 256 && i < t / kWave) ? x : 0u;
        tot += x;
    }
    __syncthreads();
    *total = tot;
    return pre + inc - v;
}

// Per-wave digit counts: for each distinct digit of the wave's valid lanes, the lowest such
// lane adds the number of lanes holding it to row w of `tbl` (one writer per address).
__device__ __forceinline__ void count_digits(uint32_t (*tbl)[256], int w, uint32_t d, bool valid) {
    const uint64_t peers = match_digit(d, valid, 8);
    const bool lead = valid && lanes_below(peers) == 0;
    const uint32_t c = (uint32_t)__popcll(peers);
    if (lead) atomicAdd(&tbl[w][d], c);
}

// One stable scatter pass of rank_sort_kernel over digit bits [shift, shift + 8): round i
// places items i*1024 .. i*1024+1023 of the pass's input (keys sk, ids sv; the first
// pass's ids are the positions themselves).  A round's rank of an item among equal digits
// is: items of that digit placed in earlier rounds (s_run), in lower waves of this round
// (s_cnt prefix) and in lower lanes of its wave (ballot match).  The two barriers of a
// round order LDS only: nothing in the block reads the round's global stores before the
// pass ends.  Loads run a group of kRankGroup rounds ahead, into the register set (A or B)
// of the group after next, at clamped positions (unconditional loads: a load under a branch
// makes the compiler wait for it where the paths join).
template <bool kFirst>
__device__ __forceinline__ void scatter_pass(const int32_t* __restrict__ sk, const int32_t* __restrict__ sv,
                                             int32_t* __restrict__ dk, int32_t* __restrict__ dv, int64_t base,
                                             int cnt, int rounds, int shift, uint32_t (*s_cnt)[256],
                                             uint32_t (*s_pre)[256], uint32_t* s_run) {
    const int t = threadIdx.x, w = t / kWave;
    auto load_group = [&](int g, uint32_t (&kk)[kRankGroup], int32_t (&vv)[kRankGroup]) {
#pragma unroll
        for (int j = 0; j < kRankGroup; ++j) {
            const int q = (g * kRankGroup + j) * kRankThreads + t;
            const int qc = q < cnt ? q : cnt - 1;
            kk[j] = (uint32_t)sk[base + qc];
            vv[j] = kFirst ? (int32_t)(base + q) : sv[base + qc];
        }
    };
    auto place_group = [&](int g, const uint32_t (&kk)[kRankGroup], const int32_t (&vv)[kRankGroup]) {
#pragma unroll
        for (int j = 0; j < kRankGroup; ++j) {
            const int i = g * kRankGroup + j;
            if (i >= rounds) break;   // uniform
            const int q = i * kRankThreads + t;
            const bool valid = q < cnt;
            const uint32_t key = kk[j];
            const uint32_t d = (key >> shift) & 255u;
            const uint64_t peers = match_digit(d, valid, 8);
            const uint32_t below = lanes_below(peers);
            const bool lead = valid && below == 0;
            const uint32_t c_lead = (uint32_t)__popcll(peers);
            if (lead) s_cnt[w][d] = c_lead;
            lds_barrier();
            if (t < 256) {
                // s_pre: where this round's first item of digit t from each wave goes
                // (s_run holds the bucket's start plus the items placed so far)
                uint32_t run = s_run[t];
#pragma unroll
                for (int k2 = 0; k2 < kRankWaves; ++k2) {
                    const uint32_t c = s_cnt[k2][t];
                    s_pre[k2][t] = run;
                    run += c;
                    s_cnt[k2][t] = 0;
                }
                s_run[t] = run;
            }
            lds_barrier();
            uint32_t at = 0;
            if (valid) at = s_pre[w][d];
            if (valid) {
                dk[base + at + below] = (int32_t)key;
                dv[base + at + below] = vv[j];
            }
        }
    };
    const int groups = (rounds + kRankGroup - 1) / kRankGroup;
    uint32_t ka_[kRankGroup], kb_[kRankGroup];
    int32_t va_[kRankGroup], vb_[kRankGroup];
    load_group(0, ka_, va_);
    for (int g = 0; g < groups; g += 2) {
        load_group(g + 1, kb_, vb_);
        place_group(g, ka_, va_);
        if (g + 1 >= groups) break;   // uniform
        load_group(g + 2, ka_, va_);
        place_group(g + 1, kb_, vb_);
    }
}

// Sorts rank r's samples by (length desc, id asc): writes len (every sample's length,
// invalid ones as 1), order and sorted_len.  Digits are the bytes of the length, low to
// high; a digit whose value is the same for every sample of the rank is skipped; each pass
// places the buckets from the highest digit value down and keeps the order within a
// bucket, so the result is by length descending, ties in sample-id order.
__global__ void __launch_bounds__(kRankThreads) rank_sort_kernel(
    const int64_t* __restrict__ tok_off, const int64_t* __restrict__ off, int32_t* __restrict__ len,
    int32_t* __restrict__ ka, int32_t* __restrict__ va, int32_t* __restrict__ kb, int32_t* __restrict__ vb,
    int32_t* __restrict__ order, int32_t* __restrict__ slen, DevStatus* st) {
    __shared__ uint32_t s_cnt[kRankWaves][256];   // first pass: digit-0 counts; passes: counts of a round
    __shared__ uint32_t s_pre[kRankWaves][256];   // first pass: digit-1 counts; passes: prefixes of a round
    __shared__ uint32_t s_hist[4][256];
    __shared__ uint32_t s_run[256];
    __shared__ uint32_t s_max;
    __shared__ unsigned long long s_bad;
    __shared__ int s_active[4];
    const int r = blockIdx.x;
    const int64_t base = off[r];
    const int cnt = (int)(off[r + 1] - base);
    if (cnt <= 0) return;
    const int t = threadIdx.x, w = t / kWave;
    for (int i = t; i < kRankWaves * 256; i += kRankThreads) {
        (&s_cnt[0][0])[i] = 0;
        (&s_pre[0][0])[i] = 0;
    }
    if (t == 0) {
        s_max = 0;
        s_bad = ~0ull;
    }
    __syncthreads();

    // lengths, validity, histograms of digits 0 and 1
    uint32_t lmax = 0;
    unsigned long long bad = ~0ull;
    for (int q0 = 0; q0 < cnt; q0 += kRankThreads * kRankItems) {
        int64_t a[kRankItems], b[kRankItems];
#pragma unroll
        for (int j = 0; j < kRankItems; ++j) {
            const int q = q0 + j * kRankThreads + t;
            const int qc = q < cnt ? q : cnt - 1;
            a[j] = tok_off[base + qc];
            b[j] = tok_off[base + qc + 1];
        }
#pragma unroll
        for (int j = 0; j < kRankItems; ++j) {
            const int q = q0 + j * kRankThreads + t;
            const bool valid = q < cnt;
            uint32_t l = 0;
            if (valid) {
                int64_t ll = b[j] - a[j];
                if (ll < 1 || ll > INT_MAX || a[j] < 0) {
                    const unsigned long long id = (unsigned long long)(base + q);
                    bad = id < bad ? id : bad;
                    ll = 1;
                }
                l = (uint32_t)ll;
                len[base + q] = (int32_t)l;
                lmax = l > lmax ? l : lmax;
            }
            count_digits(s_cnt, w, l & 255u, valid);
            count_digits(s_pre, w, (l >> 8) & 255u, valid);
        }
    }
    lmax = wave_scan_dpp<OpMax>(lmax);
    if ((t & (kWave - 1)) == kWave - 1) atomicMax(&s_max, lmax);
    if (bad != ~0ull) atomicMin(&s_bad, bad);
    __syncthreads();
    if (t < 512) {
        const int d = t & 255;
        uint32_t (*tbl)[256] = t < 256 ? s_cnt : s_pre;
        uint32_t sum = 0;
#pragma unroll
        for (int k = 0; k < kRankWaves; ++k) {
            sum += tbl[k][d];
            tbl[k][d] = 0;
        }
        s_hist[t / 256][d] = sum;
    }
    if (t == 0 && s_bad != ~0ull) {
        atomicOr(&st->err, kErrLength);
        atomicMin((unsigned long long*)&st->first_bad, s_bad);
    }
    __syncthreads();
    const uint32_t maxl = s_max;
    if (maxl >= (1u << 16)) {
        // lengths of 2^16 or more: histograms of digits 2 and 3
        for (int q0 = 0; q0 < cnt; q0 += kRankThreads) {
            const int q = q0 + t;
            const bool valid = q < cnt;
            const uint32_t l = valid ? (uint32_t)len[base + q] : 0u;
            count_digits(s_cnt, w, (l >> 16) & 255u, valid);
            count_digits(s_pre, w, l >> 24, valid);
        }
        __syncthreads();
        if (t < 512) {
            const int d = t & 255;
            uint32_t (*tbl)[256] = t < 256 ? s_cnt : s_pre;
            uint32_t sum = 0;
#pragma unroll
            for (int k = 0; k < kRankWaves; ++k) {
                sum += tbl[k][d];
                tbl[k][d] = 0;
            }
            s_hist[2 + t / 256][d] = sum;
        }
    } else if (t < 512) {
        s_hist[2 + t / 256][t & 255] = (t & 255) == 0 ? (uint32_t)cnt : 0u;
    }
    __syncthreads();
    // a digit takes part if more than one of its values occurs
    if (t < 4 * kWave) {
        const int k = t / kWave, lane = t & (kWave - 1);
        int nz = 0;
        for (int d = lane; d < 256; d += kWave) nz += s_hist[k][d] != 0;
        nz = wave_sum(nz);
        if (lane == 0) s_active[k] = nz > 1;
    }
    __syncthreads();
    int passes = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) passes += s_active[k];

    if (passes == 0) {   // every length equal: formation order is id order
        for (int q = t; q < cnt; q += kRankThreads) {
            order[base + q] = (int32_t)(base + q);
            slen[base + q] = len[base + q];
        }
        return;
    }
    int pass = 0;
    const int rounds = (cnt + kRankThreads - 1) / kRankThreads;
    for (int k = 0; k < 4; ++k) {
        if (!s_active[k]) continue;
        const bool first = pass == 0, last = pass == passes - 1;
        const int32_t* sk = first ? len : ((pass & 1) ? ka : kb);
        const int32_t* sv = (pass & 1) ? va : vb;
        int32_t* dk = last ? slen : ((pass & 1) ? kb : ka);
        int32_t* dv = last ? order : ((pass & 1) ? vb : va);
        // bucket of digit value d starts after every higher value's samples
        {
            uint32_t tot;
            const uint32_t v = t < 256 ? s_hist[k][255 - t] : 0u;
            const uint32_t ex = scan256(v, &tot);
            if (t < 256) s_run[255 - t] = ex;
        }
        __syncthreads();
        if (first)
            scatter_pass<true>(sk, sk, dk, dv, base, cnt, rounds, 8 * k, s_cnt, s_pre, s_run);
        else
            scatter_pass<false>(sk, sv, dk, dv, base, cnt, rounds, 8 * k, s_cnt, s_pre, s_run);
        __syncthreads();
        ++pass;
    }
}

// Batch size B(l) (Eq. 1), clipped to 2^31 - 1 (any larger step leaves the rank).
__device__ __forceinline__ uint32_t step_of(int32_t l, int64_t budget) {
    const int64_t b = batch_size(budget, l);
    return (uint32_t)(b < INT32_MAX ? b : INT32_MAX);
}

// Calls f(q, step) for every run start q in [lo, hi) (1 <= lo < hi <= cnt), in order: q = 1,
// and every q whose step B(l[q-1]) differs from the previous position's B(l[q-2]).  Loads
// eight lengths at a time, at clamped positions, so the loads of a batch are in flight
// together; equal neighbouring lengths skip the divisions.
template <typename F>
__device__ __forceinline__ void chunk_run_starts(const int32_t* __restrict__ slen, int64_t base, int lo, int hi,
                                                 int64_t budget, F f) {
    int32_t lp = lo >= 2 ? slen[base + lo - 2] : 0;
    uint32_t bp = lo >= 2 ? step_of(lp, budget) : 0u;
    for (int q0 = lo; q0 < hi; q0 += 8) {
        int32_t l8[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int qq = q0 + j < hi ? q0 + j : hi - 1;
            l8[j] = slen[base + qq - 1];
        }
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int q = q0 + j;
            if (q >= hi) break;
            const int32_t l = l8[j];
            if (q == 1) {
                bp = step_of(l, budget);
                f(q, bp);
            } else if (l != lp) {
                const uint32_t b = step_of(l, budget);
                if (b != bp) f(q, b);
                bp = b;
            }
            lp = l;
        }
    }
}

// Group chain of rank r from its sorted lengths.  Positions q >= 1 fall into runs of equal
// step B(l[q-1]) (the lengths are sorted, so the step never decreases along the rank).
// Inside a run of step b the chain advances by b, so one thread walks the runs and records
// each run's first chain position c; then every position's group index follows in closed
// form: the chain positions before its run, plus those of its run up to it.
__global__ void __launch_bounds__(kRankThreads) rank_walk_kernel(const int64_t* __restrict__ off,
                                                                 const int32_t* __restrict__ slen, int64_t budget,
                                                                 int32_t* __restrict__ gidx,
                                                                 int32_t* __restrict__ groups_out, DevStatus* st) {
    __shared__ uint32_t s_start[kRankRunCap + 1], s_b[kRankRunCap], s_c[kRankRunCap], s_gb[kRankRunCap];
    const int r = blockIdx.x;
    const int64_t base = off[r];
    const int cnt = (int)(off[r + 1] - base);
    const int t = threadIdx.x;
    if (cnt <= 1) {
        if (t == 0) {
            if (cnt == 1) gidx[base] = 0;
            groups_out[r] = cnt;
        }
        return;
    }
    // run starts: every thread checks a chunk of positions [1, cnt); the step is monotone, so
    // a chunk whose first position and last position have the step of the position before
    // it holds no run start
    const int span = cnt - 1;
    const int per = (span + kRankThreads - 1) / kRankThreads;
    const int lo = 1 + t * per;
    const int hi = lo + per < cnt ? lo + per : cnt;
    const bool busy = lo < hi && (lo == 1 || step_of(slen[base + lo - 2], budget) !=
                                                 step_of(slen[base + hi - 2], budget));
    uint32_t mine = 0;
    if (busy) chunk_run_starts(slen, base, lo, hi, budget, [&](int, uint32_t) { ++mine; });
    // exclusive scan of the per-thread counts over the block
    __shared__ uint32_t s_wsum[kRankWaves];
    __shared__ uint32_t s_total;
    uint32_t inc = wave_scan_dpp<OpAdd>(mine);
    if ((t & (kWave - 1)) == kWave - 1) s_wsum[t / kWave] = inc;
    __syncthreads();
    uint32_t pre = 0, tot = 0;
#pragma unroll
    for (int i = 0; i < kRankWaves; ++i) {
        pre += i < t / kWave ? s_wsum[i] : 0u;
        tot += s_wsum[i];
    }
    const uint32_t at0 = pre + inc - mine;
    if (tot > (uint32_t)kRankRunCap) {
        // more runs than the table holds (the host picks this path only when that cannot
        // happen): report, and leave the rank without groups
        if (t == 0) {
            atomicOr(&st->err, kErrInternal);
            groups_out[r] = 0;
        }
        return;
    }
    if (mine) {
        uint32_t at = at0;
        chunk_run_starts(slen, base, lo, hi, budget, [&](int q, uint32_t b) {
            s_start[at] = (uint32_t)q;
            s_b[at] = b;
            ++at;
        });
    }
    const int R = (int)tot;
    if (t == 0) s_start[R] = (uint32_t)cnt;
    __syncthreads();
    if (t == 0) {
        // positions, steps and their sums stay below 2^32 (positions < 2^31, steps <= 2^31 - 1),
        // so the walk runs on 32-bit division
        uint32_t cur = 1;   // next(0) = 1: the second group starts at position 1
        for (int i = 0; i < R; ++i) {
            const uint32_t e = s_start[i + 1], b = s_b[i];
            const bool hit = cur < e;
            s_c[i] = hit ? cur : 0xFFFFFFFFu;
            const uint32_t k = hit ? (e - cur + b - 1) / b : 0u;
            cur += k * b;
        }
    }
    __syncthreads();
    // chain positions per run and their exclusive prefix (runs dealt round robin over threads)
    {
        uint32_t carry = 0;
        for (int i0 = 0; i0 < R; i0 += kRankThreads) {
            const int i = i0 + t;
            uint32_t ng = 0;
            if (i < R) {
                const uint32_t c = s_c[i], e = s_start[i + 1], b = s_b[i];
                ng = c < e ? (e - c + b - 1) / b : 0u;
            }
            const uint32_t inc2 = wave_scan_dpp<OpAdd>(ng);
            __syncthreads();
            if ((t & (kWave - 1)) == kWave - 1) s_wsum[t / kWave] = inc2;
            __syncthreads();
            uint32_t pre2 = 0, tot2 = 0;
#pragma unroll
            for (int w2 = 0; w2 < kRankWaves; ++w2) {
                pre2 += w2 < t / kWave ? s_wsum[w2] : 0u;
                tot2 += s_wsum[w2];
            }
            if (i < R) s_gb[i] = carry + pre2 + inc2 - ng;
            carry += tot2;
        }
        if (t == 0) s_total = carry;
    }
    __syncthreads();
    // group index of every position: chain positions up to it, minus one
    for (int q = t; q < cnt; q += kRankThreads) {
        int32_t g = 0;
        if (q > 0) {
            int a = 0, z = R;   // last run with start <= q: s_start[a] <= q < s_start[z]
            while (z - a > 1) {
                const int m = (a + z) >> 1;
                if (s_start[m] <= (uint32_t)q) a = m; else z = m;
            }
            const uint32_t c = s_c[a];
            g = (int32_t)(s_gb[a] + ((uint32_t)q >= c ? ((uint32_t)q - c) / s_b[a] + 1u : 0u));
        }
        gidx[base + q] = g;
    }
    if (t == 0) groups_out[r] = (int32_t)(1 + s_total);
}

}  // namespace

// Distinct steps a rank's sorted sequence can hold: at most the distinct values of
// floor(budget / l), i.e. at most 2 sqrt(budget) + 1, at most the number of distinct
// lengths (len_range, if known, else 0) and at most the rank's positions.
static int64_t runs_bound(int64_t budget, int64_t max_cnt, int64_t len_range) {
    int64_t b = 2 * ((int64_t)std::sqrt((double)budget) + 1) + 1;
    if (len_range > 0 && len_range < b) b = len_range;
    if (max_cnt < b) b = max_cnt;
    return b;
}

// Mark scan, group index of every position, global group starts, G_r.
static int finish_groups(const Layout& L, void* ws, int W, int64_t n, const int64_t* d_off, int32_t* d_gidx,
                         int32_t* d_groups_out, RankState* d_ranks, hipStream_t s) {
    uint8_t* marks = ws_at<uint8_t>(ws, L.marks);
    int32_t* incl = ws_at<int32_t>(ws, L.incl);
    int32_t* gstart = ws_at<int32_t>(ws, L.gstart);
    ODB_TRY((device_excl_scan<uint32_t>(MarkLoad{marks}, InclStore{marks, incl}, n,
                                        ws_at<uint32_t>(ws, L.partials), s)));
    hipLaunchKernelGGL(gidx_kernel, dim3(grid_for(n, kBlock, (int64_t)num_cus() * kPlanBlocksPerCU)), dim3(kBlock), 0, s,
                       (const uint8_t*)marks, (const int32_t*)incl, d_off, (const RankState*)d_ranks, W, n,
                       d_gidx, gstart);
    ODB_LAUNCHED();
    hipLaunchKernelGGL(groups_kernel, dim3(grid_for(W, kBlock)), dim3(kBlock), 0, s, (const int32_t*)incl, d_off,
                       W, d_ranks, ws_at<int64_t>(ws, L.gbase), d_groups_out);
    ODB_LAUNCHED();
    return ODB_OK;
}

int group_sequences(const Layout& L, void* ws, int W, int64_t n, int64_t budget, const int64_t* d_off,
                    int64_t max_cnt, int64_t len_range, bool tiles_ready, const int32_t* d_slen, int32_t* d_gidx,
                    int32_t* d_groups_out, RankState* d_ranks, hipStream_t s) {
    int32_t* j0 = ws_at<int32_t>(ws, L.jmp0);
    int32_t* j1 = ws_at<int32_t>(ws, L.jmp1);
    uint8_t* marks = ws_at<uint8_t>(ws, L.marks);
    int32_t* incl = ws_at<int32_t>(ws, L.incl);
    DevStatus* st = ws_at<DevStatus>(ws, L.status);
    const unsigned grid = grid_for(n + 1, kBlock, (int64_t)num_cus() * kPlanBlocksPerCU);
    if (runs_bound(budget, max_cnt, len_range) <= kRunCap && n < INT32_MAX) {
        // run-table walk over the sort's tiles
        int64_t* d_tile_first = ws_at<int64_t>(ws, L.tile_first);
        if (!tiles_ready) {
            hipLaunchKernelGGL(sort_tiles_kernel, dim3(1), dim3(kBlock), 0, s, d_off, W, d_tile_first);
            ODB_LAUNCHED();
        }
        const unsigned tiles = (unsigned)L.num_sort_blocks;
        uint32_t* tile_runs = ws_at<uint32_t>(ws, L.counts);
        uint32_t* rank_runs = ws_at<uint32_t>(ws, L.rank_runs);
        int32_t* run_start = j0;
        int32_t* run_b = j1;
        int32_t* run_c = ws_at<int32_t>(ws, L.gsize);
        int32_t* run_g = incl;
        const RankState* cr = d_ranks;
        if (tiles > 0) {
            hipLaunchKernelGGL(run_count_kernel, dim3(tiles), dim3(kBlock), 0, s, d_off, (const int64_t*)d_tile_first,
                               W, cr, d_slen, budget, tile_runs);
            ODB_LAUNCHED();
        }
        hipLaunchKernelGGL(run_tile_scan_kernel, dim3(W), dim3(kBlock), 0, s, (const int64_t*)d_tile_first, tile_runs,
                           rank_runs);
        ODB_LAUNCHED();
        if (tiles > 0) {
            hipLaunchKernelGGL(run_write_kernel, dim3(tiles), dim3(kBlock), 0, s, d_off, (const int64_t*)d_tile_first,
                               W, cr, d_slen, budget, (const uint32_t*)tile_runs, run_start, run_b);
            ODB_LAUNCHED();
        }
        hipLaunchKernelGGL(run_chase_kernel, dim3(W), dim3(kBlock), 0, s, d_off, d_ranks, (const uint32_t*)rank_runs,
                           (const int32_t*)run_start, (const int32_t*)run_b, run_c, run_g);
        ODB_LAUNCHED();
        hipLaunchKernelGGL(rank_groups_kernel, dim3(1), dim3(kBlock), 0, s, d_ranks, W, ws_at<int64_t>(ws, L.gbase),
                           d_groups_out);
        ODB_LAUNCHED();
        if (tiles > 0) {
            hipLaunchKernelGGL(run_gidx_kernel, dim3(tiles), dim3(kBlock), 0, s, d_off, (const int64_t*)d_tile_first,
                               W, cr, d_slen, budget, (const uint32_t*)tile_runs, (const int32_t*)run_b,
                               (const int32_t*)run_c, (const int32_t*)run_g, d_gidx, ws_at<int32_t>(ws, L.gstart));
            ODB_LAUNCHED();
        }
        return ODB_OK;
    }
    hipLaunchKernelGGL(links_kernel, dim3(grid), dim3(kBlock), 0, s, d_slen, d_off,
                       (const RankState*)d_ranks, W, n, budget, j0, marks);
    ODB_LAUNCHED();
    // chains have at most max_cnt elements: ceil(log2(max_cnt + 1)) + 1 doubling rounds
    // always suffice; rounds after convergence return immediately
    int rounds = 1;
    while ((int64_t(1) << (rounds - 1)) <= max_cnt && rounds < kMaxJumpRounds) ++rounds;
    hipLaunchKernelGGL(init_jump_flags, dim3(1), dim3(64), 0, s, st);
    ODB_LAUNCHED();
    for (int k = 0; k < rounds; ++k) {
        const int32_t* jin = (k & 1) ? j1 : j0;
        int32_t* jout = (k & 1) ? j0 : j1;
        hipLaunchKernelGGL(jump_kernel, dim3(grid), dim3(kBlock), 0, s, jin, jout, marks, n, st, k);
        ODB_LAUNCHED();
    }
    return finish_groups(L, ws, W, n, d_off, d_gidx, d_groups_out, d_ranks, s);
}

}  // namespace odb

using namespace odb;

extern "C" int odb_form_groups(const odb_window_t* w, int64_t budget, int32_t* d_order, int32_t* d_sorted_len,
                               int32_t* d_group_index, int32_t* d_groups_per_rank, void* d_ws, size_t ws_bytes,
                               void* stream) {
    Layout L;
    ODB_TRY(check_workspace(w, d_ws, ws_bytes, &L));
    if (budget < 1) return set_error(ODB_E_INVALID_ARG, "budget must be >= 1");
    const int W = w->num_ranks;
    const int64_t n = w->num_samples;
    if (n > 0 && (!d_order || !d_sorted_len || !d_group_index))
        return set_error(ODB_E_INVALID_ARG, "stage-1 output pointers must not be NULL");
    if (!d_groups_per_rank) return set_error(ODB_E_INVALID_ARG, "d_groups_per_rank is NULL");
    hipStream_t s = static_cast<hipStream_t>(stream);
    ODB_TRY(upload_small(w, L, d_ws, nullptr, s));
    const int64_t* d_off = ws_at<int64_t>(d_ws, L.rank_off);
    RankState* d_ranks = ws_at<RankState>(d_ws, L.ranks);
    DevStatus* st = ws_at<DevStatus>(d_ws, L.status);
    int32_t* len = ws_at<int32_t>(d_ws, L.len);
    int64_t max_cnt = 0;
    for (int r = 0; r < W; ++r) {
        const int64_t c = w->rank_offsets[r + 1] - w->rank_offsets[r];
        if (c > max_cnt) max_cnt = c;
    }

    // one block per rank: two launches, no synchronisation (invalid lengths are grouped as
    // length 1 and reported by odb_align_groups)
    if (max_cnt <= kRankBlockMax && runs_bound(budget, max_cnt, 0) <= kRankRunCap) {
        hipLaunchKernelGGL(rank_sort_kernel, dim3(W), dim3(kRankThreads), 0, s, w->d_token_offsets, d_off, len,
                           ws_at<int32_t>(d_ws, L.keys0), ws_at<int32_t>(d_ws, L.vals0), ws_at<int32_t>(d_ws, L.keys1),
                           ws_at<int32_t>(d_ws, L.vals1), d_order, d_sorted_len, st);
        ODB_LAUNCHED();
        hipLaunchKernelGGL(rank_walk_kernel, dim3(W), dim3(kRankThreads), 0, s, d_off, (const int32_t*)d_sorted_len,
                           budget, d_group_index, d_groups_per_rank, st);
        ODB_LAUNCHED();
        return ODB_OK;
    }
    hipLaunchKernelGGL(rank_counts_kernel, dim3(grid_for(W, kBlock)), dim3(kBlock), 0, s, d_off, W, d_ranks);
    ODB_LAUNCHED();

    // (a1) lengths and their validity; the one synchronisation of this call
    hipLaunchKernelGGL(lengths_kernel, dim3(grid_for(n, kBlock, (int64_t)num_cus() * kPlanBlocksPerCU)), dim3(kBlock), 0, s,
                       w->d_token_offsets, n, len, st);
    ODB_LAUNCHED();
    DevStatus hs;
    ODB_TRY_HIP(hipMemcpyAsync(&hs, st, sizeof(DevStatus), hipMemcpyDeviceToHost, s));
    ODB_TRY_HIP(hipStreamSynchronize(s));
    if (hs.err & kErrLength)
        return set_error(ODB_E_INVALID_DATA,
                         "sample %lld has a length outside [1, 2^31) or a negative token offset",
                         (long long)hs.first_bad);
    if (n == 0) {
        hipLaunchKernelGGL(groups_kernel, dim3(grid_for(W, kBlock)), dim3(kBlock), 0, s,
                           (const int32_t*)len, d_off, W, d_ranks, ws_at<int64_t>(d_ws, L.gbase), d_groups_per_rank);
        ODB_LAUNCHED();
        return ODB_OK;
    }

    // (a2) segmented stable radix sort on key = max_l - l
    const uint32_t maxl = hs.max_len, minl = hs.min_len;
    int bits = 0;
    while (bits < 32 && ((maxl - minl) >> bits) != 0) ++bits;
    const int passes = (bits + 7) / 8;
    if (passes == 0) {
        hipLaunchKernelGGL(identity_order_kernel, dim3(grid_for(n, kBlock, (int64_t)num_cus() * kPlanBlocksPerCU)), dim3(kBlock),
                           0, s, n, (const int32_t*)len, d_order, d_sorted_len);
        ODB_LAUNCHED();
    } else {
        const int dbits = (bits + passes - 1) / passes;
        const int64_t NB = L.num_sort_blocks;
        int64_t* d_tile_first = ws_at<int64_t>(d_ws, L.tile_first);
        hipLaunchKernelGGL(sort_tiles_kernel, dim3(1), dim3(kBlock), 0, s, d_off, W, d_tile_first);
        ODB_LAUNCHED();
        uint32_t* counts = ws_at<uint32_t>(d_ws, L.counts);
        uint32_t* keys[2] = {ws_at<uint32_t>(d_ws, L.keys0), ws_at<uint32_t>(d_ws, L.keys1)};
        int32_t* vals[2] = {ws_at<int32_t>(d_ws, L.vals0), ws_at<int32_t>(d_ws, L.vals1)};
        for (int pass = 0; pass < passes; ++pass) {
            const int shift = pass * dbits;
            const bool first = pass == 0, last = pass == passes - 1;
            const uint32_t* kin = first ? nullptr : keys[(pass - 1) & 1];
            const int32_t* vin = first ? nullptr : vals[(pass - 1) & 1];
            uint32_t* kout = last ? nullptr : keys[pass & 1];
            int32_t* vout = last ? d_order : vals[pass & 1];
            if (first)
                hipLaunchKernelGGL(radix_hist_kernel<true>, dim3((unsigned)NB), dim3(kBlock), 0, s, d_off,
                                   (const int64_t*)d_tile_first, W, kin, (const int32_t*)len, maxl, shift, dbits,
                                   counts);
            else
                hipLaunchKernelGGL(radix_hist_kernel<false>, dim3((unsigned)NB), dim3(kBlock), 0, s, d_off,
                                   (const int64_t*)d_tile_first, W, kin, (const int32_t*)len, maxl, shift, dbits,
                                   counts);
            ODB_LAUNCHED();
            ODB_TRY((device_excl_scan<uint32_t>(CountLoad{counts, NB << dbits}, CountStore{counts}, (NB << dbits) + 1,
                                                ws_at<uint32_t>(d_ws, L.partials), s)));
#define ODB_SCATTER(F, La)                                                                                  \
    hipLaunchKernelGGL((radix_scatter_kernel<F, La>), dim3((unsigned)NB), dim3(kBlock), 0, s,               \
                       d_off, (const int64_t*)d_tile_first, W, kin, (const int32_t*)len, vin, maxl, shift,  \
                       dbits, (const uint32_t*)counts, kout, vout, d_sorted_len)
            if (first && last) ODB_SCATTER(true, true);
            else if (first) ODB_SCATTER(true, false);
            else if (last) ODB_SCATTER(false, true);
            else ODB_SCATTER(false, false);
#undef ODB_SCATTER
            ODB_LAUNCHED();
        }
    }

    // (a3, a4) the group chain: the multi-kernel run walk or pointer jumping.  (A large
    // rank's chain walked by one block per rank takes ~0.4 ms alone but tens of ms beside a
    // running collate, which stalls the two-stream schedule; these grid-wide kernels
    // share the GPU with it.)
    return group_sequences(L, d_ws, W, n, budget, d_off, max_cnt, n > 0 ? (int64_t)hs.max_len - hs.min_len + 1 : 0,
                           passes > 0, d_sorted_len, d_group_index, d_groups_per_rank, d_ranks, s);
}
