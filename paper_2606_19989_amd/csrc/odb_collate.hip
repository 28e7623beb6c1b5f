// Stage 4 of the ODB window pipeline: padded collation (Sec. 2.1, Fig. 1 -- every
// aligned group is padded to its own longest sample).
//
// One or two launches:
//   row_info_kernel  token start and length of every emitted row (one gather of the CSR
//                    offsets per row), so the hot loop never chases emit -> offsets; not
//                    launched when the plan brings these row records itself.
//   collate_kernel   stationary on the flat output: the four outputs share one element
//                    index space [0, padded_elems).  The output is cut into steps of
//                    kBlockStep elements; a block works through runs of kRunSteps
//                    consecutive steps, its first run by its index, later ones taken
//                    from a counter in order, so the blocks in flight read and write one
//                    compact region of every array and finish together.  In a step every
//                    lane owns kGroups groups of 4 consecutive elements (a wave's groups
//                    are 256 elements apart) and stores each group as one aligned 16-byte
//                    non-temporal store per output.
//
// Row edges.  A group whose 4 elements cross from one row into the next (the next row in
// the same tile, rows of at least 4 elements) takes the first row's part from its own
// vector load and the next row's record and first tokens from uniform-address scalar
// loads, one boundary lane of the wave at a time.  Scalar loads complete on their own
// counter, so waiting for them does not wait for the stores the wave has in flight,
// which a late vector load would (see below).  A group that crosses from the last row of
// a tile into the next tile takes the same path when the next row holds the group's
// remaining elements.  Other edge cases (rows shorter than 4, a next row too short) are
// finished element by element.
//
// Software pipeline.  On CDNA the vector-memory counter covers loads and stores alike
// and retires in order, so waiting for a load also waits for every store issued before
// it.  Under a saturated write stream that wait is long.  The kernel therefore keeps
// three steps in flight per lane: while it computes and stores step s it has the tokens
// of step s+1 and the row records of step s+2 in flight, all issued before step s's
// stores.  Each wait then targets a load issued before the previous step's stores, and
// stores drain in the background.  The loop is unrolled three times so the stages rotate
// by name instead of by register copies (a copy would wait for the load), and loads use
// clamped addresses so none is ever skipped.
//
// A group's cursor (slot, row, column) advances with the step sequence: inside a tile it
// moves by arithmetic, across tiles by a search over the tile offsets.  When a group's 4
// elements lie in one row (the common case) its tokens arrive in one 16-byte load.
#include <mutex>

#include "odb_internal.h"

namespace odb {

namespace {

constexpr int kCollateBlock = 256;
constexpr int kVec = 4;                                              // elements per group
constexpr int kGroups = 1;                                           // groups per lane per step
constexpr int64_t kGroupSpan = (int64_t)kWave * kVec;                // 256
constexpr int64_t kWaveStep = kGroupSpan * kGroups;                  // 256
constexpr int64_t kBlockStep = kWaveStep * (kCollateBlock / kWave);  // 1024
// Consecutive steps per run, a block's unit of work: the longest of 8, 16, 32 and 64 steps
// that still gives every block kRunsPerBlock runs.  Measured per run length (8/16/32/64
// steps, ms per call): 64 x 262,144 samples 26.88/26.74/26.68/26.64; 8 x 262,144 multimodal
// 15.72/15.71/15.72/15.75; 16 x 65,536 bimodal 3.91/4.00/4.05/4.09; 8 x 65,536 text
// 1.42/1.45/1.47/1.51; 2 x 2,048 0.024/0.033/0.052/0.090.  Long runs reposition less often;
// on smaller outputs short runs keep the blocks' finishing times close.
constexpr int64_t kRunSteps = 64;      // 2^6
constexpr int64_t kMinRunSteps = 8;    // 2^3
constexpr int64_t kRunsPerBlock = 128;
static_assert(kRunSteps == 64 && kMinRunSteps == 8, "the run length is 2^3 .. 2^6 steps");
// Three resident blocks (12 waves) per compute unit stream fastest (two, four, five or
// six were slower), and they leave five of the eight wave slots and about half the
// registers of every SIMD to kernels on other streams: the grouping and alignment of the next window can run
// beside this kernel instead of after it.
constexpr int kCollateBlocksPerCU = 3;

typedef int v4i __attribute__((ext_vector_type(4)));

__global__ void __launch_bounds__(kBlock) row_info_kernel(const int64_t* __restrict__ tok_off, int64_t n,
                                                          int64_t max_rows, const int32_t* __restrict__ emit,
                                                          const int64_t* __restrict__ row_off, int64_t num_slots,
                                                          int64_t* __restrict__ row_ts, int32_t* __restrict__ row_len,
                                                          int32_t* err) {
    int64_t rows = row_off[num_slots];
    if (rows > max_rows || rows < 0) {
        if (blockIdx.x == 0 && threadIdx.x == 0) atomicOr(err, 1);
        rows = rows < 0 ? 0 : max_rows;
    }
    bool bad = false;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t ri = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; ri < rows; ri += stride) {
        const int32_t s = emit[ri];
        int64_t ts = 0, l = 0;
        if (s >= 0 && s < n) {
            ts = tok_off[s];
            l = tok_off[s + 1] - ts;
        }
        if (s < 0 || s >= n || ts < 0 || l < 0 || l > 0x7FFFFFFF) {
            bad = true;
            ts = 0;
            l = 0;
        }
        row_ts[ri] = ts;
        row_len[ri] = (int32_t)l;
    }
    if (bad) atomicOr(err, 1);
}

struct Plan {
    const int64_t* __restrict__ tile_off;
    const int32_t* __restrict__ maxlen;
    const int32_t* __restrict__ rows;
    const int64_t* __restrict__ row_off;
    const int64_t* __restrict__ row_ts;
    const int32_t* __restrict__ row_len;
    const int32_t* __restrict__ tokens;
    const int64_t* __restrict__ tok_off;
    int64_t num_slots;
    int64_t n;           // samples of the window
    int64_t max_rows;    // rows addressable: the plan's row count, at most n + W - 1 (sampler
                         // padding views); set in the kernel
    int64_t tok_end;     // tokens [0, tok_end) are addressable (tok_off[n], set in the kernel)
    int32_t* err;
    unsigned long long* runs;   // counter of runs handed out after each block's first
};

// Position of a group's first element.
struct Cursor {
    int64_t t1;      // end of the slot's tile
    int32_t k;       // slot
    int32_t ri;      // emitted-row index of the current row
    int32_t ri_end;  // one past the tile's last emitted row
    int32_t ml;      // tile width
    int32_t col;     // column
};

struct RowRec {
    int64_t ts;  // first token of the row's sample
    int32_t l;   // its length
};

// Loads through these (with wave-uniform addresses) become scalar loads.
typedef __attribute__((address_space(4))) const int64_t* cptr64;
typedef __attribute__((address_space(4))) const int32_t* cptr32;
typedef __attribute__((address_space(4))) const v4i* cptrv4;

// Last slot k in [lo, num_slots) with tile_off[k] <= e, given tile_off[lo] <= e < total.
__device__ __forceinline__ int64_t advance_slot(const int64_t* __restrict__ tile_off, int64_t num_slots,
                                                int64_t lo, int64_t e) {
    if (tile_off[lo + 1] > e) return lo;
    int64_t step = 1, hi;
    for (;;) {
        hi = lo + step;
        if (hi >= num_slots) {
            hi = num_slots;
            break;
        }
        if (tile_off[hi] > e) break;
        lo = hi;
        step <<= 1;
    }
    while (hi - lo > 1) {  // tile_off[lo] <= e < tile_off[hi]
        const int64_t mid = lo + ((hi - lo) >> 1);
        if (tile_off[mid] <= e) lo = mid; else hi = mid;
    }
    return lo;
}

__device__ __forceinline__ void enter_slot(Cursor& c, int64_t k, int64_t e, const Plan& p) {
    const int64_t t0 = p.tile_off[k];
    c.k = (int32_t)k;
    c.t1 = p.tile_off[k + 1];
    int32_t ml = p.maxlen[k];
    if (ml <= 0) {
        atomicOr(p.err, 1);
        ml = 1;
    }
    c.ml = ml;
    const int64_t local = e - t0;
    int64_t row;
    if (local >= 0 && local <= 0xFFFFFFFFll) {
        const uint32_t q = (uint32_t)local / (uint32_t)ml;
        row = q;
        c.col = (int32_t)((uint32_t)local - q * (uint32_t)ml);
    } else {
        row = local / ml;
        c.col = (int32_t)(local - row * ml);
    }
    const int64_t r0 = p.row_off[k];
    c.ri = (int32_t)(r0 + row);
    c.ri_end = (int32_t)(r0 + p.rows[k]);
}

// The same search with wave-uniform lo and e, through scalar loads.
__device__ __forceinline__ int64_t advance_slot_uniform(const int64_t* __restrict__ tile_off, int64_t num_slots,
                                                        int64_t lo, int64_t e) {
    const cptr64 t = (cptr64)tile_off;
    if (t[lo + 1] > e) return lo;
    int64_t step = 1, hi;
    for (;;) {
        hi = lo + step;
        if (hi >= num_slots) {
            hi = num_slots;
            break;
        }
        if (t[hi] > e) break;
        lo = hi;
        step <<= 1;
    }
    while (hi - lo > 1) {
        const int64_t mid = lo + ((hi - lo) >> 1);
        if (t[mid] <= e) lo = mid; else hi = mid;
    }
    return lo;
}

__device__ __forceinline__ int64_t readlane64(int64_t v, int l) {
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, l);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)((uint64_t)v >> 32), l);
    return (int64_t)(((uint64_t)hi << 32) | lo);
}

// Slot entry for the lanes of a wave whose element e has passed the end of their tile
// (`cross`).  One crossing lane at a time searches for its slot and reads the slot's
// fields with wave-uniform scalar loads; every crossing lane whose element falls in that
// slot takes it, so a wave entering one tile does one search.  Scalar loads complete on
// their own counter: unlike vector loads, waiting for them does not wait for the stores
// the wave has in flight.  Called in wave-uniform control flow.
__device__ __forceinline__ void enter_slots_uniform(Cursor& c, int64_t e, bool cross, const Plan& p) {
    const int lane = threadIdx.x & (kWave - 1);
    uint64_t need = __ballot(cross);
    while (need) {
        const int l = __builtin_ctzll(need);
        const int64_t el = readlane64(e, l);
        const int64_t k = advance_slot_uniform(p.tile_off, p.num_slots, __builtin_amdgcn_readlane(c.k, l), el);
        const int64_t t0 = ((cptr64)p.tile_off)[k];
        const int64_t t1 = ((cptr64)p.tile_off)[k + 1];
        const int32_t ml_raw = ((cptr32)p.maxlen)[k];
        const int64_t r0 = ((cptr64)p.row_off)[k];
        const int32_t rows = ((cptr32)p.rows)[k];
        const bool take = ((need >> lane) & 1) && e >= t0 && e < t1;
        need &= ~(uint64_t)__ballot(take);
        if (take) {
            int32_t ml = ml_raw;
            if (ml <= 0) {
                atomicOr(p.err, 1);
                ml = 1;
            }
            c.k = (int32_t)k;
            c.t1 = t1;
            c.ml = ml;
            const int64_t local = e - t0;
            int64_t row;
            if (local <= 0xFFFFFFFFll) {
                const uint32_t q = (uint32_t)local / (uint32_t)ml;
                row = q;
                c.col = (int32_t)((uint32_t)local - q * (uint32_t)ml);
            } else {
                row = local / ml;
                c.col = (int32_t)(local - row * ml);
            }
            c.ri = (int32_t)(r0 + row);
            c.ri_end = (int32_t)(r0 + rows);
        }
    }
}

// Move a cursor forward to element e (e - delta is its current element).  Called in
// wave-uniform control flow.
__device__ __forceinline__ void advance(Cursor& c, int64_t e, int64_t delta, const Plan& p) {
    const bool cross = e >= c.t1;
    if (__ballot(cross)) enter_slots_uniform(c, e, cross, p);
    if (cross) return;
    const int64_t col = (int64_t)c.col + delta;
    if (col >= c.ml) {
        const int64_t adv = col <= 0xFFFFFFFFll ? (int64_t)((uint32_t)col / (uint32_t)c.ml) : col / c.ml;
        c.ri += (int32_t)adv;
        c.col = (int32_t)(col - adv * c.ml);
    } else {
        c.col = (int32_t)col;
    }
}

// Row record of the cursor's row.  A row index outside the tile, or a record that is not
// a token range inside the stream no longer than the tile, is a bad plan: the row is
// treated as empty and the error word is set.
__device__ __forceinline__ RowRec load_row(const Cursor& c, const Plan& p) {
    const bool ok = c.ri >= 0 && c.ri < c.ri_end && c.ri < p.max_rows;
    const int32_t i = ok ? c.ri : 0;
    RowRec r;
    r.ts = p.row_ts[i];
    r.l = p.row_len[i];
    if (!ok || r.ts < 0 || r.l < 0 || r.l > c.ml || r.ts > p.tok_end - r.l) {
        atomicOr(p.err, 1);
        r.ts = 0;
        r.l = 0;
    }
    return r;
}

// 16 bytes of tokens at the cursor (address clamped into the stream; only used when the
// group's 4 elements are real tokens of one row, which never needs the clamp).
__device__ __forceinline__ v4i load_tokens(const Cursor& c, const RowRec& r, const Plan& p) {
    int64_t a = r.ts + c.col;
    const int64_t hi = p.tok_end - kVec;
    a = a < hi ? a : hi;
    a = a > 0 ? a : 0;
    // dword-aligned 16-byte load through L2: the 128-byte line that straddles two
    // neighbouring waves' token ranges is then fetched from HBM once, not once per wave
    // (non-temporal loads fetched about 5% more bytes and ran 1.5% slower)
    return *reinterpret_cast<const v4i*>(p.tokens + a);
}

// Next step of this block's sequence, or -1 past its end: the next step of the run of
// step s, else the first step of the block's next run.  A block's first run is its index;
// later runs are taken from a counter when a block needs one, so blocks that meet cheaper
// runs take more of them (dealt statically, the blocks of one launch finished up to 15% of
// the kernel's time apart).  Thread 0 keeps the block's next run index fetched one run
// ahead (`pf`), so the atomic's latency is off the pipeline; the waves of a block cross a
// run boundary at the same step, where the index is handed to them through LDS.  Smaller
// runs for the last stretch (8 to 32 steps) trimmed the finishing tail by under 0.1%.
__device__ __forceinline__ int64_t next_step(int64_t s, int64_t nsteps, int64_t nruns, int run_shift,
                                             unsigned long long& pf,
                                             unsigned long long* runs) {
    const int64_t r = s >> run_shift;
    if (s + 1 < ((r + 1) << run_shift) && s + 1 < nsteps) return s + 1;
    __shared__ int64_t s_run;
    if (threadIdx.x == 0) {
        s_run = (int64_t)pf;
        pf = atomicAdd(runs, 1ull) + gridDim.x;
    }
    __syncthreads();
    const int64_t r2 = s_run;
    __syncthreads();
    return r2 < nruns ? r2 << run_shift : -1;
}

// One pipeline stage of a lane: where its 4 elements are, their row, their tokens.
struct Stage {
    Cursor c;
    RowRec r;
    v4i t;
};

// Values of the 4 elements at e (the stage's position); elements at or past `total` are
// left unspecified (the caller does not store them).
__device__ __forceinline__ void stage_values(const Stage& a, int64_t e, int64_t total, const Plan& p, int vec_ok,
                                             int32_t pad_id, v4i& vid, v4i& vlab, v4i& vmsk, v4i& vpos) {
    const Cursor& c = a.c;
    const RowRec& r = a.r;
    const int32_t nreal = r.l - c.col;
    // one row edge: row B's record and first tokens come through the scalar cache, one
    // boundary lane at a time (scalar loads wait on their own counter, so they never wait
    // for this wave's outstanding stores).  Row B is row ri + 1 also when row A is the last
    // row of its tile: rows and tiles are both packed in slot order, so the next row is the
    // first row of the next non-empty tile, which starts right after row A.  Its width is
    // not at hand then, so that case needs row B to hold the group's remaining elements.
    const bool same_tile = c.ri + 1 < c.ri_end;
    // column + 4 in 32-bit unsigned: a tile may be 2^31 - 1 wide, and 0 <= col < ml
    const uint32_t col4 = (uint32_t)c.col + kVec;
    bool edge = vec_ok && c.ml >= kVec && col4 > (uint32_t)c.ml && c.ri >= 0 && c.ri < c.ri_end &&
                c.ri + 1 < p.max_rows && r.ts + c.col + kVec <= p.tok_end;
    int32_t bl = 0;
    v4i bt = {0, 0, 0, 0};
    {
        uint64_t need = __ballot(edge);
        const int lane = threadIdx.x & (kWave - 1);
        while (need) {
            const int l = __builtin_ctzll(need);
            need &= need - 1;
            const int32_t ri1 = __builtin_amdgcn_readlane(c.ri, l) + 1;
            const int64_t ts = *(cptr64)(p.row_ts + ri1);
            const int32_t len = *(cptr32)(p.row_len + ri1);
            const bool fits = ts >= 0 && ts + kVec <= p.tok_end;
            const v4i h = *(cptrv4)(p.tokens + (fits ? ts : 0));
            if (lane == l) {
                bl = len;
                bt = h;
                edge = edge && fits && (same_tile || bl >= kVec - (c.ml - c.col));
            }
        }
    }
    if (edge) {
        const int32_t inA = c.ml - c.col;   // elements left in row A (1..3)
#pragma unroll
        for (int i = 0; i < kVec; ++i) {
            const bool b = i >= inA;
            const int32_t col = b ? i - inA : c.col + i;
            const int32_t len = b ? bl : r.l;
            const bool real = col < len;
            int32_t tb = bt[0];
            tb = col == 1 ? bt[1] : tb;
            tb = col == 2 ? bt[2] : tb;
            const int32_t tok = b ? tb : a.t[i];
            vid[i] = real ? tok : pad_id;
            vlab[i] = real ? tok : -100;
            vmsk[i] = real ? 1 : 0;
            vpos[i] = real ? col : 0;
        }
    } else if (vec_ok && col4 <= (uint32_t)c.ml && (nreal <= 0 || r.ts + c.col + kVec <= p.tok_end)) {
        // the 4 elements sit in one row and the vector load covered them
#pragma unroll
        for (int i = 0; i < kVec; ++i) {
            const bool real = i < nreal;
            vid[i] = real ? a.t[i] : pad_id;
            vlab[i] = real ? a.t[i] : -100;
            vmsk[i] = real ? 1 : 0;
            vpos[i] = real ? c.col + i : 0;
        }
    } else {
        // a row or tile edge inside the 4 elements: step element by element
        Cursor d = c;
        RowRec dr = r;
#pragma unroll
        for (int i = 0; i < kVec; ++i) {
            const int64_t ee = e + i;
            if (i > 0 && ee < total) {
                if (ee >= d.t1) {
                    enter_slot(d, advance_slot(p.tile_off, p.num_slots, d.k, ee), ee, p);
                    dr = load_row(d, p);
                } else if (++d.col == d.ml) {
                    d.col = 0;
                    d.ri += 1;
                    dr = load_row(d, p);
                }
            }
            const bool real = d.col < dr.l;
            const int32_t tok = real ? p.tokens[dr.ts + d.col] : 0;
            vid[i] = real ? tok : pad_id;
            vlab[i] = real ? tok : -100;
            vmsk[i] = real ? 1 : 0;
            vpos[i] = real ? d.col : 0;
        }
    }
}

// Start of a collate: the run counter and the error word of this call.
__global__ void clear_collate_kernel(unsigned long long* runs, int32_t* err) {
    if (threadIdx.x == 0) {
        *runs = 0;
        *err = 0;
    }
}

__global__ void __launch_bounds__(kCollateBlock) collate_kernel(Plan p, int32_t pad_id, int64_t capacity,
                                                                int32_t* __restrict__ o_ids,
                                                                int32_t* __restrict__ o_lab,
                                                                int32_t* __restrict__ o_msk,
                                                                int32_t* __restrict__ o_pos) {
    p.tok_end = p.tok_off[p.n];
    {
        const int64_t rows = p.row_off[p.num_slots];
        p.max_rows = rows < 0 ? 0 : (rows < p.max_rows ? rows : p.max_rows);
    }
    const int vec_ok = p.tok_end >= kVec;
    const int64_t total_plan = p.tile_off[p.num_slots];
    const int64_t total = total_plan < capacity ? total_plan : capacity;
    if (total <= 0) return;
    const int64_t nsteps = (total + kBlockStep - 1) / kBlockStep;
    // runs of 2^run_shift steps: the largest power of two from kMinRunSteps to kRunSteps that
    // still gives every block kRunsPerBlock runs
    int run_shift = 3;
    while (run_shift < 6 && ((int64_t)gridDim.x * kRunsPerBlock << (run_shift + 1)) <= nsteps) ++run_shift;
    const int64_t nruns = (nsteps + (1ll << run_shift) - 1) >> run_shift;
    if ((int64_t)blockIdx.x >= nruns) return;
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int64_t lane_off = (int64_t)wave * kWaveStep + (int64_t)lane * kVec;
    // a lane's elements may lie past the end only in the last step; clamp its position
    // so every stage has a valid cursor (the last step stores with bounds checks)
    auto elem = [&](int64_t s) {
        const int64_t e = s * kBlockStep + lane_off;
        return e < total ? e : total - 1;
    };

    // pipeline: step s0 is stored from stage a, s1's tokens load into b, s2's rows into c
    unsigned long long pf = 0;
    if (threadIdx.x == 0) pf = atomicAdd(p.runs, 1ull) + gridDim.x;
    int64_t s0 = (int64_t)blockIdx.x << run_shift;
    int64_t s1 = next_step(s0, nsteps, nruns, run_shift, pf, p.runs);
    int64_t s2 = s1 >= 0 ? next_step(s1, nsteps, nruns, run_shift, pf, p.runs) : -1;
    Stage X, Y, Z;
    {
        const int64_t e = elem(s0);
        int64_t lo = 0, hi = p.num_slots;  // last slot with tile_off <= e
        while (hi - lo > 1) {
            const int64_t mid = lo + ((hi - lo) >> 1);
            if (p.tile_off[mid] <= e) lo = mid; else hi = mid;
        }
        enter_slot(X.c, lo, e, p);
        X.r = load_row(X.c, p);
        if (vec_ok) X.t = load_tokens(X.c, X.r, p);
        Y.c = X.c;
        if (s1 >= 0) advance(Y.c, elem(s1), elem(s1) - e, p);
        Y.r = load_row(Y.c, p);
    }

    // Every load below is issued whether or not its step exists (a missing step reloads
    // its predecessor's row and tokens), and full steps store without conditions, so the
    // number of memory operations between a load and its use is the same on every path.
#define ODB_COLLATE_STEP(A, B, C)                                                             \
    {                                                                                         \
        if (s0 < 0) break;                                                                    \
        C.c = B.c;                                                                            \
        if (s2 >= 0) advance(C.c, elem(s2), elem(s2) - elem(s1), p);                          \
        C.r = load_row(C.c, p);                                                               \
        if (vec_ok) B.t = load_tokens(B.c, B.r, p);                                           \
        const int64_t e = s0 * kBlockStep + lane_off;                                         \
        v4i vid, vlab, vmsk, vpos;                                                            \
        stage_values(A, e, total, p, vec_ok, pad_id, vid, vlab, vmsk, vpos);                  \
        if ((s0 + 1) * kBlockStep <= total) {                                                 \
            __builtin_nontemporal_store(vid, reinterpret_cast<v4i*>(o_ids + e));              \
            __builtin_nontemporal_store(vlab, reinterpret_cast<v4i*>(o_lab + e));             \
            __builtin_nontemporal_store(vmsk, reinterpret_cast<v4i*>(o_msk + e));             \
            __builtin_nontemporal_store(vpos, reinterpret_cast<v4i*>(o_pos + e));             \
        } else {                                                                              \
            _Pragma("unroll") for (int i = 0; i < kVec; ++i) {                                \
                if (e + i < total) {                                                          \
                    o_ids[e + i] = vid[i];                                                    \
                    o_lab[e + i] = vlab[i];                                                   \
                    o_msk[e + i] = vmsk[i];                                                   \
                    o_pos[e + i] = vpos[i];                                                   \
                }                                                                             \
            }                                                                                 \
        }                                                                                     \
        s0 = s1;                                                                              \
        s1 = s2;                                                                              \
        s2 = s2 >= 0 ? next_step(s2, nsteps, nruns, run_shift, pf, p.runs) : -1;                         \
    }
    // unrolled three times so that no stage register is copied while its load is in flight
    for (;;) {
        ODB_COLLATE_STEP(X, Y, Z)
        ODB_COLLATE_STEP(Y, Z, X)
        ODB_COLLATE_STEP(Z, X, Y)
    }
#undef ODB_COLLATE_STEP
}


// Host checks shared by the collate entry points.  Sets *empty when there is nothing to
// write (no slots, no capacity or no samples).
int check_collate_args(const odb_window_t* w, int64_t num_slots, const int32_t* d_emit_order,
                       const int64_t* d_row_token_start, const int32_t* d_row_len, const int32_t* d_slot_rows,
                       const int32_t* d_slot_maxlen, const int64_t* d_slot_row_off, const int64_t* d_slot_tile_off,
                       int64_t out_capacity_elems, int32_t* d_input_ids, int32_t* d_labels,
                       int32_t* d_attention_mask, int32_t* d_position_ids, bool* empty) {
    if (num_slots < 0 || num_slots >= 0x7FFFFFFFll)
        return set_error(ODB_E_INVALID_ARG, "num_slots must be in [0, 2^31 - 1)");
    if (out_capacity_elems < 0) return set_error(ODB_E_INVALID_ARG, "out_capacity_elems must be >= 0");
    if ((d_row_token_start == nullptr) != (d_row_len == nullptr))
        return set_error(ODB_E_INVALID_ARG, "d_row_token_start and d_row_len are given together or not at all");
    *empty = num_slots == 0 || out_capacity_elems == 0 || w->num_samples == 0;
    if (*empty) return ODB_OK;
    if (!d_slot_rows || !d_slot_maxlen || !d_slot_row_off || !d_slot_tile_off)
        return set_error(ODB_E_INVALID_ARG, "plan arrays must not be NULL");
    if (!d_input_ids || !d_labels || !d_attention_mask || !d_position_ids)
        return set_error(ODB_E_INVALID_ARG, "output arrays must not be NULL");
    if (((reinterpret_cast<uintptr_t>(d_input_ids) | reinterpret_cast<uintptr_t>(d_labels) |
          reinterpret_cast<uintptr_t>(d_attention_mask) | reinterpret_cast<uintptr_t>(d_position_ids)) &
         15) != 0)
        return set_error(ODB_E_INVALID_ARG, "output arrays must be 16-byte aligned");
    if (!d_row_token_start && !d_emit_order) return set_error(ODB_E_INVALID_ARG, "d_emit_order is NULL");
    return ODB_OK;
}

// The launches of one collate: clear the run counter and the error word, gather the row
// records into (row_ts, row_len) when the plan brings none (capacity n + W - 1 rows),
// then the collate kernel.  `err` and `runs` are device words of the caller's choosing.
int launch_collate(const odb_window_t* w, int64_t num_slots, const int32_t* d_emit_order,
                   const int64_t* d_row_token_start, const int32_t* d_row_len, const int32_t* d_slot_rows,
                   const int32_t* d_slot_maxlen, const int64_t* d_slot_row_off, const int64_t* d_slot_tile_off,
                   int32_t pad_id, int64_t out_capacity_elems, int32_t* d_input_ids, int32_t* d_labels,
                   int32_t* d_attention_mask, int32_t* d_position_ids, bool empty, int32_t* err,
                   unsigned long long* runs, int64_t* row_ts, int32_t* row_len, hipStream_t s) {
    hipLaunchKernelGGL(clear_collate_kernel, dim3(1), dim3(64), 0, s, runs, err);
    ODB_LAUNCHED();
    if (empty) return ODB_OK;
    const int64_t n = w->num_samples;
    // a plan may list a sample more than once only through sampler padding: at most
    // W - 1 extra rows (streaming plans)
    const int64_t max_rows = n + w->num_ranks - 1;
    const int64_t* rts = d_row_token_start;
    const int32_t* rlen = d_row_len;
    if (!rts) {
        hipLaunchKernelGGL(row_info_kernel, dim3(grid_for(n, kBlock, (int64_t)num_cus() * kPlanBlocksPerCU)),
                           dim3(kBlock), 0, s, w->d_token_offsets, n, max_rows, d_emit_order, d_slot_row_off,
                           num_slots, row_ts, row_len, err);
        ODB_LAUNCHED();
        rts = row_ts;
        rlen = row_len;
    }
    Plan p{d_slot_tile_off, d_slot_maxlen, d_slot_rows, d_slot_row_off, rts, rlen, w->d_tokens,
           w->d_token_offsets, num_slots, n, max_rows, 0, err, runs};
    // kCollateBlocksPerCU blocks per compute unit, all resident at once; each starts on the
    // run of its index and then takes runs from the counter
    const unsigned grid = (unsigned)(num_cus() * kCollateBlocksPerCU);
    hipLaunchKernelGGL(collate_kernel, dim3(grid), dim3(kCollateBlock), 0, s, p, pad_id, out_capacity_elems,
                       d_input_ids, d_labels, d_attention_mask, d_position_ids);
    ODB_LAUNCHED();
    return ODB_OK;
}

}  // namespace

}  // namespace odb

using namespace odb;

extern "C" int odb_collate(const odb_window_t* w, int64_t num_slots, const int32_t* d_emit_order,
                           const int64_t* d_row_token_start, const int32_t* d_row_len, const int32_t* d_slot_rows,
                           const int32_t* d_slot_maxlen, const int64_t* d_slot_row_off,
                           const int64_t* d_slot_tile_off, int32_t pad_id, int64_t out_capacity_elems,
                           int32_t* d_input_ids, int32_t* d_labels, int32_t* d_attention_mask,
                           int32_t* d_position_ids, void* d_ws, size_t ws_bytes, void* stream) {
    Layout L;
    ODB_TRY(check_workspace(w, d_ws, ws_bytes, &L));
    bool empty = false;
    ODB_TRY(check_collate_args(w, num_slots, d_emit_order, d_row_token_start, d_row_len, d_slot_rows, d_slot_maxlen,
                               d_slot_row_off, d_slot_tile_off, out_capacity_elems, d_input_ids, d_labels,
                               d_attention_mask, d_position_ids, &empty));
    DevStatus* st = ws_at<DevStatus>(d_ws, L.status);
    return launch_collate(w, num_slots, d_emit_order, d_row_token_start, d_row_len, d_slot_rows, d_slot_maxlen,
                          d_slot_row_off, d_slot_tile_off, pad_id, out_capacity_elems, d_input_ids, d_labels,
                          d_attention_mask, d_position_ids, empty, &st->collate_err, &st->collate_runs,
                          ws_at<int64_t>(d_ws, L.row_ts), ws_at<int32_t>(d_ws, L.row_len),
                          static_cast<hipStream_t>(stream));
}

// ---------------------------------------------------------------- allocation-free variant
// odb_collate_static keeps the collate's scratch in this file-scope device array instead
// of a caller workspace: the run counter in the first 256 bytes, then, when the plan
// brings no row records, the gathered records (token starts, then lengths).  Each device
// holds its own copy until the process ends.  Host code never passes the array's name to
// a kernel (on the host it is only a stand-in for the symbol): it passes the device
// address that hipGetSymbolAddress returns, looked up once per device.
namespace odb {
namespace {

constexpr int64_t kStaticRows = ODB_COLLATE_STATIC_MAX_ROWS;
constexpr size_t kStaticHeader = 256;
constexpr size_t kStaticBytes = kStaticHeader + 12 * (size_t)kStaticRows;
constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kStaticBytes];

std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of this device's scratch array (looked up on the first call per device).
int static_scratch(void** out) {
    int dev = -1;
    ODB_TRY_HIP(hipGetDevice(&dev));
    if (dev < 0 || dev >= kMaxDevices) return set_error(ODB_E_INTERNAL, "device index %d out of range", dev);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || p == nullptr)
            return set_error(ODB_E_HIP, "hipGetSymbolAddress of the collate scratch failed on device %d: %s", dev,
                             hipGetErrorString(e));
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return ODB_OK;
}

}  // namespace
}  // namespace odb

extern "C" int odb_collate_static(const odb_window_t* w, int64_t num_slots, const int32_t* d_emit_order,
                                  const int64_t* d_row_token_start, const int32_t* d_row_len,
                                  const int32_t* d_slot_rows, const int32_t* d_slot_maxlen,
                                  const int64_t* d_slot_row_off, const int64_t* d_slot_tile_off, int32_t pad_id,
                                  int64_t out_capacity_elems, int32_t* d_input_ids, int32_t* d_labels,
                                  int32_t* d_attention_mask, int32_t* d_position_ids, int32_t* d_status,
                                  void* stream) {
    ODB_TRY(check_window(w));
    if (!d_status) return set_error(ODB_E_INVALID_ARG, "d_status is NULL");
    bool empty = false;
    ODB_TRY(check_collate_args(w, num_slots, d_emit_order, d_row_token_start, d_row_len, d_slot_rows, d_slot_maxlen,
                               d_slot_row_off, d_slot_tile_off, out_capacity_elems, d_input_ids, d_labels,
                               d_attention_mask, d_position_ids, &empty));
    const int64_t max_rows = w->num_samples + w->num_ranks - 1;
    if (!empty && !d_row_token_start && max_rows > kStaticRows)
        return set_error(ODB_E_INVALID_ARG,
                         "without row records the plan may hold %lld rows, more than the %lld the static scratch "
                         "holds: pass the plan's row records or use odb_collate with a workspace",
                         (long long)max_rows, (long long)kStaticRows);
    void* base = nullptr;
    ODB_TRY(static_scratch(&base));
    char* b = static_cast<char*>(base);
    return launch_collate(w, num_slots, d_emit_order, d_row_token_start, d_row_len, d_slot_rows, d_slot_maxlen,
                          d_slot_row_off, d_slot_tile_off, pad_id, out_capacity_elems, d_input_ids, d_labels,
                          d_attention_mask, d_position_ids, empty, d_status,
                          reinterpret_cast<unsigned long long*>(b),
                          reinterpret_cast<int64_t*>(b + kStaticHeader),
                          reinterpret_cast<int32_t*>(b + kStaticHeader + 8 * (size_t)kStaticRows),
                          static_cast<hipStream_t>(stream));
}

__global__ void clear_collate_status_kernel(DevStatus* st) {
    if (threadIdx.x == 0) st->collate_err = 0;
}

extern "C" int odb_collate_status(void* d_ws, size_t ws_bytes, void* stream) {
    if (!d_ws || ws_bytes < sizeof(DevStatus)) return set_error(ODB_E_INVALID_ARG, "workspace too small");
    hipStream_t s = static_cast<hipStream_t>(stream);
    DevStatus* st = static_cast<DevStatus*>(d_ws);  // the status word sits at offset 0
    int32_t v = 0;
    ODB_TRY_HIP(hipMemcpyAsync(&v, &st->collate_err, sizeof(v), hipMemcpyDeviceToHost, s));
    ODB_TRY_HIP(hipStreamSynchronize(s));
    hipLaunchKernelGGL(clear_collate_status_kernel, dim3(1), dim3(64), 0, s, st);
    ODB_LAUNCHED();
    if (v) return set_error(ODB_E_INVALID_DATA, "collate met an inconsistent plan");
    return ODB_OK;
}
