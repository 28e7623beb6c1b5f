// Stages 2-3 of the ODB window pipeline: Distributed Group Alignment (Eq. 3,
// Algorithm 1, termination rules of Sec. 2.3) and identity coverage (App. C).
//
// Every rank's buffer is a contiguous run of formation positions; a group is a range
// of them.  One alignment round is:
//   group_sizes        size of every group
//   adjust_kernel      per rank: the simulated all_gather of (G_r, S_r, C_r) and Eq. 3's T,
//                      then split (closed form, below) or overflow (size threshold)
//   slot_records       rows / max length / real tokens of every aligned step, and the
//                      global sample count of every step
//   finalize_kernel    per rank: the round's cut (join: all T steps; non-join: up to the
//                      first step reaching Q), which positions are emitted, where they go
//   emit_kernel        writes emitted ids (rows short to long) and the next buffer
// and rounds repeat on the returned samples until the termination rule fires.
//
// Split in closed form.  Algorithm 1 peels, one at a time, the last sample of the first
// multi-sample group met scanning the short-to-long list from its long end.  In
// formation order (longest first) that is the longest member of the first group with
// at least two samples; after k = T - G_r peels, formation positions [0, X) are
// singletons, [X, end of group j*) is one group and later groups are untouched, where
// j* is the first group whose cumulative surplus sum_{g<=j}(c_g - 1) reaches k and
// X = k + j*.
//
// Overflow.  Algorithm 1 keeps the T largest groups (stable over the short-to-long list,
// so equal sizes favour the later-formed group).  With sigma = the largest size such
// that at least T groups have size >= sigma, every group larger than sigma is kept and
// the remaining places go to the size-sigma groups with the highest formation index.
#include <algorithm>
#include <climits>
#include <cstring>
#include <vector>

#include "odb_internal.h"

namespace odb {

// A pair of int64 sums, scanned together by the generic scan (its shuffles are found by
// argument-dependent lookup, next to the scalar ones).  Trivially default-constructible, so
// it can live in LDS.
struct I64Pair {
    int64_t a, b;
    I64Pair() = default;
    __host__ __device__ constexpr I64Pair(int z) : a(z), b(z) {}
    __host__ __device__ constexpr I64Pair(int64_t x, int64_t y) : a(x), b(y) {}
};
__device__ __forceinline__ I64Pair operator+(I64Pair x, I64Pair y) { return I64Pair{x.a + y.a, x.b + y.b}; }
__device__ __forceinline__ I64Pair operator-(I64Pair x, I64Pair y) { return I64Pair{x.a - y.a, x.b - y.b}; }
__device__ __forceinline__ I64Pair& operator+=(I64Pair& x, I64Pair y) {
    x.a += y.a;
    x.b += y.b;
    return x;
}
__device__ __forceinline__ I64Pair __shfl_up(I64Pair v, unsigned int d, int width) {
    return I64Pair{::__shfl_up(v.a, d, width), ::__shfl_up(v.b, d, width)};
}
__device__ __forceinline__ I64Pair __shfl_xor(I64Pair v, int m, int width) {
    return I64Pair{::__shfl_xor(v.a, m, width), ::__shfl_xor(v.b, m, width)};
}

namespace {

template <typename T, typename Op>
__device__ __forceinline__ T block_reduce(T v, Op op) {
    __shared__ T buf[kBlock];
    buf[threadIdx.x] = v;
    __syncthreads();
    for (unsigned s = kBlock / 2; s > 0; s >>= 1) {
        if (threadIdx.x < s) buf[threadIdx.x] = op(buf[threadIdx.x], buf[threadIdx.x + s]);
        __syncthreads();
    }
    T r = buf[0];
    __syncthreads();
    return r;
}

struct MaxOp {
    __device__ int64_t operator()(int64_t a, int64_t b) const { return a > b ? a : b; }
};
struct MinOp {
    __device__ int64_t operator()(int64_t a, int64_t b) const { return a < b ? a : b; }
};
struct SumOp {
    __device__ int64_t operator()(int64_t a, int64_t b) const { return a + b; }
};

__global__ void init_align_kernel(RoundState* rs, DevInfo* info) {
    if (threadIdx.x == 0) {
        *rs = RoundState{};
        *info = DevInfo{};
    }
}

__global__ void clear_view_counters_kernel(DevInfo* info, int with_ids) {
    if (threadIdx.x == 0) {
        info->bad_views = 0;
        if (with_ids) {
            info->missing_ids = 0;
            info->duplicate_ids = 0;
        }
    }
}

__global__ void fill_i32_kernel(int32_t* p, int64_t n, int32_t v) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) p[i] = v;
}


// ---------------------------------------------------------------- round 0 inputs
// Rank state from the stage-1 group counts; G_r must be 0 exactly for empty ranks and
// at most S_r.  One block.
__global__ void __launch_bounds__(kBlock) round0_ranks_kernel(const int64_t* __restrict__ off,
                                                              const int32_t* __restrict__ groups, int W,
                                                              RankState* ranks, int64_t* __restrict__ gbase,
                                                              DevStatus* st, RoundState* rs, DevInfo* info) {
    __shared__ int64_t carry;
    if (threadIdx.x == 0) {
        carry = 0;
        *rs = RoundState{};
        *info = DevInfo{};
    }
    __syncthreads();
    for (int b = 0; b < W; b += kBlock) {
        const int r = b + threadIdx.x;
        int64_t G = 0, cnt = 0;
        if (r < W) {
            G = groups[r];
            cnt = off[r + 1] - off[r];
            if (G < 0 || G > cnt || ((cnt == 0) != (G == 0))) {
                atomicOr(&st->err, kErrGroupIndex);
                G = 0;
            }
        }
        int64_t tot;
        const int64_t ex = block_excl_sum(G, &tot);
        const int64_t c = carry;
        if (r < W) {
            RankState z = {};
            z.cnt = cnt;
            z.G = G;
            z.gbase = c + ex;
            ranks[r] = z;
            gbase[r] = c + ex;
        }
        __syncthreads();
        if (threadIdx.x == 0) carry = c + tot;
        __syncthreads();
    }
    if (threadIdx.x == 0) gbase[W] = carry;
}

// Checks that stage-1 arrays describe this window: order[p] is a sample of p's rank,
// sorted_len[p] >= 1, the order strictly (length desc, id asc) -- so each rank's segment
// is a permutation of its ids -- and the group indices run 0, 0|+1, ..., G_r - 1.
// Records every group start.  That sorted_len[p] is the CSR length of order[p] is
// checked once the plan is built (row_check_kernel, leftover_kernel), where the CSR
// offsets of every emitted sample are gathered anyway for the row records.
__global__ void __launch_bounds__(kBlock) round0_check_kernel(
    const int64_t* __restrict__ off, const RankState* __restrict__ ranks,
    int W, int64_t n, const int32_t* __restrict__ order, const int32_t* __restrict__ slen,
    const int32_t* __restrict__ gidx, int32_t* __restrict__ gstart, DevStatus* st) {
    __shared__ int64_t s_off[kLdsRanks + 1];
    off = stage_ranks(off, W, s_off);
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; p < n; p += stride) {
        const int r = rank_of(off, W, p);
        const int64_t base = off[r];
        const int64_t q = p - base, nr = ranks[r].cnt;
        const int64_t G = ranks[r].G;
        const int32_t id = order[p];
        const int32_t l = slen[p];
        bool ok = id >= base && id < base + nr && l >= 1;
        const int32_t g = gidx[p];
        bool gok = g >= 0 && g < G;
        if (q == 0) {
            gok = gok && g == 0;
        } else {
            const int32_t pl = slen[p - 1], pid = order[p - 1];
            ok = ok && (pl > l || (pl == l && pid < id));
            const int32_t d = g - gidx[p - 1];
            gok = gok && (d == 0 || d == 1);
        }
        if (q == nr - 1) gok = gok && g == G - 1;
        if (!ok) {
            atomicOr(&st->err, kErrOrder);
            atomicMin((unsigned long long*)&st->first_bad, (unsigned long long)p);
        }
        if (!gok) {
            atomicOr(&st->err, kErrGroupIndex);
            atomicMin((unsigned long long*)&st->first_bad, (unsigned long long)p);
        } else if (q == 0 || g != gidx[p - 1]) {
            gstart[ranks[r].gbase + g] = (int32_t)p;
        }
    }
}

// ---------------------------------------------------------------- one round
struct LiveLen {
    const int32_t* len;
    const int64_t* off;
    const RankState* ranks;
    int W;
    int gaps;
    __device__ int64_t operator()(int64_t i) const {
        if (!gaps) return len[i];
        const int r = rank_of(off, W, i);
        return (i - off[r] < ranks[r].cnt) ? (int64_t)len[i] : 0;
    }
};
struct LiveLenIncl {
    LiveLen ld;
    int64_t* cs;
    __device__ void operator()(int64_t i, int64_t ex) const { cs[i] = ex + ld(i); }
};

// Stage-1 arrays that round0_check_kernel found inconsistent: the round's kernels that
// index through group starts do nothing (the host reports the error at the round's
// synchronisation).
__device__ __forceinline__ bool stage1_bad(const DevStatus* st) {
    return (*(volatile const int32_t*)&st->err & (kErrOrder | kErrGroupIndex)) != 0;
}

__global__ void __launch_bounds__(kBlock) group_sizes_kernel(const int32_t* __restrict__ gstart,
                                                             const int64_t* __restrict__ gbase,
                                                             const int64_t* __restrict__ off,
                                                             const RankState* __restrict__ ranks, int W,
                                                             int32_t* __restrict__ gsize, int64_t* __restrict__ steps,
                                                             int64_t nsteps, const DevStatus* st) {
    if (stage1_bad(st)) return;
    const int64_t total = gbase[W];
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    // the round's per-step sample counts, summed by slot_records_kernel
    for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j < nsteps; j += stride) steps[j] = 0;
    for (int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; g < total; g += stride) {
        const int r = rank_of(gbase, W, g);
        const int64_t lg = g - gbase[r];
        const int64_t start = gstart[g];
        const int64_t end = (lg + 1 < ranks[r].G) ? (int64_t)gstart[g + 1] : off[r] + ranks[r].cnt;
        gsize[g] = (int32_t)(end - start);
    }
}

// Per rank (one block each): the simulated all_gather of (G_r, S_r, C_r) and Eq. 3's
// target T over the active ranks (every block computes it; block 0 also records the round's
// statistics), then this rank's action: split position or overflow selection.
__global__ void __launch_bounds__(kBlock) adjust_kernel(RankState* ranks, const int64_t* __restrict__ cap,
                                                        int has_cap, int W, RoundState* rs,
                                                        const int32_t* __restrict__ gsize,
                                                        int32_t* __restrict__ ov_slot, int32_t* __restrict__ kept,
                                                        DevStatus* st) {
    if (stage1_bad(st)) return;
    int64_t maxG = 0, minC = LLONG_MAX, minS = LLONG_MAX;
    for (int q = threadIdx.x; q < W; q += kBlock) {
        const int64_t Gq = ranks[q].G;
        if (Gq <= 0) continue;
        maxG = Gq > maxG ? Gq : maxG;
        const int64_t S = ranks[q].cnt;
        if (S > 0 && S < minS) minS = S;
        if (has_cap && cap[q] > 0 && cap[q] < minC) minC = cap[q];
    }
    maxG = block_reduce(maxG, MaxOp{});
    minC = block_reduce(minC, MinOp{});
    minS = block_reduce(minS, MinOp{});
    int64_t T = maxG;
    if (minC != LLONG_MAX && minC < T) T = minC;
    if (minS != LLONG_MAX && minS < T) T = minS;
    if (T < 1) T = 1;
    if (blockIdx.x == 0) {
        int64_t active = 0, totalG = 0, splits = 0, over = 0, changed = 0;
        for (int q = threadIdx.x; q < W; q += kBlock) {
            const int64_t Gq = ranks[q].G;
            totalG += Gq;
            if (Gq <= 0) continue;
            active += 1;
            if (Gq < T) {
                splits += T - Gq;
                changed += 1;
            } else if (Gq > T) {
                over += Gq - T;
                changed += 1;
            }
        }
        active = block_reduce(active, SumOp{});
        totalG = block_reduce(totalG, SumOp{});
        splits = block_reduce(splits, SumOp{});
        over = block_reduce(over, SumOp{});
        changed = block_reduce(changed, SumOp{});
        if (threadIdx.x == 0) {
            // App. B: the pre-alignment counts of the first exchange are exact only if no
            // active rank's groups changed; otherwise exact token weights need a second one
            rs->second_gather += changed > 0 ? 1 : 0;
            rs->T = T;
            rs->active = active;
            rs->total_groups = totalG;
            rs->splits += splits;
            rs->overflow += over;
            rs->cut = 0;
        }
    }
    const int r = blockIdx.x;
    const int64_t G = ranks[r].G;
    const int32_t action = G <= 0 ? kActInactive : (G < T ? kActSplit : (G > T ? kActOverflow : kActKeep));
    if (threadIdx.x == 0) {
        ranks[r].X = 0;
        ranks[r].jstar = 0;
        ranks[r].qcut = 0;
        ranks[r].action = action;
    }
    if (action != kActSplit && action != kActOverflow) return;
    const int64_t gb = ranks[r].gbase;
    __shared__ int64_t s_found;
    if (action == kActSplit) {
        const int64_t k = T - G;
        if (threadIdx.x == 0) s_found = -1;
        __syncthreads();
        int64_t carry = 0;
        for (int64_t b = 0; b < G; b += kBlock) {
            const int64_t j = b + threadIdx.x;
            const int64_t v = j < G ? (int64_t)gsize[gb + j] - 1 : 0;
            int64_t tot;
            const int64_t ex = block_excl_sum(v, &tot);
            if (j < G && carry + ex < k && carry + ex + v >= k) s_found = j;
            __syncthreads();
            if (s_found >= 0) break;
            carry += tot;
        }
        if (threadIdx.x == 0) {
            const int64_t js = s_found;
            if (js < 1) {
                // the group sizes do not add up to the buffer: drop the rank from this round
                // (nothing is indexed through the split) and report an internal error
                atomicOr(&st->err, kErrInternal);
                ranks[r].action = kActInactive;
            } else {
                ranks[r].jstar = js;
                ranks[r].X = k + js;
            }
        }
        return;
    }
    // overflow: sigma = largest size with at least T groups of size >= sigma
    int64_t mx = 0;
    for (int64_t j = threadIdx.x; j < G; j += kBlock) {
        const int64_t s = gsize[gb + j];
        mx = s > mx ? s : mx;
    }
    mx = block_reduce(mx, MaxOp{});
    int64_t lo = 1, hi = mx;
    while (lo < hi) {
        const int64_t mid = lo + (hi - lo + 1) / 2;
        int64_t c = 0;
        for (int64_t j = threadIdx.x; j < G; j += kBlock) c += gsize[gb + j] >= mid ? 1 : 0;
        c = block_reduce(c, SumOp{});
        if (c >= T) lo = mid; else hi = mid - 1;
    }
    const int64_t sigma = lo;
    int64_t above = 0;
    for (int64_t j = threadIdx.x; j < G; j += kBlock) above += gsize[gb + j] > sigma ? 1 : 0;
    above = block_reduce(above, SumOp{});
    const int64_t need = T - above;
    // walk groups from the highest formation index down
    int64_t ceq = 0, ckept = 0;
    for (int64_t b = 0; b < G; b += kBlock) {
        const int64_t i = b + threadIdx.x;
        const bool valid = i < G;
        const int64_t g = G - 1 - i;
        const int64_t s = valid ? gsize[gb + g] : 0;
        const int64_t eq = (valid && s == sigma) ? 1 : 0;
        int64_t teq;
        const int64_t xeq = block_excl_sum(eq, &teq);
        const int64_t keep = (valid && (s > sigma || (eq && ceq + xeq < need))) ? 1 : 0;
        int64_t tk;
        const int64_t xk = block_excl_sum(keep, &tk);
        if (valid) {
            if (keep) {
                ov_slot[gb + g] = (int32_t)(ckept + xk);
                kept[gb + ckept + xk] = (int32_t)g;
            } else {
                ov_slot[gb + g] = -1;
            }
        }
        ceq += teq;
        ckept += tk;
    }
}

// First formation position and one-past-last of adjusted group a (formation order) of a
// keep / split rank.
__device__ __forceinline__ void adjusted_range(const RankState& R, int64_t base, int64_t a,
                                               const int32_t* __restrict__ gstart,
                                               const int32_t* __restrict__ gsize, int64_t* start, int64_t* end) {
    if (a < R.X) {
        *start = base + a;
        *end = base + a + 1;
    } else if (a == R.X) {
        const int64_t g = R.gbase + R.jstar;
        *start = base + R.X;
        *end = (int64_t)gstart[g] + gsize[g];
    } else {
        const int64_t g = R.gbase + R.jstar + (a - R.X);
        *start = gstart[g];
        *end = *start + gsize[g];
    }
}

// Step j of every active rank: adjusted group T-1-j (emission runs short to long).
// Besides rows, longest length and real tokens, each record carries the approximate
// token count of App. B: rows times the mean length of the rank's buffer at the start of
// this round (the counts a rank can advertise before alignment).
__global__ void __launch_bounds__(kBlock) slot_records_kernel(
    const RankState* __restrict__ ranks, const RoundState* __restrict__ rs, const int64_t* __restrict__ off, int W,
    const int32_t* __restrict__ gstart, const int32_t* __restrict__ gsize, const int32_t* __restrict__ kept,
    const int32_t* __restrict__ cur_len, const int64_t* __restrict__ cs, int32_t* __restrict__ srows,
    int32_t* __restrict__ smax, int64_t* __restrict__ stok, double* __restrict__ sadj,
    int64_t* __restrict__ steps, const DevStatus* st) {
#pragma clang fp contract(off)
    if (stage1_bad(st)) return;
    const int64_t T = rs->T;
    const int64_t total = (int64_t)W * T;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total; idx += stride) {
        const int r = (int)(idx / T);
        const int64_t j = idx - (int64_t)r * T;
        const RankState R = ranks[r];
        if (R.action == kActInactive) continue;
        const int64_t base = off[r];
        int64_t start, end;
        if (R.action == kActOverflow) {
            const int64_t g = R.gbase + kept[R.gbase + j];
            start = gstart[g];
            end = start + gsize[g];
        } else {
            adjusted_range(R, base, T - 1 - j, gstart, gsize, &start, &end);
        }
        const int64_t rows = end - start;
        const int64_t dst = base + R.slots + j;
        srows[dst] = (int32_t)rows;
        smax[dst] = cur_len[start];
        stok[dst] = cs[end - 1] - (start > 0 ? cs[start - 1] : 0);
        // live positions of the rank are [base, base + cnt); cs is inclusive over all n
        const int64_t buf_tok = cs[base + R.cnt - 1] - (base > 0 ? cs[base - 1] : 0);
        const double mean = (double)buf_tok / (double)R.cnt;
        sadj[dst] = (double)rows * mean;
        atomicAdd((unsigned long long*)&steps[j], (unsigned long long)rows);
    }
}

// Steps of this round that are emitted: join, all T; non-join, up to the first step at
// which the cumulative global emitted count reaches the quota (Theorem 2).  Block-uniform;
// *sum and *mx receive the emitted steps' sample total and largest step.
__device__ int64_t round_cut(const int64_t* __restrict__ steps, int64_t T, int64_t before, int nonjoin,
                             int64_t quota, int64_t* sum_out, int64_t* mx_out) {
    __shared__ int64_t s_cut;
    if (threadIdx.x == 0) s_cut = T;
    __syncthreads();
    if (nonjoin) {
        int64_t carry = 0;
        for (int64_t b = 0; b < T; b += kBlock) {
            const int64_t j = b + threadIdx.x;
            const int64_t v = j < T ? steps[j] : 0;
            int64_t tot;
            const int64_t ex = block_excl_sum(v, &tot);
            if (j < T && before + carry + ex < quota && before + carry + ex + v >= quota) s_cut = j + 1;
            __syncthreads();
            if (s_cut < T) break;
            carry += tot;
        }
    }
    const int64_t cut = s_cut;
    int64_t sum = 0, mx = 0;
    for (int64_t j = threadIdx.x; j < cut; j += kBlock) {
        const int64_t v = steps[j];
        sum += v;
        mx = v > mx ? v : mx;
    }
    *sum_out = block_reduce(sum, SumOp{});
    *mx_out = block_reduce(mx, MaxOp{});
    return cut;
}

// Per rank (one block each): the round's cut (every block computes it; block 0 records it
// and the running totals, which advance_kernel makes current), then the rank's emitted
// positions and the layout of its next buffer.
__global__ void __launch_bounds__(kBlock) finalize_kernel(RankState* ranks, RoundState* rs,
                                                          const int64_t* __restrict__ steps, int nonjoin,
                                                          int64_t quota, const int64_t* __restrict__ off,
                                                          const int32_t* __restrict__ gstart,
                                                          const int32_t* __restrict__ gsize,
                                                          const int32_t* __restrict__ ov_slot,
                                                          const int32_t* __restrict__ kept,
                                                          int32_t* __restrict__ ov_lo, const DevStatus* st) {
    if (stage1_bad(st)) return;
    const int r = blockIdx.x;
    RankState& R = ranks[r];
    const int64_t T = rs->T;
    const int64_t before = rs->emitted_total;
    int64_t step_sum, step_mx;
    const int64_t cut = round_cut(steps, T, before, nonjoin, quota, &step_sum, &step_mx);
    if (r == 0 && threadIdx.x == 0) {
        rs->cut = cut;
        rs->emitted_next = before + step_sum;
        if (step_mx > rs->step_max) rs->step_max = step_mx;
        if (nonjoin && before + step_sum >= quota) rs->quota_hit = 1;
    }
    if (threadIdx.x == 0) R.ebase = R.emitted;
    if (R.action == kActInactive) {
        if (threadIdx.x == 0) R.next_cnt = 0;
        return;
    }
    const int64_t base = off[r];
    if (R.action != kActOverflow) {
        if (threadIdx.x == 0) {
            int64_t q = 0;
            if (cut < T) {
                int64_t s, e;
                adjusted_range(R, base, T - cut, gstart, gsize, &s, &e);
                q = s - base;
            }
            R.qcut = q;
            R.next_cnt = q;
            R.emitted += R.cnt - q;
            R.slots += cut;
        }
        return;
    }
    const int64_t G = R.G, gb = R.gbase;
    // emitted groups, slot order: consecutive emission offsets
    int64_t carry = 0;
    for (int64_t b = 0; b < cut; b += kBlock) {
        const int64_t j = b + threadIdx.x;
        const int64_t g = j < cut ? gb + kept[gb + j] : 0;
        const int64_t v = j < cut ? gsize[g] : 0;
        int64_t tot;
        const int64_t ex = block_excl_sum(v, &tot);
        if (j < cut) ov_lo[g] = (int32_t)(carry + ex);
        carry += tot;
    }
    const int64_t emitted_now = carry;
    // everything else, formation order: offsets in the next buffer
    carry = 0;
    for (int64_t b = 0; b < G; b += kBlock) {
        const int64_t j = b + threadIdx.x;
        const int32_t sl = j < G ? ov_slot[gb + j] : 0;
        const bool stay = j < G && (sl < 0 || sl >= cut);
        const int64_t v = stay ? gsize[gb + j] : 0;
        int64_t tot;
        const int64_t ex = block_excl_sum(v, &tot);
        if (stay) ov_lo[gb + j] = (int32_t)(carry + ex);
        carry += tot;
    }
    if (threadIdx.x == 0) {
        R.next_cnt = carry;
        R.emitted += emitted_now;
        R.slots += cut;
    }
}

__global__ void __launch_bounds__(kBlock) emit_kernel(
    const RankState* __restrict__ ranks, const RoundState* __restrict__ rs, const int64_t* __restrict__ off, int W,
    int64_t n, const int32_t* __restrict__ cur_ids, const int32_t* __restrict__ cur_len,
    const int32_t* __restrict__ gidx, const int32_t* __restrict__ gstart, const int32_t* __restrict__ gsize,
    const int32_t* __restrict__ ov_slot, const int32_t* __restrict__ ov_lo, int32_t* __restrict__ dst,
    int32_t* __restrict__ dst_len, int32_t* __restrict__ next_ids, int32_t* __restrict__ next_len,
    const DevStatus* st) {
    if (stage1_bad(st)) return;
    __shared__ int64_t s_off[kLdsRanks + 1];
    off = stage_ranks(off, W, s_off);
    const int64_t cut = rs->cut;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; p < n; p += stride) {
        const int r = rank_of(off, W, p);
        const int64_t base = off[r];
        const int64_t q = p - base;
        const RankState& R = ranks[r];
        const int64_t cnt = R.cnt;
        if (q >= cnt) continue;
        const int32_t id = cur_ids[p];
        if (R.action != kActOverflow) {
            if (q >= R.qcut) {
                const int64_t o = base + R.ebase + (cnt - 1 - q);
                dst[o] = id;
                dst_len[o] = cur_len[p];
            } else {
                next_ids[base + q] = id;
                next_len[base + q] = cur_len[p];
            }
        } else {
            const int64_t g = R.gbase + gidx[p];
            const int32_t sl = ov_slot[g];
            const int64_t st = (int64_t)gstart[g] - base;
            if (sl >= 0 && sl < cut) {
                const int64_t o = base + R.ebase + ov_lo[g] + (st + gsize[g] - 1 - q);
                dst[o] = id;
                dst_len[o] = cur_len[p];
            } else {
                const int64_t o = ov_lo[g] + (q - st);
                next_ids[base + o] = id;
                next_len[base + o] = cur_len[p];
            }
        }
    }
}

// End of a round: the next buffers' counts and the running emitted total become current.
__global__ void advance_kernel(RankState* ranks, int W, RoundState* rs) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i == 0) rs->emitted_total = rs->emitted_next;
    for (int r = i; r < W; r += gridDim.x * blockDim.x) ranks[r].cnt = ranks[r].next_cnt;
}

// ---------------------------------------------------------------- final plan
__global__ void __launch_bounds__(kBlock) plan_slots_kernel(const RankState* __restrict__ ranks,
                                                            const int64_t* __restrict__ off, int W, int64_t S,
                                                            const int32_t* __restrict__ srows,
                                                            const int32_t* __restrict__ smax,
                                                            const int64_t* __restrict__ stok,
                                                            const double* __restrict__ sadj,
                                                            int32_t* __restrict__ rows, int32_t* __restrict__ maxlen,
                                                            int64_t* __restrict__ tokens, double* __restrict__ approx,
                                                            DevInfo* info) {
    const int64_t K = (int64_t)W * S;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    int64_t real = 0;
    for (int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; k < K; k += stride) {
        const int r = (int)(k / S);
        const int64_t j = k - (int64_t)r * S;
        if (j < ranks[r].slots) {
            const int64_t src = off[r] + j;
            rows[k] = srows[src];
            maxlen[k] = smax[src];
            tokens[k] = stok[src];
            real += stok[src];
            if (approx) approx[k] = sadj[src];
        } else {
            rows[k] = 0;
            maxlen[k] = 0;
            tokens[k] = 0;
            if (approx) approx[k] = 0.0;
        }
    }
    // the plan's real tokens (Sec. 2.1 / App. I padding fraction)
    real = block_sum(real);
    if (threadIdx.x == 0 && real) atomicAdd((unsigned long long*)&info->real_tokens, (unsigned long long)real);
}

// The row and tile offsets of the slots in one scan: a slot contributes (rows, rows *
// maxlen).
struct RowsTilesLoad {
    const int32_t* rows;
    const int32_t* mx;
    int64_t K;
    __device__ I64Pair operator()(int64_t i) const {
        return i < K ? I64Pair{(int64_t)rows[i], (int64_t)rows[i] * mx[i]} : I64Pair{0, 0};
    }
};
struct RowsTilesStore {
    int64_t* row_off;
    int64_t* tile_off;
    __device__ void operator()(int64_t i, I64Pair v) const {
        row_off[i] = v.a;
        tile_off[i] = v.b;
    }
};

__global__ void __launch_bounds__(kBlock) compact_emit_kernel(const int32_t* __restrict__ stage,
                                                              const int32_t* __restrict__ stage_len,
                                                              const int64_t* __restrict__ off,
                                                              const RankState* __restrict__ ranks, int W, int64_t n,
                                                              const int64_t* __restrict__ row_off, int64_t S,
                                                              int32_t* __restrict__ emit, int32_t* __restrict__ len) {
    __shared__ int64_t s_off[kLdsRanks + 1];
    off = stage_ranks(off, W, s_off);
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; p < n; p += stride) {
        const int r = rank_of(off, W, p);
        const int64_t e = p - off[r];
        if (e < ranks[r].emitted) {
            const int64_t o = row_off[(int64_t)r * S] + e;
            emit[o] = stage[p];
            len[o] = stage_len[p];
        }
    }
}

// Row records of the emitted rows: the CSR token start of each row's sample (written
// when `ts` is not NULL) and the check that the length the plan carried for it (from
// the stage-1 sorted lengths) is the sample's CSR length.  Ids are in range here:
// round0_check_kernel verified that every rank's order is a permutation of its ids.
//
// The offsets are gathered in random order, one 128-byte line per 8-byte read unless the
// line is still cached.  A rank's rows hold only that rank's ids, whose offsets span
// 8 B per sample (2 MB at 262,144 samples), so with `xcd_ranks` set, rank r is gathered
// only by the blocks of group r mod kXcds (workgroups are dealt to the XCDs round
// robin, so block b runs on XCD b mod kXcds): each rank's offsets then stay in one XCD's
// L2 and are read from HBM about once.
constexpr int kXcds = 8;

// The CSR length of sample s against the length its plan row carries: a length outside
// [1, 2^31) or a negative offset is invalid data (grouping took such a sample as length
// 1); any other difference means the stage-1 arrays are not this window's.
__device__ __forceinline__ void check_csr_length(int32_t s, int64_t a, int64_t b, int32_t carried, DevStatus* st) {
    const int64_t l = b - a;
    if (l < 1 || l > INT_MAX || a < 0) {
        atomicOr(&st->err, kErrLength);
        atomicMin((unsigned long long*)&st->first_bad_len, (unsigned long long)s);
    } else if (l != (int64_t)carried) {
        atomicOr(&st->err, kErrSortedLen);
        atomicMin((unsigned long long*)&st->first_bad, (unsigned long long)s);
    }
}

__global__ void __launch_bounds__(kBlock) row_check_kernel(const int64_t* __restrict__ tok_off,
                                                           const int32_t* __restrict__ emit,
                                                           const int32_t* __restrict__ len,
                                                           const int64_t* __restrict__ row_off, int64_t S, int W,
                                                           int xcd_ranks, int64_t* __restrict__ ts, DevStatus* st) {
    const int group = xcd_ranks ? (int)(blockIdx.x % kXcds) : 0;
    const int groups = xcd_ranks ? kXcds : 1;
    const int64_t gb = xcd_ranks ? blockIdx.x / kXcds : blockIdx.x;   // block within its group
    const int64_t nb = xcd_ranks ? gridDim.x / kXcds : gridDim.x;
    const int64_t stride = nb * blockDim.x;
    for (int r = group; r < W; r += groups) {
        // all ranks at once in the plain mode: the rows of ranks group .. W-1 are contiguous
        const int64_t lo = row_off[(int64_t)r * S];
        const int64_t hi = row_off[(int64_t)(xcd_ranks ? r + 1 : W) * S];
        for (int64_t k = lo + gb * blockDim.x + threadIdx.x; k < hi; k += stride) {
            const int32_t s = emit[k];
            const int64_t a = tok_off[s];
            check_csr_length(s, a, tok_off[s + 1], len[k], st);
            if (ts) ts[k] = a;
        }
        if (!xcd_ranks) break;
    }
}

__global__ void __launch_bounds__(kBlock) leftover_off_kernel(const RankState* __restrict__ ranks, int W,
                                                              int64_t* __restrict__ loff) {
    __shared__ int64_t carry;
    if (threadIdx.x == 0) carry = 0;
    __syncthreads();
    for (int b = 0; b < W; b += kBlock) {
        const int r = b + threadIdx.x;
        const int64_t v = r < W ? ranks[r].cnt : 0;
        int64_t tot;
        const int64_t ex = block_excl_sum(v, &tot);
        const int64_t c = carry;
        if (r < W) loff[r] = c + ex;
        __syncthreads();
        if (threadIdx.x == 0) carry = c + tot;
        __syncthreads();
    }
    if (threadIdx.x == 0) loff[W] = carry;
}

// Left-over ids, and the length check of row_check_kernel for them.
__global__ void __launch_bounds__(kBlock) leftover_kernel(const int32_t* __restrict__ cur_ids,
                                                          const int32_t* __restrict__ cur_len,
                                                          const int64_t* __restrict__ tok_off,
                                                          const int64_t* __restrict__ off,
                                                          const RankState* __restrict__ ranks, int W, int64_t n,
                                                          const int64_t* __restrict__ loff,
                                                          int32_t* __restrict__ left, DevStatus* st) {
    __shared__ int64_t s_off[kLdsRanks + 1];
    off = stage_ranks(off, W, s_off);
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; p < n; p += stride) {
        const int r = rank_of(off, W, p);
        const int64_t q = p - off[r];
        if (q < ranks[r].cnt) {
            const int32_t s = cur_ids[p];
            left[loff[r] + q] = s;
            check_csr_length(s, tok_off[s], tok_off[s + 1], cur_len[p], st);
        }
    }
}

// ---------------------------------------------------------------- coverage
// cnt[v] += 1 for every view id (or its identity) in ids[0, m).
__global__ void __launch_bounds__(kBlock) count_kernel(const int32_t* __restrict__ ids, int64_t m, int64_t n,
                                                       const int64_t* __restrict__ identity, int64_t range,
                                                       int32_t* cnt, DevStatus* st) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < m; i += stride) {
        int64_t v = ids[i];
        if (v < 0 || v >= n) {
            atomicOr(&st->err, kErrInternal);
            continue;
        }
        if (identity) v = identity[v];
        if (v < 0 || v >= range) {
            atomicOr(&st->err, kErrIdentity);
            continue;
        }
        atomicAdd(&cnt[v], 1);
    }
}

// bad = #(cnt != 1) (views); missing = #(cnt == 0); dup = sum max(cnt - 1, 0).
__global__ void __launch_bounds__(kBlock) coverage_reduce_kernel(const int32_t* __restrict__ cnt, int64_t m,
                                                                 int want_bad, int want_ids, DevInfo* info) {
    int64_t bad = 0, miss = 0, dup = 0;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < m; i += stride) {
        const int32_t c = cnt[i];
        bad += c != 1 ? 1 : 0;
        miss += c == 0 ? 1 : 0;
        dup += c > 1 ? c - 1 : 0;
    }
    bad = block_sum(bad);
    miss = block_sum(miss);
    dup = block_sum(dup);
    if (threadIdx.x == 0) {
        if (want_bad && bad) atomicAdd((unsigned long long*)&info->bad_views, (unsigned long long)bad);
        if (want_ids && miss) atomicAdd((unsigned long long*)&info->missing_ids, (unsigned long long)miss);
        if (want_ids && dup) atomicAdd((unsigned long long*)&info->duplicate_ids, (unsigned long long)dup);
    }
}

// Sets bit v of `bits` for every view id v in ids[0, m) (ids outside [0, n) are errors).
__global__ void __launch_bounds__(kBlock) mark_views_kernel(const int32_t* __restrict__ ids, int64_t m, int64_t n,
                                                            uint32_t* bits, DevStatus* st) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < m; i += stride) {
        const int32_t v = ids[i];
        if (v < 0 || v >= n) {
            atomicOr(&st->err, kErrInternal);
            continue;
        }
        atomicOr(&bits[v >> 5], 1u << (v & 31));
    }
}

__global__ void __launch_bounds__(kBlock) popcount_kernel(const uint32_t* __restrict__ bits, int64_t words,
                                                          DevInfo* info) {
    int64_t c = 0;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < words; i += stride) c += __popc(bits[i]);
    c = block_sum(c);
    if (threadIdx.x == 0 && c) atomicAdd((unsigned long long*)&info->distinct_views, (unsigned long long)c);
}

// Coverage (App. C): a bitset over the sampler views proves "every view exactly once"
// when it holds n distinct views and n ids were listed; the exact per-view counters run
// only when it does not (run_coverage_exact).  Identities of an identity map are always
// counted exactly (duplicates are expected there: sampler padding).
int run_coverage(const odb_window_t* w, const Layout& L, void* ws, const int32_t* emitted, int64_t ne,
                 const int32_t* left, int64_t nl, hipStream_t s) {
    const int64_t n = w->num_samples;
    int32_t* cover = ws_at<int32_t>(ws, L.cover);
    DevStatus* st = ws_at<DevStatus>(ws, L.status);
    DevInfo* info = ws_at<DevInfo>(ws, L.info);
    const int64_t cap = (int64_t)num_cus() * kPlanBlocksPerCU;
    if (n > 0) {
        uint32_t* bits = reinterpret_cast<uint32_t*>(cover);
        const int64_t words = (n + 31) / 32;
        hipLaunchKernelGGL(fill_i32_kernel, dim3(grid_for(words, kBlock, cap)), dim3(kBlock), 0, s, cover, words, 0);
        ODB_LAUNCHED();
        if (ne > 0) {
            hipLaunchKernelGGL(mark_views_kernel, dim3(grid_for(ne, kBlock, cap)), dim3(kBlock), 0, s, emitted, ne, n,
                               bits, st);
            ODB_LAUNCHED();
        }
        if (nl > 0) {
            hipLaunchKernelGGL(mark_views_kernel, dim3(grid_for(nl, kBlock, cap)), dim3(kBlock), 0, s, left, nl, n,
                               bits, st);
            ODB_LAUNCHED();
        }
        hipLaunchKernelGGL(popcount_kernel, dim3(grid_for(words, kBlock, cap)), dim3(kBlock), 0, s,
                           (const uint32_t*)bits, words, info);
        ODB_LAUNCHED();
    }
    if (w->d_identity && n > 0) {
        // the identity counters reuse the bitset's memory: the popcount above has consumed it
        const int64_t nid = w->num_identities;
        hipLaunchKernelGGL(fill_i32_kernel, dim3(grid_for(nid, kBlock, cap)), dim3(kBlock), 0, s, cover, nid, 0);
        ODB_LAUNCHED();
        if (ne > 0) {
            hipLaunchKernelGGL(count_kernel, dim3(grid_for(ne, kBlock, cap)), dim3(kBlock), 0, s, emitted, ne, n,
                               w->d_identity, nid, cover, st);
            ODB_LAUNCHED();
        }
        if (nl > 0) {
            hipLaunchKernelGGL(count_kernel, dim3(grid_for(nl, kBlock, cap)), dim3(kBlock), 0, s, left, nl, n,
                               w->d_identity, nid, cover, st);
            ODB_LAUNCHED();
        }
        hipLaunchKernelGGL(coverage_reduce_kernel, dim3(grid_for(nid, kBlock, cap)), dim3(kBlock), 0, s,
                           (const int32_t*)cover, nid, 0, 1, info);
        ODB_LAUNCHED();
    }
    return ODB_OK;
}

// Exact per-view counts: bad_views (and missing / duplicates without an identity map).
// Needed only when the bitset pass found fewer than n distinct views or n != ne + nl.
int run_coverage_exact(const odb_window_t* w, const Layout& L, void* ws, const int32_t* emitted, int64_t ne,
                       const int32_t* left, int64_t nl, hipStream_t s) {
    const int64_t n = w->num_samples;
    int32_t* cover = ws_at<int32_t>(ws, L.cover);
    DevStatus* st = ws_at<DevStatus>(ws, L.status);
    DevInfo* info = ws_at<DevInfo>(ws, L.info);
    const int64_t cap = (int64_t)num_cus() * kPlanBlocksPerCU;
    hipLaunchKernelGGL(fill_i32_kernel, dim3(grid_for(n, kBlock, cap)), dim3(kBlock), 0, s, cover, n, 0);
    ODB_LAUNCHED();
    if (ne > 0) {
        hipLaunchKernelGGL(count_kernel, dim3(grid_for(ne, kBlock, cap)), dim3(kBlock), 0, s, emitted, ne, n,
                           (const int64_t*)nullptr, n, cover, st);
        ODB_LAUNCHED();
    }
    if (nl > 0) {
        hipLaunchKernelGGL(count_kernel, dim3(grid_for(nl, kBlock, cap)), dim3(kBlock), 0, s, left, nl, n,
                           (const int64_t*)nullptr, n, cover, st);
        ODB_LAUNCHED();
    }
    hipLaunchKernelGGL(coverage_reduce_kernel, dim3(grid_for(n, kBlock, cap)), dim3(kBlock), 0, s,
                       (const int32_t*)cover, n, 1, w->d_identity ? 0 : 1, info);
    ODB_LAUNCHED();
    return ODB_OK;
}

// Coverage of one rank's views, one id chunk per block, in LDS.  The views of rank r are
// its ids [off[r], off[r+1]); they may appear only in rank r's emitted rows
// (emit[row_off[r*S] .. row_off[(r+1)*S])) and leftovers (left[loff[r] .. loff[r+1])).
// Block b covers ids [lo, hi) of one rank: it scans both lists, sets bit v in `once`,
// and in `twice` if it was already set.  missing = (hi - lo) - |once|, views listed
// more than once = |twice|, extra listings = dup.  An id of another rank in these lists
// is an internal error.
constexpr int kCovBlock = 1024;

// The chunk's view of one listed id.  Ids, ranks and chunks stay below 2^31, so the
// range tests are single unsigned compares: (uint32)(x - base) < nr holds exactly for
// base <= x < base + nr, negative x included.
struct CovChunk {
    uint32_t* once;
    uint32_t* twice;
    uint32_t base, nr;  // the rank's views [base, base + nr)
    uint32_t lo, span;  // this chunk's views [lo, lo + span)
    int32_t dup, foreign;
    int first;          // chunk 0 of its rank counts the foreign ids

    __device__ __forceinline__ void add(int32_t x) {
        if ((uint32_t)x - base >= nr) {
            foreign += first;
            return;
        }
        const uint32_t d = (uint32_t)x - lo;
        if (d >= span) return;
        const uint32_t bit = 1u << (d & 31);
        if (atomicOr(&once[d >> 5], bit) & bit) {
            atomicOr(&twice[d >> 5], bit);
            dup += 1;
        }
    }
};

typedef int v4i_cov __attribute__((ext_vector_type(4)));

// Feeds ids[a, b) to the chunk: a scalar head up to the first 16-byte aligned address,
// two 16-byte loads per thread and iteration, a scalar tail.
__device__ __forceinline__ void cov_scan(CovChunk& c, const int32_t* __restrict__ ids, int64_t a, int64_t b) {
    if (b <= a) return;
    int64_t a4 = a + ((4 - ((reinterpret_cast<uintptr_t>(ids + a) >> 2) & 3)) & 3);
    if (a4 > b) a4 = b;
    const int64_t b4 = a4 + ((b - a4) & ~(int64_t)3);
    if (a + threadIdx.x < a4) c.add(ids[a + threadIdx.x]);
    if (b4 + threadIdx.x < b) c.add(ids[b4 + threadIdx.x]);
    const v4i_cov* v = reinterpret_cast<const v4i_cov*>(ids + a4);
    const int32_t nv = (int32_t)((b4 - a4) >> 2);
    for (int32_t q = threadIdx.x; q < nv; q += 2 * kCovBlock) {
        const v4i_cov x = __builtin_nontemporal_load(v + q);
        const bool two = q + kCovBlock < nv;
        const v4i_cov y = __builtin_nontemporal_load(v + (two ? q + kCovBlock : q));
#pragma unroll
        for (int k = 0; k < 4; ++k) c.add(x[k]);
        if (two) {
#pragma unroll
            for (int k = 0; k < 4; ++k) c.add(y[k]);
        }
    }
}

__global__ void __launch_bounds__(kCovBlock) coverage_lds_kernel(
    const int64_t* __restrict__ off, int W, const int64_t* __restrict__ chunk_first, int64_t C,
    const int32_t* __restrict__ emit, const int64_t* __restrict__ row_off, int64_t S,
    const int32_t* __restrict__ left, const int64_t* __restrict__ loff, int want_ids, DevInfo* info,
    DevStatus* st) {
    extern __shared__ uint32_t lds[];
    const int64_t words = C / 32;
    const int64_t b = blockIdx.x;
    const int r = rank_of(chunk_first, W, b);
    const int64_t j = b - chunk_first[r];
    const int64_t base = off[r], end = off[r + 1];
    const int64_t lo = base + j * C;
    const int64_t hi = lo + C < end ? lo + C : end;
    CovChunk c{lds, lds + words, (uint32_t)base, (uint32_t)(end - base), (uint32_t)lo, (uint32_t)(hi - lo), 0, 0,
               j == 0 ? 1 : 0};
    for (int64_t i = threadIdx.x; i < 2 * words; i += kCovBlock) lds[i] = 0;
    __syncthreads();
    cov_scan(c, emit, row_off[(int64_t)r * S], row_off[(int64_t)(r + 1) * S]);
    cov_scan(c, left, loff[r], loff[r + 1]);
    __syncthreads();
    int32_t distinct = 0, multi = 0;
    const int32_t nw = (int32_t)((hi - lo + 31) / 32);
    for (int32_t i = threadIdx.x; i < nw; i += kCovBlock) {
        distinct += __popc(c.once[i]);
        multi += __popc(c.twice[i]);
    }
    // block sums of the four counters: per-wave partials in LDS, summed by wave 0
    __shared__ int64_t part[kCovBlock / kWave][4];
    const int64_t v0 = wave_sum((int64_t)distinct), v1 = wave_sum((int64_t)multi);
    const int64_t v2 = wave_sum((int64_t)c.dup), v3 = wave_sum((int64_t)c.foreign);
    if ((threadIdx.x & (kWave - 1)) == 0) {
        int64_t* q = part[threadIdx.x / kWave];
        q[0] = v0;
        q[1] = v1;
        q[2] = v2;
        q[3] = v3;
    }
    __syncthreads();
    if (threadIdx.x < kWave) {
        const int i = threadIdx.x;
        const bool has = i < kCovBlock / kWave;
        const int64_t d_sum = wave_sum(has ? part[i][0] : (int64_t)0);
        const int64_t m_sum = wave_sum(has ? part[i][1] : (int64_t)0);
        const int64_t dup = wave_sum(has ? part[i][2] : (int64_t)0);
        const int64_t foreign = wave_sum(has ? part[i][3] : (int64_t)0);
        if (i != 0) return;
        const int64_t missing = (hi - lo) - d_sum;
        const int64_t bad = missing + m_sum;
        if (bad) atomicAdd((unsigned long long*)&info->bad_views, (unsigned long long)bad);
        if (want_ids && missing) atomicAdd((unsigned long long*)&info->missing_ids, (unsigned long long)missing);
        if (want_ids && dup) atomicAdd((unsigned long long*)&info->duplicate_ids, (unsigned long long)dup);
        if (foreign) atomicOr(&st->err, kErrInternal);
    }
}

// The plan's totals (padded elements, emitted rows, pad fraction) and the coverage chunks:
// chunk_first[r] = sum_{r' < r} ceil(n_r' / C).  One block.
__global__ void __launch_bounds__(kBlock) finish_plan_kernel(const int64_t* __restrict__ row_off,
                                                             const int64_t* __restrict__ tile_off, int64_t K,
                                                             DevInfo* info, const int64_t* __restrict__ off, int W,
                                                             int64_t C, int64_t* __restrict__ chunk_first) {
    __shared__ int64_t carry;
    if (threadIdx.x == 0) {
        carry = 0;
        info->padded_elems = K > 0 ? tile_off[K] : 0;
        info->emitted = K > 0 ? row_off[K] : 0;
        info->pad_fraction =
            info->padded_elems > 0 ? 1.0 - (double)info->real_tokens / (double)info->padded_elems : 0.0;
    }
    __syncthreads();
    for (int b = 0; b < W; b += kBlock) {
        const int r = b + threadIdx.x;
        const int64_t v = r < W ? (off[r + 1] - off[r] + C - 1) / C : 0;
        int64_t tot;
        const int64_t ex = block_excl_sum(v, &tot);
        const int64_t c = carry;
        if (r < W) chunk_first[r] = c + ex;
        __syncthreads();
        if (threadIdx.x == 0) carry = c + tot;
        __syncthreads();
    }
    if (threadIdx.x == 0) chunk_first[W] = carry;
}

// Coverage of an aligned plan: per-rank LDS bitsets for the views, global counters for
// the identities of an identity map.
int run_plan_coverage(const odb_window_t* w, const Layout& L, void* ws, const int32_t* emit,
                      const int64_t* row_off, const int64_t* tile_off, int64_t S, const int32_t* left,
                      const int64_t* loff, int64_t ne, int64_t nl, hipStream_t s) {
    const int W = w->num_ranks;
    const int64_t n = w->num_samples;
    int64_t max_nr = 0, chunks = 0;
    for (int r = 0; r < W; ++r) {
        const int64_t nr = w->rank_offsets[r + 1] - w->rank_offsets[r];
        max_nr = nr > max_nr ? nr : max_nr;
    }
    // one chunk per rank up to 131072 views (two 16 KB bitsets); larger ranks are split
    int64_t C = ((max_nr + 4095) / 4096) * 4096;
    C = C < 4096 ? 4096 : (C > 131072 ? 131072 : C);
    for (int r = 0; r < W; ++r) chunks += (w->rank_offsets[r + 1] - w->rank_offsets[r] + C - 1) / C;
    int64_t* chunk_first = ws_at<int64_t>(ws, L.tile_first);
    const int64_t* d_off = ws_at<int64_t>(ws, L.rank_off);
    hipLaunchKernelGGL(finish_plan_kernel, dim3(1), dim3(kBlock), 0, s, row_off, tile_off, (int64_t)W * S,
                       ws_at<DevInfo>(ws, L.info), d_off, W, C, chunk_first);
    ODB_LAUNCHED();
    if (n == 0) return ODB_OK;
    hipLaunchKernelGGL(coverage_lds_kernel, dim3((unsigned)chunks), dim3(kCovBlock), (size_t)(C / 4), s, d_off, W,
                       (const int64_t*)chunk_first, C, emit, row_off, S, left, loff, w->d_identity ? 0 : 1,
                       ws_at<DevInfo>(ws, L.info), ws_at<DevStatus>(ws, L.status));
    ODB_LAUNCHED();
    if (w->d_identity) {
        int32_t* cover = ws_at<int32_t>(ws, L.cover);
        DevStatus* st = ws_at<DevStatus>(ws, L.status);
        const int64_t nid = w->num_identities;
        const int64_t cap = (int64_t)num_cus() * kPlanBlocksPerCU;
        hipLaunchKernelGGL(fill_i32_kernel, dim3(grid_for(nid, kBlock, cap)), dim3(kBlock), 0, s, cover, nid, 0);
        ODB_LAUNCHED();
        if (ne > 0) {
            hipLaunchKernelGGL(count_kernel, dim3(grid_for(ne, kBlock, cap)), dim3(kBlock), 0, s, emit, ne, n,
                               w->d_identity, nid, cover, st);
            ODB_LAUNCHED();
        }
        if (nl > 0) {
            hipLaunchKernelGGL(count_kernel, dim3(grid_for(nl, kBlock, cap)), dim3(kBlock), 0, s, left, nl, n,
                               w->d_identity, nid, cover, st);
            ODB_LAUNCHED();
        }
        hipLaunchKernelGGL(coverage_reduce_kernel, dim3(grid_for(nid, kBlock, cap)), dim3(kBlock), 0, s,
                           (const int32_t*)cover, nid, 0, 1, ws_at<DevInfo>(ws, L.info));
        ODB_LAUNCHED();
    }
    return ODB_OK;
}

// Reads the coverage counters after run_coverage; runs the exact view count when the
// bitset pass did not prove that every view was listed exactly once.
int finish_coverage(const odb_window_t* w, const Layout& L, void* ws, const int32_t* emitted, int64_t ne,
                    const int32_t* left, int64_t nl, DevInfo* hi, hipStream_t s) {
    const int64_t n = w->num_samples;
    if (hi->distinct_views == n && ne + nl == n) {
        hi->bad_views = 0;
        if (!w->d_identity) {
            hi->missing_ids = 0;
            hi->duplicate_ids = 0;
        }
        return ODB_OK;
    }
    DevInfo* info = ws_at<DevInfo>(ws, L.info);
    hipLaunchKernelGGL(clear_view_counters_kernel, dim3(1), dim3(64), 0, s, info, w->d_identity ? 0 : 1);
    ODB_LAUNCHED();
    ODB_TRY(run_coverage_exact(w, L, ws, emitted, ne, left, nl, s));
    ODB_TRY_HIP(hipMemcpyAsync(hi, info, sizeof(*hi), hipMemcpyDeviceToHost, s));
    ODB_TRY_HIP(hipStreamSynchronize(s));
    return ODB_OK;
}

struct RoundBuffers {
    const int32_t* ids;
    const int32_t* len;
    const int32_t* gidx;
};

}  // namespace

}  // namespace odb

using namespace odb;

extern "C" int odb_align_groups(const odb_window_t* w, int64_t budget, const odb_align_params_t* params,
                                const int32_t* d_order, const int32_t* d_sorted_len, const int32_t* d_group_index,
                                const int32_t* d_groups_per_rank, int64_t slot_capacity, int32_t* d_emit_order,
                                int64_t* d_row_token_start, int32_t* d_row_len, int32_t* d_slot_rows, int32_t* d_slot_maxlen, int64_t* d_slot_row_off,
                                int64_t* d_slot_tile_off, int64_t* d_slot_tokens, double* d_slot_tokens_approx,
                                int32_t* d_leftover, int64_t* d_leftover_off, odb_plan_info_t* h_info, void* d_ws,
                                size_t ws_bytes, void* stream) {
    Layout L;
    ODB_TRY(check_workspace(w, d_ws, ws_bytes, &L));
    if (budget < 1) return set_error(ODB_E_INVALID_ARG, "budget must be >= 1");
    if (!params) return set_error(ODB_E_INVALID_ARG, "params is NULL");
    if (params->mode != ODB_MODE_JOIN && params->mode != ODB_MODE_NONJOIN_QUOTA)
        return set_error(ODB_E_INVALID_ARG, "unknown mode %d", params->mode);
    if (params->reserved0 != 0) return set_error(ODB_E_INVALID_ARG, "params.reserved0 must be 0");
    const bool nonjoin = params->mode == ODB_MODE_NONJOIN_QUOTA;
    if (nonjoin && params->quota < 1) return set_error(ODB_E_INVALID_ARG, "quota must be >= 1 in non-join mode");
    if (!h_info) return set_error(ODB_E_INVALID_ARG, "h_info is NULL");
    if (slot_capacity < 0) return set_error(ODB_E_INVALID_ARG, "slot_capacity must be >= 0");
    if ((d_row_token_start == nullptr) != (d_row_len == nullptr))
        return set_error(ODB_E_INVALID_ARG, "d_row_token_start and d_row_len are given together or not at all");
    const int W = w->num_ranks;
    const int64_t n = w->num_samples;
    if (n > 0 && (!d_order || !d_sorted_len || !d_group_index || !d_emit_order || !d_leftover))
        return set_error(ODB_E_INVALID_ARG, "sample arrays must not be NULL");
    if (!d_groups_per_rank || !d_slot_row_off || !d_slot_tile_off || !d_leftover_off)
        return set_error(ODB_E_INVALID_ARG, "offset arrays must not be NULL");
    if (slot_capacity > 0 && (!d_slot_rows || !d_slot_maxlen || !d_slot_tokens))
        return set_error(ODB_E_INVALID_ARG, "slot arrays must not be NULL");
    const int64_t* cap = params->slot_capacity;
    if (cap)
        for (int r = 0; r < W; ++r)
            if (cap[r] < 0) return set_error(ODB_E_INVALID_ARG, "slot_capacity[%d] must be >= 0", r);
    memset(h_info, 0, sizeof(*h_info));

    hipStream_t s = static_cast<hipStream_t>(stream);
    ODB_TRY(upload_small(w, L, d_ws, cap, s));
    const int64_t* d_off = ws_at<int64_t>(d_ws, L.rank_off);
    const int64_t* d_cap = ws_at<int64_t>(d_ws, L.cap);
    RankState* d_ranks = ws_at<RankState>(d_ws, L.ranks);
    RoundState* d_rs = ws_at<RoundState>(d_ws, L.round);
    DevStatus* st = ws_at<DevStatus>(d_ws, L.status);
    DevInfo* d_info = ws_at<DevInfo>(d_ws, L.info);
    int64_t* d_gbase = ws_at<int64_t>(d_ws, L.gbase);
    int32_t* gstart = ws_at<int32_t>(d_ws, L.gstart);
    int32_t* gsize = ws_at<int32_t>(d_ws, L.gsize);
    int64_t* cs = ws_at<int64_t>(d_ws, L.cs);
    int32_t* ov_slot = ws_at<int32_t>(d_ws, L.ov_slot);
    int32_t* ov_lo = ws_at<int32_t>(d_ws, L.ov_lo);
    int32_t* kept = ws_at<int32_t>(d_ws, L.kept);
    int32_t* srows = ws_at<int32_t>(d_ws, L.srows);
    int32_t* smax = ws_at<int32_t>(d_ws, L.smax);
    int64_t* stok = ws_at<int64_t>(d_ws, L.stok);
    double* sadj = ws_at<double>(d_ws, L.sadj);
    int64_t* steps = ws_at<int64_t>(d_ws, L.steps);
    int32_t* bids[2] = {ws_at<int32_t>(d_ws, L.buf_ids0), ws_at<int32_t>(d_ws, L.buf_ids1)};
    int32_t* blen[2] = {ws_at<int32_t>(d_ws, L.buf_len0), ws_at<int32_t>(d_ws, L.buf_len1)};
    int32_t* wgidx = ws_at<int32_t>(d_ws, L.gidx);
    int32_t* dst = nonjoin ? ws_at<int32_t>(d_ws, L.stage) : d_emit_order;
    // the length each emitted row carries (from the stage-1 sorted lengths): the row
    // records' lengths, checked against the CSR offsets once the plan is built
    int32_t* row_len = d_row_len ? d_row_len : ws_at<int32_t>(d_ws, L.row_len);
    int32_t* dst_len = nonjoin ? ws_at<int32_t>(d_ws, L.stage_len) : row_len;
    const int64_t gcap = (int64_t)num_cus() * kPlanBlocksPerCU;
    const unsigned gridn = grid_for(n, kBlock, gcap);

    hipLaunchKernelGGL(round0_ranks_kernel, dim3(1), dim3(kBlock), 0, s, d_off, d_groups_per_rank, W, d_ranks,
                       d_gbase, st, d_rs, d_info);
    ODB_LAUNCHED();
    if (n > 0) {
        hipLaunchKernelGGL(round0_check_kernel, dim3(gridn), dim3(kBlock), 0, s, d_off, (const RankState*)d_ranks, W,
                           n, d_order, d_sorted_len, d_group_index, gstart, st);
        ODB_LAUNCHED();
    }

    std::vector<int64_t> cnt(W);
    for (int r = 0; r < W; ++r) cnt[r] = w->rank_offsets[r + 1] - w->rank_offsets[r];
    RoundBuffers cur{d_order, d_sorted_len, d_group_index};
    int flip = 0;
    int64_t S = 0;
    int32_t rounds = 0;
    int32_t stop = ODB_STOP_DRAINED;
    RoundState hrs{};
    HostState hstate;
    for (;;) {
        int nonempty = 0;
        int64_t max_cnt = 0;
        for (int r = 0; r < W; ++r) {
            nonempty += cnt[r] > 0;
            if (cnt[r] > max_cnt) max_cnt = cnt[r];
        }
        if (nonempty == 0) {
            stop = ODB_STOP_DRAINED;
            break;
        }
        // non-join: a rank that is empty while others are not advertises "finished"
        if (nonjoin && nonempty < W) {
            stop = ODB_STOP_RANK_FINISHED;
            break;
        }
        if (rounds > 0) {
            ODB_TRY(group_sequences(L, d_ws, W, n, budget, d_off, max_cnt, 0, false, cur.len, wgidx, nullptr, d_ranks,
                                    s));
            cur.gidx = wgidx;
        }
        rounds += 1;
        // real tokens prefix over the live positions
        ODB_TRY((device_excl_scan<int64_t>(LiveLen{cur.len, d_off, d_ranks, W, rounds > 1 ? 1 : 0},
                                           LiveLenIncl{LiveLen{cur.len, d_off, d_ranks, W, rounds > 1 ? 1 : 0}, cs},
                                           n, ws_at<int64_t>(d_ws, L.partials), s)));
        hipLaunchKernelGGL(group_sizes_kernel, dim3(gridn), dim3(kBlock), 0, s, (const int32_t*)gstart,
                           (const int64_t*)d_gbase, d_off, (const RankState*)d_ranks, W, gsize, steps, max_cnt,
                           (const DevStatus*)st);
        ODB_LAUNCHED();
        hipLaunchKernelGGL(adjust_kernel, dim3(W), dim3(kBlock), 0, s, d_ranks, d_cap, cap ? 1 : 0, W, d_rs,
                           (const int32_t*)gsize, ov_slot, kept, st);
        ODB_LAUNCHED();
        hipLaunchKernelGGL(slot_records_kernel, dim3(gridn), dim3(kBlock), 0, s, (const RankState*)d_ranks,
                           (const RoundState*)d_rs, d_off, W, (const int32_t*)gstart, (const int32_t*)gsize,
                           (const int32_t*)kept, cur.len, (const int64_t*)cs, srows, smax, stok, sadj, steps,
                           (const DevStatus*)st);
        ODB_LAUNCHED();
        hipLaunchKernelGGL(finalize_kernel, dim3(W), dim3(kBlock), 0, s, d_ranks, d_rs, (const int64_t*)steps,
                           nonjoin ? 1 : 0, params->quota, d_off,
                           (const int32_t*)gstart, (const int32_t*)gsize, (const int32_t*)ov_slot,
                           (const int32_t*)kept, ov_lo, (const DevStatus*)st);
        ODB_LAUNCHED();
        hipLaunchKernelGGL(emit_kernel, dim3(gridn), dim3(kBlock), 0, s, (const RankState*)d_ranks,
                           (const RoundState*)d_rs, d_off, W, n, cur.ids, cur.len, cur.gidx, (const int32_t*)gstart,
                           (const int32_t*)gsize, (const int32_t*)ov_slot, (const int32_t*)ov_lo, dst, dst_len,
                           bids[flip], blen[flip], (const DevStatus*)st);
        ODB_LAUNCHED();
        hipLaunchKernelGGL(advance_kernel, dim3(grid_for(W, kBlock)), dim3(kBlock), 0, s, d_ranks, W, d_rs);
        ODB_LAUNCHED();
        ODB_TRY(read_state(L, d_ws, W, &hstate, s));
        hrs = hstate.rs;
        const DevStatus& hst = hstate.st;
        const std::vector<RankState>& hranks = hstate.ranks;
        if (hst.err & (kErrOrder | kErrGroupIndex))
            return set_error(ODB_E_INVALID_DATA,
                             "stage-1 arrays do not describe this window (first inconsistent position %lld)",
                             (long long)hst.first_bad);
        if (hst.err & kErrInternal)
            return set_error(ODB_E_INTERNAL, "alignment round %d: group sizes inconsistent", rounds);
        // every round empties part of some buffer (T >= 1 steps of >= 1 sample for each
        // active rank) and never grows one; anything else is device state this call did
        // not write, and the loop stops rather than run on it
        int64_t left_before = 0, left_after = 0;
        for (int r = 0; r < W; ++r) {
            if (hranks[r].cnt < 0 || hranks[r].cnt > cnt[r])
                return set_error(ODB_E_INTERNAL, "alignment round %d: rank %d's buffer grew", rounds, r);
            left_before += cnt[r];
            left_after += hranks[r].cnt;
        }
        if (left_after == left_before && !(nonjoin && hrs.quota_hit))
            return set_error(ODB_E_INTERNAL, "alignment round %d emitted nothing", rounds);
        S += hrs.cut;
        for (int r = 0; r < W; ++r) cnt[r] = hranks[r].cnt;
        cur = RoundBuffers{bids[flip], blen[flip], nullptr};
        flip ^= 1;
        if (nonjoin && hrs.quota_hit) {
            stop = ODB_STOP_QUOTA;
            break;
        }
    }

    const int64_t K = (int64_t)W * S;
    h_info->steps = S;
    h_info->rounds = rounds;
    h_info->stop_reason = stop;
    h_info->splits = hrs.splits;
    h_info->overflow_groups = hrs.overflow;
    h_info->max_step_samples = hrs.step_max;
    h_info->second_gather_rounds = hrs.second_gather;
    h_info->required_slot_capacity = K;
    if (K > slot_capacity)
        return set_error(ODB_E_CAPACITY, "plan needs %lld slots, capacity is %lld", (long long)K,
                         (long long)slot_capacity);

    if (K > 0) {
        hipLaunchKernelGGL(plan_slots_kernel, dim3(grid_for(K, kBlock, gcap)), dim3(kBlock), 0, s,
                           (const RankState*)d_ranks, d_off, W, S, (const int32_t*)srows, (const int32_t*)smax,
                           (const int64_t*)stok, (const double*)sadj, d_slot_rows, d_slot_maxlen, d_slot_tokens,
                           d_slot_tokens_approx, d_info);
        ODB_LAUNCHED();
    }
    ODB_TRY((device_excl_scan<I64Pair>(RowsTilesLoad{d_slot_rows, d_slot_maxlen, K},
                                       RowsTilesStore{d_slot_row_off, d_slot_tile_off}, K + 1,
                                       ws_at<I64Pair>(d_ws, L.partials), s)));
    if (nonjoin && n > 0) {
        hipLaunchKernelGGL(compact_emit_kernel, dim3(gridn), dim3(kBlock), 0, s, (const int32_t*)dst,
                           (const int32_t*)dst_len, d_off, (const RankState*)d_ranks, W, n,
                           (const int64_t*)d_slot_row_off, S, d_emit_order, row_len);
        ODB_LAUNCHED();
    }
    const int64_t nemit = hrs.emitted_total;
    if (nemit > 0 && K > 0) {
        // rank-per-XCD gathers pay off when every XCD has a rank and a rank's offsets fit
        // in its L2 with room to spare
        int64_t max_nr = 0;
        for (int r = 0; r < W; ++r) max_nr = std::max(max_nr, w->rank_offsets[r + 1] - w->rank_offsets[r]);
        const int xcd = W >= kXcds && max_nr * 8 <= (int64_t)2 << 20;
        const unsigned grid = xcd ? (unsigned)(kXcds * std::max<int64_t>(1, std::min<int64_t>(
                                        (int64_t)num_cus() * 2 / kXcds, (max_nr + kBlock - 1) / kBlock)))
                                  : grid_for(nemit, kBlock, gcap);
        hipLaunchKernelGGL(row_check_kernel, dim3(grid), dim3(kBlock), 0, s, w->d_token_offsets,
                           (const int32_t*)d_emit_order, (const int32_t*)row_len, (const int64_t*)d_slot_row_off, S,
                           W, xcd, d_row_token_start, st);
        ODB_LAUNCHED();
    }
    hipLaunchKernelGGL(leftover_off_kernel, dim3(1), dim3(kBlock), 0, s, (const RankState*)d_ranks, W,
                       d_leftover_off);
    ODB_LAUNCHED();
    int64_t nleft = 0;
    for (int r = 0; r < W; ++r) nleft += cnt[r];
    if (nleft > 0) {
        hipLaunchKernelGGL(leftover_kernel, dim3(gridn), dim3(kBlock), 0, s, cur.ids, cur.len, w->d_token_offsets,
                           d_off, (const RankState*)d_ranks, W, n, (const int64_t*)d_leftover_off, d_leftover, st);
        ODB_LAUNCHED();
    }
    // stats (Sec. 2.1 / App. I padding fraction) and coverage (App. C)
    ODB_TRY(run_plan_coverage(w, L, d_ws, d_emit_order, d_slot_row_off, d_slot_tile_off, S, d_leftover,
                              d_leftover_off, nemit, nleft, s));

    ODB_TRY(read_state(L, d_ws, W, &hstate, s));
    const DevInfo& hi = hstate.info;
    const DevStatus& hs = hstate.st;
    h_info->emitted_samples = hi.emitted;
    h_info->leftover_samples = nleft;
    h_info->real_tokens = hi.real_tokens;
    h_info->padded_elems = hi.padded_elems;
    h_info->missing_ids = hi.missing_ids;
    h_info->duplicate_ids = hi.duplicate_ids;
    h_info->bad_views = hi.bad_views;
    h_info->pad_fraction = hi.pad_fraction;
    if (hs.err & kErrLength)
        return set_error(ODB_E_INVALID_DATA,
                         "sample %lld has a length outside [1, 2^31) or a negative token offset",
                         (long long)hs.first_bad_len);
    if (hs.err & kErrSortedLen)
        return set_error(ODB_E_INVALID_DATA,
                         "stage-1 arrays do not describe this window (sorted length of sample %lld is not its CSR "
                         "length)", (long long)hs.first_bad);
    if (hs.err & kErrIdentity)
        return set_error(ODB_E_INVALID_DATA, "identity map holds a value outside [0, num_identities)");
    if ((hs.err & kErrInternal) || hi.emitted != nemit)
        return set_error(ODB_E_INTERNAL, "internal inconsistency in the aligned plan");
    if (hi.bad_views != 0)
        return set_error(ODB_E_COVERAGE, "%lld sampler views are not emitted (or left over) exactly once",
                         (long long)hi.bad_views);
    return ODB_OK;
}

extern "C" int odb_check_coverage(const odb_window_t* w, const int32_t* d_emitted, int64_t num_emitted,
                                  const int32_t* d_leftover, int64_t num_leftover, odb_plan_info_t* h_info,
                                  void* d_ws, size_t ws_bytes, void* stream) {
    Layout L;
    ODB_TRY(check_workspace(w, d_ws, ws_bytes, &L));
    if (!h_info) return set_error(ODB_E_INVALID_ARG, "h_info is NULL");
    if (num_emitted < 0 || num_leftover < 0) return set_error(ODB_E_INVALID_ARG, "negative counts");
    if ((num_emitted > 0 && !d_emitted) || (num_leftover > 0 && !d_leftover))
        return set_error(ODB_E_INVALID_ARG, "id arrays must not be NULL");
    hipStream_t s = static_cast<hipStream_t>(stream);
    ODB_TRY(upload_small(w, L, d_ws, nullptr, s));
    hipLaunchKernelGGL(init_align_kernel, dim3(1), dim3(64), 0, s, ws_at<RoundState>(d_ws, L.round),
                       ws_at<DevInfo>(d_ws, L.info));
    ODB_LAUNCHED();
    ODB_TRY(run_coverage(w, L, d_ws, d_emitted, num_emitted, d_leftover, num_leftover, s));
    DevInfo hi;
    DevStatus hs;
    ODB_TRY_HIP(hipMemcpyAsync(&hi, ws_at<DevInfo>(d_ws, L.info), sizeof(hi), hipMemcpyDeviceToHost, s));
    ODB_TRY_HIP(hipMemcpyAsync(&hs, ws_at<DevStatus>(d_ws, L.status), sizeof(hs), hipMemcpyDeviceToHost, s));
    ODB_TRY_HIP(hipStreamSynchronize(s));
    ODB_TRY(finish_coverage(w, L, d_ws, d_emitted, num_emitted, d_leftover, num_leftover, &hi, s));
    h_info->bad_views = hi.bad_views;
    h_info->missing_ids = hi.missing_ids;
    h_info->duplicate_ids = hi.duplicate_ids;
    if (hs.err & (kErrIdentity | kErrInternal))
        return set_error(ODB_E_INVALID_DATA, "an id lies outside the window or its identity outside the map");
    return ODB_OK;
}
