// The unified streaming loop (Sec. 2.3 "Unified loop and termination"; App. C, App. E):
// one logical sampler iteration of W ranks, round by round, on the device.
//
// Per-rank state (App. C): sampler-pending views R_r (a cursor into the rank's view
// sequence), the collate buffer B_r (the worker queue is folded into it: a fetched view
// lands in the buffer in the same round) and the emitted views E_r (the rank's emit
// stream).  The shuffled identity list perm[0..N) is padded by repeating it from its
// head to M = W * ceil(N / W) views (view m has identity perm[m mod N]); view m belongs
// to rank m mod W, visited in increasing m.
//
// One protocol round k takes the form of one launch and the emit of the next: launch j
// (one block per rank) does, in order,
//   booking of round j-2  the round's step sizes, the non-join quota cut (Theorem 2) and
//                         termination.  Every block computes it the same way from what the
//                         previous launch wrote (so every block knows whether to go on) and
//                         block 0 stores it; no block waits for another
//   emit of round j-1     every block reads all ranks' published fetch records (the
//                         all_gather) and derives the same round kind and target T (Eq. 3
//                         over the ready ranks); the rank commits its fetch, and in an emit
//                         round applies Algorithm 1 (split in closed form, overflow by size
//                         rank) and writes its T slot records, its emitted views and its new
//                         buffer (the overflow); finished ranks (join) write IDLE slots
//   form of round j       fetch up to rate[r] views under the depth envelope |B_r| <= D;
//                         status (finished / not ready / ready); a ready rank sorts its whole
//                         buffer by (length desc, view asc) and chases the group starts of
//                         Sec. 2.2 (threshold carry, Eq. 1).  The form is kept apart (by
//                         round parity) from the rank's committed state until the next
//                         launch's emit phase commits it, so a form made after the round
//                         that ends the iteration changes nothing
// A grid-wide barrier between the phases would need a device-scope fence in every block,
// an L2 write-back on this GPU, which beside a running collate waits behind its write
// stream; the launch boundary is the barrier instead.  Rounds are enqueued in chunks sized
// by a lower bound on the rounds left, each chunk closed by a one-block launch that books
// its last round; the host reads the done flag once per chunk, and launches enqueued after
// the stop return at once.  A final pass turns the per-rank staging into the window plan
// layout (rank-major slots, row and tile offsets), so odb_collate and odb_loss_weights
// apply unchanged, and counts coverage.
#include <algorithm>
#include <climits>
#include <cmath>
#include <cstring>
#include <vector>

#include "odb_internal.h"

namespace odb {

namespace {

constexpr int kST = 512;              // threads of a round block (one block per rank)
constexpr int kMaxDepth = 4096;       // largest outstanding-depth envelope
constexpr int64_t kMinChunk = 8;      // fewest rounds enqueued after an estimate fell short
constexpr int64_t kViewBitsLds = 64 * 1024;   // a rank's emitted-view bits in LDS up to this size

struct StreamGlobal {
    int64_t steps;       // aligned steps so far (after quota cuts)
    int64_t emitted;     // emitted views so far (after quota cuts)
    int64_t rounds;
    int64_t emit_rounds;
    int64_t skip_rounds;
    int64_t splits;
    int64_t overflow;
    int64_t second_gather;
    int64_t max_step;
    unsigned long long max_outstanding;
    int32_t done;
    int32_t stop;
    int32_t err;
};

// A rank's committed state, written by the emit phase of every round that runs.
struct RankStream {
    int64_t cursor;    // sampler position of the next fetch
    int64_t buf_n;     // |B_r|
    int64_t emitted;   // views written to the rank's emit stream (before a final quota cut)
    int64_t pad;
};

// A rank's fetch and grouping for one round (kept by round parity until committed).
struct RankForm {
    int64_t cursor;    // sampler position after the fetch
    int64_t n;         // |B_r| after the fetch, as published for the round's all_gather
    int64_t tok;       // tokens in the buffer (ready ranks)
    int32_t status;    // -1 finished, 0 not ready, G_r > 0 ready with G_r groups
    int32_t err;       // data errors met by the fetch (raised when it is committed)
};

struct StreamRec {
    int32_t kind;          // 0 emit, 1 skip, 2 stop
    int32_t changed;       // an emit round in which some ready rank had G_r != T
    int32_t booked;        // booked by the launch that closes a chunk
    int32_t pad;
    int64_t target;        // T (emit rounds)
    int64_t emitted;       // views emitted in the round (after a quota cut)
    int64_t cut;           // steps kept (emit rounds); stop reason (stop rounds)
    int64_t cum_steps;     // steps after the round
    int64_t cum_emitted;   // views emitted after the round
};

enum : int32_t { kSErrIdentity = 1, kSErrLength = 2, kSErrInternal = 4, kSErrRounds = 8 };

struct StreamArgs {
    int W;
    int mode;
    int64_t N;
    int64_t q;          // views per rank
    int64_t D;          // depth envelope
    int64_t bufsize;
    int64_t budget;
    int64_t quota;
    int64_t scap;       // staging slots per rank
    int64_t max_rounds;
    const int64_t* tok_off;
    const int32_t* perm;
    const int32_t* rate;   // [W]
    const int64_t* cap;    // [W] or null
    // every view's identity, token start and length code, rank-major (x = r * q + i is
    // view i * W + r); the code is the length, 0 for an identity outside [0, N), -1 for a
    // length outside [1, 2^31)
    const int32_t* vid;
    const int64_t* vts;
    const int32_t* vlen;
    StreamGlobal* g;
    RankStream* ranks;     // [W]
    RankForm* form;        // [2 * W], round parity major
    StreamRec* rec;
    int64_t* stepsum;      // [3 * D], round mod 3 major
    int32_t* bufv;         // [W * D]
    unsigned long long* skey;   // [W * D] sorted keys (length desc, view asc) of ready ranks
    int32_t* gs;           // [W * (D + 1)] group starts
    int32_t* srows;        // [W * scap]
    int32_t* smax;
    int64_t* stok;
    double* sadj;
    int32_t* evw;          // [W * q] emit streams
};

// Sort keys of the form phase: the buffer is padded to P = KPT * kST keys, P >= D.
inline int sort_kpt(int64_t D) {
    int64_t p = kST;
    while (p < D) p <<= 1;
    return (int)(p / kST);
}

// Dynamic LDS of a round launch: the emit tables for depth D (gtok 8 B, gsl, as, ae, cum
// 4 B per group; sorted keys 8 B and adjusted groups 4 B per position) and the form's
// radix counters (4 B per digit, slot and wave), keys (8 B), sorted lengths and
// next-start links (4 B per position) share it.
inline size_t round_lds_bytes(int64_t D) {
    const size_t emit = (size_t)(8 * D + 4 * (4 * D + 2) + 12 * D);
    const int kpt = sort_kpt(D);
    const size_t form = (size_t)(4 * (kpt <= 2 ? 32 : 16) * (kST / kWave) + 16 * kST) * kpt;
    return emit > form ? emit : form;
}

__device__ __forceinline__ int32_t view_identity(const StreamArgs& a, int64_t m) {
    return a.perm[m < a.N ? m : m % a.N];
}

// Block reductions and scans over an NT-thread block: DPP scans inside each wave, one
// LDS slot per wave across waves.  Every thread of the block must take part.
template <int NT, typename Op, typename T>
__device__ __forceinline__ T sblock_reduce(T v) {
    __shared__ T wt[NT / kWave];
    const T w = wave_last(wave_scan_dpp<Op>(v));
    if ((threadIdx.x & (kWave - 1)) == 0) wt[threadIdx.x / kWave] = w;
    __syncthreads();
    T t = wt[0];
    for (int i = 1; i < NT / kWave; ++i) t = Op::apply(t, wt[i]);
    __syncthreads();
    return t;
}

template <int NT, typename T>
__device__ __forceinline__ T sblock_sum(T v) {
    return sblock_reduce<NT, OpAdd>(v);
}

// Maximum of one non-negative value per thread.
template <int NT>
__device__ __forceinline__ int64_t sblock_max(int64_t v) {
    return sblock_reduce<NT, OpMax>(v);
}

// Exclusive scan of one value per thread over an NT-thread block; *total = sum.
template <int NT, typename T>
__device__ __forceinline__ T sblock_excl(T v, T* total) {
    __shared__ T wt[NT / kWave];
    const T inc = wave_scan_dpp<OpAdd>(v);
    const int w = threadIdx.x / kWave;
    if ((threadIdx.x & (kWave - 1)) == kWave - 1) wt[w] = inc;
    __syncthreads();
    T pre = 0, tot = 0;
    for (int i = 0; i < NT / kWave; ++i) {
        pre += i < w ? wt[i] : T(0);
        tot += wt[i];
    }
    __syncthreads();
    *total = tot;
    return pre + inc - v;
}

// The staged view table: every view's identity (perm), token start and length code (CSR
// offsets), gathered once per iteration so that a round's fetch reads its views' codes
// in order and the final pass reads identities and row records near each other.
__global__ void __launch_bounds__(256) stream_views_kernel(StreamArgs a, int32_t* vid, int64_t* vts, int32_t* vlen) {
    const int64_t M = a.q * a.W;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; x < M; x += stride) {
        const int64_t r = x / a.q, i = x - r * a.q;
        const int32_t id = view_identity(a, i * a.W + r);
        int32_t code = 0;
        int64_t t0 = 0;
        if (id >= 0 && id < a.N) {
            t0 = a.tok_off[id];
            const int64_t l = a.tok_off[id + 1] - t0;
            code = (l < 1 || l > 0x7FFFFFFF) ? -1 : (int32_t)l;
        }
        vid[x] = id;
        vts[x] = t0;
        vlen[x] = code;
    }
}

__global__ void stream_init_kernel(StreamArgs a, int64_t rounds_cap) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    const int64_t i0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i0 == 0) *a.g = StreamGlobal{};
    for (int64_t i = i0; i < a.W; i += stride) a.ranks[i] = RankStream{};
    for (int64_t i = i0; i < 2 * a.W; i += stride) a.form[i] = RankForm{};
    for (int64_t i = i0; i < rounds_cap; i += stride) a.rec[i] = StreamRec{};
    for (int64_t i = i0; i < 3 * a.D; i += stride) a.stepsum[i] = 0;
}

// ------------------------------------------------------------------ round: bookkeeping
struct Booked {
    bool done;        // the iteration ends with this round
    int64_t steps;    // aligned steps after the round
};

// Round k's bookkeeping from its record rk and the previous round's rp, both written by
// earlier launches: every block of a launch reaches the same result; `writer` stores it.
__device__ Booked book_round(const StreamArgs& a, int64_t k, const StreamRec& rk, const StreamRec& rp, bool writer) {
    if (rk.booked) return Booked{false, rk.cum_steps};   // done was seen at launch start
    StreamGlobal* g = a.g;
    StreamRec* rec = a.rec + k;
    const int64_t prev_steps = k > 0 ? rp.cum_steps : 0;
    const int64_t prev_emitted = k > 0 ? rp.cum_emitted : 0;
    const bool last = k + 1 >= a.max_rounds;
    if (rk.kind == 2) {
        if (writer && threadIdx.x == 0) {
            g->stop = (int32_t)rk.cut;
            g->done = 1;
            g->rounds = k + 1;
        }
        return Booked{true, prev_steps};
    }
    if (rk.kind == 1) {
        if (writer && threadIdx.x == 0) {
            rec->cum_steps = prev_steps;
            rec->cum_emitted = prev_emitted;
            g->skip_rounds += 1;
            g->rounds = k + 1;
            if (last) {
                atomicOr(&g->err, kSErrRounds);
                g->done = 1;
            }
        }
        return Booked{last, prev_steps};
    }
    // emit round: cumulative step sizes, the quota cut (non-join), per-round totals
    const int64_t T = rk.target;
    const bool nonjoin = a.mode == ODB_MODE_NONJOIN_QUOTA;
    if (!writer && !nonjoin) return Booked{last, prev_steps + T};
    const int64_t* ss = a.stepsum + (k % 3) * a.D;
    __shared__ int64_t s_cut;
    if (threadIdx.x == 0) s_cut = T;
    __syncthreads();
    if (nonjoin) {
        // every step holds at least one row, so the running total crosses Q at most once
        int64_t carry = 0;
        for (int64_t b = 0; b < T; b += kST) {
            const int64_t j = b + threadIdx.x;
            const int64_t v = j < T ? ss[j] : 0;
            int64_t tot;
            const int64_t ex = sblock_excl<kST>(v, &tot);
            if (j < T && prev_emitted + carry + ex < a.quota && prev_emitted + carry + ex + v >= a.quota)
                s_cut = j + 1;
            carry += tot;
        }
        __syncthreads();
    }
    const int64_t cut = s_cut;
    int64_t kept = 0, mx = 0;
    for (int64_t j = threadIdx.x; j < cut; j += kST) {
        const int64_t v = ss[j];
        kept += v;
        mx = v > mx ? v : mx;
    }
    kept = sblock_sum<kST>(kept);
    mx = sblock_max<kST>(mx);
    const bool done = cut < T || (nonjoin && prev_emitted + kept >= a.quota) || last;
    if (writer && threadIdx.x == 0) {
        rec->emitted = kept;
        rec->cut = cut;
        rec->cum_steps = prev_steps + cut;
        rec->cum_emitted = prev_emitted + kept;
        g->steps = prev_steps + cut;
        g->emitted = prev_emitted + kept;
        g->max_step = mx > g->max_step ? mx : g->max_step;
        g->emit_rounds += 1;
        g->second_gather += rk.changed ? 1 : 0;
        g->rounds = k + 1;
        if (cut < T || (nonjoin && prev_emitted + kept >= a.quota)) {
            g->stop = ODB_STOP_QUOTA;
            g->done = 1;
        } else if (last) {
            atomicOr(&g->err, kSErrRounds);
            g->done = 1;
        }
    }
    return Booked{done, prev_steps + cut};
}

// ------------------------------------------------------------------ round: align + emit
struct RoundView {
    int kind;
    int64_t T;
    int32_t stop;
};

// The all_gather: every block reduces the same W published fetch records of round k the
// same way; ft / cap_t are the record and capacity of rank threadIdx.x, loaded early.
// Each thread tallies its ranks in registers; the waves combine by DPP scans and one LDS
// slot per wave (minima as maxima of LLONG_MAX - v, so that 0 means none).
__device__ RoundView decide_round(const StreamArgs& a, int64_t k, const RankForm& ft, int64_t cap_t) {
    const RankForm* F = a.form + (k & 1) * a.W;
    int64_t cnt = 0, mg = 0, xs = 0, xc = 0;   // cnt: finished << 32 | not ready
    auto tally = [&](const RankForm& x, int64_t c) {
        if (x.status < 0) {
            cnt += 1ll << 32;
        } else if (x.status == 0) {
            cnt += 1;
        } else {
            mg = x.status > mg ? x.status : mg;
            xs = LLONG_MAX - x.n > xs ? LLONG_MAX - x.n : xs;
            if (c > 0) xc = LLONG_MAX - c > xc ? LLONG_MAX - c : xc;
        }
    };
    if ((int)threadIdx.x < a.W) tally(ft, cap_t);
    for (int r = threadIdx.x + kST; r < a.W; r += kST) tally(F[r], a.cap ? a.cap[r] : 0);
    cnt = wave_last(wave_scan_dpp<OpAdd>(cnt));
    mg = wave_last(wave_scan_dpp<OpMax>(mg));
    xs = wave_last(wave_scan_dpp<OpMax>(xs));
    xc = wave_last(wave_scan_dpp<OpMax>(xc));
    __shared__ int64_t part[4][kST / kWave];
    const int w = threadIdx.x / kWave;
    if ((threadIdx.x & (kWave - 1)) == 0) {
        part[0][w] = cnt;
        part[1][w] = mg;
        part[2][w] = xs;
        part[3][w] = xc;
    }
    __syncthreads();
    cnt = 0;
    mg = xs = xc = 0;
    for (int i = 0; i < kST / kWave; ++i) {
        cnt += part[0][i];
        mg = part[1][i] > mg ? part[1][i] : mg;
        xs = part[2][i] > xs ? part[2][i] : xs;
        xc = part[3][i] > xc ? part[3][i] : xc;
    }
    const int64_t fin = cnt >> 32, unready = cnt & 0xFFFFFFFFll;
    const int64_t minS = LLONG_MAX - xs, minC = LLONG_MAX - xc;
    RoundView v{0, 0, 0};
    if (fin == a.W) {
        v.kind = 2;
        v.stop = ODB_STOP_DRAINED;
    } else if (a.mode == ODB_MODE_NONJOIN_QUOTA && fin > 0) {
        v.kind = 2;
        v.stop = ODB_STOP_RANK_FINISHED;
    } else if (unready > 0) {
        v.kind = 1;
    } else {
        int64_t T = mg;
        if (minC < T) T = minC;
        if (minS < T) T = minS;
        v.T = T < 1 ? 1 : T;
    }
    return v;
}

// LDS of the emit phase for depth D: gtok (8 B per group), gsl, as, ae, cum (4 B per
// group), then the rank's sorted keys kl (8 B per position) and adjusted groups apos
// (4 B per position).
struct EmitLds {
    unsigned long long* gtok;
    int32_t *gsl, *as, *ae, *cum;
    unsigned long long* kl;
    int32_t* apos;
};

__device__ __forceinline__ EmitLds emit_lds(unsigned char* lds, int64_t D) {
    EmitLds e;
    e.gtok = reinterpret_cast<unsigned long long*>(lds);
    e.gsl = reinterpret_cast<int32_t*>(e.gtok + D);
    e.as = e.gsl + (D + 1);
    e.ae = e.as + D;
    e.cum = e.ae + D;
    e.kl = reinterpret_cast<unsigned long long*>(e.cum + (D + 1));   // 24 D + 8 bytes in
    e.apos = reinterpret_cast<int32_t*>(e.kl + D);
    return e;
}

__device__ __forceinline__ int32_t key_view(unsigned long long key) { return (int32_t)(key & 0xFFFFFFFFull); }
__device__ __forceinline__ int32_t key_len(unsigned long long key) {
    return (int32_t)(0x7FFFFFFFll - (int64_t)(key >> 32));
}
__device__ __forceinline__ unsigned long long make_key(int64_t l, int64_t m) {
    return ((unsigned long long)(0x7FFFFFFFll - l) << 32) | (unsigned long long)(uint32_t)m;
}

// Algorithm 1 and the emission of round k for ready rank r = blockIdx.x, whose G group
// starts and n sorted keys are in LDS: T slot records at steps base.., the emitted views
// and the returns (overflow), compacted in sorted order into kl[0..) and the rank's
// buffer.  Returns the number of returns.
__device__ int64_t emit_rank(const StreamArgs& a, int64_t k, int64_t base, const EmitLds& L, int64_t T, int64_t G,
                             int64_t n, int64_t tok, int64_t ebase) {
    const int r = blockIdx.x;
    int32_t *gsl = L.gsl, *as = L.as, *ae = L.ae, *cum = L.cum, *apos = L.apos;
    unsigned long long *gtok = L.gtok, *kl = L.kl;
    __shared__ int64_t s_X, s_jstar;
    __shared__ int32_t s_bad;
    for (int64_t i = threadIdx.x; i < T; i += kST) gtok[i] = 0;
    if (threadIdx.x == 0) {
        s_bad = 0;
        s_X = 0;
        s_jstar = 0;
    }
    __syncthreads();
    // the adjusted groups [as[t], ae[t]) in formation order
    if (G < T) {
        // split, closed form: positions [0, X) become singletons, [X, end of group j*)
        // stays one group, later groups are unchanged; j* is the first group whose
        // cumulative surplus sum (c_g - 1) reaches k = T - G
        if (threadIdx.x == 0) s_jstar = -1;
        __syncthreads();
        const int64_t need = T - G;
        int64_t carry = 0;
        for (int64_t b = 0; b < G; b += kST) {
            const int64_t g = b + threadIdx.x;
            const int64_t v = g < G ? (int64_t)(gsl[g + 1] - gsl[g]) - 1 : 0;
            int64_t tot;
            const int64_t ex = carry + sblock_excl<kST>(v, &tot);
            if (g < G && ex < need && ex + v >= need) {   // surpluses are >= 0: one crossing
                s_jstar = g;
                s_X = gsl[g] + (need - ex);
            }
            carry += tot;
        }
        __syncthreads();
        const int64_t X = s_X, js = s_jstar < 0 ? 0 : s_jstar;
        if (threadIdx.x == 0 && (s_jstar < 0 || X + 1 + (G - 1 - s_jstar) != T)) s_bad = 1;
        for (int64_t t = threadIdx.x; t < T; t += kST) {
            if (t < X) {
                as[t] = (int32_t)t;
                ae[t] = (int32_t)(t + 1);
            } else if (t == X) {
                as[t] = (int32_t)X;
                ae[t] = gsl[js + 1];
            } else {
                const int64_t g = js + (t - X);
                as[t] = g < G ? gsl[g] : (int32_t)n;
                ae[t] = g < G ? gsl[g + 1] : (int32_t)n;
            }
        }
        __syncthreads();
        for (int64_t p = threadIdx.x; p < n; p += kST) {
            int64_t ap;
            if (p < X) {
                ap = p;
            } else if (p < gsl[js + 1]) {
                ap = X;
            } else {
                // formation group of p (> j*): binary search over the group starts
                int64_t lo = js + 1, hi = G;
                while (hi - lo > 1) {
                    const int64_t mid = (lo + hi) >> 1;
                    if (gsl[mid] <= p) lo = mid; else hi = mid;
                }
                ap = X + (lo - js);
            }
            apos[p] = (int32_t)ap;
        }
    } else if (G > T) {
        // overflow: keep the T groups first by (size desc, formation index desc)
        for (int64_t g = threadIdx.x; g < G; g += kST) {
            const int32_t cg = gsl[g + 1] - gsl[g];
            int64_t rank = 0;
            for (int64_t h = 0; h < G; ++h) {
                const int32_t ch = gsl[h + 1] - gsl[h];
                rank += (ch > cg || (ch == cg && h > g)) ? 1 : 0;
            }
            cum[g] = rank < T ? 1 : 0;   // kept flag, turned into the kept index below
        }
        __syncthreads();
        int64_t carry = 0;
        for (int64_t b = 0; b < G; b += kST) {
            const int64_t g = b + threadIdx.x;
            const int32_t f = g < G ? cum[g] : 0;
            int32_t tot;
            const int32_t ex = sblock_excl<kST>(f, &tot);
            if (g < G && f) {
                const int64_t ki = carry + ex;
                as[ki] = gsl[g];
                ae[ki] = gsl[g + 1];
            }
            carry += tot;
        }
        __syncthreads();
        if (threadIdx.x == 0 && carry != T) s_bad = 1;
        for (int64_t p = threadIdx.x; p < n; p += kST) apos[p] = -1;
        __syncthreads();
        for (int64_t t = threadIdx.x; t < T; t += kST)
            for (int64_t p = as[t]; p < ae[t]; ++p) apos[p] = (int32_t)t;
    } else {
        for (int64_t t = threadIdx.x; t < T; t += kST) {
            as[t] = gsl[t];
            ae[t] = gsl[t + 1];
        }
        __syncthreads();
        for (int64_t t = threadIdx.x; t < T; t += kST)
            for (int64_t p = as[t]; p < ae[t]; ++p) apos[p] = (int32_t)t;
    }
    __syncthreads();
    // rows prefix over the adjusted groups, tokens per adjusted group.  Without overflow
    // the adjusted groups tile positions 0..n in order, so the prefix is the group start
    if (G <= T) {
        for (int64_t t = threadIdx.x; t < T; t += kST) cum[t] = as[t];
        if (threadIdx.x == 0) cum[T] = (int32_t)n;
    } else {
        int64_t carry = 0;
        for (int64_t b = 0; b < T; b += kST) {
            const int64_t t = b + threadIdx.x;
            const int32_t rows = t < T ? ae[t] - as[t] : 0;
            int32_t tot;
            const int32_t ex = sblock_excl<kST>(rows, &tot);
            if (t < T) cum[t] = (int32_t)(carry + ex);
            carry += tot;
        }
        if (threadIdx.x == 0) cum[T] = (int32_t)carry;
    }
    // tokens per adjusted group: a group's positions are contiguous, so each wave sums its
    // piece of a group with a DPP scan and adds it with one atomic (a per-position atomic
    // would queue up to a wave of lanes on one LDS address)
    for (int64_t b = 0; b < n; b += kST) {
        const int64_t p = b + threadIdx.x;
        const int lane = threadIdx.x & (kWave - 1);
        const int32_t t = p < n ? apos[p] : -1;
        const int64_t l = t >= 0 ? key_len(kl[p]) : 0;
        const int64_t inc = wave_scan_dpp<OpAdd>(l);
        const int32_t t_prev = __shfl_up(t, 1, kWave), t_next = __shfl_down(t, 1, kWave);
        const int head = wave_scan_dpp<OpMax>((lane == 0 || t_prev != t) ? lane : 0);
        const int64_t before = __shfl(inc, head > 0 ? head - 1 : 0, kWave);
        if (t >= 0 && (lane == kWave - 1 || t_next != t))
            atomicAdd(&gtok[t], (unsigned long long)(inc - (head > 0 ? before : 0)));
    }
    __syncthreads();
    const int64_t E = cum[T];
    const double mean = (double)tok / (double)n;
    int64_t* stepsum = a.stepsum + (k % 3) * a.D;
    // slot records: step j of the round is adjusted group T-1-j (short to long).  Steps at
    // or past the capacity are not staged: when the iteration's final step count S fits
    // the capacity they all lie past S (a non-join quota cut can drop the round's last
    // steps), and otherwise the call reports ODB_E_CAPACITY from S
    for (int64_t t = threadIdx.x; t < T; t += kST) {
        const int64_t j = T - 1 - t;
        const int64_t x = base + j;
        const int32_t rows = ae[t] - as[t];
        if (x < a.scap) {
            const int64_t o = (int64_t)r * a.scap + x;
            a.srows[o] = rows;
            a.smax[o] = rows > 0 ? key_len(kl[as[t]]) : 0;
            a.stok[o] = (int64_t)gtok[t];
            a.sadj[o] = (double)rows * mean;
        }
        atomicAdd((unsigned long long*)&stepsum[j], (unsigned long long)rows);
    }
    // emitted views (rows of a group run from its last position to its first); returns
    // are compacted in place, in sorted order, into kl[0..) and the buffer: a position
    // never moves up and every read of a chunk precedes the scan's barriers, so no key
    // is overwritten before it is read
    int32_t* ev = a.evw + (int64_t)r * a.q;
    int32_t* buf = a.bufv + (int64_t)r * a.D;
    int64_t nret = 0;
    if (G <= T) {   // every position is emitted
        for (int64_t p = threadIdx.x; p < n; p += kST) {
            const int32_t t = apos[p];
            const int64_t e = ebase + E - cum[t + 1] + (ae[t] - 1 - p);
            if (e < a.q) ev[e] = key_view(kl[p]); else s_bad = 1;
        }
    } else for (int64_t b = 0; b < n; b += kST) {
        const int64_t p = b + threadIdx.x;
        const unsigned long long key = p < n ? kl[p] : 0ull;
        const int32_t t = p < n ? apos[p] : 0;
        if (p < n && t >= 0) {
            const int64_t e = ebase + E - cum[t + 1] + (ae[t] - 1 - p);
            if (e < a.q) ev[e] = key_view(key); else s_bad = 1;
        }
        const int32_t ret = (p < n && t < 0) ? 1 : 0;
        int32_t tot;
        const int32_t ex = sblock_excl<kST>(ret, &tot);
        if (ret) {
            kl[nret + ex] = key;
            buf[nret + ex] = key_view(key);
        }
        nret += tot;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        a.ranks[r].emitted = ebase + E;
        a.ranks[r].buf_n = nret;
        if (E + nret != n) s_bad = 1;
        if (G < T) atomicAdd((unsigned long long*)&a.g->splits, (unsigned long long)(T - G));
        if (G > T) atomicAdd((unsigned long long*)&a.g->overflow, (unsigned long long)(G - T));
        if (G != T) atomicOr(&a.rec[k].changed, 1);
        if (s_bad) atomicOr(&a.g->err, kSErrInternal);
    }
    return nret;
}

// ------------------------------------------------------------------ round: fetch + form
// Key of view m from its staged length code; flags bad data.
__device__ __forceinline__ unsigned long long staged_key(int32_t code, int64_t m, int32_t* err) {
    int64_t l = code;
    if (code <= 0) {
        *err |= code == 0 ? kSErrIdentity : kSErrLength;
        l = 1;
    }
    return make_key(l, m);
}

// Launch j: books round j-2, emits round j-1, forms round j (see the top of this file).
// Global loads are issued in two batches ahead of the work that needs them (the
// control state, then the rank's group starts, sorted keys and the next fetch's length
// codes), so that a round costs few memory round trips beside a running collate.
template <int KPT>
__global__ void __launch_bounds__(kST) stream_round_kernel(StreamArgs a, int64_t j) {
    constexpr int P = KPT * kST;
    extern __shared__ unsigned long long s_dyn[];
    unsigned char* lds = reinterpret_cast<unsigned char*>(s_dyn);
    const int r = blockIdx.x;
    const int tid = threadIdx.x;
    // ---- first batch: control state and the fetch records published for round j-1
    const int32_t done = a.g->done;   // written by an earlier launch
    const int64_t kb = j >= 2 ? j - 2 : 0;
    const StreamRec rk = a.rec[kb];
    const StreamRec rp = a.rec[kb > 0 ? kb - 1 : 0];
    const RankForm* Fe = a.form + ((j + 1) & 1) * a.W;   // round j-1
    RankForm ft{}, fr{};
    int64_t cap_t = 0;
    if (j >= 1) {
        if (tid < a.W) {
            ft = Fe[tid];
            cap_t = a.cap ? a.cap[tid] : 0;
        }
        fr = Fe[r];
    }
    const int64_t ebase = a.ranks[r].emitted;
    const int64_t rate = a.rate[r];
    if (done) return;
    // the first batch is complete here (one wait), so the second one below is not drained
    // by a later first use of this batch
    asm volatile("" ::"v"(ft.status), "v"(ft.n), "v"(cap_t));
    // ---- second batch, before the booking and the round decision are known: this rank's
    // group starts and sorted keys (used if round j-1 emits) and the length codes of the
    // views round j can fetch
    const bool may_emit = j >= 1 && fr.status > 0;
    const int64_t G = may_emit ? fr.status : 0;
    const int64_t n = may_emit ? fr.n : 0;
    const int32_t* gsg = a.gs + (int64_t)r * (a.D + 1);
    const unsigned long long* skey = a.skey + (int64_t)r * a.D;
    int32_t gv[KPT + 1];
    unsigned long long kv[KPT];
#pragma unroll
    for (int c = 0; c <= KPT; ++c) {
        const int64_t i = tid + c * kST;
        gv[c] = i <= G ? gsg[i] : 0;
    }
#pragma unroll
    for (int c = 0; c < KPT; ++c) {
        const int64_t i = tid + c * kST;
        kv[c] = i < n ? skey[i] : 0ull;
    }
    const int64_t cursor = j >= 1 ? fr.cursor : 0;   // committed by the emit phase below
    int64_t fmax = a.q - cursor;
    fmax = fmax < rate ? fmax : rate;
    fmax = fmax < a.D ? fmax : a.D;
    const int32_t* vlen_r = a.vlen + (int64_t)r * a.q;
    int32_t code[KPT];
#pragma unroll
    for (int c = 0; c < KPT; ++c) {
        const int64_t i = tid + c * kST;
        code[c] = i < fmax ? vlen_r[cursor + i] : 1;
    }
    int64_t base = 0;
    if (j >= 2) {
        const Booked b = book_round(a, j - 2, rk, rp, r == 0);
        if (b.done) return;
        base = b.steps;
    }
    // the step sums of round j, added up by the next launch: last read when round j-3
    // was booked
    if (r == 0) {
        int64_t* ss = a.stepsum + (j % 3) * a.D;
        for (int64_t i = tid; i < a.D; i += kST) ss[i] = 0;
    }
    const EmitLds L = emit_lds(lds, a.D);
    __shared__ int32_t s_err;
    if (tid == 0) s_err = 0;
    __syncthreads();
    // ---- emit phase of round j-1: the all_gather, the commit of the rank's fetch, and
    // in an emit round the rank's groups
    int64_t n0 = 0;          // the rank's buffer after round j-1
    bool in_lds = false;     // its keys are in L.kl[0..n0)
    if (j >= 1) {
        const RoundView v = decide_round(a, j - 1, ft, cap_t);
        if (r == 0 && tid == 0) {
            a.rec[j - 1].kind = v.kind;
            a.rec[j - 1].target = v.T;
            a.rec[j - 1].cut = v.kind == 2 ? v.stop : 0;
        }
        if (tid == 0) {
            a.ranks[r].cursor = fr.cursor;
            a.ranks[r].buf_n = fr.n;
            atomicMax(&a.g->max_outstanding, (unsigned long long)fr.n);
            if (fr.err) atomicOr(&a.g->err, fr.err);
        }
        if (v.kind == 2) return;   // a stop round: the next launch's booking ends the iteration
        n0 = fr.n;
        if (v.kind == 0 && fr.status < 0) {   // finished rank in join mode: IDLE slots
            for (int64_t t = tid; t < v.T; t += kST) {
                const int64_t x = base + t;
                if (x < a.scap) {   // steps past the capacity are not staged (see the slot records)
                    const int64_t o = (int64_t)r * a.scap + x;
                    a.srows[o] = 0;
                    a.smax[o] = 0;
                    a.stok[o] = 0;
                    a.sadj[o] = 0.0;
                }
            }
        } else if (v.kind == 0) {
#pragma unroll
            for (int c = 0; c <= KPT; ++c) {
                const int64_t i = tid + c * kST;
                if (i <= G) L.gsl[i] = gv[c];
            }
#pragma unroll
            for (int c = 0; c < KPT; ++c) {
                const int64_t i = tid + c * kST;
                if (i < n) L.kl[i] = kv[c];
            }
            n0 = emit_rank(a, j - 1, base, L, v.T, G, n, fr.tok, ebase);
            in_lds = true;
        }
    }
    // ---- form phase of round j: fetch, status, and for a ready rank sort and group starts
    int32_t* buf = a.bufv + (int64_t)r * a.D;
    int64_t f = a.D - n0;
    f = f < fmax ? f : fmax;
    f = f > 0 ? f : 0;
    const int64_t nn = n0 + f;
    const bool drained = cursor + f == a.q;
    const bool finished = drained && nn == 0;
    const bool ready = !finished && (nn >= a.bufsize || drained);
    RankForm* F = a.form + (j & 1) * a.W + r;
    // the fetched views join the buffer (a ready rank keeps them there when another rank
    // is not ready and the round is a skip round)
    int32_t err = 0;
    unsigned long long fk[KPT];
#pragma unroll
    for (int c = 0; c < KPT; ++c) {
        const int64_t i = tid + c * kST;
        fk[c] = 0;
        if (i < f) {
            const int64_t m = (cursor + i) * a.W + r;
            buf[n0 + i] = (int32_t)m;
            if (ready) fk[c] = staged_key(code[c], m, &err);
        }
    }
    if (!ready) {
        if (tid == 0) *F = RankForm{cursor + f, nn, 0, finished ? -1 : 0, 0};
        return;
    }
    // keys of the whole buffer into kl[0..nn): the returns are there already when the
    // rank emitted in this launch, otherwise they are read back
    if (!in_lds) {
        for (int64_t i = tid; i < n0; i += kST) {
            const int64_t m = buf[i];
            L.kl[i] = staged_key(vlen_r[m / a.W], m, &err);
        }
    }
#pragma unroll
    for (int c = 0; c < KPT; ++c) {
        const int64_t i = tid + c * kST;
        if (i < f) L.kl[n0 + i] = fk[c];
    }
    if (err) atomicOr(&s_err, err);
    __syncthreads();
    unsigned long long x[KPT];
    int64_t tok = 0, mylen = 0;
#pragma unroll
    for (int c = 0; c < KPT; ++c) {
        const int64_t i = tid + c * kST;
        x[c] = i < nn ? L.kl[i] : ~0ull;
        const int64_t l = i < nn ? key_len(x[c]) : 0;
        tok += l;
        mylen = l > mylen ? l : mylen;
    }
    tok = sblock_sum<kST>(tok);
    const int64_t maxlen = sblock_max<kST>(mylen);
    // sort to (length desc, view asc).  The buffer is already in view order within each
    // length: the returns come first, sorted, and every fetched view follows all views
    // fetched before it.  So a stable LSD radix sort on the length alone, digits taken
    // descending, gives that order (5-bit digits up to two keys per thread, 4-bit
    // beyond, so that the counters fit one scan).  A digit's rank among equal digits comes from
    // lane ballots; the counts per (digit, slot, wave) are scanned in that order, which is
    // the order of positions t + c * kST.
    constexpr int kWaves = kST / kWave;
    constexpr int kDig = KPT <= 2 ? 5 : 4;   // digit bits
    constexpr int kBins = 1 << kDig;
    constexpr int kCnt = kBins * KPT * kWaves;
    int32_t* cnt = reinterpret_cast<int32_t*>(lds);                                         // [kCnt]
    unsigned long long* sk_l = reinterpret_cast<unsigned long long*>(lds + 4 * kCnt);        // [P]
    int32_t* len = reinterpret_cast<int32_t*>(sk_l + P);                                     // [P]
    int32_t* nxt = len + P;                                                                  // [P]
    const int wv = tid / kWave;
    const int bits = 32 - __clz((int)maxlen);
    for (int sh = 0; sh < bits; sh += kDig) {
        for (int i = tid; i < kCnt; i += kST) cnt[i] = 0;
        __syncthreads();
        int dg[KPT], drank[KPT];   // digit, rank among equal digits of the wave
#pragma unroll
        for (int c = 0; c < KPT; ++c) {
            const bool valid = tid + c * kST < nn;
            const int d = (kBins - 1) - ((key_len(x[c]) >> sh) & (kBins - 1));
            uint64_t m = __ballot(valid);
#pragma unroll
            for (int bt = 0; bt < kDig; ++bt) {
                const bool on = (d >> bt) & 1;
                const uint64_t bb = __ballot(valid && on);
                m &= on ? bb : ~bb;
            }
            dg[c] = d;
            drank[c] = lanes_below(m);
            if (valid && drank[c] == 0) cnt[(d * KPT + c) * kWaves + wv] = __popcll(m);
        }
        __syncthreads();
        int carry = 0;
        for (int b0 = 0; b0 < kCnt; b0 += kST) {
            const int i = b0 + tid;
            const int v = i < kCnt ? cnt[i] : 0;
            int tot;
            const int ex = sblock_excl<kST>(v, &tot);
            if (i < kCnt) cnt[i] = carry + ex;
            carry += tot;
        }
        __syncthreads();
#pragma unroll
        for (int c = 0; c < KPT; ++c)
            if (tid + c * kST < nn) sk_l[cnt[(dg[c] * KPT + c) * kWaves + wv] + drank[c]] = x[c];
        __syncthreads();
#pragma unroll
        for (int c = 0; c < KPT; ++c) {
            const int64_t i = tid + c * kST;
            x[c] = i < nn ? sk_l[i] : ~0ull;
        }
    }
    __syncthreads();
    unsigned long long* sk = a.skey + (int64_t)r * a.D;
#pragma unroll
    for (int c = 0; c < KPT; ++c) {
        const int64_t i = tid + c * kST;
        if (i < nn) {
            sk[i] = x[c];
            len[i] = key_len(x[c]);
        }
    }
    __syncthreads();
    // Sec. 2.2: the group starting at p holds B(l) samples, l = the length just before p
    // (the shortest of the previous group); the first group is a singleton
#pragma unroll
    for (int c = 0; c < KPT; ++c) {
        const int64_t i = tid + c * kST;
        if (i < nn) {
            const int64_t nx = i == 0 ? 1 : i + batch_size(a.budget, len[i - 1]);
            nxt[i] = (int32_t)(nx < nn ? nx : nn);
        }
    }
    __syncthreads();
    if (tid == 0) {
        // one thread walks the links (about one per group); pointer doubling over all
        // positions took longer, each of its rounds needing two block barriers
        int32_t* gs = a.gs + (int64_t)r * (a.D + 1);
        int64_t p = 0, g = 0;
        while (p < nn) {
            gs[g++] = (int32_t)p;
            p = nxt[p];
        }
        gs[g] = (int32_t)nn;
        *F = RankForm{cursor + f, nn, tok, (int32_t)g, s_err};
    }
}

// Books round k at the end of a chunk of launches, so that the host sees its outcome.
__global__ void __launch_bounds__(kST) stream_book_kernel(StreamArgs a, int64_t k) {
    const int32_t done = a.g->done;   // written by an earlier launch
    const StreamRec rk = a.rec[k];
    const StreamRec rp = a.rec[k > 0 ? k - 1 : 0];
    if (done) return;
    book_round(a, k, rk, rp, true);
    if (threadIdx.x == 0) a.rec[k].booked = 1;
}

// ------------------------------------------------------------------ final plan
__global__ void stream_slots_kernel(StreamArgs a, int64_t S, int32_t* rows, int32_t* maxlen, int64_t* tokens,
                                    double* approx) {
    const int64_t K = (int64_t)a.W * S;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; x < K; x += stride) {
        const int64_t r = x / S, j = x - r * S;
        const int64_t o = r * a.scap + j;
        rows[x] = a.srows[o];
        maxlen[x] = a.smax[o];
        tokens[x] = a.stok[o];
        if (approx) approx[x] = a.sadj[o];
    }
}

// Rank r's emitted views (slot order, row order), their identities and, when asked for,
// the row records (token start and length of each identity), read from the staged view
// table; blockIdx.x is the rank, blockIdx.y a slice of its stream.
__global__ void __launch_bounds__(256) stream_emit_out_kernel(StreamArgs a, int64_t S, const int64_t* row_off,
                                                              int32_t* emit_views, int32_t* emit_order,
                                                              int64_t* row_ts, int32_t* row_len) {
    const int r = blockIdx.x;
    const int64_t lo = row_off[(int64_t)r * S], hi = row_off[(int64_t)(r + 1) * S];
    const int32_t* ev = a.evw + (int64_t)r * a.q;
    const int64_t M = a.q * a.W;
    const int64_t stride = (int64_t)gridDim.y * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.y * blockDim.x + threadIdx.x; i < hi - lo; i += stride) {
        const int32_t m = ev[i];
        if (m < 0 || m >= M) continue;   // a library error, counted by the view bits
        const int64_t x = (int64_t)r * a.q + m / a.W;
        emit_views[lo + i] = m;
        emit_order[lo + i] = a.vid[x];
        if (row_ts) {
            row_ts[lo + i] = a.vts[x];
            row_len[lo + i] = a.vlen[x];
        }
    }
}

// Emitted-view bits, word-interleaved over ranks: bit i & 31 of word (i / 32) * W + r is
// view i * W + r (the i-th view of rank r), so the words of the W ranks for the same 32
// views are adjacent.
__device__ __forceinline__ bool view_emitted(const uint32_t* vbits, int64_t W, int64_t r, int64_t i) {
    return (vbits[(i >> 5) * W + r] >> (i & 31)) & 1;
}

// Rank r = blockIdx.x: the bits of its emitted views, set in LDS (a bit already set is a
// view emitted twice, a view of another rank or outside [0, M) is a library error; both
// count as bad views), then written out.  kLds: the rank's q bits fit in LDS; otherwise
// the bits are set in global memory, cleared beforehand.
template <bool kLds>
__global__ void __launch_bounds__(1024) stream_view_bits_kernel(StreamArgs a, int64_t S, const int64_t* row_off,
                                                                uint32_t* vbits, unsigned long long* bad_views) {
    extern __shared__ uint32_t s_bits[];
    const int r = blockIdx.x;
    const int64_t W = a.W, M = a.q * a.W, qw = (a.q + 31) / 32;
    const int64_t lo = row_off[(int64_t)r * S], hi = row_off[(int64_t)(r + 1) * S];
    const int32_t* ev = a.evw + (int64_t)r * a.q;
    if (kLds) {
        for (int64_t k = threadIdx.x; k < qw; k += blockDim.x) s_bits[k] = 0;
        __syncthreads();
    }
    unsigned long long bad = 0;
    for (int64_t e = threadIdx.x; e < hi - lo; e += blockDim.x) {
        const int64_t m = ev[e];
        if (m < 0 || m >= M || m % W != r) {
            bad += 1;
            continue;
        }
        const int64_t i = m / W;
        const uint32_t b = 1u << (i & 31);
        const uint32_t old = kLds ? atomicOr(&s_bits[i >> 5], b) : atomicOr(&vbits[(i >> 5) * W + r], b);
        bad += (old & b) ? 1 : 0;
    }
    if (kLds) {
        __syncthreads();
        for (int64_t k = threadIdx.x; k < qw; k += blockDim.x) vbits[k * W + r] = s_bits[k];
    }
    bad = wave_sum(bad);
    if ((threadIdx.x & (kWave - 1)) == 0 && bad) atomicAdd(bad_views, bad);
}

struct RowsLoadS {
    const int32_t* rows;
    int64_t K;
    __device__ int64_t operator()(int64_t i) const { return i < K ? (int64_t)rows[i] : 0; }
};
struct TileLoadS {
    const int32_t* rows;
    const int32_t* mx;
    int64_t K;
    __device__ int64_t operator()(int64_t i) const { return i < K ? (int64_t)rows[i] * mx[i] : 0; }
};
struct StoreS {
    int64_t* out;
    __device__ void operator()(int64_t i, int64_t v) const { out[i] = v; }
};

struct LeftFlag {
    StreamArgs a;
    const uint32_t* vbits;
    // rank-major position x = r * q + i <-> view m = i * W + r
    __device__ int64_t operator()(int64_t x) const {
        const int64_t r = x / a.q, i = x - r * a.q;
        return view_emitted(vbits, a.W, r, i) ? 0 : 1;
    }
};
struct LeftStore {
    StreamArgs a;
    const uint32_t* vbits;
    int32_t* left;
    int64_t* left_off;
    __device__ void operator()(int64_t x, int64_t ex) const {
        const int64_t r = x / a.q, i = x - r * a.q;
        if (i == 0) left_off[r] = ex;
        if (!view_emitted(vbits, a.W, r, i)) left[ex] = (int32_t)(i * a.W + r);
    }
};

struct StreamTotals {
    unsigned long long real_tokens;
    unsigned long long bad_views;
    unsigned long long missing_ids;
    unsigned long long duplicate_ids;
};

// Real tokens over the slots, and the identity counts.  perm is a permutation of [0, N),
// so identity perm[m] (m < N) is carried by the views m, m + N, m + 2N, ... below M (the
// padding repeats the list from its head) and by nothing else: its emission count is the
// sum of those views' bits.
__global__ void __launch_bounds__(256) stream_totals_kernel(StreamArgs a, int64_t K, const int64_t* tokens,
                                                            const uint32_t* vbits, StreamTotals* t) {
    const int64_t M = a.q * a.W;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    unsigned long long tok = 0, bad = 0, miss = 0, dup = 0;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < K; i += stride) tok += tokens[i];
    for (int64_t m = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; m < a.N; m += stride) {
        int64_t c = 0;
        for (int64_t v = m; v < M; v += a.N) c += view_emitted(vbits, a.W, v % a.W, v / a.W) ? 1 : 0;
        miss += c == 0;
        dup += c > 0 ? (unsigned long long)(c - 1) : 0ull;
    }
    __shared__ unsigned long long part[4][256 / kWave];
    const int w = threadIdx.x / kWave;
    tok = wave_sum(tok);
    bad = wave_sum(bad);
    miss = wave_sum(miss);
    dup = wave_sum(dup);
    if ((threadIdx.x & (kWave - 1)) == 0) {
        part[0][w] = tok;
        part[1][w] = bad;
        part[2][w] = miss;
        part[3][w] = dup;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        unsigned long long v[4] = {0, 0, 0, 0};
        for (int f = 0; f < 4; ++f)
            for (int i = 0; i < 256 / kWave; ++i) v[f] += part[f][i];
        if (v[0]) atomicAdd(&t->real_tokens, v[0]);
        if (v[1]) atomicAdd(&t->bad_views, v[1]);
        if (v[2]) atomicAdd(&t->missing_ids, v[2]);
        if (v[3]) atomicAdd(&t->duplicate_ids, v[3]);
    }
}

__global__ void fill_i64s_kernel(int64_t* p, int64_t n) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) p[i] = 0;
}

__global__ void fill_i32_kernel(int32_t* p, int64_t n) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) p[i] = 0;
}

__global__ void clear_totals_kernel(StreamTotals* t) {
    if (threadIdx.x == 0) *t = StreamTotals{};
}

struct StreamLayout {
    size_t g, ranks, form, rec, stepsum, bufv, skey, gs, srows, smax, stok, sadj, evw, vbits, vid, vts, vlen,
        totals, partials, rate, cap, total;
};

// Workspace layout of a streaming iteration after the window workspace (`at` bytes).
// Returns false when the slot capacity or the round limit asks for more than kMaxStreamBytes
// of workspace (every size is checked before it is multiplied, so none wraps).
constexpr int64_t kMaxStreamBytes = int64_t(1) << 50;

bool stream_layout(size_t at, int64_t W, int64_t N, int64_t D, int64_t scap, int64_t rounds, StreamLayout* L) {
    const int64_t q = N > 0 ? (N + W - 1) / W : 0;
    const int64_t M = q * W;
    // per-rank staging slots and round records, bounded before any product is formed
    if (scap < 0 || rounds < 1 || scap > kMaxStreamBytes / 8 / W || rounds > kMaxStreamBytes / 64) return false;
    const int64_t K1 = W * scap + 1;
    const int64_t scan_n = (K1 > M + 1 ? K1 : M + 1);
    size_t o = at;
    auto take = [&](size_t bytes) {
        size_t x = o;
        o = (o + (bytes ? bytes : 1) + 255) & ~(size_t)255;
        return x;
    };
    L->g = take(sizeof(StreamGlobal));
    L->ranks = take(sizeof(RankStream) * W);
    L->form = take(sizeof(RankForm) * 2 * W);
    L->rec = take(sizeof(StreamRec) * rounds);
    L->stepsum = take(8 * 3 * D);
    L->bufv = take(4 * W * D);
    L->skey = take(8 * W * D);
    L->gs = take(4 * W * (D + 1));
    L->srows = take(4 * W * scap);
    L->smax = take(4 * W * scap);
    L->stok = take(8 * W * scap);
    L->sadj = take(8 * W * scap);
    L->evw = take(4 * (M > 0 ? M : 1));
    L->vbits = take(4 * W * ((q + 31) / 32));
    L->vid = take(4 * (M > 0 ? M : 1));
    L->vts = take(8 * (M > 0 ? M : 1));
    L->vlen = take(4 * (M > 0 ? M : 1));
    L->totals = take(sizeof(StreamTotals));
    L->partials = take(8 * (scan_n / kScanTile + 4));
    L->rate = take(4 * W);
    L->cap = take(8 * W);
    L->total = o;
    return o - at <= (size_t)kMaxStreamBytes;
}

// A lower bound on the rounds still to run after the committed state `hr`: a rank fetches
// at most rate[r] views a round, and its last fetch is followed by the round that finds
// it finished (join: every rank; non-join: the first); a non-join quota needs at least
// (Q - emitted) / (W * D) more rounds, since a round emits at most a full buffer per rank.
int64_t stream_rounds_left(const StreamArgs& a, const int32_t* rate, const std::vector<RankStream>& hr,
                           const StreamGlobal& hg, int64_t at_least) {
    int64_t hi = 0, lo = LLONG_MAX;
    for (int r = 0; r < a.W; ++r) {
        const int64_t need = (a.q - hr[r].cursor + rate[r] - 1) / rate[r];
        hi = std::max(hi, need);
        lo = std::min(lo, need);
    }
    const bool nonjoin = a.mode == ODB_MODE_NONJOIN_QUOTA;
    int64_t b = (nonjoin ? lo : hi) + 1;
    if (nonjoin) {
        const int64_t per = (int64_t)a.W * a.D;
        b = std::min(b, std::max<int64_t>(1, (a.quota - hg.emitted + per - 1) / per));
    }
    return std::max(b, at_least);
}

int check_stream_params(const odb_window_t* w, const odb_stream_params_t* p, int64_t slot_capacity) {
    if (!p) return set_error(ODB_E_INVALID_ARG, "params is NULL");
    if (p->mode != ODB_MODE_JOIN && p->mode != ODB_MODE_NONJOIN_QUOTA)
        return set_error(ODB_E_INVALID_ARG, "unknown mode %d", p->mode);
    if (p->reserved0 != 0) return set_error(ODB_E_INVALID_ARG, "params.reserved0 must be 0");
    if (p->mode == ODB_MODE_NONJOIN_QUOTA && p->quota < 1)
        return set_error(ODB_E_INVALID_ARG, "quota must be >= 1 in non-join mode");
    if (p->buffer_size < 1 || p->depth < p->buffer_size || p->depth > kMaxDepth)
        return set_error(ODB_E_INVALID_ARG, "need 1 <= buffer_size <= depth <= %d", kMaxDepth);
    if (p->max_rounds < 1) return set_error(ODB_E_INVALID_ARG, "max_rounds must be >= 1");
    if (slot_capacity < 0) return set_error(ODB_E_INVALID_ARG, "slot_capacity must be >= 0");
    if (!p->rate) return set_error(ODB_E_INVALID_ARG, "rate is NULL");
    for (int r = 0; r < w->num_ranks; ++r) {
        if (p->rate[r] < 1) return set_error(ODB_E_INVALID_ARG, "rate[%d] must be >= 1", r);
        if (p->slot_capacity && p->slot_capacity[r] < 0)
            return set_error(ODB_E_INVALID_ARG, "slot_capacity[%d] must be >= 0", r);
    }
    if (w->num_samples + w->num_ranks >= 0x7FFFFFFFll)
        return set_error(ODB_E_INVALID_ARG, "N + W must stay below 2^31 (view ids are int32)");
    return ODB_OK;
}

}  // namespace

}  // namespace odb

using namespace odb;

extern "C" size_t odb_stream_workspace_size(const odb_window_t* w, int32_t depth, int64_t slot_capacity,
                                            int64_t max_rounds) {
    Layout L;
    if (!make_layout(w, &L)) return 0;
    if (depth < 1 || depth > kMaxDepth || slot_capacity < 0 || max_rounds < 1) return 0;
    StreamLayout S;
    if (!stream_layout(L.total, w->num_ranks, w->num_samples, depth, slot_capacity / w->num_ranks, max_rounds, &S))
        return 0;
    return S.total;
}

extern "C" int odb_stream_plan(const odb_window_t* w, const int32_t* d_perm, int64_t budget,
                               const odb_stream_params_t* params, int64_t slot_capacity, int32_t* d_emit_order,
                               int32_t* d_emit_views, int64_t* d_row_token_start, int32_t* d_row_len,
                               int32_t* d_slot_rows, int32_t* d_slot_maxlen,
                               int64_t* d_slot_row_off, int64_t* d_slot_tile_off, int64_t* d_slot_tokens,
                               double* d_slot_tokens_approx, int32_t* d_left_views, int64_t* d_left_off,
                               odb_stream_round_t* h_trace, odb_stream_info_t* h_info, void* d_ws, size_t ws_bytes,
                               void* stream) {
    Layout L;
    if (!make_layout(w, &L)) return set_error(ODB_E_INVALID_ARG, "bad window");
    if (budget < 1) return set_error(ODB_E_INVALID_ARG, "budget must be >= 1");
    ODB_TRY(check_stream_params(w, params, slot_capacity));
    if (!h_info) return set_error(ODB_E_INVALID_ARG, "h_info is NULL");
    if ((d_row_token_start == nullptr) != (d_row_len == nullptr))
        return set_error(ODB_E_INVALID_ARG, "d_row_token_start and d_row_len are given together or not at all");
    const int W = w->num_ranks;
    const int64_t N = w->num_samples;
    const int64_t q = N > 0 ? (N + W - 1) / W : 0;
    const int64_t M = q * W;
    const int64_t scap = slot_capacity / W;
    if (N > 0 && !d_perm) return set_error(ODB_E_INVALID_ARG, "d_perm is NULL");
    if (M > 0 && (!d_emit_order || !d_emit_views || !d_left_views))
        return set_error(ODB_E_INVALID_ARG, "view arrays must not be NULL");
    if (!d_slot_row_off || !d_slot_tile_off || !d_left_off)
        return set_error(ODB_E_INVALID_ARG, "offset arrays must not be NULL");
    if (scap > 0 && (!d_slot_rows || !d_slot_maxlen || !d_slot_tokens))
        return set_error(ODB_E_INVALID_ARG, "slot arrays must not be NULL");
    StreamLayout SL;
    if (!stream_layout(L.total, W, N, params->depth, scap, params->max_rounds, &SL))
        return set_error(ODB_E_INVALID_ARG, "slot_capacity (%lld) or max_rounds (%lld) asks for more than 2^50 bytes of "
                         "workspace", (long long)slot_capacity, (long long)params->max_rounds);
    if (!d_ws) return set_error(ODB_E_INVALID_ARG, "workspace is NULL");
    if (reinterpret_cast<uintptr_t>(d_ws) & 255) return set_error(ODB_E_INVALID_ARG, "workspace must be 256-byte aligned");
    if (ws_bytes < SL.total)
        return set_error(ODB_E_WORKSPACE, "workspace has %zu bytes, %zu needed", ws_bytes, SL.total);
    memset(h_info, 0, sizeof(*h_info));
    hipStream_t s = static_cast<hipStream_t>(stream);
    // the window part of the workspace: rank offsets and a cleared status word, as after
    // odb_align_groups, so odb_collate / odb_collate_status work on this workspace
    ODB_TRY(upload_small(w, L, d_ws, nullptr, s));

    StreamArgs a{};
    a.W = W;
    a.mode = params->mode;
    a.N = N;
    a.q = q;
    a.D = params->depth;
    a.bufsize = params->buffer_size;
    a.budget = budget;
    a.quota = params->quota;
    a.scap = scap;
    a.max_rounds = params->max_rounds;
    a.tok_off = w->d_token_offsets;
    a.perm = d_perm;
    a.rate = ws_at<int32_t>(d_ws, SL.rate);
    a.cap = params->slot_capacity ? ws_at<int64_t>(d_ws, SL.cap) : nullptr;
    a.g = ws_at<StreamGlobal>(d_ws, SL.g);
    a.ranks = ws_at<RankStream>(d_ws, SL.ranks);
    a.form = ws_at<RankForm>(d_ws, SL.form);
    a.rec = ws_at<StreamRec>(d_ws, SL.rec);
    a.stepsum = ws_at<int64_t>(d_ws, SL.stepsum);
    a.bufv = ws_at<int32_t>(d_ws, SL.bufv);
    a.skey = ws_at<unsigned long long>(d_ws, SL.skey);
    a.gs = ws_at<int32_t>(d_ws, SL.gs);
    a.srows = ws_at<int32_t>(d_ws, SL.srows);
    a.smax = ws_at<int32_t>(d_ws, SL.smax);
    a.stok = ws_at<int64_t>(d_ws, SL.stok);
    a.sadj = ws_at<double>(d_ws, SL.sadj);
    a.evw = ws_at<int32_t>(d_ws, SL.evw);
    a.vid = ws_at<int32_t>(d_ws, SL.vid);
    a.vts = ws_at<int64_t>(d_ws, SL.vts);
    a.vlen = ws_at<int32_t>(d_ws, SL.vlen);
    ODB_TRY_HIP(hipMemcpyAsync(const_cast<int32_t*>(a.rate), params->rate, 4 * W, hipMemcpyHostToDevice, s));
    if (a.cap)
        ODB_TRY_HIP(hipMemcpyAsync(const_cast<int64_t*>(a.cap), params->slot_capacity, 8 * W, hipMemcpyHostToDevice, s));
    if (M > 0) {
        hipLaunchKernelGGL(stream_views_kernel, dim3(grid_for(M, 256, (int64_t)num_cus() * kPlanBlocksPerCU)),
                           dim3(256), 0, s, a, const_cast<int32_t*>(a.vid), const_cast<int64_t*>(a.vts),
                           const_cast<int32_t*>(a.vlen));
        ODB_LAUNCHED();
    }
    hipLaunchKernelGGL(stream_init_kernel, dim3(grid_for(std::max<int64_t>(params->max_rounds, W), 256, 1024)),
                       dim3(256), 0, s, a, params->max_rounds);
    ODB_LAUNCHED();

    // rounds, in chunks, until the done flag is up
    const int kpt = sort_kpt(a.D);
    const size_t lds = round_lds_bytes(a.D);
    auto launch_round = [&](int64_t j) {
        switch (kpt) {
            case 1: hipLaunchKernelGGL(stream_round_kernel<1>, dim3(W), dim3(kST), lds, s, a, j); break;
            case 2: hipLaunchKernelGGL(stream_round_kernel<2>, dim3(W), dim3(kST), lds, s, a, j); break;
            case 4: hipLaunchKernelGGL(stream_round_kernel<4>, dim3(W), dim3(kST), lds, s, a, j); break;
            default: hipLaunchKernelGGL(stream_round_kernel<8>, dim3(W), dim3(kST), lds, s, a, j); break;
        }
    };
    static_assert(kMaxDepth <= 8 * kST, "sort slots per thread");
    StreamGlobal hg{};
    std::vector<RankStream> hr(W);   // committed state after the last booked round
    launch_round(0);                  // round 0's form
    ODB_LAUNCHED();
    for (int64_t k0 = 0; k0 < a.max_rounds;) {
        // rounds k0 .. k0+cnt-1: launch k+1 emits round k; the chunk's last round is then
        // booked on its own
        const int64_t cnt = std::min<int64_t>(a.max_rounds - k0, stream_rounds_left(a, params->rate, hr, hg,
                                                                                    k0 == 0 ? 1 : kMinChunk));
        for (int64_t k = k0; k < k0 + cnt; ++k) {
            launch_round(k + 1);
            ODB_LAUNCHED();
        }
        hipLaunchKernelGGL(stream_book_kernel, dim3(1), dim3(kST), 0, s, a, k0 + cnt - 1);
        ODB_LAUNCHED();
        ODB_TRY_HIP(hipMemcpyAsync(&hg, a.g, sizeof(hg), hipMemcpyDeviceToHost, s));
        ODB_TRY_HIP(hipMemcpyAsync(hr.data(), a.ranks, sizeof(RankStream) * W, hipMemcpyDeviceToHost, s));
        ODB_TRY_HIP(hipStreamSynchronize(s));
        if (hg.done) break;
        k0 += cnt;
    }
    if (hg.err & kSErrIdentity) return set_error(ODB_E_INVALID_DATA, "perm holds a value outside [0, N)");
    if (hg.err & kSErrLength) return set_error(ODB_E_INVALID_DATA, "a sample has length < 1 or >= 2^31");
    if (hg.err & kSErrInternal) return set_error(ODB_E_INTERNAL, "streaming round state inconsistent");
    h_info->rounds = hg.rounds;
    if (!hg.done || (hg.err & kSErrRounds)) {
        h_info->rounds = a.max_rounds;
        return set_error(ODB_E_CAPACITY, "the iteration did not finish within %lld rounds",
                         (long long)a.max_rounds);
    }
    const int64_t S = hg.steps;
    const int64_t K = (int64_t)W * S;
    h_info->steps = S;
    h_info->emit_rounds = hg.emit_rounds;
    h_info->skip_rounds = hg.skip_rounds;
    h_info->stop_reason = hg.stop;
    h_info->views = M;
    h_info->emitted_views = hg.emitted;
    h_info->max_step_samples = hg.max_step;
    h_info->splits = hg.splits;
    h_info->overflow_groups = hg.overflow;
    h_info->second_gather_rounds = hg.second_gather;
    h_info->max_outstanding = (int64_t)hg.max_outstanding;
    h_info->required_slot_capacity = K;
    if (S > scap)
        return set_error(ODB_E_CAPACITY, "plan needs %lld slots, capacity is %lld", (long long)K,
                         (long long)slot_capacity);

    // plan arrays in the window layout
    const int64_t gcap = (int64_t)num_cus() * kPlanBlocksPerCU;
    int64_t* partials = ws_at<int64_t>(d_ws, SL.partials);
    if (K > 0) {
        hipLaunchKernelGGL(stream_slots_kernel, dim3(grid_for(K, 256, gcap)), dim3(256), 0, s, a, S, d_slot_rows,
                           d_slot_maxlen, d_slot_tokens, d_slot_tokens_approx);
        ODB_LAUNCHED();
    }
    ODB_TRY((device_excl_scan<int64_t>(RowsLoadS{d_slot_rows, K}, StoreS{d_slot_row_off}, K + 1, partials, s)));
    ODB_TRY((device_excl_scan<int64_t>(TileLoadS{d_slot_rows, d_slot_maxlen, K}, StoreS{d_slot_tile_off}, K + 1,
                                       partials, s)));
    uint32_t* vbits = ws_at<uint32_t>(d_ws, SL.vbits);
    const int64_t qw = (q + 31) / 32;
    const bool bits_in_lds = 4 * qw <= kViewBitsLds;
    StreamTotals* tot = ws_at<StreamTotals>(d_ws, SL.totals);
    if (!bits_in_lds && qw > 0) {
        hipLaunchKernelGGL(fill_i32_kernel, dim3(grid_for(W * qw, 256, gcap)), dim3(256), 0, s,
                           reinterpret_cast<int32_t*>(vbits), W * qw);
        ODB_LAUNCHED();
    }
    hipLaunchKernelGGL(clear_totals_kernel, dim3(1), dim3(64), 0, s, tot);
    ODB_LAUNCHED();
    if (K > 0) {
        hipLaunchKernelGGL(stream_emit_out_kernel, dim3(W, 64), dim3(256), 0, s, a, S, (const int64_t*)d_slot_row_off,
                           d_emit_views, d_emit_order, d_row_token_start, d_row_len);
        ODB_LAUNCHED();
    }
    if (M > 0) {
        if (bits_in_lds)
            hipLaunchKernelGGL(stream_view_bits_kernel<true>, dim3(W), dim3(1024), 4 * qw, s, a, S,
                               (const int64_t*)d_slot_row_off, vbits, &tot->bad_views);
        else
            hipLaunchKernelGGL(stream_view_bits_kernel<false>, dim3(W), dim3(1024), 0, s, a, S,
                               (const int64_t*)d_slot_row_off, vbits, &tot->bad_views);
        ODB_LAUNCHED();
    }
    hipLaunchKernelGGL(fill_i64s_kernel, dim3(1), dim3(256), 0, s, d_left_off, (int64_t)W + 1);
    ODB_LAUNCHED();
    ODB_TRY((device_excl_scan<int64_t>(LeftFlag{a, vbits}, LeftStore{a, vbits, d_left_views, d_left_off}, M,
                                       partials, s)));
    hipLaunchKernelGGL(stream_totals_kernel, dim3(grid_for(std::max<int64_t>(std::max(K, N), 1), 256, gcap)),
                       dim3(256), 0, s, a, K, (const int64_t*)d_slot_tokens, (const uint32_t*)vbits, tot);
    ODB_LAUNCHED();
    StreamTotals ht{};
    int64_t padded = 0, nleft = 0;
    ODB_TRY_HIP(hipMemcpyAsync(&ht, tot, sizeof(ht), hipMemcpyDeviceToHost, s));
    ODB_TRY_HIP(hipMemcpyAsync(&padded, d_slot_tile_off + K, 8, hipMemcpyDeviceToHost, s));
    ODB_TRY_HIP(hipMemcpyAsync(hr.data(), a.ranks, sizeof(RankStream) * W, hipMemcpyDeviceToHost, s));
    if (M > 0) ODB_TRY_HIP(hipMemcpyAsync(&nleft, partials + (M + kScanTile - 1) / kScanTile, 8,
                                          hipMemcpyDeviceToHost, s));
    std::vector<StreamRec> hrec(h_trace ? hg.rounds : 0);
    if (h_trace && hg.rounds > 0)
        ODB_TRY_HIP(hipMemcpyAsync(hrec.data(), a.rec, sizeof(StreamRec) * hg.rounds, hipMemcpyDeviceToHost, s));
    ODB_TRY_HIP(hipStreamSynchronize(s));
    // the left-over offsets end with the total; the scan left off[W] unset
    ODB_TRY_HIP(hipMemcpyAsync(d_left_off + W, &nleft, 8, hipMemcpyHostToDevice, s));
    ODB_TRY_HIP(hipStreamSynchronize(s));
    int64_t fetched = 0;
    for (int r = 0; r < W; ++r) fetched += hr[r].cursor;
    h_info->real_tokens = (int64_t)ht.real_tokens;
    h_info->padded_elems = padded;
    h_info->pad_fraction = padded > 0 ? 1.0 - (double)ht.real_tokens / (double)padded : 0.0;
    h_info->undelivered_views = fetched - hg.emitted;
    h_info->pending_views = M - fetched;
    h_info->bad_views = (int64_t)ht.bad_views;
    h_info->missing_ids = (int64_t)ht.missing_ids;
    h_info->duplicate_ids = (int64_t)ht.duplicate_ids;
    if (h_trace) {
        int64_t phi = M;
        for (int64_t i = 0; i < hg.rounds; ++i) {
            phi -= hrec[i].kind == 0 ? hrec[i].emitted : 0;
            h_trace[i].kind = hrec[i].kind;
            h_trace[i].reserved0 = 0;
            h_trace[i].target = hrec[i].kind == 0 ? hrec[i].target : 0;
            h_trace[i].emitted = hrec[i].kind == 0 ? hrec[i].emitted : 0;
            h_trace[i].phi = phi;
        }
    }
    if (nleft != M - hg.emitted || ht.bad_views != 0)
        return set_error(ODB_E_INTERNAL, "streaming plan does not account for every view exactly once");
    return ODB_OK;
}
