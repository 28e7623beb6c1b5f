// ROI length sketch (Sec. 1 defines the length heterogeneity CV = sigma / mu of realised
// post-pipeline lengths; the practical-guidance section screens a 1k-5k sample with CV
// and the short-sample fraction f_s = Pr[l < L_max / 4]: CV >= 0.8 or f_s > 0.2 marks a
// high-return workload).
//
// The device computes exact integer moments of the sketched lengths in one pass: count,
// sum l, sum l^2 (as the separate sums of the high and low 32-bit halves of every l^2, so
// nothing overflows for up to 2^31 samples), the count of 4 l < L_max, min and max.  The
// host turns them into CV = sqrt(n sum l^2 - (sum l)^2) / sum l with a 128-bit integer
// numerator, so the only rounding is in the final conversion, root and quotient.
//
// Bytes: 8 B (two token offsets, one of them shared with the neighbour) read per sketched
// sample, plus 4 B per id when ids are given; one block-level reduction and six 64-bit
// atomics per block.
#include <cmath>

#include "odb_internal.h"

namespace odb {

namespace {

struct DevSketch {
    int64_t n;
    int64_t short_n;
    int64_t s1;
    int64_t s2_hi;
    int64_t s2_lo;
    unsigned long long min_len;
    unsigned long long max_len;
    int32_t err;
    int32_t pad;
};

enum : int32_t { kSketchBadId = 1, kSketchBadLength = 2 };

__global__ void sketch_init_kernel(DevSketch* d) {
    if (threadIdx.x == 0) {
        *d = DevSketch{};
        d->min_len = ~0ull;
    }
}

template <typename T>
__device__ __forceinline__ T wave_min(T v) {
#pragma unroll
    for (int d = kWave / 2; d > 0; d >>= 1) {
        const T o = __shfl_xor(v, d, kWave);
        v = o < v ? o : v;
    }
    return v;
}

template <typename T>
__device__ __forceinline__ T wave_max(T v) {
#pragma unroll
    for (int d = kWave / 2; d > 0; d >>= 1) {
        const T o = __shfl_xor(v, d, kWave);
        v = o > v ? o : v;
    }
    return v;
}

__global__ void __launch_bounds__(kBlock) sketch_kernel(const int64_t* __restrict__ tok_off, int64_t n,
                                                        const int32_t* __restrict__ ids, int64_t count,
                                                        int64_t budget, DevSketch* __restrict__ out) {
    int64_t cnt = 0, short_n = 0, s1 = 0, s2_hi = 0, s2_lo = 0;
    unsigned long long mn = ~0ull, mx = 0;
    int32_t err = 0;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count; i += stride) {
        const int64_t s = ids ? (int64_t)ids[i] : i;
        if (s < 0 || s >= n) {
            err |= kSketchBadId;
            continue;
        }
        const int64_t l = tok_off[s + 1] - tok_off[s];
        if (l < 1 || l > 0x7FFFFFFFll) {
            err |= kSketchBadLength;
            continue;
        }
        const uint64_t sq = (uint64_t)l * (uint64_t)l;
        cnt += 1;
        s1 += l;
        s2_hi += (int64_t)(sq >> 32);
        s2_lo += (int64_t)(sq & 0xFFFFFFFFull);
        short_n += 4 * l < budget ? 1 : 0;
        mn = (unsigned long long)l < mn ? (unsigned long long)l : mn;
        mx = (unsigned long long)l > mx ? (unsigned long long)l : mx;
    }
    cnt = wave_sum(cnt);
    short_n = wave_sum(short_n);
    s1 = wave_sum(s1);
    s2_hi = wave_sum(s2_hi);
    s2_lo = wave_sum(s2_lo);
    mn = wave_min(mn);
    mx = wave_max(mx);
    __shared__ int64_t part[5][kBlock / kWave];
    __shared__ unsigned long long ext[2][kBlock / kWave];
    __shared__ int32_t berr;
    if (threadIdx.x == 0) berr = 0;
    __syncthreads();
    if (err) atomicOr(&berr, err);
    const int wave = threadIdx.x / kWave;
    if ((threadIdx.x & (kWave - 1)) == 0) {
        part[0][wave] = cnt;
        part[1][wave] = short_n;
        part[2][wave] = s1;
        part[3][wave] = s2_hi;
        part[4][wave] = s2_lo;
        ext[0][wave] = mn;
        ext[1][wave] = mx;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        int64_t v[5] = {0, 0, 0, 0, 0};
        unsigned long long bmn = ~0ull, bmx = 0;
        for (int w = 0; w < kBlock / kWave; ++w) {
            for (int f = 0; f < 5; ++f) v[f] += part[f][w];
            bmn = ext[0][w] < bmn ? ext[0][w] : bmn;
            bmx = ext[1][w] > bmx ? ext[1][w] : bmx;
        }
        if (v[0] > 0) {
            atomicAdd((unsigned long long*)&out->n, (unsigned long long)v[0]);
            atomicAdd((unsigned long long*)&out->short_n, (unsigned long long)v[1]);
            atomicAdd((unsigned long long*)&out->s1, (unsigned long long)v[2]);
            atomicAdd((unsigned long long*)&out->s2_hi, (unsigned long long)v[3]);
            atomicAdd((unsigned long long*)&out->s2_lo, (unsigned long long)v[4]);
            atomicMin(&out->min_len, bmn);
            atomicMax(&out->max_len, bmx);
        }
        if (berr) atomicOr(&out->err, berr);
    }
}

}  // namespace

}  // namespace odb

using namespace odb;

extern "C" int odb_length_sketch(const odb_window_t* w, const int32_t* d_ids, int64_t count, int64_t budget,
                                 odb_length_sketch_t* h_out, void* d_ws, size_t ws_bytes, void* stream) {
    Layout L;
    ODB_TRY(check_workspace(w, d_ws, ws_bytes, &L));
    if (!h_out) return set_error(ODB_E_INVALID_ARG, "h_out is NULL");
    if (budget < 1) return set_error(ODB_E_INVALID_ARG, "budget must be >= 1");
    if (count < 0 || count > 0x7FFFFFFFll) return set_error(ODB_E_INVALID_ARG, "count must be in [0, 2^31)");
    if (!d_ids && count > w->num_samples)
        return set_error(ODB_E_INVALID_ARG, "count exceeds the window's %lld samples", (long long)w->num_samples);
    static_assert(sizeof(DevSketch) <= 256, "sketch record must fit its workspace slot");
    *h_out = odb_length_sketch_t{};
    hipStream_t s = static_cast<hipStream_t>(stream);
    DevSketch* d = ws_at<DevSketch>(d_ws, L.sketch);
    hipLaunchKernelGGL(sketch_init_kernel, dim3(1), dim3(64), 0, s, d);
    ODB_LAUNCHED();
    if (count > 0) {
        hipLaunchKernelGGL(sketch_kernel, dim3(grid_for(count, kBlock, (int64_t)num_cus() * 8)), dim3(kBlock), 0, s,
                           w->d_token_offsets, w->num_samples, d_ids, count, budget, d);
        ODB_LAUNCHED();
    }
    DevSketch h;
    ODB_TRY_HIP(hipMemcpyAsync(&h, d, sizeof(h), hipMemcpyDeviceToHost, s));
    ODB_TRY_HIP(hipStreamSynchronize(s));
    if (h.err & kSketchBadId) return set_error(ODB_E_INVALID_DATA, "a sketch id lies outside the window");
    if (h.err & kSketchBadLength) return set_error(ODB_E_INVALID_DATA, "a sketched sample has length < 1 or >= 2^31");
    h_out->samples = h.n;
    h_out->short_samples = h.short_n;
    h_out->sum_len = h.s1;
    h_out->sum_sq_hi = (uint64_t)h.s2_hi;
    h_out->sum_sq_lo = (uint64_t)h.s2_lo;
    if (h.n == 0) return ODB_OK;
    h_out->min_len = (int64_t)h.min_len;
    h_out->max_len = (int64_t)h.max_len;
    // n^2 sigma^2 = n sum l^2 - (sum l)^2, exact: n < 2^31 and sum l^2 < 2^93
    const unsigned __int128 s2 = ((unsigned __int128)(uint64_t)h.s2_hi << 32) + (uint64_t)h.s2_lo;
    const unsigned __int128 num = (unsigned __int128)(uint64_t)h.n * s2 -
                                  (unsigned __int128)(uint64_t)h.s1 * (uint64_t)h.s1;
    h_out->mean = (double)h.s1 / (double)h.n;
    h_out->cv = std::sqrt((double)num) / (double)h.s1;
    h_out->short_fraction = (double)h.short_n / (double)h.n;
    h_out->high_roi = (h_out->cv >= 0.8 || h_out->short_fraction > 0.2) ? 1 : 0;
    return ODB_OK;
}
