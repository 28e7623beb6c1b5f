// Loss-scaling weights of an aligned plan (Sec. 2.3 "Loss scaling", Eq. 2, App. B, and
// the three scaling modes of the loss-scaling ablation in App. N).
//
// At step j every rank r trains on its slot (r, j).  DDP averages the ranks' per-token
// mean losses, so rank r pre-scales its mean by W * w_{r,j}; the exact token-level weight
// w = t_{r,j} / sum_r t_{r,j} makes the result the per-token mean over the whole step.
// The sample-level weight uses the slot's rows instead of its tokens, the approximate
// token-level weight the approximate token counts that alignment records per slot.
//
// One thread per step.  Slots are rank-major (k = r * S + j), so at a fixed rank the
// threads of a wave read consecutive slots.  The sums over ranks run in rank order and
// each fp64 operation is rounded on its own (contraction off), which makes the weights
// reproducible bit for bit on any device or host that follows the same order.
#include "odb_internal.h"

namespace odb {

namespace {

__global__ void __launch_bounds__(kBlock) loss_weights_kernel(int W, int64_t S, int mode,
                                                              const int32_t* __restrict__ rows,
                                                              const int64_t* __restrict__ tokens,
                                                              const double* __restrict__ approx,
                                                              double* __restrict__ weight,
                                                              int64_t* __restrict__ step_tokens,
                                                              int64_t* __restrict__ step_samples) {
#pragma clang fp contract(off)
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j < S; j += stride) {
        int64_t t_sum = 0, n_sum = 0;
        double a_sum = 0.0;
        for (int r = 0; r < W; ++r) {
            const int64_t k = (int64_t)r * S + j;
            t_sum += tokens[k];
            n_sum += rows[k];
            if (mode == ODB_WEIGHT_TOKEN_APPROX) a_sum = a_sum + approx[k];
        }
        for (int r = 0; r < W; ++r) {
            const int64_t k = (int64_t)r * S + j;
            double w = 0.0;
            if (mode == ODB_WEIGHT_SAMPLE) {
                if (n_sum > 0) w = (double)rows[k] / (double)n_sum;
            } else if (mode == ODB_WEIGHT_TOKEN_APPROX) {
                if (a_sum > 0.0) w = approx[k] / a_sum;
            } else {
                if (t_sum > 0) w = (double)tokens[k] / (double)t_sum;
            }
            weight[k] = w;
        }
        if (step_tokens) step_tokens[j] = t_sum;
        if (step_samples) step_samples[j] = n_sum;
    }
}

}  // namespace

}  // namespace odb

using namespace odb;

extern "C" int odb_loss_weights(int32_t num_ranks, int64_t steps, int32_t mode, const int32_t* d_slot_rows,
                                const int64_t* d_slot_tokens, const double* d_slot_tokens_approx, double* d_weight,
                                int64_t* d_step_tokens, int64_t* d_step_samples, void* stream) {
    if (num_ranks < 1) return set_error(ODB_E_INVALID_ARG, "num_ranks must be >= 1");
    if (steps < 0) return set_error(ODB_E_INVALID_ARG, "steps must be >= 0");
    if (steps > INT64_MAX / num_ranks) return set_error(ODB_E_INVALID_ARG, "num_ranks * steps overflows");
    if (mode != ODB_WEIGHT_SAMPLE && mode != ODB_WEIGHT_TOKEN_APPROX && mode != ODB_WEIGHT_TOKEN_EXACT)
        return set_error(ODB_E_INVALID_ARG, "unknown loss-weight mode %d", mode);
    if (steps == 0) return ODB_OK;
    if (!d_slot_rows || !d_slot_tokens || !d_weight)
        return set_error(ODB_E_INVALID_ARG, "slot arrays and d_weight must not be NULL");
    if (mode == ODB_WEIGHT_TOKEN_APPROX && !d_slot_tokens_approx)
        return set_error(ODB_E_INVALID_ARG, "the approximate mode needs d_slot_tokens_approx");
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipLaunchKernelGGL(loss_weights_kernel, dim3(grid_for(steps, kBlock, (int64_t)num_cus() * 8)), dim3(kBlock), 0,
                       s, (int)num_ranks, steps, (int)mode, d_slot_rows, d_slot_tokens, d_slot_tokens_approx, d_weight,
                       d_step_tokens, d_step_samples);
    ODB_LAUNCHED();
    return ODB_OK;
}
