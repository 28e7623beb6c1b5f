/*
 * The window pipeline driven from plain C through include/odb.h, with no Python and no
 * torch: device memory from the HIP runtime API, then odb_form_groups ->
 * odb_align_groups (retried once with the slot capacity the plan reports) ->
 * odb_collate and odb_collate_static (into a second set of outputs) -> odb_loss_weights,
 * odb_check_coverage over the plan's emitted and left-over ids, and odb_length_sketch
 * over every sample; every output is written to a file for the test to compare with the
 * oracle.
 *
 *   window_pipeline IN OUT BUDGET MODE QUOTA
 *
 * IN (little-endian): int64 W, n, T; int64 rank_offsets[W+1]; int64 token_offsets[n+1];
 * int32 tokens[T].
 * OUT: int64 info[15] (steps, rounds, stop_reason, emitted_samples, leftover_samples,
 * real_tokens, padded_elems, max_step_samples, splits, overflow_groups, missing_ids,
 * duplicate_ids, bad_views, second_gather_rounds, required_slot_capacity), double
 * pad_fraction, int64 capacity_retries; int32 order[n], sorted_len[n], group_index[n],
 * groups_per_rank[W]; int32 emit_order[emitted]; int32 slot_rows[K], slot_maxlen[K];
 * int64 slot_row_off[K+1], slot_tile_off[K+1], slot_tokens[K]; int32 leftover[leftover];
 * int64 leftover_off[W+1]; int32 input_ids[P], labels[P], attention_mask[P],
 * position_ids[P]; the same four arrays from odb_collate_static and its int32 status;
 * double weight[K] (exact token-level mode); int64 sketch[7] (samples, short_samples,
 * sum_len, sum_sq_hi, sum_sq_lo, min_len, max_len), double sketch[3] (mean, cv,
 * short_fraction), int64 high_roi; int64 coverage[3] (bad_views, missing_ids,
 * duplicate_ids); with K = W * steps and P = padded_elems.
 *
 * Exit status 0 on success; otherwise the failing call and its message go to stderr.
 */
#define __HIP_PLATFORM_AMD__ 1
#include <hip/hip_runtime_api.h>

#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "odb.h"

static int fail(const char* what, int status) {
    fprintf(stderr, "%s: %s (%s)\n", what, odb_status_string(status), odb_last_error_message());
    return 1;
}

#define HIP_CHECK(call)                                                                  \
    do {                                                                                 \
        hipError_t e_ = (call);                                                          \
        if (e_ != hipSuccess) {                                                          \
            fprintf(stderr, "%s: %s\n", #call, hipGetErrorString(e_));                   \
            exit(2);                                                                     \
        }                                                                                \
    } while (0)

static void* dev_alloc(size_t bytes) {
    void* p = NULL;
    HIP_CHECK(hipMalloc(&p, bytes ? bytes : 16));
    return p;
}

static void read_exact(FILE* f, void* dst, size_t bytes) {
    if (bytes && fread(dst, 1, bytes, f) != bytes) {
        fprintf(stderr, "short input file\n");
        exit(2);
    }
}

static void* host_alloc(size_t bytes) {
    void* p = malloc(bytes ? bytes : 16);
    if (!p) {
        fprintf(stderr, "out of host memory\n");
        exit(2);
    }
    return p;
}

/* Copy `bytes` of device memory to the output file. */
static void dump(FILE* f, const void* d, size_t bytes) {
    void* h = host_alloc(bytes);
    if (bytes) HIP_CHECK(hipMemcpy(h, d, bytes, hipMemcpyDeviceToHost));
    if (bytes && fwrite(h, 1, bytes, f) != bytes) {
        fprintf(stderr, "short write\n");
        exit(2);
    }
    free(h);
}

int main(int argc, char** argv) {
    if (argc != 6) {
        fprintf(stderr, "usage: %s IN OUT BUDGET MODE QUOTA\n", argv[0]);
        return 2;
    }
    const int64_t budget = strtoll(argv[3], NULL, 10);
    const int32_t mode = (int32_t)strtol(argv[4], NULL, 10);
    const int64_t quota = strtoll(argv[5], NULL, 10);

    FILE* in = fopen(argv[1], "rb");
    if (!in) {
        fprintf(stderr, "cannot open %s\n", argv[1]);
        return 2;
    }
    int64_t hdr[3];
    read_exact(in, hdr, sizeof hdr);
    const int64_t W = hdr[0], n = hdr[1], T = hdr[2];
    int64_t* rank_off = host_alloc(sizeof(int64_t) * (size_t)(W + 1));
    int64_t* tok_off = host_alloc(sizeof(int64_t) * (size_t)(n + 1));
    int32_t* tokens = host_alloc(sizeof(int32_t) * (size_t)T);
    read_exact(in, rank_off, sizeof(int64_t) * (size_t)(W + 1));
    read_exact(in, tok_off, sizeof(int64_t) * (size_t)(n + 1));
    read_exact(in, tokens, sizeof(int32_t) * (size_t)T);
    fclose(in);

    int64_t* d_tok_off = dev_alloc(sizeof(int64_t) * (size_t)(n + 1));
    int32_t* d_tokens = dev_alloc(sizeof(int32_t) * (size_t)T);
    HIP_CHECK(hipMemcpy(d_tok_off, tok_off, sizeof(int64_t) * (size_t)(n + 1), hipMemcpyHostToDevice));
    if (T) HIP_CHECK(hipMemcpy(d_tokens, tokens, sizeof(int32_t) * (size_t)T, hipMemcpyHostToDevice));

    odb_window_t w;
    memset(&w, 0, sizeof w);
    w.num_ranks = (int32_t)W;
    w.num_samples = n;
    w.rank_offsets = rank_off;
    w.d_token_offsets = d_tok_off;
    w.d_tokens = d_tokens;
    w.d_identity = NULL;
    w.num_identities = 0;

    const size_t ws_bytes = odb_workspace_size(&w);
    if (ws_bytes == 0) return fail("odb_workspace_size", ODB_E_INVALID_ARG);
    void* d_ws = dev_alloc(ws_bytes);
    hipStream_t stream;
    HIP_CHECK(hipStreamCreate(&stream));

    /* stage 1 */
    int32_t* d_order = dev_alloc(sizeof(int32_t) * (size_t)n);
    int32_t* d_sorted_len = dev_alloc(sizeof(int32_t) * (size_t)n);
    int32_t* d_group_index = dev_alloc(sizeof(int32_t) * (size_t)n);
    int32_t* d_groups = dev_alloc(sizeof(int32_t) * (size_t)W);
    int st = odb_form_groups(&w, budget, d_order, d_sorted_len, d_group_index, d_groups, d_ws, ws_bytes, stream);
    if (st != ODB_OK) return fail("odb_form_groups", st);

    /* stages 2-3: start with room for one step per rank, take the capacity the plan
       reports and call again */
    odb_align_params_t params;
    memset(&params, 0, sizeof params);
    params.mode = mode;
    params.quota = quota;
    params.slot_capacity = NULL;
    int32_t* d_emit = dev_alloc(sizeof(int32_t) * (size_t)n);
    int64_t* d_row_ts = dev_alloc(sizeof(int64_t) * (size_t)n);
    int32_t* d_row_len = dev_alloc(sizeof(int32_t) * (size_t)n);
    int32_t* d_leftover = dev_alloc(sizeof(int32_t) * (size_t)n);
    int64_t* d_leftover_off = dev_alloc(sizeof(int64_t) * (size_t)(W + 1));
    int64_t cap = W;
    int64_t retries = 0;
    odb_plan_info_t info;
    int32_t *d_rows = NULL, *d_maxlen = NULL;
    int64_t *d_row_off = NULL, *d_tile_off = NULL, *d_slot_tok = NULL;
    for (;;) {
        d_rows = dev_alloc(sizeof(int32_t) * (size_t)cap);
        d_maxlen = dev_alloc(sizeof(int32_t) * (size_t)cap);
        d_row_off = dev_alloc(sizeof(int64_t) * (size_t)(cap + 1));
        d_tile_off = dev_alloc(sizeof(int64_t) * (size_t)(cap + 1));
        d_slot_tok = dev_alloc(sizeof(int64_t) * (size_t)cap);
        st = odb_align_groups(&w, budget, &params, d_order, d_sorted_len, d_group_index, d_groups, cap, d_emit,
                              d_row_ts, d_row_len, d_rows, d_maxlen, d_row_off, d_tile_off, d_slot_tok, NULL,
                              d_leftover, d_leftover_off, &info, d_ws, ws_bytes, stream);
        if (st != ODB_E_CAPACITY || retries > 0) break;
        cap = info.required_slot_capacity;
        retries += 1;
        HIP_CHECK(hipFree(d_rows));
        HIP_CHECK(hipFree(d_maxlen));
        HIP_CHECK(hipFree(d_row_off));
        HIP_CHECK(hipFree(d_tile_off));
        HIP_CHECK(hipFree(d_slot_tok));
        /* the stage-1 outputs are unchanged: the alignment reads them again */
    }
    if (st != ODB_OK) return fail("odb_align_groups", st);
    const int64_t K = W * info.steps;
    const int64_t P = info.padded_elems;

    /* stage 4 */
    int32_t* d_out[4];
    for (int i = 0; i < 4; ++i) d_out[i] = dev_alloc(sizeof(int32_t) * (size_t)P);
    st = odb_collate(&w, K, d_emit, d_row_ts, d_row_len, d_rows, d_maxlen, d_row_off, d_tile_off, 0, P, d_out[0],
                     d_out[1], d_out[2], d_out[3], d_ws, ws_bytes, stream);
    if (st != ODB_OK) return fail("odb_collate", st);
    st = odb_collate_status(d_ws, ws_bytes, stream);
    if (st != ODB_OK) return fail("odb_collate_status", st);
    /* the allocation-free variant, same plan, its own outputs and status word */
    int32_t* d_static_out[4];
    for (int i = 0; i < 4; ++i) d_static_out[i] = dev_alloc(sizeof(int32_t) * (size_t)P);
    int32_t* d_static_status = dev_alloc(sizeof(int32_t));
    st = odb_collate_static(&w, K, d_emit, d_row_ts, d_row_len, d_rows, d_maxlen, d_row_off, d_tile_off, 0, P,
                            d_static_out[0], d_static_out[1], d_static_out[2], d_static_out[3], d_static_status,
                            stream);
    if (st != ODB_OK) return fail("odb_collate_static", st);

    /* exact token-level loss-scaling weights (Eq. 2) */
    double* d_weight = dev_alloc(sizeof(double) * (size_t)K);
    st = odb_loss_weights((int32_t)W, info.steps, ODB_WEIGHT_TOKEN_EXACT, d_rows, d_slot_tok, NULL, d_weight, NULL,
                          NULL, stream);
    if (st != ODB_OK) return fail("odb_loss_weights", st);
    HIP_CHECK(hipStreamSynchronize(stream));
    /* the return-on-investment screen over every sample of the window */
    odb_length_sketch_t sk;
    st = odb_length_sketch(&w, NULL, n, budget, &sk, d_ws, ws_bytes, stream);
    if (st != ODB_OK) return fail("odb_length_sketch", st);
    /* the identity-coverage self-check on its own, over the plan's emitted and left-over ids */
    odb_plan_info_t cov;
    memset(&cov, 0, sizeof cov);
    st = odb_check_coverage(&w, d_emit, info.emitted_samples, d_leftover, info.leftover_samples, &cov, d_ws, ws_bytes,
                            stream);
    if (st != ODB_OK) return fail("odb_check_coverage", st);

    FILE* out = fopen(argv[2], "wb");
    if (!out) {
        fprintf(stderr, "cannot open %s\n", argv[2]);
        return 2;
    }
    const int64_t fields[15] = {info.steps, info.rounds, info.stop_reason, info.emitted_samples,
                                info.leftover_samples, info.real_tokens, info.padded_elems,
                                info.max_step_samples, info.splits, info.overflow_groups, info.missing_ids,
                                info.duplicate_ids, info.bad_views, info.second_gather_rounds,
                                info.required_slot_capacity};
    if (fwrite(fields, sizeof fields, 1, out) != 1 || fwrite(&info.pad_fraction, sizeof(double), 1, out) != 1 ||
        fwrite(&retries, sizeof retries, 1, out) != 1) {
        fprintf(stderr, "short write\n");
        return 2;
    }
    dump(out, d_order, sizeof(int32_t) * (size_t)n);
    dump(out, d_sorted_len, sizeof(int32_t) * (size_t)n);
    dump(out, d_group_index, sizeof(int32_t) * (size_t)n);
    dump(out, d_groups, sizeof(int32_t) * (size_t)W);
    dump(out, d_emit, sizeof(int32_t) * (size_t)info.emitted_samples);
    dump(out, d_rows, sizeof(int32_t) * (size_t)K);
    dump(out, d_maxlen, sizeof(int32_t) * (size_t)K);
    dump(out, d_row_off, sizeof(int64_t) * (size_t)(K + 1));
    dump(out, d_tile_off, sizeof(int64_t) * (size_t)(K + 1));
    dump(out, d_slot_tok, sizeof(int64_t) * (size_t)K);
    dump(out, d_leftover, sizeof(int32_t) * (size_t)info.leftover_samples);
    dump(out, d_leftover_off, sizeof(int64_t) * (size_t)(W + 1));
    for (int i = 0; i < 4; ++i) dump(out, d_out[i], sizeof(int32_t) * (size_t)P);
    for (int i = 0; i < 4; ++i) dump(out, d_static_out[i], sizeof(int32_t) * (size_t)P);
    dump(out, d_static_status, sizeof(int32_t));
    dump(out, d_weight, sizeof(double) * (size_t)K);
    const int64_t sk_int[7] = {sk.samples, sk.short_samples, sk.sum_len, (int64_t)sk.sum_sq_hi, (int64_t)sk.sum_sq_lo,
                               sk.min_len, sk.max_len};
    const double sk_real[3] = {sk.mean, sk.cv, sk.short_fraction};
    const int64_t sk_roi = sk.high_roi;
    if (fwrite(sk_int, sizeof sk_int, 1, out) != 1 || fwrite(sk_real, sizeof sk_real, 1, out) != 1 ||
        fwrite(&sk_roi, sizeof sk_roi, 1, out) != 1) {
        fprintf(stderr, "short write\n");
        return 2;
    }
    const int64_t cov_out[3] = {cov.bad_views, cov.missing_ids, cov.duplicate_ids};
    if (fwrite(cov_out, sizeof cov_out, 1, out) != 1) {
        fprintf(stderr, "short write\n");
        return 2;
    }
    fclose(out);

    void* bufs[] = {d_tok_off, d_tokens, d_ws, d_order, d_sorted_len, d_group_index, d_groups, d_emit, d_row_ts,
                    d_row_len, d_leftover, d_leftover_off, d_rows, d_maxlen, d_row_off, d_tile_off, d_slot_tok,
                    d_out[0], d_out[1], d_out[2], d_out[3], d_weight, d_static_out[0], d_static_out[1],
                    d_static_out[2], d_static_out[3], d_static_status};
    for (size_t i = 0; i < sizeof bufs / sizeof bufs[0]; ++i) HIP_CHECK(hipFree(bufs[i]));
    HIP_CHECK(hipStreamDestroy(stream));
    free(rank_off);
    free(tok_off);
    free(tokens);
    return 0;
}
