/*
 * One logical iteration of the streaming protocol driven from plain C through
 * include/odb.h: odb_stream_workspace_size + odb_stream_plan (retried once with the slot
 * capacity the first call reports) -> odb_collate -> odb_loss_weights, every output
 * written to a file for the test to compare with the oracle.
 *
 *   stream_pipeline IN OUT BUDGET MODE QUOTA BUFFER DEPTH MAX_ROUNDS
 *
 * IN (little-endian): int64 W, N, T; int64 token_offsets[N+1]; int32 tokens[T];
 * int32 perm[N]; int32 rate[W].
 * OUT: int64 info[20] (steps, rounds, emit_rounds, skip_rounds, stop_reason, views,
 * emitted_views, undelivered_views, pending_views, real_tokens, padded_elems,
 * max_step_samples, splits, overflow_groups, missing_ids, duplicate_ids, bad_views,
 * second_gather_rounds, max_outstanding, required_slot_capacity), double pad_fraction,
 * int64 capacity_retries; int64 trace[rounds][4] (kind, target, emitted, phi);
 * int32 emit_views[E], emit_order[E]; int64 row_token_start[E]; int32 row_len[E];
 * int32 slot_rows[K], slot_maxlen[K]; int64 slot_row_off[K+1], slot_tile_off[K+1],
 * slot_tokens[K]; int32 left_views[M-E]; int64 left_off[W+1]; int32 input_ids[P],
 * labels[P], attention_mask[P], position_ids[P]; double weight[K] (exact token-level
 * mode), with E = emitted_views, M = views, K = W * steps and P = padded_elems.
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

static void* host_alloc(size_t bytes) {
    void* p = malloc(bytes ? bytes : 16);
    if (!p) {
        fprintf(stderr, "out of host memory\n");
        exit(2);
    }
    return p;
}

static void read_exact(FILE* f, void* dst, size_t bytes) {
    if (bytes && fread(dst, 1, bytes, f) != bytes) {
        fprintf(stderr, "short input file\n");
        exit(2);
    }
}

static void write_exact(FILE* f, const void* src, size_t bytes) {
    if (bytes && fwrite(src, 1, bytes, f) != bytes) {
        fprintf(stderr, "short write\n");
        exit(2);
    }
}

/* Copy `bytes` of device memory to the output file. */
static void dump(FILE* f, const void* d, size_t bytes) {
    void* h = host_alloc(bytes);
    if (bytes) HIP_CHECK(hipMemcpy(h, d, bytes, hipMemcpyDeviceToHost));
    write_exact(f, h, bytes);
    free(h);
}

/* The slot arrays of one capacity. */
typedef struct slots {
    int32_t* rows;
    int32_t* maxlen;
    int64_t* row_off;
    int64_t* tile_off;
    int64_t* tokens;
} slots_t;

static slots_t slots_alloc(int64_t cap) {
    slots_t s;
    s.rows = dev_alloc(sizeof(int32_t) * (size_t)cap);
    s.maxlen = dev_alloc(sizeof(int32_t) * (size_t)cap);
    s.row_off = dev_alloc(sizeof(int64_t) * (size_t)(cap + 1));
    s.tile_off = dev_alloc(sizeof(int64_t) * (size_t)(cap + 1));
    s.tokens = dev_alloc(sizeof(int64_t) * (size_t)cap);
    return s;
}

static void slots_free(slots_t s) {
    HIP_CHECK(hipFree(s.rows));
    HIP_CHECK(hipFree(s.maxlen));
    HIP_CHECK(hipFree(s.row_off));
    HIP_CHECK(hipFree(s.tile_off));
    HIP_CHECK(hipFree(s.tokens));
}

int main(int argc, char** argv) {
    if (argc != 9) {
        fprintf(stderr, "usage: %s IN OUT BUDGET MODE QUOTA BUFFER DEPTH MAX_ROUNDS\n", argv[0]);
        return 2;
    }
    const int64_t budget = strtoll(argv[3], NULL, 10);
    const int32_t mode = (int32_t)strtol(argv[4], NULL, 10);
    const int64_t quota = strtoll(argv[5], NULL, 10);
    const int32_t buffer_size = (int32_t)strtol(argv[6], NULL, 10);
    const int32_t depth = (int32_t)strtol(argv[7], NULL, 10);
    const int64_t max_rounds = strtoll(argv[8], NULL, 10);

    FILE* in = fopen(argv[1], "rb");
    if (!in) {
        fprintf(stderr, "cannot open %s\n", argv[1]);
        return 2;
    }
    int64_t hdr[3];
    read_exact(in, hdr, sizeof hdr);
    const int64_t W = hdr[0], N = hdr[1], T = hdr[2];
    int64_t* tok_off = host_alloc(sizeof(int64_t) * (size_t)(N + 1));
    int32_t* tokens = host_alloc(sizeof(int32_t) * (size_t)T);
    int32_t* perm = host_alloc(sizeof(int32_t) * (size_t)N);
    int32_t* rate = host_alloc(sizeof(int32_t) * (size_t)W);
    read_exact(in, tok_off, sizeof(int64_t) * (size_t)(N + 1));
    read_exact(in, tokens, sizeof(int32_t) * (size_t)T);
    read_exact(in, perm, sizeof(int32_t) * (size_t)N);
    read_exact(in, rate, sizeof(int32_t) * (size_t)W);
    fclose(in);

    /* the streaming loop does not use the window's rank split; any valid one will do */
    int64_t* rank_off = host_alloc(sizeof(int64_t) * (size_t)(W + 1));
    for (int64_t r = 0; r <= W; ++r) rank_off[r] = r * N / W;

    int64_t* d_tok_off = dev_alloc(sizeof(int64_t) * (size_t)(N + 1));
    int32_t* d_tokens = dev_alloc(sizeof(int32_t) * (size_t)T);
    int32_t* d_perm = dev_alloc(sizeof(int32_t) * (size_t)N);
    HIP_CHECK(hipMemcpy(d_tok_off, tok_off, sizeof(int64_t) * (size_t)(N + 1), hipMemcpyHostToDevice));
    if (T) HIP_CHECK(hipMemcpy(d_tokens, tokens, sizeof(int32_t) * (size_t)T, hipMemcpyHostToDevice));
    if (N) HIP_CHECK(hipMemcpy(d_perm, perm, sizeof(int32_t) * (size_t)N, hipMemcpyHostToDevice));

    odb_window_t w;
    memset(&w, 0, sizeof w);
    w.num_ranks = (int32_t)W;
    w.num_samples = N;
    w.rank_offsets = rank_off;
    w.d_token_offsets = d_tok_off;
    w.d_tokens = d_tokens;

    odb_stream_params_t params;
    memset(&params, 0, sizeof params);
    params.mode = mode;
    params.buffer_size = buffer_size;
    params.depth = depth;
    params.quota = quota;
    params.rate = rate;
    params.slot_capacity = NULL;
    params.max_rounds = max_rounds;

    const int64_t M = W * ((N + W - 1) / W);
    int32_t* d_emit_order = dev_alloc(sizeof(int32_t) * (size_t)M);
    int32_t* d_emit_views = dev_alloc(sizeof(int32_t) * (size_t)M);
    int64_t* d_row_ts = dev_alloc(sizeof(int64_t) * (size_t)M);
    int32_t* d_row_len = dev_alloc(sizeof(int32_t) * (size_t)M);
    int32_t* d_left_views = dev_alloc(sizeof(int32_t) * (size_t)M);
    int64_t* d_left_off = dev_alloc(sizeof(int64_t) * (size_t)(W + 1));
    odb_stream_round_t* trace = host_alloc(sizeof(odb_stream_round_t) * (size_t)max_rounds);

    /* room for one step per rank first, then the capacity the iteration reports; the
       workspace size depends on the slot capacity */
    int64_t cap = W, retries = 0;
    odb_stream_info_t info;
    slots_t sl;
    void* d_ws = NULL;
    size_t ws_bytes = 0;
    int st;
    for (;;) {
        ws_bytes = odb_stream_workspace_size(&w, depth, cap, max_rounds);
        if (ws_bytes == 0) return fail("odb_stream_workspace_size", ODB_E_INVALID_ARG);
        d_ws = dev_alloc(ws_bytes);
        sl = slots_alloc(cap);
        st = odb_stream_plan(&w, d_perm, budget, &params, cap, d_emit_order, d_emit_views, d_row_ts, d_row_len,
                             sl.rows, sl.maxlen, sl.row_off, sl.tile_off, sl.tokens, NULL, d_left_views, d_left_off,
                             trace, &info, d_ws, ws_bytes, NULL);
        if (st != ODB_E_CAPACITY || retries > 0 || info.required_slot_capacity <= cap) break;
        cap = info.required_slot_capacity;
        retries += 1;
        slots_free(sl);
        HIP_CHECK(hipFree(d_ws));
    }
    if (st != ODB_OK) return fail("odb_stream_plan", st);
    const int64_t K = W * info.steps;
    const int64_t P = info.padded_elems;
    const int64_t E = info.emitted_views;

    int32_t* d_out[4];
    for (int i = 0; i < 4; ++i) d_out[i] = dev_alloc(sizeof(int32_t) * (size_t)P);
    st = odb_collate(&w, K, d_emit_order, d_row_ts, d_row_len, sl.rows, sl.maxlen, sl.row_off, sl.tile_off, 0, P,
                     d_out[0], d_out[1], d_out[2], d_out[3], d_ws, ws_bytes, NULL);
    if (st != ODB_OK) return fail("odb_collate", st);
    st = odb_collate_status(d_ws, ws_bytes, NULL);
    if (st != ODB_OK) return fail("odb_collate_status", st);
    double* d_weight = dev_alloc(sizeof(double) * (size_t)K);
    st = odb_loss_weights((int32_t)W, info.steps, ODB_WEIGHT_TOKEN_EXACT, sl.rows, sl.tokens, NULL, d_weight, NULL,
                          NULL, NULL);
    if (st != ODB_OK) return fail("odb_loss_weights", st);
    HIP_CHECK(hipDeviceSynchronize());

    FILE* out = fopen(argv[2], "wb");
    if (!out) {
        fprintf(stderr, "cannot open %s\n", argv[2]);
        return 2;
    }
    const int64_t fields[20] = {info.steps, info.rounds, info.emit_rounds, info.skip_rounds, info.stop_reason,
                                info.views, info.emitted_views, info.undelivered_views, info.pending_views,
                                info.real_tokens, info.padded_elems, info.max_step_samples, info.splits,
                                info.overflow_groups, info.missing_ids, info.duplicate_ids, info.bad_views,
                                info.second_gather_rounds, info.max_outstanding, info.required_slot_capacity};
    write_exact(out, fields, sizeof fields);
    write_exact(out, &info.pad_fraction, sizeof(double));
    write_exact(out, &retries, sizeof retries);
    for (int64_t i = 0; i < info.rounds; ++i) {
        const int64_t rec[4] = {trace[i].kind, trace[i].target, trace[i].emitted, trace[i].phi};
        write_exact(out, rec, sizeof rec);
    }
    dump(out, d_emit_views, sizeof(int32_t) * (size_t)E);
    dump(out, d_emit_order, sizeof(int32_t) * (size_t)E);
    dump(out, d_row_ts, sizeof(int64_t) * (size_t)E);
    dump(out, d_row_len, sizeof(int32_t) * (size_t)E);
    dump(out, sl.rows, sizeof(int32_t) * (size_t)K);
    dump(out, sl.maxlen, sizeof(int32_t) * (size_t)K);
    dump(out, sl.row_off, sizeof(int64_t) * (size_t)(K + 1));
    dump(out, sl.tile_off, sizeof(int64_t) * (size_t)(K + 1));
    dump(out, sl.tokens, sizeof(int64_t) * (size_t)K);
    dump(out, d_left_views, sizeof(int32_t) * (size_t)(M - E));
    dump(out, d_left_off, sizeof(int64_t) * (size_t)(W + 1));
    for (int i = 0; i < 4; ++i) dump(out, d_out[i], sizeof(int32_t) * (size_t)P);
    dump(out, d_weight, sizeof(double) * (size_t)K);
    fclose(out);

    slots_free(sl);
    void* bufs[] = {d_tok_off, d_tokens, d_perm, d_emit_order, d_emit_views, d_row_ts, d_row_len, d_left_views,
                    d_left_off, d_ws, d_out[0], d_out[1], d_out[2], d_out[3], d_weight};
    for (size_t i = 0; i < sizeof bufs / sizeof bufs[0]; ++i) HIP_CHECK(hipFree(bufs[i]));
    free(tok_off);
    free(tokens);
    free(perm);
    free(rate);
    free(rank_off);
    free(trace);
    return 0;
}
