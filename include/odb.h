/*
 * odb.h -- C ABI of the MI355X (gfx950) Online Dynamic Batching window pipeline.
 *
 * One call sequence turns a window of realised samples, split over W simulated DDP
 * ranks, into step-aligned, padded training tiles:
 *
 *   odb_form_groups   length-aware grouping of every rank's buffer      (Sec. 2.2, Eq. 1)
 *   odb_align_groups  Distributed Group Alignment: target, split,       (Eq. 3, Algorithm 1,
 *                     overflow recirculation, join / non-join quota      Sec. 2.3, Thm 1-2)
 *                     termination, slot plan, stats, identity coverage  (App. C)
 *   odb_collate       pad every aligned group to its own longest sample (Sec. 2.1, Fig. 1)
 *   odb_loss_weights  per-step, per-rank loss-scaling weights          (Eq. 2, App. B)
 *   odb_length_sketch CV and short-sample fraction of sketched lengths  (Sec. 1, practical
 *                     (return-on-investment screen)                      guidance section)
 *   odb_stream_plan   the unified streaming loop: one logical sampler    (Sec. 2.3, App. C,
 *                     iteration, round by round (fetch, skip, emit,       App. E)
 *                     stop), into the same plan layout
 *
 * Conventions shared by every entry point
 *   - Pointers named d_* are device pointers (HIP global memory on the current device);
 *     all other pointers are host pointers.  The caller owns every buffer; the library
 *     allocates no device memory (scratch comes from the caller's workspace), keeps no
 *     pointer after returning and holds no state except a thread-local error message and
 *     the fixed per-device scratch array of odb_collate_static.
 *   - `stream` is a hipStream_t (NULL = the legacy default stream).  Work is enqueued
 *     on it in order.  odb_align_groups synchronises `stream` because its output sizes
 *     are data dependent; odb_form_groups does so only on its multi-block path (ranks of
 *     more than 16,384 samples, or budgets of millions); odb_collate does not.
 *   - Every call returns an odb_status_t.  Argument errors are detected on the host
 *     before anything is launched.  Data errors found on the device are reported at the
 *     call's synchronisation point.  On any error the outputs are unspecified.  No C++
 *     exception crosses this interface.
 *   - Calls on distinct streams with distinct workspaces may run concurrently.
 *
 * Window layout (odb_window_t)
 *   Samples are numbered 0..n-1; that number is the sample id used in every output.
 *   Rank r owns the contiguous id range [rank_offsets[r], rank_offsets[r+1]).  Sample i
 *   has realised length l_i = d_token_offsets[i+1] - d_token_offsets[i] and its tokens
 *   are d_tokens[d_token_offsets[i] .. d_token_offsets[i+1]).
 */
#ifndef ODB_H_
#define ODB_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum odb_status {
    ODB_OK = 0,
    ODB_E_INVALID_ARG = 1,   /* bad argument, detected on the host                      */
    ODB_E_INVALID_DATA = 2,  /* bad window contents (l < 1, l >= 2^31, bad plan arrays)  */
    ODB_E_WORKSPACE = 3,     /* workspace smaller than odb_workspace_size()              */
    ODB_E_CAPACITY = 4,      /* slot arrays too small; see required_slot_capacity        */
    ODB_E_HIP = 5,           /* a HIP runtime call failed                                */
    ODB_E_COVERAGE = 6,      /* coverage self-check failed: some view not emitted once   */
    ODB_E_INTERNAL = 7
} odb_status_t;

typedef enum odb_mode {
    ODB_MODE_JOIN = 0,           /* default: drain every buffer, each view emitted once (Thm 1) */
    ODB_MODE_NONJOIN_QUOTA = 1   /* stop at the first step reaching the sample quota (Thm 2)   */
} odb_mode_t;

typedef enum odb_stop_reason {
    ODB_STOP_DRAINED = 0,        /* every rank's buffer emptied                               */
    ODB_STOP_QUOTA = 1,          /* non-join: cumulative emitted samples reached the quota    */
    ODB_STOP_RANK_FINISHED = 2   /* non-join: a rank ran empty while others still had samples */
} odb_stop_reason_t;

/* A window of realised samples over W simulated DDP ranks. */
typedef struct odb_window {
    int32_t num_ranks;               /* W >= 1                                              */
    int32_t reserved0;               /* must be 0                                           */
    int64_t num_samples;             /* n, 0 <= n < 2^31 - 1                                */
    const int64_t* rank_offsets;     /* HOST [W+1]; 0 = off[0] <= ... <= off[W] = n          */
    const int64_t* d_token_offsets;  /* [n+1]; l_i = off[i+1] - off[i] must lie in [1, 2^31) */
    const int32_t* d_tokens;         /* token stream addressed by d_token_offsets            */
    const int64_t* d_identity;       /* [n] dataset identity of every sampler view, or NULL  */
    int64_t num_identities;          /* identities lie in [0, num_identities) (NULL map: n)  */
} odb_window_t;

/* Human-readable name of a status code (static storage). */
const char* odb_status_string(int status);

/* Detail of the last failing call on this thread ("" if none). */
const char* odb_last_error_message(void);

/* Bytes of device workspace that odb_form_groups / odb_align_groups / odb_collate need
 * for this window (the same workspace serves all three).  Returns 0 on a bad window. */
size_t odb_workspace_size(const odb_window_t* w);

/*
 * Stage 1: length-aware grouping (Sec. 2.2; batch size rule Eq. 1; App. D example).
 *
 * Every rank's samples are ordered by realised length, longest first, equal lengths by
 * ascending sample id ("formation order").  Walking that order with a running threshold
 * t (initially 1), a group is closed as soon as it holds t samples and t becomes
 * B(l) = max(floor(budget / l), 1) of the sample just added; samples left over at the
 * end of the buffer form one last group.
 *
 *   budget              L_max >= 1, padded-token budget of a group
 *   d_order             [n] out: formation order, rank segments in place (global sample ids)
 *   d_sorted_len        [n] out: l of d_order[p]
 *   d_group_index       [n] out: 0-based formation group index of position p within its rank
 *   d_groups_per_rank   [W] out: G_r, groups formed by rank r
 *   d_ws / ws_bytes     workspace of at least odb_workspace_size(w) bytes, 256-B aligned
 *
 * Two paths, equal results:
 *   - every rank holds at most 16,384 samples and its distinct batch sizes fit a
 *     3,840-entry table (budget < 3,682,561, or ranks of at most 3,840 samples): one block
 *     per rank sorts and walks its samples; two kernels, asynchronous.  A sample whose
 *     length lies outside [1, 2^31), or whose token offset is negative, is grouped as if
 *     its length were 1, and odb_align_groups on these outputs returns ODB_E_INVALID_DATA
 *     naming the first such sample.
 *   - otherwise a multi-block radix sort and run walk (or pointer jumping for budgets
 *     whose batch sizes may exceed the table); this path synchronises `stream` once, to
 *     size its radix passes from the window's length range, and returns
 *     ODB_E_INVALID_DATA itself for such a sample (message names the first one).
 */
int odb_form_groups(const odb_window_t* w, int64_t budget,
                    int32_t* d_order, int32_t* d_sorted_len, int32_t* d_group_index,
                    int32_t* d_groups_per_rank, void* d_ws, size_t ws_bytes, void* stream);

/* Alignment parameters. */
typedef struct odb_align_params {
    int32_t mode;                    /* odb_mode_t                                          */
    int32_t reserved0;               /* must be 0                                           */
    int64_t quota;                   /* sample quota Q >= 1 (non-join only)                 */
    const int64_t* slot_capacity;    /* HOST [W] output-slot capacity C_r >= 0 per round, or
                                        NULL (no limit); C_r = 0 takes no part in the minimum */
} odb_align_params_t;

/* Summary of an aligned plan. */
typedef struct odb_plan_info {
    int64_t steps;                   /* S: aligned steps (slots per rank)                   */
    int32_t rounds;                  /* alignment rounds run                                */
    int32_t stop_reason;             /* odb_stop_reason_t                                   */
    int64_t emitted_samples;         /* sum of rows over all slots                          */
    int64_t leftover_samples;        /* samples not emitted (non-join only)                 */
    int64_t real_tokens;             /* sum of l over emitted samples                       */
    int64_t padded_elems;            /* sum of rows * maxlen over all slots                 */
    int64_t max_step_samples;        /* S_max: largest global sample count of one step      */
    int64_t splits;                  /* singletons extracted by split, all rounds           */
    int64_t overflow_groups;         /* groups returned by overflow, all rounds             */
    int64_t missing_ids;             /* identities in [0, N_id) neither emitted nor leftover */
    int64_t duplicate_ids;           /* extra emissions of an identity beyond its first     */
    int64_t bad_views;               /* sampler views not emitted/leftover exactly once     */
    double  pad_fraction;            /* 1 - real_tokens / padded_elems (0 if nothing padded) */
    int64_t required_slot_capacity;  /* W * S; set on ODB_E_CAPACITY and on success         */
    int64_t second_gather_rounds;    /* rounds in which some active rank had G_r != T, i.e.
                                        rounds whose pre-alignment counts are not the
                                        post-alignment ones, so exact token-level loss
                                        scaling needs a second exchange (App. B)             */
} odb_plan_info_t;

/*
 * Stages 2-3: Distributed Group Alignment (Eq. 3, Algorithm 1, Sec. 2.3) + coverage (App. C).
 *
 * Inputs are the outputs of odb_form_groups for the same window and budget.  Each
 * round gathers every rank's group count G_r and buffered count S_r (the simulated
 * all_gather), computes T = max(min(max_{G_r>0} G_r, C+_min, S+_min), 1) over the active
 * ranks, splits (peels the longest member of the first multi-sample group, counting from
 * the longest group, into a singleton until G_r = T) or overflows (keeps the T largest
 * groups, ties to the shorter samples, and returns the rest to the buffer).  Join mode
 * repeats rounds on the returned samples until every buffer is empty; ranks with an
 * empty buffer receive IDLE slots (rows = 0).  Non-join mode stops at the first step
 * whose cumulative global emitted count reaches `quota`, or at the start of a round in
 * which some rank is empty while others are not; un-emitted samples become leftovers.
 *
 * Output layout.  Slot k = r * S + j is rank r's j-th aligned step (rank-major).  A rank's
 * groups are emitted short to long and each group's rows run short to long (the reverse
 * of formation order).  Tiles are packed back to back in slot order.
 *   slot_capacity     capacity of the slot arrays in slots; >= W * S is required
 *   d_emit_order      [n] out: emitted ids; slot k's rows are
 *                     d_emit_order[d_slot_row_off[k] .. d_slot_row_off[k+1])
 *   d_row_token_start [n] out, or NULL (then d_row_len must be NULL too): row records,
 *   d_row_len         [n] out   parallel to d_emit_order: d_token_offsets[s] and l_s of
 *                     the row's sample s.  odb_collate reads them instead of gathering
 *                     the CSR offsets of the emitted ids itself.
 *   d_slot_rows       [slot_capacity] out: rows of slot k (0 = IDLE)
 *   d_slot_maxlen     [slot_capacity] out: longest l in slot k (0 = IDLE)
 *   d_slot_row_off    [slot_capacity+1] out: exclusive prefix sum of rows
 *   d_slot_tile_off   [slot_capacity+1] out: exclusive prefix sum of rows * maxlen
 *   d_slot_tokens     [slot_capacity] out: real tokens of slot k
 *   d_slot_tokens_approx [slot_capacity] out, or NULL: approximate token count of slot k
 *                     for approximate token-level loss scaling (App. B): rows of the slot
 *                     times the mean length of its rank's buffer at the start of the
 *                     slot's alignment round (fp64, rows * (tokens / samples), each
 *                     operation rounded to nearest); 0 for IDLE slots
 *   d_leftover        [n] out: un-emitted ids of every rank in formation order, rank-major
 *   d_leftover_off    [W+1] out: rank r's leftovers are [off[r], off[r+1])
 *   h_info            host out: plan summary (always filled when the plan was built)
 *
 * Synchronises `stream` once per alignment round and once at the end: twice for windows
 * that align in one round (every rank buffering the same number of samples, no capacity
 * limit, as in all of the benchmark windows), each time with one device-to-host copy.
 * Returns
 * ODB_E_CAPACITY (with h_info->required_slot_capacity) if slot_capacity < W * S,
 * ODB_E_INVALID_DATA if a sample's CSR length lies outside [1, 2^31) or its token offset
 * is negative (the message names the first such sample), or if the stage-1 arrays are
 * inconsistent (an order that is not each
 * rank's ids by (length desc, id asc), a group index that does not step by 0 or 1, a
 * sorted length < 1 or different from the sample's CSR length; the last is checked
 * once the plan is built, against every emitted and left-over sample), and
 * ODB_E_COVERAGE if the coverage self-check finds a view that is not emitted (or left
 * over) exactly once.
 */
int odb_align_groups(const odb_window_t* w, int64_t budget, const odb_align_params_t* params,
                     const int32_t* d_order, const int32_t* d_sorted_len,
                     const int32_t* d_group_index, const int32_t* d_groups_per_rank,
                     int64_t slot_capacity,
                     int32_t* d_emit_order, int64_t* d_row_token_start, int32_t* d_row_len,
                     int32_t* d_slot_rows, int32_t* d_slot_maxlen,
                     int64_t* d_slot_row_off, int64_t* d_slot_tile_off, int64_t* d_slot_tokens,
                     double* d_slot_tokens_approx, int32_t* d_leftover, int64_t* d_leftover_off,
                     odb_plan_info_t* h_info, void* d_ws, size_t ws_bytes, void* stream);

/*
 * Stage 4: padded collation (Sec. 2.1 and Fig. 1: each aligned group is padded to its
 * own longest sample).
 *
 * Writes four flat int32 arrays of length tile_off[num_slots] (= padded_elems).  Slot
 * k's tile is elements [tile_off[k], tile_off[k+1]) viewed row-major as
 * [rows[k], maxlen[k]].  Element (i, c) of a tile whose row i holds sample s:
 *   c <  l_s : input_ids = labels = token c of s, attention_mask = 1, position_ids = c
 *   c >= l_s : input_ids = pad_id, labels = -100, attention_mask = 0, position_ids = 0
 *
 *   num_slots           W * S from odb_align_groups or odb_stream_plan (>= 0)
 *   plan arrays         as written by odb_align_groups or odb_stream_plan (device); the
 *                       emitted rows number at most n + W - 1 (sampler padding views)
 *   d_row_token_start,  the plan's row records (token start and length of each emitted
 *   d_row_len           row), or both NULL: then the rows' samples are read from
 *                       d_emit_order and their CSR offsets gathered here (one more
 *                       kernel, one random 16-byte read per row); with row records
 *                       d_emit_order is not read and may be NULL
 *   out_capacity_elems  length of each output array; elements beyond it are not written
 *   d_ws / ws_bytes     the workspace: a status word, the counter from which the kernel's
 *                       blocks take runs of steps, and the gathered row records when none
 *                       are passed; two collates in flight at once need two workspaces
 *
 * Asynchronous (a clear of the counter and the status word, and one kernel with row
 * records, one kernel more without).  Accesses are bounds-checked against the window
 * and the plan: a row record outside the token stream or longer than its tile, or an
 * emitted id outside [0, n), sets the workspace's collate status word (such a row is
 * written as padding).  Each odb_collate clears that word when it starts; no other
 * entry point touches it, so odb_collate_status() reports the last collate on the
 * workspace even after later grouping or alignment calls on it.
 */
int odb_collate(const odb_window_t* w, int64_t num_slots,
                const int32_t* d_emit_order, const int64_t* d_row_token_start,
                const int32_t* d_row_len, const int32_t* d_slot_rows,
                const int32_t* d_slot_maxlen, const int64_t* d_slot_row_off,
                const int64_t* d_slot_tile_off, int32_t pad_id, int64_t out_capacity_elems,
                int32_t* d_input_ids, int32_t* d_labels, int32_t* d_attention_mask,
                int32_t* d_position_ids, void* d_ws, size_t ws_bytes, void* stream);

/* Rows of gathered row records the static scratch of odb_collate_static holds. */
#define ODB_COLLATE_STATIC_MAX_ROWS 2097152

/*
 * odb_collate without a workspace, for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid allocation).  Same
 * arguments, checks and outputs as odb_collate; it allocates nothing and synchronises
 * nothing.  Its scratch (the kernel's run counter and, when the plan brings no row
 * records, the gathered records) is a fixed array inside the library: 25,166,080 bytes per
 * device, held from the first call on that device until the process ends.
 *
 *   d_status   [1] device out: set to 0 when the call starts, nonzero if the plan is
 *              inconsistent (the cases odb_collate reports through odb_collate_status)
 *
 * Without row records the window may hold at most ODB_COLLATE_STATIC_MAX_ROWS - W + 1
 * samples (n + W - 1 rows); a larger window returns ODB_E_INVALID_ARG before anything
 * is launched (pass the plan's row records, or use odb_collate).  Every call on a device
 * shares that device's scratch: calls that overlap on one device race, so keep them on
 * one stream or order them with events.
 */
int odb_collate_static(const odb_window_t* w, int64_t num_slots,
                       const int32_t* d_emit_order, const int64_t* d_row_token_start,
                       const int32_t* d_row_len, const int32_t* d_slot_rows,
                       const int32_t* d_slot_maxlen, const int64_t* d_slot_row_off,
                       const int64_t* d_slot_tile_off, int32_t pad_id, int64_t out_capacity_elems,
                       int32_t* d_input_ids, int32_t* d_labels, int32_t* d_attention_mask,
                       int32_t* d_position_ids, int32_t* d_status, void* stream);

/* Synchronises `stream` and returns ODB_OK, or ODB_E_INVALID_DATA if the last
 * odb_collate on this workspace met an inconsistent plan (and clears the word). */
int odb_collate_status(void* d_ws, size_t ws_bytes, void* stream);

/*
 * Identity coverage self-check on its own (App. C, terminal identity coverage): counts
 * every sampler view over `emitted` and `leftover` ids and every identity over the same
 * union.  Fills h_info->bad_views, missing_ids and duplicate_ids only.  Synchronises.
 */
int odb_check_coverage(const odb_window_t* w, const int32_t* d_emitted, int64_t num_emitted,
                       const int32_t* d_leftover, int64_t num_leftover,
                       odb_plan_info_t* h_info, void* d_ws, size_t ws_bytes, void* stream);

/* Loss-scaling weight modes (App. B and the loss-scaling ablation of App. N). */
typedef enum odb_weight_mode {
    ODB_WEIGHT_SAMPLE = 0,         /* n_{r,j} / sum_r n_{r,j}                                  */
    ODB_WEIGHT_TOKEN_APPROX = 1,   /* a_{r,j} / sum_r a_{r,j}, a = d_slot_tokens_approx         */
    ODB_WEIGHT_TOKEN_EXACT = 2     /* t_{r,j} / sum_r t_{r,j}, t = real tokens (Eq. 2)          */
} odb_weight_mode_t;

/*
 * Loss-scaling weights of an aligned plan (Sec. 2.3 "Loss scaling", Eq. 2, App. B).
 *
 * At step j rank r pre-scales its per-token mean loss by W * weight[r * S + j]; DDP's
 * mean over ranks then equals sum_r weight * mean loss of rank r, which for the exact
 * token-level mode is the per-token mean over the whole step.  n = rows, t = real
 * tokens, a = approximate tokens of the slot, all as written by odb_align_groups.
 *
 *   num_ranks, steps        W >= 1 and S >= 0 of the plan (W * S slots, rank-major)
 *   mode                    odb_weight_mode_t
 *   d_slot_rows             [W*S] rows per slot
 *   d_slot_tokens           [W*S] real tokens per slot
 *   d_slot_tokens_approx    [W*S] approximate tokens per slot (read only in the
 *                           approximate mode; may be NULL otherwise)
 *   d_weight                [W*S] out: fp64 weight of every slot; IDLE slots get 0
 *   d_step_tokens           [S] out, or NULL: sum_r t_{r,j}
 *   d_step_samples          [S] out, or NULL: sum_r n_{r,j}
 *
 * Sums over ranks run in rank order; every product, sum and quotient is one fp64
 * operation rounded to nearest (no fused multiply-add), so results are reproducible
 * bit for bit.  A step whose denominator is 0 gets zero weights.  Asynchronous (one
 * kernel); needs no workspace.
 */
int odb_loss_weights(int32_t num_ranks, int64_t steps, int32_t mode, const int32_t* d_slot_rows,
                     const int64_t* d_slot_tokens, const double* d_slot_tokens_approx, double* d_weight,
                     int64_t* d_step_tokens, int64_t* d_step_samples, void* stream);

/* Moments of a length sketch (see odb_length_sketch). */
typedef struct odb_length_sketch {
    int64_t  samples;         /* n: sketched samples                                     */
    int64_t  short_samples;   /* samples with l < L_max / 4 (tested as 4 l < L_max)      */
    int64_t  sum_len;         /* sum of l                                                */
    uint64_t sum_sq_hi;       /* sum of l^2 = sum_sq_hi * 2^32 + sum_sq_lo (exact)       */
    uint64_t sum_sq_lo;
    int64_t  min_len;         /* 0 if n = 0                                              */
    int64_t  max_len;
    double   mean;            /* sum_len / n                                             */
    double   cv;              /* population sigma / mu = sqrt(n sum l^2 - (sum l)^2) / sum l */
    double   short_fraction;  /* f_s = short_samples / n                                 */
    int32_t  high_roi;        /* cv >= 0.8 or f_s > 0.2                                  */
    int32_t  reserved0;
} odb_length_sketch_t;

/*
 * Return-on-investment screen (Sec. 1 defines CV = sigma / mu of realised lengths; the
 * practical-guidance section screens a 1k-5k sketch with CV and f_s = Pr[l < L_max / 4]
 * and flags CV >= 0.8 or f_s > 0.2 as a high-return workload).
 *
 *   d_ids     [count] sample ids of the sketch (device), or NULL: samples 0 .. count-1
 *   count     sketch size, 0 <= count < 2^31 (<= n when d_ids is NULL); ids may repeat
 *   budget    L_max >= 1 that f_s is measured against
 *   h_out     host out
 *
 * Integer fields are exact.  mean, cv and short_fraction are computed on the host from
 * them (cv from an exact 128-bit numerator).  Synchronises `stream`.  Returns
 * ODB_E_INVALID_DATA if an id lies outside the window or a sketched length is < 1.
 */
int odb_length_sketch(const odb_window_t* w, const int32_t* d_ids, int64_t count, int64_t budget,
                      odb_length_sketch_t* h_out, void* d_ws, size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------- unified loop */

/* Parameters of one logical sampler iteration of the streaming protocol. */
typedef struct odb_stream_params {
    int32_t mode;                  /* odb_mode_t: join (drain, then stop) or non-join quota  */
    int32_t buffer_size;           /* views a rank collects before it groups, >= 1           */
    int32_t depth;                 /* outstanding-depth envelope D: most views a rank holds
                                      fetched but not emitted; buffer_size <= D <= 4096      */
    int32_t reserved0;             /* must be 0                                              */
    int64_t quota;                 /* non-join sample quota Q >= 1                           */
    const int32_t* rate;           /* HOST [W] views rank r's workers deliver per round, >= 1 */
    const int64_t* slot_capacity;  /* HOST [W] output-slot capacity C_r >= 0, or NULL        */
    int64_t max_rounds;            /* protocol rounds (>= 1) after which the call fails; also
                                      the length of the workspace's round record             */
} odb_stream_params_t;

/* One protocol round. */
typedef struct odb_stream_round {
    int32_t kind;                  /* 0 emit, 1 skip (some unfinished rank not ready), 2 stop */
    int32_t reserved0;
    int64_t target;                /* T of an emit round, else 0                             */
    int64_t emitted;               /* views emitted in the round (after a quota cut)         */
    int64_t phi;                   /* potential after the round: views not yet emitted      */
} odb_stream_round_t;

/* Summary of one logical iteration. */
typedef struct odb_stream_info {
    int64_t steps;                 /* S: aligned steps                                       */
    int64_t rounds;                /* protocol rounds, including the one that saw the stop   */
    int64_t emit_rounds;
    int64_t skip_rounds;
    int32_t stop_reason;           /* odb_stop_reason_t                                      */
    int32_t reserved0;
    int64_t views;                 /* M = W * ceil(N / W) sampler views                      */
    int64_t emitted_views;
    int64_t undelivered_views;     /* fetched but not emitted at the stop (eta_logical * N)  */
    int64_t pending_views;         /* never fetched                                          */
    int64_t real_tokens;
    int64_t padded_elems;
    int64_t max_step_samples;
    int64_t splits;
    int64_t overflow_groups;
    int64_t missing_ids;           /* identities with no emitted view                        */
    int64_t duplicate_ids;         /* emitted views beyond the first of their identity       */
    int64_t bad_views;             /* views emitted more than once (0 unless the library errs) */
    int64_t second_gather_rounds;  /* emit rounds in which some ready rank had G_r != T     */
    int64_t max_outstanding;       /* largest |B_r| after a fetch (<= depth)                 */
    double  pad_fraction;
    int64_t required_slot_capacity;/* W * S; set on ODB_E_CAPACITY and on success            */
} odb_stream_info_t;

/* Bytes of device workspace odb_stream_plan needs (0 for invalid arguments, and for a
 * slot_capacity or max_rounds that would ask for more than 2^50 bytes).  The workspace
 * starts with the window workspace, so odb_collate can reuse it. */
size_t odb_stream_workspace_size(const odb_window_t* w, int32_t depth, int64_t slot_capacity,
                                 int64_t max_rounds);

/*
 * One logical iteration of the unified loop (Sec. 2.3 "Unified loop and termination",
 * App. C state and transition rules, App. E state machine) over the window's samples
 * taken as dataset identities 0..N-1 (rank_offsets of the window are not used; W is
 * num_ranks).
 *
 * Sampler: d_perm [N] is the iteration's shuffled identity list, a permutation of [0, N)
 * drawn by the caller (entries outside [0, N) among the fetched views are rejected,
 * repeated entries are not detected: missing_ids and duplicate_ids are counted from the
 * emitted views under the permutation contract); it is padded by repeating it from its
 * head to M = W * ceil(N / W) views,
 * view m has identity perm[m mod N] and belongs to rank m mod W (stride sharding), and a
 * rank visits its views in increasing m.
 * Round: every rank moves up to rate[r] views into its buffer (never above depth); a rank
 * is finished when it has nothing pending or buffered, ready when its buffer holds
 * buffer_size views or nothing is pending.  Join stops when every rank is finished,
 * non-join when any is (or at the quota).  Otherwise, if an unfinished rank is not ready
 * the round is a skip round; else every ready rank groups its whole buffer (Sec. 2.2,
 * ties by view index), T follows Eq. 3 over the ready ranks (S_r = buffered views), and
 * Algorithm 1 splits or overflows; each ready rank emits T steps, finished ranks IDLE
 * slots, and overflow stays buffered.  Non-join stops after the first step at which the
 * cumulative emitted count reaches `quota`.
 *
 * Outputs use the plan layout of odb_align_groups (slot k = r * S + j; rows of a group
 * from its shortest member), so odb_collate and odb_loss_weights take them unchanged:
 *   d_emit_order     [M] out: identities of the emitted views, slot order, row order
 *   d_emit_views     [M] out: the emitted views themselves
 *   d_row_token_start, d_row_len  [M] out, or both NULL: row records of the emitted
 *                    views (token start and length of their identities), as odb_align_groups
 *   slot arrays      as odb_align_groups, capacity slot_capacity (W * S needed)
 *   d_left_views     [M] out: un-emitted views, per rank in increasing view index
 *   d_left_off       [W+1] out
 *   h_trace          [max_rounds] host out, or NULL: one record per round
 * Rounds are enqueued in chunks, each as long as a lower bound on the rounds left (from
 * the sampler cursors, the rates and, non-join, the quota; at least 8 after the first);
 * the call synchronises `stream` once per chunk and at the end.  Returns ODB_E_CAPACITY if
 * slot_capacity < W * S (required_slot_capacity tells the size) or the iteration needs
 * more than max_rounds rounds, ODB_E_INVALID_DATA for a perm entry outside [0, N) or a
 * sample length < 1 met among the views the iteration fetches.
 */
int odb_stream_plan(const odb_window_t* w, const int32_t* d_perm, int64_t budget,
                    const odb_stream_params_t* params, int64_t slot_capacity,
                    int32_t* d_emit_order, int32_t* d_emit_views, int64_t* d_row_token_start,
                    int32_t* d_row_len, int32_t* d_slot_rows,
                    int32_t* d_slot_maxlen, int64_t* d_slot_row_off, int64_t* d_slot_tile_off,
                    int64_t* d_slot_tokens, double* d_slot_tokens_approx, int32_t* d_left_views,
                    int64_t* d_left_off, odb_stream_round_t* h_trace, odb_stream_info_t* h_info,
                    void* d_ws, size_t ws_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* ODB_H_ */
