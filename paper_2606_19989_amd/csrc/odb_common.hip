// Host-side plumbing shared by every entry point: error strings, workspace layout,
// window validation and small uploads.
#include <atomic>
#include <cstdarg>
#include <cstdio>
#include <cstring>

#include "odb_internal.h"

namespace odb {

namespace {
thread_local char g_msg[1024] = {0};

size_t align_up(size_t x) { return (x + 255) & ~size_t(255); }
}  // namespace

int set_error(int code, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_msg, sizeof(g_msg), fmt, ap);
    va_end(ap);
    return code;
}

const char* last_error() { return g_msg; }

int check_window(const odb_window_t* w) {
    if (!w) return set_error(ODB_E_INVALID_ARG, "window is NULL");
    if (w->num_ranks < 1) return set_error(ODB_E_INVALID_ARG, "num_ranks must be >= 1 (got %d)", w->num_ranks);
    if (w->reserved0 != 0) return set_error(ODB_E_INVALID_ARG, "window.reserved0 must be 0");
    if (w->num_samples < 0 || w->num_samples >= 0x7FFFFFFFll)
        return set_error(ODB_E_INVALID_ARG, "num_samples must be in [0, 2^31 - 1) (got %lld)",
                         (long long)w->num_samples);
    if (!w->rank_offsets) return set_error(ODB_E_INVALID_ARG, "rank_offsets is NULL");
    if (w->rank_offsets[0] != 0 || w->rank_offsets[w->num_ranks] != w->num_samples)
        return set_error(ODB_E_INVALID_ARG, "rank_offsets must start at 0 and end at num_samples");
    for (int r = 0; r < w->num_ranks; ++r)
        if (w->rank_offsets[r + 1] < w->rank_offsets[r])
            return set_error(ODB_E_INVALID_ARG, "rank_offsets must be non-decreasing (rank %d)", r);
    if (w->num_samples > 0 && (!w->d_token_offsets || !w->d_tokens))
        return set_error(ODB_E_INVALID_ARG, "d_token_offsets / d_tokens must not be NULL");
    if (w->d_identity && w->num_identities < 1)
        return set_error(ODB_E_INVALID_ARG, "num_identities must be >= 1 with an identity map");
    if (w->num_identities < 0 || w->num_identities >= 0x7FFFFFFFll)
        return set_error(ODB_E_INVALID_ARG, "num_identities out of range");
    return ODB_OK;
}

bool make_layout(const odb_window_t* w, Layout* L) {
    if (check_window(w) != ODB_OK) return false;
    const int64_t W = w->num_ranks;
    const int64_t n = w->num_samples;
    const int64_t nid = w->d_identity ? w->num_identities : n;
    int64_t nb = 0, max_nr = 0;
    for (int64_t r = 0; r < W; ++r) {
        int64_t nr = w->rank_offsets[r + 1] - w->rank_offsets[r];
        nb += (nr + kSortTile - 1) / kSortTile;
        if (nr > max_nr) max_nr = nr;
    }
    const int64_t n1 = n + 1;
    int64_t scan_max = n1;
    if (256 * nb > scan_max) scan_max = 256 * nb;
    if (W * max_nr + 1 > scan_max) scan_max = W * max_nr + 1;
    const int64_t partials = scan_max / kScanTile + 4;

    size_t o = 0;
    auto take = [&](size_t bytes) {
        size_t at = o;
        o = align_up(o + (bytes ? bytes : 1));
        return at;
    };
    // status, round, info and ranks first and in this order: one copy reads them all
    L->status = take(sizeof(DevStatus));
    L->round = take(sizeof(RoundState));
    L->info = take(sizeof(DevInfo));
    L->ranks = take(sizeof(RankState) * W);
    L->sketch = take(256);
    L->rank_off = take(8 * (W + 1));
    L->cap = take(8 * W);
    L->gbase = take(8 * (W + 1));
    L->tile_first = take(8 * (W + 1));
    L->rank_runs = take(4 * (W + 1));
    L->len = take(4 * n1);
    L->keys0 = take(4 * n1);
    L->keys1 = take(4 * n1);
    L->vals0 = take(4 * n1);
    L->vals1 = take(4 * n1);
    L->counts = take(4 * (256 * nb + 1));
    L->partials = take(16 * partials);   // room for pairs of int64 sums
    L->jmp0 = take(4 * n1);
    L->jmp1 = take(4 * n1);
    L->marks = take(n1);
    L->incl = take(4 * n1);
    L->gstart = take(4 * n1);
    L->gsize = take(4 * n1);
    L->gmax = take(4 * n1);
    L->sadj = take(8 * n1);
    L->cs = take(8 * n1);
    L->ov_slot = take(4 * n1);
    L->ov_lo = take(4 * n1);
    L->kept = take(4 * n1);
    L->srows = take(4 * n1);
    L->smax = take(4 * n1);
    L->stok = take(8 * n1);
    L->steps = take(8 * n1);
    L->buf_ids0 = take(4 * n1);
    L->buf_ids1 = take(4 * n1);
    L->buf_len0 = take(4 * n1);
    L->buf_len1 = take(4 * n1);
    L->gidx = take(4 * n1);
    L->stage = take(4 * n1);
    L->stage_len = take(4 * n1);
    L->cover = take(4 * ((nid > n ? nid : n) + 1));
    L->row_ts = take(8 * (n1 + W));
    L->row_len = take(4 * (n1 + W));
    L->total = o;
    L->num_sort_blocks = nb;
    L->partials_len = partials;
    return true;
}

int check_workspace(const odb_window_t* w, void* d_ws, size_t ws_bytes, Layout* L) {
    ODB_TRY(check_window(w));
    if (!make_layout(w, L)) return set_error(ODB_E_INVALID_ARG, "bad window");
    if (!d_ws) return set_error(ODB_E_INVALID_ARG, "workspace is NULL");
    if (reinterpret_cast<uintptr_t>(d_ws) & 255)
        return set_error(ODB_E_INVALID_ARG, "workspace must be 256-byte aligned");
    if (ws_bytes < L->total)
        return set_error(ODB_E_WORKSPACE, "workspace has %zu bytes, %zu needed", ws_bytes, L->total);
    return ODB_OK;
}

// Small host arrays reach the device as kernel arguments, kValuesPerLaunch values per
// launch: no host-to-device copy (which, from pageable memory, may wait for the stream)
// and nothing a graph capture could not record.
constexpr int kValuesPerLaunch = 64;
struct Values64 {
    int64_t v[kValuesPerLaunch];
};

// Stores values [first, first + count) of an array; the first launch of a call also
// resets the status word.  The collate's error word is left alone: odb_collate clears it
// when it starts and odb_collate_status when it has read it, so a plan call made on the
// same workspace in between does not erase a collate error.
__global__ void store_values_kernel(Values64 vals, int64_t* dst, int count, DevStatus* st) {
    const int t = threadIdx.x;
    if (t < count) dst[t] = vals.v[t];
    if (st) {
        if (t == 0) {
            st->err = 0;
            st->first_bad = 0x7FFFFFFFFFFFFFFFll;
            st->first_bad_len = 0x7FFFFFFFFFFFFFFFll;
            st->min_len = 0xFFFFFFFFu;
            st->max_len = 0;
        }
        if (t < kMaxJumpRounds) st->jump_changed[t] = 0;
    }
}

static int store_values(const int64_t* src, int64_t count, int64_t* dst, DevStatus* st, hipStream_t s) {
    int64_t a = 0;
    do {
        Values64 v{};
        const int64_t left = count - a;
        const int c = (int)(left < kValuesPerLaunch ? (left > 0 ? left : 0) : kValuesPerLaunch);
        for (int i = 0; i < c; ++i) v.v[i] = src[a + i];
        hipLaunchKernelGGL(store_values_kernel, dim3(1), dim3(kValuesPerLaunch), 0, s, v, dst + a, c,
                           a == 0 ? st : (DevStatus*)nullptr);
        ODB_LAUNCHED();
        a += kValuesPerLaunch;
    } while (a < count);
    return ODB_OK;
}

int upload_small(const odb_window_t* w, const Layout& L, void* ws, const int64_t* cap, hipStream_t s) {
    const int W = w->num_ranks;
    ODB_TRY(store_values(w->rank_offsets, W + 1, ws_at<int64_t>(ws, L.rank_off), ws_at<DevStatus>(ws, L.status), s));
    if (cap) ODB_TRY(store_values(cap, W, ws_at<int64_t>(ws, L.cap), nullptr, s));
    return ODB_OK;
}

int read_state(const Layout& L, void* ws, int W, HostState* h, hipStream_t s) {
    const size_t bytes = L.ranks + sizeof(RankState) * (size_t)W - L.status;
    h->buf.resize(bytes);
    ODB_TRY_HIP(hipMemcpyAsync(h->buf.data(), ws_at<char>(ws, L.status), bytes, hipMemcpyDeviceToHost, s));
    ODB_TRY_HIP(hipStreamSynchronize(s));
    const char* b = h->buf.data();
    memcpy(&h->st, b, sizeof(DevStatus));
    memcpy(&h->rs, b + (L.round - L.status), sizeof(RoundState));
    memcpy(&h->info, b + (L.info - L.status), sizeof(DevInfo));
    h->ranks.resize((size_t)W);
    memcpy(h->ranks.data(), b + (L.ranks - L.status), sizeof(RankState) * (size_t)W);
    return ODB_OK;
}

int num_cus() {
    // per device, looked up once; threads that race on the first lookup store the same value
    static std::atomic<int> cached[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    int v = cached[dev].load(std::memory_order_relaxed);
    if (!v) {
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0)
            v = 256;
        cached[dev].store(v, std::memory_order_relaxed);
    }
    return v;
}

}  // namespace odb

extern "C" {

const char* odb_status_string(int status) {
    switch (status) {
        case ODB_OK: return "ODB_OK";
        case ODB_E_INVALID_ARG: return "ODB_E_INVALID_ARG";
        case ODB_E_INVALID_DATA: return "ODB_E_INVALID_DATA";
        case ODB_E_WORKSPACE: return "ODB_E_WORKSPACE";
        case ODB_E_CAPACITY: return "ODB_E_CAPACITY";
        case ODB_E_HIP: return "ODB_E_HIP";
        case ODB_E_COVERAGE: return "ODB_E_COVERAGE";
        case ODB_E_INTERNAL: return "ODB_E_INTERNAL";
        default: return "ODB_E_UNKNOWN";
    }
}

const char* odb_last_error_message(void) { return odb::last_error(); }

size_t odb_workspace_size(const odb_window_t* w) {
    odb::Layout L;
    if (!odb::make_layout(w, &L)) return 0;
    return L.total;
}

}  // extern "C"
