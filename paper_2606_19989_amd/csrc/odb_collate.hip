// Stage 4 of the ODB window pipeline: padded collation (Sec. 2.1, Fig. 1 -- every
// aligned group is padded to its own longest sample).
//
// The kernel is stationary on the flat output: all four outputs share one element index
// space [0, padded_elems), every lane owns 4 consecutive elements, so each lane issues one
// aligned 16-byte non-temporal store per output whatever the row length.  A block owns a
// contiguous span of the output and walks it in 1024-element steps; each lane keeps the
// tile (slot) index of its current element and advances it by a galloping search over
// the tile offsets, so long tiles cost one cached compare per step and runs of tiny tiles
// stay logarithmic.  Row, column and sample come from the tile's max length and row
// offset; real columns read the sample's tokens from the CSR stream.
#include "odb_internal.h"

namespace odb {

namespace {

constexpr int kCollateBlock = 256;
constexpr int kVec = 4;
constexpr int64_t kChunk = (int64_t)kCollateBlock * kVec;

typedef int v4i __attribute__((ext_vector_type(4)));

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
    // tile_off[lo] <= e < tile_off[hi]
    while (hi - lo > 1) {
        const int64_t mid = lo + ((hi - lo) >> 1);
        if (tile_off[mid] <= e) lo = mid; else hi = mid;
    }
    return lo;
}

struct RowCursor {
    int64_t k;      // slot
    int64_t t1;     // end of the slot's tile
    int32_t ml;     // tile width (max length)
    int32_t col;    // column of the current element
    int64_t row;    // row of the current element
    int64_t ts;     // first token of the row's sample
    int32_t l;      // length of the row's sample
};

__device__ __forceinline__ void load_row(RowCursor& c, const int64_t* __restrict__ tok_off,
                                         const int32_t* __restrict__ emit, const int32_t* __restrict__ rows,
                                         const int64_t* __restrict__ row_off, int64_t n, int32_t* err) {
    const int64_t ri = row_off[c.k] + c.row;
    bool ok = c.row < rows[c.k] && ri >= 0 && ri < n;
    int32_t s = ok ? emit[ri] : 0;
    ok = ok && s >= 0 && s < n;
    if (ok) {
        c.ts = tok_off[s];
        const int64_t l = tok_off[s + 1] - c.ts;
        ok = c.ts >= 0 && l >= 0 && l <= 0x7FFFFFFF;
        c.l = ok ? (int32_t)l : 0;
    } else {
        c.ts = 0;
        c.l = 0;
    }
    if (!ok) atomicOr(err, 1);
}

__device__ __forceinline__ void enter_slot(RowCursor& c, int64_t e, const int64_t* __restrict__ tile_off,
                                           const int32_t* __restrict__ maxlen, const int64_t* __restrict__ tok_off,
                                           const int32_t* __restrict__ emit, const int32_t* __restrict__ rows,
                                           const int64_t* __restrict__ row_off, int64_t n, int32_t* err) {
    const int64_t t0 = tile_off[c.k];
    c.t1 = tile_off[c.k + 1];
    c.ml = maxlen[c.k];
    const int64_t local = e - t0;
    if (c.ml <= 0) {
        atomicOr(err, 1);
        c.ml = 1;
    }
    if (c.t1 - t0 <= 0xFFFFFFFFll) {
        const uint32_t q = (uint32_t)local / (uint32_t)c.ml;
        c.row = q;
        c.col = (int32_t)((uint32_t)local - q * (uint32_t)c.ml);
    } else {
        c.row = local / c.ml;
        c.col = (int32_t)(local - c.row * c.ml);
    }
    load_row(c, tok_off, emit, rows, row_off, n, err);
}

template <bool kAligned>
__global__ void __launch_bounds__(kCollateBlock) collate_kernel(
    const int64_t* __restrict__ tok_off, const int32_t* __restrict__ tokens, int64_t n,
    const int32_t* __restrict__ emit, int64_t num_slots, const int32_t* __restrict__ rows,
    const int32_t* __restrict__ maxlen, const int64_t* __restrict__ row_off, const int64_t* __restrict__ tile_off,
    int32_t pad_id, int64_t capacity, int32_t* __restrict__ o_ids, int32_t* __restrict__ o_lab,
    int32_t* __restrict__ o_msk, int32_t* __restrict__ o_pos, int32_t* err) {
    const int64_t total_plan = tile_off[num_slots];
    const int64_t total = total_plan < capacity ? total_plan : capacity;
    if (total <= 0) return;
    const int64_t nchunks = (total + kChunk - 1) / kChunk;
    const int64_t per = (nchunks + gridDim.x - 1) / gridDim.x;
    const int64_t c0 = (int64_t)blockIdx.x * per;
    const int64_t c1 = c0 + per < nchunks ? c0 + per : nchunks;
    if (c0 >= c1) return;
    int64_t e = c0 * kChunk + (int64_t)threadIdx.x * kVec;
    if (e >= total) return;
    RowCursor c;
    {
        // last slot with tile_off[k] <= e
        int64_t lo = 0, hi = num_slots;
        while (hi - lo > 1) {
            const int64_t mid = lo + ((hi - lo) >> 1);
            if (tile_off[mid] <= e) lo = mid; else hi = mid;
        }
        c.k = lo;
    }
    c.t1 = -1;
    for (int64_t ci = c0; ci < c1; ++ci, e += kChunk) {
        if (e >= total) break;
        if (e >= c.t1) {
            c.k = advance_slot(tile_off, num_slots, c.k, e);
            enter_slot(c, e, tile_off, maxlen, tok_off, emit, rows, row_off, n, err);
        } else {
            // same tile: move the cursor forward by kChunk elements
            // col < ml <= 2^31 - 1, so col + kChunk fits in 32 unsigned bits
            const uint32_t local_col = (uint32_t)c.col + (uint32_t)kChunk;
            if (local_col >= (uint32_t)c.ml) {
                const uint32_t adv = local_col / (uint32_t)c.ml;
                c.row += adv;
                c.col = (int32_t)(local_col - adv * (uint32_t)c.ml);
                load_row(c, tok_off, emit, rows, row_off, n, err);
            } else {
                c.col = (int32_t)local_col;
            }
        }
        v4i vid, vlab, vmsk, vpos;
        RowCursor d = c;  // cursor for the 4 elements of this step
#pragma unroll
        for (int i = 0; i < kVec; ++i) {
            const int64_t ee = e + i;
            if (i > 0 && ee < total) {
                if (ee >= d.t1) {
                    d.k = advance_slot(tile_off, num_slots, d.k, ee);
                    enter_slot(d, ee, tile_off, maxlen, tok_off, emit, rows, row_off, n, err);
                } else if (++d.col == d.ml) {
                    d.col = 0;
                    d.row += 1;
                    load_row(d, tok_off, emit, rows, row_off, n, err);
                }
            }
            const bool real = d.col < d.l;
            const int32_t tok = real ? tokens[d.ts + d.col] : 0;
            vid[i] = real ? tok : pad_id;
            vlab[i] = real ? tok : -100;
            vmsk[i] = real ? 1 : 0;
            vpos[i] = real ? d.col : 0;
        }
        if (kAligned && e + kVec <= total) {
            __builtin_nontemporal_store(vid, reinterpret_cast<v4i*>(o_ids + e));
            __builtin_nontemporal_store(vlab, reinterpret_cast<v4i*>(o_lab + e));
            __builtin_nontemporal_store(vmsk, reinterpret_cast<v4i*>(o_msk + e));
            __builtin_nontemporal_store(vpos, reinterpret_cast<v4i*>(o_pos + e));
        } else {
#pragma unroll
            for (int i = 0; i < kVec; ++i) {
                if (e + i < total) {
                    o_ids[e + i] = vid[i];
                    o_lab[e + i] = vlab[i];
                    o_msk[e + i] = vmsk[i];
                    o_pos[e + i] = vpos[i];
                }
            }
        }
    }
}

}  // namespace

}  // namespace odb

using namespace odb;

extern "C" int odb_collate(const odb_window_t* w, int64_t num_slots, const int32_t* d_emit_order,
                           const int32_t* d_slot_rows, const int32_t* d_slot_maxlen, const int64_t* d_slot_row_off,
                           const int64_t* d_slot_tile_off, int32_t pad_id, int64_t out_capacity_elems,
                           int32_t* d_input_ids, int32_t* d_labels, int32_t* d_attention_mask,
                           int32_t* d_position_ids, void* d_ws, size_t ws_bytes, void* stream) {
    Layout L;
    ODB_TRY(check_workspace(w, d_ws, ws_bytes, &L));
    if (num_slots < 0) return set_error(ODB_E_INVALID_ARG, "num_slots must be >= 0");
    if (out_capacity_elems < 0) return set_error(ODB_E_INVALID_ARG, "out_capacity_elems must be >= 0");
    if (num_slots == 0 || out_capacity_elems == 0) return ODB_OK;
    if (!d_slot_rows || !d_slot_maxlen || !d_slot_row_off || !d_slot_tile_off)
        return set_error(ODB_E_INVALID_ARG, "plan arrays must not be NULL");
    if (!d_input_ids || !d_labels || !d_attention_mask || !d_position_ids)
        return set_error(ODB_E_INVALID_ARG, "output arrays must not be NULL");
    if (w->num_samples > 0 && !d_emit_order) return set_error(ODB_E_INVALID_ARG, "d_emit_order is NULL");
    hipStream_t s = static_cast<hipStream_t>(stream);
    const bool aligned = ((reinterpret_cast<uintptr_t>(d_input_ids) | reinterpret_cast<uintptr_t>(d_labels) |
                           reinterpret_cast<uintptr_t>(d_attention_mask) |
                           reinterpret_cast<uintptr_t>(d_position_ids)) &
                          15) == 0;
    const unsigned grid = (unsigned)num_cus() * 8;
    int32_t* err = &ws_at<DevStatus>(d_ws, L.status)->collate_err;
    if (aligned)
        hipLaunchKernelGGL(collate_kernel<true>, dim3(grid), dim3(kCollateBlock), 0, s, w->d_token_offsets,
                           w->d_tokens, w->num_samples, d_emit_order, num_slots, d_slot_rows, d_slot_maxlen,
                           d_slot_row_off, d_slot_tile_off, pad_id, out_capacity_elems, d_input_ids, d_labels,
                           d_attention_mask, d_position_ids, err);
    else
        hipLaunchKernelGGL(collate_kernel<false>, dim3(grid), dim3(kCollateBlock), 0, s, w->d_token_offsets,
                           w->d_tokens, w->num_samples, d_emit_order, num_slots, d_slot_rows, d_slot_maxlen,
                           d_slot_row_off, d_slot_tile_off, pad_id, out_capacity_elems, d_input_ids, d_labels,
                           d_attention_mask, d_position_ids, err);
    ODB_LAUNCHED();
    return ODB_OK;
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
