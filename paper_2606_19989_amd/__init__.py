"""Python binding of libodb, the MI355X Online Dynamic Batching window pipeline.

The functions named ``odb_*`` mirror the C ABI in ``include/odb.h`` one to one: they
convert torch device tensors and host arrays into the pointers and structs the library
takes, call it, and turn its status into an exception.  All computation happens in the
HIP kernels of ``libodb.so``; there is no fallback path -- if the library is missing or
fails to load, every call raises.

:class:`Pipeline` owns the device buffers of one window and runs the three stages
(grouping, alignment, collation) in order on one stream, and on request the loss-scaling
weights of the aligned plan.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libodb.so")

ODB_OK = 0
ODB_E_INVALID_ARG = 1
ODB_E_INVALID_DATA = 2
ODB_E_WORKSPACE = 3
ODB_E_CAPACITY = 4
ODB_E_HIP = 5
ODB_E_COVERAGE = 6
ODB_E_INTERNAL = 7

ODB_MODE_JOIN = 0
ODB_MODE_NONJOIN_QUOTA = 1
ODB_STOP_DRAINED, ODB_STOP_QUOTA, ODB_STOP_RANK_FINISHED = 0, 1, 2
ODB_WEIGHT_SAMPLE, ODB_WEIGHT_TOKEN_APPROX, ODB_WEIGHT_TOKEN_EXACT = 0, 1, 2

EXPORTED = [
    "odb_status_string", "odb_last_error_message", "odb_workspace_size", "odb_form_groups",
    "odb_align_groups", "odb_collate", "odb_collate_status", "odb_check_coverage", "odb_loss_weights",
    "odb_length_sketch", "odb_stream_workspace_size", "odb_stream_plan", "odb_collate_static",
]
ODB_COLLATE_STATIC_MAX_ROWS = 2097152


class OdbError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{message} [status {status}]")
        self.status = status


class Window(ctypes.Structure):
    _fields_ = [
        ("num_ranks", ctypes.c_int32),
        ("reserved0", ctypes.c_int32),
        ("num_samples", ctypes.c_int64),
        ("rank_offsets", ctypes.c_void_p),
        ("d_token_offsets", ctypes.c_void_p),
        ("d_tokens", ctypes.c_void_p),
        ("d_identity", ctypes.c_void_p),
        ("num_identities", ctypes.c_int64),
    ]


class AlignParams(ctypes.Structure):
    _fields_ = [
        ("mode", ctypes.c_int32),
        ("reserved0", ctypes.c_int32),
        ("quota", ctypes.c_int64),
        ("slot_capacity", ctypes.c_void_p),
    ]


class PlanInfo(ctypes.Structure):
    _fields_ = [
        ("steps", ctypes.c_int64),
        ("rounds", ctypes.c_int32),
        ("stop_reason", ctypes.c_int32),
        ("emitted_samples", ctypes.c_int64),
        ("leftover_samples", ctypes.c_int64),
        ("real_tokens", ctypes.c_int64),
        ("padded_elems", ctypes.c_int64),
        ("max_step_samples", ctypes.c_int64),
        ("splits", ctypes.c_int64),
        ("overflow_groups", ctypes.c_int64),
        ("missing_ids", ctypes.c_int64),
        ("duplicate_ids", ctypes.c_int64),
        ("bad_views", ctypes.c_int64),
        ("pad_fraction", ctypes.c_double),
        ("required_slot_capacity", ctypes.c_int64),
        ("second_gather_rounds", ctypes.c_int64),
    ]

    def as_dict(self) -> dict:
        return {f: getattr(self, f) for f, _ in self._fields_}


class LengthSketch(ctypes.Structure):
    _fields_ = [
        ("samples", ctypes.c_int64),
        ("short_samples", ctypes.c_int64),
        ("sum_len", ctypes.c_int64),
        ("sum_sq_hi", ctypes.c_uint64),
        ("sum_sq_lo", ctypes.c_uint64),
        ("min_len", ctypes.c_int64),
        ("max_len", ctypes.c_int64),
        ("mean", ctypes.c_double),
        ("cv", ctypes.c_double),
        ("short_fraction", ctypes.c_double),
        ("high_roi", ctypes.c_int32),
        ("reserved0", ctypes.c_int32),
    ]


class StreamParams(ctypes.Structure):
    _fields_ = [
        ("mode", ctypes.c_int32),
        ("buffer_size", ctypes.c_int32),
        ("depth", ctypes.c_int32),
        ("reserved0", ctypes.c_int32),
        ("quota", ctypes.c_int64),
        ("rate", ctypes.c_void_p),
        ("slot_capacity", ctypes.c_void_p),
        ("max_rounds", ctypes.c_int64),
    ]


class StreamRound(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("reserved0", ctypes.c_int32), ("target", ctypes.c_int64),
                ("emitted", ctypes.c_int64), ("phi", ctypes.c_int64)]


class StreamInfo(ctypes.Structure):
    _fields_ = [
        ("steps", ctypes.c_int64),
        ("rounds", ctypes.c_int64),
        ("emit_rounds", ctypes.c_int64),
        ("skip_rounds", ctypes.c_int64),
        ("stop_reason", ctypes.c_int32),
        ("reserved0", ctypes.c_int32),
        ("views", ctypes.c_int64),
        ("emitted_views", ctypes.c_int64),
        ("undelivered_views", ctypes.c_int64),
        ("pending_views", ctypes.c_int64),
        ("real_tokens", ctypes.c_int64),
        ("padded_elems", ctypes.c_int64),
        ("max_step_samples", ctypes.c_int64),
        ("splits", ctypes.c_int64),
        ("overflow_groups", ctypes.c_int64),
        ("missing_ids", ctypes.c_int64),
        ("duplicate_ids", ctypes.c_int64),
        ("bad_views", ctypes.c_int64),
        ("second_gather_rounds", ctypes.c_int64),
        ("max_outstanding", ctypes.c_int64),
        ("pad_fraction", ctypes.c_double),
        ("required_slot_capacity", ctypes.c_int64),
    ]

    def as_dict(self) -> dict:
        return {f: getattr(self, f) for f, _ in self._fields_ if f != "reserved0"}


_lib = None


def load():
    """Load libodb.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                               "or python -m paper_2606_19989_amd.build")
        lib = ctypes.CDLL(LIB_PATH)
        P, I32, I64, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
        W = ctypes.POINTER(Window)
        lib.odb_status_string.restype = ctypes.c_char_p
        lib.odb_status_string.argtypes = [ctypes.c_int]
        lib.odb_last_error_message.restype = ctypes.c_char_p
        lib.odb_last_error_message.argtypes = []
        lib.odb_workspace_size.restype = SZ
        lib.odb_workspace_size.argtypes = [W]
        lib.odb_form_groups.restype = ctypes.c_int
        lib.odb_form_groups.argtypes = [W, I64, P, P, P, P, P, SZ, P]
        lib.odb_align_groups.restype = ctypes.c_int
        lib.odb_align_groups.argtypes = [W, I64, ctypes.POINTER(AlignParams), P, P, P, P, I64,
                                         P, P, P, P, P, P, P, P, P, P, P, ctypes.POINTER(PlanInfo), P, SZ, P]
        lib.odb_collate.restype = ctypes.c_int
        lib.odb_collate.argtypes = [W, I64, P, P, P, P, P, P, P, I32, I64, P, P, P, P, P, SZ, P]
        lib.odb_collate_static.restype = ctypes.c_int
        lib.odb_collate_static.argtypes = [W, I64, P, P, P, P, P, P, P, I32, I64, P, P, P, P, P, P]
        lib.odb_collate_status.restype = ctypes.c_int
        lib.odb_collate_status.argtypes = [P, SZ, P]
        lib.odb_check_coverage.restype = ctypes.c_int
        lib.odb_check_coverage.argtypes = [W, P, I64, P, I64, ctypes.POINTER(PlanInfo), P, SZ, P]
        lib.odb_loss_weights.restype = ctypes.c_int
        lib.odb_loss_weights.argtypes = [I32, I64, I32, P, P, P, P, P, P, P]
        lib.odb_length_sketch.restype = ctypes.c_int
        lib.odb_length_sketch.argtypes = [W, P, I64, I64, ctypes.POINTER(LengthSketch), P, SZ, P]
        lib.odb_stream_workspace_size.restype = SZ
        lib.odb_stream_workspace_size.argtypes = [W, I32, I64, I64]
        lib.odb_stream_plan.restype = ctypes.c_int
        lib.odb_stream_plan.argtypes = [W, P, I64, ctypes.POINTER(StreamParams), I64, P, P, P, P, P, P, P, P, P, P, P, P,
                                        P, ctypes.POINTER(StreamInfo), P, SZ, P]
        _lib = lib
    return _lib


def _check(status: int):
    if status != ODB_OK:
        lib = load()
        raise OdbError(status, f"{lib.odb_status_string(status).decode()}: "
                               f"{lib.odb_last_error_message().decode()}")


def _dptr(t) -> Optional[int]:
    """Device pointer of a contiguous torch tensor on a GPU (None passes NULL)."""
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("expected a device tensor")
    if not t.is_contiguous():
        raise ValueError("expected a contiguous tensor")
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def _sync_current(device):
    """Waits for the current stream of a GPU device (no-op elsewhere)."""
    import torch
    if torch.device(device).type == "cuda":
        torch.cuda.current_stream(device).synchronize()


class DeviceWindow:
    """A window resident in device memory, with its C descriptor.

    rank_offsets stays on the host (int64 numpy, W+1 entries); token_offsets (int64,
    n+1), tokens (int32) and the optional identity map (int64, n) are device tensors.
    """

    def __init__(self, rank_offsets, token_offsets, tokens, identity=None, num_identities: int = 0):
        self.rank_offsets = np.ascontiguousarray(rank_offsets, dtype=np.int64)
        self.token_offsets = token_offsets
        self.tokens = tokens
        self.identity = identity
        self.num_ranks = len(self.rank_offsets) - 1
        self.num_samples = int(self.rank_offsets[-1])
        self.struct = Window(self.num_ranks, 0, self.num_samples,
                             self.rank_offsets.ctypes.data_as(ctypes.c_void_p).value,
                             _dptr(token_offsets), _dptr(tokens), _dptr(identity),
                             int(num_identities) if identity is not None else 0)

    @property
    def ref(self):
        return ctypes.byref(self.struct)


def odb_workspace_size(win: DeviceWindow) -> int:
    v = load().odb_workspace_size(win.ref)
    if v == 0:
        _check(ODB_E_INVALID_ARG)
    return int(v)


def odb_form_groups(win, budget, order, sorted_len, group_index, groups_per_rank, ws, stream=None):
    _check(load().odb_form_groups(win.ref, int(budget), _dptr(order), _dptr(sorted_len), _dptr(group_index),
                                  _dptr(groups_per_rank), _dptr(ws), ws.numel() * ws.element_size(),
                                  _stream(stream)))


def odb_align_groups(win, budget, mode, quota, slot_capacity_per_rank, order, sorted_len, group_index,
                     groups_per_rank, slot_capacity, emit_order, slot_rows, slot_maxlen, slot_row_off,
                     slot_tile_off, slot_tokens, leftover, leftover_off, ws, stream=None, raise_on_capacity=True,
                     slot_tokens_approx=None, row_token_start=None, row_len=None):
    cap = None
    if slot_capacity_per_rank is not None:
        cap = np.ascontiguousarray(slot_capacity_per_rank, dtype=np.int64)
    params = AlignParams(int(mode), 0, int(quota), None if cap is None else cap.ctypes.data_as(ctypes.c_void_p).value)
    info = PlanInfo()
    st = load().odb_align_groups(win.ref, int(budget), ctypes.byref(params), _dptr(order), _dptr(sorted_len),
                                 _dptr(group_index), _dptr(groups_per_rank), int(slot_capacity), _dptr(emit_order),
                                 _dptr(row_token_start), _dptr(row_len), _dptr(slot_rows), _dptr(slot_maxlen), _dptr(slot_row_off), _dptr(slot_tile_off),
                                 _dptr(slot_tokens), _dptr(slot_tokens_approx), _dptr(leftover), _dptr(leftover_off),
                                 ctypes.byref(info),
                                 _dptr(ws), ws.numel() * ws.element_size(), _stream(stream))
    if st == ODB_E_CAPACITY and not raise_on_capacity:
        return st, info.as_dict()
    _check(st)
    return st, info.as_dict()


def odb_collate(win, num_slots, emit_order, slot_rows, slot_maxlen, slot_row_off, slot_tile_off, pad_id,
                out_capacity, input_ids, labels, attention_mask, position_ids, ws, stream=None, row_token_start=None,
                row_len=None):
    _check(load().odb_collate(win.ref, int(num_slots), _dptr(emit_order), _dptr(row_token_start), _dptr(row_len),
                              _dptr(slot_rows), _dptr(slot_maxlen),
                              _dptr(slot_row_off), _dptr(slot_tile_off), int(pad_id), int(out_capacity),
                              _dptr(input_ids), _dptr(labels), _dptr(attention_mask), _dptr(position_ids),
                              _dptr(ws), ws.numel() * ws.element_size(), _stream(stream)))


def odb_collate_static(win, num_slots, emit_order, slot_rows, slot_maxlen, slot_row_off, slot_tile_off, pad_id,
                       out_capacity, input_ids, labels, attention_mask, position_ids, status, stream=None,
                       row_token_start=None, row_len=None):
    """odb_collate without a workspace (the library's fixed scratch); ``status`` is a
    device int32 tensor of one element that receives 0 or the plan-error flag."""
    _check(load().odb_collate_static(win.ref, int(num_slots), _dptr(emit_order), _dptr(row_token_start),
                                     _dptr(row_len), _dptr(slot_rows), _dptr(slot_maxlen), _dptr(slot_row_off),
                                     _dptr(slot_tile_off), int(pad_id), int(out_capacity), _dptr(input_ids),
                                     _dptr(labels), _dptr(attention_mask), _dptr(position_ids), _dptr(status),
                                     _stream(stream)))


def odb_collate_status(ws, stream=None):
    _check(load().odb_collate_status(_dptr(ws), ws.numel() * ws.element_size(), _stream(stream)))


def odb_check_coverage(win, emitted, num_emitted, leftover, num_leftover, ws, stream=None) -> dict:
    info = PlanInfo()
    _check(load().odb_check_coverage(win.ref, _dptr(emitted), int(num_emitted), _dptr(leftover), int(num_leftover),
                                     ctypes.byref(info), _dptr(ws), ws.numel() * ws.element_size(),
                                     _stream(stream)))
    return info.as_dict()


def odb_loss_weights(num_ranks, steps, mode, slot_rows, slot_tokens, slot_tokens_approx, weight,
                     step_tokens=None, step_samples=None, stream=None):
    _check(load().odb_loss_weights(int(num_ranks), int(steps), int(mode), _dptr(slot_rows), _dptr(slot_tokens),
                                   _dptr(slot_tokens_approx), _dptr(weight), _dptr(step_tokens), _dptr(step_samples),
                                   _stream(stream)))


def odb_length_sketch(win, ids, count, budget, ws, stream=None) -> dict:
    """CV, f_s and exact length moments of a sketch (ids: device int32 tensor or None for
    samples 0 .. count-1); ``sum_sq`` is returned as one Python integer."""
    out = LengthSketch()
    _check(load().odb_length_sketch(win.ref, _dptr(ids), int(count), int(budget), ctypes.byref(out), _dptr(ws),
                                    ws.numel() * ws.element_size(), _stream(stream)))
    d = {f: getattr(out, f) for f, _ in out._fields_ if f != "reserved0"}
    d["sum_sq"] = (int(d.pop("sum_sq_hi")) << 32) + int(d.pop("sum_sq_lo"))
    return d


class Pipeline:
    """Device buffers of one window and the three-stage call sequence.

    Slot arrays start at ``W * max_r n_r`` capacity unless ``slot_capacity`` is given;
    outputs of :meth:`collate` are allocated (or reused) at ``padded_elems``.
    """

    def __init__(self, win: DeviceWindow, budget: int, mode: str = "join", quota: int = 0,
                 capacity=None, pad_id: int = 0, slot_capacity: Optional[int] = None):
        import torch

        self.torch = torch
        self.win = win
        self.budget = int(budget)
        self.mode = ODB_MODE_NONJOIN_QUOTA if mode == "nonjoin" else ODB_MODE_JOIN
        self.quota = int(quota)
        self.capacity = capacity
        self.pad_id = int(pad_id)
        dev = win.token_offsets.device
        self.device = dev
        n, W = win.num_samples, win.num_ranks
        n1 = max(n, 1)
        i32 = dict(dtype=torch.int32, device=dev)
        i64 = dict(dtype=torch.int64, device=dev)
        self.ws = torch.empty(odb_workspace_size(win), dtype=torch.uint8, device=dev)
        self.order = torch.empty(n1, **i32)
        self.sorted_len = torch.empty(n1, **i32)
        self.group_index = torch.empty(n1, **i32)
        self.groups_per_rank = torch.empty(W, **i32)
        self.emit_order = torch.empty(n1, **i32)
        self.row_token_start = torch.empty(n1, **i64)
        self.row_len = torch.empty(n1, **i32)
        self.leftover = torch.empty(n1, **i32)
        self.leftover_off = torch.empty(W + 1, **i64)
        if slot_capacity is None:
            sizes = np.diff(win.rank_offsets)
            slot_capacity = int(W * (sizes.max() if len(sizes) else 0))
        self._alloc_slots(max(int(slot_capacity), 1))
        self.info = None
        self.outputs = None

    def _alloc_slots(self, cap: int):
        torch = self.torch
        self.slot_capacity = cap
        self.slot_rows = torch.empty(cap, dtype=torch.int32, device=self.device)
        self.slot_maxlen = torch.empty(cap, dtype=torch.int32, device=self.device)
        self.slot_tokens = torch.empty(cap, dtype=torch.int64, device=self.device)
        self.slot_tokens_approx = torch.empty(cap, dtype=torch.float64, device=self.device)
        self.slot_row_off = torch.empty(cap + 1, dtype=torch.int64, device=self.device)
        self.slot_tile_off = torch.empty(cap + 1, dtype=torch.int64, device=self.device)
        # buffers may be used on another stream than the one they were allocated on
        _sync_current(self.device)

    def form(self, stream=None):
        odb_form_groups(self.win, self.budget, self.order, self.sorted_len, self.group_index,
                        self.groups_per_rank, self.ws, stream)

    def align(self, stream=None) -> dict:
        args = lambda: (self.win, self.budget, self.mode, self.quota, self.capacity, self.order, self.sorted_len,
                        self.group_index, self.groups_per_rank, self.slot_capacity, self.emit_order,
                        self.slot_rows, self.slot_maxlen, self.slot_row_off, self.slot_tile_off, self.slot_tokens,
                        self.leftover, self.leftover_off, self.ws, stream)
        # both argument sets are read when the call is made: a retry after ODB_E_CAPACITY
        # must pass the reallocated slot arrays, every one of them
        rec = lambda: dict(slot_tokens_approx=self.slot_tokens_approx, row_token_start=self.row_token_start,
                           row_len=self.row_len)
        st, info = odb_align_groups(*args(), raise_on_capacity=False, **rec())
        if st == ODB_E_CAPACITY:
            self._alloc_slots(int(info["required_slot_capacity"]))
            st, info = odb_align_groups(*args(), **rec())
        self.info = info
        return info

    @property
    def num_slots(self) -> int:
        return self.win.num_ranks * int(self.info["steps"])

    def alloc_outputs(self, elems: int):
        torch = self.torch
        elems = max(int(elems), 1)
        if self.outputs is None or self.outputs[0].numel() < elems:
            self.outputs = tuple(torch.empty(elems, dtype=torch.int32, device=self.device) for _ in range(4))
            # the allocator may hand out memory freed by work still queued on the current
            # stream; the library may write it on another stream
            _sync_current(self.device)
        return self.outputs

    def collate(self, stream=None):
        P = int(self.info["padded_elems"])
        outs = self.alloc_outputs(P)
        odb_collate(self.win, self.num_slots, self.emit_order, self.slot_rows, self.slot_maxlen, self.slot_row_off,
                    self.slot_tile_off, self.pad_id, P, *outs, self.ws, stream, row_token_start=self.row_token_start,
                    row_len=self.row_len)
        return tuple(o[:P] for o in outs)

    def loss_weights(self, mode: int = ODB_WEIGHT_TOKEN_EXACT, stream=None):
        """Per-slot loss-scaling weights (rank-major, W * S) and the per-step sums of real
        tokens and samples over ranks, as device tensors."""
        torch = self.torch
        S = int(self.info["steps"])
        K = self.num_slots
        if getattr(self, "_weights", None) is None or self._weights[0].numel() < max(K, 1) \
                or self._weights[1].numel() < max(S, 1):
            self._weights = (torch.empty(max(K, 1), dtype=torch.float64, device=self.device),
                             torch.empty(max(S, 1), dtype=torch.int64, device=self.device),
                             torch.empty(max(S, 1), dtype=torch.int64, device=self.device))
        wt, st, ss = self._weights
        odb_loss_weights(self.win.num_ranks, S, mode, self.slot_rows, self.slot_tokens, self.slot_tokens_approx,
                         wt, st, ss, stream)
        return wt[:K], st[:S], ss[:S]

    def run(self, stream=None):
        self.form(stream)
        self.align(stream)
        return self.collate(stream)


def stream_round_bound(num_samples: int, num_ranks: int, buffer_size: int, rate) -> int:
    """Rounds one logical iteration can take: at most ceil(N/W) emitting rounds, between
    them at most ceil(buffer_size / min rate) fill rounds, and the stop round."""
    q = -(-int(num_samples) // int(num_ranks)) if num_samples else 0
    fill = -(-int(buffer_size) // int(np.min(rate)))
    return q + (q + 1) * fill + 2


class StreamPipeline:
    """Device buffers of one streaming iteration (odb_stream_plan) and its collate and
    loss weights (odb_collate / odb_loss_weights on the streaming plan)."""

    def __init__(self, win: DeviceWindow, perm, budget: int, buffer_size: int = 1024, depth: Optional[int] = None,
                 rate=None, mode: str = "join", quota: int = 0, capacity=None, pad_id: int = 0,
                 max_rounds: Optional[int] = None, slot_capacity: Optional[int] = None):
        import torch

        self.torch = torch
        self.win = win
        self.perm = perm
        self.budget = int(budget)
        W, N = win.num_ranks, win.num_samples
        self.W, self.N = W, N
        self.q = -(-N // W) if N else 0
        self.M = self.q * W
        depth = int(buffer_size if depth is None else depth)
        rate = np.full(W, buffer_size, np.int32) if rate is None else np.ascontiguousarray(rate, dtype=np.int32)
        self.rate = rate
        self.cap = None if capacity is None else np.ascontiguousarray(capacity, dtype=np.int64)
        if max_rounds is None:
            max_rounds = stream_round_bound(N, W, buffer_size, rate)
        self.params = StreamParams(ODB_MODE_NONJOIN_QUOTA if mode == "nonjoin" else ODB_MODE_JOIN, int(buffer_size),
                                   depth, 0, int(quota), rate.ctypes.data_as(ctypes.c_void_p).value,
                                   None if self.cap is None else self.cap.ctypes.data_as(ctypes.c_void_p).value,
                                   int(max_rounds))
        self.pad_id = int(pad_id)
        dev = win.token_offsets.device
        self.device = dev
        m1 = max(self.M, 1)
        self.emit_order = torch.empty(m1, dtype=torch.int32, device=dev)
        self.emit_views = torch.empty(m1, dtype=torch.int32, device=dev)
        self.row_token_start = torch.empty(m1, dtype=torch.int64, device=dev)
        self.row_len = torch.empty(m1, dtype=torch.int32, device=dev)
        self.left_views = torch.empty(m1, dtype=torch.int32, device=dev)
        self.left_off = torch.empty(W + 1, dtype=torch.int64, device=dev)
        self._alloc_slots(max(int(slot_capacity if slot_capacity is not None else W * max(self.q, 1)), W))
        self.trace = (StreamRound * max(int(max_rounds), 1))()
        self.info = None
        self.outputs = None

    def _alloc_slots(self, cap: int):
        torch = self.torch
        cap = (cap + self.W - 1) // self.W * self.W
        self.slot_capacity = cap
        d = self.device
        self.slot_rows = torch.empty(cap, dtype=torch.int32, device=d)
        self.slot_maxlen = torch.empty(cap, dtype=torch.int32, device=d)
        self.slot_tokens = torch.empty(cap, dtype=torch.int64, device=d)
        self.slot_tokens_approx = torch.empty(cap, dtype=torch.float64, device=d)
        self.slot_row_off = torch.empty(cap + 1, dtype=torch.int64, device=d)
        self.slot_tile_off = torch.empty(cap + 1, dtype=torch.int64, device=d)
        size = load().odb_stream_workspace_size(self.win.ref, self.params.depth, cap, self.params.max_rounds)
        if size == 0:
            _check(ODB_E_INVALID_ARG)
        self.ws = torch.empty(size, dtype=torch.uint8, device=d)
        # buffers may be used on another stream than the one they were allocated on
        _sync_current(d)

    def _call(self, stream):
        info = StreamInfo()
        st = load().odb_stream_plan(self.win.ref, _dptr(self.perm), self.budget, ctypes.byref(self.params),
                                    self.slot_capacity, _dptr(self.emit_order), _dptr(self.emit_views),
                                    _dptr(self.row_token_start), _dptr(self.row_len), _dptr(self.slot_rows), _dptr(self.slot_maxlen), _dptr(self.slot_row_off),
                                    _dptr(self.slot_tile_off), _dptr(self.slot_tokens),
                                    _dptr(self.slot_tokens_approx), _dptr(self.left_views), _dptr(self.left_off),
                                    ctypes.cast(self.trace, ctypes.c_void_p), ctypes.byref(info), _dptr(self.ws),
                                    self.ws.numel(), _stream(stream))
        return st, info.as_dict()

    def plan(self, stream=None) -> dict:
        st, info = self._call(stream)
        if st == ODB_E_CAPACITY and info["required_slot_capacity"] > self.slot_capacity:
            self._alloc_slots(int(info["required_slot_capacity"]))
            st, info = self._call(stream)
        _check(st)
        self.info = info
        return info

    def trace_array(self) -> np.ndarray:
        """Rounds as rows (kind, target, emitted, phi)."""
        n = int(self.info["rounds"])
        return np.array([(self.trace[i].kind, self.trace[i].target, self.trace[i].emitted, self.trace[i].phi)
                         for i in range(n)], dtype=np.int64).reshape(-1, 4)

    @property
    def num_slots(self) -> int:
        return self.W * int(self.info["steps"])

    def collate(self, stream=None):
        torch = self.torch
        P = int(self.info["padded_elems"])
        if self.outputs is None or self.outputs[0].numel() < max(P, 1):
            self.outputs = tuple(torch.empty(max(P, 1), dtype=torch.int32, device=self.device) for _ in range(4))
            _sync_current(self.device)
        odb_collate(self.win, self.num_slots, self.emit_order, self.slot_rows, self.slot_maxlen, self.slot_row_off,
                    self.slot_tile_off, self.pad_id, P, *self.outputs, self.ws, stream,
                    row_token_start=self.row_token_start, row_len=self.row_len)
        return tuple(o[:P] for o in self.outputs)

    def loss_weights(self, mode: int = ODB_WEIGHT_TOKEN_EXACT, stream=None):
        """As Pipeline.loss_weights; the output buffers are kept and reused (views of
        them are returned), so a call on another stream never writes freed memory."""
        torch = self.torch
        S, K = int(self.info["steps"]), self.num_slots
        if getattr(self, "_weights", None) is None or self._weights[0].numel() < max(K, 1) \
                or self._weights[1].numel() < max(S, 1):
            self._weights = (torch.empty(max(K, 1), dtype=torch.float64, device=self.device),
                             torch.empty(max(S, 1), dtype=torch.int64, device=self.device),
                             torch.empty(max(S, 1), dtype=torch.int64, device=self.device))
        wt, st, ss = self._weights
        odb_loss_weights(self.W, S, mode, self.slot_rows, self.slot_tokens, self.slot_tokens_approx, wt, st, ss,
                         stream)
        return wt[:K], st[:S], ss[:S]
