"""CPU reference oracle for the ODB window pipeline -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py``
may import this package.  It wraps ``odb_oracle.cpp`` (plain single-threaded C++,
built with g++) and adds :func:`collate_elements`, a numpy statement of the collate
rule evaluated at individual output positions so full-size GPU outputs can be spot
checked without materialising the whole oracle output.

The oracle shares no code with the HIP library: it is compiled from its own source by
its own compiler, and neither side imports or links the other.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "odb_oracle.cpp")
_LIB = os.path.join(_HERE, "libodb_oracle.so")

MODE_JOIN = 0
MODE_NONJOIN = 1
STOP_DRAINED, STOP_QUOTA, STOP_RANK_FINISHED = 0, 1, 2
WEIGHT_SAMPLE, WEIGHT_TOKEN_APPROX, WEIGHT_TOKEN_EXACT = 0, 1, 2


def build(force: bool = True) -> str:
    """Compile the oracle with g++ (always when ``force``)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp"
        # -ffp-contract=off: every fp64 product and sum is rounded on its own, as written
        subprocess.check_call(["g++", "-O2", "-std=c++17", "-ffp-contract=off", "-shared", "-fPIC", "-Wall", "-Wextra",
                               _SRC, "-o", tmp])
        os.replace(tmp, _LIB)
    return _LIB


class _Info(ctypes.Structure):
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
        ("second_gather_rounds", ctypes.c_int64),
    ]


class _StreamInfo(ctypes.Structure):
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
    ]


class _StreamRound(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("reserved0", ctypes.c_int32), ("target", ctypes.c_int64),
                ("emitted", ctypes.c_int64), ("phi", ctypes.c_int64)]


ROUND_EMIT, ROUND_SKIP, ROUND_STOP = 0, 1, 2

_lib = None


def _bind(path: str):
    lib = ctypes.CDLL(path)
    P = ctypes.c_void_p
    lib.oracle_plan.restype = P
    lib.oracle_plan.argtypes = [ctypes.c_int32, ctypes.c_int64, P, P, P, ctypes.c_int64,
                                ctypes.c_int64, ctypes.c_int32, ctypes.c_int64, P]
    lib.oracle_last_error.restype = ctypes.c_char_p
    lib.oracle_free.argtypes = [P]
    lib.oracle_info.argtypes = [P, ctypes.POINTER(_Info)]
    lib.oracle_form.argtypes = [P, P, P, P, P]
    lib.oracle_slots.argtypes = [P, P, P, P, P, P]
    lib.oracle_emit.argtypes = [P, P, P, P]
    lib.oracle_collate.argtypes = [P, P, P, ctypes.c_int32, P, P, P, P]
    lib.oracle_collate_rank.argtypes = [P, ctypes.c_int32, P, P, ctypes.c_int32, P, P, P, P]
    lib.oracle_collate_rank.restype = ctypes.c_int
    lib.oracle_collate_rank_all.argtypes = [P, ctypes.c_int32, P, P, ctypes.c_int32, P, P, P, P]
    lib.oracle_collate_rank_all.restype = ctypes.c_int
    lib.oracle_round_targets.argtypes = [P, P]
    lib.oracle_slots_approx.argtypes = [P, P]
    lib.oracle_loss_weights.argtypes = [P, ctypes.c_int32, P, P, P]
    lib.oracle_loss_weights.restype = ctypes.c_int
    lib.oracle_stream.restype = P
    lib.oracle_stream.argtypes = [ctypes.c_int32, ctypes.c_int64, P, P, ctypes.c_int64, ctypes.c_int32,
                                  ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, P, P, ctypes.c_int64]
    lib.oracle_stream_free.argtypes = [P]
    lib.oracle_stream_info.argtypes = [P, ctypes.POINTER(_StreamInfo)]
    lib.oracle_stream_trace.argtypes = [P, P]
    lib.oracle_stream_views.argtypes = [P, P, P, P]
    return lib


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build(force=True)
        _lib = _bind(_LIB)
    return _lib


def _use_library(path: str) -> None:
    """Test hook: make every oracle call go to the library at `path` (used to check that
    the pins reject deliberately mutated builds of the oracle)."""
    global _lib
    _lib = _bind(path)


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


class OracleError(ValueError):
    pass


@dataclass
class Plan:
    W: int
    n: int
    info: dict
    # first formation
    order: np.ndarray
    sorted_len: np.ndarray
    group_index: np.ndarray
    groups_per_rank: np.ndarray
    # aligned plan
    slot_rows: np.ndarray
    slot_maxlen: np.ndarray
    slot_row_off: np.ndarray
    slot_tile_off: np.ndarray
    slot_tokens: np.ndarray
    slot_tokens_approx: np.ndarray
    emit_order: np.ndarray
    leftover: np.ndarray
    leftover_off: np.ndarray
    round_targets: np.ndarray
    _handle: int = 0

    @property
    def steps(self) -> int:
        return int(self.info["steps"])

    @property
    def num_slots(self) -> int:
        return self.W * self.steps

    @property
    def padded_elems(self) -> int:
        return int(self.info["padded_elems"])

    def __del__(self):
        if self._handle and _lib is not None:
            _lib.oracle_free(ctypes.c_void_p(self._handle))
            self._handle = 0

    def collate(self, tok_off: np.ndarray, tokens: np.ndarray, pad_id: int = 0):
        """Full collate: four flat int32 arrays of length padded_elems."""
        lib = _load()
        P = self.padded_elems
        outs = [np.empty(P, dtype=np.int32) for _ in range(4)]
        tok_off = np.ascontiguousarray(tok_off, dtype=np.int64)
        tokens = np.ascontiguousarray(tokens, dtype=np.int32)
        lib.oracle_collate(ctypes.c_void_p(self._handle), _ptr(tok_off), _ptr(tokens), int(pad_id),
                           *[_ptr(o) for o in outs])
        return tuple(outs)

    def loss_weights(self, mode: int = WEIGHT_TOKEN_EXACT):
        """Loss-scaling weights of every slot (rank-major, like the slot tables) and the
        per-step sums of real tokens and of samples over ranks (Eq. 2, App. B)."""
        lib = _load()
        K, S = self.num_slots, self.steps
        wt = np.empty(K, np.float64)
        st = np.empty(S, np.int64)
        ss = np.empty(S, np.int64)
        if lib.oracle_loss_weights(ctypes.c_void_p(self._handle), int(mode), _ptr(wt), _ptr(st), _ptr(ss)) != 0:
            raise OracleError(f"unknown loss-weight mode {mode}")
        return wt, st, ss

    def collate_rank(self, r: int, tok_off: np.ndarray, rank_tokens: np.ndarray, pad_id: int = 0,
                     whole_stream: bool = False):
        """Rank r's tiles only: four int32 arrays covering output positions
        [slot_tile_off[r * steps], slot_tile_off[(r + 1) * steps]).  ``rank_tokens`` holds
        the CSR positions owned by rank r's samples (from its first sample's offset), or,
        with ``whole_stream``, the whole token stream (streaming plans, whose rows are
        identities from anywhere in the dataset)."""
        lib = _load()
        if not 0 <= r < self.W:
            raise OracleError(f"rank {r} out of range")
        S = self.steps
        P = int(self.slot_tile_off[(r + 1) * S] - self.slot_tile_off[r * S])
        outs = [np.empty(P, dtype=np.int32) for _ in range(4)]
        tok_off = np.ascontiguousarray(tok_off, dtype=np.int64)
        rank_tokens = np.ascontiguousarray(rank_tokens, dtype=np.int32)
        fn = lib.oracle_collate_rank_all if whole_stream else lib.oracle_collate_rank
        if fn(ctypes.c_void_p(self._handle), int(r), _ptr(tok_off), _ptr(rank_tokens), int(pad_id),
              *[_ptr(o) for o in outs]) != 0:
            raise OracleError(f"rank {r} out of range")
        return tuple(outs)


def plan(rank_off, tok_off, budget: int, mode: int = MODE_JOIN, quota: int = 0,
         capacity=None, identity=None, num_identities: int = 0) -> Plan:
    lib = _load()
    rank_off = np.ascontiguousarray(rank_off, dtype=np.int64)
    tok_off = np.ascontiguousarray(tok_off, dtype=np.int64)
    W = len(rank_off) - 1
    n = len(tok_off) - 1
    cap = None if capacity is None else np.ascontiguousarray(capacity, dtype=np.int64)
    ident = None if identity is None else np.ascontiguousarray(identity, dtype=np.int64)
    h = lib.oracle_plan(W, n, _ptr(rank_off), _ptr(tok_off), _ptr(ident), int(num_identities),
                        int(budget), int(mode), int(quota), _ptr(cap))
    if not h:
        raise OracleError(lib.oracle_last_error().decode())
    info = _Info()
    lib.oracle_info(ctypes.c_void_p(h), ctypes.byref(info))
    d = {f: getattr(info, f) for f, _ in _Info._fields_}
    S = d["steps"]
    K = W * S
    order = np.empty(n, np.int32)
    slen = np.empty(n, np.int32)
    gidx = np.empty(n, np.int32)
    G = np.empty(W, np.int32)
    lib.oracle_form(ctypes.c_void_p(h), _ptr(order), _ptr(slen), _ptr(gidx), _ptr(G))
    rows = np.empty(K, np.int32)
    mx = np.empty(K, np.int32)
    ro = np.empty(K + 1, np.int64)
    to = np.empty(K + 1, np.int64)
    tk = np.empty(K, np.int64)
    lib.oracle_slots(ctypes.c_void_p(h), _ptr(rows), _ptr(mx), _ptr(ro), _ptr(to), _ptr(tk))
    ta = np.empty(K, np.float64)
    lib.oracle_slots_approx(ctypes.c_void_p(h), _ptr(ta))
    emit = np.empty(d["emitted_samples"], np.int32)
    left = np.empty(d["leftover_samples"], np.int32)
    loff = np.empty(W + 1, np.int64)
    lib.oracle_emit(ctypes.c_void_p(h), _ptr(emit), _ptr(left), _ptr(loff))
    rt = np.empty(d["rounds"], np.int64)
    lib.oracle_round_targets(ctypes.c_void_p(h), _ptr(rt))
    return Plan(W, n, d, order, slen, gidx, G, rows, mx, ro, to, tk, ta, emit, left, loff, rt, _handle=h)


def plan_window(w, **overrides) -> Plan:
    """Convenience: run :func:`plan` on a ``synth.Window``."""
    kw = dict(budget=w.budget, mode=MODE_NONJOIN if w.mode == "nonjoin" else MODE_JOIN,
              quota=w.quota, capacity=w.capacity, identity=w.identity,
              num_identities=w.num_identities)
    kw.update(overrides)
    return plan(w.rank_off, w.tok_off, **kw)


def collate_elements(p: Plan, tok_off: np.ndarray, token_at, idx: np.ndarray, pad_id: int = 0):
    """Collate values at flat output positions ``idx`` (Sec. 2.1 pad-to-max rule).

    ``token_at(k)`` returns the token ids at global CSR positions ``k`` (numpy int64).
    Returns four int32 arrays aligned with ``idx``.
    """
    idx = np.asarray(idx, dtype=np.int64)
    k = np.searchsorted(p.slot_tile_off, idx, side="right") - 1   # slot holding each element
    local = idx - p.slot_tile_off[k]
    ml = p.slot_maxlen[k].astype(np.int64)
    row = local // ml
    col = local - row * ml
    s = p.emit_order[p.slot_row_off[k] + row].astype(np.int64)
    start = tok_off[s]
    l = tok_off[s + 1] - start
    real = col < l
    tok = np.where(real, token_at(np.where(real, start + col, 0)), 0).astype(np.int32)
    ids = np.where(real, tok, pad_id).astype(np.int32)
    lab = np.where(real, tok, -100).astype(np.int32)
    msk = real.astype(np.int32)
    pos = np.where(real, col, 0).astype(np.int32)
    return ids, lab, msk, pos


def length_sketch(tok_off: np.ndarray, ids: Optional[np.ndarray], budget: int) -> dict:
    """ROI sketch of realised lengths (Sec. 1 defines CV = sigma / mu of post-pipeline
    lengths; the practical-guidance section screens a 1k-5k sketch with CV and
    f_s = Pr[l < L_max / 4], flagging CV >= 0.8 or f_s > 0.2 as high ROI).

    ``ids`` are the sketched sample ids (None: every sample).  sigma is the population
    standard deviation (reading: the sketch is the population being described).  The
    moments are exact Python integers; CV is sqrt(sum (l - mu)^2 / n) / mu evaluated as
    one correctly rounded conversion of the exact rational CV^2 and one square root.
    """
    from fractions import Fraction
    import math

    tok_off = np.asarray(tok_off, dtype=np.int64)
    n_all = len(tok_off) - 1
    ids = np.arange(n_all, dtype=np.int64) if ids is None else np.asarray(ids, dtype=np.int64)
    if ids.size and (ids.min() < 0 or ids.max() >= n_all):
        raise OracleError("sketch id outside the window")
    lens = [int(tok_off[i + 1] - tok_off[i]) for i in ids]
    if any(l < 1 for l in lens):
        raise OracleError("sample length < 1")
    n = len(lens)
    out = dict(samples=n, short_samples=0, sum_len=0, sum_sq=0, min_len=0, max_len=0,
               mean=0.0, cv=0.0, short_fraction=0.0, high_roi=0)
    if n == 0:
        return out
    s1 = sum(lens)
    s2 = sum(l * l for l in lens)
    mu = Fraction(s1, n)
    var = sum((Fraction(l) - mu) ** 2 for l in lens) / n if n <= 20000 else Fraction(n * s2 - s1 * s1, n * n)
    short = sum(1 for l in lens if Fraction(l) < Fraction(budget, 4))
    cv = math.sqrt(float(var / (mu * mu)))
    out.update(short_samples=short, sum_len=s1, sum_sq=s2, min_len=min(lens), max_len=max(lens),
               mean=s1 / n, cv=cv, short_fraction=short / n, high_roi=int(cv >= 0.8 or short / n > 0.2))
    return out


class StreamPlan(Plan):
    """One logical iteration of the unified loop: a window-format plan over identities
    plus the streaming record (``sinfo``, per-round ``trace``, emitted and un-emitted
    views)."""

    def __init__(self, handle, W, N, sinfo, trace, emit_views, left_views, left_off):
        lib = _load()
        info = _Info()
        lib.oracle_info(ctypes.c_void_p(handle), ctypes.byref(info))
        d = {f: getattr(info, f) for f, _ in _Info._fields_}
        S = d["steps"]
        K = W * S
        rows = np.empty(K, np.int32)
        mx = np.empty(K, np.int32)
        ro = np.empty(K + 1, np.int64)
        to = np.empty(K + 1, np.int64)
        tk = np.empty(K, np.int64)
        lib.oracle_slots(ctypes.c_void_p(handle), _ptr(rows), _ptr(mx), _ptr(ro), _ptr(to), _ptr(tk))
        ta = np.empty(K, np.float64)
        lib.oracle_slots_approx(ctypes.c_void_p(handle), _ptr(ta))
        emit = np.empty(d["emitted_samples"], np.int32)
        left = np.empty(d["leftover_samples"], np.int32)
        loff = np.empty(W + 1, np.int64)
        lib.oracle_emit(ctypes.c_void_p(handle), _ptr(emit), _ptr(left), _ptr(loff))
        z32, z64 = np.zeros(0, np.int32), np.zeros(0, np.int64)
        super().__init__(W, N, d, z32, z32, z32, z32, rows, mx, ro, to, tk, ta, emit, left, loff, z64,
                         _handle=0)
        self._stream_handle = handle
        self.sinfo = sinfo
        self.trace = trace
        self.emit_views = emit_views
        self.left_views = left_views
        self.left_off = left_off

    @property
    def _h(self):
        return self._stream_handle

    def __del__(self):
        if getattr(self, "_stream_handle", 0) and _lib is not None:
            _lib.oracle_stream_free(ctypes.c_void_p(self._stream_handle))
            self._stream_handle = 0

    def loss_weights(self, mode: int = WEIGHT_TOKEN_EXACT):
        self._handle = self._stream_handle
        try:
            return super().loss_weights(mode)
        finally:
            self._handle = 0

    def collate(self, tok_off, tokens, pad_id: int = 0):
        self._handle = self._stream_handle
        try:
            return super().collate(tok_off, tokens, pad_id)
        finally:
            self._handle = 0

    def collate_rank(self, r: int, tok_off, tokens, pad_id: int = 0, whole_stream: bool = True):
        """Rank r's tiles; ``tokens`` is the whole token stream."""
        if not whole_stream:
            raise OracleError("a streaming plan's rows need the whole token stream")
        self._handle = self._stream_handle
        try:
            return super().collate_rank(r, tok_off, tokens, pad_id, whole_stream=True)
        finally:
            self._handle = 0


def stream(tok_off, perm, W: int, budget: int, mode: int = MODE_JOIN, quota: int = 0, buffer_size: int = 1024,
           depth: Optional[int] = None, rate=None, capacity=None, max_rounds: Optional[int] = None) -> StreamPlan:
    """One logical iteration of the unified loop (Sec. 2.3, App. C) over identities
    0..N-1 with lengths from ``tok_off``, the shuffled identity list ``perm``, ``W``
    ranks, the collate buffer size, the outstanding-depth envelope ``depth`` (default
    buffer_size) and per-rank arrival rates (views per round, default buffer_size)."""
    lib = _load()
    tok_off = np.ascontiguousarray(tok_off, dtype=np.int64)
    N = len(tok_off) - 1
    perm = np.ascontiguousarray(perm, dtype=np.int32)
    if len(perm) != N:
        raise OracleError("perm must hold N entries")
    depth = buffer_size if depth is None else int(depth)
    rate = np.full(W, buffer_size, np.int32) if rate is None else np.ascontiguousarray(rate, dtype=np.int32)
    cap = None if capacity is None else np.ascontiguousarray(capacity, dtype=np.int64)
    if max_rounds is None:
        # at most ceil(N/W) emitting rounds, at most ceil(buffer / min rate) fill rounds
        # before each, and the round that observes the stop
        q = -(-N // W) if N else 0
        max_rounds = q + (q + 1) * -(-int(buffer_size) // max(1, int(rate.min()))) + 2
    h = lib.oracle_stream(int(W), N, _ptr(tok_off), _ptr(perm), int(budget), int(mode), int(quota),
                          int(buffer_size), int(depth), _ptr(rate), _ptr(cap), int(max_rounds))
    if not h:
        raise OracleError(lib.oracle_last_error().decode())
    si = _StreamInfo()
    lib.oracle_stream_info(ctypes.c_void_p(h), ctypes.byref(si))
    sinfo = {f: getattr(si, f) for f, _ in _StreamInfo._fields_ if f != "reserved0"}
    tr = (_StreamRound * max(sinfo["rounds"], 1))()
    lib.oracle_stream_trace(ctypes.c_void_p(h), ctypes.cast(tr, ctypes.c_void_p))
    trace = np.array([(tr[i].kind, tr[i].target, tr[i].emitted, tr[i].phi) for i in range(sinfo["rounds"])],
                     dtype=np.int64).reshape(-1, 4)
    ev = np.empty(sinfo["emitted_views"], np.int32)
    lv = np.empty(sinfo["views"] - sinfo["emitted_views"], np.int32)
    lo = np.empty(W + 1, np.int64)
    lib.oracle_stream_views(ctypes.c_void_p(h), _ptr(ev), _ptr(lv), _ptr(lo))
    return StreamPlan(h, int(W), N, sinfo, trace, ev, lv, lo)
