"""Seeded synthetic ODB windows.

This module only *draws inputs*: per-rank sample lengths, the CSR token offsets
that those lengths imply, token ids from a counter-based hash, and optional
sampler-view identity maps.  It holds none of the batching method's arithmetic
(no B(l), no grouping, no alignment, no collation), so both the CPU oracle and
the HIP path can be fed from it without sharing any of the method's code.

Length recipes follow the workload shapes the paper measures on (the per-dataset
length table and the six synthetic correctness-audit distributions in the
experimental-setup appendix); the datasets themselves are not available, so these
parametric draws stand in for them.

Lognormal parameterisation: ``mean`` and ``cv`` describe the *unclipped*
lognormal, i.e. sigma^2 = ln(1 + cv^2), mu = ln(mean) - sigma^2 / 2.  Values are
rounded half-to-even (``numpy.rint``) and then clipped.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Callable, Dict, List, Optional

import numpy as np

VOCAB = 151936
_M32 = 0xFFFFFFFF


# --------------------------------------------------------------------------------------
# Counter-based token ids.  tok(k) depends only on the global token index k, so any
# slice of the CSR token stream can be regenerated anywhere (host or device) without
# materialising the rest.  The mixer is the public-domain "lowbias32" integer hash
# (two multiply-xorshift rounds); multiplications are split into 16-bit halves so every
# intermediate stays below 2^63 in signed int64 arithmetic on any torch device.
# --------------------------------------------------------------------------------------
def _mul32(x, c: int):
    lo = c & 0xFFFF
    hi = c >> 16
    return (x * lo + (((x * hi) & 0xFFFF) << 16)) & _M32


def _mix32(x):
    x = x ^ (x >> 16)
    x = _mul32(x, 0x7FEB352D)
    x = x ^ (x >> 15)
    x = _mul32(x, 0x846CA68B)
    x = x ^ (x >> 16)
    return x


TOKEN_SEED = 0x5EED


def token_ids(k):
    """Token id at global CSR position ``k`` (int64 torch tensor or numpy array).

    Returns the same container type with int64 values uniform on [0, VOCAB).
    """
    hi = _mix32(((k >> 32) + TOKEN_SEED) & _M32)
    h = _mix32((k & _M32) ^ hi)
    return (h * VOCAB) >> 32


def fill_tokens_torch(total: int, device, chunk: int = 1 << 27):
    """Materialise the whole token stream [0, total) as int32 on ``device``."""
    import torch

    out = torch.empty(total, dtype=torch.int32, device=device)
    for s in range(0, total, chunk):
        e = min(total, s + chunk)
        idx = torch.arange(s, e, dtype=torch.int64, device=device)
        out[s:e] = token_ids(idx).to(torch.int32)
        del idx
    return out


def device_tensors(w: "Window", device="cuda", tokens=None):
    """Device copies of a window's CSR offsets, token stream and identity map.

    Tokens are generated directly on the device unless given.  Returns
    (token_offsets int64, tokens int32, identity int64 or None).
    """
    import torch

    tok_off = torch.from_numpy(w.tok_off).to(device)
    if tokens is None:
        tokens = fill_tokens_torch(max(w.total_tokens, 1), device)
    ident = None if w.identity is None else torch.from_numpy(w.identity).to(device)
    return tok_off, tokens, ident


def tokens_numpy(start: int, stop: int) -> np.ndarray:
    idx = np.arange(start, stop, dtype=np.int64)
    return token_ids(idx).astype(np.int32)


# --------------------------------------------------------------------------------------
# Window container
# --------------------------------------------------------------------------------------
@dataclass
class Window:
    """A window of realised samples split over ``W`` simulated ranks.

    rank_off[W+1]  int64, rank r owns samples [rank_off[r], rank_off[r+1])
    lengths[n]     int64, realised token length of every sample (>= 1 unless a test
                   deliberately builds invalid data)
    tok_off[n+1]   int64, CSR offsets, tok_off[i+1] - tok_off[i] = lengths[i]
    identity[n]    optional int64 dataset identity of each sampler view
    """

    name: str
    rank_off: np.ndarray
    lengths: np.ndarray
    budget: int
    mode: str = "join"            # "join" | "nonjoin"
    quota: int = 0                # non-join sample quota Q
    capacity: Optional[np.ndarray] = None   # per-rank output-slot capacity C_r
    identity: Optional[np.ndarray] = None
    num_identities: int = 0
    tok_off: np.ndarray = field(init=False)

    def __post_init__(self):
        self.rank_off = np.ascontiguousarray(self.rank_off, dtype=np.int64)
        self.lengths = np.ascontiguousarray(self.lengths, dtype=np.int64)
        self.tok_off = np.zeros(len(self.lengths) + 1, dtype=np.int64)
        np.cumsum(self.lengths, out=self.tok_off[1:])
        if self.identity is not None:
            self.identity = np.ascontiguousarray(self.identity, dtype=np.int64)

    @property
    def W(self) -> int:
        return len(self.rank_off) - 1

    @property
    def n(self) -> int:
        return len(self.lengths)

    @property
    def total_tokens(self) -> int:
        return int(self.tok_off[-1])

    def tokens_numpy(self) -> np.ndarray:
        return tokens_numpy(0, self.total_tokens)


def window_from_ranks(name: str, per_rank: List[np.ndarray], budget: int, **kw) -> Window:
    lens = [np.asarray(x, dtype=np.int64).reshape(-1) for x in per_rank]
    off = np.zeros(len(lens) + 1, dtype=np.int64)
    off[1:] = np.cumsum([len(x) for x in lens])
    flat = np.concatenate(lens) if lens else np.zeros(0, dtype=np.int64)
    return Window(name=name, rank_off=off, lengths=flat, budget=budget, **kw)


# --------------------------------------------------------------------------------------
# Length recipes
# --------------------------------------------------------------------------------------
def lognormal(rng: np.random.Generator, mean: float, cv: float, size: int) -> np.ndarray:
    s2 = math.log1p(cv * cv)
    mu = math.log(mean) - s2 / 2.0
    return rng.lognormal(mu, math.sqrt(s2), size)


def _clip_round(x: np.ndarray, lo: int, hi: int) -> np.ndarray:
    return np.clip(np.rint(x), lo, hi).astype(np.int64)


def _draw_lognormal_ranks(seed, W, n_r, mean, cv, lo, hi):
    rng = np.random.default_rng(seed)
    return [_clip_round(lognormal(rng, mean, cv, n_r), lo, hi) for _ in range(W)]


def _draw_multimodal_ranks(seed, W, n_r):
    # text part ~ LN(300, 0.7), at least 1 token, plus K ~ Poisson(1.5) images, each
    # expanding to 4*U{16..640} visual tokens (multiples of 4 in [64, 2560]).
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(W):
        text = np.maximum(1, np.rint(lognormal(rng, 300.0, 0.7, n_r))).astype(np.int64)
        k = rng.poisson(1.5, n_r).astype(np.int64)
        img = rng.integers(16, 641, size=int(k.sum()), dtype=np.int64) * 4
        owner = np.repeat(np.arange(n_r), k)
        vis = np.bincount(owner, weights=img, minlength=n_r).astype(np.int64)
        out.append(np.clip(text + vis, 1, 16384).astype(np.int64))
    return out


def _draw_bimodal_ranks(seed, W, n_r):
    # 90% LN(200, 0.3) / 10% LN(8000, 0.3), clipped to [1, 32768].
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(W):
        u = rng.random(n_r)
        a = lognormal(rng, 200.0, 0.3, n_r)
        b = lognormal(rng, 8000.0, 0.3, n_r)
        out.append(_clip_round(np.where(u < 0.9, a, b), 1, 32768))
    return out


@dataclass(frozen=True)
class Workload:
    name: str
    W: int
    n_per_rank: int
    budget: int
    mode: str
    description: str
    draw: Callable[[int], List[np.ndarray]]
    seed: int = 0

    def window(self, ranks: Optional[int] = None) -> Window:
        per_rank = self.draw(self.seed)
        if ranks is not None:
            per_rank = per_rank[:ranks]
        n = sum(len(x) for x in per_rank)
        quota = n if self.mode == "nonjoin" else 0
        return window_from_ranks(self.name, per_rank, self.budget, mode=self.mode, quota=quota)


# The five benchmark workloads (sizes as stated: simulated ranks x samples per rank).
WORKLOADS: Dict[str, Workload] = {
    "ln512_w2x2048": Workload(
        "ln512_w2x2048", 2, 2048, 16384, "join",
        "2 ranks x 2,048 samples, lognormal mean 512 CV 0.5 clipped [16,4096], budget 16384, join",
        lambda s: _draw_lognormal_ranks(s, 2, 2048, 512.0, 0.5, 16, 4096)),
    "text_w8x65536": Workload(
        "text_w8x65536", 8, 65536, 65536, "join",
        "8 ranks x 65,536 text-like samples, lognormal mean 700 CV 0.8 clipped [8,8192], budget 65536, join",
        lambda s: _draw_lognormal_ranks(s, 8, 65536, 700.0, 0.8, 8, 8192)),
    "mm_w8x262144": Workload(
        "mm_w8x262144", 8, 262144, 131072, "join",
        "8 ranks x 262,144 multimodal samples, text LN(300,0.7) + Poisson(1.5) images x 4*U{16..640} "
        "visual tokens, clipped [1,16384], budget 131072, join",
        lambda s: _draw_multimodal_ranks(s, 8, 262144)),
    "bimodal_w16x65536": Workload(
        "bimodal_w16x65536", 16, 65536, 262144, "nonjoin",
        "16 ranks x 65,536 samples, 90% LN(200,0.3) / 10% LN(8000,0.3) clipped [1,32768], budget 262144, "
        "non-join sample-quota mode with Q = N",
        lambda s: _draw_bimodal_ranks(s, 16, 65536)),
    "ln480_w64x262144": Workload(
        "ln480_w64x262144", 64, 262144, 131072, "join",
        "64 ranks x 262,144 samples (16,777,216 total), lognormal mean 480 CV 1.2 clipped [8,16384], "
        "budget 131072, join, full collate",
        lambda s: _draw_lognormal_ranks(s, 64, 262144, 480.0, 1.2, 8, 16384)),
}

# Order of the five workloads, smallest first.
WORKLOAD_ORDER = ["ln512_w2x2048", "text_w8x65536", "mm_w8x262144", "bimodal_w16x65536", "ln480_w64x262144"]


# --------------------------------------------------------------------------------------
# The six 1000-sample correctness-audit distributions (experimental-setup appendix).
# The paper names longtail "90% short / 10% long" and bimodal "50/50" without ranges;
# the ranges below are this repository's choice.
# --------------------------------------------------------------------------------------
def audit_lengths(kind: str, n: int = 1000, seed: int = 0) -> np.ndarray:
    rng = np.random.default_rng(seed)
    if kind == "uniform_narrow":
        return rng.integers(64, 513, n, dtype=np.int64)
    if kind == "uniform_wide":
        return rng.integers(64, 2049, n, dtype=np.int64)
    if kind == "longtail":
        short = rng.integers(32, 257, n, dtype=np.int64)
        long_ = rng.integers(1024, 2049, n, dtype=np.int64)
        return np.where(rng.random(n) < 0.9, short, long_)
    if kind == "bimodal":
        a = rng.integers(64, 257, n, dtype=np.int64)
        b = rng.integers(1536, 2049, n, dtype=np.int64)
        return np.where(rng.random(n) < 0.5, a, b)
    if kind == "all_long":
        return rng.integers(1800, 2049, n, dtype=np.int64)
    if kind == "all_short":
        return rng.integers(32, 65, n, dtype=np.int64)
    raise ValueError(kind)


AUDIT_KINDS = ["uniform_narrow", "uniform_wide", "longtail", "bimodal", "all_long", "all_short"]


def sampler_views(num_identities: int, W: int, seed: int = 0):
    """Sampler views the way a distributed sampler with drop_last=False assigns them.

    A seeded permutation of the identities is padded by wrap-around repetition of its
    head to M = W * ceil(N / W) entries and dealt to ranks by striding (rank r takes
    entries r, r+W, ...).  Returns (per-rank identity arrays, q, P).
    """
    q = -(-num_identities // W)
    M = W * q
    perm = np.random.default_rng(seed).permutation(num_identities).astype(np.int64)
    pad = M - num_identities
    if pad:
        reps = -(-pad // num_identities)
        perm = np.concatenate([perm] + [perm] * reps)[:M]
    return [perm[r:M:W] for r in range(W)], q, pad


def audit_window(kind: str, W: int, n: int = 1000, budget: int = 4096, seed: int = 0,
                 mode: str = "join", quota: int = 0) -> Window:
    """One audit distribution dealt to W ranks through sampler views (identity map set)."""
    lens_by_id = audit_lengths(kind, n, seed)
    views, q, pad = sampler_views(n, W, seed + 1)
    ident = np.concatenate(views)
    per_rank = [lens_by_id[v] for v in views]
    w = window_from_ranks(f"audit_{kind}_w{W}", per_rank, budget, mode=mode, quota=quota,
                          identity=ident, num_identities=n)
    return w
