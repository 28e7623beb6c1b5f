"""The pipeline driven from plain C (tests/c_abi/*.c: hipMalloc'd buffers, include/odb.h,
no Python in the loop), compared with the oracle.  Window: grouping, alignment (after the
one retry with the slot capacity the first call reports), the collated tiles (from
odb_collate and from odb_collate_static), the exact token-level loss weights, the
coverage check of the emitted and left-over ids and the length sketch of the whole
window.  Streaming: one logical iteration (round trace, plan,
row records, leftovers, after the same retry), its collated tiles and weights."""
import os
import subprocess

import numpy as np
import pytest

import oracle
import synth
from _parity import INFO_EXACT, PAD_FRACTION_RTOL, log

pytestmark = pytest.mark.gpu

HERE = os.path.dirname(os.path.abspath(__file__))
BIN = os.path.join(HERE, "c_abi", "window_pipeline")
STREAM_BIN = os.path.join(HERE, "c_abi", "stream_pipeline")
INFO_FIELDS = INFO_EXACT[:13] + ["second_gather_rounds", "required_slot_capacity"]
STREAM_FIELDS = ["steps", "rounds", "emit_rounds", "skip_rounds", "stop_reason", "views", "emitted_views",
                 "undelivered_views", "pending_views", "real_tokens", "padded_elems", "max_step_samples", "splits",
                 "overflow_groups", "missing_ids", "duplicate_ids", "bad_views", "second_gather_rounds",
                 "max_outstanding", "required_slot_capacity"]


def _window(case):
    rng = np.random.default_rng(73)
    if case == "join_small":
        per = [np.clip(np.rint(synth.lognormal(rng, 700.0, 0.8, 3000)), 8, 8192) for _ in range(3)]
        return synth.window_from_ranks("c_join_small", per, 16384)
    if case == "nonjoin":
        per = [rng.integers(1, 4000, int(k)) for k in (2500, 900, 4100, 3000)]
        n = sum(len(x) for x in per)
        return synth.window_from_ranks("c_nonjoin", per, 20000, mode="nonjoin", quota=n // 2)
    if case == "multi_block":
        per = [np.clip(np.rint(synth.lognormal(rng, 480.0, 1.2, 20000)), 8, 16384) for _ in range(2)]
        return synth.window_from_ranks("c_multi_block", per, 65536)
    raise ValueError(case)


class _Reader:
    def __init__(self, raw):
        self.raw, self.at = raw, 0

    def take(self, dtype, count):
        a = np.frombuffer(self.raw, dtype=dtype, count=count, offset=self.at)
        self.at += a.nbytes
        return a


@pytest.mark.parametrize("case", ["join_small", "nonjoin", "multi_block"])
def test_window_pipeline_from_c(case, tmp_path):
    assert os.path.exists(BIN), "tests/c_abi/window_pipeline is missing: run __graft_entry__.build()"
    w = _window(case)
    tokens = w.tokens_numpy()
    src, dst = tmp_path / "in.bin", tmp_path / "out.bin"
    with open(src, "wb") as f:
        np.array([w.W, w.n, len(tokens)], np.int64).tofile(f)
        w.rank_off.tofile(f)
        w.tok_off.tofile(f)
        tokens.astype(np.int32).tofile(f)
    mode = 1 if w.mode == "nonjoin" else 0
    log(f"case {w.name}: W={w.W} n={w.n} budget={w.budget} mode={w.mode}")
    r = subprocess.run([BIN, str(src), str(dst), str(w.budget), str(mode), str(w.quota)], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 0, r.stderr

    ref = oracle.plan_window(w)
    rd = _Reader(open(dst, "rb").read())
    info = dict(zip(INFO_FIELDS, rd.take(np.int64, 15).tolist()))
    pad_fraction = float(rd.take(np.float64, 1)[0])
    retries = int(rd.take(np.int64, 1)[0])
    K = w.W * ref.steps
    for f in INFO_FIELDS[:-1]:
        assert info[f] == ref.info[f], (f, info[f], ref.info[f])
    assert info["required_slot_capacity"] == K
    rf = ref.info["pad_fraction"]
    assert abs(pad_fraction - rf) <= PAD_FRACTION_RTOL * max(abs(rf), 1e-300) or pad_fraction == rf
    # the first call had room for one step per rank
    assert retries == (1 if ref.steps > 1 else 0), retries
    n, E, Lf = w.n, ref.info["emitted_samples"], ref.info["leftover_samples"]
    for name, dtype, count, want in [
        ("order", np.int32, n, ref.order), ("sorted_len", np.int32, n, ref.sorted_len),
        ("group_index", np.int32, n, ref.group_index), ("groups_per_rank", np.int32, w.W, ref.groups_per_rank),
        ("emit_order", np.int32, E, ref.emit_order), ("slot_rows", np.int32, K, ref.slot_rows),
        ("slot_maxlen", np.int32, K, ref.slot_maxlen), ("slot_row_off", np.int64, K + 1, ref.slot_row_off),
        ("slot_tile_off", np.int64, K + 1, ref.slot_tile_off), ("slot_tokens", np.int64, K, ref.slot_tokens),
        ("leftover", np.int32, Lf, ref.leftover), ("leftover_off", np.int64, w.W + 1, ref.leftover_off),
    ]:
        assert np.array_equal(rd.take(dtype, count), want), name
    P = ref.padded_elems
    want = ref.collate(w.tok_off, tokens, 0)
    for entry in ("odb_collate", "odb_collate_static"):
        for name, e in zip(["input_ids", "labels", "attention_mask", "position_ids"], want):
            got = rd.take(np.int32, P)
            assert np.array_equal(got, e), (entry, name, int(np.count_nonzero(got != e)))
    assert int(rd.take(np.int32, 1)[0]) == 0, "odb_collate_static status"
    wt = rd.take(np.float64, K)
    ewt, _, _ = ref.loss_weights(oracle.WEIGHT_TOKEN_EXACT)
    assert np.array_equal(wt.view(np.int64), ewt.view(np.int64)), "loss weights"
    samples, short, sum_len, sq_hi, sq_lo, min_len, max_len = rd.take(np.int64, 7).tolist()
    mean, cv, short_fraction = rd.take(np.float64, 3).tolist()
    high_roi = int(rd.take(np.int64, 1)[0])
    sk = oracle.length_sketch(w.tok_off, None, w.budget)
    assert (samples, short, sum_len, (sq_hi << 32) + (sq_lo & 0xFFFFFFFFFFFFFFFF), min_len, max_len, high_roi) == \
        (sk["samples"], sk["short_samples"], sk["sum_len"], sk["sum_sq"], sk["min_len"], sk["max_len"],
         sk["high_roi"])
    assert short_fraction == sk["short_fraction"]
    assert abs(mean - sk["mean"]) <= 2.0 ** -52 * sk["mean"]
    assert abs(cv - sk["cv"]) <= 1e-15 * max(sk["cv"], 1e-300), (cv, sk["cv"])
    # every sample emitted or left over exactly once
    assert rd.take(np.int64, 3).tolist() == [0, 0, 0], "coverage"
    assert rd.at == len(rd.raw), "trailing output"


@pytest.mark.parametrize("case", ["join", "nonjoin"])
def test_stream_iteration_from_c(case, tmp_path):
    assert os.path.exists(STREAM_BIN), "tests/c_abi/stream_pipeline is missing: run __graft_entry__.build()"
    rng = np.random.default_rng(79)
    N, W, budget, buffer_size, depth = 6007, 5, 8192, 64, 96
    lens = np.clip(np.rint(synth.lognormal(rng, 300.0, 1.0, N)), 1, 4000).astype(np.int64)
    tok_off = np.zeros(N + 1, np.int64)
    np.cumsum(lens, out=tok_off[1:])
    tokens = synth.tokens_numpy(0, int(tok_off[-1]))
    perm = rng.permutation(N).astype(np.int32)
    rate = rng.integers(8, 40, W).astype(np.int32)
    mode, quota = (0, 0) if case == "join" else (1, N // 3)
    q = -(-N // W)
    max_rounds = q + (q + 1) * -(-buffer_size // int(rate.min())) + 2
    src, dst = tmp_path / "in.bin", tmp_path / "out.bin"
    with open(src, "wb") as f:
        np.array([W, N, len(tokens)], np.int64).tofile(f)
        tok_off.tofile(f)
        tokens.astype(np.int32).tofile(f)
        perm.tofile(f)
        rate.tofile(f)
    log(f"stream case c_{case}: N={N} W={W} budget={budget} buffer={buffer_size} depth={depth} quota={quota}")
    r = subprocess.run([STREAM_BIN, str(src), str(dst), str(budget), str(mode), str(quota), str(buffer_size),
                        str(depth), str(max_rounds)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr

    ref = oracle.stream(tok_off, perm, W, budget, mode=oracle.MODE_NONJOIN if mode else oracle.MODE_JOIN,
                        quota=quota, buffer_size=buffer_size, depth=depth, rate=rate)
    rd = _Reader(open(dst, "rb").read())
    info = dict(zip(STREAM_FIELDS, rd.take(np.int64, 20).tolist()))
    pad_fraction = float(rd.take(np.float64, 1)[0])
    retries = int(rd.take(np.int64, 1)[0])
    for f in STREAM_FIELDS[:-1]:
        assert info[f] == ref.sinfo[f], (f, info[f], ref.sinfo[f])
    S, M, E = ref.steps, ref.sinfo["views"], ref.sinfo["emitted_views"]
    K = W * S
    assert info["required_slot_capacity"] == K
    rf = ref.sinfo["pad_fraction"]
    assert abs(pad_fraction - rf) <= PAD_FRACTION_RTOL * max(abs(rf), 1e-300) or pad_fraction == rf
    assert retries == (1 if S > 1 else 0), retries
    assert np.array_equal(rd.take(np.int64, 4 * info["rounds"]).reshape(-1, 4), ref.trace), "trace"
    ids = np.asarray(ref.emit_order, dtype=np.int64)
    for name, dtype, count, want in [
        ("emit_views", np.int32, E, ref.emit_views), ("emit_order", np.int32, E, ref.emit_order),
        ("row_token_start", np.int64, E, tok_off[ids]), ("row_len", np.int32, E, lens[ids]),
        ("slot_rows", np.int32, K, ref.slot_rows), ("slot_maxlen", np.int32, K, ref.slot_maxlen),
        ("slot_row_off", np.int64, K + 1, ref.slot_row_off), ("slot_tile_off", np.int64, K + 1, ref.slot_tile_off),
        ("slot_tokens", np.int64, K, ref.slot_tokens), ("left_views", np.int32, M - E, ref.left_views),
        ("left_off", np.int64, W + 1, ref.left_off),
    ]:
        assert np.array_equal(rd.take(dtype, count), want), name
    P = int(ref.sinfo["padded_elems"])
    for name, want in zip(["input_ids", "labels", "attention_mask", "position_ids"], ref.collate(tok_off, tokens, 0)):
        got = rd.take(np.int32, P)
        assert np.array_equal(got, want), (name, int(np.count_nonzero(got != want)))
    wt = rd.take(np.float64, K)
    ewt, _, _ = ref.loss_weights(oracle.WEIGHT_TOKEN_EXACT)
    assert np.array_equal(wt.view(np.int64), ewt.view(np.int64)), "loss weights"
    assert rd.at == len(rd.raw), "trailing output"
