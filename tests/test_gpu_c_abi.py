"""The window pipeline driven from plain C (tests/c_abi/window_pipeline.c: hipMalloc'd
buffers, include/odb.h, no Python in the loop), compared with the oracle: grouping,
alignment (after the one retry with the slot capacity the first call reports), the
collated tiles and the exact token-level loss weights."""
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
INFO_FIELDS = INFO_EXACT[:13] + ["second_gather_rounds", "required_slot_capacity"]


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
    for name, want in zip(["input_ids", "labels", "attention_mask", "position_ids"],
                          ref.collate(w.tok_off, tokens, 0)):
        got = rd.take(np.int32, P)
        assert np.array_equal(got, want), (name, int(np.count_nonzero(got != want)))
    wt = rd.take(np.float64, K)
    ewt, _, _ = ref.loss_weights(oracle.WEIGHT_TOKEN_EXACT)
    assert np.array_equal(wt.view(np.int64), ewt.view(np.int64)), "loss weights"
    assert rd.at == len(rd.raw), "trailing output"
