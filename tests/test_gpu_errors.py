"""GPU tests of the window path's data-error, capacity and status branches, called
through the C ABI: bad CSR lengths are reported with the first bad sample, a slot
capacity below W * S is reported with the capacity the plan needs (and Pipeline.align
then reallocates and matches the oracle), and the collate status word survives later
plan calls on the same workspace."""
import numpy as np
import pytest

import oracle
import synth
from _parity import compare_collate_full, compare_loss_weights, compare_plan, log, run_gpu

pytestmark = pytest.mark.gpu


def _window_with_offsets(tok_off, W):
    """A device window over explicit CSR offsets (possibly invalid); the token stream is a
    small array the grouping and alignment stages never read."""
    import torch
    import paper_2606_19989_amd as odb

    n = len(tok_off) - 1
    rank_off = np.linspace(0, n, W + 1).astype(np.int64)
    d_off = torch.from_numpy(np.ascontiguousarray(tok_off, dtype=np.int64)).cuda()
    toks = torch.zeros(64, dtype=torch.int32, device="cuda")
    return odb.DeviceWindow(rank_off, d_off, toks, None, 0)


def _bad_offsets(kind, rng):
    lens = rng.integers(1, 3000, 6000).astype(np.int64)
    off = np.zeros(len(lens) + 1, np.int64)
    np.cumsum(lens, out=off[1:])
    if kind == "zero_length":
        first = 777
        off[first + 1:] -= lens[first]           # sample 777 has length 0
        off[4001 + 1:] -= lens[4001]              # and a later one
    elif kind == "decreasing_offset":
        first = 1000
        off[first + 1] = off[first] - 5           # sample 1000 has length -5
    elif kind == "length_2p31":
        first = 2500
        off[first + 1:] += (1 << 31) - lens[first]    # sample 2500 has length exactly 2^31
    elif kind == "negative_offset":
        first = 0
        off[:] -= 3                               # sample 0 starts at token -3
    else:
        raise ValueError(kind)
    return off, first


@pytest.mark.parametrize("kind", ["zero_length", "decreasing_offset", "length_2p31", "negative_offset"])
def test_window_rejects_bad_lengths(kind):
    # l < 1, l >= 2^31 and negative token offsets are invalid data (a length the batch
    # size rule of Eq. 1 cannot take); the first such sample is named, and the same
    # workspace then serves a valid window
    import torch
    import paper_2606_19989_amd as odb

    rng = np.random.default_rng(41)
    off, first = _bad_offsets(kind, rng)
    log(f"bad lengths: {kind}, first bad sample {first}")
    dwin = _window_with_offsets(off, 3)
    pipe = odb.Pipeline(dwin, 16384)
    with pytest.raises(odb.OdbError) as e:
        pipe.form()
        pipe.align()
    assert e.value.status == odb.ODB_E_INVALID_DATA, str(e.value)
    assert f"sample {first} " in str(e.value), str(e.value)
    torch.cuda.synchronize()
    # the workspace recovers: a valid window of the same shape on it
    lens = rng.integers(1, 3000, 6000)
    w = synth.window_from_ranks("after_error", [lens[:2000], lens[2000:4000], lens[4000:]], 16384)
    tok_off, toks, _ = synth.device_tensors(w, "cuda")
    good = odb.DeviceWindow(w.rank_off, tok_off, toks, None, 0)
    pipe2 = odb.Pipeline(good, w.budget)
    pipe2.ws = pipe.ws
    pipe2.form()
    pipe2.align()
    compare_plan(w, pipe2, oracle.plan_window(w))


@pytest.mark.parametrize("mode", ["join", "nonjoin"])
def test_align_reports_capacity_and_pipeline_retries(mode):
    # slot arrays below W * S: ODB_E_CAPACITY with the capacity the plan needs; the
    # Pipeline then reallocates and its plan and outputs equal the oracle's
    import torch
    import paper_2606_19989_amd as odb

    rng = np.random.default_rng(43)
    per = [rng.integers(1, 3000, 4000), rng.integers(1, 3000, 900), rng.integers(1, 3000, 2500)]
    n = sum(len(x) for x in per)
    w = synth.window_from_ranks(f"capacity_{mode}", per, 12000, mode=mode, quota=n // 2 if mode == "nonjoin" else 0)
    ref = oracle.plan_window(w)
    need = w.W * ref.steps
    log(f"capacity: {mode}, plan needs {need} slots")
    tok_off, toks, _ = synth.device_tensors(w, "cuda")
    dwin = odb.DeviceWindow(w.rank_off, tok_off, toks, None, 0)
    for cap in (1, need - 1):
        pipe = odb.Pipeline(dwin, w.budget, mode=w.mode, quota=w.quota, slot_capacity=cap)
        pipe.form()
        st, info = odb.odb_align_groups(dwin, w.budget, pipe.mode, pipe.quota, None, pipe.order, pipe.sorted_len,
                                        pipe.group_index, pipe.groups_per_rank, pipe.slot_capacity, pipe.emit_order,
                                        pipe.slot_rows, pipe.slot_maxlen, pipe.slot_row_off, pipe.slot_tile_off,
                                        pipe.slot_tokens, pipe.leftover, pipe.leftover_off, pipe.ws,
                                        raise_on_capacity=False, slot_tokens_approx=pipe.slot_tokens_approx,
                                        row_token_start=pipe.row_token_start, row_len=pipe.row_len)
        assert st == odb.ODB_E_CAPACITY
        assert info["required_slot_capacity"] == need and info["steps"] == ref.steps
        with pytest.raises(odb.OdbError) as e:
            odb.odb_align_groups(dwin, w.budget, pipe.mode, pipe.quota, None, pipe.order, pipe.sorted_len,
                                 pipe.group_index, pipe.groups_per_rank, pipe.slot_capacity, pipe.emit_order,
                                 pipe.slot_rows, pipe.slot_maxlen, pipe.slot_row_off, pipe.slot_tile_off,
                                 pipe.slot_tokens, pipe.leftover, pipe.leftover_off, pipe.ws)
        assert e.value.status == odb.ODB_E_CAPACITY and str(need) in str(e.value)
        # Pipeline.align reallocates the slot arrays to the reported size and retries
        pipe.align()
        assert pipe.slot_capacity == need
        outs = pipe.collate()
        torch.cuda.synchronize()
        odb.odb_collate_status(pipe.ws)
        compare_plan(w, pipe, ref)
        compare_collate_full(w, outs, ref)
        compare_loss_weights(pipe, ref)


def test_collate_status_survives_plan_calls():
    # a collate error stays readable after grouping and alignment calls on the same
    # workspace; reading it clears it; a fresh workspace full of ones reports no error
    import torch
    import paper_2606_19989_amd as odb

    w = synth.WORKLOADS["ln512_w2x2048"].window()
    tok_off, toks, ident = synth.device_tensors(w, "cuda")
    dwin = odb.DeviceWindow(w.rank_off, tok_off, toks, ident, w.num_identities)
    pipe = odb.Pipeline(dwin, w.budget)
    pipe.ws.fill_(255)
    pipe.run()
    torch.cuda.synchronize()
    odb.odb_collate_status(pipe.ws)
    ref = oracle.plan_window(w)
    good = int(pipe.row_token_start[5])
    pipe.row_token_start[5] = int(w.tok_off[-1])   # a row record past the end of the stream
    pipe.collate()
    pipe.row_token_start[5] = good
    pipe.form()
    pipe.align()
    torch.cuda.synchronize()
    with pytest.raises(odb.OdbError) as e:
        odb.odb_collate_status(pipe.ws)
    assert e.value.status == odb.ODB_E_INVALID_DATA
    odb.odb_collate_status(pipe.ws)          # cleared by the read
    outs = pipe.collate()
    torch.cuda.synchronize()
    odb.odb_collate_status(pipe.ws)
    compare_plan(w, pipe, ref)
    compare_collate_full(w, outs, ref)


def test_pointer_jumping_full_size():
    # group discovery by pointer jumping over the next-group-start links on the largest
    # window (64 ranks x 262,144 samples, lengths 8..16384): a budget of 2^26 gives more
    # distinct batch sizes per rank than the run walk's table holds, so every rank's chain
    # is found by doubling rounds.  Every plan array and the loss weights are compared
    # exactly (groups of up to 2^26 padded elements: the collate is not run here)
    import torch

    w = synth.WORKLOADS["ln480_w64x262144"].window()
    w.budget = 1 << 26
    lens = np.diff(w.tok_off)
    rng_len = int(lens.max() - lens.min() + 1)
    runs_bound = min(2 * (int(np.sqrt(w.budget)) + 1) + 1, rng_len)
    assert runs_bound > 4096, runs_bound
    log(f"pointer jumping: n={w.n} budget={w.budget} distinct-step bound {runs_bound}")
    ref = oracle.plan_window(w)
    log(f"  oracle plan done: steps={ref.steps} groups={int(ref.groups_per_rank.sum())}")
    pipe, _ = run_gpu(w, collate=False)
    compare_plan(w, pipe, ref)
    compare_loss_weights(pipe, ref)
    log("  plan and loss weights equal")
    del pipe
    torch.cuda.empty_cache()
