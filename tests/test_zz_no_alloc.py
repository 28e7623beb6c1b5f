"""odb_collate_static (the collate without a workspace, for callers that cannot allocate)
against odb_collate on the same plans, through the C ABI: two calls in a row, the second
on a smaller window, with and without the plan's row records; the status output; the
host-side size limit, and a window at that limit."""
import numpy as np
import pytest

import synth
from _parity import log

pytestmark = pytest.mark.gpu


def _planned(w):
    import torch
    import paper_2606_19989_amd as odb

    tok_off, toks, ident = synth.device_tensors(w, "cuda")
    dwin = odb.DeviceWindow(w.rank_off, tok_off, toks, ident, w.num_identities)
    pipe = odb.Pipeline(dwin, w.budget, mode=w.mode, quota=w.quota)
    pipe.form()
    pipe.align()
    outs = pipe.collate()
    torch.cuda.synchronize()
    odb.odb_collate_status(pipe.ws)
    return pipe, tuple(o.clone() for o in outs)


def _static(pipe, rows, status, fill=-9):
    import torch
    import paper_2606_19989_amd as odb

    P = int(pipe.info["padded_elems"])
    outs = tuple(torch.full((max(P, 1),), fill, dtype=torch.int32, device="cuda") for _ in range(4))
    rec = dict(row_token_start=pipe.row_token_start, row_len=pipe.row_len) if rows else {}
    odb.odb_collate_static(pipe.win, pipe.num_slots, pipe.emit_order, pipe.slot_rows, pipe.slot_maxlen,
                           pipe.slot_row_off, pipe.slot_tile_off, pipe.pad_id, P, *outs, status, **rec)
    return tuple(o[:P] for o in outs)


@pytest.mark.parametrize("rows", [True, False])
def test_static_collate_equals_workspace_collate(rows):
    import torch

    big = synth.WORKLOADS["ln512_w2x2048"].window()
    rng = np.random.default_rng(57)
    small = synth.window_from_ranks("small", [rng.integers(1, 900, 700), rng.integers(1, 900, 301),
                                              rng.integers(1, 900, 40)], 4096)
    status = torch.full((1,), 77, dtype=torch.int32, device="cuda")
    for w in (big, small):
        log(f"static collate: {w.name} n={w.n} row records={rows}")
        pipe, want = _planned(w)
        got = _static(pipe, rows, status)
        torch.cuda.synchronize()
        assert int(status.item()) == 0
        for name, g, e in zip(["input_ids", "labels", "attention_mask", "position_ids"], got, want):
            assert torch.equal(g, e), name
        del pipe


def test_static_collate_reports_a_bad_row_record():
    import torch

    w = synth.WORKLOADS["ln512_w2x2048"].window()
    pipe, want = _planned(w)
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    good = int(pipe.row_token_start[5])
    pipe.row_token_start[5] = int(w.tok_off[-1])   # a row record past the end of the stream
    _static(pipe, True, status)
    torch.cuda.synchronize()
    assert int(status.item()) != 0
    pipe.row_token_start[5] = good
    got = _static(pipe, True, status)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    for g, e in zip(got, want):
        assert torch.equal(g, e)


def test_static_collate_rejects_windows_beyond_the_scratch():
    # without row records a window of more than ODB_COLLATE_STATIC_MAX_ROWS - W + 1
    # samples is refused on the host, before any launch
    import torch
    import paper_2606_19989_amd as odb

    n = odb.ODB_COLLATE_STATIC_MAX_ROWS
    tok_off = torch.arange(n + 1, dtype=torch.int64, device="cuda")
    toks = torch.zeros(n, dtype=torch.int32, device="cuda")
    dwin = odb.DeviceWindow(np.array([0, n // 2, n], np.int64), tok_off, toks)
    one = torch.zeros(4, dtype=torch.int64, device="cuda")
    i32 = torch.zeros(4, dtype=torch.int32, device="cuda")
    outs = [torch.zeros(4, dtype=torch.int32, device="cuda") for _ in range(4)]
    with pytest.raises(odb.OdbError) as e:
        odb.odb_collate_static(dwin, 1, i32, i32, i32, one, one, 0, 4, *outs, i32[:1])
    assert e.value.status == odb.ODB_E_INVALID_ARG and "static scratch" in str(e.value)
    lib = odb.load()
    assert b"static scratch" in lib.odb_last_error_message()
    # with row records the same window is accepted (a plan of one empty slot: nothing to
    # write)
    zero = torch.zeros(2, dtype=torch.int64, device="cuda")
    status = torch.full((1,), 5, dtype=torch.int32, device="cuda")
    odb.odb_collate_static(dwin, 1, None, i32, i32, zero, zero, 0, 4, *outs, status,
                           row_token_start=one, row_len=i32)
    torch.cuda.synchronize()
    assert int(status.item()) == 0


def test_static_collate_at_the_scratch_limit():
    # without row records, a window of exactly ODB_COLLATE_STATIC_MAX_ROWS - W + 1
    # samples (n + W - 1 rows, the scratch's last row included) is accepted and collates
    # like odb_collate
    import torch
    import paper_2606_19989_amd as odb

    W = 2
    n = odb.ODB_COLLATE_STATIC_MAX_ROWS - W + 1
    rng = np.random.default_rng(59)
    w = synth.window_from_ranks("at_limit", [rng.integers(1, 4, n // 2), rng.integers(1, 4, n - n // 2)], 4096)
    log(f"static collate at the scratch limit: n={w.n} W={w.W}")
    pipe, want = _planned(w)
    status = torch.full((1,), 77, dtype=torch.int32, device="cuda")
    got = _static(pipe, False, status)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    for name, g, e in zip(["input_ids", "labels", "attention_mask", "position_ids"], got, want):
        assert torch.equal(g, e), name
