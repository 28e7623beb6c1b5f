"""Host logic of the Python binding, without a GPU: the Pipeline's retry after
ODB_E_CAPACITY passes every reallocated slot array (the library is replaced by a
recorder; nothing is launched)."""
import ctypes
import types

import numpy as np

import paper_2606_19989_amd as odb


def _fake_window():
    import torch

    ro = np.array([0, 5, 9], np.int64)
    win = types.SimpleNamespace(num_ranks=2, num_samples=9, rank_offsets=ro,
                                token_offsets=torch.zeros(10, dtype=torch.int64))
    # host fields only: odb_workspace_size never dereferences the device pointers
    win.struct = odb.Window(2, 0, 9, ro.ctypes.data_as(ctypes.c_void_p).value, 0x1000, 0x2000, None, 0)
    win.ref = ctypes.byref(win.struct)
    return win


def test_pipeline_capacity_retry_passes_the_reallocated_slot_arrays(monkeypatch):
    calls = []

    def recorder(*args, raise_on_capacity=True, **kw):
        calls.append((args, kw))
        if len(calls) == 1:
            return odb.ODB_E_CAPACITY, {"required_slot_capacity": 7, "steps": 3}
        return odb.ODB_OK, {"required_slot_capacity": 7, "steps": 3}

    monkeypatch.setattr(odb, "odb_align_groups", recorder)
    pipe = odb.Pipeline(_fake_window(), 100, slot_capacity=1)
    pipe.align()
    assert len(calls) == 2
    (a1, k1), (a2, k2) = calls
    assert a1[9] == 1 and a2[9] == 7 == pipe.slot_capacity
    # slot_rows, slot_maxlen, slot_tokens (capacity) and the two offset arrays (+1)
    for i, size in ((11, 7), (12, 7), (15, 7), (13, 8), (14, 8)):
        assert a2[i].numel() == size, i
        assert a1[i].numel() == (1 if size == 7 else 2), i
    assert k2["slot_tokens_approx"].numel() == 7 and k2["slot_tokens_approx"] is pipe.slot_tokens_approx
    assert k1["slot_tokens_approx"].numel() == 1
    assert k2["row_token_start"] is pipe.row_token_start and k2["row_len"] is pipe.row_len
