"""The C-ABI library without a GPU: it loads, exports what include/odb.h declares, and
rejects bad arguments on the host before touching the device."""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_2606_19989_amd as odb

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    text = open(os.path.join(ROOT, "include", "odb.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(odb_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = odb.load()
    names = _declared()
    assert set(names) == set(odb.EXPORTED)
    for name in names:
        assert hasattr(lib, name), name


def test_status_strings():
    lib = odb.load()
    assert lib.odb_status_string(0) == b"ODB_OK"
    assert lib.odb_status_string(4) == b"ODB_E_CAPACITY"
    assert lib.odb_status_string(99) == b"ODB_E_UNKNOWN"


def _window(rank_off, n=None):
    ro = np.asarray(rank_off, dtype=np.int64)
    w = odb.Window(len(ro) - 1, 0, int(ro[-1]) if n is None else n,
                   ro.ctypes.data_as(ctypes.c_void_p).value, 0x1000, 0x2000, None, 0)
    return w, ro


def test_workspace_size_grows_with_window():
    lib = odb.load()
    w1, k1 = _window([0, 100, 200])
    w2, k2 = _window([0, 100000, 200000])
    s1 = lib.odb_workspace_size(ctypes.byref(w1))
    s2 = lib.odb_workspace_size(ctypes.byref(w2))
    assert 0 < s1 < s2
    assert s2 >= 200000 * 64   # tens of bytes of scratch per sample


@pytest.mark.parametrize("rank_off,n", [([0, 5, 3, 6], None), ([1, 5], None), ([0, 5], 6), ([0], 0)])
def test_bad_windows_rejected_on_host(rank_off, n):
    lib = odb.load()
    w, keep = _window(rank_off, n)
    assert lib.odb_workspace_size(ctypes.byref(w)) == 0
    st = lib.odb_form_groups(ctypes.byref(w), 10, None, None, None, None, None, 0, None)
    assert st == odb.ODB_E_INVALID_ARG
    assert lib.odb_last_error_message() != b""


def test_bad_arguments_rejected_on_host():
    lib = odb.load()
    w, keep = _window([0, 4])
    size = lib.odb_workspace_size(ctypes.byref(w))
    fake_ws = 0x100000  # never dereferenced: every call below fails its host checks first
    # workspace too small
    st = lib.odb_form_groups(ctypes.byref(w), 10, 1, 1, 1, 1, fake_ws, size - 1, None)
    assert st == odb.ODB_E_WORKSPACE
    # misaligned workspace
    st = lib.odb_form_groups(ctypes.byref(w), 10, 1, 1, 1, 1, fake_ws + 8, size, None)
    assert st == odb.ODB_E_INVALID_ARG
    # budget < 1
    st = lib.odb_form_groups(ctypes.byref(w), 0, 1, 1, 1, 1, fake_ws, size, None)
    assert st == odb.ODB_E_INVALID_ARG
    # non-join without quota, unknown mode, negative capacity
    info = odb.PlanInfo()
    for mode, quota, cap in [(1, 0, None), (7, 1, None), (0, 0, np.array([-1], dtype=np.int64))]:
        p = odb.AlignParams(mode, 0, quota, None if cap is None else cap.ctypes.data_as(ctypes.c_void_p).value)
        st = lib.odb_align_groups(ctypes.byref(w), 10, ctypes.byref(p), 1, 1, 1, 1, 16, 1, None, None, 1, 1, 1, 1,
                                  1, None, 1, 1, ctypes.byref(info), fake_ws, size, None)
        assert st == odb.ODB_E_INVALID_ARG, (mode, quota, cap)
    # row records come as a pair or not at all
    p = odb.AlignParams(0, 0, 0, None)
    for ts, ln in [(1, None), (None, 1)]:
        st = lib.odb_align_groups(ctypes.byref(w), 10, ctypes.byref(p), 1, 1, 1, 1, 16, 1, ts, ln, 1, 1, 1, 1,
                                  1, None, 1, 1, ctypes.byref(info), fake_ws, size, None)
        assert st == odb.ODB_E_INVALID_ARG
        st = lib.odb_collate(ctypes.byref(w), 3, 1, ts, ln, 1, 1, 1, 1, 0, 10, 1, 1, 1, 1, fake_ws, size, None)
        assert st == odb.ODB_E_INVALID_ARG
    # collate with negative sizes
    st = lib.odb_collate(ctypes.byref(w), -1, 1, None, None, 1, 1, 1, 1, 0, 10, 1, 1, 1, 1, fake_ws, size, None)
    assert st == odb.ODB_E_INVALID_ARG
    st = lib.odb_collate(ctypes.byref(w), 3, 1, None, None, 1, 1, 1, 1, 0, -5, 1, 1, 1, 1, fake_ws, size, None)
    assert st == odb.ODB_E_INVALID_ARG
    # collate without row records needs the emitted ids
    st = lib.odb_collate(ctypes.byref(w), 3, None, None, None, 1, 1, 1, 1, 0, 10, 16, 16, 16, 16, fake_ws, size,
                         None)
    assert st == odb.ODB_E_INVALID_ARG


def test_loss_weights_arguments_checked_on_host():
    lib = odb.load()
    # no GPU call happens: each of these fails (or finishes, for zero steps) on the host
    assert lib.odb_loss_weights(0, 5, 2, 1, 1, None, 1, None, None, None) == odb.ODB_E_INVALID_ARG
    assert lib.odb_loss_weights(2, -1, 2, 1, 1, None, 1, None, None, None) == odb.ODB_E_INVALID_ARG
    assert lib.odb_loss_weights(2, 5, 3, 1, 1, None, 1, None, None, None) == odb.ODB_E_INVALID_ARG
    assert lib.odb_loss_weights(2, 5, 2, None, 1, None, 1, None, None, None) == odb.ODB_E_INVALID_ARG
    assert lib.odb_loss_weights(2, 5, 2, 1, 1, None, None, None, None, None) == odb.ODB_E_INVALID_ARG
    # the approximate mode needs the approximate counts
    assert lib.odb_loss_weights(2, 5, odb.ODB_WEIGHT_TOKEN_APPROX, 1, 1, None, 1, None, None, None) == \
        odb.ODB_E_INVALID_ARG
    assert lib.odb_loss_weights(2 ** 30, 2 ** 40, 2, 1, 1, None, 1, None, None, None) == odb.ODB_E_INVALID_ARG
    assert lib.odb_loss_weights(3, 0, 0, None, None, None, None, None, None, None) == odb.ODB_OK


def test_length_sketch_arguments_checked_on_host():
    lib = odb.load()
    w, keep = _window([0, 4, 9])
    size = lib.odb_workspace_size(ctypes.byref(w))
    fake_ws = 0x100000  # never dereferenced: every call below fails its host checks first
    out = odb.LengthSketch()
    ref = ctypes.byref(out)
    assert lib.odb_length_sketch(ctypes.byref(w), None, 3, 10, None, fake_ws, size, None) == odb.ODB_E_INVALID_ARG
    assert lib.odb_length_sketch(ctypes.byref(w), None, 3, 0, ref, fake_ws, size, None) == odb.ODB_E_INVALID_ARG
    assert lib.odb_length_sketch(ctypes.byref(w), None, -1, 10, ref, fake_ws, size, None) == odb.ODB_E_INVALID_ARG
    assert lib.odb_length_sketch(ctypes.byref(w), None, 10, 10, ref, fake_ws, size, None) == odb.ODB_E_INVALID_ARG
    assert lib.odb_length_sketch(ctypes.byref(w), 1, 2 ** 31, 10, ref, fake_ws, size, None) == odb.ODB_E_INVALID_ARG
    assert lib.odb_length_sketch(ctypes.byref(w), None, 3, 10, ref, fake_ws, size - 1, None) == odb.ODB_E_WORKSPACE


def test_stream_arguments_checked_on_host():
    lib = odb.load()
    w, keep = _window([0, 4, 9])
    assert lib.odb_stream_workspace_size(ctypes.byref(w), 64, 100, 50) > lib.odb_workspace_size(ctypes.byref(w))
    assert lib.odb_stream_workspace_size(ctypes.byref(w), 4097, 100, 50) == 0     # deeper than the LDS sort
    assert lib.odb_stream_workspace_size(ctypes.byref(w), 64, -1, 50) == 0
    assert lib.odb_stream_workspace_size(ctypes.byref(w), 64, 100, 0) == 0
    # capacities and round limits whose workspace would pass 2^50 bytes (sizes that would
    # wrap if multiplied unchecked) are refused, not wrapped
    for cap, rounds in ((1 << 62, 50), ((1 << 63) - 1, 50), (100, 1 << 62), (100, (1 << 63) - 1)):
        assert lib.odb_stream_workspace_size(ctypes.byref(w), 64, cap, rounds) == 0, (cap, rounds)
    fake_ws = 0x100000  # never dereferenced: every call below fails its host checks first
    rate = np.array([4, 4], dtype=np.int32)
    bad_rate = np.array([4, 0], dtype=np.int32)
    info = odb.StreamInfo()

    def call(params, budget=10, cap=16, ts=None, ln=None):
        return lib.odb_stream_plan(ctypes.byref(w), 1, budget, params, cap, 1, 1, ts, ln, 1, 1, 1, 1, 1, None, 1, 1,
                                   None, ctypes.byref(info), fake_ws, 1 << 40, None)

    ptr = lambda a: a.ctypes.data_as(ctypes.c_void_p).value
    good = dict(mode=0, buffer_size=4, depth=8, reserved0=0, quota=0, rate=ptr(rate), slot_capacity=None, max_rounds=9)
    for bad in (dict(mode=5), dict(buffer_size=0), dict(buffer_size=9), dict(depth=5000, buffer_size=8),
                dict(reserved0=1), dict(mode=1, quota=0), dict(rate=None), dict(rate=ptr(bad_rate)),
                dict(max_rounds=0)):
        p = odb.StreamParams(**{**good, **bad})
        assert call(ctypes.byref(p)) == odb.ODB_E_INVALID_ARG, bad
    assert call(None) == odb.ODB_E_INVALID_ARG
    p = odb.StreamParams(**good)
    assert call(ctypes.byref(p), budget=0) == odb.ODB_E_INVALID_ARG
    assert call(ctypes.byref(p), cap=-1) == odb.ODB_E_INVALID_ARG
    assert call(ctypes.byref(p), cap=(1 << 63) - 1) == odb.ODB_E_INVALID_ARG
    p_rounds = odb.StreamParams(**{**good, "max_rounds": (1 << 63) - 1})
    assert call(ctypes.byref(p_rounds)) == odb.ODB_E_INVALID_ARG
    assert b"2^50 bytes" in lib.odb_last_error_message()
    assert call(ctypes.byref(p), ts=1) == odb.ODB_E_INVALID_ARG
    assert call(ctypes.byref(p), ln=1) == odb.ODB_E_INVALID_ARG


def test_binding_raises_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(odb, "_lib", None)
    monkeypatch.setattr(odb, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(RuntimeError):
        odb.load()
