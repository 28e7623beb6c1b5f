"""Pins for the oracle's unified streaming loop (no GPU).

The streaming model is tied to the already-pinned window oracle (it must reduce to it
exactly when every rank buffers its whole share in the first round), to Theorem 1
(join: every sampler view emitted once, identity coverage with the sampler's padding as
the only duplicates), to App. C's No-Leak invariant and Lyapunov potential (emit rounds
lower it by what they emit, skip rounds leave it), to the round-count bound, to the
non-join envelope eta_logical <= W * D / N and quota closure, and to skip-round timing
worked out by hand.
"""

import numpy as np
import pytest

import oracle


def offsets(lens):
    return np.concatenate([[0], np.cumsum(np.asarray(lens, dtype=np.int64))])


def view_identity(perm, N, W):
    q = -(-N // W)
    m = np.arange(q * W)
    return perm[m % N], q


def random_case(rng):
    N = int(rng.integers(1, 3000))
    W = int(rng.integers(1, 7))
    lens = rng.integers(1, int(rng.integers(2, 3000)), size=N)
    perm = rng.permutation(N).astype(np.int32)
    buf = int(rng.integers(1, 400))
    depth = buf + int(rng.integers(0, 300))
    rate = rng.integers(1, depth + 1, size=W)
    return N, W, lens, perm, buf, depth, rate


@pytest.mark.parametrize("mode", ["join", "nonjoin"])
def test_reduces_to_the_window_pipeline(mode):
    # buffer = depth = rate = a rank's whole share: round 1 buffers everything, later
    # rounds regroup overflow, exactly the window pipeline's join / non-join rounds
    rng = np.random.default_rng(61)
    for t in range(25):
        N = int(rng.integers(1, 2000))
        W = int(rng.integers(1, 6))
        lens = rng.integers(1, int(rng.integers(2, 3000)), size=N)
        perm = rng.permutation(N).astype(np.int32)
        ident, q = view_identity(perm, N, W)
        budget = int(rng.integers(1, 20000))
        quota = int(rng.integers(1, q * W + 2))
        cap = rng.integers(0, 5, size=W) if t % 3 == 1 else None
        m_mode = oracle.MODE_NONJOIN if mode == "nonjoin" else oracle.MODE_JOIN
        sp = oracle.stream(offsets(lens), perm, W, budget, mode=m_mode, quota=quota, buffer_size=q, depth=q,
                           rate=np.full(W, q), capacity=cap)
        # the same views as a window: rank r holds its views in increasing m
        order = np.concatenate([np.arange(r, q * W, W) for r in range(W)])
        rank_off = np.arange(W + 1) * q
        wp = oracle.plan(rank_off, offsets(lens[ident[order]]), budget, mode=m_mode, quota=quota, capacity=cap)
        for f in ("steps", "stop_reason", "emitted_samples", "real_tokens", "padded_elems", "max_step_samples",
                  "splits", "overflow_groups", "second_gather_rounds"):
            assert sp.info[f] == wp.info[f], (t, f, sp.info[f], wp.info[f])
        assert sp.sinfo["emit_rounds"] == wp.info["rounds"]
        for f in ("slot_rows", "slot_maxlen", "slot_row_off", "slot_tile_off", "slot_tokens"):
            assert np.array_equal(getattr(sp, f), getattr(wp, f)), (t, f)
        assert np.array_equal(sp.slot_tokens_approx, wp.slot_tokens_approx)
        assert np.array_equal(sp.emit_views, order[wp.emit_order])           # window index -> view
        assert np.array_equal(sp.emit_order, ident[order[wp.emit_order]])    # view -> identity


def test_join_theorem_1_and_no_leak():
    rng = np.random.default_rng(62)
    for t in range(40):
        N, W, lens, perm, buf, depth, rate = random_case(rng)
        sp = oracle.stream(offsets(lens), perm, W, int(rng.integers(1, 20000)), buffer_size=buf, depth=depth,
                           rate=rate)
        si = sp.sinfo
        q = -(-N // W)
        M = q * W
        assert si["views"] == M and si["stop_reason"] == oracle.STOP_DRAINED
        assert si["emitted_views"] == M and si["undelivered_views"] == 0 and si["pending_views"] == 0
        assert sorted(sp.emit_views.tolist()) == list(range(M))        # every view exactly once
        assert si["bad_views"] == 0 and si["missing_ids"] == 0 and si["duplicate_ids"] == M - N
        counts = np.bincount(sp.emit_order, minlength=N)
        assert counts.min() == 1 and counts.sum() == M
        # each rank emits exactly its own views
        S = sp.steps
        for r in range(W):
            a, b = sp.slot_row_off[r * S], sp.slot_row_off[(r + 1) * S]
            assert np.all(sp.emit_views[a:b] % W == r)


def test_lyapunov_potential_and_round_bounds():
    rng = np.random.default_rng(63)
    for t in range(40):
        N, W, lens, perm, buf, depth, rate = random_case(rng)
        mode = oracle.MODE_NONJOIN if t % 2 else oracle.MODE_JOIN
        sp = oracle.stream(offsets(lens), perm, W, int(rng.integers(1, 20000)), mode=mode,
                           quota=int(rng.integers(1, N + 2)), buffer_size=buf, depth=depth, rate=rate)
        si, tr = sp.sinfo, sp.trace
        M = si["views"]
        assert len(tr) == si["rounds"] == si["emit_rounds"] + si["skip_rounds"] + (1 if tr[-1, 0] == 2 else 0)
        phi = M
        for kind, T, emitted, after in tr:
            if kind == oracle.ROUND_EMIT:
                assert T >= 1 and emitted >= 1 and after == phi - emitted     # strict decrease
            else:
                assert emitted == 0 and after == phi                           # skip / stop: unchanged
            phi = after
        assert phi == M - si["emitted_views"]
        q = -(-N // W)
        assert si["emit_rounds"] <= q                                          # Thm 3: <= ceil(N/W) emitting rounds
        fill = -(-buf // int(rate.min()))
        assert si["skip_rounds"] <= (si["emit_rounds"] + 1) * fill             # bounded skip epilogues
        assert si["max_outstanding"] <= depth                                  # the envelope


def test_nonjoin_envelope_and_quota_closure():
    rng = np.random.default_rng(64)
    seen = set()
    for t in range(60):
        N, W, lens, perm, buf, depth, rate = random_case(rng)
        quota = int(rng.integers(1, N + 2))
        sp = oracle.stream(offsets(lens), perm, W, int(rng.integers(1, 20000)), mode=oracle.MODE_NONJOIN,
                           quota=quota, buffer_size=buf, depth=depth, rate=rate)
        si = sp.sinfo
        seen.add(si["stop_reason"])
        # Lemma (logical-discard bound): fetched but not emitted <= W * D
        assert si["undelivered_views"] <= W * depth
        assert si["undelivered_views"] / N <= W * depth / N
        assert si["emitted_views"] + si["undelivered_views"] + si["pending_views"] == si["views"]
        assert si["bad_views"] == 0
        if si["stop_reason"] == oracle.STOP_QUOTA:
            assert quota <= si["emitted_views"] <= quota + si["max_step_samples"]   # Thm 2
        # left-over views: exactly the un-emitted ones, per rank in increasing view index
        left = set(sp.left_views.tolist())
        assert left.isdisjoint(sp.emit_views.tolist()) and len(left) + si["emitted_views"] == si["views"]
        for r in range(W):
            lv = sp.left_views[sp.left_off[r]:sp.left_off[r + 1]]
            assert np.all(lv % W == r) and np.all(np.diff(lv) > 0)
    assert oracle.STOP_QUOTA in seen and oracle.STOP_RANK_FINISHED in seen


def test_skip_rounds_by_hand():
    # W = 2, 12 samples of length 10, buffer 4, rate (1, 4): rank 0 needs 4 rounds to
    # fill, so rounds 1-3 skip and round 4 emits; budget 20 -> groups of sizes 1, 2, 1
    # (threshold t: 1, then B(10) = 2, trailing 1) on both ranks, T = 3
    N, W = 12, 2
    sp = oracle.stream(offsets([10] * N), np.arange(N, dtype=np.int32), W, 20, buffer_size=4, depth=4,
                       rate=[1, 4])
    tr = sp.trace
    assert list(tr[:4, 0]) == [1, 1, 1, 0]
    assert tr[3, 1] == 3 and tr[3, 2] == 8 and tr[3, 3] == 12 - 8
    # round 5: rank 1 fetches its last 2 views (sampler drained, so ready); rank 0 holds
    # 1 view with 1 still pending, so it is not ready: skip.  Round 6: rank 0 fetches its
    # last view and is ready with 2; each rank forms groups of sizes 1, 1 and T = 2.
    # Round 7 observes that both ranks are finished.
    assert list(tr[4:, 0]) == [1, 0, 2]
    assert tr[5, 1] == 2 and tr[5, 2] == 4 and tr[5, 3] == 0
    assert sp.sinfo["emit_rounds"] == 2 and sp.sinfo["skip_rounds"] == 4 and sp.sinfo["rounds"] == 7
    assert sp.steps == 5 and sp.slot_rows[:5].tolist() == [1, 2, 1, 1, 1]


def test_idle_slots_for_finished_ranks():
    # rank 1 has one short view; rank 0's long buffer overflows into a second round in
    # which rank 1 is finished and sends IDLE slots
    lens = [5000, 5000, 5000, 1] + [5000] * 2
    N, W = 6, 2
    perm = np.array([0, 3, 1, 4, 2, 5], dtype=np.int32)      # rank 0: 0, 1, 2; rank 1: 3, 4, 5
    sp = oracle.stream(offsets(lens), perm, W, 5000, buffer_size=3, depth=3, rate=[3, 3],
                       capacity=[1, 1])
    S = sp.steps
    assert sp.sinfo["stop_reason"] == oracle.STOP_DRAINED and sp.sinfo["emitted_views"] == 6
    assert S == 3 and sp.slot_rows.reshape(W, S).min(axis=0).tolist() == [1, 1, 1]


def test_sampler_padding_reuses_the_head_of_the_list():
    N, W = 10, 4           # M = 12: views 10, 11 are perm[0], perm[1]
    perm = np.array([9, 3, 7, 1, 0, 2, 4, 6, 8, 5], dtype=np.int32)
    sp = oracle.stream(offsets(np.arange(1, N + 1)), perm, W, 100, buffer_size=3, depth=3)
    ident = dict(zip(sp.emit_views.tolist(), sp.emit_order.tolist()))
    assert ident[10] == 9 and ident[11] == 3
    assert sp.sinfo["duplicate_ids"] == 2


def test_invalid_inputs():
    off = offsets([3, 4, 5])
    with pytest.raises(oracle.OracleError):
        oracle.stream(off, np.array([0, 0, 1]), 2, 10)
    with pytest.raises(oracle.OracleError):
        oracle.stream(off, np.array([0, 1, 2]), 2, 10, rate=[0, 1])
    with pytest.raises(oracle.OracleError):
        oracle.stream(off, np.array([0, 1, 2]), 2, 10, buffer_size=4, depth=3)
    with pytest.raises(oracle.OracleError):
        oracle.stream(off, np.array([0, 1, 2]), 2, 10, buffer_size=1, rate=[1, 1], max_rounds=2)
