"""GPU parity: the HIP pipeline, called through the C ABI, against the CPU oracle.

Small and adversarial windows are compared element by element on every output; the
benchmark workloads are compared exactly on every plan array and on sampled collate
outputs (plus whole-output properties), in the launch configuration the benchmark uses.
"""
import numpy as np
import pytest

import oracle
import synth
from _parity import (collate_properties, compare_collate_by_rank, compare_collate_full, compare_collate_sampled,
                     compare_loss_weights, compare_plan, log, run_gpu)

pytestmark = pytest.mark.gpu


def win(per_rank, budget, **kw):
    return synth.window_from_ranks("t", [np.asarray(x, dtype=np.int64) for x in per_rank], budget, **kw)


def check_full(w, pad_id=0):
    log(f"case {w.name}: W={w.W} n={w.n} budget={w.budget} mode={w.mode} quota={w.quota} "
        f"cap={None if w.capacity is None else list(w.capacity)}")
    ref = oracle.plan_window(w)
    pipe, outs = run_gpu(w, pad_id=pad_id)
    compare_plan(w, pipe, ref)
    compare_collate_full(w, outs, ref, pad_id)
    compare_loss_weights(pipe, ref)
    return pipe, ref


def adversarial_windows():
    rng = np.random.default_rng(100)
    out = []
    add = lambda name, per, budget, **kw: out.append(
        synth.window_from_ranks(name, [np.asarray(x, dtype=np.int64) for x in per], budget, **kw))
    add("worked_example", [[100, 200, 500, 800]], 1000)
    add("all_equal", [[64] * 700, [64] * 513], 4096)
    add("ascending", [np.arange(1, 3001), np.arange(5, 900)], 8192)
    add("descending", [np.arange(3000, 0, -1)], 5000)
    add("heavy_ties", [rng.integers(1, 4, 5000) for _ in range(3)], 64)
    add("single_sample_ranks", [[7], [9], [1]], 100)
    add("empty_ranks", [[], rng.integers(1, 500, 300), [], rng.integers(1, 500, 40), []], 2000)
    add("longer_than_budget", [rng.integers(900, 3000, 200), rng.integers(1, 100, 900)], 1000)
    add("budget_below_min", [rng.integers(50, 300, 400), rng.integers(50, 300, 10)], 49)
    add("one_rank", [rng.integers(1, 4000, 10000)], 16384)
    add("tiny_budget_one", [rng.integers(1, 5, 300)], 1)
    add("capacity_overflow", [rng.integers(1, 600, 900), rng.integers(1, 600, 500), rng.integers(1, 600, 50)], 3000,
        capacity=np.array([5, 0, 3]))
    add("capacity_one", [rng.integers(1, 300, 120), rng.integers(1, 300, 80)], 600, capacity=np.array([1, 1]))
    add("unequal_buffers", [rng.integers(1, 2000, 4000), rng.integers(1, 2000, 37), rng.integers(1, 2000, 1)], 8192)
    n4 = 4000 + 800 + 3
    for q in (1, 777, n4 - 1, n4, n4 + 1):
        add(f"nonjoin_q{q}", [rng.integers(1, 3000, 4000), rng.integers(1, 3000, 800), rng.integers(1, 3000, 3)],
            12000, mode="nonjoin", quota=q)
    add("nonjoin_capacity", [rng.integers(1, 900, 700), rng.integers(1, 900, 600)], 2500, mode="nonjoin",
        quota=1000, capacity=np.array([2, 4]))
    add("nonjoin_empty_rank", [rng.integers(1, 900, 70), [], rng.integers(1, 900, 5)], 2500, mode="nonjoin", quota=10)
    add("empty_window", [[], []], 100)
    # group discovery: a huge budget with a wide length range takes the pointer-jumping
    # path; a 4M budget with lengths up to 5000 gives ~4000 distinct steps, close to the
    # run walk's LDS table
    add("huge_budget_jumping", [rng.integers(1, 20000, 9000), rng.integers(1, 20000, 5000)], 1 << 40)
    add("many_step_runs", [rng.integers(1, 5000, 12000), rng.integers(1, 5000, 7000)], 4_000_000)
    per = [rng.integers(100, 3000, 47 - r) for r in range(15)] + [np.zeros(0, np.int64)]
    add("empty_rank_audit_w16", per, 8192)
    # narrow tiles (widths 3..9, a few rows each): groups straddle tile edges at every
    # offset, the next tile's first row is sometimes shorter than the group's remainder,
    # and an empty rank leaves zero-size IDLE tiles between non-empty ones
    add("narrow_tile_edges", [rng.integers(3, 10, 3000), [], rng.integers(3, 10, 1500), rng.integers(1, 4, 700)], 24)
    add("narrow_tile_edges_nonjoin", [rng.integers(3, 10, 3000), rng.integers(3, 10, 1501)], 31, mode="nonjoin",
        quota=2500)
    # more ranks than the LDS rank table (1024) and than a block's threads, some empty
    add("many_ranks_w1500", [rng.integers(1, 2000, int(rng.integers(0, 12))) for _ in range(1500)], 8192)
    per = [rng.integers(1, 2000, int(rng.integers(1, 9))) for _ in range(700)]
    add("many_ranks_w700_nonjoin", per, 6000, mode="nonjoin", quota=sum(len(x) for x in per) // 2)
    return out


@pytest.mark.parametrize("idx", range(len(adversarial_windows())))
def test_adversarial_window(idx):
    w = adversarial_windows()[idx]
    check_full(w, pad_id=idx + 3)


@pytest.mark.parametrize("kind", synth.AUDIT_KINDS)
def test_audit_distributions(kind):
    for W, mode in ((3, "join"), (8, "join"), (3, "nonjoin")):
        w = synth.audit_window(kind, W, budget=4096, mode=mode, quota=1000)
        pipe, ref = check_full(w)
        if mode == "join":
            _, q, P = synth.sampler_views(1000, W, seed=1)
            assert pipe.info["missing_ids"] == 0 and pipe.info["duplicate_ids"] == P


def test_random_small_windows():
    rng = np.random.default_rng(7)
    for t in range(40):
        W = int(rng.integers(1, 6))
        per = [rng.integers(1, int(rng.integers(2, 3000)), size=int(rng.integers(0, 400))) for _ in range(W)]
        n = sum(len(x) for x in per)
        mode = "nonjoin" if t % 3 == 2 else "join"
        cap = rng.integers(0, 6, size=W) if t % 4 == 1 else None
        w = win(per, int(rng.integers(1, 20000)), mode=mode, quota=int(rng.integers(1, n + 2)), capacity=cap)
        w.name = f"random_{t}"
        check_full(w, pad_id=int(rng.integers(0, 5)))


def test_random_medium_windows():
    # windows past the one-block-per-rank limit (ranks of up to 60,000 samples) in random
    # shapes: 1-24 ranks of unequal sizes, uniform, lognormal and bimodal lengths, budgets
    # from below the longest sample to 2^23 (where a wide length range sends group
    # discovery to pointer jumping), join and non-join modes, per-rank slot capacities
    import torch

    rng = np.random.default_rng(2025)
    for t in range(14):
        W = int(rng.integers(1, 25))
        big = int(rng.integers(0, W))
        kind = t % 3
        per = []
        for r in range(W):
            m = int(rng.integers(16385, 60000)) if r == big else int(rng.integers(0, 9000))
            if kind == 0:
                x = rng.integers(1, int(rng.integers(2, 3000)), size=m)
            elif kind == 1:
                x = np.clip(np.rint(synth.lognormal(rng, 200, 1.5, m)), 1, 8000).astype(np.int64)
            else:
                x = np.where(rng.random(m) < 0.9, rng.integers(8, 300, size=m), rng.integers(2000, 8000, size=m))
            per.append(x)
        jump = t % 5 == 4
        if jump:   # lengths 1 and 8000 in the window: more distinct steps than the run table holds
            per[big] = np.concatenate([per[big], [1, 8000]])
        n = sum(len(x) for x in per)
        budget = 1 << 23 if jump else int(rng.integers(2000, 300000))
        mode = "nonjoin" if t % 4 == 3 else "join"
        cap = rng.integers(0, 40, size=W) if t % 6 == 1 else None
        w = win(per, budget, mode=mode, quota=int(rng.integers(1, n + 2)), capacity=cap)
        w.name = f"random_medium_{t}"
        if jump:
            log(f"case {w.name}: W={w.W} n={w.n} budget={w.budget} mode={w.mode} (plan only)")
            ref = oracle.plan_window(w)
            pipe, _ = run_gpu(w, tokens=torch.zeros(64, dtype=torch.int32, device="cuda"), collate=False)
            compare_plan(w, pipe, ref)
            compare_loss_weights(pipe, ref)
        else:
            check_full(w, pad_id=int(rng.integers(0, 5)))


def test_sampler_padding_identity_coverage():
    # identity-coverage audit arithmetic: N = 57,284 over 8 ranks leaves P = 4 padding views
    views, q, P = synth.sampler_views(57284, 8, seed=3)
    rng = np.random.default_rng(3)
    lens = rng.integers(16, 12110, size=57284)
    w = win([lens[v] for v in views], 12288, identity=np.concatenate(views), num_identities=57284)
    w.name = "sampler_padding_57284"
    pipe, ref = check_full(w)
    assert pipe.info["missing_ids"] == 0 and pipe.info["duplicate_ids"] == P == 4


def test_workload_small_full():
    w = synth.WORKLOADS["ln512_w2x2048"].window()
    check_full(w)


@pytest.mark.parametrize("name", ["text_w8x65536", "bimodal_w16x65536", "mm_w8x262144", "ln480_w64x262144"])
def test_workload_full_size(name):
    # the launch configuration the benchmark times; every output element is compared
    w = synth.WORKLOADS[name].window()
    log(f"workload {name}: n={w.n} tokens={w.total_tokens}")
    ref = oracle.plan_window(w)
    log(f"  oracle plan done: steps={ref.steps} padded={ref.padded_elems}")
    pipe, outs = run_gpu(w)
    log("  gpu pipeline done")
    compare_plan(w, pipe, ref)
    compare_loss_weights(pipe, ref)
    log("  plan and loss weights equal")
    compare_collate_sampled(w, outs, ref)
    collate_properties(outs, ref)
    compare_collate_by_rank(w, outs, ref, pipe.win.tokens)
    log("  every output element equal")
    del pipe, outs
    import torch
    torch.cuda.empty_cache()


@pytest.mark.parametrize("case", ["at_block_limit", "past_block_limit", "wide_lengths", "one_length_per_rank",
                                  "long_rank", "tile_edges", "many_ranks", "many_ranks_jump", "max_lengths",
                                  "max_lengths_one_block", "budget_int64_max", "budget_int64_max_jump"])
def test_grouping_paths(case):
    # The two grouping paths (one block per rank up to 16,384 samples per rank, the
    # multi-block sort and run-table walk beyond) at the limit; lengths up to 2^25 (all
    # four byte digits of the one-block sort in use) with the collate left out (the token
    # stream of such lengths would not fit); equal lengths within each rank (no digit
    # varies); a rank of 700,000 samples (342 sort tiles: the per-rank scan of the tiles'
    # run counts takes two passes of its block) beside one of 3; ranks one position past,
    # at and one short of a tile edge, with empty and one-sample ranks; 1,100 ranks (more
    # than the rank table kernels stage in LDS) with one past the one-block limit, grouped
    # by the run-table walk and, at budget 2^23 with lengths 1..8000, by pointer jumping;
    # lengths over the whole valid range [1, 2^31 - 1] (31-bit keys: four radix passes of
    # 8-bit digits; with ranks of at most 16,384 samples, the one-block sort's top byte)
    # at a budget of 2^40 (64-bit batch sizes), plan only; a budget of 2^63 - 1 (batch
    # sizes past any rank: every group after the first takes the rest of its rank), on the
    # one-block path and on pointer jumping (plan only there)
    import torch

    rng = np.random.default_rng(61)
    if case == "at_block_limit":
        per = [rng.integers(1, 5000, 16384), rng.integers(1, 5000, 100), rng.integers(1, 5000, 16384)]
        w = win(per, 20000)
    elif case == "past_block_limit":
        per = [rng.integers(1, 5000, 16385), rng.integers(1, 5000, 5)]
        w = win(per, 20000)
    elif case == "wide_lengths":
        per = [np.concatenate([rng.integers(1, 1 << 25, 3000), rng.integers(1, 300, 1000)]) for _ in range(3)]
        w = win(per, 1 << 21)
    elif case == "long_rank":
        per = [rng.integers(1, 3000, 700000), rng.integers(1, 3000, 3)]
        w = win(per, 20000)
    elif case == "tile_edges":
        per = [rng.integers(1, 5000, 10 * 2048 + 1), rng.integers(1, 5000, 10 * 2048),
               np.zeros(0, np.int64), rng.integers(1, 5000, 10 * 2048 - 1), rng.integers(1, 5000, 1),
               rng.integers(1, 5000, 2)]
        w = win(per, 20000)
    elif case in ("many_ranks", "many_ranks_jump"):
        per = [rng.integers(1, 3000, 20000)] + [rng.integers(1, 3000, int(rng.integers(0, 21))) for _ in range(1099)]
        if case == "many_ranks_jump":
            per[0] = np.concatenate([per[0], [1, 8000]])
        w = win(per, (1 << 23) if case == "many_ranks_jump" else 20000)
    elif case == "max_lengths":
        top = (1 << 31) - 1
        per = [np.concatenate([rng.integers(1, top, 17000), [top, 1, top]]), rng.integers(1, top, 3),
               np.zeros(0, np.int64), np.concatenate([rng.integers(1, top, 2000), [top, top, 1]])]
        w = win(per, 1 << 40)
    elif case == "budget_int64_max":
        per = [rng.integers(1, 3000, 2000), rng.integers(1, 3000, 500), np.array([1, 1, 2])]
        w = win(per, (1 << 63) - 1)
    elif case == "budget_int64_max_jump":
        per = [rng.integers(1, 20000, 17000), rng.integers(1, 100, 5)]
        w = win(per, (1 << 63) - 1)
    elif case == "max_lengths_one_block":
        top = (1 << 31) - 1
        per = [np.concatenate([rng.integers(1, top, 2000), [top, 1, top]]), rng.integers(1, top, 3)]
        w = win(per, 1 << 40)
    else:
        per = [np.full(3000, 77), np.full(10, 5000), np.full(1, 1)]
        w = win(per, 9000)
    w.name = f"paths_{case}"
    log(f"case {w.name}: W={w.W} n={w.n} budget={w.budget}")
    ref = oracle.plan_window(w)
    if case in ("wide_lengths", "long_rank", "many_ranks_jump", "max_lengths", "max_lengths_one_block",
                "budget_int64_max_jump"):
        pipe, _ = run_gpu(w, tokens=torch.zeros(64, dtype=torch.int32, device="cuda"), collate=False)
        compare_plan(w, pipe, ref)
        compare_loss_weights(pipe, ref)
    else:
        pipe, outs = run_gpu(w)
        compare_plan(w, pipe, ref)
        compare_collate_full(w, outs, ref)
        compare_loss_weights(pipe, ref)


def _numpy_coverage(ids, n, identity=None, nid=0):
    cnt = np.bincount(ids, minlength=n)
    bad = int((cnt != 1).sum())
    if identity is None:
        return bad, int((cnt == 0).sum()), int(np.maximum(cnt - 1, 0).sum())
    icnt = np.bincount(identity[ids], minlength=nid)
    return bad, int((icnt == 0).sum()), int(np.maximum(icnt - 1, 0).sum())


@pytest.mark.parametrize("case", ["permutation", "duplicates", "missing_and_dup", "identity_map"])
def test_check_coverage_entry_point(case):
    import torch
    import paper_2606_19989_amd as odb

    rng = np.random.default_rng(21)
    n = 100_003
    w = win([rng.integers(1, 50, 60_000), rng.integers(1, 50, n - 60_000)], 4096)
    ids = rng.permutation(n).astype(np.int32)
    identity, nid = None, 0
    if case == "duplicates":
        ids[5] = ids[6]
    elif case == "missing_and_dup":
        ids[:100] = ids[100:200]
    elif case == "identity_map":
        nid = 70_000
        identity = np.concatenate([np.arange(nid), rng.integers(0, nid, n - nid)]).astype(np.int64)
        w.identity, w.num_identities = identity, nid
    tok_off, toks, ident = synth.device_tensors(w, "cuda")
    dwin = odb.DeviceWindow(w.rank_off, tok_off, toks, ident, nid)
    ws = torch.empty(odb.odb_workspace_size(dwin), dtype=torch.uint8, device="cuda")
    emitted = torch.from_numpy(ids[:70_000].copy()).cuda()
    left = torch.from_numpy(ids[70_000:].copy()).cuda()
    log(f"coverage case {case}")
    info = odb.odb_check_coverage(dwin, emitted, emitted.numel(), left, left.numel(), ws)
    bad, miss, dup = _numpy_coverage(ids.astype(np.int64), n, identity, nid)
    assert (info["bad_views"], info["missing_ids"], info["duplicate_ids"]) == (bad, miss, dup)


SKETCH_CV_RTOL = 1e-15   # both sides: a few correctly rounded fp64 operations on exact integers


def _compare_sketch(got, want):
    for f in ("samples", "short_samples", "sum_len", "sum_sq", "min_len", "max_len", "high_roi"):
        assert got[f] == want[f], (f, got[f], want[f])
    assert got["short_fraction"] == want["short_fraction"]
    assert abs(got["mean"] - want["mean"]) <= 2.0 ** -52 * want["mean"]
    assert abs(got["cv"] - want["cv"]) <= SKETCH_CV_RTOL * max(want["cv"], 1e-300), (got["cv"], want["cv"])


@pytest.mark.parametrize("name", list(synth.WORKLOADS))
def test_length_sketch(name):
    # the screen the practical-guidance section prescribes: a 1k-5k sketch (ids drawn
    # without replacement), plus leading prefixes of the window
    import torch
    import paper_2606_19989_amd as odb

    w = synth.WORKLOADS[name].window()
    tok_off = torch.from_numpy(w.tok_off).cuda()
    win = odb.DeviceWindow(w.rank_off, tok_off, torch.zeros(4, dtype=torch.int32, device="cuda"), None, 0)
    ws = torch.empty(odb.odb_workspace_size(win), dtype=torch.uint8, device="cuda")
    rng = np.random.default_rng(51)
    log(f"sketch {name}: n={w.n}")
    for k in (1000, 5000):
        ids = rng.choice(w.n, size=min(k, w.n), replace=False).astype(np.int32)
        got = odb.odb_length_sketch(win, torch.from_numpy(ids).cuda(), len(ids), w.budget, ws)
        _compare_sketch(got, oracle.length_sketch(w.tok_off, ids, w.budget))
    for count in (0, 1, min(w.n, 100_000)):
        got = odb.odb_length_sketch(win, None, count, w.budget, ws)
        _compare_sketch(got, oracle.length_sketch(w.tok_off, np.arange(count), w.budget))
    del ws, tok_off


def test_length_sketch_whole_window_and_edge_cases():
    import torch
    import paper_2606_19989_amd as odb

    w = synth.WORKLOADS["text_w8x65536"].window()
    tok_off = torch.from_numpy(w.tok_off).cuda()
    win = odb.DeviceWindow(w.rank_off, tok_off, torch.zeros(4, dtype=torch.int32, device="cuda"), None, 0)
    ws = torch.empty(odb.odb_workspace_size(win), dtype=torch.uint8, device="cuda")
    log("sketch whole window text_w8x65536")
    got = odb.odb_length_sketch(win, None, w.n, w.budget, ws)
    _compare_sketch(got, oracle.length_sketch(w.tok_off, None, w.budget))
    for budget in (1, 4, 700 * 4, 700 * 4 + 1, 1 << 40):
        ids = np.array([0, 0, 5, w.n - 1, 5], dtype=np.int32)   # repeated ids count every time
        got = odb.odb_length_sketch(win, torch.from_numpy(ids).cuda(), len(ids), budget, ws)
        _compare_sketch(got, oracle.length_sketch(w.tok_off, ids, budget))
    # an id outside the window is caught by the kernel's own bounds check
    bad = torch.tensor([3, w.n], dtype=torch.int32, device="cuda")
    with pytest.raises(odb.OdbError) as e:
        odb.odb_length_sketch(win, bad, 2, w.budget, ws)
    assert e.value.status == odb.ODB_E_INVALID_DATA


def test_length_sketch_sums_past_64_bits():
    # lengths near 2^31: the sum of squares passes 2^64 (the 128-bit accumulation), at a
    # budget of 2^40 (the short-sample test 4 l < L_max in 64 bits)
    import torch
    import paper_2606_19989_amd as odb

    rng = np.random.default_rng(53)
    n = 6000
    lens = np.concatenate([rng.integers(1 << 30, 1 << 31, n - 4), [(1 << 31) - 1, 1, (1 << 31) - 1, 7]])
    off = np.zeros(n + 1, np.int64)
    np.cumsum(lens, out=off[1:])
    tok_off = torch.from_numpy(off).cuda()
    win = odb.DeviceWindow(np.array([0, n], np.int64), tok_off, torch.zeros(4, dtype=torch.int32, device="cuda"),
                           None, 0)
    ws = torch.empty(odb.odb_workspace_size(win), dtype=torch.uint8, device="cuda")
    want = oracle.length_sketch(off, None, 1 << 40)
    assert want["sum_sq"] >= 1 << 64
    log("sketch past 64 bits")
    _compare_sketch(odb.odb_length_sketch(win, None, n, 1 << 40, ws), want)
    ids = rng.integers(0, n, 5000).astype(np.int32)   # with repeats
    for budget in (1 << 40, 1 << 33, 7):
        got = odb.odb_length_sketch(win, torch.from_numpy(ids).cuda(), len(ids), budget, ws)
        _compare_sketch(got, oracle.length_sketch(off, ids, budget))


def test_collate_tile_width_at_the_length_limit():
    # tiles 2^31 - 1 and 2^31 - 2 elements wide (the longest valid samples): a 4-element
    # group that starts 1 to 3 columns before a row's end must still take the row-edge
    # path there (column + 4 is past 2^31); every element around each row edge and a
    # random sample are checked against the oracle's per-element rule
    import torch

    top = (1 << 31) - 1
    for lens, name in (([top, top, top - 1], "width_2p31m1"), ([top - 1, top - 1, 5, top - 2], "width_2p31m2")):
        w = win([np.array(lens, np.int64)], 1 << 40)
        w.name = name
        log(f"collate at the length limit: {name}, {int(w.tok_off[-1])} tokens")
        ref = oracle.plan_window(w)
        pipe, outs = run_gpu(w)
        compare_plan(w, pipe, ref)
        P = ref.padded_elems
        edges = []
        for k in range(len(ref.slot_rows)):
            t0, ml, rows = int(ref.slot_tile_off[k]), int(ref.slot_maxlen[k]), int(ref.slot_rows[k])
            for r in range(1, rows + 1):
                edges.append(np.arange(t0 + r * ml - 24, t0 + r * ml + 24))
        idx = np.concatenate(edges + [np.random.default_rng(5).integers(0, P, 20000), [0, P - 1]])
        idx = np.unique(idx[(idx >= 0) & (idx < P)])
        want = oracle.collate_elements(ref, w.tok_off, synth.token_ids, idx, 0)
        ti = torch.from_numpy(idx).cuda()
        for label, g, e in zip(["input_ids", "labels", "attention_mask", "position_ids"], outs, want):
            got = g[ti].cpu().numpy()
            bad = np.nonzero(got != e)[0]
            assert len(bad) == 0, f"{name} {label}: {len(bad)} mismatches, first at {idx[bad[0]]}"
        del pipe, outs, ti
        torch.cuda.synchronize()
        torch.cuda.empty_cache()


def test_collate_from_emit_order():
    # odb_collate without row records gathers them from the emitted ids itself; both
    # routes give the oracle's outputs
    import torch
    import paper_2606_19989_amd as odb

    for w in (synth.WORKLOADS["ln512_w2x2048"].window(), adversarial_windows()[4], adversarial_windows()[16]):
        log(f"collate from emit order: {w.name}")
        ref = oracle.plan_window(w)
        pipe, outs = run_gpu(w, pad_id=3)
        P = int(pipe.info["padded_elems"])
        alt = tuple(torch.empty(max(P, 1), dtype=torch.int32, device="cuda") for _ in range(4))
        odb.odb_collate(pipe.win, pipe.num_slots, pipe.emit_order, pipe.slot_rows, pipe.slot_maxlen,
                        pipe.slot_row_off, pipe.slot_tile_off, 3, P, *alt, pipe.ws)
        torch.cuda.synchronize()
        odb.odb_collate_status(pipe.ws)
        compare_collate_full(w, tuple(a[:P] for a in alt), ref, 3)
        for a, b in zip(alt, outs):
            assert torch.equal(a[:P], b)


def test_collate_output_capacity():
    # outputs shorter than the padded size: the first out_capacity elements are the
    # oracle's and nothing at or past out_capacity is written, with and without row
    # records, at capacities that end inside a group, a step and a run of steps
    import torch
    import paper_2606_19989_amd as odb

    w = synth.WORKLOADS["ln512_w2x2048"].window()
    ref = oracle.plan_window(w)
    pipe, outs = run_gpu(w, pad_id=5)
    compare_collate_full(w, outs, ref, 5)
    P = int(pipe.info["padded_elems"])
    assert P > 70000
    sentinel = -12345
    for cap in (0, 1, 3, 1023, 1025, 65 * 1024 + 7, P - 1):
        for records in (True, False):
            log(f"collate with out_capacity={cap} of {P}, row records={records}")
            alt = tuple(torch.full((P + 64,), sentinel, dtype=torch.int32, device="cuda") for _ in range(4))
            rec = dict(row_token_start=pipe.row_token_start, row_len=pipe.row_len) if records else {}
            odb.odb_collate(pipe.win, pipe.num_slots, pipe.emit_order, pipe.slot_rows, pipe.slot_maxlen,
                            pipe.slot_row_off, pipe.slot_tile_off, 5, cap, *alt, pipe.ws, **rec)
            torch.cuda.synchronize()
            odb.odb_collate_status(pipe.ws)
            for a, b in zip(alt, outs):
                assert torch.equal(a[:cap], b[:cap])
                assert bool((a[cap:] == sentinel).all())


def test_concurrent_collates():
    # two collates in flight at once on two streams, each with its own workspace (and so
    # its own run counter) and outputs, repeated: both give the oracle's outputs
    import torch
    import paper_2606_19989_amd as odb

    w = synth.WORKLOADS["ln512_w2x2048"].window()
    ref = oracle.plan_window(w)
    pipes = []
    for pad in (2, 9):
        pipe, outs = run_gpu(w, pad_id=pad)
        compare_collate_full(w, outs, ref, pad)
        pipes.append((pipe, outs, pad))
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    P = int(pipes[0][0].info["padded_elems"])
    alts = [tuple(torch.full((P,), -1, dtype=torch.int32, device="cuda") for _ in range(4)) for _ in pipes]
    torch.cuda.synchronize()
    for rep in range(3):
        log(f"two concurrent collates, repetition {rep}")
        for (pipe, _, pad), alt, st in zip(pipes, alts, streams):
            odb.odb_collate(pipe.win, pipe.num_slots, pipe.emit_order, pipe.slot_rows, pipe.slot_maxlen,
                            pipe.slot_row_off, pipe.slot_tile_off, pad, P, *alt, pipe.ws, st,
                            row_token_start=pipe.row_token_start, row_len=pipe.row_len)
        torch.cuda.synchronize()
        for (pipe, outs, _), alt in zip(pipes, alts):
            odb.odb_collate_status(pipe.ws)
            for a, b in zip(alt, outs):
                assert torch.equal(a, b)
            for a in alt:
                a.fill_(-1)
        torch.cuda.synchronize()


def _formed(w):
    import torch
    import paper_2606_19989_amd as odb

    tok_off, toks, ident = synth.device_tensors(w, "cuda")
    win_ = odb.DeviceWindow(w.rank_off, tok_off, toks, ident, w.num_identities)
    pipe = odb.Pipeline(win_, w.budget, mode=w.mode, quota=w.quota, capacity=w.capacity)
    pipe.form()
    torch.cuda.synchronize()
    return pipe


@pytest.mark.parametrize("mode", ["join", "nonjoin"])
def test_align_rejects_a_wrong_sorted_length(mode):
    # a stage-1 sorted length that keeps the order valid but is not the sample's CSR
    # length is found once the plan is built (emitted rows, or leftovers in non-join)
    import paper_2606_19989_amd as odb

    rng = np.random.default_rng(31)
    w = win([rng.integers(10, 3000, 5000), rng.integers(10, 3000, 3000)], 8192, mode=mode,
            quota=2000 if mode == "nonjoin" else 0)
    pipe = _formed(w)
    ref = oracle.plan_window(w)
    slen = pipe.sorted_len.cpu().numpy()
    # a position strictly inside a run of descending lengths: lowering its length by one
    # keeps (length desc, id asc).  Non-join emits the shortest samples first, so a long
    # one (an early position) is left over and checked on that path
    cand = [p for p in range(1, 4999) if slen[p - 1] > slen[p] > slen[p + 1] + 1]
    p = cand[len(cand) // 2] if mode == "join" else cand[0]
    order = pipe.order.cpu().numpy()
    if mode == "nonjoin":
        assert order[p] in set(ref.leftover.tolist())
    bad = pipe.sorted_len.clone()
    bad[p] -= 1
    pipe.sorted_len.copy_(bad)
    log(f"wrong sorted length at position {p} ({mode}); the oracle leaves {ref.info['leftover_samples']} over")
    with pytest.raises(odb.OdbError) as e:
        pipe.align()
    assert e.value.status == odb.ODB_E_INVALID_DATA
    assert "sorted length" in str(e.value)


def test_collate_flags_a_bad_row_record():
    # a row record outside the token stream is written as padding and reported
    import torch
    import paper_2606_19989_amd as odb

    w = synth.WORKLOADS["ln512_w2x2048"].window()
    pipe, outs = run_gpu(w)
    P = int(pipe.info["padded_elems"])
    pipe.row_token_start[5] = int(w.tok_off[-1])   # starts at the end of the stream
    pipe.collate()
    torch.cuda.synchronize()
    with pytest.raises(odb.OdbError) as e:
        odb.odb_collate_status(pipe.ws)
    assert e.value.status == odb.ODB_E_INVALID_DATA
    pipe.row_token_start[5] = int(w.tok_off[int(pipe.emit_order[5])])
    pipe.collate()
    torch.cuda.synchronize()
    odb.odb_collate_status(pipe.ws)
    ref = oracle.plan_window(w)
    compare_collate_full(w, tuple(o[:P] for o in pipe.outputs), ref)


def test_two_stream_schedule():
    # the benchmark's schedule: step i+1's plan on one stream beside step i's collate on
    # another, two plan buffers, one set of outputs; after several steps the outputs and
    # both plans are the oracle's
    import torch
    import paper_2606_19989_amd as odb
    import bench

    w = synth.WORKLOADS["text_w8x65536"].window()
    log(f"two-stream schedule on {w.name}")
    plan_stream, collate_stream = torch.cuda.Stream(), torch.cuda.Stream()
    tok_off, toks, ident = synth.device_tensors(w, "cuda")
    dwin = odb.DeviceWindow(w.rank_off, tok_off, toks, ident, w.num_identities)
    pipes = [odb.Pipeline(dwin, w.budget, mode=w.mode, quota=w.quota) for _ in range(2)]
    for p in pipes:
        p.run()
        pipes[1].outputs = pipes[0].outputs
    torch.cuda.synchronize()
    pipes[0].outputs[0].fill_(-7)
    sec, coll, _ = bench.pipelined_steps(pipes, plan_stream, collate_stream, 5)
    assert len(coll) == 5 and sec > 0
    ref = oracle.plan_window(w)
    for p in pipes:
        odb.odb_collate_status(p.ws)
        compare_plan(w, p, ref)
    P = ref.padded_elems
    outs = tuple(o[:P] for o in pipes[0].outputs)
    compare_collate_sampled(w, outs, ref)
    collate_properties(outs, ref)
    compare_collate_by_rank(w, outs, ref, toks)
