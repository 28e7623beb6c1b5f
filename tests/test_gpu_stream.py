"""GPU parity of the unified streaming loop (odb_stream_plan) with the oracle: every plan
array, the per-round trace, the summary, the loss weights bit for bit and, on small
cases, every collate element."""
import numpy as np
import pytest

import oracle
import synth
from _parity import compare_row_records, log

pytestmark = pytest.mark.gpu

STREAM_INFO_EXACT = ["steps", "rounds", "emit_rounds", "skip_rounds", "stop_reason", "views", "emitted_views",
                     "undelivered_views", "pending_views", "real_tokens", "padded_elems", "max_step_samples",
                     "splits", "overflow_groups", "missing_ids", "duplicate_ids", "bad_views",
                     "second_gather_rounds", "max_outstanding"]


def offsets(lens):
    return np.concatenate([[0], np.cumsum(np.asarray(lens, dtype=np.int64))])


def run_case(name, lens, perm, W, budget, buffer_size, depth, rate, mode="join", quota=0, cap=None, pad_id=0,
             full_collate=True, tokens=None, max_rounds=None, device_perm=None, slot_capacity=None):
    import torch
    import paper_2606_19989_amd as odb

    N = len(lens)
    log(f"stream case {name}: N={N} W={W} budget={budget} buffer={buffer_size} depth={depth} mode={mode} "
        f"quota={quota} rate={list(rate)[:8]}")
    tok_off = offsets(lens)
    m_mode = oracle.MODE_NONJOIN if mode == "nonjoin" else oracle.MODE_JOIN
    ref = oracle.stream(tok_off, perm, W, budget, mode=m_mode, quota=quota, buffer_size=buffer_size, depth=depth,
                        rate=rate, capacity=cap)
    rank_off = np.linspace(0, N, W + 1).astype(np.int64)   # not used by the streaming loop
    d_tok_off = torch.from_numpy(tok_off).cuda()
    toks = tokens if tokens is not None else synth.fill_tokens_torch(int(tok_off[-1]), "cuda")
    win = odb.DeviceWindow(rank_off, d_tok_off, toks, None, 0)
    dperm = perm if device_perm is None else device_perm
    sp = odb.StreamPipeline(win, torch.from_numpy(np.asarray(dperm, dtype=np.int32)).cuda(), budget,
                            buffer_size=buffer_size, depth=depth, rate=rate, mode=mode, quota=quota, capacity=cap,
                            pad_id=pad_id, max_rounds=max_rounds, slot_capacity=slot_capacity)
    info = sp.plan()
    torch.cuda.synchronize()
    for f in STREAM_INFO_EXACT:
        assert info[f] == ref.sinfo[f], (f, info[f], ref.sinfo[f])
    assert abs(info["pad_fraction"] - ref.sinfo["pad_fraction"]) <= 1e-12 * max(ref.sinfo["pad_fraction"], 1e-300)
    assert np.array_equal(sp.trace_array(), ref.trace), "trace"
    S, K, M = ref.steps, W * ref.steps, ref.sinfo["views"]
    E = ref.sinfo["emitted_views"]
    h = lambda t, k: t[:k].cpu().numpy()
    assert np.array_equal(h(sp.slot_rows, K), ref.slot_rows), "slot_rows"
    assert np.array_equal(h(sp.slot_maxlen, K), ref.slot_maxlen), "slot_maxlen"
    assert np.array_equal(h(sp.slot_tokens, K), ref.slot_tokens), "slot_tokens"
    assert np.array_equal(h(sp.slot_tokens_approx, K).view(np.int64), ref.slot_tokens_approx.view(np.int64))
    assert np.array_equal(h(sp.slot_row_off, K + 1), ref.slot_row_off), "slot_row_off"
    assert np.array_equal(h(sp.slot_tile_off, K + 1), ref.slot_tile_off), "slot_tile_off"
    assert np.array_equal(h(sp.emit_views, E), ref.emit_views), "emit_views"
    assert np.array_equal(h(sp.emit_order, E), ref.emit_order), "emit_order"
    compare_row_records(tok_off, sp, ref.emit_order)
    assert np.array_equal(h(sp.left_views, M - E), ref.left_views), "left_views"
    assert np.array_equal(h(sp.left_off, W + 1), ref.left_off), "left_off"
    for m in (oracle.WEIGHT_SAMPLE, oracle.WEIGHT_TOKEN_APPROX, oracle.WEIGHT_TOKEN_EXACT):
        wt, st, ss = sp.loss_weights(m)
        ewt, est, ess = ref.loss_weights(m)
        assert np.array_equal(wt.cpu().numpy().view(np.int64), ewt.view(np.int64)), ("weights", m)
        assert np.array_equal(st.cpu().numpy(), est) and np.array_equal(ss.cpu().numpy(), ess)
    if full_collate:
        outs = sp.collate()
        torch.cuda.synchronize()
        odb.odb_collate_status(sp.ws)
        want = ref.collate(tok_off, toks.cpu().numpy(), pad_id)
        for name_, g, e in zip(["input_ids", "labels", "attention_mask", "position_ids"], outs, want):
            assert np.array_equal(g.cpu().numpy(), e), name_
    return sp, ref


def edge_cases():
    rng = np.random.default_rng(71)
    out = []
    add = lambda name, lens, W, budget, buf, depth, rate, **kw: out.append(
        (name, np.asarray(lens, dtype=np.int64), W, budget, buf, depth, np.asarray(rate, dtype=np.int32), kw))
    add("empty", [], 3, 100, 4, 4, [4, 4, 4])
    add("one_sample_four_ranks", [7], 4, 100, 2, 3, [1, 2, 3, 1])           # padding wraps N = 1 times 3
    add("fewer_samples_than_ranks", [5, 9, 2], 5, 12, 1, 1, [1] * 5)
    add("buffer_one", rng.integers(1, 50, 40), 3, 30, 1, 1, [1, 1, 1])
    add("slow_rank", rng.integers(1, 900, 700), 4, 4096, 64, 64, [1, 64, 64, 64])
    add("deep_envelope", rng.integers(1, 900, 3000), 3, 8192, 128, 1024, [300, 17, 128])
    add("tiny_budget", rng.integers(1, 9, 500), 2, 1, 50, 80, [20, 80])
    add("overflow_capacity", rng.integers(1, 600, 1500), 3, 3000, 200, 256, [256, 100, 50], cap=np.array([3, 0, 5]))
    add("max_depth", rng.integers(1, 3000, 20000), 2, 16384, 4096, 4096, [4096, 4096])
    # depth 1500: four sort keys per thread; skip rounds while the slow rank fills
    add("depth_1500", rng.integers(1, 5000, 12000), 3, 12000, 1200, 1500, [1500, 700, 1500])
    # one rank with 600,000 views: its emitted-view bits exceed the LDS budget and are set
    # in global memory
    add("long_rank", rng.integers(1, 12, 600000), 1, 64, 1024, 1024, [1024])
    # more ranks than a round block has threads (the round decision loops over them)
    add("many_ranks", rng.integers(1, 300, 4000), 600, 2000, 4, 4, [2] * 600)
    n = 2003
    for q in (1, 500, n + 1):
        add(f"nonjoin_q{q}", rng.integers(1, 2000, n), 4, 6000, 100, 150, [150, 90, 40, 150], mode="nonjoin",
            quota=q)
    add("nonjoin_capacity", rng.integers(1, 900, 900), 2, 2500, 64, 64, [64, 7], mode="nonjoin", quota=700,
        cap=np.array([2, 4]))
    return out


@pytest.mark.parametrize("idx", range(len(edge_cases())))
def test_stream_edge_cases(idx):
    name, lens, W, budget, buf, depth, rate, kw = edge_cases()[idx]
    perm = np.random.default_rng(idx).permutation(len(lens)).astype(np.int32)
    run_case(name, lens, perm, W, budget, buf, depth, rate, pad_id=idx, **kw)


def test_stream_random_small():
    rng = np.random.default_rng(72)
    for t in range(30):
        N = int(rng.integers(1, 3000))
        W = int(rng.integers(1, 9))
        lens = rng.integers(1, int(rng.integers(2, 4000)), size=N)
        buf = int(rng.integers(1, 300))
        depth = buf + int(rng.integers(0, 200))
        rate = rng.integers(1, depth + 1, size=W).astype(np.int32)
        mode = "nonjoin" if t % 3 == 2 else "join"
        cap = rng.integers(0, 6, size=W) if t % 4 == 1 else None
        run_case(f"random_{t}", lens, rng.permutation(N).astype(np.int32), W, int(rng.integers(1, 30000)), buf, depth,
                 rate, mode=mode, quota=int(rng.integers(1, N + 2)), cap=cap, pad_id=t % 5)


def _stream_pipeline(lens, perm, W, budget, buffer_size, depth, rate, **kw):
    import torch
    import paper_2606_19989_amd as odb

    tok_off = offsets(lens)
    win = odb.DeviceWindow(np.linspace(0, len(lens), W + 1).astype(np.int64), torch.from_numpy(tok_off).cuda(),
                           synth.fill_tokens_torch(int(tok_off[-1]), "cuda"), None, 0)
    return odb.StreamPipeline(win, torch.from_numpy(np.asarray(perm, dtype=np.int32)).cuda(), budget,
                              buffer_size=buffer_size, depth=depth, rate=np.asarray(rate, dtype=np.int32), **kw)


@pytest.mark.parametrize("mode", ["join", "nonjoin"])
def test_stream_round_limit(mode):
    # rounds are enqueued in chunks sized by a lower bound on the rounds left (a slow rank
    # makes the first bound short, so later chunks follow): a limit equal to the rounds
    # the iteration takes passes and matches the oracle, one round fewer is a capacity
    # error, and so is a limit of one round
    import paper_2606_19989_amd as odb

    rng = np.random.default_rng(76)
    N, W = 700, 4
    lens = rng.integers(1, 900, N)
    perm = rng.permutation(N).astype(np.int32)
    rate = np.array([3, 64, 64, 64], np.int32)
    kw = dict(mode=mode, quota=N // 2 if mode == "nonjoin" else 0)
    m_mode = oracle.MODE_NONJOIN if mode == "nonjoin" else oracle.MODE_JOIN
    ref = oracle.stream(offsets(lens), perm, W, 4096, mode=m_mode, quota=kw["quota"], buffer_size=64, depth=64,
                        rate=rate)
    R = int(ref.sinfo["rounds"])
    log(f"round limit {mode}: the iteration takes {R} rounds")
    assert R > 20
    run_case(f"round_limit_{mode}", lens, perm, W, 4096, 64, 64, rate, max_rounds=R, **kw)
    for limit in (R - 1, 1):
        sp = _stream_pipeline(lens, perm, W, 4096, 64, 64, rate, max_rounds=limit, **kw)
        with pytest.raises(odb.OdbError) as e:
            sp.plan()
        assert e.value.status == odb.ODB_E_CAPACITY, limit


@pytest.mark.parametrize("bad", ["perm", "length"])
def test_stream_rejects_bad_data(bad):
    import paper_2606_19989_amd as odb

    rng = np.random.default_rng(77)
    N, W = 60, 3
    lens = rng.integers(1, 50, N)
    perm = rng.permutation(N).astype(np.int32)
    if bad == "perm":
        perm[17] = N       # outside [0, N)
    else:
        lens[perm[17]] = 0
    sp = _stream_pipeline(lens, perm, W, 200, 4, 4, [4, 4, 4])
    with pytest.raises(odb.OdbError) as e:
        sp.plan()
    assert e.value.status == odb.ODB_E_INVALID_DATA


def test_stream_ignores_views_after_the_stop():
    # the grouping of the round after the one that meets a non-join quota runs before the
    # quota is known, and must leave no trace: a perm entry outside [0, N) for a view only
    # that round fetches does not fail the call, and the plan is the one of the valid perm
    rng = np.random.default_rng(78)
    N, W = 40, 2
    lens = rng.integers(1, 30, N)
    perm = rng.permutation(N).astype(np.int32)
    bad = perm.copy()
    bad[8] = N          # view 8: rank 0's first view of the second round
    sp, ref = run_case("stop_then_bad_view", lens, perm, W, 100, 4, 4, [4, 4], mode="nonjoin", quota=1,
                       device_perm=bad)
    assert ref.sinfo["rounds"] == 1 and ref.sinfo["stop_reason"] == oracle.STOP_QUOTA


def test_stream_window_workload():
    # the multimodal window's samples as a dataset streamed through 8 ranks with the
    # paper's default buffer of 1024 and unequal worker throughput
    w = synth.WORKLOADS["mm_w8x262144"].window()
    lens = np.diff(w.tok_off)
    rng = np.random.default_rng(73)
    perm = rng.permutation(len(lens)).astype(np.int32)
    rate = np.array([1024, 512, 1024, 256, 1024, 1024, 768, 1024], dtype=np.int32)
    import torch
    import paper_2606_19989_amd as odb

    from _parity import compare_collate_by_rank_whole_stream

    toks = synth.fill_tokens_torch(int(w.tok_off[-1]), "cuda")
    sp, ref = run_case("mm_stream", lens, perm, 8, w.budget, 1024, 1024, rate, full_collate=False, tokens=toks)
    outs = sp.collate()
    torch.cuda.synchronize()
    odb.odb_collate_status(sp.ws)
    compare_collate_by_rank_whole_stream(w.tok_off, outs, ref, toks)
    log("  every stream collate element equal")
    del sp, outs, toks
    torch.cuda.empty_cache()


@pytest.mark.parametrize("quota_div", [1, 3])
def test_stream_bimodal_nonjoin(quota_div):
    # the bimodal 16-rank window's 1.05M samples streamed in non-join mode with two worker
    # rates and a depth of 2048 (four sort keys per thread): quota N stops when the fast
    # ranks finish, quota N/3 at the quota; plan, trace, weights and every collate element
    # exact
    import torch
    import paper_2606_19989_amd as odb

    from _parity import compare_collate_by_rank_whole_stream, compare_collate_sampled

    w = synth.WORKLOADS["bimodal_w16x65536"].window()
    lens = np.diff(w.tok_off)
    perm = np.random.default_rng(79).permutation(len(lens)).astype(np.int32)
    toks = synth.fill_tokens_torch(int(w.tok_off[-1]), "cuda")
    sp, ref = run_case(f"bimodal_nonjoin_q{quota_div}", lens, perm, 16, 32768, 1024, 2048,
                       np.array([1024, 512] * 8, np.int32), mode="nonjoin", quota=len(lens) // quota_div,
                       full_collate=False, tokens=toks)
    assert ref.sinfo["stop_reason"] == (oracle.STOP_RANK_FINISHED if quota_div == 1 else oracle.STOP_QUOTA)
    outs = sp.collate()
    torch.cuda.synchronize()
    odb.odb_collate_status(sp.ws)
    compare_collate_sampled(w, outs, ref)
    compare_collate_by_rank_whole_stream(w.tok_off, outs, ref, toks)
    log("  every stream collate element equal")
    del sp, outs, toks
    torch.cuda.empty_cache()


def test_stream_full_size():
    # the largest window's 16.7M samples streamed by 64 ranks with the paper's buffer
    # of 1024 and a budget in its L_max range; the benchmark times this configuration.
    # Plan, trace, weights and every collate element (8.5 G per output) are compared
    # exactly
    import torch

    from _parity import collate_properties, compare_collate_by_rank_whole_stream, compare_collate_sampled

    w = synth.WORKLOADS["ln480_w64x262144"].window()
    lens = np.diff(w.tok_off)
    perm = np.random.default_rng(74).permutation(len(lens)).astype(np.int32)
    toks = synth.fill_tokens_torch(int(w.tok_off[-1]), "cuda")
    sp, ref = run_case("ln480_stream", lens, perm, 64, 16384, 1024, 1024, np.full(64, 1024, np.int32),
                       full_collate=False, tokens=toks)
    outs = sp.collate()
    torch.cuda.synchronize()
    import paper_2606_19989_amd as odb
    odb.odb_collate_status(sp.ws)
    compare_collate_sampled(w, outs, ref)
    collate_properties(outs, ref)
    log("  stream collate sampled and properties equal")
    compare_collate_by_rank_whole_stream(w.tok_off, outs, ref, toks)
    log("  every stream collate element equal")
    del sp, outs, toks
    torch.cuda.empty_cache()


def test_stream_two_stream_schedule():
    # the benchmark's streaming schedule: iteration i+1's odb_stream_plan on one stream
    # beside iteration i's collate on another, two plan buffers, one set of outputs
    import torch
    import paper_2606_19989_amd as odb
    import bench

    from _parity import collate_properties, compare_collate_sampled

    w = synth.WORKLOADS["text_w8x65536"].window()
    lens = np.diff(w.tok_off)
    N, W = len(lens), 8
    perm = np.random.default_rng(75).permutation(N).astype(np.int32)
    log(f"two-stream streaming schedule: N={N} W={W}")
    ref = oracle.stream(w.tok_off, perm, W, 16384, buffer_size=1024, depth=1024, rate=np.full(W, 1024))
    plan_stream, collate_stream = torch.cuda.Stream(), torch.cuda.Stream()
    toks = synth.fill_tokens_torch(int(w.tok_off[-1]), "cuda")
    win = odb.DeviceWindow(np.linspace(0, N, W + 1).astype(np.int64), torch.from_numpy(w.tok_off).cuda(), toks,
                           None, 0)
    d_perm = torch.from_numpy(perm).cuda()
    sps = [odb.StreamPipeline(win, d_perm, 16384, buffer_size=1024, depth=1024, rate=np.full(W, 1024, np.int32))
           for _ in range(2)]
    for sp in sps:
        sp.plan()
        sp.collate()
        sps[1].outputs = sps[0].outputs
    torch.cuda.synchronize()
    sps[0].outputs[0].fill_(-7)
    sec, coll, _ = bench.pipelined_steps(sps, plan_stream, collate_stream, 5, plan=bench.stream_plan,
                                         weights=bench.stream_weights)
    assert len(coll) == 5 and sec > 0
    S, E = ref.steps, ref.sinfo["emitted_views"]
    for sp in sps:
        odb.odb_collate_status(sp.ws)
        assert sp.info["steps"] == S
        assert np.array_equal(sp.slot_tile_off[:W * S + 1].cpu().numpy(), ref.slot_tile_off)
        assert np.array_equal(sp.emit_order[:E].cpu().numpy(), ref.emit_order)
        compare_row_records(w.tok_off, sp, ref.emit_order)
    outs = tuple(o[:ref.padded_elems] for o in sps[0].outputs)
    compare_collate_sampled(w, outs, ref)
    collate_properties(outs, ref)
    wt, st, ss = sps[0].loss_weights(oracle.WEIGHT_TOKEN_EXACT)
    ewt, est, ess = ref.loss_weights(oracle.WEIGHT_TOKEN_EXACT)
    assert np.array_equal(wt.cpu().numpy().view(np.int64), ewt.view(np.int64))


def test_stream_quota_cut_retry_at_the_reported_capacity():
    # room for one step per rank first: the call reports W * S and the retry at exactly
    # that capacity must succeed even though the round that reaches the quota stages more
    # steps than the cut keeps
    rng = np.random.default_rng(79)
    N, W = 6007, 5
    lens = np.clip(np.rint(synth.lognormal(rng, 300.0, 1.0, N)), 1, 4000).astype(np.int64)
    perm = rng.permutation(N).astype(np.int32)
    rate = rng.integers(8, 40, W).astype(np.int32)
    sp, ref = run_case("quota_cut_retry", lens, perm, W, 8192, 64, 96, rate, mode="nonjoin", quota=N // 3,
                       slot_capacity=W)
    assert sp.slot_capacity == W * ref.steps


@pytest.mark.parametrize("mode", ["join", "nonjoin"])
def test_stream_max_lengths(mode):
    # lengths over the whole valid range [1, 2^31 - 1] (31-bit sort keys: seven 5-bit
    # digit passes) at a budget of 2^40 (64-bit batch sizes); plan and weights only, the
    # token stream would not fit
    import torch

    rng = np.random.default_rng(78)
    top = (1 << 31) - 1
    lens = np.concatenate([rng.integers(1, top, 600), [top, 1, top], rng.integers(1, 50, 300)])
    perm = rng.permutation(len(lens)).astype(np.int32)
    run_case(f"max_lengths_{mode}", lens, perm, 3, 1 << 40, 64, 96, [64, 30, 64], mode=mode,
             quota=len(lens) // 2 if mode == "nonjoin" else 0, full_collate=False,
             tokens=torch.zeros(64, dtype=torch.int32, device="cuda"))


def test_stream_budget_int64_max():
    # a budget of 2^63 - 1: every group after a round's first takes the rest of the buffer
    rng = np.random.default_rng(80)
    lens = rng.integers(1, 3000, 2500)
    perm = rng.permutation(len(lens)).astype(np.int32)
    run_case("budget_int64_max", lens, perm, 3, (1 << 63) - 1, 128, 200, [128, 50, 128])
