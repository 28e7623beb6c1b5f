"""Shared helpers for the GPU parity tests: run the HIP pipeline through the C ABI and
compare it with the CPU oracle on the same seeded window."""
import sys

import numpy as np

import oracle
import synth

INFO_EXACT = ["steps", "rounds", "stop_reason", "emitted_samples", "leftover_samples", "real_tokens",
              "padded_elems", "max_step_samples", "splits", "overflow_groups", "missing_ids", "duplicate_ids",
              "bad_views", "second_gather_rounds"]
PAD_FRACTION_RTOL = 1e-12


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def run_gpu(w, pad_id=0, tokens=None, collate=True):
    import torch
    import paper_2606_19989_amd as odb

    tok_off, toks, ident = synth.device_tensors(w, "cuda", tokens)
    win = odb.DeviceWindow(w.rank_off, tok_off, toks, ident, w.num_identities)
    pipe = odb.Pipeline(win, w.budget, mode=w.mode, quota=w.quota, capacity=w.capacity, pad_id=pad_id)
    pipe.form()
    pipe.align()
    outs = pipe.collate() if collate else None
    torch.cuda.synchronize()
    if collate:
        odb.odb_collate_status(pipe.ws)
    return pipe, outs


def h(t, k=None):
    x = t if k is None else t[:k]
    return x.cpu().numpy()


def compare_plan(w, pipe, ref):
    n, W = w.n, w.W
    info = pipe.info
    for f in INFO_EXACT:
        assert info[f] == ref.info[f], (f, info[f], ref.info[f])
    pf, rf = info["pad_fraction"], ref.info["pad_fraction"]
    assert abs(pf - rf) <= PAD_FRACTION_RTOL * max(abs(rf), 1e-300) or pf == rf, (pf, rf)
    if n:
        assert np.array_equal(h(pipe.order, n), ref.order), "order"
        assert np.array_equal(h(pipe.sorted_len, n), ref.sorted_len), "sorted_len"
        assert np.array_equal(h(pipe.group_index, n), ref.group_index), "group_index"
    assert np.array_equal(h(pipe.groups_per_rank), ref.groups_per_rank), "groups_per_rank"
    K = W * ref.steps
    assert np.array_equal(h(pipe.slot_rows, K), ref.slot_rows), "slot_rows"
    assert np.array_equal(h(pipe.slot_maxlen, K), ref.slot_maxlen), "slot_maxlen"
    assert np.array_equal(h(pipe.slot_tokens, K), ref.slot_tokens), "slot_tokens"
    # fp64, same operations in the same order on both sides: equal bit for bit
    assert np.array_equal(h(pipe.slot_tokens_approx, K).view(np.int64), ref.slot_tokens_approx.view(np.int64)), \
        "slot_tokens_approx"
    assert np.array_equal(h(pipe.slot_row_off, K + 1), ref.slot_row_off), "slot_row_off"
    assert np.array_equal(h(pipe.slot_tile_off, K + 1), ref.slot_tile_off), "slot_tile_off"
    E, Lf = ref.info["emitted_samples"], ref.info["leftover_samples"]
    assert np.array_equal(h(pipe.emit_order, E), ref.emit_order), "emit_order"
    compare_row_records(w.tok_off, pipe, ref.emit_order)
    assert np.array_equal(h(pipe.leftover, Lf), ref.leftover), "leftover"
    assert np.array_equal(h(pipe.leftover_off), ref.leftover_off), "leftover_off"


def compare_row_records(tok_off, pipe, emit_order):
    """Row records of the plan: token start and length of each emitted row's sample,
    read off the CSR offsets at the oracle's emitted ids."""
    E = len(emit_order)
    ids = np.asarray(emit_order, dtype=np.int64)
    assert np.array_equal(h(pipe.row_token_start, E), tok_off[ids]), "row_token_start"
    assert np.array_equal(h(pipe.row_len, E), (tok_off[ids + 1] - tok_off[ids]).astype(np.int32)), "row_len"


def compare_loss_weights(pipe, ref):
    """Every mode's per-slot weights (bit for bit) and per-step sums (Eq. 2, App. B)."""
    import torch

    for mode in (oracle.WEIGHT_SAMPLE, oracle.WEIGHT_TOKEN_APPROX, oracle.WEIGHT_TOKEN_EXACT):
        wt, st, ss = pipe.loss_weights(mode)
        torch.cuda.synchronize()
        ewt, est, ess = ref.loss_weights(mode)
        got = h(wt)
        assert np.array_equal(got.view(np.int64), ewt.view(np.int64)), \
            (mode, int(np.count_nonzero(got != ewt)), float(np.max(np.abs(got - ewt), initial=0.0)))
        assert np.array_equal(h(st), est), ("step tokens", mode)
        assert np.array_equal(h(ss), ess), ("step samples", mode)


def compare_collate_full(w, outs, ref, pad_id=0):
    want = ref.collate(w.tok_off, w.tokens_numpy(), pad_id)
    for name, g, e in zip(["input_ids", "labels", "attention_mask", "position_ids"], outs, want):
        got = h(g)
        assert got.shape == e.shape, name
        if not np.array_equal(got, e):
            bad = np.nonzero(got != e)[0]
            raise AssertionError(f"{name}: {len(bad)} mismatches, first at {bad[0]}: {got[bad[0]]} vs {e[bad[0]]}")


def compare_collate_sampled(w, outs, ref, pad_id=0, samples=200000, seed=0):
    """Spot-check collate outputs at random positions plus every tile's first and last
    element, against the oracle's per-element collate rule."""
    import torch

    P = ref.padded_elems
    rng = np.random.default_rng(seed)
    idx = rng.integers(0, P, size=samples)
    starts = ref.slot_tile_off[:-1][ref.slot_rows > 0]
    ends = ref.slot_tile_off[1:][ref.slot_rows > 0] - 1
    idx = np.unique(np.concatenate([idx, starts, ends, [0, P - 1]]))
    want = oracle.collate_elements(ref, w.tok_off, synth.token_ids, idx, pad_id)
    ti = torch.from_numpy(idx).to(outs[0].device)
    for name, g, e in zip(["input_ids", "labels", "attention_mask", "position_ids"], outs, want):
        got = g[ti].cpu().numpy()
        if not np.array_equal(got, e):
            bad = np.nonzero(got != e)[0]
            raise AssertionError(f"{name}: {len(bad)} sampled mismatches, first at {idx[bad[0]]}")


def compare_collate_by_rank(w, outs, ref, tokens_dev, pad_id=0, check_tokens=100_000, seed=0):
    """Every element of the four outputs, one rank at a time: the oracle collates rank r's
    tiles from that rank's token range and the GPU outputs' slice is copied back.  The
    token range comes from the device token stream (written by the seeded generator, not
    by the library); a sample of it is checked against the generator first."""
    rng = np.random.default_rng(seed)
    S = ref.steps
    for r in range(w.W):
        a, b = int(w.tok_off[w.rank_off[r]]), int(w.tok_off[w.rank_off[r + 1]])
        toks = tokens_dev[a:b].cpu().numpy()
        if b > a:
            k = np.unique(np.concatenate([rng.integers(a, b, size=min(check_tokens, b - a)), [a, b - 1]]))
            assert np.array_equal(toks[k - a], synth.token_ids(k).astype(np.int32)), f"token stream, rank {r}"
        want = ref.collate_rank(r, w.tok_off, toks, pad_id)
        lo, hi = int(ref.slot_tile_off[r * S]), int(ref.slot_tile_off[(r + 1) * S])
        for name, g, e in zip(["input_ids", "labels", "attention_mask", "position_ids"], outs, want):
            got = g[lo:hi].cpu().numpy()
            if not np.array_equal(got, e):
                bad = np.nonzero(got != e)[0]
                raise AssertionError(f"{name}: rank {r}: {len(bad)} mismatches, first at {lo + bad[0]}: "
                                     f"{got[bad[0]]} vs {e[bad[0]]}")
        del toks, want


def collate_properties(outs, ref, pad_id=0, chunk=1 << 30):
    """Whole-output properties that hold at any size (evaluated chunk by chunk, so the
    temporaries stay small next to outputs of 100+ GB)."""
    import torch

    ids, lab, msk, pos = outs
    P = ref.padded_elems
    assert ids.numel() == P
    real = 0
    for a in range(0, P, chunk):
        b = min(P, a + chunk)
        m = msk[a:b]
        real += int(m.sum(dtype=torch.int64))
        pad = m == 0
        assert int(pad.logical_and(lab[a:b] != -100).sum()) == 0
        assert int(pad.logical_and(ids[a:b] != pad_id).sum()) == 0
        assert int(pad.logical_and(pos[a:b] != 0).sum()) == 0
        assert int((m == 1).logical_and(ids[a:b] != lab[a:b]).sum()) == 0
        del m, pad
    assert real == ref.info["real_tokens"]
    return real


def compare_collate_by_rank_whole_stream(tok_off, outs, ref, tokens_dev, pad_id=0, check_tokens=1_000_000, seed=0):
    """Every element of the four outputs of a plan whose rows come from anywhere in the
    token stream (streaming plans: a rank's views are identities spread over the whole
    dataset).  The device token stream (written by the seeded generator) is copied back
    once and a sample of it checked against the generator; then, rank by rank, the
    oracle collates that rank's tiles from it and the GPU slice is compared."""
    rng = np.random.default_rng(seed)
    toks = tokens_dev.cpu().numpy()
    if len(toks):
        k = np.unique(np.concatenate([rng.integers(0, len(toks), size=min(check_tokens, len(toks))),
                                      [0, len(toks) - 1]]))
        assert np.array_equal(toks[k], synth.token_ids(k).astype(np.int32)), "token stream"
    S = ref.steps
    for r in range(ref.W):
        want = ref.collate_rank(r, tok_off, toks, pad_id, whole_stream=True)
        lo, hi = int(ref.slot_tile_off[r * S]), int(ref.slot_tile_off[(r + 1) * S])
        for name, g, e in zip(["input_ids", "labels", "attention_mask", "position_ids"], outs, want):
            got = g[lo:hi].cpu().numpy()
            if not np.array_equal(got, e):
                bad = np.nonzero(got != e)[0]
                raise AssertionError(f"{name}: rank {r}: {len(bad)} mismatches, first at {lo + bad[0]}: "
                                     f"{got[bad[0]]} vs {e[bad[0]]}")
        del want
        if r % 8 == 7 or r == ref.W - 1:
            log(f"  ranks 0-{r}: every collate element equal")
    del toks
