"""Pins for the CPU oracle (no GPU).

Each test ties the oracle to something other than itself: values the paper prints for
its worked example, closed forms that follow from Eq. 1 / Eq. 3, brute-force search
over all cuts on tiny inputs, a second (closed-form) statement of the split rule, the
theorems' invariants, torch's own ``pad_sequence`` for the collate, and the sampler
arithmetic of the identity-coverage audit.
"""
import itertools
import math
import os

import numpy as np
import pytest
import torch

import oracle
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def win(per_rank, budget, **kw):
    return synth.window_from_ranks("t", [np.asarray(x, dtype=np.int64) for x in per_rank], budget, **kw)


def rank_slots(p, r):
    """Rank r's aligned steps as lists of sample ids (rows in order)."""
    S = p.steps
    out = []
    for j in range(S):
        k = r * S + j
        out.append([int(x) for x in p.emit_order[p.slot_row_off[k]:p.slot_row_off[k + 1]]])
    return out


def formation_groups(p, w, r):
    """Rank r's first-formation groups as lists of formation positions (rank-local)."""
    a, b = w.rank_off[r], w.rank_off[r + 1]
    gi = p.group_index[a:b]
    groups = []
    for pos, g in enumerate(gi):
        if g == len(groups):
            groups.append([])
        groups[g].append(pos)
    return groups


def B(L, l):  # Eq. 1, restated for test arithmetic
    return max(L // l, 1)


# ----------------------------------------------------------------------------- App. D
def _read_worked_example():
    budget, lengths, groups = None, None, []
    with open(os.path.join(GOLDEN, "appD_worked_example.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, rest = line.split(None, 1)
            if key == "budget":
                budget = int(rest)
            elif key == "lengths":
                lengths = [int(x) for x in rest.split()]
            elif key == "group":
                members, padded_to, padded = [x.strip() for x in rest.split("|")]
                groups.append(([int(x) for x in members.split()], int(padded_to), int(padded)))
    return budget, lengths, groups


def test_worked_example_appD():
    budget, lengths, groups = _read_worked_example()
    w = win([lengths], budget)
    p = oracle.plan_window(w)
    slots = rank_slots(p, 0)
    got = [[int(w.lengths[x]) for x in g] for g in slots]
    assert got == [g[0] for g in groups]
    assert list(p.slot_maxlen) == [g[1] for g in groups]
    assert list(p.slot_rows.astype(np.int64) * p.slot_maxlen) == [g[2] for g in groups]
    real = sum(lengths)
    padded = sum(g[2] for g in groups)
    assert p.info["real_tokens"] == real and p.info["padded_elems"] == padded
    # pad% = 1 - sum(L_real) / sum(L_compute), in fp64
    assert p.info["pad_fraction"] == 1.0 - real / padded
    assert abs(p.info["pad_fraction"] - 1.0 / 17.0) <= 1e-12 * (1.0 / 17.0)


# ----------------------------------------------------------------------------- Eq. 1
@pytest.mark.parametrize("l,L", [(1, 1), (3, 10), (5, 10), (7, 100), (100, 99), (64, 4096), (33, 1000)])
def test_equal_lengths_closed_form(l, L):
    # all lengths equal: the first group is a singleton, then every group has b = B(l)
    # samples except a shorter trailing one  =>  G = 1 + ceil((n - 1) / b)
    b = B(L, l)
    ns = list(range(1, 41))
    w = win([[l] * n for n in ns], L)
    p = oracle.plan_window(w)
    for r, n in enumerate(ns):
        assert p.groups_per_rank[r] == 1 + math.ceil((n - 1) / b)
        sizes = [len(g) for g in formation_groups(p, w, r)]
        assert sizes[0] == 1 and all(s == b for s in sizes[1:-1]) and 1 <= sizes[-1] <= b


def test_budget_below_every_length_gives_singletons():
    rng = np.random.default_rng(1)
    per = [rng.integers(50, 500, size=k) for k in (1, 5, 17, 64)]
    w = win(per, 49)
    p = oracle.plan_window(w)
    assert list(p.groups_per_rank) == [1, 5, 17, 64]
    assert np.all(p.slot_rows[p.slot_rows > 0] == 1)


# ----------------------------------------------------------------------------- sort key
def test_formation_order_is_length_desc_id_asc():
    rng = np.random.default_rng(2)
    per = [rng.integers(1, 6, size=k) for k in (0, 1, 7, 100, 333)]  # heavy ties
    w = win(per, 8)
    p = oracle.plan_window(w)
    for r in range(w.W):
        a, b = w.rank_off[r], w.rank_off[r + 1]
        ids = np.arange(a, b)
        expect = ids[np.lexsort((ids, -w.lengths[a:b]))]
        assert np.array_equal(p.order[a:b], expect)
        assert np.array_equal(p.sorted_len[a:b], w.lengths[expect])


# ----------------------------------------------------------------------------- brute force
def _valid_cuts(sorted_lens, L):
    """All cuts of the visiting sequence satisfying the declarative grouping rule."""
    n = len(sorted_lens)
    sols = []
    for mask in range(1 << (n - 1)):
        bounds = [0] + [i + 1 for i in range(n - 1) if mask >> i & 1] + [n]
        sizes = [bounds[i + 1] - bounds[i] for i in range(len(bounds) - 1)]
        ok = sizes[0] == 1
        for g in range(1, len(sizes)):
            want = B(L, sorted_lens[bounds[g] - 1])  # B of the previous group's last sample
            if g < len(sizes) - 1:
                ok &= sizes[g] == want
            else:
                ok &= 1 <= sizes[g] <= want
        if ok:
            sols.append(sizes)
    return sols


def test_grouping_matches_exhaustive_cut_search():
    alphabet = [1, 2, 3, 5]
    budgets = [1, 2, 4, 7, 10]
    vectors = [v for n in range(1, 7) for v in itertools.product(alphabet, repeat=n)]
    for L in budgets:
        w = win([list(v) for v in vectors], L)
        p = oracle.plan_window(w)
        for r, v in enumerate(vectors):
            a = w.rank_off[r]
            sl = [int(x) for x in p.sorted_len[a:a + len(v)]]
            assert sl == sorted(v, reverse=True)
            sols = _valid_cuts(sl, L)
            assert len(sols) == 1
            sizes = [len(g) for g in formation_groups(p, w, r)]
            assert sizes == sols[0], (v, L)


def test_budget_invariant_on_every_slot():
    rng = np.random.default_rng(3)
    for L in (10, 100, 1000, 4096):
        per = [rng.integers(1, 3000, size=k) for k in (0, 1, 2, 50, 400)]
        for cap in (None, [3, 1, 2, 5, 4]):
            w = win(per, L, capacity=None if cap is None else np.array(cap))
            p = oracle.plan_window(w)
            rows = p.slot_rows.astype(np.int64)
            ok = (rows <= 1) | (rows * p.slot_maxlen <= L)
            assert ok.all()


# ----------------------------------------------------------------------------- Eq. 3
def _target(G, S, C):
    act = [r for r in range(len(G)) if G[r] > 0]
    if not act:
        return None
    t = max(G[r] for r in act)
    cs = [C[r] for r in act if C is not None and C[r] > 0]
    ss = [S[r] for r in act if S[r] > 0]
    if cs:
        t = min(t, min(cs))
    if ss:
        t = min(t, min(ss))
    return max(t, 1)


def test_alignment_target_eq3():
    L = 10
    # rank 0: ten samples of length 5 -> groups 1,2,2,2,2,1 (G=6); rank 1: 3 samples (G=2);
    # rank 2 empty and therefore not active.
    w = win([[5] * 10, [5] * 3, []], L)
    p = oracle.plan_window(w)
    assert list(p.groups_per_rank) == [6, 2, 0]
    assert p.round_targets[0] == _target([6, 2, 0], [10, 3, 0], None) == 3
    # capacity: only positive capacities of active ranks count (rank 2's 1 is ignored)
    w = win([[5] * 10, [5] * 9, []], L, capacity=np.array([4, 0, 1]))
    p = oracle.plan_window(w)
    G = [int(x) for x in p.groups_per_rank]
    assert p.round_targets[0] == _target(G, [10, 9, 0], [4, 0, 1]) == 4
    # unlimited capacity, equal buffers: the target is the largest group count
    rng = np.random.default_rng(4)
    for _ in range(20):
        per = [rng.integers(1, 200, size=64) for _ in range(5)]
        w = win(per, 512)
        p = oracle.plan_window(w)
        G = [int(x) for x in p.groups_per_rank]
        assert p.round_targets[0] == max(G)
        assert p.info["rounds"] == 1 and p.info["overflow_groups"] == 0
        assert p.info["splits"] == sum(max(G) - g for g in G)


# ----------------------------------------------------------------------------- split
def _split_closed_form(sizes, k):
    """Formation-order groups after k extractions, as (start, end) ranges.

    Peeling the longest member of the first non-singleton group in formation order,
    k times, leaves positions [0, X) as singletons and [X, end of group j*) as one group,
    where j* is the first group at which the cumulative surplus sum(c_g - 1) reaches k.
    """
    starts = np.concatenate([[0], np.cumsum(sizes)[:-1]])
    surplus = np.cumsum(np.asarray(sizes) - 1)
    j = int(np.searchsorted(surplus, k))          # first j with surplus[j] >= k
    before = int(surplus[j - 1]) if j > 0 else 0
    X = int(starts[j]) + (k - before)
    out = [(i, i + 1) for i in range(X)]
    out.append((X, int(starts[j] + sizes[j])))
    out += [(int(starts[g]), int(starts[g] + sizes[g])) for g in range(j + 1, len(sizes))]
    return out


def test_split_matches_closed_form():
    rng = np.random.default_rng(5)
    for trial in range(300):
        L = int(rng.integers(20, 400))
        big = rng.integers(1, 60, size=int(rng.integers(40, 120)))
        small = rng.integers(1, 60, size=int(rng.integers(8, 40)))
        w = win([big, small], L)
        p = oracle.plan_window(w)
        T = int(p.round_targets[0])
        G1 = int(p.groups_per_rank[1])
        if p.info["rounds"] != 1 or G1 >= T:
            continue
        groups = formation_groups(p, w, 1)
        sizes = [len(g) for g in groups]
        expect = _split_closed_form(sizes, T - G1)
        a = w.rank_off[1]
        posmap = {int(x): i for i, x in enumerate(p.order[a:w.rank_off[2]])}
        got = []
        for g in rank_slots(p, 1):
            ps = [posmap[x] for x in g]
            assert ps == sorted(ps, reverse=True)          # rows run short to long
            got.append((min(ps), max(ps) + 1))
        assert got == expect[::-1]                         # emitted short to long
        assert len(got) == T


def test_split_refines_and_preserves():
    rng = np.random.default_rng(6)
    for _ in range(100):
        per = [rng.integers(1, 100, size=int(rng.integers(1, 80))) for _ in range(4)]
        w = win(per, int(rng.integers(50, 500)))
        p = oracle.plan_window(w)
        if p.info["rounds"] != 1:
            continue
        for r in range(w.W):
            a = w.rank_off[r]
            form = p.group_index[a:w.rank_off[r + 1]]
            where = {int(x): int(form[i]) for i, x in enumerate(p.order[a:w.rank_off[r + 1]])}
            slots = [g for g in rank_slots(p, r) if g]
            assert len(slots) == p.round_targets[0]
            for g in slots:
                assert len({where[x] for x in g}) == 1       # each new group inside one old group
            assert sorted(x for g in slots for x in g) == list(range(a, w.rank_off[r + 1]))


# ----------------------------------------------------------------------------- overflow
def test_overflow_keeps_largest_groups():
    rng = np.random.default_rng(7)
    checked = 0
    for _ in range(200):
        per = [rng.integers(1, 120, size=int(rng.integers(20, 200))) for _ in range(3)]
        cap = rng.integers(1, 6, size=3)
        w = win(per, int(rng.integers(100, 1000)), capacity=cap)
        p = oracle.plan_window(w)
        T = int(p.round_targets[0])
        for r in range(w.W):
            G = int(p.groups_per_rank[r])
            if G <= T:
                continue
            checked += 1
            groups = formation_groups(p, w, r)
            a = w.rank_off[r]
            ids = [[int(p.order[a + i]) for i in g] for g in groups]
            kept = [sorted(g) for g in rank_slots(p, r)[:T]]
            # stable sort of the short-to-long list by size, descending
            short_to_long = list(range(G))[::-1]
            ranked = sorted(short_to_long, key=lambda g: -len(groups[g]))
            expect = sorted(sorted(ids[g]) for g in ranked[:T])
            assert sorted(kept) == expect
            kmin = min(len(g) for g in kept)
            assert all(len(groups[g]) <= kmin for g in ranked[T:])
        # join: everything still emitted exactly once over the extra rounds
        assert p.info["bad_views"] == 0 and p.info["emitted_samples"] == w.n
    assert checked > 50


# ----------------------------------------------------------------------------- Theorem 1
def _check_join(p, w):
    assert p.info["stop_reason"] == oracle.STOP_DRAINED
    assert p.info["emitted_samples"] == w.n and p.info["leftover_samples"] == 0
    assert p.info["bad_views"] == 0
    assert sorted(p.emit_order.tolist()) == list(range(w.n))
    S = p.steps
    assert S == int(p.round_targets.sum())
    # IDLE slots: a rank's real steps form a prefix; once idle it stays idle (its buffer
    # is empty and nothing arrives within a window)
    for r in range(w.W):
        rows = p.slot_rows[r * S:(r + 1) * S]
        real = rows > 0
        k = int(real.sum())
        assert real[:k].all() and not real[k:].any()
        assert int(rows.sum()) == w.rank_off[r + 1] - w.rank_off[r]


def test_join_emits_every_view_once():
    rng = np.random.default_rng(8)
    for t in range(60):
        W = int(rng.integers(1, 7))
        per = [rng.integers(1, 300, size=int(rng.integers(0, 150))) for _ in range(W)]
        cap = rng.integers(0, 8, size=W) if t % 3 == 0 else None
        w = win(per, int(rng.integers(1, 2000)), capacity=cap)
        _check_join(oracle.plan_window(w), w)


def test_empty_rank_audit_shape():
    # two-node empty-rank audit (App. F table): 16 ranks assigned 47 - r views for
    # r < 15 and rank 15 empty; join mode must give rank 15 only IDLE slots.
    rng = np.random.default_rng(9)
    per = [rng.integers(100, 3000, size=47 - r) for r in range(15)] + [np.zeros(0, np.int64)]
    w = win(per, 8192)
    p = oracle.plan_window(w)
    _check_join(p, w)
    S = p.steps
    assert (p.slot_rows[15 * S:] == 0).all()
    assert w.n == sum(47 - r for r in range(15))


# ----------------------------------------------------------------------------- Theorem 2
def test_nonjoin_quota_closure():
    rng = np.random.default_rng(10)
    for t in range(80):
        W = int(rng.integers(1, 6))
        per = [rng.integers(1, 400, size=int(rng.integers(1, 120))) for _ in range(W)]
        n = sum(len(x) for x in per)
        Q = int([1, rng.integers(1, n + 1), max(n - 1, 1), n, n + 1][t % 5])
        cap = rng.integers(1, 5, size=W) if t % 4 == 0 else None
        w = win(per, int(rng.integers(50, 3000)), mode="nonjoin", quota=Q, capacity=cap)
        p = oracle.plan_window(w)
        I = p.info
        # No-Leak: emitted and leftover partition the window
        both = np.concatenate([p.emit_order, p.leftover])
        assert sorted(both.tolist()) == list(range(n)) and I["bad_views"] == 0
        S = p.steps
        steps = [int(p.slot_rows[[r * S + j for r in range(W)]].sum()) for j in range(S)]
        assert sum(steps) == I["emitted_samples"]
        if I["stop_reason"] == oracle.STOP_QUOTA:
            assert Q <= I["emitted_samples"] <= Q + I["max_step_samples"]
            assert sum(steps[:-1]) < Q           # the cut is the first step reaching Q
        elif I["stop_reason"] == oracle.STOP_DRAINED:
            assert I["emitted_samples"] == n < Q
        else:
            assert I["stop_reason"] == oracle.STOP_RANK_FINISHED
        # leftovers of every rank are in visiting order
        for r in range(W):
            lo = p.leftover[p.leftover_off[r]:p.leftover_off[r + 1]]
            assert np.array_equal(lo, lo[np.lexsort((lo, -w.lengths[lo]))])


def test_nonjoin_finished_rank_stops():
    w = win([[10, 20], [], [30]], 100, mode="nonjoin", quota=3)
    p = oracle.plan_window(w)
    assert p.info["stop_reason"] == oracle.STOP_RANK_FINISHED
    assert p.steps == 0 and p.info["leftover_samples"] == 3


# ----------------------------------------------------------------------------- coverage
def _read_sampler_padding():
    rows = []
    with open(os.path.join(GOLDEN, "sampler_padding.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                rows.append(tuple(int(x) for x in line.split()))
    return rows


@pytest.mark.parametrize("N,W,q,P", _read_sampler_padding())
def test_identity_closure_sampler_padding(N, W, q, P):
    views, q2, P2 = synth.sampler_views(N, W, seed=11)
    assert (q2, P2) == (q, P)
    rng = np.random.default_rng(12)
    lens_by_id = rng.integers(16, 4096, size=N)
    w = win([lens_by_id[v] for v in views], 16384, identity=np.concatenate(views), num_identities=N)
    p = oracle.plan_window(w)
    assert p.info["bad_views"] == 0
    assert p.info["missing_ids"] == 0              # eta_identity = 0
    assert p.info["duplicate_ids"] == P            # surplus = sampler padding
    S = p.steps
    per_rank = [int(p.slot_rows[r * S:(r + 1) * S].sum()) for r in range(W)]
    assert per_rank == [q] * W                     # every rank emits q views


@pytest.mark.parametrize("kind", synth.AUDIT_KINDS)
def test_audit_distributions(kind):
    for W in (3, 8):
        w = synth.audit_window(kind, W, budget=4096)
        p = oracle.plan_window(w)
        _, q, P = synth.sampler_views(1000, W, seed=1)
        assert p.info["missing_ids"] == 0 and p.info["duplicate_ids"] == P
        wq = synth.audit_window(kind, W, budget=4096, mode="nonjoin", quota=1000)
        pq = oracle.plan_window(wq)
        emitted = pq.info["emitted_samples"]
        assert max(0.0, 1.0 - emitted / 1000) == 0.0   # eta_quota = 0
        assert emitted <= 1000 + pq.info["max_step_samples"]


# ----------------------------------------------------------------------------- collate
def _pad_sequence_tiles(p, w, tokens, pad_id):
    from torch.nn.utils.rnn import pad_sequence
    outs = [[], [], [], []]
    for k in range(p.num_slots):
        rows = p.emit_order[p.slot_row_off[k]:p.slot_row_off[k + 1]]
        if len(rows) == 0:
            continue
        seqs = [torch.from_numpy(tokens[w.tok_off[s]:w.tok_off[s + 1]].astype(np.int64)) for s in rows]
        ones = [torch.ones(len(x), dtype=torch.int64) for x in seqs]
        ar = [torch.arange(len(x), dtype=torch.int64) for x in seqs]
        outs[0].append(pad_sequence(seqs, batch_first=True, padding_value=pad_id).reshape(-1))
        outs[1].append(pad_sequence(seqs, batch_first=True, padding_value=-100).reshape(-1))
        outs[2].append(pad_sequence(ones, batch_first=True, padding_value=0).reshape(-1))
        outs[3].append(pad_sequence(ar, batch_first=True, padding_value=0).reshape(-1))
    return [torch.cat(o).numpy().astype(np.int32) if o else np.zeros(0, np.int32) for o in outs]


@pytest.mark.parametrize("mode", ["join", "nonjoin"])
def test_collate_matches_pad_sequence(mode):
    rng = np.random.default_rng(13)
    for t in range(12):
        W = int(rng.integers(1, 5))
        per = [rng.integers(1, 90, size=int(rng.integers(0, 40))) for _ in range(W)]
        n = sum(len(x) for x in per)
        w = win(per, int(rng.integers(20, 400)), mode=mode, quota=max(1, n // 2))
        p = oracle.plan_window(w)
        tokens = w.tokens_numpy()
        pad_id = int(rng.integers(0, 1000))
        got = p.collate(w.tok_off, tokens, pad_id)
        want = _pad_sequence_tiles(p, w, tokens, pad_id)
        for g, e in zip(got, want):
            assert np.array_equal(g, e)
        assert len(got[0]) == p.slot_tile_off[-1] == p.info["padded_elems"]


def test_collate_elements_agrees_with_full_collate():
    rng = np.random.default_rng(14)
    w = win([rng.integers(1, 300, size=200) for _ in range(3)], 1500)
    p = oracle.plan_window(w)
    tokens = w.tokens_numpy()
    full = p.collate(w.tok_off, tokens, 7)
    idx = rng.integers(0, p.padded_elems, size=5000)
    part = oracle.collate_elements(p, w.tok_off, synth.token_ids, idx, 7)
    for f, s in zip(full, part):
        assert np.array_equal(f[idx], s)



@pytest.mark.parametrize("mode", ["join", "nonjoin"])
def test_collate_rank_is_the_rank_slice_of_full_collate(mode):
    # per-rank collate (used to compare full-size windows rank by rank) reads only that
    # rank's token range and reproduces exactly its slice of the whole-window collate
    rng = np.random.default_rng(16)
    per = [rng.integers(1, 300, size=int(k)) for k in (150, 0, 90, 1, 200)]
    n = sum(len(x) for x in per)
    w = win(per, 1200, mode=mode, quota=n // 3)
    p = oracle.plan_window(w)
    tokens = w.tokens_numpy()
    full = p.collate(w.tok_off, tokens, 9)
    S = p.steps
    for r in range(w.W):
        a, b = w.tok_off[w.rank_off[r]], w.tok_off[w.rank_off[r + 1]]
        part = p.collate_rank(r, w.tok_off, tokens[a:b].copy(), 9)
        lo, hi = p.slot_tile_off[r * S], p.slot_tile_off[(r + 1) * S]
        for f, g in zip(full, part):
            assert np.array_equal(f[lo:hi], g)
    with pytest.raises(oracle.OracleError):
        p.collate_rank(w.W, w.tok_off, tokens, 9)


# ----------------------------------------------------------------------------- stats
def test_stats_are_exact_sums():
    rng = np.random.default_rng(15)
    w = win([rng.integers(1, 5000, size=300) for _ in range(4)], 20000)
    p = oracle.plan_window(w)
    assert p.info["real_tokens"] == int(w.lengths.sum()) == int(p.slot_tokens.sum())
    assert p.info["padded_elems"] == int((p.slot_rows.astype(np.int64) * p.slot_maxlen).sum())
    assert p.info["pad_fraction"] == 1.0 - p.info["real_tokens"] / p.info["padded_elems"]


# ----------------------------------------------------------------------------- invalid
def test_invalid_inputs_rejected():
    w = win([[3, 0, 2]], 10)
    with pytest.raises(oracle.OracleError):
        oracle.plan_window(w)
    with pytest.raises(oracle.OracleError):
        oracle.plan(np.array([0, 2, 1, 3]), np.array([0, 1, 2, 3]), 10)
    with pytest.raises(oracle.OracleError):
        oracle.plan(np.array([0, 3]), np.array([0, 1, 2, 3]), 10, mode=oracle.MODE_NONJOIN, quota=0)
