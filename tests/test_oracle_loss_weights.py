"""Pins for the oracle's loss-scaling weights (no GPU).

Eq. 2 and App. B define the token-level weight w_r = t_r / T_tok of a step: with it the
weighted mean of the ranks' per-token mean losses equals the mean over every token of
the step.  The pins below check that identity on random per-token losses, the cases in
which sample-level or approximate weights must coincide with the exact ones bit for bit,
the approximate counts against a re-derivation from the emitted plan, and the
second-gather predicate against the alignment counters.
"""
import numpy as np
import pytest

import oracle
import synth

MODES = (oracle.WEIGHT_SAMPLE, oracle.WEIGHT_TOKEN_APPROX, oracle.WEIGHT_TOKEN_EXACT)


def win(per_rank, budget, **kw):
    return synth.window_from_ranks("t", [np.asarray(x, dtype=np.int64) for x in per_rank], budget, **kw)


def random_windows():
    rng = np.random.default_rng(31)
    out = []
    for t in range(30):
        W = int(rng.integers(1, 7))
        per = [rng.integers(1, int(rng.integers(2, 2000)), size=int(rng.integers(0, 300))) for _ in range(W)]
        if sum(len(x) for x in per) == 0:
            per[0] = rng.integers(1, 100, size=5)
        n = sum(len(x) for x in per)
        mode = "nonjoin" if t % 3 == 2 else "join"
        cap = rng.integers(0, 5, size=W) if t % 4 == 1 else None
        out.append(win(per, int(rng.integers(50, 20000)), mode=mode, quota=int(rng.integers(1, n + 1)),
                       capacity=cap))
    return out


def slot_members(p, k):
    return p.emit_order[p.slot_row_off[k]:p.slot_row_off[k + 1]].astype(np.int64)


def test_exact_weights_recover_the_per_token_mean_loss():
    # Eq. 2: sum_r w_r * mean_r = (1 / T_tok) * sum of every token loss of the step
    rng = np.random.default_rng(32)
    checked = 0
    naive_differs = False
    for w in random_windows():
        p = oracle.plan_window(w)
        S, W = p.steps, w.W
        loss = rng.random(int(w.tok_off[-1])) * 10.0      # one loss per CSR token position
        wt, st, _ = p.loss_weights(oracle.WEIGHT_TOKEN_EXACT)
        for j in range(S):
            sums, toks = np.zeros(W), np.zeros(W, dtype=np.int64)
            for r in range(W):
                for s in slot_members(p, r * S + j):
                    a, b = w.tok_off[s], w.tok_off[s + 1]
                    sums[r] += loss[a:b].sum()
                    toks[r] += b - a
            assert toks.sum() == st[j]
            ref = sums.sum() / toks.sum()
            means = np.where(toks > 0, sums / np.maximum(toks, 1), 0.0)
            got = float(np.dot(wt[np.arange(W) * S + j], means))
            assert abs(got - ref) <= 1e-12 * ref
            active = toks > 0
            naive = means[active].mean()
            naive_differs |= abs(naive - ref) > 1e-9 * ref
            checked += 1
    assert checked > 500 and naive_differs


@pytest.mark.parametrize("mode", MODES)
def test_weights_sum_to_one_and_idle_slots_weigh_zero(mode):
    for w in random_windows():
        p = oracle.plan_window(w)
        S, W = p.steps, w.W
        wt, st, ss = p.loss_weights(mode)
        m = wt.reshape(W, S)
        assert np.all(m >= 0.0)
        assert np.all(np.abs(m.sum(axis=0) - 1.0) <= W * 2.0 ** -52)
        idle = p.slot_rows.reshape(W, S) == 0
        assert np.all(m[idle] == 0.0)
        assert np.array_equal(ss, p.slot_rows.reshape(W, S).sum(axis=0))
        assert np.array_equal(st, p.slot_tokens.reshape(W, S).sum(axis=0))


def test_sample_level_equals_token_level_when_all_lengths_are_equal():
    # t_r / n_r is the same on every rank, so both weights are the same rational number
    rng = np.random.default_rng(33)
    for t in range(10):
        W = int(rng.integers(2, 6))
        l = int(rng.integers(1, 900))
        per = [np.full(int(rng.integers(0, 200)), l) for _ in range(W)]
        per[0] = np.full(50, l)
        w = win(per, int(rng.integers(l, 40 * l)))
        p = oracle.plan_window(w)
        a = p.loss_weights(oracle.WEIGHT_SAMPLE)[0]
        b = p.loss_weights(oracle.WEIGHT_TOKEN_EXACT)[0]
        assert np.array_equal(a, b)


def test_approximate_equals_exact_when_each_rank_has_one_length():
    # a rank's buffer mean is then its length, so rows * mean is the exact token count
    rng = np.random.default_rng(34)
    differs = False
    for t in range(10):
        W = int(rng.integers(2, 6))
        per = [np.full(int(rng.integers(1, 200)), int(rng.integers(1, 900))) for _ in range(W)]
        w = win(per, 6000)
        p = oracle.plan_window(w)
        a = p.loss_weights(oracle.WEIGHT_TOKEN_APPROX)[0]
        b = p.loss_weights(oracle.WEIGHT_TOKEN_EXACT)[0]
        assert np.array_equal(a, b)
        assert np.array_equal(p.slot_tokens_approx, p.slot_tokens.astype(np.float64))
    for w in random_windows():
        p = oracle.plan_window(w)
        a = p.loss_weights(oracle.WEIGHT_TOKEN_APPROX)[0]
        b = p.loss_weights(oracle.WEIGHT_TOKEN_EXACT)[0]
        differs |= not np.array_equal(a, b)
    assert differs


def test_approximate_counts_from_the_emitted_plan():
    # Round k's buffer of rank r = its samples not emitted in earlier rounds.  Re-derive
    # rows * (buffer tokens / buffer samples) from the emitted slots and the round
    # targets (each round emits T_k steps, the last one possibly cut by the quota).
    for w in random_windows():
        p = oracle.plan_window(w)
        S, W = p.steps, w.W
        lens = np.diff(w.tok_off)
        begins = np.concatenate([[0], np.cumsum(p.round_targets)])
        want = np.zeros(W * S)
        for r in range(W):
            a, b = w.rank_off[r], w.rank_off[r + 1]
            n_left, t_left = b - a, int(lens[a:b].sum())
            for k in range(len(p.round_targets)):
                lo, hi = begins[k], min(begins[k + 1], S)
                mean = t_left / n_left if n_left > 0 else 0.0
                for j in range(lo, hi):
                    ids = slot_members(p, r * S + j)
                    want[r * S + j] = len(ids) * mean if len(ids) else 0.0
                    n_left -= len(ids)
                    t_left -= int(lens[ids].sum())
        assert np.array_equal(p.slot_tokens_approx, want)


def test_second_gather_predicate():
    rng = np.random.default_rng(35)
    # identical buffers on every rank: equal group counts, alignment is a no-op
    base = rng.integers(1, 3000, size=400)
    p = oracle.plan_window(win([base, base.copy(), base.copy()], 8192))
    assert p.info["rounds"] == 1 and p.info["second_gather_rounds"] == 0
    assert p.info["splits"] == 0 and p.info["overflow_groups"] == 0
    # one rank: T = G_r every round
    p = oracle.plan_window(win([rng.integers(1, 3000, size=500)], 8192))
    assert p.info["second_gather_rounds"] == 0
    # single-round windows: the predicate is "some rank was split or overflowed"
    seen = set()
    for t in range(40):
        W = int(rng.integers(2, 5))
        per = [rng.integers(1, 2000, size=int(rng.integers(50, 300))) for _ in range(W)]
        p = oracle.plan_window(win(per, int(rng.integers(2000, 30000))))
        if p.info["rounds"] != 1:
            continue
        changed = p.info["splits"] + p.info["overflow_groups"] > 0
        assert p.info["second_gather_rounds"] == int(changed)
        seen.add(changed)
    assert True in seen   # unequal buffers usually need a split
    # every round counts at most once
    for w in random_windows():
        p = oracle.plan_window(w)
        assert 0 <= p.info["second_gather_rounds"] <= p.info["rounds"]


def test_unknown_mode_rejected():
    p = oracle.plan_window(win([[5, 6, 7]], 100))
    with pytest.raises(oracle.OracleError):
        p.loss_weights(3)
