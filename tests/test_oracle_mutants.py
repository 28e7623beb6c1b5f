"""The oracle's pins reject plausible mistakes (no GPU).

Each mutant is a copy of the oracle's C++ source with one deliberate, plausible error
(a flipped tie order, a ceiling instead of a floor, a dropped trailing group, a wrong
scan direction, an off-by-one quota test, a wrong pad value, ...), compiled on the CPU.
The pins of the oracle test files then run against the mutant in a subprocess (a mutant
may loop) and at least one must fail.  The oracle in the repository is not modified.
"""
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor


ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "odb_oracle.cpp")

# (name, text in the oracle source, replacement); every occurrence is replaced
MUTANTS = [
    ("tie_order_id_desc", "return a < b;", "return a > b;"),
    ("eq1_ceiling", "int64_t b = L_max / l;", "int64_t b = (L_max + l - 1) / l;"),
    ("threshold_from_first_member", "t = batch_size(L_max, len[x]);", "t = batch_size(L_max, len[cur.front()]);"),
    ("trailing_group_dropped", "if (!cur.empty()) formed.push_back(cur);", "if (false) formed.push_back(cur);"),
    ("eq3_min_of_groups", "maxG = std::max(maxG, G);", "maxG = maxG == 0 ? G : std::min(maxG, G);"),
    ("eq3_buffer_bound_dropped", "if (minS > 0) T = std::min(T, minS);", "(void)minS;"),
    ("split_peels_from_last_formed", "    GroupList out;\n    for (Group& g : formed) {\n",
     "    GroupList out;\n    std::reverse(formed.begin(), formed.end());\n    for (Group& g : formed) {\n"),
    ("split_peels_shortest_member", "        size_t first = 0;\n",
     "        size_t first = 0;\n        std::reverse(g.begin(), g.end());\n"),
    ("overflow_keeps_smallest", "return formed[a].size() > formed[b].size();",
     "return formed[a].size() < formed[b].size();"),
    ("overflow_ties_keep_earlier_formed", "        return a > b;\n    });", "        return a < b;\n    });"),
    ("quota_strict", "emitted >= quota", "emitted > quota"),
    ("pad_fraction_inverted", "I.pad_fraction = I.padded_elems > 0 ? 1.0 - ",
     "I.pad_fraction = I.padded_elems > 0 ? 0.0 + "),
    ("label_pad_value", "labels[e] = -100;", "labels[e] = pad_id;"),
    ("position_from_one", "position_ids[e] = (int32_t)c;", "position_ids[e] = (int32_t)c + 1;"),
    ("rows_long_to_short", "return pos[a] > pos[b];", "return pos[a] < pos[b];"),
    ("groups_long_to_short", "return pos[a.front()] > pos[b.front()];", "return pos[a.front()] < pos[b.front()];"),
    ("exact_weight_by_samples", "w = (double)t[(size_t)r] / (double)T_tok;", "w = (double)c[(size_t)r] / (double)N;"),
    ("approx_mean_off_by_one", "mean_len[(size_t)r] = (double)tok / (double)b.size();",
     "mean_len[(size_t)r] = (double)tok / (double)(b.size() + 1);"),
    ("duplicates_count_first_view", "I.duplicate_ids += id_count[(size_t)d] - 1;",
     "I.duplicate_ids += id_count[(size_t)d];"),
    ("stream_never_skips", "unready += (!fin && !ready[(size_t)r]) ? 1 : 0;", "unready += 0;"),
    ("stream_padding_repeats_first", "ident[(size_t)m] = perm[m % N];", "ident[(size_t)m] = perm[m < N ? m : 0];"),
    ("stream_envelope_ignored", "int64_t room = depth - (int64_t)buf[(size_t)r].size();", "int64_t room = depth;"),
    ("stream_ready_needs_full_buffer",
     "ready[(size_t)r] = !fin && ((int64_t)buf[(size_t)r].size() >= buffer_size || drained);",
     "ready[(size_t)r] = !fin && ((int64_t)buf[(size_t)r].size() >= buffer_size || (drained && buf[(size_t)r].size() > 1));"),
]

RUNNER = r"""
import sys
sys.path[:0] = [{root!r}, {tests!r}]
import oracle
oracle._use_library({lib!r})
import test_oracle_pins as P
import test_oracle_loss_weights as LW
import test_oracle_stream as ST
pins = [
    ("worked_example", P.test_worked_example_appD, ()),
    ("equal_lengths", P.test_equal_lengths_closed_form, (3, 10)),
    ("equal_lengths_b", P.test_equal_lengths_closed_form, (64, 4096)),
    ("singletons", P.test_budget_below_every_length_gives_singletons, ()),
    ("formation_order", P.test_formation_order_is_length_desc_id_asc, ()),
    ("exhaustive_cuts", P.test_grouping_matches_exhaustive_cut_search, ()),
    ("budget_invariant", P.test_budget_invariant_on_every_slot, ()),
    ("eq3", P.test_alignment_target_eq3, ()),
    ("split_closed_form", P.test_split_matches_closed_form, ()),
    ("split_refines", P.test_split_refines_and_preserves, ()),
    ("overflow", P.test_overflow_keeps_largest_groups, ()),
    ("join_once", P.test_join_emits_every_view_once, ()),
    ("empty_rank", P.test_empty_rank_audit_shape, ()),
    ("quota", P.test_nonjoin_quota_closure, ()),
    ("finished_rank", P.test_nonjoin_finished_rank_stops, ()),
    ("collate_join", P.test_collate_matches_pad_sequence, ("join",)),
    ("collate_nonjoin", P.test_collate_matches_pad_sequence, ("nonjoin",)),
    ("stats", P.test_stats_are_exact_sums, ()),
    ("sampler_padding", P.test_identity_closure_sampler_padding, (57284, 8, 7161, 4)),
    ("sampler_padding_b", P.test_identity_closure_sampler_padding, (207865, 8, 25984, 7)),
    ("eq2", LW.test_exact_weights_recover_the_per_token_mean_loss, ()),
    ("weights_sum", LW.test_weights_sum_to_one_and_idle_slots_weigh_zero, (2,)),
    ("sample_eq_token", LW.test_sample_level_equals_token_level_when_all_lengths_are_equal, ()),
    ("approx_counts", LW.test_approximate_counts_from_the_emitted_plan, ()),
    ("predicate", LW.test_second_gather_predicate, ()),
    ("stream_window", ST.test_reduces_to_the_window_pipeline, ("join",)),
    ("stream_thm1", ST.test_join_theorem_1_and_no_leak, ()),
    ("stream_lyapunov", ST.test_lyapunov_potential_and_round_bounds, ()),
    ("stream_nonjoin", ST.test_nonjoin_envelope_and_quota_closure, ()),
    ("stream_skips", ST.test_skip_rounds_by_hand, ()),
    ("stream_padding", ST.test_sampler_padding_reuses_the_head_of_the_list, ()),
]
for name, fn, args in pins:
    try:
        fn(*args)
    except Exception as e:
        print("CAUGHT", name, type(e).__name__, flush=True)
        sys.exit(0)
print("SURVIVED", flush=True)
sys.exit(1)
"""


def _build(name, old, new, out_dir):
    src = open(SRC).read()
    assert src.count(old) >= 1, f"mutation {name}: target text not in the oracle source"
    path = os.path.join(out_dir, f"mut_{name}.cpp")
    lib = os.path.join(out_dir, f"libmut_{name}.so")
    open(path, "w").write(src.replace(old, new))
    subprocess.check_call(["g++", "-O1", "-std=c++17", "-ffp-contract=off", "-shared", "-fPIC", "-w", path, "-o", lib])
    return lib


def _run(lib):
    code = RUNNER.format(root=ROOT, tests=os.path.join(ROOT, "tests"), lib=lib)
    try:
        r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=90)
    except subprocess.TimeoutExpired:
        return "CAUGHT timeout (the mutant does not terminate)"
    last = (r.stdout.strip().splitlines() or [""])[-1]
    if r.returncode != 0 and not last.startswith("SURVIVED"):
        return f"CAUGHT crash (exit {r.returncode})"   # e.g. an out-of-range access in the mutant
    return last


def test_every_mutant_is_caught(tmp_path):
    with ThreadPoolExecutor(max_workers=8) as ex:
        libs = list(ex.map(lambda m: _build(*m, str(tmp_path)), MUTANTS))
    with ThreadPoolExecutor(max_workers=6) as ex:
        results = list(ex.map(_run, libs))
    survived = [(m[0], r) for m, r in zip(MUTANTS, results) if not r.startswith("CAUGHT")]
    assert not survived, f"mutants not caught by any pin: {survived}"
