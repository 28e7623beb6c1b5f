// Reference oracle for the Online Dynamic Batching window pipeline.
//
// TEST INFRASTRUCTURE ONLY.  This file is a plain, slow, single-threaded CPU
// statement of what the batching method computes on one window of realised samples.
// Only the test suite, the smoke check and the benchmark's CPU-baseline leg load it;
// the HIP library never includes, links or calls anything here, and this file uses
// nothing from the HIP library.
//
// Every step follows the paper's own description, with plain containers:
//   * batch size rule                           Eq. 1, Sec. 2.2
//   * sort + threshold-carry grouping           Sec. 2.2 and the worked example (App. D)
//   * alignment target over active ranks        Eq. 3 (App. A)
//   * split / overflow adjustment               App. A, Algorithm 1
//   * join (drain-then-signal) termination      Sec. 2.3, Theorem 1
//   * non-join sample-quota termination         Sec. 2.3, Theorem 2, App. C (quota closure)
//   * IDLE slots for ranks with nothing to send Sec. 2.1 and Algorithm 1's postcondition
//   * collate = pad every group to its own max  Sec. 2.1 / Fig. 1 ("pad to l_max")
//   * padding fraction                          throughput-decomposition definition (App. I)
//   * identity coverage                         App. C (terminal identity coverage)
//   * loss-scaling weights (sample, approximate  Eq. 2 (Sec. 2.3 "Loss scaling"), App. B,
//     and exact token level), second-gather      and the loss-scaling ablation (App. N)
//     predicate
// Where the paper is silent the oracle takes the readings documented in the
// repository's design notes (tie order, list order, trailing group, canonical
// emission order, pad values); each is marked "reading" below.
//
// Build: g++ -O2 -std=c++17 -ffp-contract=off -shared -fPIC odb_oracle.cpp -o libodb_oracle.so

#include <algorithm>
#include <cstddef>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <limits>
#include <new>
#include <string>
#include <vector>

namespace {

enum { MODE_JOIN = 0, MODE_NONJOIN = 1 };
enum { STOP_DRAINED = 0, STOP_QUOTA = 1, STOP_RANK_FINISHED = 2 };

using Group = std::vector<int32_t>;   // sample ids
using GroupList = std::vector<Group>;

struct Info {
    int64_t steps;
    int32_t rounds;
    int32_t stop_reason;
    int64_t emitted_samples;
    int64_t leftover_samples;
    int64_t real_tokens;
    int64_t padded_elems;
    int64_t max_step_samples;
    int64_t splits;
    int64_t overflow_groups;
    int64_t missing_ids;
    int64_t duplicate_ids;
    int64_t bad_views;
    double pad_fraction;
    int64_t second_gather_rounds;   // rounds whose alignment changed some active rank's groups
};

struct Result {
    int32_t W = 0;
    int64_t n = 0;
    std::vector<int64_t> rank_off;
    std::vector<int64_t> len;                 // realised length of every sample
    // first formation of every rank's full buffer (Sec. 2.2)
    std::vector<int32_t> order, sorted_len, group_index, groups_per_rank;
    // aligned plan: slots[r][j] = members of rank r's j-th step in row order (empty = IDLE)
    std::vector<std::vector<Group>> slots;
    // slots_approx[r][j]: approximate post-alignment token count of slot (r, j) for the
    // approximate token-level loss weights (App. B): rows * mean length of the rank's
    // buffer before that round's alignment; 0 for IDLE slots
    std::vector<std::vector<double>> slots_approx;
    std::vector<std::vector<int32_t>> leftover;
    std::vector<int64_t> round_target;       // T of every alignment round (Eq. 3)
    Info info{};
};

// Eq. 1: B(l) = max(floor(L_max / l), 1).
int64_t batch_size(int64_t L_max, int64_t l) {
    int64_t b = L_max / l;
    return b > 1 ? b : 1;
}

// Sec. 2.2: sort the buffer by realised length and walk it from the longest to the
// shortest sample with a running group-size threshold t (initially 1).  Each sample is
// appended to the current group; when the group's size reaches t it is finalised and
// t becomes B(l) of the sample just added (the shortest so far).
//   reading (tie order): equal lengths are visited in ascending sample id, i.e. the
//     visiting order is (length descending, id ascending).
//   reading (trailing group): samples left in an unfinished group when the buffer is
//     exhausted form one last group, so nothing in the window is dropped.
// Returns groups in formation order (longest first), members in visiting order; the
// visiting order itself is written to *visit.
GroupList form_groups(const std::vector<int32_t>& buffer, const std::vector<int64_t>& len,
                      int64_t L_max, std::vector<int32_t>* visit) {
    std::vector<int32_t> s(buffer);
    std::stable_sort(s.begin(), s.end(), [&](int32_t a, int32_t b) {
        if (len[a] != len[b]) return len[a] > len[b];
        return a < b;
    });
    GroupList formed;
    Group cur;
    int64_t t = 1;
    for (int32_t x : s) {
        cur.push_back(x);
        if ((int64_t)cur.size() >= t) {
            formed.push_back(cur);
            t = batch_size(L_max, len[x]);
            cur.clear();
        }
    }
    if (!cur.empty()) formed.push_back(cur);
    if (visit) *visit = s;
    return formed;
}

// Algorithm 1, split branch (reading R4).  A rank with fewer than T groups makes up the
// difference with singletons peeled off multi-sample groups.  Read against the App. D
// list (short groups first, members ascending), the group it peels from is the one
// holding the longest samples among those with two or more members, and the sample it
// peels is that group's longest.  Over the formation-order list (longest group first,
// members longest first) this means: the first group in formation order that still has
// two or more members gives up its first member, one peel at a time, until the rank has
// T groups or every group is a singleton.  A group that is down to one member is passed
// and the next one gives.  The peeled singleton goes in front of its donor (where in the
// list is immaterial: the emission order is canonical).  Returns the number of peels.
int64_t split_to(GroupList& formed, int64_t T) {
    int64_t need = T - (int64_t)formed.size();
    int64_t peels = 0;
    GroupList out;
    for (Group& g : formed) {
        size_t first = 0;
        while (need > 0 && g.size() - first >= 2) {
            out.push_back(Group{g[first]});
            ++first;
            --need;
            ++peels;
        }
        out.push_back(Group(g.begin() + (std::ptrdiff_t)first, g.end()));
    }
    formed.swap(out);
    return peels;
}

// Algorithm 1, overflow branch (reading R6).  A rank with more than T groups keeps the T
// largest and sends the samples of the others back to its buffer.  Equal sizes are
// decided in favour of the group formed later (shorter samples): the App. D list puts
// later-formed groups first and the paper's sort by size keeps their relative order.
// Works on the formation-order list; the kept groups stay in formation order.
void overflow_to(GroupList& formed, int64_t T, std::vector<int32_t>& returned) {
    std::vector<size_t> rank_of_group(formed.size());
    for (size_t g = 0; g < formed.size(); ++g) rank_of_group[g] = g;
    std::sort(rank_of_group.begin(), rank_of_group.end(), [&](size_t a, size_t b) {
        if (formed[a].size() != formed[b].size()) return formed[a].size() > formed[b].size();
        return a > b;
    });
    std::vector<char> keep(formed.size(), 0);
    for (size_t i = 0; i < (size_t)T && i < rank_of_group.size(); ++i) keep[rank_of_group[i]] = 1;
    GroupList kept;
    for (size_t g = 0; g < formed.size(); ++g) {
        if (keep[g]) {
            kept.push_back(formed[g]);
        } else {
            for (int32_t x : formed[g]) returned.push_back(x);
        }
    }
    formed.swap(kept);
}

// reading (emission order): a rank's aligned groups are emitted short to long and each
// group's rows run short to long; concretely groups are ordered by their members'
// positions in this round's visiting order, latest first, and so are the rows.
void canonicalize(GroupList& list, const std::vector<int64_t>& pos) {
    for (Group& g : list)
        std::sort(g.begin(), g.end(), [&](int32_t a, int32_t b) { return pos[a] > pos[b]; });
    std::sort(list.begin(), list.end(),
              [&](const Group& a, const Group& b) { return pos[a.front()] > pos[b.front()]; });
}

std::string g_err;

bool fail(const std::string& m) {
    g_err = m;
    return false;
}

bool run(Result& R, int32_t W, int64_t n, const int64_t* rank_off, const int64_t* tok_off,
         const int64_t* identity, int64_t num_identities, int64_t L_max, int32_t mode,
         int64_t quota, const int64_t* capacity) {
    if (W < 1) return fail("W must be >= 1");
    if (n < 0 || n >= (int64_t)std::numeric_limits<int32_t>::max()) return fail("n out of range");
    if (L_max < 1) return fail("budget must be >= 1");
    if (mode != MODE_JOIN && mode != MODE_NONJOIN) return fail("bad mode");
    if (mode == MODE_NONJOIN && quota < 1) return fail("quota must be >= 1 in non-join mode");
    if (rank_off[0] != 0 || rank_off[W] != n) return fail("rank offsets must span [0, n)");
    for (int32_t r = 0; r < W; ++r)
        if (rank_off[r + 1] < rank_off[r]) return fail("rank offsets must be non-decreasing");
    if (capacity)
        for (int32_t r = 0; r < W; ++r)
            if (capacity[r] < 0) return fail("capacity must be >= 0");
    R.W = W;
    R.n = n;
    R.rank_off.assign(rank_off, rank_off + W + 1);
    R.len.resize((size_t)n);
    for (int64_t i = 0; i < n; ++i) {
        int64_t l = tok_off[i + 1] - tok_off[i];   // realised post-pipeline length
        if (l < 1 || l > (int64_t)std::numeric_limits<int32_t>::max())
            return fail("sample " + std::to_string(i) + " has invalid length " + std::to_string(l));
        R.len[(size_t)i] = l;
    }
    if (identity) {
        if (num_identities < 1) return fail("num_identities must be >= 1 with an identity map");
        for (int64_t i = 0; i < n; ++i)
            if (identity[i] < 0 || identity[i] >= num_identities) return fail("identity out of range");
    }

    // ---- first formation of every rank's whole buffer (Sec. 2.2) ----
    R.order.resize((size_t)n);
    R.sorted_len.resize((size_t)n);
    R.group_index.resize((size_t)n);
    R.groups_per_rank.assign((size_t)W, 0);
    for (int32_t r = 0; r < W; ++r) {
        std::vector<int32_t> buf;
        for (int64_t i = rank_off[r]; i < rank_off[r + 1]; ++i) buf.push_back((int32_t)i);
        std::vector<int32_t> visit;
        GroupList formed = form_groups(buf, R.len, L_max, &visit);
        int64_t p = rank_off[r];
        for (size_t g = 0; g < formed.size(); ++g)
            for (int32_t x : formed[g]) {
                R.order[(size_t)p] = x;
                R.sorted_len[(size_t)p] = (int32_t)R.len[(size_t)x];
                R.group_index[(size_t)p] = (int32_t)g;
                ++p;
            }
        R.groups_per_rank[(size_t)r] = (int32_t)formed.size();
    }

    // ---- alignment rounds ----
    std::vector<std::vector<int32_t>> buf((size_t)W);
    for (int32_t r = 0; r < W; ++r)
        for (int64_t i = rank_off[r]; i < rank_off[r + 1]; ++i) buf[(size_t)r].push_back((int32_t)i);
    R.slots.assign((size_t)W, {});
    R.slots_approx.assign((size_t)W, {});
    std::vector<int64_t> pos((size_t)n, -1);
    Info& I = R.info;
    int64_t S = 0, emitted = 0;
    int32_t stop = STOP_DRAINED;
    for (;;) {
        int32_t nonempty = 0;
        for (int32_t r = 0; r < W; ++r) nonempty += buf[(size_t)r].empty() ? 0 : 1;
        if (nonempty == 0) { stop = STOP_DRAINED; break; }
        // Non-join: a rank with nothing left while others still hold samples advertises
        // "finished" (n_groups = -1) and the logical iteration ends (Sec. 2.3).
        if (mode == MODE_NONJOIN && nonempty < W) { stop = STOP_RANK_FINISHED; break; }
        I.rounds += 1;

        // Grouping of every buffer (Sec. 2.2), groups in formation order.
        std::vector<GroupList> list((size_t)W);
        for (int32_t r = 0; r < W; ++r) {
            std::vector<int32_t> visit;
            list[(size_t)r] = form_groups(buf[(size_t)r], R.len, L_max, &visit);
            for (size_t p = 0; p < visit.size(); ++p) pos[(size_t)visit[p]] = (int64_t)p;
        }

        // Eq. 3 over the active ranks A = {r : G_r > 0}; the minima over capacity and
        // buffered count only consider positive values; an absent capacity array means
        // no capacity limit.
        int64_t maxG = 0, minC = 0, minS = 0;
        for (int32_t r = 0; r < W; ++r) {
            int64_t G = (int64_t)list[(size_t)r].size();
            if (G <= 0) continue;
            maxG = std::max(maxG, G);
            int64_t Sr = (int64_t)buf[(size_t)r].size();
            if (Sr > 0) minS = (minS == 0) ? Sr : std::min(minS, Sr);
            if (capacity && capacity[r] > 0) minC = (minC == 0) ? capacity[r] : std::min(minC, capacity[r]);
        }
        int64_t T = maxG;
        if (minC > 0) T = std::min(T, minC);
        if (minS > 0) T = std::min(T, minS);
        T = std::max<int64_t>(T, 1);
        R.round_target.push_back(T);

        // App. B: what a rank can advertise before alignment is its buffer's sample and
        // token counts; the approximate mode prices an adjusted group at its row count
        // times the buffer's mean tokens per sample.  The exact mode needs post-alignment
        // counts, i.e. a second exchange, unless alignment left every active rank's
        // groups as they were (G_r = T for all r in A).
        std::vector<double> mean_len((size_t)W, 0.0);
        bool noop = true;
        for (int32_t r = 0; r < W; ++r) {
            const std::vector<int32_t>& b = buf[(size_t)r];
            if (b.empty()) continue;
            int64_t tok = 0;
            for (int32_t x : b) tok += R.len[(size_t)x];
            mean_len[(size_t)r] = (double)tok / (double)b.size();
            if ((int64_t)list[(size_t)r].size() != T) noop = false;
        }
        if (!noop) I.second_gather_rounds += 1;

        // Algorithm 1 on every active rank.
        std::vector<std::vector<int32_t>> returned((size_t)W);
        for (int32_t r = 0; r < W; ++r) {
            GroupList& L = list[(size_t)r];
            int64_t G = (int64_t)L.size();
            if (G == 0) continue;
            if (G < T) {
                I.splits += split_to(L, T);
            } else if (G > T) {
                I.overflow_groups += G - T;
                overflow_to(L, T, returned[(size_t)r]);
            }
            canonicalize(L, pos);
        }

        // Emit the round's T aligned steps; inactive ranks send IDLE slots.  In non-join
        // mode the trainer stops after the first step whose cumulative global emitted
        // count reaches the quota (Theorem 2).
        int64_t cut = T;
        bool quota_hit = false;
        for (int64_t j = 0; j < T; ++j) {
            int64_t step = 0;
            for (int32_t r = 0; r < W; ++r)
                if (!list[(size_t)r].empty()) step += (int64_t)list[(size_t)r][(size_t)j].size();
            emitted += step;
            I.max_step_samples = std::max(I.max_step_samples, step);
            if (mode == MODE_NONJOIN && emitted >= quota) {
                cut = j + 1;
                quota_hit = true;
                break;
            }
        }
        for (int32_t r = 0; r < W; ++r) {
            GroupList& L = list[(size_t)r];
            std::vector<int32_t> next;
            for (int64_t j = 0; j < cut; ++j) {
                R.slots[(size_t)r].push_back(L.empty() ? Group{} : L[(size_t)j]);
                R.slots_approx[(size_t)r].push_back(L.empty() ? 0.0
                                                               : (double)L[(size_t)j].size() * mean_len[(size_t)r]);
            }
            for (size_t j = (size_t)cut; j < L.size(); ++j)
                for (int32_t x : L[j]) next.push_back(x);
            for (int32_t x : returned[(size_t)r]) next.push_back(x);
            buf[(size_t)r] = next;
        }
        S += cut;
        if (quota_hit) { stop = STOP_QUOTA; break; }
    }
    I.steps = S;
    I.stop_reason = stop;
    I.emitted_samples = emitted;

    // Un-emitted samples (non-join only) stay with their rank, in visiting order
    // (length descending, id ascending) -- the No-Leak lemma (App. C).
    R.leftover.assign((size_t)W, {});
    for (int32_t r = 0; r < W; ++r) {
        std::vector<int32_t> left = buf[(size_t)r];
        std::stable_sort(left.begin(), left.end(), [&](int32_t a, int32_t b) {
            if (R.len[a] != R.len[b]) return R.len[a] > R.len[b];
            return a < b;
        });
        R.leftover[(size_t)r] = left;
        I.leftover_samples += (int64_t)left.size();
    }

    // Stats: real tokens and padded area; pad% = 1 - sum(L_real) / sum(L_compute).
    for (int32_t r = 0; r < W; ++r)
        for (const Group& g : R.slots[(size_t)r]) {
            int64_t mx = 0;
            for (int32_t x : g) {
                I.real_tokens += R.len[(size_t)x];
                mx = std::max(mx, R.len[(size_t)x]);
            }
            I.padded_elems += mx * (int64_t)g.size();
        }
    I.pad_fraction = I.padded_elems > 0 ? 1.0 - (double)I.real_tokens / (double)I.padded_elems : 0.0;

    // Coverage: every sampler view must be emitted exactly once (join) or sit in exactly
    // one of emitted / leftover (non-join); identities are counted over the same union.
    std::vector<int64_t> view_count((size_t)n, 0);
    int64_t N_id = identity ? num_identities : n;
    std::vector<int64_t> id_count((size_t)N_id, 0);
    auto count = [&](int32_t x) {
        view_count[(size_t)x] += 1;
        id_count[(size_t)(identity ? identity[x] : x)] += 1;
    };
    for (int32_t r = 0; r < W; ++r) {
        for (const Group& g : R.slots[(size_t)r])
            for (int32_t x : g) count(x);
        for (int32_t x : R.leftover[(size_t)r]) count(x);
    }
    for (int64_t i = 0; i < n; ++i) I.bad_views += view_count[(size_t)i] != 1 ? 1 : 0;
    for (int64_t d = 0; d < N_id; ++d) {
        if (id_count[(size_t)d] == 0) I.missing_ids += 1;
        if (id_count[(size_t)d] > 1) I.duplicate_ids += id_count[(size_t)d] - 1;
    }
    return true;
}

// ------------------------------------------------------------------ unified loop
// The streaming protocol of Sec. 2.3 ("Unified loop and termination") and App. C/E,
// with the per-rank state of App. C: sampler-pending views R_r, the collate buffer B_r
// (the worker queue is folded into it: a fetched view lands in the buffer in the same
// round), and emitted views E_r.
//   reading (sampler): the shuffled identity list perm[0..N) is padded to
//     M = W * ceil(N / W) views by repeating it from its head (view m has identity
//     perm[m mod N]), and view m belongs to rank m mod W (stride sharding); a rank visits
//     its views in increasing m.
//   reading (arrivals): in every round rank r moves up to rate[r] views from R_r to B_r,
//     in sampler order, without exceeding the outstanding-depth envelope |B_r| <= D.
//   reading (status): a rank is finished when R_r and B_r are empty (n_groups = -1); it
//     is ready when |B_r| >= buffer_size or R_r is empty and B_r is not; a ready rank
//     groups its whole buffer (n_groups = G_r > 0), an unready one reports 0.
//   reading (round kinds): join stops when every rank is finished; non-join stops when
//     any rank is finished (logical stop) or the quota is reached.  Otherwise, if some
//     unfinished rank is not ready the round is a skip round (no rank emits); else every
//     ready rank's buffer is grouped (Sec. 2.2), aligned (Eq. 3 over the ready ranks,
//     Algorithm 1) and emitted, finished ranks send IDLE slots, and overflow stays in B.
//   Ties in the length order break by view index m.
struct StreamInfo {
    int64_t steps;
    int64_t rounds;              // protocol rounds including the one that observed the stop
    int64_t emit_rounds;
    int64_t skip_rounds;
    int32_t stop_reason;
    int32_t reserved0;
    int64_t views;               // M
    int64_t emitted_views;
    int64_t undelivered_views;   // fetched but not emitted at the stop (sum over ranks of |B_r|)
    int64_t pending_views;       // never fetched (sum of |R_r|)
    int64_t real_tokens;
    int64_t padded_elems;
    int64_t max_step_samples;
    int64_t splits;
    int64_t overflow_groups;
    int64_t missing_ids;
    int64_t duplicate_ids;
    int64_t bad_views;
    int64_t second_gather_rounds;
    int64_t max_outstanding;     // largest |B_r| seen after a fetch
    double pad_fraction;
};

struct StreamRound {
    int32_t kind;      // 0 emit, 1 skip, 2 stop
    int32_t reserved0;
    int64_t target;    // T of an emit round, 0 otherwise
    int64_t emitted;   // views emitted in the round
    int64_t phi;       // potential after the round: views not yet emitted (App. C, Lyapunov)
};

struct StreamResult : Result {                      // the plan: slots hold identities
    StreamInfo sinfo{};
    std::vector<StreamRound> trace;
    std::vector<std::vector<int32_t>> emit_views;  // per rank, slot order, row order
    std::vector<std::vector<int32_t>> left_views;  // per rank, increasing m
};

bool run_stream(StreamResult& SR, int32_t W, int64_t N, const int64_t* tok_off, const int32_t* perm,
                int64_t L_max, int32_t mode, int64_t quota, int64_t buffer_size, int64_t depth,
                const int32_t* rate, const int64_t* capacity, int64_t max_rounds) {
    if (W < 1) return fail("W must be >= 1");
    if (N < 0 || N >= (int64_t)std::numeric_limits<int32_t>::max() / 2) return fail("N out of range");
    if (L_max < 1) return fail("budget must be >= 1");
    if (mode != MODE_JOIN && mode != MODE_NONJOIN) return fail("bad mode");
    if (mode == MODE_NONJOIN && quota < 1) return fail("quota must be >= 1 in non-join mode");
    if (buffer_size < 1 || depth < buffer_size) return fail("need 1 <= buffer_size <= depth");
    for (int32_t r = 0; r < W; ++r)
        if (rate[r] < 1) return fail("rate must be >= 1");
    if (capacity)
        for (int32_t r = 0; r < W; ++r)
            if (capacity[r] < 0) return fail("capacity must be >= 0");
    Result& R = SR;
    R.W = W;
    R.n = N;
    R.len.resize((size_t)N);
    for (int64_t i = 0; i < N; ++i) {
        int64_t l = tok_off[i + 1] - tok_off[i];
        if (l < 1 || l > (int64_t)std::numeric_limits<int32_t>::max())
            return fail("sample " + std::to_string(i) + " has invalid length " + std::to_string(l));
        R.len[(size_t)i] = l;
    }
    std::vector<char> seen((size_t)N, 0);
    for (int64_t i = 0; i < N; ++i) {
        if (perm[i] < 0 || perm[i] >= N || seen[(size_t)perm[i]]) return fail("perm is not a permutation");
        seen[(size_t)perm[i]] = 1;
    }
    const int64_t q = N > 0 ? (N + W - 1) / W : 0;   // views per rank
    const int64_t M = q * W;
    std::vector<int32_t> ident((size_t)M);
    std::vector<int64_t> vlen((size_t)M);
    for (int64_t m = 0; m < M; ++m) {
        ident[(size_t)m] = perm[m % N];
        vlen[(size_t)m] = R.len[(size_t)ident[(size_t)m]];
    }
    std::vector<int64_t> cursor((size_t)W, 0);          // next sampler position of each rank
    std::vector<std::vector<int32_t>> buf((size_t)W);   // B_r (view ids)
    R.slots.assign((size_t)W, {});
    R.slots_approx.assign((size_t)W, {});
    SR.emit_views.assign((size_t)W, {});
    std::vector<int64_t> pos((size_t)M, -1);
    StreamInfo& I = SR.sinfo;
    I.views = M;
    int64_t S = 0, emitted = 0;
    int32_t stop = STOP_DRAINED;
    for (;;) {
        if (I.rounds >= max_rounds) return fail("max_rounds exceeded");
        I.rounds += 1;
        // fetch (R -> B), bounded by the rank's rate and the envelope
        for (int32_t r = 0; r < W; ++r) {
            int64_t room = depth - (int64_t)buf[(size_t)r].size();
            int64_t f = std::min<int64_t>({(int64_t)rate[r], room, q - cursor[(size_t)r]});
            for (int64_t i = 0; i < f; ++i) buf[(size_t)r].push_back((int32_t)((cursor[(size_t)r] + i) * W + r));
            cursor[(size_t)r] += std::max<int64_t>(f, 0);
            I.max_outstanding = std::max(I.max_outstanding, (int64_t)buf[(size_t)r].size());
        }
        int32_t finished = 0, unready = 0;
        std::vector<char> ready((size_t)W, 0);
        for (int32_t r = 0; r < W; ++r) {
            bool drained = cursor[(size_t)r] == q;
            bool fin = drained && buf[(size_t)r].empty();
            finished += fin ? 1 : 0;
            ready[(size_t)r] = !fin && ((int64_t)buf[(size_t)r].size() >= buffer_size || drained);
            unready += (!fin && !ready[(size_t)r]) ? 1 : 0;
        }
        StreamRound rec{};
        if (finished == W) {
            stop = STOP_DRAINED;
            rec.kind = 2;
        } else if (mode == MODE_NONJOIN && finished > 0) {
            stop = STOP_RANK_FINISHED;
            rec.kind = 2;
        } else if (unready > 0) {
            rec.kind = 1;
        }
        if (rec.kind != 0) {
            rec.phi = M - emitted;
            SR.trace.push_back(rec);
            if (rec.kind == 2) break;
            I.skip_rounds += 1;
            continue;
        }
        I.emit_rounds += 1;
        // group every ready buffer (Sec. 2.2), groups in formation order
        std::vector<GroupList> list((size_t)W);
        std::vector<double> mean_len((size_t)W, 0.0);
        for (int32_t r = 0; r < W; ++r) {
            if (!ready[(size_t)r]) continue;
            std::vector<int32_t> visit;
            list[(size_t)r] = form_groups(buf[(size_t)r], vlen, L_max, &visit);
            for (size_t p = 0; p < visit.size(); ++p) pos[(size_t)visit[p]] = (int64_t)p;
            int64_t tok = 0;
            for (int32_t v : buf[(size_t)r]) tok += vlen[(size_t)v];
            mean_len[(size_t)r] = (double)tok / (double)buf[(size_t)r].size();
        }
        // Eq. 3 over the ready ranks
        int64_t maxG = 0, minC = 0, minS = 0;
        for (int32_t r = 0; r < W; ++r) {
            int64_t G = (int64_t)list[(size_t)r].size();
            if (G <= 0) continue;
            maxG = std::max(maxG, G);
            int64_t Sr = (int64_t)buf[(size_t)r].size();
            minS = (minS == 0) ? Sr : std::min(minS, Sr);
            if (capacity && capacity[r] > 0) minC = (minC == 0) ? capacity[r] : std::min(minC, capacity[r]);
        }
        int64_t T = maxG;
        if (minC > 0) T = std::min(T, minC);
        if (minS > 0) T = std::min(T, minS);
        T = std::max<int64_t>(T, 1);
        bool noop = true;
        std::vector<std::vector<int32_t>> returned((size_t)W);
        for (int32_t r = 0; r < W; ++r) {
            GroupList& L = list[(size_t)r];
            int64_t G = (int64_t)L.size();
            if (G == 0) continue;
            if (G != T) noop = false;
            if (G < T) {
                I.splits += split_to(L, T);
            } else if (G > T) {
                I.overflow_groups += G - T;
                overflow_to(L, T, returned[(size_t)r]);
            }
            canonicalize(L, pos);
        }
        if (!noop) I.second_gather_rounds += 1;
        int64_t cut = T;
        bool quota_hit = false;
        int64_t round_emitted = 0;
        for (int64_t j = 0; j < T; ++j) {
            int64_t step = 0;
            for (int32_t r = 0; r < W; ++r)
                if (!list[(size_t)r].empty()) step += (int64_t)list[(size_t)r][(size_t)j].size();
            emitted += step;
            round_emitted += step;
            I.max_step_samples = std::max(I.max_step_samples, step);
            if (mode == MODE_NONJOIN && emitted >= quota) {
                cut = j + 1;
                quota_hit = true;
                break;
            }
        }
        for (int32_t r = 0; r < W; ++r) {
            GroupList& L = list[(size_t)r];
            std::vector<int32_t> keep;
            for (int64_t j = 0; j < cut; ++j) {
                Group ids;
                if (!L.empty())
                    for (int32_t v : L[(size_t)j]) {
                        ids.push_back(ident[(size_t)v]);
                        SR.emit_views[(size_t)r].push_back(v);
                    }
                R.slots[(size_t)r].push_back(ids);
                R.slots_approx[(size_t)r].push_back(L.empty() ? 0.0 : (double)L[(size_t)j].size() * mean_len[(size_t)r]);
            }
            if (!ready[(size_t)r]) continue;   // a finished rank's buffer is empty
            for (size_t j = (size_t)cut; j < L.size(); ++j)
                for (int32_t v : L[j]) keep.push_back(v);
            for (int32_t v : returned[(size_t)r]) keep.push_back(v);
            buf[(size_t)r] = keep;
        }
        S += cut;
        rec.kind = 0;
        rec.target = T;
        rec.emitted = round_emitted;
        rec.phi = M - emitted;
        SR.trace.push_back(rec);
        if (quota_hit) {
            stop = STOP_QUOTA;
            break;
        }
    }
    I.steps = S;
    I.stop_reason = stop;
    I.emitted_views = emitted;
    // Stats as in the window pipeline (real tokens, padded area, pad fraction).
    for (int32_t r = 0; r < W; ++r)
        for (const Group& g : R.slots[(size_t)r]) {
            int64_t mx = 0;
            for (int32_t x : g) {
                I.real_tokens += R.len[(size_t)x];
                mx = std::max(mx, R.len[(size_t)x]);
            }
            I.padded_elems += mx * (int64_t)g.size();
        }
    I.pad_fraction = I.padded_elems > 0 ? 1.0 - (double)I.real_tokens / (double)I.padded_elems : 0.0;
    // Undelivered and pending views, and the No-Leak check over every view's state.
    std::vector<int32_t> state((size_t)M, 0);
    for (int32_t r = 0; r < W; ++r) {
        for (int32_t v : SR.emit_views[(size_t)r]) state[(size_t)v] += 1;
        for (int32_t v : buf[(size_t)r]) state[(size_t)v] += 1;
        for (int64_t i = cursor[(size_t)r]; i < q; ++i) state[(size_t)(i * W + r)] += 1;
        I.undelivered_views += (int64_t)buf[(size_t)r].size();
        I.pending_views += q - cursor[(size_t)r];
    }
    SR.left_views.assign((size_t)W, {});
    R.leftover.assign((size_t)W, {});
    std::vector<char> is_emitted((size_t)M, 0);
    for (int32_t r = 0; r < W; ++r)
        for (int32_t v : SR.emit_views[(size_t)r]) is_emitted[(size_t)v] = 1;
    for (int32_t r = 0; r < W; ++r)
        for (int64_t i = 0; i < q; ++i) {
            int32_t v = (int32_t)(i * W + r);
            if (!is_emitted[(size_t)v]) {
                SR.left_views[(size_t)r].push_back(v);
                R.leftover[(size_t)r].push_back(ident[(size_t)v]);
            }
        }
    std::vector<int64_t> id_count((size_t)N, 0);
    for (int64_t m = 0; m < M; ++m) {
        if (state[(size_t)m] != 1) I.bad_views += 1;
        id_count[(size_t)ident[(size_t)m]] += 1;   // every view is emitted or left over
    }
    // identity coverage of what was emitted (join: every identity, P duplicates)
    std::vector<int64_t> emit_count((size_t)N, 0);
    for (int32_t r = 0; r < W; ++r)
        for (int32_t v : SR.emit_views[(size_t)r]) emit_count[(size_t)ident[(size_t)v]] += 1;
    for (int64_t d = 0; d < N; ++d) {
        if (emit_count[(size_t)d] == 0) I.missing_ids += 1;
        if (emit_count[(size_t)d] > 1) I.duplicate_ids += emit_count[(size_t)d] - 1;
    }
    // the window-level summary the shared accessors read
    Info& PI = R.info;
    PI.steps = S;
    PI.rounds = (int32_t)std::min<int64_t>(I.emit_rounds, std::numeric_limits<int32_t>::max());
    PI.stop_reason = stop;
    PI.emitted_samples = emitted;
    PI.leftover_samples = M - emitted;
    PI.real_tokens = I.real_tokens;
    PI.padded_elems = I.padded_elems;
    PI.max_step_samples = I.max_step_samples;
    PI.splits = I.splits;
    PI.overflow_groups = I.overflow_groups;
    PI.missing_ids = I.missing_ids;
    PI.duplicate_ids = I.duplicate_ids;
    PI.bad_views = I.bad_views;
    PI.pad_fraction = I.pad_fraction;
    PI.second_gather_rounds = I.second_gather_rounds;
    R.rank_off.assign((size_t)W + 1, 0);
    return true;
}

}  // namespace

extern "C" {

typedef Info oracle_info_t;

const char* oracle_last_error(void) { return g_err.c_str(); }

// Runs grouping, alignment, stats and coverage on one window.  Returns an opaque handle
// (free with oracle_free) or NULL on invalid input (message via oracle_last_error).
void* oracle_plan(int32_t W, int64_t n, const int64_t* rank_off, const int64_t* tok_off,
                  const int64_t* identity, int64_t num_identities, int64_t budget, int32_t mode,
                  int64_t quota, const int64_t* capacity) {
    Result* R = new (std::nothrow) Result();
    if (!R) return nullptr;
    if (!run(*R, W, n, rank_off, tok_off, identity, num_identities, budget, mode, quota, capacity)) {
        delete R;
        return nullptr;
    }
    return R;
}

void oracle_free(void* h) { delete static_cast<Result*>(h); }

// Alignment target of every round; out must hold info.rounds entries.
void oracle_round_targets(void* h, int64_t* out) {
    const Result& R = *static_cast<Result*>(h);
    std::copy(R.round_target.begin(), R.round_target.end(), out);
}

void oracle_info(void* h, oracle_info_t* out) { *out = static_cast<Result*>(h)->info; }

void oracle_form(void* h, int32_t* order, int32_t* sorted_len, int32_t* group_index,
                 int32_t* groups_per_rank) {
    const Result& R = *static_cast<Result*>(h);
    std::copy(R.order.begin(), R.order.end(), order);
    std::copy(R.sorted_len.begin(), R.sorted_len.end(), sorted_len);
    std::copy(R.group_index.begin(), R.group_index.end(), group_index);
    std::copy(R.groups_per_rank.begin(), R.groups_per_rank.end(), groups_per_rank);
}

// Slot tables, rank-major (slot k = r * steps + j).  row_off / tile_off have
// W * steps + 1 entries (exclusive prefix sums of rows and of rows * maxlen).
void oracle_slots(void* h, int32_t* rows, int32_t* maxlen, int64_t* row_off, int64_t* tile_off,
                  int64_t* tokens) {
    const Result& R = *static_cast<Result*>(h);
    int64_t k = 0, ro = 0, to = 0;
    for (int32_t r = 0; r < R.W; ++r)
        for (const Group& g : R.slots[(size_t)r]) {
            int64_t mx = 0, tk = 0;
            for (int32_t x : g) {
                mx = std::max(mx, R.len[(size_t)x]);
                tk += R.len[(size_t)x];
            }
            rows[k] = (int32_t)g.size();
            maxlen[k] = (int32_t)mx;
            tokens[k] = tk;
            row_off[k] = ro;
            tile_off[k] = to;
            ro += (int64_t)g.size();
            to += (int64_t)g.size() * mx;
            ++k;
        }
    row_off[k] = ro;
    tile_off[k] = to;
}

// Approximate post-alignment token count of every slot (same layout as oracle_slots).
void oracle_slots_approx(void* h, double* tokens_approx) {
    const Result& R = *static_cast<Result*>(h);
    int64_t k = 0;
    for (int32_t r = 0; r < R.W; ++r)
        for (double a : R.slots_approx[(size_t)r]) tokens_approx[k++] = a;
}

// Loss-scaling weights (Eq. 2, App. B) of every slot, rank-major like the slot tables:
// at step j rank r pre-scales its mean loss by W * weight[r * steps + j], so that the
// mean over ranks equals sum_r weight * mean loss of rank r.
//   mode 0, sample level:            n_{r,j} / sum_r n_{r,j}
//   mode 1, approximate token level: a_{r,j} / sum_r a_{r,j}, a = rows * buffer mean length
//   mode 2, exact token level:       t_{r,j} / sum_r t_{r,j}  (t = real tokens of the slot)
// The sums run over ranks in rank order; a step whose sum is zero gets zero weights.
// step_tokens / step_samples (may be NULL) receive sum_r t_{r,j} and sum_r n_{r,j}.
int oracle_loss_weights(void* h, int32_t mode, double* weight, int64_t* step_tokens, int64_t* step_samples) {
    const Result& R = *static_cast<Result*>(h);
    if (mode < 0 || mode > 2) return -1;
    const int64_t S = R.info.steps;
    for (int64_t j = 0; j < S; ++j) {
        int64_t T_tok = 0, N = 0;
        double A = 0.0;
        std::vector<int64_t> t((size_t)R.W), c((size_t)R.W);
        for (int32_t r = 0; r < R.W; ++r) {
            const Group& g = R.slots[(size_t)r][(size_t)j];
            int64_t tk = 0;
            for (int32_t x : g) tk += R.len[(size_t)x];
            t[(size_t)r] = tk;
            c[(size_t)r] = (int64_t)g.size();
            T_tok += tk;
            N += (int64_t)g.size();
            A = A + R.slots_approx[(size_t)r][(size_t)j];
        }
        for (int32_t r = 0; r < R.W; ++r) {
            double w = 0.0;
            if (mode == 0 && N > 0) w = (double)c[(size_t)r] / (double)N;
            if (mode == 1 && A > 0.0) w = R.slots_approx[(size_t)r][(size_t)j] / A;
            if (mode == 2 && T_tok > 0) w = (double)t[(size_t)r] / (double)T_tok;
            weight[(int64_t)r * S + j] = w;
        }
        if (step_tokens) step_tokens[j] = T_tok;
        if (step_samples) step_samples[j] = N;
    }
    return 0;
}

// emit_order: emitted sample ids rank-major, slot order, row order.  leftover: the
// un-emitted ids of every rank (rank-major) with leftover_off[W+1].
void oracle_emit(void* h, int32_t* emit_order, int32_t* leftover, int64_t* leftover_off) {
    const Result& R = *static_cast<Result*>(h);
    int64_t e = 0;
    for (int32_t r = 0; r < R.W; ++r)
        for (const Group& g : R.slots[(size_t)r])
            for (int32_t x : g) emit_order[e++] = x;
    int64_t o = 0;
    for (int32_t r = 0; r < R.W; ++r) {
        leftover_off[r] = o;
        for (int32_t x : R.leftover[(size_t)r]) leftover[o++] = x;
    }
    leftover_off[R.W] = o;
}

// Collate (Sec. 2.1): every aligned group becomes a [rows, max_len] tile padded on the
// right.  reading (values): input_ids = labels = token, attention_mask = 1,
// position_ids = column for real tokens; pad_id, -100, 0, 0 for padding.  Tiles are
// packed back to back in rank-major slot order.  Writes the tiles of ranks
// [r_begin, r_end) from element 0 of the outputs; tokens[k - tok_base] is the token at
// CSR position k.
static void collate_ranks(const Result& R, int32_t r_begin, int32_t r_end, const int64_t* tok_off,
                          const int32_t* tokens, int64_t tok_base, int32_t pad_id, int32_t* input_ids,
                          int32_t* labels, int32_t* attention_mask, int32_t* position_ids) {
    int64_t e = 0;
    for (int32_t r = r_begin; r < r_end; ++r)
        for (const Group& g : R.slots[(size_t)r]) {
            int64_t mx = 0;
            for (int32_t x : g) mx = std::max(mx, R.len[(size_t)x]);
            for (int32_t x : g) {
                int64_t l = R.len[(size_t)x];
                for (int64_t c = 0; c < mx; ++c, ++e) {
                    if (c < l) {
                        int32_t t = tokens[tok_off[x] + c - tok_base];
                        input_ids[e] = t;
                        labels[e] = t;
                        attention_mask[e] = 1;
                        position_ids[e] = (int32_t)c;
                    } else {
                        input_ids[e] = pad_id;
                        labels[e] = -100;
                        attention_mask[e] = 0;
                        position_ids[e] = 0;
                    }
                }
            }
        }
}

// The whole window: outputs hold info.padded_elems elements.
void oracle_collate(void* h, const int64_t* tok_off, const int32_t* tokens, int32_t pad_id,
                    int32_t* input_ids, int32_t* labels, int32_t* attention_mask,
                    int32_t* position_ids) {
    const Result& R = *static_cast<Result*>(h);
    collate_ranks(R, 0, R.W, tok_off, tokens, 0, pad_id, input_ids, labels, attention_mask, position_ids);
}

// One rank's tiles (its slots r * steps ... (r + 1) * steps - 1).  tokens holds the CSR
// positions [tok_off[rank_off[r]], tok_off[rank_off[r + 1]]) only, which is all that
// rank's samples own.  Returns 0, or -1 for a rank out of range.
int oracle_collate_rank(void* h, int32_t r, const int64_t* tok_off, const int32_t* tokens, int32_t pad_id,
                        int32_t* input_ids, int32_t* labels, int32_t* attention_mask,
                        int32_t* position_ids) {
    const Result& R = *static_cast<Result*>(h);
    if (r < 0 || r >= R.W) return -1;
    const int64_t base = tok_off[R.rank_off[(size_t)r]];
    collate_ranks(R, r, r + 1, tok_off, tokens, base, pad_id, input_ids, labels, attention_mask, position_ids);
    return 0;
}

// One rank's tiles as oracle_collate_rank, with `tokens` the whole token stream (CSR
// position k at tokens[k]): for streaming plans, whose rows carry identities from anywhere
// in the dataset.  Returns 0, or -1 for a rank out of range.
int oracle_collate_rank_all(void* h, int32_t r, const int64_t* tok_off, const int32_t* tokens, int32_t pad_id,
                            int32_t* input_ids, int32_t* labels, int32_t* attention_mask,
                            int32_t* position_ids) {
    const Result& R = *static_cast<Result*>(h);
    if (r < 0 || r >= R.W) return -1;
    collate_ranks(R, r, r + 1, tok_off, tokens, 0, pad_id, input_ids, labels, attention_mask, position_ids);
    return 0;
}

// ------------------------------------------------------------------ unified loop API
// One logical iteration of the streaming protocol over identities 0..N-1 (lengths from
// tok_off).  Returns a handle whose plan the window accessors above read (slots hold
// identities; leftover lists the identities of un-emitted views), or NULL.
void* oracle_stream(int32_t W, int64_t N, const int64_t* tok_off, const int32_t* perm, int64_t budget,
                    int32_t mode, int64_t quota, int64_t buffer_size, int64_t depth, const int32_t* rate,
                    const int64_t* capacity, int64_t max_rounds) {
    StreamResult* SR = new (std::nothrow) StreamResult();
    if (!SR) return nullptr;
    if (!run_stream(*SR, W, N, tok_off, perm, budget, mode, quota, buffer_size, depth, rate, capacity,
                    max_rounds)) {
        delete SR;
        return nullptr;
    }
    // the handle is the window plan it contains, so every window accessor applies
    return static_cast<Result*>(SR);
}

static StreamResult* stream_of(void* h) { return static_cast<StreamResult*>(static_cast<Result*>(h)); }

void oracle_stream_free(void* h) { delete stream_of(h); }

void oracle_stream_info(void* h, StreamInfo* out) { *out = stream_of(h)->sinfo; }

// Per-round trace; out must hold info.rounds records.
void oracle_stream_trace(void* h, StreamRound* out) {
    const StreamResult* SR = stream_of(h);
    std::copy(SR->trace.begin(), SR->trace.end(), out);
}

// Emitted views (rank-major, slot order, row order) and un-emitted views per rank in
// increasing view index, with left_off[W + 1].
void oracle_stream_views(void* h, int32_t* emit_views, int32_t* left_views, int64_t* left_off) {
    const StreamResult* SR = stream_of(h);
    int64_t e = 0, o = 0;
    for (const auto& v : SR->emit_views)
        for (int32_t x : v) emit_views[e++] = x;
    for (size_t r = 0; r < SR->left_views.size(); ++r) {
        left_off[r] = o;
        for (int32_t x : SR->left_views[r]) left_views[o++] = x;
    }
    left_off[SR->left_views.size()] = o;
}

}  // extern "C"
