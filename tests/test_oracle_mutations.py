"""The pins must catch plausible mistakes: each case plants one mistake in a
copy of the oracle source (on the CPU), builds it, and requires the pin
suite to fail against the mutant."""
import os
import shutil
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "ewsjf_oracle.cpp")

# (name, original text, planted mistake)
MUTANTS = [
    ("qf_zero_based_queue_index", "(double)(q + 1) / (b + 1.0)", "(double)(q) / (b + 1.0)"),
    ("qf_drops_plus_one", "(double)(q + 1) / (b + 1.0)", "(double)(q + 1) / (b)"),
    ("fairness_term_dropped", "+ w_fair * std::log(b + 1.0)", ""),
    ("log_of_b_not_b_plus_1", "std::log(b + 1.0)", "std::log(b)"),
    ("wait_sign_flipped", "(double)now - (double)arrival;", "(double)arrival - (double)now;"),
    ("cost_drops_linear_term", "c0 + c1 * b + c2 * b * b", "c0 + c2 * b * b"),
    ("compute_score_inverted", "const double cs = W / C;", "const double cs = C / W;"),
    ("urgency_weight_operands_swapped", "(double)th[2] * m + (double)th[3]", "(double)th[3] * m + (double)th[2]"),
    ("prune_merges_highest_utility", "if (i == 0 || u < best_u)", "if (i == 0 || u > best_u)"),
    ("prune_density_off_by_one", "(double)((int64_t)q[i].hi - (int64_t)q[i].lo + 1)",
     "(double)((int64_t)q[i].hi - (int64_t)q[i].lo + 2)"),
    ("prune_ignores_mean_distance", "(std::fabs(m_b - m_a) + eps)", "(1.0 + eps)"),
    ("split_uses_count_not_gaps", "members_minus_one = VC - 1;", "members_minus_one = VC;"),
    ("split_threshold_without_alpha", "const double rhs = alpha * (double)span;",
     "const double rhs = (double)span;"),
    ("equal_width_denominator", "* (int64_t)K / width;", "* (int64_t)K / (width - 1 + (width == 1));"),
    ("select_tie_prefers_high_id", "(s[a] == s[b] && a < b)", "(s[a] == s[b] && a > b)"),
    ("route_lower_bound", "std::upper_bound(bounds, bounds + (k - 1), b)", "std::lower_bound(bounds, bounds + (k - 1), b)"),
    ("kmeans_wrong_count", "(s2 * s2) / n2", "(s2 * s2) / n1"),
    ("mean_inverted", "mean[i] = (double)q[i].S / (double)q[i].n;", "mean[i] = (double)q[i].n / (double)q[i].S;"),
    ("window_not_clamped", "x = std::min(std::max(x, 1), max_len);", "x = std::max(x, 1);"),
    # Algorithm 1 (tactical step)
    ("fifo_newest_first", "return x.arrival < y.arrival || (x.arrival == y.arrival && x.id < y.id);",
     "return x.arrival > y.arrival || (x.arrival == y.arrival && x.id < y.id);"),
    ("fifo_tie_prefers_high_id", "(x.arrival == y.arrival && x.id < y.id)", "(x.arrival == y.arrival && x.id > y.id)"),
    ("argmax_takes_lowest_score", "(prim < 0 || head_score[q] > head_score[prim])",
     "(prim < 0 || head_score[q] < head_score[prim])"),
    ("argmax_tie_to_high_index", "(prim < 0 || head_score[q] > head_score[prim])",
     "(prim < 0 || head_score[q] >= head_score[prim])"),
    ("backfill_ignores_head_scores", "if (adj.size() == 2 && head_score[adj[1]] > head_score[adj[0]])",
     "if (false)"),
    ("backfill_skips_upper_neighbour", "if (prim + 1 < k && !fifo[prim + 1].empty()) adj.push_back(prim + 1);", ""),
    ("empty_count_never_reset", "      empty_cnt[q] = 0;\n", "\n"),
    ("empty_threshold_off_by_one", "if (empty_cnt[q] > empty_threshold)", "if (empty_cnt[q] >= empty_threshold)"),
    ("absorber_highest_utility", "utility(qs[r - 1], qs[r], eps) <= utility(qs[r], qs[r + 1], eps)",
     "utility(qs[r - 1], qs[r], eps) > utility(qs[r], qs[r + 1], eps)"),
    ("absorber_drops_counts", "A = {A.n + qs[r].n, A.S + qs[r].S,", "A = {A.n, A.S + qs[r].S,"),
    ("removal_rebuilds_bounds_from_lo", "if (q > 0) bounds[q - 1] = bnd[q - 1];",
     "if (q > 0) bounds[q - 1] = qs[q].lo;"),
    ("removal_deletes_the_far_boundary", "bnd.erase(bnd.begin() + std::min(r, a));",
     "bnd.erase(bnd.begin() + (a < r ? r : r + 1 < (int32_t)bnd.size() ? r + 1 : r - 1));"),
    # Algorithm 2 (bubble queues)
    ("bubble_lower_tolerance_strict", "if (10 * b <= 11 * max_len_i) return i;", "if (10 * b < 11 * max_len_i) return i;"),
    ("bubble_upper_tolerance_factor", "if (10 * b >= 9 * min_len_next) return i + 1;",
     "if (10 * b >= 8 * min_len_next) return i + 1;"),
    ("bubble_max_len_is_hi", "const int64_t max_len = (int64_t)chi[i] + 1, min_len = clo[i + 1];",
     "const int64_t max_len = (int64_t)chi[i], min_len = clo[i + 1];"),
    ("bubble_available_off_by_one", "const int64_t available = min_len - max_len;",
     "const int64_t available = min_len - max_len + 1;"),
    ("bubble_not_centred", "const int64_t new_min = std::max(b - range / 2, max_len);",
     "const int64_t new_min = std::max(b - range, max_len);"),
    ("bubble_upper_edge_unclipped", "std::min(b - range / 2 + range, min_len)", "(b - range / 2 + range)"),
    ("bubble_profile_is_its_width", "1, b, (double)b, next_ident", "1, range, (double)b, next_ident"),
    ("bubble_cap_off_by_one", "if (t < 0 && m < max_queues)", "if (t < 0 && m <= max_queues)"),
    ("nearer_tie_goes_high", "return b - hi_i <= lo_next - b ? i : i + 1;", "return b - hi_i < lo_next - b ? i : i + 1;"),
    ("dispatch_in_id_order", "  std::stable_sort(order.begin(), order.end(), older);\n", "\n"),
    ("gapped_route_without_tolerance", "const int32_t t = tolerance(b, (int64_t)hi[i] + 1, lo[i + 1], i);",
     "const int32_t t = -1;"),
    ("below_first_goes_up", "    *q = 0;\n    return false;", "    *q = k > 1 ? 1 : 0;\n    return false;"),
]


def _run_mutant(args):
    name, orig, bad = args
    src = open(SRC).read()
    assert src.count(orig) >= 1, name
    mutated = src.replace(orig, bad, 1)
    d = tempfile.mkdtemp(prefix=f"mut_{name}_")
    try:
        cpp = os.path.join(d, "m.cpp")
        so = os.path.join(d, "m.so")
        open(cpp, "w").write(mutated)
        subprocess.run(["g++", "-std=c++17", "-O1", "-ffp-contract=off", "-fPIC", "-shared", cpp, "-o", so],
                       check=True, capture_output=True)
        env = dict(os.environ, EWSJF_ORACLE_LIB=so)
        r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                            os.path.join(ROOT, "tests", "test_oracle_pins.py"),
                            os.path.join(ROOT, "tests", "test_oracle_tactical.py"),
                            os.path.join(ROOT, "tests", "test_oracle_bubble.py")],
                           cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
        return name, r.returncode
    finally:
        shutil.rmtree(d, ignore_errors=True)


def test_pins_catch_every_planted_mistake():
    with ThreadPoolExecutor(max_workers=4) as ex:
        results = list(ex.map(_run_mutant, MUTANTS))
    survivors = [n for n, rc in results if rc == 0]
    assert not survivors, f"pins did not catch: {survivors}"


@pytest.mark.parametrize("name,orig,bad", MUTANTS[:1])
def test_unmutated_source_passes(name, orig, bad):
    assert open(SRC).read().count(orig) == 1
