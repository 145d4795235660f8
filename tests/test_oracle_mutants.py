"""Plant plausible mistakes in copies of the oracle and require that the pin
suite catches every one of them (CPU only).

Each mutant is one textual edit of ``oracle/sf_oracle.c``; the edited copy is
compiled into a temporary library and run through every pin.  A mutant that
passes all pins would mean the pins leave that part of the oracle unchecked.
"""
import os

import pytest

import oracle
import pins

SRC = os.path.join(os.path.dirname(oracle.__file__), "sf_oracle.c")

# (function, anchor, replacement): the anchor must occur exactly once in the
# body of that function
MUTANTS = {
    # frontier
    "tie_to_highest_rank": ("sfo_frontier", "r < R && L < 0", "r < R"),
    "no_prefix_reset": ("sfo_frontier", "(s > 0 ? P[(int64_t)(s - 1) * R + r] : 0)",
                        "(s > 0 ? P[(int64_t)(s - 1) * R + r] : P[(int64_t)(S - 1) * R + r])"),
    "stage_max_not_prefix": ("sfo_frontier", "(s > 0 ? P[(int64_t)(s - 1) * R + r] : 0) + ", ""),
    "transposed_layout": ("sfo_frontier", "+ m[(int64_t)s * R + r];", "+ m[(int64_t)r * S + s];"),
    "exclusive_prefix": ("sfo_frontier", "+ m[(int64_t)s * R + r];",
                         "+ (s > 0 ? m[(int64_t)(s - 1) * R + r] : 0);"),
    "absolute_not_advance": ("sfo_frontier", "F[s] - (s > 0 ? F[s - 1] : 0)", "F[s]"),
    "sign_flip": ("sfo_frontier", "F[s] - (s > 0 ? F[s - 1] : 0)", "(s > 0 ? F[s - 1] : 0) - F[s]"),
    "rank_relabel": ("sfo_frontier", "lead[t * S + s] = L;", "lead[t * S + s] = R - 1 - L;"),
    "max_skips_last_rank": ("sfo_frontier", "for (int32_t r = 1; r < R; ++r)\n                if (row[r] > best)",
                            "for (int32_t r = 1; r < R - 1; ++r)\n                if (row[r] > best)"),
    "skip_first_rank_in_prefix": ("sfo_frontier", "for (int32_t r = 0; r < R; ++r)\n                P[",
                                  "for (int32_t r = 1; r < R; ++r)\n                P["),
    # window summary
    "last_window_short": ("sfo_window_summary", "int64_t t1 = t0 + window < T ? t0 + window : T;",
                          "int64_t t1 = t0 + window < T ? t0 + window : T - 1;"),
    "exposed_drops_first_step": ("sfo_window_summary",
                                 "for (int64_t t = t0; t < t1; ++t) sum += inc[t * S + s];",
                                 "for (int64_t t = t0 + 1; t < t1; ++t) sum += inc[t * S + s];"),
    "rank0_not_counted": ("sfo_window_summary", "if (r >= 0 && r < R) c[r] += 1;",
                          "if (r > 0 && r < R) c[r] += 1;"),
    "top_stage_tie_to_higher": ("sfo_window_summary",
                                "if (exposed[w * S + s] > exposed[w * S + s1]) s1 = s;",
                                "if (exposed[w * S + s] >= exposed[w * S + s1]) s1 = s;"),
    "second_stage_may_repeat_first": ("sfo_window_summary", "if (s == s1) continue;", ""),
    "modal_rank_tie_to_higher": ("sfo_window_summary", "if (c[r] > best) {",
                                 "if (c[r] >= best && c[r] > 0) {"),
    "top2_ascending": ("sfo_window_summary",
                       "if (s2 < 0 || exposed[w * S + s] > exposed[w * S + s2]) s2 = s;",
                       "if (s2 < 0 || exposed[w * S + s] < exposed[w * S + s2]) s2 = s;"),
    # exposed time led per (window, stage, rank) and its top-2
    "le_weight_is_count": ("sfo_window_lead_exposed", "if (r >= 0 && r < R) e[r] += inc[t * S + s];",
                           "if (r >= 0 && r < R) e[r] += 1;"),
    "le_rank0_not_counted": ("sfo_window_lead_exposed", "if (r >= 0 && r < R) e[r] += inc[t * S + s];",
                             "if (r > 0 && r < R) e[r] += inc[t * S + s];"),
    "le_drops_last_step": ("sfo_window_lead_exposed", "int64_t t1 = t0 + window < T ? t0 + window : T;",
                           "int64_t t1 = t0 + window < T ? t0 + window - 1 : T;"),
    "le_wrong_stage_weight": ("sfo_window_lead_exposed", "if (r >= 0 && r < R) e[r] += inc[t * S + s];",
                              "if (r >= 0 && r < R) e[r] += inc[t * S + (S - 1 - s)];"),
    "le_first_stage_tie_to_higher": ("sfo_window_lead_exposed", "if (s1 < 0 || tot > e1) {",
                                     "if (s1 < 0 || tot >= e1) {"),
    "le_second_not_demoted": ("sfo_window_lead_exposed", "s2 = s1;\n                e2 = e1;\n", ""),
    "le_rank_tie_to_higher": ("sfo_window_lead_exposed", "if (e[r] > best) {",
                              "if (e[r] >= best && e[r] > 0) {"),
    "le_rank_first_nonzero": ("sfo_window_lead_exposed", "best = e[r];", "best = INT64_MAX;"),
    # leader switches between confident unique leaders
    "sw_ties_not_unique": ("sfo_window_leader_switches", "ties[i] == 1 &&", "ties[i] >= 1 &&"),
    "sw_gap_strict": ("sfo_window_leader_switches", "gap[i] >= min_gap", "gap[i] > min_gap"),
    "sw_single_rank_not_confident": ("sfo_window_leader_switches", " || gap[i] < 0", ""),
    "sw_prev_not_updated": ("sfo_window_leader_switches", "prev = lead[i];\n", ""),
    "sw_prev_from_any_boundary": ("sfo_window_leader_switches", "if (!confident) continue;",
                                  "if (!confident) { prev = lead[i]; have_prev = 1; continue; }"),
    "sw_eligible_counts_all": ("sfo_window_leader_switches",
                               "if (!confident) continue;\n                n_el += 1;",
                               "n_el += 1;\n                if (!confident) continue;"),
    "sw_first_compares_rank0": ("sfo_window_leader_switches", "int have_prev = 0;", "int have_prev = 1;"),
    "sw_short_window": ("sfo_window_leader_switches", "int64_t t1 = t0 + window < T ? t0 + window : T;",
                        "int64_t t1 = t0 + window < T ? t0 + window - 1 : T;"),
    # localization evidence and baselines
    "ev_tie_to_highest_rank": ("sfo_frontier_evidence", "r < R && L < 0", "r < R"),
    "ev_no_prefix_reset": ("sfo_frontier_evidence", "(s > 0 ? P[(int64_t)(s - 1) * R + r] : 0)",
                           "(s > 0 ? P[(int64_t)(s - 1) * R + r] : P[(int64_t)(S - 1) * R + r])"),
    "ev_absolute_not_advance": ("sfo_frontier_evidence", "F[s] - (s > 0 ? F[s - 1] : 0)", "F[s]"),
    "ev_tie_count_excludes_leader": ("sfo_frontier_evidence", "if (row[r] == best) n_tie += 1;",
                                     "if (row[r] == best && r != L) n_tie += 1;"),
    "ev_runner_up_may_be_leader": ("sfo_frontier_evidence",
                                   "if (r != L && (!have_second || row[r] > second)) {",
                                   "if (!have_second || row[r] > second) {"),
    "ev_gap_sign": ("sfo_frontier_evidence", "gap[i] = have_second ? best - second : -1;",
                    "gap[i] = have_second ? second - best : -1;"),
    "ev_single_rank_gap_zero": ("sfo_frontier_evidence", "gap[i] = have_second ? best - second : -1;",
                                "gap[i] = have_second ? best - second : 0;"),
    "ev_stage_max_of_prefix": ("sfo_frontier_evidence", "if (ds[r] > dmax) dmax = ds[r];",
                               "if (row[r] > dmax) dmax = row[r];"),
    "ev_stage_sum_skips_rank0": ("sfo_frontier_evidence", "dsum += ds[r];",
                                 "if (r) dsum += ds[r];"),
    # ingest
    "ingest_residual_unclamped": ("sfo_ingest", "d[(t * S + K) * R + r] = e > 0 ? e : 0;",
                                  "d[(t * S + K) * R + r] = e;"),
    "ingest_overlap_sign": ("sfo_ingest", "o[t * R + r] = e < 0 ? -e : 0;",
                            "o[t * R + r] = e < 0 ? e : 0;"),
    "ingest_residual_first": ("sfo_ingest", "d[(t * S + k) * R + r] = xs[k];",
                              "d[(t * S + k + 1) * R + r] = xs[k];"),
    "ingest_wall_of_next_rank": ("sfo_ingest", "const int64_t e = w[(int64_t)r * T + t] - explicit_sum;",
                                 "const int64_t e = w[(int64_t)((r + 1) % R) * T + t] - explicit_sum;"),
    # routing set
    "route_ascending": ("sfo_route", "while (j > 0 && ex[ord[j - 1]] < ex[s]) {",
                        "while (j > 0 && ex[ord[j - 1]] > ex[s]) {"),
    "route_tie_to_higher_stage": ("sfo_route", "while (j > 0 && ex[ord[j - 1]] < ex[s]) {",
                                  "while (j > 0 && ex[ord[j - 1]] <= ex[s]) {"),
    "route_strict_threshold": ("sfo_route", "while (k < S && (__int128)tau_den * cum < need) {",
                               "while (k < S && (__int128)tau_den * cum <= need) {"),
    "route_tau_inverted": ("sfo_route", "const __int128 need = (__int128)tau_num * total;",
                           "const __int128 need = (__int128)tau_den * total;"),
    # direct-exposure gain
    "gain_unclipped": ("sfo_exposure_gain", "if (b < *cell) *cell = b;", "*cell = b;"),
    "gain_replaces_next_stage": ("sfo_exposure_gain", "int64_t* cell = m + (int64_t)s * R + r;",
                                 "int64_t* cell = m + (int64_t)((s + 1) % S) * R + r;"),
    "gain_baseline_of_window0": ("sfo_exposure_gain", "const int64_t b = btilde[(w * S + s) * R + r];",
                                 "const int64_t b = btilde[(0 * S + s) * R + r];"),
    "gain_window_sum_skips_first": ("sfo_exposure_gain", "wgain[w * S + s] += g;",
                                    "if (t % window) wgain[w * S + s] += g;"),
    "gain_frontier_misses_last_stage": ("last_frontier", "for (int32_t s = 0; s < S; ++s) {",
                                        "for (int32_t s = 0; s < S - 1; ++s) {"),
    # lag
    "lag_upper_median": ("sfo_frontier_lag", "const int64_t median = sorted[(R - 1) / 2];",
                         "const int64_t median = sorted[R / 2];"),
    "lag_of_durations": ("sfo_frontier_lag", "memcpy(sorted, P, sizeof(int64_t) * (size_t)R);",
                         "memcpy(sorted, row, sizeof(int64_t) * (size_t)R);"),
    "lag_increment_not_reset": ("sfo_frontier_lag", "int64_t L_prev = 0;",
                                "static int64_t L_prev = 0;"),
    "lag_against_min": ("sfo_frontier_lag", "const int64_t median = sorted[(R - 1) / 2];",
                        "const int64_t median = sorted[0];"),
    # raw rank spread
    "spread_upper_median": ("sfo_rank_spread", "sorted[R - 1] - sorted[(R - 1) / 2];",
                            "sorted[R - 1] - sorted[R / 2];"),
    "spread_from_min": ("sfo_rank_spread", "sorted[R - 1] - sorted[(R - 1) / 2];",
                        "sorted[(R - 1) / 2] - sorted[0];"),
    "spread_window_overwrites": ("sfo_rank_spread", "wspread[w * S + s] += x;",
                                 "wspread[w * S + s] = x;"),
    "spread_drops_last_rank": ("sfo_rank_spread", "qsort(sorted, (size_t)R, sizeof(int64_t), cmp_i64);",
                               "qsort(sorted, (size_t)(R > 1 ? R - 1 : R), sizeof(int64_t), cmp_i64);"),
    # range status
    "range_inclusive_bound": ("sfo_range_status", "if (row[r] < 0 || row[r] >= limit - P[r]) {",
                              "if (row[r] < 0 || row[r] > limit - P[r]) {"),
    "range_ignores_negative": ("sfo_range_status", "if (row[r] < 0 || row[r] >= limit - P[r]) {",
                               "if (row[r] >= limit - P[r]) {"),
    "range_durations_not_prefixes": ("sfo_range_status", "P[r] += row[r];", ""),
    "range_carries_across_steps": ("sfo_range_status", "for (int32_t r = 0; r < R; ++r) P[r] = 0;", ""),
    # per-rank window median
    "median_upper": ("sfo_window_median", "med[(w * S + s) * (int64_t)R + r] = col[(n - 1) / 2];",
                     "med[(w * S + s) * (int64_t)R + r] = col[n / 2];"),
    "median_drops_last_step": ("sfo_window_median", "const int64_t n = t1 - t0;",
                               "const int64_t n = t1 - t0 - (t1 - t0 > 1);"),
    "median_stage_zero_only": ("sfo_window_median", "col[t - t0] = d[(t * S + s) * (int64_t)R + r];",
                               "col[t - t0] = d[(t * S + 0) * (int64_t)R + r];"),
    "median_unsorted": ("sfo_window_median", "qsort(col, (size_t)n, sizeof(int64_t), cmp_i64);", ""),
}


def _function_span(source, name):
    """[start, end) of the definition of C function ``name`` in ``source``."""
    import re
    m = re.search(r"^\w[^\n;]*\b%s\(" % name, source, flags=re.M)
    assert m, name
    end = source.index("\n}\n", m.start()) + 3
    return m.start(), end


def _run_all(o):
    """Names of the pins that fail for oracle ``o``."""
    failed = []
    for pin in pins.FRONTIER_PINS:
        try:
            pin(o.frontier)
        except AssertionError:
            failed.append(pin.__name__)
    for pin in pins.SUMMARY_PINS:
        try:
            pin(o.frontier, o.window_summary)
        except AssertionError:
            failed.append(pin.__name__)
    for pin in pins.LEAD_PINS:
        try:
            pin(o.frontier, o.window_lead_exposed)
        except AssertionError:
            failed.append(pin.__name__)
    try:
        pins.pin_lead_top2_cases(o.frontier, o.window_lead_exposed, o.window_summary)
    except AssertionError:
        failed.append("pin_lead_top2_cases")
    for pin in pins.SWITCH_PINS:
        try:
            pin(o.frontier_evidence, o.window_leader_switches)
        except AssertionError:
            failed.append(pin.__name__)
    for pin in pins.EVIDENCE_PINS:
        try:
            pin(o.frontier_evidence)
        except AssertionError:
            failed.append(pin.__name__)
    for pin in pins.INGEST_PINS:
        try:
            pin(o.ingest)
        except AssertionError:
            failed.append(pin.__name__)
    for pin in pins.ROUTE_PINS:
        try:
            pin(o.route)
        except AssertionError:
            failed.append(pin.__name__)
    for pin in pins.GAIN_PINS:
        try:
            pin(o.exposure_gain)
        except AssertionError:
            failed.append(pin.__name__)
    for pin in pins.LAG_PINS:
        try:
            pin(o.frontier_lag)
        except AssertionError:
            failed.append(pin.__name__)
    for pin in pins.SPREAD_PINS:
        try:
            pin(o.rank_spread)
        except AssertionError:
            failed.append(pin.__name__)
    try:
        pins.pin_spread_first_boundary_is_lag(o.rank_spread, o.frontier_lag)
    except AssertionError:
        failed.append("pin_spread_first_boundary_is_lag")
    for pin in pins.MEDIAN_PINS:
        try:
            pin(o.window_median)
        except AssertionError:
            failed.append(pin.__name__)
    for pin in pins.RANGE_PINS:
        try:
            pin(o.range_status)
        except AssertionError:
            failed.append(pin.__name__)
    return failed


@pytest.fixture(scope="module")
def source():
    with open(SRC) as fh:
        return fh.read()


def test_unmutated_copy_passes(source, tmp_path):
    src = tmp_path / "copy.c"
    src.write_text(source)
    lib = oracle.build(force=True, src=str(src), out=str(tmp_path / "libcopy.so"))
    assert _run_all(oracle.COracle(lib)) == []


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, source, tmp_path):
    func, old, new = MUTANTS[name]
    a, b = _function_span(source, func)
    body = source[a:b]
    assert body.count(old) == 1, "mutation anchor must occur once in %s: %r" % (func, old)
    src = tmp_path / ("%s.c" % name)
    src.write_text(source[:a] + body.replace(old, new) + source[b:])
    lib = oracle.build(force=True, src=str(src), out=str(tmp_path / ("lib%s.so" % name)))
    failed = _run_all(oracle.COracle(lib))
    assert failed, "mutant %s passed every pin" % name
