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

MUTANTS = {
    # frontier
    "tie_to_highest_rank": ("if (P[r] > F) {", "if (P[r] >= F) {"),
    "no_prefix_reset": ("for (int32_t r = 0; r < R; ++r) P[r] = 0;", ""),
    "stage_max_not_prefix": ("P[r] += row[r];", "P[r] = row[r];"),
    "transposed_layout": ("P[r] += row[r];", "P[r] += d[(t * R + r) * (int64_t)S + s];"),
    "absolute_not_advance": ("F_prev = F;", ""),
    "sign_flip": ("inc[t * S + s] = F - F_prev;", "inc[t * S + s] = F_prev - F;"),
    "rank_relabel": ("L = r;", "L = R - 1 - r;"),
    "start_leader_minus_one": ("int32_t L = 0;", "int32_t L = -1;"),
    "skip_first_rank_in_prefix": ("for (int32_t r = 0; r < R; ++r) P[r] += row[r];",
                                  "for (int32_t r = 1; r < R; ++r) P[r] += row[r];"),
    # window summary
    "last_window_short": ("int64_t t1 = t0 + window < T ? t0 + window : T;",
                          "int64_t t1 = t0 + window < T ? t0 + window : T - 1;"),
    "exposed_drops_first_step": ("for (int64_t t = t0; t < t1; ++t) sum += inc[t * S + s];",
                                 "for (int64_t t = t0 + 1; t < t1; ++t) sum += inc[t * S + s];"),
    "rank0_not_counted": ("if (r >= 0 && r < R) c[r] += 1;", "if (r > 0 && r < R) c[r] += 1;"),
    "top_stage_tie_to_higher": ("if (exposed[w * S + s] > exposed[w * S + s1]) s1 = s;",
                                "if (exposed[w * S + s] >= exposed[w * S + s1]) s1 = s;"),
    "second_stage_may_repeat_first": ("if (s == s1) continue;", ""),
    "modal_rank_tie_to_higher": ("if (c[r] > best) {", "if (c[r] >= best && c[r] > 0) {"),
    "top2_ascending": ("if (s2 < 0 || exposed[w * S + s] > exposed[w * S + s2]) s2 = s;",
                       "if (s2 < 0 || exposed[w * S + s] < exposed[w * S + s2]) s2 = s;"),
}


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
    old, new = MUTANTS[name]
    assert source.count(old) == 1, "mutation anchor must occur exactly once: %r" % old
    src = tmp_path / ("%s.c" % name)
    src.write_text(source.replace(old, new))
    lib = oracle.build(force=True, src=str(src), out=str(tmp_path / ("lib%s.so" % name)))
    failed = _run_all(oracle.COracle(lib))
    assert failed, "mutant %s passed every pin" % name
