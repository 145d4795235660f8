"""Pins of the frontier-accounting oracle to facts outside the oracle itself.

Each ``pin_*`` takes a frontier function ``f(d[T,S,R]) -> (inc, lead)`` and
(where needed) a summary function ``g(inc, lead, R, window) -> (exposed,
counts, top2)`` and raises ``AssertionError`` on a violation.  The suite in
``test_oracle_pins.py`` applies them to the oracle; ``test_oracle_mutants.py``
applies them to copies of the oracle with planted mistakes and requires that
every mistake is caught by at least one pin.

What pins what:
  * printed worked examples (Sec. 2, Fig. fig:frontier-accounting, Sec. 4);
  * Theorem 1 (telescoping: advances sum to the largest rank total) and the
    nonnegativity of advances stated after Eq. (1);
  * the slack identity, Eq. (3), an independent formula for each advance;
  * Propositions 1 and 2 (max overcount / average undercount bounds, with the
    tight constructions of Appendix D);
  * the measurement-error stability proposition of Appendix D;
  * the R = 1 edge case (Sec. 3: the frontier is the rank's own vector);
  * brute force over every small integer matrix;
  * structural invariants: rank relabelling, stage refinement (the
    accumulation-expansion remark of Sec. 3), zero stages, step chunking;
  * the hand-built single-rank data stall of the Sec. 2 pattern.
"""
from __future__ import annotations

import itertools
import os

import numpy as np

MS = 1_000_000

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


# ----------------------------------------------------------------------------
# helpers that do not restate the frontier recursion


def load_golden(name: str) -> dict:
    """Parse one fixture of tests/golden (see the files for the format)."""
    rows, out = {}, {}
    with open(os.path.join(GOLDEN, name)) as fh:
        for line in fh:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            key, *vals = line.split()
            if key == "d":
                rows[int(vals[0])] = [int(v) for v in vals[1:]]
            elif key == "stages":
                out["stages"] = vals
            else:
                out[key] = [int(v) for v in vals]
    R = len(rows)
    # fixture rows are per rank; the oracle layout is [T][S][R]
    out["d"] = np.array([[rows[r] for r in range(R)]], dtype=np.int64).transpose(0, 2, 1).copy()
    return out


GOLDEN_FILES = ["motivating_example.txt", "frontier_figure.txt", "non_identifiable_pair.txt"]


def rank_totals(d):
    """[T, R] total duration of every rank (sum over all stages)."""
    return d.sum(axis=1)


def random_cases(seed=0):
    """A mix of tie-free and tie-heavy random inputs of several shapes."""
    rng = np.random.Generator(np.random.PCG64(seed))
    cases = []
    for (T, S, R) in [(50, 6, 8), (40, 3, 1), (30, 1, 5), (25, 12, 33), (20, 7, 64), (10, 5, 130)]:
        cases.append(rng.integers(0, 10**9, size=(T, S, R), dtype=np.int64))
        cases.append(rng.integers(0, 4, size=(T, S, R), dtype=np.int64))  # many ties
    return cases


def stall_case():
    """Hand-built single-rank data stall (Sec. 2 pattern) with four ranks.

    All ranks share the base stage durations (20, 60, 120, 2, 15, 3) ms of
    (data, fwd, bwd, callback, optim, other).  Rank 2's data stage is 30 ms
    late; ranks 0, 1 and 3 observe the same delay as 30 ms of backward wait.
    """
    base = np.array([20, 60, 120, 2, 15, 3], dtype=np.int64) * MS
    d = np.repeat(base[:, None], 4, axis=1)
    d[0, 2] += 30 * MS
    for r in (0, 1, 3):
        d[2, r] += 30 * MS
    return d[None].copy()


# ----------------------------------------------------------------------------
# frontier pins


def pin_golden(f):
    for name in GOLDEN_FILES:
        g = load_golden(name)
        inc, lead = f(g["d"])
        assert inc[0].tolist() == g["inc"], (name, inc[0].tolist())
        assert lead[0].tolist() == g["lead"], (name, lead[0].tolist())
        assert int(inc[0].sum()) == g["makespan"][0], name
        if "stage_max_total" in g:
            # the per-stage max baseline printed beside the frontier
            assert int(g["d"][0].max(axis=1).sum()) == g["stage_max_total"][0]


def pin_stall(f):
    """Sec. 2 pattern: the delay is charged once, to data, on the stalled
    rank; backward is not inflated by the wait of the other ranks."""
    d = stall_case()
    inc, lead = f(d)
    assert inc[0].tolist() == [50 * MS, 60 * MS, 120 * MS, 2 * MS, 15 * MS, 3 * MS], inc
    # data led by the stalled rank; from bwd on all four ranks tie at the
    # same prefix and the lowest index leads
    assert lead[0].tolist() == [2, 2, 0, 0, 0, 0], lead
    assert int(inc[0].sum()) == 250 * MS == int(rank_totals(d).max())
    # the naive per-stage max double counts the wait
    assert int(d[0].max(axis=1).sum()) == 280 * MS


def pin_telescoping(f):
    """Theorem 1 and a >= 0 (Sec. 3)."""
    for d in random_cases(1):
        inc, lead = f(d)
        assert inc.shape == d.shape[:2] and lead.shape == d.shape[:2]
        assert (inc >= 0).all()
        assert np.array_equal(inc.sum(axis=1), rank_totals(d).max(axis=1))


def pin_slack_identity(f):
    """Eq. (3): a[t,s] = max_r (d[t,r,s] - lambda[t,r,s]) with
    lambda[t,r,s] = F[t,s-1] - P[t,r,s-1]; every lambda >= 0."""
    for d in random_cases(2):
        inc, _ = f(d)
        T, S, R = d.shape
        F = np.cumsum(inc, axis=1)  # frontier from the function under test
        for t in range(T):
            P_prev = np.zeros(R, dtype=np.int64)
            F_prev = 0
            for s in range(S):
                lam = F_prev - P_prev
                assert (lam >= 0).all()
                assert inc[t, s] == (d[t, s] - lam).max()
                P_prev = P_prev + d[t, s]
                F_prev = F[t, s]


def pin_single_rank(f):
    """Sec. 3 edge case: with R = 1 the frontier is the rank's own vector."""
    rng = np.random.Generator(np.random.PCG64(3))
    d = rng.integers(0, 10**9, size=(17, 9, 1), dtype=np.int64)
    inc, lead = f(d)
    assert np.array_equal(inc, d[:, :, 0])
    assert (lead == 0).all()


def pin_props(f):
    """Propositions 1 and 2 (integer form) and their tight constructions
    (Appendix D)."""
    for d in random_cases(4):
        inc, _ = f(d)
        T, S, R = d.shape
        F = inc.sum(axis=1)
        M = d.max(axis=2).sum(axis=1)          # sum_s max_r d
        tot = d.sum(axis=(1, 2))               # R * mean-based summary
        assert (F <= M).all() and (M <= min(R, S) * F).all()
        assert (F <= tot).all() and (tot <= R * F).all()
    # Prop. 1 tight: D on min(R,S) distinct (rank, stage) pairs, one per rank
    for R, S in [(3, 5), (6, 4), (5, 5)]:
        D = 7 * MS
        d = np.zeros((1, S, R), dtype=np.int64)
        for k in range(min(R, S)):
            d[0, k, k] = D
        inc, _ = f(d)
        assert int(inc.sum()) == D
        assert int(d[0].max(axis=1).sum()) == min(R, S) * int(inc.sum())
    # Prop. 2 tight: one rank carries total D, the others zero
    R, S = 5, 4
    d = np.zeros((1, S, R), dtype=np.int64)
    d[0, :, 3] = [1 * MS, 2 * MS, 3 * MS, 4 * MS]
    inc, lead = f(d)
    assert int(inc.sum()) == 10 * MS == int(d.sum())
    assert lead[0].tolist() == [3, 3, 3, 3]


def pin_stability(f):
    """Appendix D: every duration moved by at most eps moves the frontier
    at 1-based boundary s by at most s*eps and the advance by at most
    (2s-1)*eps."""
    rng = np.random.Generator(np.random.PCG64(5))
    for (T, S, R) in [(40, 6, 8), (20, 12, 50)]:
        d = rng.integers(10**6, 10**8, size=(T, S, R), dtype=np.int64)
        for eps in (1, 1000, 10**6):
            e = rng.integers(-eps, eps + 1, size=d.shape, dtype=np.int64)
            inc0, _ = f(d)
            inc1, _ = f(d + e)
            F0, F1 = np.cumsum(inc0, axis=1), np.cumsum(inc1, axis=1)
            s1 = np.arange(1, S + 1)
            assert (np.abs(F1 - F0) <= s1 * eps).all()
            assert (np.abs(inc1 - inc0) <= (2 * s1 - 1) * eps).all()
            # the bound is reached: one rank's first stages all move by +eps
    d = np.zeros((1, 4, 2), dtype=np.int64) + 5 * MS
    e = np.zeros_like(d)
    e[0, :, 0] = 1000
    inc0, _ = f(d)
    inc1, _ = f(d + e)
    assert (np.cumsum(inc1 - inc0, axis=1) == 1000 * np.arange(1, 5)).all()


def _brute_prefix_max(case, R, S):
    """Largest total of the first s+1 stages over ranks, and the lowest rank
    reaching it, by summing each rank's stages from scratch."""
    inc, lead = [], []
    prev = 0
    for s in range(S):
        sums = [sum(case[j][r] for j in range(s + 1)) for r in range(R)]
        best = max(sums)
        inc.append(best - prev)
        lead.append(min(r for r in range(R) if sums[r] == best))
        prev = best
    return inc, lead


def pin_bruteforce(f):
    """Every d in {0,1,2}^(S x R) for four small shapes."""
    for (R, S) in [(2, 2), (2, 3), (3, 2), (3, 3)]:
        cases = list(itertools.product(range(3), repeat=R * S))
        d = np.array(cases, dtype=np.int64).reshape(len(cases), S, R)
        inc, lead = f(d)
        for i, flat in enumerate(cases):
            case = [list(flat[s * R:(s + 1) * R]) for s in range(S)]
            ei, el = _brute_prefix_max(case, R, S)
            assert inc[i].tolist() == ei, (R, S, case)
            assert lead[i].tolist() == el, (R, S, case)


def pin_permutation(f):
    """Relabelling ranks permutes leaders where the leader is unique; at a
    tie the leader is the lowest relabelled index of the tie set."""
    rng = np.random.Generator(np.random.PCG64(6))
    for d in random_cases(7):
        T, S, R = d.shape
        perm = rng.permutation(R)            # new rank k holds old rank perm[k]
        inv = np.argsort(perm)               # old rank r becomes inv[r]
        inc0, lead0 = f(d)
        inc1, lead1 = f(d[:, :, perm])
        assert np.array_equal(inc0, inc1)
        P = np.cumsum(d, axis=1)
        for t in range(T):
            for s in range(S):
                ties = np.flatnonzero(P[t, s] == P[t, s].max())
                assert lead0[t, s] == ties.min()
                assert lead1[t, s] == inv[ties].min()


def pin_structure(f):
    """Stage refinement, zero stages, constant shifts, scaling, step order
    and step chunking (steps are independent, Sec. 3)."""
    rng = np.random.Generator(np.random.PCG64(8))
    d = rng.integers(0, 10**7, size=(30, 6, 11), dtype=np.int64)
    inc, lead = f(d)
    # refinement: split stage 2 into two consecutive sub-stages on every rank
    frac = rng.integers(0, 10**7, size=(30, 11), dtype=np.int64)
    part = np.minimum(frac, d[:, 2])
    dr = np.concatenate([d[:, :2], part[:, None], (d[:, 2] - part)[:, None], d[:, 3:]], axis=1)
    ir, lr = f(dr)
    assert np.array_equal(ir[:, 2] + ir[:, 3], inc[:, 2])
    assert np.array_equal(np.delete(ir, [2, 3], axis=1), np.delete(inc, 2, axis=1))
    assert np.array_equal(lr[:, 3], lead[:, 2])
    # appending a zero stage: zero advance, leader of the last boundary kept
    dz = np.concatenate([d, np.zeros((30, 1, 11), dtype=np.int64)], axis=1)
    iz, lz = f(dz)
    assert (iz[:, -1] == 0).all() and np.array_equal(lz[:, -1], lead[:, -1])
    # adding c to stage 4 on every rank adds c to that advance only
    dc = d.copy()
    dc[:, 4] += 12345
    ic, lc = f(dc)
    expect = inc.copy()
    expect[:, 4] += 12345
    assert np.array_equal(ic, expect) and np.array_equal(lc, lead)
    # scaling every duration scales every advance
    i3, l3 = f(3 * d)
    assert np.array_equal(i3, 3 * inc) and np.array_equal(l3, lead)
    # steps are independent: reversing steps reverses results
    ib, lb = f(d[::-1].copy())
    assert np.array_equal(ib, inc[::-1]) and np.array_equal(lb, lead[::-1])
    # chunks concatenate
    i1, l1 = f(d[:13])
    i2, l2 = f(d[13:])
    assert np.array_equal(np.concatenate([i1, i2]), inc)
    assert np.array_equal(np.concatenate([l1, l2]), lead)


def pin_twin(f, pyref):
    """Agreement with the pure-Python statement on small random inputs."""
    for d in random_cases(9):
        small = d[:6]
        inc, lead = f(small)
        pi, pl = pyref.frontier(small.tolist())
        assert inc.tolist() == pi and lead.tolist() == pl


FRONTIER_PINS = [pin_golden, pin_stall, pin_telescoping, pin_slack_identity,
                 pin_single_rank, pin_props, pin_stability, pin_bruteforce,
                 pin_permutation, pin_structure]


# ----------------------------------------------------------------------------
# window-summary pins


def _expected_counts(lead, R, t0, t1):
    """Leader histogram of steps [t0, t1) per stage with np.bincount."""
    S = lead.shape[1]
    out = np.zeros((S, R), dtype=np.int64)
    for s in range(S):
        v = lead[t0:t1, s]
        v = v[(v >= 0) & (v < R)]
        out[s] = np.bincount(v, minlength=R)[:R]
    return out


def pin_summary_mass(f, g):
    """Counts sum to the window length; exposed totals sum to the window's
    exposed makespan (Theorem 1 summed over the window); the last window
    is the remainder."""
    for d in random_cases(10):
        T, S, R = d.shape
        inc, lead = f(d)
        for window in (1, 7, T, T + 3):
            ex, cnt, top2 = g(inc, lead, R, window)
            W = -(-T // window)
            assert ex.shape == (W, S) and cnt.shape == (W, S, R) and top2.shape == (W, 2, 2)
            for w in range(W):
                t0, t1 = w * window, min((w + 1) * window, T)
                assert (cnt[w].sum(axis=1) == t1 - t0).all()
                assert int(ex[w].sum()) == int(rank_totals(d[t0:t1]).max(axis=1).sum())
                assert np.array_equal(ex[w], inc[t0:t1].sum(axis=0))
                assert np.array_equal(cnt[w], _expected_counts(lead, R, t0, t1))


def pin_summary_top2(f, g):
    """Top-2 routing on constructed windows: order by exposed total, lower
    stage on ties; modal leader, lower rank on ties, -1 with no leader."""
    R = 4
    # one window of 6 steps, S = 4; exposed totals (5, 9, 9, 1) by construction
    inc = np.array([[5, 9, 9, 1]] + [[0, 0, 0, 0]] * 5, dtype=np.int64)
    lead = np.array([[0, 1, 3, 0],
                     [0, 2, 3, 0],
                     [1, 2, 0, 0],
                     [1, 1, 0, 0],
                     [2, 3, 0, 0],
                     [2, 3, 0, 0]], dtype=np.int32)
    ex, cnt, top2 = g(inc, lead, R, 6)
    assert ex.tolist() == [[5, 9, 9, 1]]
    # stage 1 (tie with 2 at 9 -> lower index) counts r1:2 r2:2 r3:2 -> r1
    # stage 2 counts r0:4 r3:2 -> r0
    assert top2.tolist() == [[[1, 1], [2, 0]]]
    # S = 1: the second pair is padding
    ex, cnt, top2 = g(np.array([[3], [4]], dtype=np.int64), np.array([[2], [2]], dtype=np.int32), 3, 5)
    assert top2.tolist() == [[[0, 2], [-1, -1]]]
    # all-zero exposed: stages 0 and 1; leaders outside [0, R) are not counted
    inc = np.zeros((3, 3), dtype=np.int64)
    lead = np.array([[-1, 5, 0], [7, 1, 0], [-2, 1, 0]], dtype=np.int32)
    ex, cnt, top2 = g(inc, lead, 2, 3)
    assert cnt[0].tolist() == [[0, 0], [0, 2], [3, 0]]
    assert top2.tolist() == [[[0, -1], [1, 1]]]
    # the stall case routes to the data stage and the stalled rank
    d = np.repeat(stall_case(), 10, axis=0)
    d[5:, 0, 2] -= 30 * MS          # the stall on only half of the steps
    d[5:, 2, [0, 1, 3]] -= 30 * MS
    inc, lead = f(d)
    ex, cnt, top2 = g(inc, lead, 4, 10)
    # data: the stalled rank leads the 5 stalled steps; the 5 clean steps
    # are four-way ties that go to rank 0
    assert cnt[0, 0].tolist() == [5, 0, 5, 0]
    assert ex[0, 0] == 5 * 50 * MS + 5 * 20 * MS
    # bwd is a four-way tie on every step: never charged to the waiting ranks
    assert cnt[0, 2].tolist() == [10, 0, 0, 0]
    assert ex[0, 2] == 10 * 120 * MS


def pin_summary_bruteforce(f, g):
    """Every leader pattern of a tiny window set against bincount."""
    R, S, T = 2, 2, 3
    inc = np.arange(T * S, dtype=np.int64).reshape(T, S) * 3 + 1
    for flat in itertools.product(range(R), repeat=T * S):
        lead = np.array(flat, dtype=np.int32).reshape(T, S)
        for window in (1, 2, 3):
            ex, cnt, top2 = g(inc, lead, R, window)
            for w in range(-(-T // window)):
                t0, t1 = w * window, min((w + 1) * window, T)
                c = _expected_counts(lead, R, t0, t1)
                assert np.array_equal(cnt[w], c)
                e = inc[t0:t1].sum(axis=0)
                order = np.lexsort((np.arange(S), -e))
                for k in range(2):
                    sk = int(order[k])
                    rk = int(np.argmax(c[sk])) if c[sk].max() > 0 else -1
                    assert top2[w, k].tolist() == [sk, rk]


def pin_summary_twin(f, g, pyref):
    for d in random_cases(11):
        small = d[:9]
        T, S, R = small.shape
        inc, lead = f(small)
        for window in (2, 4, 9):
            ex, cnt, top2 = g(inc, lead, R, window)
            pe, pc, pt = pyref.window_summary(inc.tolist(), lead.tolist(), R, window)
            assert ex.tolist() == pe and cnt.tolist() == pc and top2.tolist() == pt


SUMMARY_PINS = [pin_summary_mass, pin_summary_top2, pin_summary_bruteforce]


# ----------------------------------------------------------------------------
# exposed time led per (window, stage, rank): every advance goes to the rank
# that attains the frontier (the leader)


def pin_lead_golden(f, le):
    """The printed worked examples: the whole advance of each boundary goes
    to its leader, in one window."""
    for name in GOLDEN_FILES:
        g = load_golden(name)
        d = g["d"]
        inc, lead = f(d)
        T, S, R = d.shape
        out, _ = le(inc, lead, R, T)
        want = np.zeros((1, S, R), dtype=np.int64)
        for s, (a, r) in enumerate(zip(g["inc"], g["lead"])):
            want[0, s, r] = a
        assert np.array_equal(out, want), name


def pin_lead_stall(f, le):
    """The Sec. 2 stall on half of ten steps: the data stage's exposed time
    goes to the stalled rank for the stalled steps (50 ms each) and to rank 0
    for the clean four-way ties (20 ms each); backward never goes to the
    waiting ranks.  By count the data stage is a 5-5 tie that goes to rank
    0; by exposed time led it goes to the stalled rank."""
    d = np.repeat(stall_case(), 10, axis=0)
    d[5:, 0, 2] -= 30 * MS
    d[5:, 2, [0, 1, 3]] -= 30 * MS
    inc, lead = f(d)
    out, top2 = le(inc, lead, 4, 10)
    assert out[0, 0].tolist() == [5 * 20 * MS, 0, 5 * 50 * MS, 0]
    assert out[0, 2].tolist() == [10 * 120 * MS, 0, 0, 0]
    # stage totals: bwd 1200 ms, fwd 600 ms, data 350 ms
    assert top2[0].tolist() == [[2, 0], [1, 0]]
    # with the step time of the model stages cut, data becomes the top stage
    d2 = d.copy()
    d2[:, 1:3] //= 10
    inc2, lead2 = f(d2)
    _, top2 = le(inc2, lead2, 4, 10)
    assert top2[0, 0].tolist() == [0, 2]


def pin_lead_single_rank(f, le):
    """R = 1: every advance is the rank's own duration (Sec. 3), so the
    single rank holds the window sums of its durations."""
    d = random_cases(13)[0][:, :, :1].copy()
    T, S, _ = d.shape
    inc, lead = f(d)
    for window in (1, 4, T):
        out, top2 = le(inc, lead, 1, window)
        for w in range(-(-T // window)):
            t0, t1 = w * window, min((w + 1) * window, T)
            assert np.array_equal(out[w, :, 0], d[t0:t1, :, 0].sum(axis=0))
            for k in range(2):
                assert top2[w, k, 1] == (0 if out[w, top2[w, k, 0], 0] > 0 else -1)


def pin_lead_mass_and_support(f, le):
    """Per window and stage the ranks' shares add up to the stage's exposed
    total, and by Theorem 1 over all stages to the window's exposed
    makespan; shares are nonnegative, and only ranks that led the stage at
    some step of the window hold any.  Windows add up."""
    for d in random_cases(14):
        T, S, R = d.shape
        inc, lead = f(d)
        for window in (1, 5, T, T + 2):
            out, _ = le(inc, lead, R, window)
            assert out.shape == (-(-T // window), S, R)
            assert (out >= 0).all()
            for w in range(out.shape[0]):
                t0, t1 = w * window, min((w + 1) * window, T)
                assert np.array_equal(out[w].sum(axis=1), inc[t0:t1].sum(axis=0))
                assert int(out[w].sum()) == int(rank_totals(d[t0:t1]).max(axis=1).sum())
                for s in range(S):
                    led = set(lead[t0:t1, s].tolist())
                    assert all(r in led for r in np.nonzero(out[w, s])[0].tolist())
        if T >= 4:
            whole, _ = le(inc, lead, R, T)
            halves, _ = le(inc, lead, R, -(-T // 2))
            assert np.array_equal(halves.sum(axis=0), whole[0])


def pin_lead_relabel(f, le):
    """Relabelling the ranks (tie-free data) relabels the shares and the
    suspect ranks."""
    rng = np.random.Generator(np.random.PCG64(15))
    d = rng.integers(0, 10**9, size=(12, 5, 7), dtype=np.int64)
    perm = rng.permutation(7)
    inc, lead = f(d)
    inc2, lead2 = f(d[:, :, perm])
    a, ta = le(inc, lead, 7, 4)
    b, tb = le(inc2, lead2, 7, 4)
    # new rank j is old rank perm[j]
    assert np.array_equal(b, a[:, :, perm])
    assert np.array_equal(tb[:, :, 0], ta[:, :, 0])
    assert np.array_equal(perm[tb[:, :, 1]], ta[:, :, 1])


def pin_lead_counts_and_bincount(f, le):
    """Against the leader counts and numpy: with every advance of a stage
    equal to c the share is c times the rank's count, and in general it is
    numpy's weighted bincount of the leaders; leaders outside [0, R) count
    nowhere.  The suspects are the two stages of largest window total
    (numpy lexsort, lower stage first on ties), each with numpy's first
    argmax of its shares (-1 when every share is 0).  Brute force over
    every leader pattern of a tiny window set."""
    R, S, T = 3, 2, 4
    inc = np.arange(T * S, dtype=np.int64).reshape(T, S) * 5 + 2
    for flat in itertools.product(range(-1, R + 1), repeat=T * S // 2):
        lead = np.array(flat + flat, dtype=np.int32).reshape(T, S)
        for window in (1, 3, 4):
            out, top2 = le(inc, lead, R, window)
            for w in range(-(-T // window)):
                t0, t1 = w * window, min((w + 1) * window, T)
                for s in range(S):
                    v = lead[t0:t1, s]
                    keep = (v >= 0) & (v < R)
                    want = np.bincount(v[keep], weights=inc[t0:t1, s][keep], minlength=R)[:R]
                    assert np.array_equal(out[w, s], want.astype(np.int64))
                e = inc[t0:t1].sum(axis=0)
                order = np.lexsort((np.arange(S), -e))
                for k in range(2):
                    sk = int(order[k])
                    rk = int(np.argmax(out[w, sk])) if out[w, sk].max() > 0 else -1
                    assert top2[w, k].tolist() == [sk, rk]
    c = np.full((T, S), 7, dtype=np.int64)
    lead = np.array([[0, 2], [2, 2], [0, 1], [0, 0]], dtype=np.int32)
    assert np.array_equal(le(c, lead, R, T)[0][0], 7 * _expected_counts(lead, R, 0, T))


def pin_lead_top2_cases(f, le, g):
    """Constructed windows: the count-modal rank and the rank that led the
    most exposed time differ when few long advances outweigh many short
    ones; with equal advances they agree with the window summary's top-2
    (every stage and rank, ties included); S = 1 pads; zero totals give
    rank -1."""
    R = 4
    # stage 0: rank 1 leads 4 steps of 1, rank 3 leads 2 steps of 10
    # (total 24); stage 1: ranks 2 and 0 each lead 3 steps of 5 (total 30)
    inc = np.array([[1, 5], [1, 5], [10, 5], [1, 5], [10, 5], [1, 5]], dtype=np.int64)
    lead = np.array([[1, 2], [1, 0], [3, 2], [1, 0], [3, 2], [1, 0]], dtype=np.int32)
    out, top2 = le(inc, lead, R, 6)
    assert out[0].tolist() == [[0, 4, 0, 20], [15, 0, 15, 0]]
    assert top2.tolist() == [[[1, 0], [0, 3]]]
    _, _, t_count = g(inc, lead, R, 6)
    assert t_count.tolist() == [[[1, 0], [0, 1]]]
    # equal advances per stage: same picks as the count-based top-2
    for d in random_cases(17):
        T, S, R = d.shape
        _, lead = f(d)
        cinc = np.tile(np.arange(S, dtype=np.int64)[::-1] % 3 + 1, (T, 1))
        for window in (3, T):
            _, tw = le(cinc, lead, R, window)
            _, _, tc = g(cinc, lead, R, window)
            assert np.array_equal(tw, tc)
    # S = 1 pads the second pair; zero advances lead to no rank
    _, top2 = le(np.array([[0], [0]], dtype=np.int64), np.array([[1], [1]], dtype=np.int32), 2, 2)
    assert top2.tolist() == [[[0, -1], [-1, -1]]]
    _, top2 = le(np.array([[3], [4]], dtype=np.int64), np.array([[2], [2]], dtype=np.int32), 3, 5)
    assert top2.tolist() == [[[0, 2], [-1, -1]]]


def pin_lead_twin(f, le, pyref):
    for d in random_cases(16):
        small = d[:9]
        T, S, R = small.shape
        inc, lead = f(small)
        for window in (2, 4, 9):
            out, top2 = le(inc, lead, R, window)
            po, pt = pyref.window_lead_exposed(inc.tolist(), lead.tolist(), R, window)
            assert out.tolist() == po and top2.tolist() == pt


LEAD_PINS = [pin_lead_golden, pin_lead_stall, pin_lead_single_rank, pin_lead_mass_and_support,
             pin_lead_relabel, pin_lead_counts_and_bincount]


# ----------------------------------------------------------------------------
# leader switches between confident unique leaders (Sec. 4 localization
# evidence)


def _switches_by_runs(lead, gap, ties, window, min_gap):
    """The definition restated through runs: in each window the qualifying
    leaders of a stage, in step order, form maximal runs of equal ranks; the
    switches are the runs minus one (0 when nothing qualifies)."""
    T, S = lead.shape
    W = -(-T // window)
    sw = np.zeros((W, S), dtype=np.int64)
    el = np.zeros((W, S), dtype=np.int64)
    for w in range(W):
        for s in range(S):
            seq = [int(lead[t, s]) for t in range(w * window, min((w + 1) * window, T))
                   if ties[t, s] == 1 and (gap[t, s] >= min_gap or gap[t, s] < 0)]
            runs = len([k for k, _ in itertools.groupby(seq)])
            el[w, s] = len(seq)
            sw[w, s] = max(runs - 1, 0)
    return sw, el


def pin_switch_stall(e, sw):
    """The Sec. 2 stall on every other step of ten: the stalled steps have a
    unique data leader 30 ms ahead of the other three ranks, the clean steps
    are four-way ties and never qualify.  One stalled rank: no switch; the
    stall alternating between ranks 1 and 2: a switch at every qualifying
    step after the first; a gap threshold above 30 ms: nothing qualifies."""
    d = np.repeat(stall_case(), 10, axis=0)
    d[1::2, 0, 2] -= 30 * MS           # clean on odd steps
    d[1::2, 2, [0, 1, 3]] -= 30 * MS
    ev = e(d)
    n, el = sw(ev["lead"], ev["gap"], ev["ties"], 10, 0)
    assert el[0, 0] == 5 and n[0, 0] == 0
    # backward: a four-way tie at every step (also where the wait absorbs
    # the stall), so nothing qualifies
    assert el[0, 2] == 0 and n[0, 2] == 0
    d2 = d.copy()
    for t in (2, 6):                   # the stall moves to rank 1 there
        d2[t, 0, 2] -= 30 * MS
        d2[t, 0, 1] += 30 * MS
        d2[t, 2, 2] += 30 * MS
        d2[t, 2, 1] -= 30 * MS
    ev2 = e(d2)
    n2, el2 = sw(ev2["lead"], ev2["gap"], ev2["ties"], 10, 0)
    assert ev2["lead"][::2, 0].tolist() == [2, 1, 2, 1, 2]
    assert el2[0, 0] == 5 and n2[0, 0] == 4
    # two windows of five steps: the seam between them drops one switch
    n5, el5 = sw(ev2["lead"], ev2["gap"], ev2["ties"], 5, 0)
    assert el5[:, 0].tolist() == [3, 2] and n5[:, 0].tolist() == [2, 1]
    n3, el3 = sw(ev2["lead"], ev2["gap"], ev2["ties"], 10, 30 * MS + 1)
    assert el3[0, 0] == 0 and n3[0, 0] == 0
    n4, el4 = sw(ev2["lead"], ev2["gap"], ev2["ties"], 10, 30 * MS)
    assert el4[0, 0] == 5 and n4[0, 0] == 4


def pin_switch_runs(e, sw):
    """Against the run-count restatement on random evidence arrays (ties and
    gaps drawn so that about half the boundaries qualify), several windows
    and thresholds, and against numpy's diff on the qualifying leaders."""
    rng = np.random.Generator(np.random.PCG64(18))
    for (T, S) in [(1, 1), (7, 3), (50, 6), (129, 2), (300, 12)]:
        lead = rng.integers(0, 4, size=(T, S), dtype=np.int32)
        ties = rng.choice(np.array([1, 1, 1, 2, 3], dtype=np.int32), size=(T, S))
        gap = np.where(ties == 1, rng.integers(-1, 100, size=(T, S)), 0).astype(np.int64)
        for window in (1, 4, 7, T, T + 5):
            for min_gap in (0, 1, 50, 99, 100):
                n, el = sw(lead, gap, ties, window, min_gap)
                rn, rel = _switches_by_runs(lead, gap, ties, window, min_gap)
                assert np.array_equal(n, rn) and np.array_equal(el, rel)
                for w in range(n.shape[0]):
                    t0, t1 = w * window, min((w + 1) * window, T)
                    for s in range(S):
                        m = (ties[t0:t1, s] == 1) & ((gap[t0:t1, s] >= min_gap) | (gap[t0:t1, s] < 0))
                        q = lead[t0:t1, s][m]
                        assert n[w, s] == np.count_nonzero(np.diff(q))
                        assert el[w, s] == m.sum()


def pin_switch_bruteforce(e, sw):
    """Every leader pattern in {0,1,2}^6 with every qualifying mask of one
    stage: the switches are the boundaries where the qualifying leader
    changes, counted by hand."""
    T = 6
    for flat in itertools.product(range(3), repeat=T):
        lead = np.array(flat, dtype=np.int32).reshape(T, 1)
        for mask in range(1 << T):
            q = np.array([(mask >> t) & 1 for t in range(T)], dtype=bool).reshape(T, 1)
            ties = np.where(q, 1, 2).astype(np.int32)
            gap = np.where(q, 5, 0).astype(np.int64)
            n, el = sw(lead, gap, ties, 3, 1)
            for w in range(2):
                chosen = [flat[t] for t in range(3 * w, 3 * w + 3) if q[t, 0]]
                want = sum(1 for i in range(1, len(chosen)) if chosen[i] != chosen[i - 1])
                assert n[w, 0] == want and el[w, 0] == len(chosen)


def pin_switch_invariants(e, sw):
    """R = 1 qualifies every boundary (no runner-up) and never switches;
    switches < eligible whenever something qualifies; relabelling the
    leaders changes nothing; a larger threshold never adds qualifying
    boundaries; at threshold 0 every unique leader qualifies; windows add up
    in the eligible counts, and joining windows adds at most one switch per
    seam."""
    for d in random_cases(19):
        T, S, R = d.shape
        ev = e(d)
        lead, gap, ties = ev["lead"], ev["gap"], ev["ties"]
        n, el = sw(lead, gap, ties, T, 0)
        if R == 1:
            assert (el == T).all() and (n == 0).all()
        assert np.array_equal(el[0], (ties == 1).sum(axis=0))
        assert ((n < el) | ((n == 0) & (el == 0))).all()
        perm = np.random.Generator(np.random.PCG64(R)).permutation(R).astype(np.int32)
        n2, el2 = sw(perm[lead], gap, ties, T, 0)
        assert np.array_equal(n, n2) and np.array_equal(el, el2)
        prev = el
        for g in (1, 10, 10**6, 10**9):
            _, elg = sw(lead, gap, ties, T, g)
            assert (elg <= prev).all()
            prev = elg
        if T >= 4:
            half = -(-T // 2)
            nh, elh = sw(lead, gap, ties, half, 0)
            assert np.array_equal(elh.sum(axis=0), el[0])
            assert (nh.sum(axis=0) <= n[0]).all() and (n[0] <= nh.sum(axis=0) + 1).all()


def pin_switch_twin(e, sw, pyref):
    for d in random_cases(21):
        small = d[:12]
        ev = e(small)
        T, S, _ = small.shape
        for window, min_gap in ((3, 0), (5, 7), (12, 10**8)):
            n, el = sw(ev["lead"], ev["gap"], ev["ties"], window, min_gap)
            pn, pel = pyref.window_leader_switches(ev["lead"].tolist(), ev["gap"].tolist(),
                                                   ev["ties"].tolist(), window, min_gap)
            assert n.tolist() == pn and el.tolist() == pel


SWITCH_PINS = [pin_switch_stall, pin_switch_runs, pin_switch_bruteforce, pin_switch_invariants]


# ----------------------------------------------------------------------------
# localization evidence and per-stage baselines (Sec. 4; Props. 1-2)
#
# Each pin takes ``e(d) -> dict`` with [T, S] arrays inc, lead, gap, ties,
# stage_max, stage_sum.


def _as_frontier(e):
    def f(d):
        out = e(d)
        return out["inc"], out["lead"]
    return f


def pin_ev_frontier_part(e):
    """The frontier part of the evidence pass meets every frontier pin."""
    f = _as_frontier(e)
    for pin in FRONTIER_PINS:
        pin(f)


def pin_ev_golden(e):
    g = load_golden("motivating_example.txt")
    out = e(g["d"])
    assert out["stage_max"][0].tolist() == g["stage_max"]
    assert int(out["stage_max"][0].sum()) == g["stage_max_total"][0]


def pin_ev_stall(e):
    """The Sec. 2 pattern: a 30 ms margin at data and fwd, then a four-way
    tie; the per-stage max of bwd counts the wait (150 ms)."""
    out = e(stall_case())
    assert out["gap"][0].tolist() == [30 * MS, 30 * MS, 0, 0, 0, 0]
    assert out["ties"][0].tolist() == [1, 1, 4, 4, 4, 4]
    assert out["stage_max"][0].tolist() == [50 * MS, 60 * MS, 150 * MS, 2 * MS, 15 * MS, 3 * MS]
    assert out["stage_sum"][0].tolist() == [110 * MS, 240 * MS, 570 * MS, 8 * MS, 60 * MS, 12 * MS]


def pin_ev_bruteforce(e):
    """Every d in {0,1,2}^(S x R) for four small shapes: prefixes summed
    from scratch, sorted; the gap is the difference of the two largest, the
    tie count the multiplicity of the largest."""
    for (R, S) in [(2, 2), (2, 3), (3, 2), (3, 3)]:
        cases = list(itertools.product(range(3), repeat=R * S))
        d = np.array(cases, dtype=np.int64).reshape(len(cases), S, R)
        out = e(d)
        for i, flat in enumerate(cases):
            case = [list(flat[s * R:(s + 1) * R]) for s in range(S)]
            for s in range(S):
                sums = sorted((sum(case[j][r] for j in range(s + 1)) for r in range(R)), reverse=True)
                assert out["gap"][i, s] == sums[0] - sums[1], (case, s)
                assert out["ties"][i, s] == sums.count(sums[0]), (case, s)
                assert out["stage_max"][i, s] == max(case[s])
                assert out["stage_sum"][i, s] == sum(case[s])


def pin_ev_props(e):
    """Props. 1 and 2 on the baselines this pass reports, with the tight
    constructions of Appendix D."""
    for d in random_cases(12):
        out = e(d)
        T, S, R = d.shape
        F = out["inc"].sum(axis=1)
        M = out["stage_max"].sum(axis=1)
        tot = out["stage_sum"].sum(axis=1)                     # = R * Mbar
        assert (F <= M).all() and (M <= min(R, S) * F).all()
        assert (F <= tot).all() and (tot <= R * F).all()
        assert np.array_equal(out["stage_sum"], d.sum(axis=2))    # library sum
        assert np.array_equal(out["stage_max"], d.max(axis=2))    # library max
    for R, S in [(3, 5), (6, 4)]:
        d = np.zeros((1, S, R), dtype=np.int64)
        for k in range(min(R, S)):
            d[0, k, k] = 9 * MS
        out = e(d)
        assert int(out["stage_max"].sum()) == min(R, S) * int(out["inc"].sum())
    d = np.zeros((1, 4, 5), dtype=np.int64)
    d[0, :, 2] = [1 * MS, 2 * MS, 3 * MS, 4 * MS]
    out = e(d)
    assert int(out["stage_sum"].sum()) == int(out["inc"].sum())  # Mbar = F / R
    assert out["gap"][0].tolist() == [1 * MS, 3 * MS, 6 * MS, 10 * MS]


def pin_ev_invariants(e):
    """Relabelling ranks leaves the evidence unchanged; gap 0 exactly at
    ties; R = 1 has no runner-up."""
    rng = np.random.Generator(np.random.PCG64(13))
    for d in random_cases(14):
        T, S, R = d.shape
        out = e(d)
        assert (out["ties"] >= 1).all()
        if R >= 2:
            assert (out["gap"] >= 0).all()
            assert np.array_equal(out["gap"] == 0, out["ties"] >= 2)
        else:
            assert (out["gap"] == -1).all() and (out["ties"] == 1).all()
        perm = rng.permutation(R)
        out2 = e(d[:, :, perm])
        for k in ("inc", "gap", "ties", "stage_max", "stage_sum"):
            assert np.array_equal(out[k], out2[k]), k


def pin_ev_twin(e, pyref):
    for d in random_cases(15):
        small = d[:5]
        out = e(small)
        ref = pyref.frontier_evidence(small.tolist())
        for k, v in ref.items():
            assert out[k].tolist() == v, k


EVIDENCE_PINS = [pin_ev_frontier_part, pin_ev_golden, pin_ev_stall, pin_ev_bruteforce,
                 pin_ev_props, pin_ev_invariants]


# ----------------------------------------------------------------------------
# ingest (Appendix A closure) and routing candidate set (Sec. 4)
#
# ingest pins take ``g(x[R,T,K], w[R,T]) -> (d[T,K+1,R], o[T,R])``; route pins
# take ``c(exposed[W,S], num, den) -> (order[W,S], size[W])``.


def pin_ingest_closure(g):
    """Appendix A: the residual is max(0, e), the overlap max(0, -e), with
    e = w - (explicit stages); so the stages minus the overlap give back w,
    and residual and overlap are never both positive."""
    rng = np.random.Generator(np.random.PCG64(30))
    for (R, T, K) in [(1, 5, 1), (3, 7, 5), (8, 40, 5), (33, 9, 11)]:
        x = rng.integers(0, 10**6, size=(R, T, K), dtype=np.int64)
        w = x.sum(axis=2) + rng.integers(-3 * 10**5, 3 * 10**5, size=(R, T), dtype=np.int64)
        w[0, 0] = x[0, 0].sum()          # exact closure: both zero
        d, o = g(x, w)
        assert d.shape == (T, K + 1, R) and o.shape == (T, R)
        assert np.array_equal(d[:, :K, :], x.transpose(1, 2, 0))    # library transpose
        assert np.array_equal(d.sum(axis=1) - o, w.T)
        assert (d[:, K, :] >= 0).all() and (o >= 0).all()
        assert not ((d[:, K, :] > 0) & (o > 0)).any()
        assert d[0, K, 0] == 0 and o[0, 0] == 0


def pin_ingest_roundtrip(g):
    """A [T][S][R] matrix whose last stage is the residual of the others comes
    back unchanged from its per-rank explicit stages and rank totals."""
    rng = np.random.Generator(np.random.PCG64(31))
    d0 = rng.integers(0, 10**7, size=(20, 6, 13), dtype=np.int64)
    x = d0[:, :5, :].transpose(2, 0, 1).copy()
    w = d0.sum(axis=1).T.copy()
    d, o = g(x, w)
    assert np.array_equal(d, d0) and (o == 0).all()


def pin_ingest_twin(g, pyref):
    rng = np.random.Generator(np.random.PCG64(32))
    x = rng.integers(0, 100, size=(4, 6, 3), dtype=np.int64)
    w = rng.integers(0, 400, size=(4, 6), dtype=np.int64)
    d, o = g(x, w)
    pd, po = pyref.ingest(x.tolist(), w.tolist())
    assert d.tolist() == pd and o.tolist() == po


def _route_by_lexsort(ex, num, den):
    order = np.lexsort((np.arange(len(ex)), -ex))
    cum = np.concatenate([[0], np.cumsum(ex[order])])
    need = num * int(ex.sum())
    k = next(i for i in range(len(ex) + 1) if i == len(ex) or den * int(cum[i]) >= need)
    return order, k


def pin_route_definition(c):
    """Sec. 4: the smallest leading-share prefix reaching tau, on constructed
    windows and against a sort by numpy's lexsort with a cumulative sum."""
    ex = np.array([[50, 30, 15, 5], [5, 5, 5, 5], [0, 0, 0, 0], [10, 0, 0, 0],
                   [1, 2, 3, 4], [7, 9, 9, 1]], dtype=np.int64)
    order, size = c(ex, 4, 5)
    assert size.tolist() == [2, 4, 0, 1, 3, 3]
    assert order[5].tolist() == [1, 2, 0, 3]                 # tie 9/9: lower stage first
    rng = np.random.Generator(np.random.PCG64(33))
    for S in (1, 2, 6, 12, 40):
        ex = rng.integers(0, 5, size=(30, S), dtype=np.int64) * rng.integers(1, 10**6)
        for num, den in ((4, 5), (7, 10), (9, 10), (1, 1), (0, 1), (1, 3)):
            order, size = c(ex, num, den)
            for w in range(len(ex)):
                eo, ek = _route_by_lexsort(ex[w], num, den)
                assert order[w].tolist() == eo.tolist() and size[w] == ek


def pin_route_properties(c):
    """Larger tau never shrinks the set; tau = 0 gives the empty set; tau = 1
    reaches every stage with nonzero exposure; the first two stages are the
    top-2 stages."""
    rng = np.random.Generator(np.random.PCG64(34))
    ex = rng.integers(0, 10**6, size=(50, 8), dtype=np.int64)
    ex[::5, 3:] = 0
    sizes = [c(ex, n, 10)[1] for n in range(11)]
    for a, b in zip(sizes, sizes[1:]):
        assert (a <= b).all()
    assert (sizes[0] == 0).all()
    assert np.array_equal(sizes[10], (ex > 0).sum(axis=1))
    order, _ = c(ex, 4, 5)
    for w in range(len(ex)):
        first = int(np.argmax(ex[w]))
        assert order[w, 0] == first


def pin_route_bruteforce(c):
    """Every exposure vector in {0,1,2,3}^4 at tau 4/5 and 1/2."""
    vecs = np.array(list(itertools.product(range(4), repeat=4)), dtype=np.int64)
    for num, den in ((4, 5), (1, 2)):
        order, size = c(vecs, num, den)
        for i, ex in enumerate(vecs):
            best = None
            for k in range(5):
                for subset in itertools.combinations(range(4), k):
                    if den * int(ex[list(subset)].sum()) >= num * int(ex.sum()):
                        best = k
                        break
                if best is not None:
                    break
            # the smallest subset of any stages equals the smallest leading prefix
            assert size[i] == best, (ex, num, den)


def pin_route_twin(c, pyref):
    rng = np.random.Generator(np.random.PCG64(35))
    ex = rng.integers(0, 6, size=(40, 5), dtype=np.int64)
    order, size = c(ex, 4, 5)
    po, ps = pyref.route(ex.tolist(), 4, 5)
    assert order.tolist() == po and size.tolist() == ps


INGEST_PINS = [pin_ingest_closure, pin_ingest_roundtrip]
ROUTE_PINS = [pin_route_definition, pin_route_properties, pin_route_bruteforce]


# ----------------------------------------------------------------------------
# direct-exposure gain, Eq. (4)
#
# Pins take ``x(d[T,S,R], btilde[W,S,R], window) -> dict`` with gain [T,S],
# makespan [T], window_gain [W,S], window_makespan [W].

_BASE6 = np.array([20, 60, 120, 2, 15, 3], dtype=np.int64) * MS


def _gain_by_numpy(d, btilde, window):
    """F[t,S] is the largest rank total (Theorem 1); replacing stage s by
    min(d, btilde) changes each rank's total only through that stage."""
    T, S, R = d.shape
    F = d.sum(axis=1).max(axis=1)
    gain = np.empty((T, S), dtype=np.int64)
    for t in range(T):
        b = btilde[t // window]
        for s in range(S):
            m = d[t].copy()
            m[s] = np.minimum(m[s], b[s])
            gain[t, s] = F[t] - m.sum(axis=0).max()
    return F, gain


def pin_gain_sync_wait(x):
    """Sec. 4: the Sec. 2 stall has a large data share but no single-stage
    gain against a no-stall baseline, because the other ranks' wait stays in
    place when only one stage is replaced."""
    d = stall_case()
    bt = np.repeat(_BASE6[:, None], 4, axis=1)[None]
    out = x(d, bt, 1)
    assert out["gain"][0].tolist() == [0] * 6
    assert out["makespan"][0] == 250 * MS


def pin_gain_direct(x):
    """A delay no other rank waits for is directly exposed: replacing that
    stage removes it from the makespan."""
    d = np.repeat(np.repeat(_BASE6[:, None], 4, axis=1)[None], 3, axis=0)
    d[:, 4, 1] += 50 * MS                      # rank 1's optimizer, every step
    d[1, 0, 3] += 7 * MS                       # and a small data delay on step 1
    bt = np.repeat(_BASE6[:, None], 4, axis=1)[None]
    out = x(d, bt, 3)
    assert out["gain"].tolist() == [[0, 0, 0, 0, 50 * MS, 0],
                                    [0, 0, 0, 0, 43 * MS, 0],
                                    [0, 0, 0, 0, 50 * MS, 0]]
    assert out["makespan"].tolist() == [270 * MS, 270 * MS, 270 * MS]
    assert out["window_gain"][0].tolist() == [0, 0, 0, 0, 143 * MS, 0]
    assert out["window_makespan"].tolist() == [810 * MS]


def pin_gain_bounds(x):
    """0 <= gain <= the largest reduction of any rank at that stage; a
    baseline at or above every duration gives 0; a zero baseline removes the
    stage; window sums are the sums of the steps."""
    rng = np.random.Generator(np.random.PCG64(40))
    for (T, S, R, window) in [(20, 6, 8, 7), (9, 3, 1, 4), (12, 12, 33, 12), (5, 2, 64, 1)]:
        d = rng.integers(0, 10**6, size=(T, S, R), dtype=np.int64)
        W = -(-T // window)
        bt = rng.integers(0, 10**6, size=(W, S, R), dtype=np.int64)
        out = x(d, bt, window)
        F, g = _gain_by_numpy(d, bt, window)
        assert np.array_equal(out["makespan"], F) and np.array_equal(out["gain"], g)
        for t in range(T):
            red = np.maximum(0, d[t] - bt[t // window]).max(axis=1)
            assert (out["gain"][t] >= 0).all() and (out["gain"][t] <= red).all()
        for w in range(W):
            sl = slice(w * window, min(T, (w + 1) * window))
            assert np.array_equal(out["window_gain"][w], out["gain"][sl].sum(axis=0))
            assert out["window_makespan"][w] == out["makespan"][sl].sum()
        hi = np.full_like(bt, 10**7)
        assert (x(d, hi, window)["gain"] == 0).all()
        zero = np.zeros_like(bt)
        gz = x(d, zero, window)["gain"]
        tot = d.sum(axis=1)
        for s in range(S):
            assert np.array_equal(gz[:, s], F - (tot - d[:, s]).max(axis=1))


def pin_gain_bruteforce(x):
    """Every d and btilde in {0,1,2}^(S x R) for R = S = 2 (6561 pairs)."""
    R, S = 2, 2
    mats = np.array(list(itertools.product(range(3), repeat=R * S)), dtype=np.int64).reshape(-1, S, R)
    n = len(mats)
    d = np.repeat(mats, n, axis=0)
    bt = np.tile(mats, (n, 1, 1))
    out = x(d, bt, 1)
    F = d.sum(axis=1).max(axis=1)
    for s in range(S):
        m = d.copy()
        m[:, s] = np.minimum(d[:, s], bt[:, s])
        assert np.array_equal(out["gain"][:, s], F - m.sum(axis=1).max(axis=1))


def pin_gain_twin(x, pyref):
    rng = np.random.Generator(np.random.PCG64(41))
    d = rng.integers(0, 50, size=(7, 4, 5), dtype=np.int64)
    bt = rng.integers(0, 50, size=(3, 4, 5), dtype=np.int64)
    out = x(d, bt, 3)
    ref = pyref.exposure_gain(d.tolist(), bt.tolist(), 3)
    for k, v in ref.items():
        assert out[k].tolist() == v, k


GAIN_PINS = [pin_gain_sync_wait, pin_gain_direct, pin_gain_bounds, pin_gain_bruteforce]


# ----------------------------------------------------------------------------
# lag of the frontier over the median rank (Sec. 4)
#
# Pins take ``l(d[T,S,R]) -> (lag[T,S], lag_inc[T,S])``.


def pin_lag_stall(l):
    """The Sec. 2 pattern: the stalled rank opens a 30 ms lag at data that
    closes (-30 ms increment) at bwd, where the others' wait levels them."""
    lag, inc = l(stall_case())
    assert lag[0].tolist() == [30 * MS, 30 * MS, 0, 0, 0, 0]
    assert inc[0].tolist() == [30 * MS, 0, -30 * MS, 0, 0, 0]


def pin_lag_library_median(l):
    """Odd R: numpy's median; even R: the lower middle of numpy's sort."""
    rng = np.random.Generator(np.random.PCG64(50))
    for (T, S, R) in [(20, 6, 7), (15, 5, 8), (10, 4, 1), (8, 3, 2), (6, 12, 129), (5, 6, 1000),
                      (12, 4, 3)]:
        for hi in (10**9, 3):
            d = rng.integers(0, hi + 1, size=(T, S, R), dtype=np.int64)
            lag, inc = l(d)
            P = np.cumsum(d, axis=1)
            F = P.max(axis=2)
            if R % 2:
                med = np.median(P, axis=2).astype(np.int64)
            else:
                med = np.sort(P, axis=2)[:, :, (R - 1) // 2]
            assert np.array_equal(lag, F - med)
            assert np.array_equal(np.cumsum(inc, axis=1), lag)
            assert (lag >= 0).all()
            if R == 1:
                assert (lag == 0).all()
            if R == 2:
                assert np.array_equal(lag, P.max(axis=2) - P.min(axis=2))


def pin_lag_invariants(l):
    """Relabelling ranks and adding one constant to a stage of every rank
    leave the lag unchanged; scaling scales it."""
    rng = np.random.Generator(np.random.PCG64(51))
    d = rng.integers(0, 10**6, size=(30, 6, 33), dtype=np.int64)
    lag, inc = l(d)
    lag2, _ = l(d[:, :, rng.permutation(33)])
    assert np.array_equal(lag, lag2)
    dc = d.copy()
    dc[:, 3] += 777
    assert np.array_equal(l(dc)[0], lag)
    assert np.array_equal(l(5 * d)[0], 5 * lag)


def pin_lag_bruteforce(l):
    """Every d in {0,1,2}^(S x R) for (R, S) in {(3, 2), (4, 2), (2, 3)}."""
    for (R, S) in [(3, 2), (4, 2), (2, 3)]:
        cases = list(itertools.product(range(3), repeat=R * S))
        d = np.array(cases, dtype=np.int64).reshape(len(cases), S, R)
        lag, inc = l(d)
        for i, flat in enumerate(cases):
            prev = 0
            for s in range(S):
                sums = sorted(sum(flat[j * R + r] for j in range(s + 1)) for r in range(R))
                L = sums[-1] - sums[(R - 1) // 2]
                assert lag[i, s] == L and inc[i, s] == L - prev
                prev = L


def pin_lag_twin(l, pyref):
    rng = np.random.Generator(np.random.PCG64(52))
    d = rng.integers(0, 20, size=(6, 5, 9), dtype=np.int64)
    lag, inc = l(d)
    pl, pi = pyref.frontier_lag(d.tolist())
    assert lag.tolist() == pl and inc.tolist() == pi


LAG_PINS = [pin_lag_stall, pin_lag_library_median, pin_lag_invariants, pin_lag_bruteforce]


# ----------------------------------------------------------------------------
# raw rank spread (Sec. 6.2) and the per-rank window median (Eq. (4))
#
# Spread pins take ``sp(d[T,S,R], window) -> (spread[T,S], wspread[W,S])``;
# window-median pins take ``wm(d[T,S,R], window) -> med[W,S,R]``.


def _lower_median_by_count(xs):
    """The lower median of ``xs`` from its defining property, without
    sorting: the value m with #{x < m} <= k < #{x <= m}, k = (n-1)//2."""
    k = (len(xs) - 1) // 2
    for m in xs:
        if sum(x < m for x in xs) <= k < sum(x <= m for x in xs):
            return m
    raise AssertionError("no lower median")


def _window_sums(x, window):
    T = x.shape[0]
    return np.stack([x[t0:t0 + window].sum(axis=0) for t0 in range(0, T, window)])


def pin_spread_stall(sp):
    """The Sec. 2 pattern, by hand: at data the stalled rank is 30 ms above
    the median of the four ranks; at bwd the three waiting ranks are 30 ms
    above the stalled one, but they are the median, so the spread is 0."""
    spread, wspread = sp(stall_case(), 1)
    assert spread[0].tolist() == [30 * MS, 0, 0, 0, 0, 0]
    assert wspread.tolist() == spread.tolist()


def pin_spread_library(sp):
    """numpy's max and median (odd R) or the lower middle of numpy's sort
    (even R); window sums by numpy."""
    rng = np.random.Generator(np.random.PCG64(60))
    for (T, S, R, window) in [(20, 6, 7, 5), (15, 5, 8, 4), (10, 4, 1, 3), (8, 3, 2, 8),
                              (6, 12, 129, 1), (5, 6, 1000, 2), (13, 4, 3, 20)]:
        for hi in (10**9, 3):
            d = rng.integers(0, hi + 1, size=(T, S, R), dtype=np.int64)
            spread, wspread = sp(d, window)
            if R % 2:
                med = np.median(d, axis=2).astype(np.int64)
            else:
                med = np.sort(d, axis=2)[:, :, (R - 1) // 2]
            assert np.array_equal(spread, d.max(axis=2) - med)
            assert np.array_equal(wspread, _window_sums(spread, window))
            assert (spread >= 0).all()
            if R == 1:
                assert (spread == 0).all()
            if R == 2:
                assert np.array_equal(spread, d.max(axis=2) - d.min(axis=2))


def pin_spread_first_boundary_is_lag(sp, l):
    """At the first boundary a rank's prefix is its duration, so the spread
    of stage 0 equals the lag of stage 0; with S = 1 they agree everywhere."""
    rng = np.random.Generator(np.random.PCG64(61))
    d = rng.integers(0, 10**6, size=(25, 5, 31), dtype=np.int64)
    spread, _ = sp(d, 7)
    lag, _ = l(d)
    assert np.array_equal(spread[:, 0], lag[:, 0])
    assert np.array_equal(sp(d[:, :1], 7)[0], l(d[:, :1])[0])


def pin_spread_invariants(sp):
    """Relabelling ranks, adding one constant to every rank of a stage, and
    reordering stages act as they must; scaling scales."""
    rng = np.random.Generator(np.random.PCG64(62))
    d = rng.integers(0, 10**6, size=(30, 6, 33), dtype=np.int64)
    spread, wspread = sp(d, 10)
    assert np.array_equal(sp(d[:, :, rng.permutation(33)], 10)[0], spread)
    dc = d.copy()
    dc[:, 2] += 12345
    assert np.array_equal(sp(dc, 10)[0], spread)
    order = rng.permutation(6)
    assert np.array_equal(sp(d[:, order], 10)[0], spread[:, order])
    assert np.array_equal(sp(3 * d, 10)[0], 3 * spread)
    assert np.array_equal(sp(d, 1)[1], spread)
    assert np.array_equal(sp(d, 1000)[1][0], spread.sum(axis=0))


def pin_spread_bruteforce(sp):
    """Every row in {0,1,2,3}^R for R in 1..5, the median by its counting
    definition."""
    for R in range(1, 6):
        rows = list(itertools.product(range(4), repeat=R))
        d = np.array(rows, dtype=np.int64).reshape(len(rows), 1, R)
        spread, _ = sp(d, 1)
        for i, row in enumerate(rows):
            assert spread[i, 0] == max(row) - _lower_median_by_count(list(row))


def pin_spread_twin(sp, pyref):
    rng = np.random.Generator(np.random.PCG64(63))
    d = rng.integers(0, 20, size=(7, 5, 9), dtype=np.int64)
    spread, wspread = sp(d, 3)
    ps, pw = pyref.rank_spread(d.tolist(), 3)
    assert spread.tolist() == ps and wspread.tolist() == pw


SPREAD_PINS = [pin_spread_stall, pin_spread_library, pin_spread_invariants, pin_spread_bruteforce]


def pin_median_identity_window(wm):
    """A window of one step: the median is the step itself."""
    rng = np.random.Generator(np.random.PCG64(70))
    d = rng.integers(0, 10**9, size=(9, 4, 5), dtype=np.int64)
    assert np.array_equal(wm(d, 1), d)


def pin_median_library(wm):
    """numpy's median over each window's steps (odd n) or the lower middle
    of numpy's sort (even n), the last window shorter."""
    rng = np.random.Generator(np.random.PCG64(71))
    for (T, S, R, window) in [(21, 3, 5, 7), (20, 2, 4, 8), (7, 3, 6, 100), (50, 1, 3, 2),
                              (30, 4, 17, 10), (11, 2, 2, 3)]:
        d = rng.integers(0, 10**9, size=(T, S, R), dtype=np.int64)
        med = wm(d, window)
        W = (T + window - 1) // window
        assert med.shape == (W, S, R)
        for w in range(W):
            blk = d[w * window:(w + 1) * window]
            n = blk.shape[0]
            want = (np.median(blk, axis=0).astype(np.int64) if n % 2
                    else np.sort(blk, axis=0)[(n - 1) // 2])
            assert np.array_equal(med[w], want), (T, window, w)


def pin_median_invariants(wm):
    """Reordering the steps inside a window leaves its medians unchanged;
    a shift or a positive scale of the data moves them alike; a constant
    series is its own median; the median lies within the window's range."""
    rng = np.random.Generator(np.random.PCG64(72))
    d = rng.integers(0, 10**6, size=(40, 3, 6), dtype=np.int64)
    med = wm(d, 10)
    perm = np.concatenate([w * 10 + rng.permutation(10) for w in range(4)])
    assert np.array_equal(wm(d[perm], 10), med)
    assert np.array_equal(wm(d + 999, 10), med + 999)
    assert np.array_equal(wm(7 * d, 10), 7 * med)
    c = np.full((12, 2, 3), 42, dtype=np.int64)
    assert (wm(c, 5) == 42).all()
    blocks = d.reshape(4, 10, 3, 6)
    assert (med >= blocks.min(axis=1)).all() and (med <= blocks.max(axis=1)).all()


def pin_median_bruteforce(wm):
    """Every sequence in {0,1,2,3}^n for n in 1..6 (one stage, one rank), the
    median by its counting definition."""
    for n in range(1, 7):
        seqs = list(itertools.product(range(4), repeat=n))
        for seq in seqs:
            d = np.array(seq, dtype=np.int64).reshape(n, 1, 1)
            assert wm(d, n)[0, 0, 0] == _lower_median_by_count(list(seq))


def pin_median_twin(wm, pyref):
    rng = np.random.Generator(np.random.PCG64(73))
    d = rng.integers(0, 30, size=(11, 3, 4), dtype=np.int64)
    assert wm(d, 4).tolist() == pyref.window_median(d.tolist(), 4)


MEDIAN_PINS = [pin_median_identity_window, pin_median_library, pin_median_invariants,
               pin_median_bruteforce]


# ----------------------------------------------------------------------------
# range status of the data contract (Sec. 3: d >= 0; prefixes below 2^47)
#
# Pins take ``rs(d[T,S,R]) -> 0 or 2``.

LIMIT = 1 << 47


def pin_range_edges(rs):
    """The bound is exclusive, on prefixes as well as on single durations."""
    z = np.zeros((2, 3, 4), dtype=np.int64)
    assert rs(z) == 0
    d = z.copy(); d[1, 2, 3] = -1
    assert rs(d) == 2                                   # one negative duration
    d = z.copy(); d[0, 0, 0] = LIMIT - 1
    assert rs(d) == 0                                   # largest allowed prefix
    d = z.copy(); d[0, 0, 0] = LIMIT
    assert rs(d) == 2                                   # one duration at the bound
    d = z.copy(); d[0, :, 2] = [LIMIT // 2, LIMIT // 4, LIMIT // 4 - 1]
    assert rs(d) == 0                                   # a prefix of 2^47 - 1
    d[0, 2, 2] += 1
    assert rs(d) == 2                                   # the same prefix reaching 2^47
    d = z.copy(); d[:, :, 1] = LIMIT // 3               # each step's prefix is 3 * floor(2^47 / 3)
    assert rs(d) == 0                                   # steps are separate: no carry across steps
    d = z.copy(); d[0, 0, 0] = np.iinfo(np.int64).max
    assert rs(d) == 2
    d = z.copy(); d[0, 0, 0] = np.iinfo(np.int64).min
    assert rs(d) == 2


def pin_range_library(rs):
    """numpy's cumulative sums (exact here: every value is small or the
    first prefix already crosses) and sign test on random inputs."""
    rng = np.random.Generator(np.random.PCG64(80))
    for _ in range(40):
        T, S, R = rng.integers(1, 6, size=3)
        d = rng.integers(0, 1 << 46, size=(T, S, R), dtype=np.int64)
        if rng.random() < 0.3:
            d[rng.integers(T), rng.integers(S), rng.integers(R)] = -int(rng.integers(1, 10))
        want = 2 if ((d < 0).any() or (np.cumsum(np.maximum(d, 0), axis=1) >= LIMIT).any()) else 0
        assert rs(d) == want


def pin_range_twin(rs, pyref):
    rng = np.random.Generator(np.random.PCG64(81))
    for _ in range(20):
        d = rng.integers(-2, 1 << 45, size=(3, 6, 5), dtype=np.int64)
        assert rs(d) == pyref.range_status(d.tolist())


RANGE_PINS = [pin_range_edges, pin_range_library]
