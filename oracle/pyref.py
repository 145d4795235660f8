"""Pure-Python statement of frontier accounting, for tiny inputs.

TEST INFRASTRUCTURE ONLY (same rules as the rest of ``oracle``).  It restates
the definitions of Sec. 3 (Eq. (1), Eq. (2)) and the top-2 routing of Sec. 4
as literal Python loops over lists, with the same readings as
``sf_oracle.c``, so that the C oracle can be cross-checked on small inputs by
a second, independently written statement.
"""
from __future__ import annotations


def _prefix_matrix(step):
    """``P[s][r] = sum_{j<=s} step[j][r]`` (Eq. (1)), row by row."""
    P = []
    for s, row in enumerate(step):
        P.append([(P[s - 1][r] if s else 0) + x for r, x in enumerate(row)])
    return P


def frontier(d):
    """``d[t][s][r]`` nested lists of ints -> ``(inc[t][s], lead[t][s])``.

    Eq. (1) per step: the prefix matrix, then the frontier of every boundary
    with its lowest leader, then the differences of the frontier."""
    inc, lead = [], []
    for step in d:
        P = _prefix_matrix(step)
        F = [max(row) for row in P]
        lead.append([row.index(f) for row, f in zip(P, F)])  # first (lowest) rank attaining F
        inc.append([f - (F[s - 1] if s else 0) for s, f in enumerate(F)])
    return inc, lead


def window_summary(inc, lead, R, window):
    """Returns ``(exposed[w][s], counts[w][s][r], top2[w][k][2])``."""
    T = len(inc)
    S = len(inc[0]) if T else 0
    W = (T + window - 1) // window
    exposed, counts, top2 = [], [], []
    for w in range(W):
        steps = range(w * window, min((w + 1) * window, T))
        ex_w = [sum(inc[t][s] for t in steps) for s in range(S)]
        c_w = [[sum(1 for t in steps if lead[t][s] == r) for r in range(R)]
               for s in range(S)]
        order = sorted(range(S), key=lambda s: (-ex_w[s], s))
        picks = order[:2] + [-1] * (2 - len(order[:2]))
        t2 = []
        for sk in picks:
            if sk < 0:
                t2.append([-1, -1])
                continue
            m = max(c_w[sk])
            t2.append([sk, c_w[sk].index(m) if m > 0 else -1])
        exposed.append(ex_w)
        counts.append(c_w)
        top2.append(t2)
    return exposed, counts, top2


def window_lead_exposed(inc, lead, R, window):
    """Returns ``(lead_exposed[w][s][r], top2[w][k][2])``: per window and
    stage, the advances whose leader is rank r, summed (leaders outside
    [0, R) not counted); the top-2 stages by window total, each with the rank
    that led the most exposed time (lowest on ties, -1 if none led any)."""
    T = len(inc)
    S = len(inc[0]) if T else 0
    W = (T + window - 1) // window
    out, top2 = [], []
    for w in range(W):
        steps = range(w * window, min((w + 1) * window, T))
        le_w = [[sum(inc[t][s] for t in steps if lead[t][s] == r) for r in range(R)]
                for s in range(S)]
        totals = [sum(inc[t][s] for t in steps) for s in range(S)]
        order = sorted(range(S), key=lambda s: (-totals[s], s))
        picks = order[:2] + [-1] * (2 - len(order[:2]))
        t2 = []
        for sk in picks:
            if sk < 0:
                t2.append([-1, -1])
                continue
            m = max(le_w[sk])
            t2.append([sk, le_w[sk].index(m) if m > 0 else -1])
        out.append(le_w)
        top2.append(t2)
    return out, top2


def window_leader_switches(lead, gap, ties, window, min_gap=0):
    """Returns ``(switches[w][s], eligible[w][s])``: per window and stage,
    the qualifying boundaries (a single rank at the frontier, ahead by at
    least min_gap, or with no runner-up) and how often their leader changes
    from one qualifying boundary to the next."""
    T = len(lead)
    S = len(lead[0]) if T else 0
    W = (T + window - 1) // window
    switches, eligible = [], []
    for w in range(W):
        sw_w, el_w = [], []
        for s in range(S):
            seq = [lead[t][s] for t in range(w * window, min((w + 1) * window, T))
                   if ties[t][s] == 1 and (gap[t][s] >= min_gap or gap[t][s] < 0)]
            el_w.append(len(seq))
            sw_w.append(sum(1 for a, b in zip(seq, seq[1:]) if a != b))
        switches.append(sw_w)
        eligible.append(el_w)
    return switches, eligible


def frontier_evidence(d):
    """``d[t][s][r]`` -> dict of [t][s] lists: inc, lead, gap, ties,
    stage_max, stage_sum (same readings as the C oracle), in the order of
    ``frontier``: prefix matrix, per-boundary quantities, differences."""
    out = {k: [] for k in ("inc", "lead", "gap", "ties", "stage_max", "stage_sum")}
    for step in d:
        P = _prefix_matrix(step)
        F = [max(row) for row in P]
        leaders = [row.index(f) for row, f in zip(P, F)]
        gaps = []
        for row, L in zip(P, leaders):
            others = sorted(row[:L] + row[L + 1:])
            gaps.append(row[L] - others[-1] if others else -1)
        out["lead"].append(leaders)
        out["gap"].append(gaps)
        out["ties"].append([row.count(f) for row, f in zip(P, F)])
        out["stage_max"].append([max(x) for x in step])
        out["stage_sum"].append([sum(x) for x in step])
        out["inc"].append([f - (F[s - 1] if s else 0) for s, f in enumerate(F)])
    return out


def ingest(x, w):
    """``x[r][t][k]``, ``w[r][t]`` -> ``(d[t][s][r], o[t][r])`` with the
    residual stage appended last (Appendix A)."""
    R = len(x)
    T = len(x[0]) if R else 0
    K = len(x[0][0]) if T else 0
    d = [[[0] * R for _ in range(K + 1)] for _ in range(T)]
    o = [[0] * R for _ in range(T)]
    for r in range(R):
        for t in range(T):
            for k in range(K):
                d[t][k][r] = x[r][t][k]
            e = w[r][t] - sum(x[r][t])
            d[t][K][r] = max(0, e)
            o[t][r] = max(0, -e)
    return d, o


def route(exposed, tau_num=4, tau_den=5):
    """Stage order by (exposed desc, stage asc) and the smallest prefix size
    whose exposed sum reaches tau_num / tau_den of the total."""
    order, size = [], []
    for ex in exposed:
        ordw = sorted(range(len(ex)), key=lambda s: (-ex[s], s))
        total = sum(ex)
        k, cum = 0, 0
        while k < len(ex) and tau_den * cum < tau_num * total:
            cum += ex[ordw[k]]
            k += 1
        order.append(ordw)
        size.append(k)
    return order, size


def exposure_gain(d, btilde, window):
    """Eq. (4) on nested lists: d[t][s][r], btilde[w][s][r] -> dict of
    gain[t][s], makespan[t], window_gain[w][s], window_makespan[w]."""
    def last_frontier(step):
        return max(sum(step[s][r] for s in range(len(step))) for r in range(len(step[0])))

    T = len(d)
    S = len(d[0]) if T else 0
    W = (T + window - 1) // window
    out = {"gain": [], "makespan": [], "window_gain": [[0] * S for _ in range(W)],
           "window_makespan": [0] * W}
    for t, step in enumerate(d):
        w = t // window
        F = last_frontier(step)
        g = []
        for s in range(S):
            m = [row[:] for row in step]
            m[s] = [min(v, b) for v, b in zip(step[s], btilde[w][s])]
            g.append(F - last_frontier(m))
            out["window_gain"][w][s] += g[-1]
        out["gain"].append(g)
        out["makespan"].append(F)
        out["window_makespan"][w] += F
    return out


def frontier_lag(d):
    """d[t][s][r] -> (lag[t][s], lag_inc[t][s]) with the lower median."""
    lag, inc = [], []
    for step in d:
        R = len(step[0])
        P = [0] * R
        prev = 0
        lt, it = [], []
        for row in step:
            P = [p + v for p, v in zip(P, row)]
            srt = sorted(P)
            L = srt[-1] - srt[(R - 1) // 2]
            lt.append(L)
            it.append(L - prev)
            prev = L
        lag.append(lt)
        inc.append(it)
    return lag, inc


def rank_spread(d, window):
    """d[t][s][r] -> (spread[t][s], window sums[w][s]): max minus lower
    median over ranks (Sec. 6.2)."""
    spread = [[max(row) - sorted(row)[(len(row) - 1) // 2] for row in step] for step in d]
    T, S = len(d), len(d[0]) if d else 0
    W = (T + window - 1) // window
    wsum = [[0] * S for _ in range(W)]
    for t in range(T):
        for s in range(S):
            wsum[t // window][s] += spread[t][s]
    return spread, wsum


def window_median(d, window):
    """d[t][s][r] -> med[w][s][r]: lower median over each window's steps
    (the per-rank window-median baseline of Eq. (4))."""
    T = len(d)
    S, R = len(d[0]), len(d[0][0])
    out = []
    for t0 in range(0, T, window):
        steps = d[t0:t0 + window]
        out.append([[sorted(st[s][r] for st in steps)[(len(steps) - 1) // 2] for r in range(R)]
                    for s in range(S)])
    return out


def range_status(d):
    """2 if some duration is negative or some prefix reaches 2**47, else 0."""
    for step in d:
        P = [0] * len(step[0])
        for row in step:
            for r, x in enumerate(row):
                if x < 0:
                    return 2
                P[r] += x
                if P[r] >= 1 << 47:
                    return 2
    return 0
