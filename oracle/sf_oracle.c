/*
 * sf_oracle.c -- reference CPU statement of StageFrontier frontier
 * accounting.  TEST INFRASTRUCTURE ONLY: nothing in the product library
 * calls, links or includes this file.  It exists so that the tests, the
 * smoke check and the CPU baseline of the benchmark have an obviously
 * correct answer to compare the GPU path against.
 *
 * The method is exact (no approximation, heuristic or iteration), so this
 * file is its definition written out as nested loops, in signed int64
 * nanoseconds, in the paper's order of operations:
 *
 *   Sec. 3, Eq. (1):  P[t,r,s] = sum_{j<=s} d[t,r,j]
 *                     F[t,s]   = max_r P[t,r,s]
 *                     a[t,s]   = F[t,s] - F[t,s-1],  F[t,0] = 0 (1-based s)
 *   Each step is independent (Sec. 3 processes steps one at a time); per
 *   step the oracle forms P, then F and the leaders, then the advances.
 *   Sec. 3, Eq. (2):  the window share numerator sum_{t in window} a[t,s].
 *   Sec. 4: top-2 routing = the two stages with the highest shares.
 *   Sec. 4, localization evidence: the tie set of the frontier and the gap
 *   between the largest and the second-largest prefix at each boundary.
 *   Appendix A, closure: with rank-local step wall time w[t,r] and the
 *   explicit stage durations, e = w - sum of the explicit stages, the
 *   residual stage is max(0, e) and the overlap error max(0, -e).
 *   Sec. 4, routing candidate set: the smallest prefix of stages, ordered by
 *   share, whose cumulative share reaches tau_C.
 *   Sec. 4, lag: L[t,s] = max_r P[t,r,s] - median_r P[t,r,s] and its
 *   increment L[t,s] - L[t,s-1] (L[t,-1] = 0, like F).
 *   Sec. 4, Eq. (4), direct exposure: replace stage s on every rank by the
 *   clipped baseline b = min(d, btilde), recompute the frontier, and take
 *   F[t,S] - F^(s<-b)[t,S]; G_s is its window sum over the window sum of
 *   F[t,S].
 *   Sec. 3, Props. 1 and 2: the per-stage max and mean baselines
 *   M_t = sum_s max_r d and Mbar_t = sum_s (1/R) sum_r d, kept per stage as
 *   max_r d[t,r,s] and sum_r d[t,r,s].
 *   Sec. 6.2, raw rank spread (a dispersion baseline scored on the same
 *   window matrix): max_r d[t,r,s] - median_r d[t,r,s], summed over the
 *   steps of a window.
 *   Sec. 4, Eq. (4), per-rank window median: a candidate baseline btilde,
 *   the median over the steps of a window of d[t,r,s], per stage and rank.
 *   Sec. 3 and Sec. 4, rank attribution: every advance a[t,s] is
 *   attributed to the rank attaining the frontier (the leader); per window,
 *   stage and rank, the exposed time that rank led is the sum of the
 *   window's advances of that stage whose leader is that rank; the top-2
 *   suspects weighted this way pair the two stages of the window summary
 *   with the rank that led the most exposed time of each.
 *   Sec. 4 and App. C, leader switches: per window and stage, the number
 *   of times the leader changes between consecutive confident unique
 *   leaders (boundaries whose frontier is attained by one rank only, ahead
 *   of the runner-up by at least a caller-given gap), and how many
 *   boundaries qualify.
 *   Sec. 3, the data contract: durations are nonnegative; with the
 *   library's packed keys every prefix must also stay below 2^47 ns.  The
 *   range status is 2 (SF_ERANGE) when some d < 0 or some prefix of
 *   nonnegative durations reaches 2^47, else 0.
 *
 * Readings where the paper leaves a choice open (each is a reading of the
 * paper, not a statement it makes):
 *   - leader = lowest rank index attaining F (the paper reports a tie set);
 *   - the leader is emitted and counted at every boundary, also where a = 0;
 *   - top-2 orders stages by the exposed window total (equivalently by the
 *     share, whose denominator is common), lower stage index on ties, and
 *     pairs each with its most frequent leader, lower rank on ties, -1 when
 *     that stage has no counted leader;
 *   - W = ceil(T / window); the last window may be shorter;
 *   - leaders outside [0, R) are not counted;
 *   - the gap is F minus the second-largest prefix over ranks (0 when two or
 *     more ranks attain F); with R = 1 there is no runner-up and the gap
 *     is -1.
 *
 *   - the gathered per-rank buffers are [R][T][K] (each rank's steps, each
 *     step's K explicit stages) and the residual is appended as the last
 *     stage, S = K + 1, as in the default stage taxonomy;
 *   - the baseline btilde of Eq. (4) is given per window, per stage and per
 *     rank ([W][S][R]), which covers a per-rank window median, a cohort
 *     median or a no-stall reference; the library returns the numerators
 *     and the denominator of G_s as int64 sums, never their quotient;
 *   - the median of the lag is the lower median, the element of rank
 *     floor((R - 1) / 2) in ascending order (the middle element for odd R;
 *     the lower middle for even R, which keeps the lag integer); the raw
 *     rank spread and the window median take the lower median likewise
 *     (over ranks, and over the n steps of a window: rank floor((n-1)/2));
 *   - the routing set orders stages like top-2 (exposed total descending,
 *     lower stage first) and compares shares exactly: k stages suffice when
 *     tau_den * (their exposed sum) >= tau_num * (window total);
 *   - a boundary's leader is confident and unique when its tie-set size is
 *     1 and its gap is at least min_gap (a gap of -1, R = 1, has no
 *     runner-up and qualifies); switches are counted between consecutive
 *     qualifying boundaries of the same stage inside one window (each
 *     window starts afresh), and the paper's switch-rate gates, whose
 *     values it does not state, are left to the caller.
 *
 * Layout: d is [T][S][R] (rank fastest), increments, leaders, gaps and tie
 * counts [T][S], switch and eligible counts [W][S],
 * exposed [W][S], counts and exposed time led [W][S][R], top2 [W][2][2],
 * route order [W][S] and route size [W].
 *
 * Parity status: every function here is pinned by the CPU test suite
 * (printed worked examples, closed forms, brute force); see tests/.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* Frontier advances and leaders, Eq. (1), taken in the order the equation
 * defines them, one step at a time:
 *   (i)   the rank-local prefix matrix P[s][r] = sum_{j<=s} d[t][j][r], each
 *         row the previous row plus the stage's durations;
 *   (ii)  the frontier F[s] = max_r P[s][r], then the leader: the lowest rank
 *         whose prefix equals F[s];
 *   (iii) the advances a[s] = F[s] - F[s-1], with F[-1] = 0 (the paper's
 *         F_{t,0} = 0 in 1-based stages).
 * Returns 0, or -1 if scratch cannot be allocated. */
int sfo_frontier(const int64_t* d, int64_t T, int32_t R, int32_t S,
                 int64_t* inc, int32_t* lead)
{
    int64_t* P = (int64_t*)calloc((size_t)S * (size_t)R, sizeof(int64_t));
    int64_t* F = (int64_t*)malloc(sizeof(int64_t) * (size_t)S);
    if (!P || !F) {
        free(P);
        free(F);
        return -1;
    }
    for (int64_t t = 0; t < T; ++t) {
        const int64_t* m = d + t * S * (int64_t)R; /* d[t][s][r] = m[s * R + r] */
        /* (i) the prefix matrix of the step */
        for (int32_t s = 0; s < S; ++s)
            for (int32_t r = 0; r < R; ++r)
                P[(int64_t)s * R + r] = (s > 0 ? P[(int64_t)(s - 1) * R + r] : 0) + m[(int64_t)s * R + r];
        /* (ii) the frontier of every boundary and its lowest leader */
        for (int32_t s = 0; s < S; ++s) {
            const int64_t* row = P + (int64_t)s * R;
            int64_t best = row[0];
            for (int32_t r = 1; r < R; ++r)
                if (row[r] > best) best = row[r];
            F[s] = best;
            int32_t L = -1;
            for (int32_t r = 0; r < R && L < 0; ++r)
                if (row[r] == best) L = r;
            lead[t * S + s] = L;
        }
        /* (iii) the advances */
        for (int32_t s = 0; s < S; ++s) inc[t * S + s] = F[s] - (s > 0 ? F[s - 1] : 0);
    }
    free(P);
    free(F);
    return 0;
}

/* Window reduction of per-step results: Eq. (2) numerators, leader counts
 * and top-2 routing. */
void sfo_window_summary(const int64_t* inc, const int32_t* lead,
                        int64_t T, int32_t R, int32_t S, int64_t window,
                        int64_t* exposed, int32_t* counts, int32_t* top2)
{
    int64_t W = (T + window - 1) / window;
    for (int64_t w = 0; w < W; ++w) {
        int64_t t0 = w * window;
        int64_t t1 = t0 + window < T ? t0 + window : T;

        for (int32_t s = 0; s < S; ++s) {
            int64_t sum = 0;
            for (int64_t t = t0; t < t1; ++t) sum += inc[t * S + s];
            exposed[w * S + s] = sum;

            int32_t* c = counts + (w * S + s) * (int64_t)R;
            for (int32_t r = 0; r < R; ++r) c[r] = 0;
            for (int64_t t = t0; t < t1; ++t) {
                int32_t r = lead[t * S + s];
                if (r >= 0 && r < R) c[r] += 1;
            }
        }

        /* first stage: largest exposed, lower index on ties */
        int32_t s1 = 0;
        for (int32_t s = 1; s < S; ++s)
            if (exposed[w * S + s] > exposed[w * S + s1]) s1 = s;
        /* second stage: same rule among the remaining stages */
        int32_t s2 = -1;
        for (int32_t s = 0; s < S; ++s) {
            if (s == s1) continue;
            if (s2 < 0 || exposed[w * S + s] > exposed[w * S + s2]) s2 = s;
        }

        int32_t pick[2] = {s1, s2};
        for (int k = 0; k < 2; ++k) {
            int32_t sk = pick[k];
            int32_t rk = -1;
            if (sk >= 0) {
                const int32_t* c = counts + (w * S + sk) * (int64_t)R;
                int32_t best = 0;
                for (int32_t r = 0; r < R; ++r) {
                    if (c[r] > best) {
                        best = c[r];
                        rk = r;
                    }
                }
            }
            top2[w * 4 + 2 * k + 0] = sk;
            top2[w * 4 + 2 * k + 1] = rk;
        }
    }
}

/* Exposed time led per (window, stage, rank): the sum of a window's
 * advances of stage s whose leader is rank r.  Leaders outside [0, R) are
 * not counted.  lead_exposed is [W][S][R].  top2 is [W][2][2]: the same two
 * stages as sfo_window_summary (largest window total of the advances, lower
 * stage first on ties), each paired with the rank that led the most exposed
 * time of that stage (lowest rank on ties; -1 if no rank led any). */
void sfo_window_lead_exposed(const int64_t* inc, const int32_t* lead, int64_t T, int32_t R,
                             int32_t S, int64_t window, int64_t* lead_exposed, int32_t* top2)
{
    int64_t W = (T + window - 1) / window;
    for (int64_t w = 0; w < W; ++w) {
        int64_t t0 = w * window;
        int64_t t1 = t0 + window < T ? t0 + window : T;
        for (int32_t s = 0; s < S; ++s) {
            int64_t* e = lead_exposed + (w * S + s) * (int64_t)R;
            for (int32_t r = 0; r < R; ++r) e[r] = 0;
            for (int64_t t = t0; t < t1; ++t) {
                int32_t r = lead[t * S + s];
                if (r >= 0 && r < R) e[r] += inc[t * S + s];
            }
        }

        /* the stage totals, recomputed from the advances */
        int32_t s1 = -1, s2 = -1;
        int64_t e1 = 0, e2 = 0;
        for (int32_t s = 0; s < S; ++s) {
            int64_t tot = 0;
            for (int64_t t = t0; t < t1; ++t) tot += inc[t * S + s];
            if (s1 < 0 || tot > e1) {
                s2 = s1;
                e2 = e1;
                s1 = s;
                e1 = tot;
            } else if (s2 < 0 || tot > e2) {
                s2 = s;
                e2 = tot;
            }
        }

        int32_t pick[2] = {s1, s2};
        for (int k = 0; k < 2; ++k) {
            int32_t sk = pick[k];
            int32_t rk = -1;
            if (sk >= 0) {
                const int64_t* e = lead_exposed + (w * S + sk) * (int64_t)R;
                int64_t best = 0;
                for (int32_t r = 0; r < R; ++r) {
                    if (e[r] > best) {
                        best = e[r];
                        rk = r;
                    }
                }
            }
            top2[w * 4 + 2 * k + 0] = sk;
            top2[w * 4 + 2 * k + 1] = rk;
        }
    }
}

/* Leader switches between confident unique leaders, per window and stage.
 * A boundary (t, s) qualifies when ties[t][s] == 1 and (gap[t][s] >= min_gap
 * or gap[t][s] < 0).  eligible[w][s] counts the qualifying boundaries of
 * window w; switches[w][s] counts those whose leader differs from the
 * leader of the previous qualifying boundary of the same stage and window. */
void sfo_window_leader_switches(const int32_t* lead, const int64_t* gap, const int32_t* ties,
                                int64_t T, int32_t S, int64_t window, int64_t min_gap,
                                int32_t* switches, int32_t* eligible)
{
    int64_t W = (T + window - 1) / window;
    for (int64_t w = 0; w < W; ++w) {
        int64_t t0 = w * window;
        int64_t t1 = t0 + window < T ? t0 + window : T;
        for (int32_t s = 0; s < S; ++s) {
            int32_t n_sw = 0, n_el = 0;
            int32_t prev = 0;
            int have_prev = 0;
            for (int64_t t = t0; t < t1; ++t) {
                const int64_t i = t * S + s;
                const int confident = ties[i] == 1 && (gap[i] >= min_gap || gap[i] < 0);
                if (!confident) continue;
                n_el += 1;
                if (have_prev && lead[i] != prev) n_sw += 1;
                prev = lead[i];
                have_prev = 1;
            }
            switches[w * S + s] = n_sw;
            eligible[w * S + s] = n_el;
        }
    }
}

/* Localization evidence and per-stage baselines of every boundary, with the
 * frontier advances and leaders of sfo_frontier, in the same order:
 *   (i)   the prefix matrix P[s][r] of the step;
 *   (ii)  per boundary: F[s] = max_r P[s][r]; the leader, the lowest rank
 *         attaining it; the tie set size #{r : P[s][r] = F[s]}; the runner-up,
 *         the largest prefix of a rank other than the leader, and the gap
 *         F[s] minus it (-1 when there is no other rank); the stage's max and
 *         sum of d over ranks;
 *   (iii) the advances a[s] = F[s] - F[s-1], F[-1] = 0.
 * Returns 0, or -1 if scratch cannot be allocated. */
int sfo_frontier_evidence(const int64_t* d, int64_t T, int32_t R, int32_t S,
                          int64_t* inc, int32_t* lead, int64_t* gap,
                          int32_t* ties, int64_t* stage_max, int64_t* stage_sum)
{
    int64_t* P = (int64_t*)calloc((size_t)S * (size_t)R, sizeof(int64_t));
    int64_t* F = (int64_t*)malloc(sizeof(int64_t) * (size_t)S);
    if (!P || !F) {
        free(P);
        free(F);
        return -1;
    }
    for (int64_t t = 0; t < T; ++t) {
        const int64_t* m = d + t * S * (int64_t)R;
        /* (i) */
        for (int32_t s = 0; s < S; ++s)
            for (int32_t r = 0; r < R; ++r)
                P[(int64_t)s * R + r] = (s > 0 ? P[(int64_t)(s - 1) * R + r] : 0) + m[(int64_t)s * R + r];
        /* (ii) */
        for (int32_t s = 0; s < S; ++s) {
            const int64_t* row = P + (int64_t)s * R;
            const int64_t* ds = m + (int64_t)s * R;
            int64_t best = row[0];
            for (int32_t r = 1; r < R; ++r)
                if (row[r] > best) best = row[r];
            F[s] = best;
            int32_t L = -1;
            for (int32_t r = 0; r < R && L < 0; ++r)
                if (row[r] == best) L = r;
            int32_t n_tie = 0;
            for (int32_t r = 0; r < R; ++r)
                if (row[r] == best) n_tie += 1;
            int64_t second = 0;
            int have_second = 0;
            for (int32_t r = 0; r < R; ++r) {
                if (r != L && (!have_second || row[r] > second)) {
                    second = row[r];
                    have_second = 1;
                }
            }
            int64_t dmax = ds[0], dsum = 0;
            for (int32_t r = 0; r < R; ++r) {
                if (ds[r] > dmax) dmax = ds[r];
                dsum += ds[r];
            }
            const int64_t i = t * S + s;
            lead[i] = L;
            gap[i] = have_second ? best - second : -1;
            ties[i] = n_tie;
            stage_max[i] = dmax;
            stage_sum[i] = dsum;
        }
        /* (iii) */
        for (int32_t s = 0; s < S; ++s) inc[t * S + s] = F[s] - (s > 0 ? F[s - 1] : 0);
    }
    free(P);
    free(F);
    return 0;
}

/* Ingest of gathered per-rank stage buffers (Appendix A closure): x is
 * [R][T][K] explicit stage durations, w is [R][T] step wall times.  Writes
 * d [T][K+1][R] with the residual stage last and the overlap error o [T][R]. */
void sfo_ingest(const int64_t* x, const int64_t* w, int64_t T, int32_t R, int32_t K,
                int64_t* d, int64_t* o)
{
    const int32_t S = K + 1;
    for (int32_t r = 0; r < R; ++r) {
        for (int64_t t = 0; t < T; ++t) {
            const int64_t* xs = x + ((int64_t)r * T + t) * K;
            int64_t explicit_sum = 0;
            for (int32_t k = 0; k < K; ++k) {
                d[(t * S + k) * R + r] = xs[k];
                explicit_sum += xs[k];
            }
            const int64_t e = w[(int64_t)r * T + t] - explicit_sum;
            d[(t * S + K) * R + r] = e > 0 ? e : 0;
            o[t * R + r] = e < 0 ? -e : 0;
        }
    }
}

/* Routing candidate set per window (Sec. 4): order[w] lists the stages by
 * exposed total, descending, lower stage first on ties; size[w] is the
 * smallest k whose first k stages reach tau = tau_num / tau_den of the
 * window total. */
void sfo_route(const int64_t* exposed, int64_t W, int32_t S, int64_t tau_num,
               int64_t tau_den, int32_t* order, int32_t* size)
{
    for (int64_t w = 0; w < W; ++w) {
        const int64_t* ex = exposed + w * S;
        int32_t* ord = order + w * S;
        /* insertion sort by (exposed desc, stage asc) */
        for (int32_t s = 0; s < S; ++s) {
            int32_t j = s;
            while (j > 0 && ex[ord[j - 1]] < ex[s]) {
                ord[j] = ord[j - 1];
                --j;
            }
            ord[j] = s;
        }
        __int128 total = 0;
        for (int32_t s = 0; s < S; ++s) total += ex[s];
        const __int128 need = (__int128)tau_num * total;
        __int128 cum = 0;
        int32_t k = 0;
        while (k < S && (__int128)tau_den * cum < need) {
            cum += ex[ord[k]];
            ++k;
        }
        size[w] = k;
    }
}

/* Frontier at the last boundary of one step, F[t,S] = max over ranks of the
 * rank's total, from its own running prefixes (Eq. (1)). */
static int64_t last_frontier(const int64_t* m, int32_t R, int32_t S, int64_t* P)
{
    for (int32_t r = 0; r < R; ++r) P[r] = 0;
    int64_t F = 0;
    for (int32_t s = 0; s < S; ++s) {
        for (int32_t r = 0; r < R; ++r) P[r] += m[(int64_t)s * R + r];
        F = P[0];
        for (int32_t r = 1; r < R; ++r)
            if (P[r] > F) F = P[r];
    }
    return F;
}

/* Direct-exposure gain, Eq. (4): for every step and stage s, the frontier is
 * recomputed on a copy of the step whose stage s holds min(d, btilde) on
 * every rank.  Per step: gain[t][s] = F[t,S] - F^(s<-b)[t,S] and
 * makespan[t] = F[t,S]; per window w: wgain[w][s] and wmakespan[w] are their
 * sums.  Returns 0, or -1 if scratch cannot be allocated. */
int sfo_exposure_gain(const int64_t* d, const int64_t* btilde, int64_t T, int32_t R,
                      int32_t S, int64_t window, int64_t* gain, int64_t* makespan,
                      int64_t* wgain, int64_t* wmakespan)
{
    const int64_t n = (int64_t)S * R;
    int64_t* m = (int64_t*)malloc(sizeof(int64_t) * (size_t)(n > 0 ? n : 1));
    int64_t* P = (int64_t*)malloc(sizeof(int64_t) * (size_t)(R > 0 ? R : 1));
    if (!m || !P) {
        free(m);
        free(P);
        return -1;
    }
    const int64_t W = (T + window - 1) / window;
    for (int64_t i = 0; i < W * S; ++i) wgain[i] = 0;
    for (int64_t i = 0; i < W; ++i) wmakespan[i] = 0;
    for (int64_t t = 0; t < T; ++t) {
        const int64_t w = t / window;
        const int64_t* step = d + t * n;
        const int64_t F = last_frontier(step, R, S, P);
        makespan[t] = F;
        wmakespan[w] += F;
        for (int32_t s = 0; s < S; ++s) {
            /* the step with stage s replaced by the clipped baseline */
            for (int64_t i = 0; i < n; ++i) m[i] = step[i];
            for (int32_t r = 0; r < R; ++r) {
                const int64_t b = btilde[(w * S + s) * R + r];
                int64_t* cell = m + (int64_t)s * R + r;
                if (b < *cell) *cell = b;
            }
            const int64_t g = F - last_frontier(m, R, S, P);
            gain[t * S + s] = g;
            wgain[w * S + s] += g;
        }
    }
    free(m);
    free(P);
    return 0;
}

static int cmp_i64(const void* a, const void* b)
{
    const int64_t x = *(const int64_t*)a, y = *(const int64_t*)b;
    return (x > y) - (x < y);
}

/* Lag of the frontier over the median rank (Sec. 4) and its increment.
 * The median is taken with a library sort of a copy of the prefixes.
 * Returns 0, or -1 if scratch cannot be allocated. */
int sfo_frontier_lag(const int64_t* d, int64_t T, int32_t R, int32_t S, int64_t* lag,
                     int64_t* lag_inc)
{
    int64_t* P = (int64_t*)malloc(sizeof(int64_t) * (size_t)(R > 0 ? R : 1));
    int64_t* sorted = (int64_t*)malloc(sizeof(int64_t) * (size_t)(R > 0 ? R : 1));
    if (!P || !sorted) {
        free(P);
        free(sorted);
        return -1;
    }
    for (int64_t t = 0; t < T; ++t) {
        for (int32_t r = 0; r < R; ++r) P[r] = 0;
        int64_t L_prev = 0;
        for (int32_t s = 0; s < S; ++s) {
            const int64_t* row = d + (t * S + s) * (int64_t)R;
            for (int32_t r = 0; r < R; ++r) P[r] += row[r];
            memcpy(sorted, P, sizeof(int64_t) * (size_t)R);
            qsort(sorted, (size_t)R, sizeof(int64_t), cmp_i64);
            const int64_t F = sorted[R - 1];
            const int64_t median = sorted[(R - 1) / 2];
            const int64_t L = F - median;
            lag[t * S + s] = L;
            lag_inc[t * S + s] = L - L_prev;
            L_prev = L;
        }
    }
    free(P);
    free(sorted);
    return 0;
}

/* Raw rank spread of Sec. 6.2: spread[t][s] = max_r d - median_r d at every
 * step and stage (lower median, by a library sort of a copy of the row),
 * and its sums over the steps of each window, wspread[W][S].
 * Returns 0, or -1 if scratch cannot be allocated. */
int sfo_rank_spread(const int64_t* d, int64_t T, int32_t R, int32_t S, int64_t window,
                    int64_t* spread, int64_t* wspread)
{
    int64_t* sorted = (int64_t*)malloc(sizeof(int64_t) * (size_t)(R > 0 ? R : 1));
    if (!sorted) return -1;
    const int64_t W = T / window + (T % window != 0);
    for (int64_t i = 0; i < W * S; ++i) wspread[i] = 0;
    for (int64_t t = 0; t < T; ++t) {
        const int64_t w = t / window;
        for (int32_t s = 0; s < S; ++s) {
            const int64_t* row = d + (t * S + s) * (int64_t)R;
            memcpy(sorted, row, sizeof(int64_t) * (size_t)R);
            qsort(sorted, (size_t)R, sizeof(int64_t), cmp_i64);
            const int64_t x = sorted[R - 1] - sorted[(R - 1) / 2];
            spread[t * S + s] = x;
            wspread[w * S + s] += x;
        }
    }
    free(sorted);
    return 0;
}

/* Per-rank window median, a candidate baseline btilde of Eq. (4) (Sec. 4):
 * med[w][s][r] = the lower median of d[t][s][r] over the n steps t of
 * window w (the element of rank floor((n-1)/2) of a library sort).
 * Returns 0, or -1 if scratch cannot be allocated. */
int sfo_window_median(const int64_t* d, int64_t T, int32_t R, int32_t S, int64_t window,
                      int64_t* med)
{
    int64_t* col = (int64_t*)malloc(sizeof(int64_t) * (size_t)(window < T ? window : (T > 0 ? T : 1)));
    if (!col) return -1;
    const int64_t W = T / window + (T % window != 0);
    for (int64_t w = 0; w < W; ++w) {
        const int64_t t0 = w * window;
        const int64_t t1 = t0 + window < T ? t0 + window : T;
        const int64_t n = t1 - t0;
        for (int32_t s = 0; s < S; ++s) {
            for (int32_t r = 0; r < R; ++r) {
                for (int64_t t = t0; t < t1; ++t) col[t - t0] = d[(t * S + s) * (int64_t)R + r];
                qsort(col, (size_t)n, sizeof(int64_t), cmp_i64);
                med[(w * S + s) * (int64_t)R + r] = col[(n - 1) / 2];
            }
        }
    }
    free(col);
    return 0;
}

/* Range status of the data contract (Sec. 3: nonnegative durations; prefixes
 * below 2^47 ns for the library's packed keys): 2 (SF_ERANGE) if some
 * d[t][s][r] < 0 or some prefix P[t][r][s] >= 2^47, else 0.  A rank stops
 * accumulating once it is flagged, so nothing overflows.
 * Returns the status, or -1 if scratch cannot be allocated. */
int sfo_range_status(const int64_t* d, int64_t T, int32_t R, int32_t S)
{
    const int64_t limit = (int64_t)1 << 47;
    int64_t* P = (int64_t*)malloc(sizeof(int64_t) * (size_t)(R > 0 ? R : 1));
    if (!P) return -1;
    int status = 0;
    for (int64_t t = 0; t < T && status == 0; ++t) {
        for (int32_t r = 0; r < R; ++r) P[r] = 0;
        for (int32_t s = 0; s < S && status == 0; ++s) {
            const int64_t* row = d + (t * S + s) * (int64_t)R;
            for (int32_t r = 0; r < R; ++r) {
                if (row[r] < 0 || row[r] >= limit - P[r]) {
                    status = 2;
                    break;
                }
                P[r] += row[r];
            }
        }
    }
    free(P);
    return status;
}
