/*
 * stagefrontier.h -- C ABI of libstagefrontier.
 *
 * StageFrontier frontier accounting over per-rank ordered stage durations
 * (Sec. 3 "Frontier Accounting", Eq. (1) and Eq. (2); window reduction and
 * top-2 routing of Sec. 4), computed on an AMD Instinct MI355X (gfx950).
 *
 * Notation (Sec. 3): d[t][s][r] >= 0 is the duration of ordered stage s on
 * rank r in training step t.  With 0-based stage indices
 *     P[t][r][s] = sum_{j <= s} d[t][j][r]          rank-local prefix
 *     F[t][s]    = max_r P[t][r][s]                 frontier
 *     a[t][s]    = F[t][s] - F[t][s-1],  F[t][-1] = 0   frontier advance
 * and the leader of boundary (t, s) is the lowest rank index r with
 * P[t][r][s] == F[t][s].
 *
 * Conventions shared by every entry point:
 *  - All array pointers are DEVICE pointers (hipMalloc'd memory or memory
 *    the device can address).  Arrays are dense, row-major, with no padding.
 *  - Every call that takes a stream is asynchronous on that stream: it
 *    validates its arguments on the host, enqueues kernels and returns.
 *    Outputs are valid once the stream has reached that point.  A NULL
 *    stream means the legacy default stream.
 *  - The caller allocates and frees every buffer.  The library allocates no
 *    memory, never synchronises a stream and keeps no mutable global state,
 *    so calls are reentrant and may be issued from several host threads.
 *  - Inputs are read only.  Output arrays must not overlap each other or
 *    any input (checked: SF_EINVAL).
 *  - Errors found on the host are returned before anything is enqueued.
 *    SF_EHIP reports a failed kernel launch; nothing is left enqueued by
 *    the failing call after its first failed launch.
 */
#ifndef STAGEFRONTIER_H
#define STAGEFRONTIER_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* hipStream_t, passed as an opaque pointer so that the header needs no HIP
 * include.  NULL selects the default stream. */
typedef void* sf_stream_t;

/* Status codes returned by every int-returning entry point. */
enum {
    SF_OK = 0,
    SF_EINVAL = 1, /* bad argument: NULL pointer, size out of range,
                      misaligned pointer, overlapping outputs, overflow   */
    SF_ERANGE = 2, /* data outside the contract (sf_frontier_checked's
                      status word; never returned by a call)             */
    SF_EHIP = 3    /* the HIP runtime rejected a kernel launch            */
};

/* Largest rank count: the leader is carried in 16 bits of a packed
 * (prefix, rank) key. */
#define SF_MAX_R 65536
/* Stage counts are unbounded (up to the size overflow checks): Sec. 3
 * expands every accumulation micro-step into its own stages before the
 * frontier is taken, so S grows with the accumulation count. */
/* Every rank-local prefix P[t][r][s] must be below this many ns (about
 * 39 hours) so that the packed key fits in 64 bits. */
#define SF_MAX_PREFIX_NS ((int64_t)1 << 47)

/*
 * sf_frontier -- per-step frontier advances and leaders (Sec. 3, Eq. (1);
 * the single streaming pass over steps, stages and ranks of Sec. 3).
 *
 *   durations      [T][S][R] int64, ns; rank index fastest.  Read once.
 *   T              number of steps, 0 <= T.  T == 0 is a no-op (pointers
 *                  may then be NULL).
 *   R              number of ranks, 1 <= R <= SF_MAX_R.
 *   S              number of ordered stages, 1 <= S (any count whose
 *                  arrays fit in int64 byte sizes: SF_EINVAL on overflow).
 *   out_increment  [T][S] int64, ns: a[t][s].  Written.  With S above 512
 *                  it also holds intermediate per-stage maxima while the
 *                  call runs, so it must not be read before the stream has
 *                  passed the call (true of every output anyway).
 *   out_leader     [T][S] int32: lowest rank attaining F[t][s].  Written.
 *   stream         HIP stream the work is enqueued on.
 *
 * Data preconditions (not checked): every d >= 0 (Sec. 3 requires
 * nonnegative durations) and every prefix P < SF_MAX_PREFIX_NS.  Outputs
 * are unspecified when they are violated.  Pointers must be aligned to
 * their element size (checked).
 *
 * Steps are independent, so a long step axis may be processed in chunks:
 * pass durations + t0*S*R, out_increment + t0*S, out_leader + t0*S with
 * T = chunk length.  The result equals one call over the whole range.
 *
 * Returns SF_OK, SF_EINVAL or SF_EHIP.
 */
int sf_frontier(const int64_t* durations, int64_t T, int32_t R, int32_t S,
                int64_t* out_increment, int32_t* out_leader,
                sf_stream_t stream);

/*
 * sf_frontier_checked -- sf_frontier, verifying the data contract on the
 * same pass: if some duration lies outside [0, SF_MAX_PREFIX_NS) or some
 * prefix P[t][r][s] reaches SF_MAX_PREFIX_NS, SF_ERANGE is OR-ed into
 * *status.  The word is the caller's: the library never clears it, so one
 * word can collect several calls; clear it before the first.  Where the
 * contract holds the outputs equal sf_frontier's, and *status is untouched.
 *
 *   durations, T, R, S, out_increment, out_leader, stream: as for
 *                  sf_frontier.
 *   status         device uint32, 4-byte aligned, overlapping no array of
 *                  the call.
 *
 * Data errors are reported only through *status, once the stream has
 * reached this call.  Returns SF_OK, SF_EINVAL (also for a NULL status) or
 * SF_EHIP.
 */
int sf_frontier_checked(const int64_t* durations, int64_t T, int32_t R, int32_t S,
                        int64_t* out_increment, int32_t* out_leader, uint32_t* status,
                        sf_stream_t stream);

/*
 * sf_frontier_evidence -- the sf_frontier pass plus, at every boundary, the
 * localization evidence of Sec. 4 (the frontier tie set and the gap between
 * the largest and second-largest prefix) and the per-stage terms of the
 * max and mean baselines that Props. 1 and 2 compare the frontier with
 * (M_t = sum_s max_r d, Mbar_t = sum_s (1/R) sum_r d).  One read of the
 * durations produces all six outputs.
 *
 *   durations, T, R, S, out_increment, out_leader: as for sf_frontier (the
 *                  outputs are identical to sf_frontier's).
 *   out_gap        [T][S] int64, ns: F[t][s] minus the second-largest prefix
 *                  over ranks (0 exactly when two or more ranks attain F);
 *                  -1 when R == 1 (no runner-up).
 *   out_ties       [T][S] int32: number of ranks r with P[t][r][s] == F[t][s]
 *                  (>= 1); the leader is the lowest of them.
 *   out_stage_max  [T][S] int64, ns: max over r of d[t][s][r].
 *   out_stage_sum  [T][S] int64, ns: sum over r of d[t][s][r].
 *   stream         HIP stream.
 *
 * Preconditions, alignment (element size), chunking and overlap rules as
 * for sf_frontier; additionally T <= INT32_MAX.  Any S: past 819 stages the
 * per-stage partial results of a step are kept in its own output rows
 * instead of on chip (slower, same results).
 * Returns SF_OK, SF_EINVAL or SF_EHIP.
 */
int sf_frontier_evidence(const int64_t* durations, int64_t T, int32_t R, int32_t S,
                         int64_t* out_increment, int32_t* out_leader,
                         int64_t* out_gap, int32_t* out_ties,
                         int64_t* out_stage_max, int64_t* out_stage_sum,
                         sf_stream_t stream);

/*
 * sf_ingest -- the step before the path: gathered per-rank stage buffers to
 * the [T][S][R] layout, with the closure of Appendix A.  For each rank r and
 * step t, with w[r][t] the rank-local step wall time and x[r][t][k] the K
 * explicit stage durations, e = w - sum_k x; the residual stage
 * ("step.other", last in the default taxonomy) is max(0, e) and the
 * overlap error is max(0, -e).
 *
 *   stages         [R][T][K] int64 ns, each rank's buffer as gathered
 *                  (steps, then explicit stages).  May be NULL when K == 0.
 *   wall           [R][T] int64 ns.
 *   T, R, K        0 <= T, 1 <= R <= SF_MAX_R, 0 <= K <= INT32_MAX - 2.
 *                  Up to 511 explicit stages a rank's segment of a step is
 *                  staged in LDS; beyond, each thread walks its (step, rank)
 *                  segment in global memory (slower, same results).
 *                  T == 0 is a no-op.
 *   out_durations  [T][K+1][R] int64: stage k < K is x, stage K the residual.
 *   out_overlap    [T][R] int64.
 *   stream         HIP stream.
 *
 * Pointers 8-byte aligned; outputs must not overlap inputs or each other.
 * Returns SF_OK, SF_EINVAL or SF_EHIP.
 */
int sf_ingest(const int64_t* stages, const int64_t* wall, int64_t T, int32_t R,
              int32_t K, int64_t* out_durations, int64_t* out_overlap,
              sf_stream_t stream);

/*
 * sf_route -- the routing candidate set of Sec. 4 per window: the smallest
 * prefix of stages, ordered by share, whose cumulative share reaches
 * tau_C = tau_num / tau_den (the paper's default is 0.80 = 4/5).  Shares of
 * a window have a common denominator (Eq. (2)), so the order and the test
 * use the exposed totals of sf_window_summary directly:
 * k stages suffice when tau_den * (sum of their totals) >= tau_num * (sum of
 * all totals), evaluated exactly in 128-bit integers.
 *
 *   stage_exposed  [W][S] int64 (out_stage_exposed of sf_window_summary).
 *   W, S           0 <= W, 1 <= S.  W == 0 is a no-op.
 *   tau_num, tau_den  0 <= tau_num <= tau_den, 1 <= tau_den <= INT32_MAX.
 *   out_order      [W][S] int32: stages by total, descending; the lower
 *                  stage first on ties (so the first two are the top-2
 *                  stages of sf_window_summary).
 *   out_size       [W] int32: the candidate-set size k (0 when the window
 *                  total is 0 or tau is 0); the set is out_order[w][0..k).
 *   stream         HIP stream.
 *
 * Returns SF_OK, SF_EINVAL or SF_EHIP.
 */
int sf_route(const int64_t* stage_exposed, int64_t W, int32_t S, int64_t tau_num,
             int64_t tau_den, int32_t* out_order, int32_t* out_size,
             sf_stream_t stream);

/*
 * sf_exposure_gain -- the direct-exposure score of Eq. (4) (Sec. 4).  For
 * every step t and stage s, stage s of every rank is replaced by the clipped
 * baseline b = min(d, btilde) and the frontier is recomputed; the gain is
 * F[t][S-1] - F^(s<-b)[t][S-1] >= 0.  Per window, G_s = out_window_gain[w][s]
 * / out_window_makespan[w]; the quotient is left to the caller.
 *
 *   durations            [T][S][R] int64 ns (as for sf_frontier).
 *   baseline             [W][S][R] int64 ns: btilde for the steps of window
 *                        w (a per-rank window median, a cohort median, a
 *                        no-stall reference, ...).
 *   T, R, S, window      as for sf_window_summary.  Up to 64 stages the
 *                        per-stage deltas are held in registers and the
 *                        durations read once; past 64 a two-pass kernel
 *                        reads each step's durations twice (slower, same
 *                        results).  From 4097 to 16384 ranks (up to 16
 *                        stages, even R, 16-byte aligned inputs) a step's
 *                        durations are read once into rank totals and the
 *                        baseline only for the ranks near the frontier; a
 *                        step that the bound does not settle is read again
 *                        over all ranks (same results).
 *   out_gain             [T][S] int64: the gain of each step and stage.
 *   out_makespan         [T] int64: F[t][S-1], the step's exposed makespan.
 *   out_window_gain      [W][S] int64: window sums of out_gain.
 *   out_window_makespan  [W] int64: window sums of out_makespan.
 *   stream               HIP stream.
 *
 * Preconditions as for sf_frontier, and every baseline value must lie in
 * [0, SF_MAX_PREFIX_NS).  Pointers 8-byte aligned; outputs must not overlap
 * inputs or each other.  Returns SF_OK, SF_EINVAL or SF_EHIP.
 */
int sf_exposure_gain(const int64_t* durations, const int64_t* baseline, int64_t T,
                     int32_t R, int32_t S, int64_t window, int64_t* out_gain,
                     int64_t* out_makespan, int64_t* out_window_gain,
                     int64_t* out_window_makespan, sf_stream_t stream);

/*
 * sf_frontier_lag -- the lag of the frontier over the median rank, one of
 * the localization signals of Sec. 4: L[t][s] = F[t][s] - median_r P[t][r][s],
 * and its increment L[t][s] - L[t][s-1] (L[t][-1] = 0).  The median is the
 * lower median: the prefix of rank floor((R - 1) / 2) in ascending order
 * (the middle one for odd R), so the lag is an exact integer.
 *
 *   durations      [T][S][R] int64 ns (as for sf_frontier).
 *   T, R, S        0 <= T <= INT32_MAX, 1 <= R <= SF_MAX_R, 1 <= S.  A
 *                  step's values are held on chip up to 16384 ranks (up to
 *                  32768 for even R with a 16-byte aligned base); beyond
 *                  that a kernel re-reads them from global memory at every
 *                  select pass (slower, same results).
 *                  T == 0 is a no-op.
 *   out_lag        [T][S] int64 ns, >= 0.
 *   out_lag_inc    [T][S] int64 ns.
 *   stream         HIP stream.
 *
 * Preconditions, alignment, chunking and overlap rules as for sf_frontier.
 * Returns SF_OK, SF_EINVAL or SF_EHIP.
 */
int sf_frontier_lag(const int64_t* durations, int64_t T, int32_t R, int32_t S,
                    int64_t* out_lag, int64_t* out_lag_inc, sf_stream_t stream);

/*
 * sf_rank_spread -- the raw rank spread, the dispersion baseline of Sec. 6.2
 * that ranks stages by sum over steps of (max_r d - median_r d):
 * spread[t][s] = max_r d[t][s][r] - the lower median over r of d[t][s][r]
 * (rank floor((R - 1) / 2) in ascending order, as for sf_frontier_lag), and
 * its sums over the steps of each window.
 *
 *   durations          [T][S][R] int64 ns (as for sf_frontier).
 *   T, R, S            0 <= T <= INT32_MAX, 1 <= R <= SF_MAX_R, 1 <= S
 *                      (above 16384 ranks as for sf_frontier_lag).
 *                      T == 0 is a no-op.
 *   window             steps per window, >= 1 (windows as for
 *                      sf_window_summary).
 *   out_spread         [T][S] int64 ns, >= 0.
 *   out_window_spread  [W][S] int64 ns: window sums of out_spread.
 *   stream             HIP stream.
 *
 * Preconditions and alignment as for sf_frontier; outputs must not overlap
 * the input or each other.  Returns SF_OK, SF_EINVAL or SF_EHIP.
 */
int sf_rank_spread(const int64_t* durations, int64_t T, int32_t R, int32_t S,
                   int64_t window, int64_t* out_spread, int64_t* out_window_spread,
                   sf_stream_t stream);

/*
 * sf_window_median -- the per-rank window median, a candidate baseline
 * btilde of Eq. (4) (Sec. 4): out_median[w][s][r] is the lower median of
 * d[t][s][r] over the n steps t of window w (the value of rank
 * floor((n - 1) / 2) in ascending order).  Its output is laid out as the
 * baseline argument of sf_exposure_gain.
 *
 *   durations   [T][S][R] int64 ns (as for sf_frontier).
 *   T, R, S     0 <= T, 1 <= R <= SF_MAX_R, 1 <= S.  T == 0 is a no-op.
 *   window      steps per window, >= 1 (windows as for sf_window_summary).
 *               Windows of up to 1024 steps are held on chip in tiles of
 *               ranks; longer ones are selected from global memory, one
 *               column at a time (slower, same results).
 *   out_median  [W][S][R] int64 ns.
 *   stream      HIP stream.
 *
 * Pointers 8-byte aligned; the output must not overlap the input.  Returns
 * SF_OK, SF_EINVAL or SF_EHIP.
 */
int sf_window_median(const int64_t* durations, int64_t T, int32_t R, int32_t S,
                     int64_t window, int64_t* out_median, sf_stream_t stream);

/*
 * sf_num_windows -- number of windows W = ceil(T / window) that
 * sf_window_summary produces.  Sec. 3 reduces the per-step advances over
 * windows of N consecutive steps (Eq. (2)) and lets a window close early;
 * the paper does not say how a step count that is not a multiple of N ends,
 * so the last window holds the remaining T - (W-1)*window steps (a shorter
 * window, never a dropped one).  Returns -1 when T < 0 or window < 1.
 * Host only; no device work.
 */
int64_t sf_num_windows(int64_t T, int64_t window);

/*
 * sf_window_summary -- window reduction of the per-step results (Eq. (2) of
 * Sec. 3: numerators of the stage shares; leader counts; the top-2 stage
 * routing of Sec. 4).
 *
 *   increment          [T][S] int64 from sf_frontier.
 *   leader             [T][S] int32 from sf_frontier.  Entries outside
 *                      [0, R) are not counted anywhere.
 *   T, R, S            as for sf_frontier (T == 0 is a no-op).
 *   window             steps per window, >= 1.  Window w covers steps
 *                      [w*window, min((w+1)*window, T)).
 *   out_stage_exposed  [W][S] int64: sum over the window of a[t][s].  The
 *                      share A_s of Eq. (2) is this value divided by the
 *                      sum over s of the same row (Theorem 1).
 *   out_lead_counts    [W][S][R] int32: number of steps of the window whose
 *                      leader at stage s is rank r (zeros included).
 *   out_top2           [W][2][2] int32: {{s1, r1}, {s2, r2}}.  s1, s2 are
 *                      the two stages with the largest exposed totals
 *                      (ties go to the lower stage index); rk is the rank
 *                      with the largest lead count at stage sk (ties go to
 *                      the lower rank; -1 if that count is 0).  When S == 1
 *                      the second pair is {-1, -1}.
 *   stream             HIP stream.
 *
 * The sums are exact in int64 unless they overflow: a window total is at
 * most window * max F, so any window below 65536 steps is exact at the
 * prefix bound, and any window below 2^28 steps with step times under
 * 2^35 ns (about 34 s).
 *
 * Returns SF_OK, SF_EINVAL or SF_EHIP.
 */
int sf_window_summary(const int64_t* increment, const int32_t* leader,
                      int64_t T, int32_t R, int32_t S, int64_t window,
                      int64_t* out_stage_exposed, int32_t* out_lead_counts,
                      int32_t* out_top2, sf_stream_t stream);

/*
 * sf_frontier_summary -- sf_frontier followed by sf_window_summary over the
 * same steps, as one call: the per-step accounting of Sec. 3 (Eq. (1)) and
 * its reduction over windows (Eq. (2) numerators, lead counts, the top-2 of
 * Sec. 4).  Small inputs (R <= 256, S <= 64, min(window, T) <= 1024 and
 * T * S * R <= 2^20 samples) run as ONE kernel launch, one workgroup per
 * window, for callers bound by launch latency (a per-step or per-window
 * serving loop); larger ones run the two calls' kernels.  Every output is
 * identical to sf_frontier's and sf_window_summary's.
 *
 *   durations          [T][S][R] int64 ns (as for sf_frontier).
 *   T, R, S, window    as for sf_window_summary (T == 0 is a no-op).
 *   out_increment      [T][S] int64, out_leader [T][S] int32: as for
 *                      sf_frontier.
 *   out_stage_exposed  [W][S] int64, out_lead_counts [W][S][R] int32,
 *   out_top2           [W][2][2] int32: as for sf_window_summary.
 *   stream             HIP stream.
 *
 * Preconditions as for sf_frontier.  Pointers aligned to their element
 * size; no two arrays may overlap.  Returns SF_OK, SF_EINVAL or SF_EHIP.
 */
int sf_frontier_summary(const int64_t* durations, int64_t T, int32_t R, int32_t S,
                        int64_t window, int64_t* out_increment, int32_t* out_leader,
                        int64_t* out_stage_exposed, int32_t* out_lead_counts,
                        int32_t* out_top2, sf_stream_t stream);

/*
 * sf_window_lead_exposed -- the exposed time each rank led, per window and
 * stage.  Every advance a[t][s] is attributed to the rank attaining the
 * frontier (Sec. 3), so summing a window's advances of stage s by leader
 * splits the stage's exposed total (the Eq. (2) numerator) over ranks:
 * the rank-level counterpart of the stage shares, and the exposed-time
 * weighting of the top-2 rank localization of Sec. 4.
 *
 *   increment, leader, T, R, S, window: as for sf_window_summary.
 *   out_lead_exposed   [W][S][R] int64: sum of a[t][s] over the steps t of
 *                      window w whose leader at stage s is rank r (zeros
 *                      included).  Leaders outside [0, R) count nowhere,
 *                      so a row sums to out_stage_exposed[w][s] whenever
 *                      every leader of the window lies in [0, R).
 *   out_top2           [W][2][2] int32: {{s1, r1}, {s2, r2}}.  s1, s2 are
 *                      the stages of sf_window_summary's top-2 (largest
 *                      window total of a[t][s], the lower stage on ties);
 *                      rk is the rank that led the most exposed time of
 *                      stage sk (the lower rank on ties; -1 if no entry of
 *                      that row is positive).  When S == 1 the second pair
 *                      is {-1, -1}.
 *   stream             HIP stream.
 *
 * Exactness as for sf_window_summary.  Pointers aligned to their element
 * size; outputs must not overlap inputs or each other.  Returns SF_OK,
 * SF_EINVAL or SF_EHIP.
 */
int sf_window_lead_exposed(const int64_t* increment, const int32_t* leader, int64_t T,
                           int32_t R, int32_t S, int64_t window, int64_t* out_lead_exposed,
                           int32_t* out_top2, sf_stream_t stream);

/*
 * sf_window_leader_switches -- leader-switch evidence of Sec. 4: per window
 * and stage, how often the frontier's leader changes, counted only between
 * confident unique leaders.  A boundary (t, s) qualifies when one rank
 * alone attains F[t][s] (tie-set size 1) and leads the runner-up by at least
 * min_gap ns (a boundary with no runner-up, R == 1, qualifies).  The paper's
 * gates on the switch rate and on the qualifying fraction (App. C) state no
 * values; they are left to the caller, who has both counts.
 *
 *   leader         [T][S] int32 (out_leader of sf_frontier_evidence).
 *   gap            [T][S] int64 (out_gap of sf_frontier_evidence).
 *   ties           [T][S] int32 (out_ties of sf_frontier_evidence).
 *   T, S, window   0 <= T, 1 <= S, 1 <= window, and
 *                  min(window, T) <= INT32_MAX.  T == 0 is a no-op.
 *                  Window w covers steps [w*window, min((w+1)*window, T)).
 *   min_gap        the confidence threshold on the gap, ns.
 *   out_switches   [W][S] int32: the qualifying boundaries of window w and
 *                  stage s whose leader differs from the leader of the
 *                  previous qualifying boundary of the same stage and
 *                  window (each window starts afresh).
 *   out_eligible   [W][S] int32: the qualifying boundaries of window w and
 *                  stage s.  out_switches <= max(out_eligible - 1, 0).
 *   stream         HIP stream.
 *
 * Pointers aligned to their element size; outputs must not overlap inputs
 * or each other.  Returns SF_OK, SF_EINVAL or SF_EHIP.
 */
int sf_window_leader_switches(const int32_t* leader, const int64_t* gap, const int32_t* ties,
                              int64_t T, int32_t S, int64_t window, int64_t min_gap,
                              int32_t* out_switches, int32_t* out_eligible, sf_stream_t stream);

/*
 * sf_read_xor -- plain-read calibration (a measurement aid, not part of the
 * paper's method): the XOR of the 64-bit words of every SF_XOR_PIECE_BYTES
 * piece of a device buffer.  It reads each byte exactly once with the
 * streaming loads of the frontier pass and does nothing else, so its rate
 * is the device's practical read ceiling, against which the single-pass
 * kernels (Eq. (1) reads each duration once) are measured.  The words also
 * serve as a cheap per-piece checksum of a buffer, e.g. after an upload.
 *
 *   buf       device buffer, 16-byte aligned, read only.  May be NULL when
 *             bytes == 0.
 *   bytes     buffer length, a multiple of 8, >= 0 (0 is a no-op).
 *   out_xor   device uint64_t[sf_read_xor_pieces(bytes)], 8-byte aligned,
 *             disjoint from buf.  Word i is the XOR of the little-endian
 *             64-bit words in bytes [i * SF_XOR_PIECE_BYTES,
 *             min((i + 1) * SF_XOR_PIECE_BYTES, bytes)) of buf.  The XOR of
 *             all its words is the XOR of the whole buffer.
 *   stream    HIP stream.
 *
 * Returns SF_OK, SF_EINVAL (alignment, length, NULL, overlap, or more than
 * 2^31 - 1 pieces) or SF_EHIP.
 */
#define SF_XOR_PIECE_BYTES 262144
int sf_read_xor(const void* buf, int64_t bytes, uint64_t* out_xor, sf_stream_t stream);

/*
 * sf_read_xor_pieces -- number of words sf_read_xor writes for a buffer of
 * `bytes` bytes: ceil(bytes / SF_XOR_PIECE_BYTES).  Returns -1 when
 * bytes < 0.  Host only; no device work.
 */
int64_t sf_read_xor_pieces(int64_t bytes);

/* sf_strerror -- static, NUL-terminated description of a status code. */
const char* sf_strerror(int status);

/* sf_version -- static, NUL-terminated library version string. */
const char* sf_version(void);

#ifdef __cplusplus
}
#endif

#endif /* STAGEFRONTIER_H */
