// gain.hip -- direct-exposure gain, Eq. (4).  Replacing stage s of every rank by
// b = min(d, btilde) changes the last frontier F[t,S] = max_r P[t,r,S] only
// through the rank totals: F^(s<-b)[t,S] = max_r (P[t,r,S] - delta[r,s]) with
// delta = max(0, d - btilde).  Step group layout as in k_frontier; each lane
// keeps its ranks' totals and the deltas of all stages in registers (the
// stage loop is unrolled to SMAX, rows past S re-read row 0 and are
// ignored), then every stage's candidate max and the plain max go through
// the idempotent DPP max, so lane slots past R (which re-read rank r0) need
// no masking.  When a step spans several rank tiles (and up to 16 stages)
// a lane keeps its running maxima over the tiles in registers and the group
// reduces once per step; otherwise the group reduces every tile.  Partial
// maxima of several groups meet in LDS.
//
// Past 4096 ranks (up to 16384, 16 stages) k_exposure_gain_near takes the
// maximum over the ranks near the frontier first and over all ranks only
// when a bound requires it.

#include "sf_device.h"
#include "sf_host.h"
#include "sf_select.h"

namespace sfk {

template <int VEC, int K, int G, int WG, int SMAX, bool RUN>
__global__ __launch_bounds__(WG) void k_exposure_gain(
    const int64_t* __restrict__ d, const int64_t* __restrict__ btilde, int64_t T, int R, int S,
    int64_t window, int64_t* __restrict__ gain, int64_t* __restrict__ makespan)
{
    static_assert(K % VEC == 0 && (WG % G == 0 || G == WG), "shape");
    constexpr int SUB = G < 64 ? G : 64;
    constexpr int SPW = WG / G;
    constexpr int SPS = G / SUB;
    constexpr int NLD = K / VEC;
    constexpr int RT = G * K;
    constexpr int NCOL = SMAX + 1;  // SMAX replaced-stage maxima, then F
    static_assert(!RUN || SMAX <= 16, "running maxima of up to 16 stages");

    __shared__ u64 tab[(WG / SUB) * NCOL];

    const int tid = threadIdx.x;
    const int gl = tid % G;
    const int slot = tid / SUB;
    const bool writer = (tid % SUB) == SUB - 1;
    const int64_t tb = xcd_block() * SPW;
    const int64_t t = tb + tid / G;

    if (t < T) {
        const int64_t* dt = d + t * (int64_t)S * R;
        const int64_t* bw = btilde + (t / window) * (int64_t)S * R;
        u64 run[RUN ? NCOL : 1];  // RUN: this lane's maxima so far ([SMAX] is F)
#pragma unroll
        for (int c = 0; c < (RUN ? NCOL : 1); ++c) run[c] = 0;
        for (int r0 = 0; r0 < R; r0 += RT) {
            int idx[NLD];
#pragma unroll
            for (int l = 0; l < NLD; ++l) {
                const int r = r0 + (l * G + gl) * VEC;
                idx[l] = r < R ? r : r0;
            }
            int64_t tot[K];
            int64_t dl[K][SMAX];
#pragma unroll
            for (int k = 0; k < K; ++k) tot[k] = 0;
#pragma unroll
            for (int s = 0; s < SMAX; ++s) {
                const int sr = s < S ? s : 0;
                const int64_t* row = dt + (int64_t)sr * R;
                const int64_t* brow = bw + (int64_t)sr * R;
#pragma unroll
                for (int l = 0; l < NLD; ++l) {
                    int64_t x[VEC], y[VEC];
                    if (VEC == 2) {
                        const v2i64 a = __builtin_nontemporal_load(reinterpret_cast<const v2i64*>(row + idx[l]));
                        const v2i64 b = *reinterpret_cast<const v2i64*>(brow + idx[l]);
                        x[0] = a.x;
                        x[VEC - 1] = a.y;
                        y[0] = b.x;
                        y[VEC - 1] = b.y;
                    } else {
                        x[0] = __builtin_nontemporal_load(row + idx[l]);
                        y[0] = brow[idx[l]];
                    }
#pragma unroll
                    for (int e = 0; e < VEC; ++e) {
                        const int k = l * VEC + e;
                        const int64_t red = x[e] - y[e];
                        dl[k][s] = red > 0 ? red : 0;
                        if (s < S) tot[k] += x[e];
                    }
                }
            }
            u64 fmax = 0;
#pragma unroll
            for (int k = 0; k < K; ++k) fmax = umax64(fmax, (u64)tot[k]);
            if constexpr (RUN) {
                run[SMAX] = umax64(run[SMAX], fmax);
            } else {
                fmax = group_max<SUB>(fmax);
                if (writer) {
                    u64* p = &tab[slot * NCOL + SMAX];
                    *p = (r0 == 0) ? fmax : umax64(*p, fmax);
                }
            }
#pragma unroll
            for (int s = 0; s < SMAX; ++s) {
                if (s < S) {
                    u64 m = 0;
#pragma unroll
                    for (int k = 0; k < K; ++k) m = umax64(m, (u64)(tot[k] - dl[k][s]));
                    if constexpr (RUN) {
                        run[s] = umax64(run[s], m);
                    } else {
                        m = group_max<SUB>(m);
                        if (writer) {
                            u64* p = &tab[slot * NCOL + s];
                            *p = (r0 == 0) ? m : umax64(*p, m);
                        }
                    }
                }
            }
        }
        if constexpr (RUN) {
            // one reduction per step over the group
#pragma unroll
            for (int c = 0; c < (RUN ? NCOL : 1); ++c) {
                if (c < S || c == SMAX) {
                    const u64 m = group_max<SUB>(run[c]);
                    if (writer) tab[slot * NCOL + c] = m;
                }
            }
        }
    }
    __syncthreads();

    for (int i = tid; i < SPW * S; i += WG) {
        const int jj = i / S;
        const int s = i - jj * S;
        const int64_t tt = tb + jj;
        if (tt >= T) break;
        u64 F = 0, Fr = 0;
#pragma unroll
        for (int qd = 0; qd < SPS; ++qd) {
            F = umax64(F, tab[(jj * SPS + qd) * NCOL + SMAX]);
            Fr = umax64(Fr, tab[(jj * SPS + qd) * NCOL + s]);
        }
        gain[tt * S + s] = (int64_t)F - (int64_t)Fr;
        if (s == 0) makespan[tt] = (int64_t)F;
    }
}

// Any number of stages (past what the registers of k_exposure_gain hold):
// for each rank tile the step group makes two passes over the stages, the
// rank totals first and then every stage's candidate max (the durations of
// the tile are read twice).  The group's last lane keeps the maxima over
// tiles in the step's own out_gain row (the replaced-stage maxima) and
// out_makespan entry (F), and after a barrier the workgroup turns the rows
// into gains.  Slots past R re-read rank r0, which cannot change a max.
template <int VEC, int K, int G, int WG>
__global__ __launch_bounds__(WG) void k_exposure_gain_wide(
    const int64_t* __restrict__ d, const int64_t* __restrict__ btilde, int64_t T, int R, int S,
    int64_t window, int64_t* __restrict__ gain, int64_t* __restrict__ makespan)
{
    static_assert(K % VEC == 0 && G <= 64 && WG % G == 0, "one writer lane per step");
    constexpr int SPW = WG / G;
    constexpr int NLD = K / VEC;
    constexpr int RT = G * K;
    const int tid = threadIdx.x;
    const int gl = tid % G;
    const bool writer = gl == G - 1;
    const int64_t tb = xcd_block() * SPW;
    const int64_t t = tb + tid / G;
    if (t < T) {
        const int64_t* dt = d + t * (int64_t)S * R;
        const int64_t* bw = btilde + (t / window) * (int64_t)S * R;
        u64* fr = reinterpret_cast<u64*>(gain) + t * S;  // replaced-stage maxima so far
        u64* fm = reinterpret_cast<u64*>(makespan) + t;  // F so far
        for (int r0 = 0; r0 < R; r0 += RT) {
            int idx[NLD];
#pragma unroll
            for (int l = 0; l < NLD; ++l) {
                const int r = r0 + (l * G + gl) * VEC;
                idx[l] = r < R ? r : r0;
            }
            auto load = [&](const int64_t* row, int l, int64_t* x) {
                if (VEC == 2) {
                    const v2i64 a = *reinterpret_cast<const v2i64*>(row + idx[l]);
                    x[0] = a.x;
                    x[VEC - 1] = a.y;
                } else {
                    x[0] = row[idx[l]];
                }
            };
            int64_t tot[K];
#pragma unroll
            for (int k = 0; k < K; ++k) tot[k] = 0;
            for (int s = 0; s < S; ++s) {
#pragma unroll
                for (int l = 0; l < NLD; ++l) {
                    int64_t x[VEC];
                    load(dt + (int64_t)s * R, l, x);
#pragma unroll
                    for (int e = 0; e < VEC; ++e) tot[l * VEC + e] += x[e];
                }
            }
            u64 f = 0;
#pragma unroll
            for (int k = 0; k < K; ++k) f = umax64(f, (u64)tot[k]);
            f = group_max<G>(f);
            if (writer) *fm = r0 == 0 ? f : umax64(*fm, f);
            for (int s = 0; s < S; ++s) {
                u64 m = 0;
#pragma unroll
                for (int l = 0; l < NLD; ++l) {
                    int64_t x[VEC], y[VEC];
                    load(dt + (int64_t)s * R, l, x);
                    load(bw + (int64_t)s * R, l, y);
#pragma unroll
                    for (int e = 0; e < VEC; ++e) {
                        const int64_t red = x[e] - y[e];
                        m = umax64(m, (u64)(tot[l * VEC + e] - (red > 0 ? red : 0)));
                    }
                }
                m = group_max<G>(m);
                if (writer) fr[s] = r0 == 0 ? m : umax64(fr[s], m);
            }
        }
    }
    __syncthreads();  // the writer lanes' maxima are visible to the workgroup
    for (int i = tid; i < SPW * S; i += WG) {
        const int jj = i / S;
        const int64_t tt = tb + jj;
        if (tt >= T) break;
        const int64_t idx = tt * S + (i - jj * S);
        gain[idx] = makespan[tt] - gain[idx];
    }
}

// Steps of 4097 to 16384 ranks and up to 16 stages: the ranks near the
// frontier first.  Replacing stage s lowers a rank's total by delta >= 0, so
// with v = F - P_S (F = max_r P_S) a rank whose v is at least D contributes
// at most F - D to max_r (P_S - delta); when the maximum over the set
// Q = {r : v < D} reaches F - D it is the maximum over all ranks.  One
// workgroup per step keeps the rank totals in registers (16 per lane: one
// pass over the step's durations, two chunks of loads per stage, the waves
// kept on one stage row by a barrier), picks D by radix passes over v
// (256-bin histograms, as in the selects) so that Q holds at least kNearMin
// ranks (every rank up to the one of rank kNearMin - 1 in ascending v, and
// the rest of its bin in the last pass) and at most kNearCap, reads the
// durations and baseline of Q's ranks only, and folds every stage's maximum
// over Q with LDS atomics.  If some stage's maximum falls below F - D (a
// gain larger than D), or more than kNearCap ranks sit at the smallest
// values of v, the workgroup makes a second pass over the step's durations
// and baseline and takes the maxima over all ranks.  The totals are 64-bit
// (32-bit ones ran 0.5% faster but made every step past 2^32 ns, 4.3 s, a
// second launch).  Measured on MI355X: one 16-wave workgroup per CU beat
// two at a 64-VGPR cap by 5%; loading a stage in one chunk, 3% slower;
// without the stage barrier, 2% slower; at 4096 ranks the per-step kernel
// stays ahead (0.63 against 0.64-0.66 ms).
constexpr int kNearMin = 32;
constexpr int kNearCap = 512;

// digit and candidate tests of the bound's radix passes, on 64-bit values or
// on 32-bit ones (totals spanning less than 2^32: lo <= 24, hi <= 32, a
// prefix below 2^(32 - hi)), which keep the shifts and compares in single
// VALU instructions
__device__ __forceinline__ int near_first_bin(u64 v, int lo) { return sel_first_bin(v, lo); }
__device__ __forceinline__ int near_bin(u64 v, int lo, int hi, u64 prefix) { return sel_bin(v, lo, hi, prefix); }
__device__ __forceinline__ int near_first_bin(uint32_t v, int lo) { return (int)(v >> lo); }
__device__ __forceinline__ int near_bin(uint32_t v, int lo, int hi, u64 prefix)
{
    return (hi >= 32 || (v >> hi) == (uint32_t)prefix) ? (int)((v >> lo) & ((1u << (hi - lo)) - 1u)) : -1;
}
constexpr int kNearK = 16;  // ranks per lane

template <int WG, bool FULL>
__global__ __launch_bounds__(WG) __attribute__((amdgpu_waves_per_eu(4))) void k_exposure_gain_near(
    const int64_t* __restrict__ d, const int64_t* __restrict__ btilde, int64_t T, int R, int S,
    int64_t window, int64_t* __restrict__ gain, int64_t* __restrict__ makespan)
{
    constexpr int K = kNearK;
    constexpr int NW = WG / 64;
    constexpr int NLD = K / 2;
    constexpr int CH = 2;  // chunks of loads per stage
    constexpr int SMAX = 16;
    __shared__ __align__(16) uint32_t hist[kSelWords];
    __shared__ u64 red_max[NW], red_min[NW];
    __shared__ uint32_t sel[3];
    __shared__ int q_rank[kNearCap];
    __shared__ u64 q_tot[kNearCap];
    __shared__ uint32_t q_n, all_ranks;
    __shared__ int top_rank;  // a rank whose total is F
    __shared__ u64 cand[SMAX];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int64_t t = xcd_block();
    if (t >= T) return;  // uniform (the grid is T)
    const int64_t* dt = d + t * (int64_t)S * R;
    const int64_t* bw = btilde + (t / window) * (int64_t)S * R;

    bool ok[NLD];
    int idx[NLD];
#pragma unroll
    for (int l = 0; l < NLD; ++l) {
        const int r = (l * WG + tid) * 2;
        ok[l] = FULL || r < R;
        idx[l] = ok[l] ? r : 0;
    }
    // the rank totals P_S (slots past R stay 0 and are left out below)
    u64 tot[K];
#pragma unroll
    for (int k = 0; k < K; ++k) tot[k] = 0;
    for (int s = 0; s < S; ++s) {
        const auto rs = buffer_rsrc(dt + (int64_t)s * R, (uint32_t)R * 8u);
#pragma unroll
        for (int ch = 0; ch < CH; ++ch) {
            v2i64 xs[NLD / CH];
#pragma unroll
            for (int l = 0; l < NLD / CH; ++l) {
                const int ll = ch * (NLD / CH) + l;
                xs[l] = FULL ? buffer_load16_nt(rs, (uint32_t)tid * 16u, (uint32_t)(ll * WG * 16))
                             : buffer_load16_nt(rs, (uint32_t)idx[ll] * 8u, 0u);
            }
            __builtin_amdgcn_sched_barrier(0);  // the chunk's loads all in flight first
#pragma unroll
            for (int l = 0; l < NLD / CH; ++l) {
                const int ll = ch * (NLD / CH) + l;
                tot[2 * ll] += ok[ll] ? (u64)xs[l].x : 0ull;
                tot[2 * ll + 1] += ok[ll] ? (u64)xs[l].y : 0ull;
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        __builtin_amdgcn_s_barrier();  // the waves read a stage's row together
    }
    // F and the smallest total over the workgroup
    u64 mx = 0, mn = ~0ull;
#pragma unroll
    for (int k = 0; k < K; ++k) {
        if (ok[k / 2]) {
            mx = umax64(mx, tot[k]);
            mn = umin64(mn, tot[k]);
        }
    }
    mx = group_max<64>(mx);
    mn = ~group_max<64>(~mn);
    if (lane == 63) {
        red_max[wave] = mx;
        red_min[wave] = mn;
    }
    if (tid < SMAX) cand[tid] = 0;
    if (tid == 0) {
        q_n = 0;
        all_ranks = 0;
    }
    __syncthreads();
    u64 F = 0, Pmin = ~0ull;
#pragma unroll
    for (int i = 0; i < NW; ++i) {
        F = umax64(F, red_max[i]);
        Pmin = umin64(Pmin, red_min[i]);
    }
    // the bound D: Q = {v < D} with kNearMin <= |Q| <= kNearCap, by radix
    // passes over v = F - P_S; in 32 bits when the totals span less than
    // 2^32 (every workload here), else in 64
    u64 D = 0;
    bool have_q = false;
    auto find_bound = [&](auto vt) {
        typedef decltype(vt) VT;
        VT v[K];
#pragma unroll
        for (int k = 0; k < K; ++k) v[k] = (VT)(F - tot[k]);
        int lo = sel_first_lo(F - Pmin), hi = 64;
        u64 prefix = 0;
        uint32_t kk = kNearMin - 1;  // R > 4096 ranks
        uint32_t below = 0;          // ranks in Q for certain (below the bracket)
        bool first = true;
        for (;;) {
            for (int i = tid; i < kSelWords; i += WG) hist[i] = 0;
            __syncthreads();
#pragma unroll
            for (int k = 0; k < K; ++k) {
                if (ok[k / 2]) {
                    const int bin = first ? near_first_bin(v[k], lo) : near_bin(v[k], lo, hi, prefix);
                    if (bin >= 0) atomicAdd(&hist[bin], 1u);
                }
            }
            __syncthreads();
            if (wave == 0) {
                uint32_t k2 = kk, dg, cn;
                sel_scan_wave(hist, lane, k2, dg, cn);
                if (lane == 0) {
                    sel[0] = dg;
                    sel[1] = k2;
                    sel[2] = cn;
                }
            }
            __syncthreads();
            const uint32_t dg = sel[0], kin = sel[1], cn = sel[2];
            const uint32_t lower = kk - kin;  // candidates in the lower bins of this pass
            prefix = first ? (u64)dg : (prefix << (hi - lo)) | (u64)dg;
            first = false;
            hi = lo;
            if (below + lower + cn <= (uint32_t)kNearCap) {
                D = (prefix + 1) << hi;
                have_q = true;
                return;
            }
            if (hi == 0) return;  // more than kNearCap ranks up to one value of v
            below += lower;
            kk = kin;
            lo = lo > 8 ? lo - 8 : 0;
        }
    };
    if (F != Pmin) {
        if (F - Pmin <= 0xFFFFFFFFull)
            find_bound((uint32_t)0);
        else
            find_bound((u64)0);
        // sel and hist are not touched again in this step
    }
    if (have_q) {
        // Q into LDS: a wave scan of the per-lane counts, one atomic per wave
        uint32_t cm = 0;
#pragma unroll
        for (int k = 0; k < K; ++k) cm |= (ok[k / 2] && F - tot[k] < D) ? (1u << k) : 0u;
        const uint32_t nc = (uint32_t)__popc(cm);
        const uint32_t incl = wave_scan_incl(nc);
        const uint32_t total = (uint32_t)__builtin_amdgcn_readlane((int)incl, 63);
        uint32_t wb = 0;
        if (lane == 63 && total != 0) wb = atomicAdd(&q_n, total);
        uint32_t pos = (uint32_t)__builtin_amdgcn_readlane((int)wb, 63) + incl - nc;
#pragma unroll
        for (int k = 0; k < K; ++k) {
            if ((cm >> k) & 1u) {
                if (pos < (uint32_t)kNearCap) {
                    q_rank[pos] = idx[k / 2] + (k & 1);
                    q_tot[pos] = tot[k];
                }
                ++pos;
            }
            if (ok[k / 2] && tot[k] == F) top_rank = idx[k / 2] + (k & 1);  // any one of them
        }
        __syncthreads();
        // first a rank whose total is F, for every stage: its replaced-stage
        // total F - delta bounds the stage's maximum from below, so only
        // ranks of Q whose total exceeds it can raise it (fewer scattered
        // reads: each costs a cache line)
        if (tid < S) {
            const int64_t e = dt[(int64_t)tid * R + top_rank] - bw[(int64_t)tid * R + top_rank];
            cand[tid] = F - (u64)(e > 0 ? e : 0);
        }
        __syncthreads();
        const uint32_t nq = min(q_n, (uint32_t)kNearCap);
        const uint32_t np = nq * (uint32_t)S;
        // the (rank of Q, stage) pairs left: four per thread in flight at once
        for (uint32_t i0 = tid; i0 < np; i0 += 4 * WG) {
            int64_t x[4], y[4];
            u64 tq[4];
            int sj[4];
            bool need[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const uint32_t i = i0 + (uint32_t)(j * WG);
                const uint32_t ii = i < np ? i : 0u;
                const uint32_t q = ii / (uint32_t)S;
                const int s = (int)(ii - q * (uint32_t)S);
                tq[j] = q_tot[q];
                sj[j] = s;
                need[j] = i < np && tq[j] > cand[s];  // cand only grows: a stale read is safe
                x[j] = 0;
                y[j] = 0;
                if (need[j]) {
                    const int r = q_rank[q];
                    x[j] = dt[(int64_t)s * R + r];
                    y[j] = bw[(int64_t)s * R + r];
                }
            }
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                if (need[j]) {
                    const int64_t e = x[j] - y[j];  // b >= 0: max(e, 0) <= x <= the total
                    atomicMax(&cand[sj[j]], tq[j] - (u64)(e > 0 ? e : 0));
                }
            }
        }
        __syncthreads();
        if (tid < S && cand[tid] + D < F) all_ranks = 1;  // a gain above D
        __syncthreads();
    }
    if (!have_q || all_ranks != 0) {
        // every rank: a second pass over the step's durations and baseline
        if (have_q) {
            if (tid < SMAX) cand[tid] = 0;  // the check above has read them
            __syncthreads();
        }
        for (int s = 0; s < S; ++s) {
            const auto rd = buffer_rsrc(dt + (int64_t)s * R, (uint32_t)R * 8u);
            const auto rb = buffer_rsrc(bw + (int64_t)s * R, (uint32_t)R * 8u);
            u64 m = 0;
#pragma unroll
            for (int ch = 0; ch < CH; ++ch) {
                v2i64 xs[NLD / CH], ys[NLD / CH];
#pragma unroll
                for (int l = 0; l < NLD / CH; ++l) {
                    const int ll = ch * (NLD / CH) + l;
                    const uint32_t vo = FULL ? (uint32_t)tid * 16u : (uint32_t)idx[ll] * 8u;
                    const uint32_t so = FULL ? (uint32_t)(ll * WG * 16) : 0u;
                    xs[l] = buffer_load16_nt(rd, vo, so);
                    ys[l] = buffer_load16_nt(rb, vo, so);
                }
#pragma unroll
                for (int l = 0; l < NLD / CH; ++l) {
                    const int ll = ch * (NLD / CH) + l;
#pragma unroll
                    for (int e = 0; e < 2; ++e) {
                        const int64_t e64 = (e == 0 ? xs[l].x : xs[l].y) - (e == 0 ? ys[l].x : ys[l].y);
                        const u64 c = tot[2 * ll + e] - (u64)(e64 > 0 ? e64 : 0);
                        m = ok[ll] ? umax64(m, c) : m;
                    }
                }
            }
            m = group_max<64>(m);
            if (lane == 63) atomicMax(&cand[s], m);
        }
        __syncthreads();
    }
    if (tid < S) gain[t * S + tid] = (int64_t)(F - cand[tid]);
    if (tid == 0) makespan[t] = (int64_t)F;
}

struct GainVariant {
    const void* fn;
    int G, WG;
};

template <int VEC, int K, int G, int WG, int SMAX, bool RUN = false>
GainVariant gain_variant()
{
    return GainVariant{reinterpret_cast<const void*>(&k_exposure_gain<VEC, K, G, WG, SMAX, RUN>), G,
                       WG};
}

// Two ranks per lane keep the deltas of up to 32 stages in registers
// (K = 1 at 64); G covers R in one tile up to 256 * K ranks, larger R loops
// over tiles.  Chosen by measurement on MI355X (wider K held more registers
// and ran up to 2x slower).
template <int VEC, int K, int SMAX>
GainVariant pick_gain_g(int R)
{
    if (R <= 16 * K) return gain_variant<VEC, K, 16, 64, SMAX>();
    if (R <= 64 * K) return gain_variant<VEC, K, 64, 256, SMAX>();
    // four or more tiles per step: running maxima (measured: 1-2% faster at
    // 4096 and 16384 ranks; at one or two tiles they only cost registers)
    if (SMAX <= 16 && R > 3 * 256 * K) return gain_variant<VEC, K, 256, 256, SMAX, (SMAX <= 16)>();
    return gain_variant<VEC, K, 256, 256, SMAX>();
}

template <int SMAX>
GainVariant pick_gain_s(int R, bool vec2)
{
    return vec2 ? pick_gain_g<2, 2, SMAX>(R) : pick_gain_g<1, 2, SMAX>(R);
}

// SMAX close above S: every unrolled stage past S still issues its two loads
// and holds its deltas, so 12 stages under SMAX = 16 ran 14-18% slower than
// under SMAX = 12 (and 6 under 8, 9% slower) on MI355X.
constexpr int kGainRegS = 64;  // stages whose deltas k_exposure_gain keeps in registers

GainVariant pick_gain(int R, int S, bool vec2)
{
    if (S <= 4) return pick_gain_s<4>(R, vec2);
    if (S <= 6) return pick_gain_s<6>(R, vec2);
    if (S <= 8) return pick_gain_s<8>(R, vec2);
    if (S <= 12) return pick_gain_s<12>(R, vec2);
    if (S <= 16) return pick_gain_s<16>(R, vec2);
    if (S <= 24) return pick_gain_s<24>(R, vec2);
    if (S <= 32) return pick_gain_s<32>(R, vec2);
    return pick_gain_g<1, 1, 64>(R);  // S <= kGainRegS
}

}  // namespace sfk

using namespace sfk;

SF_API int sf_exposure_gain(const int64_t* durations, const int64_t* baseline, int64_t T,
                            int32_t R, int32_t S, int64_t window, int64_t* out_gain,
                            int64_t* out_makespan, int64_t* out_window_gain,
                            int64_t* out_window_makespan, sf_stream_t stream)
{
    if (T < 0 || R < 1 || R > SF_MAX_R || S < 1 || window < 1) return SF_EINVAL;
    if (!fits(T, S, R, 8)) return SF_EINVAL;
    if (T == 0) return SF_OK;
    const int64_t W = sf_num_windows(T, window);
    if (!fits(W, S, R, 8)) return SF_EINVAL;
    const void* bufs[6] = {durations, baseline, out_gain, out_makespan, out_window_gain,
                           out_window_makespan};
    const int64_t sizes[6] = {T * S * (int64_t)R * 8, W * S * (int64_t)R * 8, T * S * 8, T * 8,
                              W * S * 8, W * 8};
    for (int a = 0; a < 6; ++a)
        if (!bufs[a] || !aligned(bufs[a], 8)) return SF_EINVAL;
    for (int a = 0; a < 6; ++a)
        for (int b = (a < 2 ? 2 : a + 1); b < 6; ++b)
            if (!disjoint(bufs[a], sizes[a], bufs[b], sizes[b])) return SF_EINVAL;

    const bool vec2 = (R % 2 == 0) && aligned(durations, 16) && aligned(baseline, 16);
    int Ri = R, Si = S;
    void* a1[] = {(void*)&durations, (void*)&baseline, (void*)&T, (void*)&Ri, (void*)&Si,
                  (void*)&window, (void*)&out_gain, (void*)&out_makespan};
    if (vec2 && S <= 16 && R > kNearK * 256 && R <= kNearK * 1024 && T <= INT32_MAX) {
        // the ranks near the frontier (all ranks where the bound does not settle it)
        const int WG = R <= kNearK * 512 ? 512 : 1024;
        const bool full = R == kNearK * WG;
        const void* fn =
            WG == 512 ? (full ? reinterpret_cast<const void*>(&k_exposure_gain_near<512, true>)
                              : reinterpret_cast<const void*>(&k_exposure_gain_near<512, false>))
                      : (full ? reinterpret_cast<const void*>(&k_exposure_gain_near<1024, true>)
                              : reinterpret_cast<const void*>(&k_exposure_gain_near<1024, false>));
        int rc = launch(fn, dim3((unsigned)T), dim3(WG), a1, 0, stream);
        if (rc != SF_OK) return rc;
        rc = launch_window_sum(out_gain, T, S, window, W, out_window_gain, stream);
        if (rc != SF_OK) return rc;
        return launch_window_sum(out_makespan, T, 1, window, W, out_window_makespan, stream);
    }
    const GainVariant v =
        S <= kGainRegS ? pick_gain(R, S, vec2)
                       : GainVariant{vec2 ? reinterpret_cast<const void*>(&k_exposure_gain_wide<2, 2, 64, 256>)
                                          : reinterpret_cast<const void*>(&k_exposure_gain_wide<1, 2, 64, 256>),
                                     64, 256};
    const int spw = v.WG / v.G;
    const int64_t blocks = (T + spw - 1) / spw;
    if (blocks > INT32_MAX) return SF_EINVAL;
    int rc = launch(v.fn, dim3((unsigned)blocks), dim3(v.WG), a1, 0, stream);
    if (rc != SF_OK) return rc;
    rc = launch_window_sum(out_gain, T, S, window, W, out_window_gain, stream);
    if (rc != SF_OK) return rc;
    return launch_window_sum(out_makespan, T, 1, window, W, out_window_makespan, stream);
}
