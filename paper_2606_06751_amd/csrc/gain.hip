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

#include "sf_device.h"
#include "sf_host.h"

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
            if (RUN) {
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
                    if (RUN) {
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
        if (RUN) {
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
    const GainVariant v =
        S <= kGainRegS ? pick_gain(R, S, vec2)
                       : GainVariant{vec2 ? reinterpret_cast<const void*>(&k_exposure_gain_wide<2, 2, 64, 256>)
                                          : reinterpret_cast<const void*>(&k_exposure_gain_wide<1, 2, 64, 256>),
                                     64, 256};
    const int spw = v.WG / v.G;
    const int64_t blocks = (T + spw - 1) / spw;
    if (blocks > INT32_MAX) return SF_EINVAL;
    int Ri = R, Si = S;
    void* a1[] = {(void*)&durations, (void*)&baseline, (void*)&T, (void*)&Ri, (void*)&Si,
                  (void*)&window, (void*)&out_gain, (void*)&out_makespan};
    int rc = launch(v.fn, dim3((unsigned)blocks), dim3(v.WG), a1, 0, stream);
    if (rc != SF_OK) return rc;
    rc = launch_window_sum(out_gain, T, S, window, W, out_window_gain, stream);
    if (rc != SF_OK) return rc;
    return launch_window_sum(out_makespan, T, 1, window, W, out_window_makespan, stream);
}
