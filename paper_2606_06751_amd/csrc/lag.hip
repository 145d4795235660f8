// lag.hip -- lag kernel (Sec. 4): L[t,s] = max_r P - median_r P with the lower median
// (rank floor((R-1)/2) in ascending order) and its increment.
//
// One workgroup per step holds all R prefixes in registers (K per lane), and
// the next stage's durations are loaded while the current boundary is
// resolved.  At each boundary one block reduction gives F = max P and Pmin
// (and, for large R, the mean and standard deviation of P); the prefixes
// are rebased to u = P - Pmin (so the lag is F - Pmin - u(median)), and the
// median of u is found exactly by radix select.
//
// The first pass histograms 256 equal bins: over [0, F - Pmin] for small R,
// and for large R over a window around the mean.  For any distribution
// |mean - median| <= sd, so [mean - sd, mean + sd] (widened for rounding)
// holds the median, and the values below it are only counted.  Stragglers
// stretch F - Pmin far beyond the spread of the bulk, so bins over the whole
// range would leave most prefixes in a few bins; the window keeps the first
// pass selective.  Should rounding still leave the target rank outside the
// window, the pass is redone over [0, F - Pmin].  Later passes take 8 bits
// at a time of the values left, which after the first pass (usually a few
// per thousand of R) are compacted into an LDS list; a digit that isolates
// a single value ends the selection.

#include <math.h>

#include "sf_device.h"
#include "sf_host.h"

namespace sfk {

constexpr int kLagBins = 256;                // bins per histogram (8-bit digits)
constexpr int kLagPerLane = kLagBins / 64;   // bins scanned by each lane of wave 0
// bin b lives at word b + b / kLagPerLane: the bins a lane of wave 0 scans
// start kLagPerLane + 1 (odd) words after the previous lane's, so the scan
// reads hit distinct banks
constexpr int kLagBinWords = kLagBins + kLagBins / kLagPerLane;
constexpr int kLagBelow = kLagBinWords;      // count of values under the window
constexpr int kLagWords = kLagBinWords + 1;

__device__ __forceinline__ int lag_slot(int b) { return b + b / kLagPerLane; }

// DPP lane move of a 32-bit value in which lanes outside the row/bank masks,
// and lanes whose source lies outside their row, read 0
template <int CTRL, int ROW_MASK = 0xF, int BANK_MASK = 0xF>
__device__ __forceinline__ uint32_t dpp0(uint32_t v)
{
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, ROW_MASK, BANK_MASK, true);
}

template <int CTRL, int ROW_MASK = 0xF, int BANK_MASK = 0xF>
__device__ __forceinline__ u64 dpp0_64(u64 v)
{
    return ((u64)dpp0<CTRL, ROW_MASK, BANK_MASK>((uint32_t)(v >> 32)) << 32) |
           dpp0<CTRL, ROW_MASK, BANK_MASK>((uint32_t)v);
}

// inclusive prefix sum over the 64 lanes: row_shr 1..3 of the input, then
// row_shr 4 and 8 of the partial sums, then the row totals carried across
// rows by row_bcast 15 and 31
__device__ __forceinline__ uint32_t wave_scan_incl(uint32_t v)
{
    uint32_t t = v + dpp0<0x111>(v);
    t += dpp0<0x112>(v);
    t += dpp0<0x113>(v);
    t += dpp0<0x114, 0xF, 0xE>(t);
    t += dpp0<0x118, 0xF, 0xC>(t);
    t += dpp0<0x142, 0xA>(t);
    t += dpp0<0x143, 0xC>(t);
    return t;
}

// sum over each row of 16 lanes (in every lane of the row), by moves that
// pair distinct lanes: quad_perm [1,0,3,2], [2,3,0,1], row_half_mirror,
// row_mirror
template <typename V, typename MV>
__device__ __forceinline__ V row_sum(V v, MV move)
{
    v += move.template operator()<0xB1>(v);
    v += move.template operator()<0x4E>(v);
    v += move.template operator()<0x141>(v);
    v += move.template operator()<0x140>(v);
    return v;
}

struct MoveU64 {
    template <int CTRL>
    __device__ __forceinline__ u64 operator()(u64 v) const { return dpp0_64<CTRL>(v); }
};
struct MoveF64 {
    template <int CTRL>
    __device__ __forceinline__ double operator()(double v) const
    {
        return __longlong_as_double((long long)dpp0_64<CTRL>((u64)__double_as_longlong(v)));
    }
};

// sum over the 64 lanes, valid in lane 63 (rows 1 and 3 take row 0's and
// row 2's totals by row_bcast 15, then rows 2 and 3 take lane 31's)
__device__ __forceinline__ u64 wave_sum_u64(u64 v)
{
    v = row_sum(v, MoveU64{});
    v += dpp0_64<0x142, 0xA>(v);
    v += dpp0_64<0x143, 0xC>(v);
    return v;
}

__device__ __forceinline__ double wave_sum_f64(double v)
{
    v = row_sum(v, MoveF64{});
    v += __longlong_as_double((long long)dpp0_64<0x142, 0xA>((u64)__double_as_longlong(v)));
    v += __longlong_as_double((long long)dpp0_64<0x143, 0xC>((u64)__double_as_longlong(v)));
    return v;
}

// lane L's value, in every lane
template <int L>
__device__ __forceinline__ u64 lane_bcast(u64 v)
{
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, L);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), L);
    return ((u64)hi << 32) | lo;
}

template <int L>
__device__ __forceinline__ double lane_bcast_f64(double v)
{
    return __longlong_as_double((long long)lane_bcast<L>((u64)__double_as_longlong(v)));
}

// Add the active lanes' bins (-1: none) to the histogram.  When every active
// lane has the same bin one lane adds them all, so they do not serialise on
// one word.
__device__ __forceinline__ void lag_hist_add(uint32_t* h, int bin)
{
    const int first = __builtin_amdgcn_readfirstlane(bin);
    if (__ballot(bin != first) == 0) {
        const u64 active = __ballot(1);
        if (first >= 0 && (int)(threadIdx.x & 63) == __builtin_ctzll(active))
            atomicAdd(&h[lag_slot(first)], (uint32_t)__popcll(active));
    } else if (bin >= 0) {
        atomicAdd(&h[lag_slot(bin)], 1u);
    }
}

// Selection state: the candidates are the keys v with v >> hi == prefix,
// and a pass histograms their bits [lo, hi) (hi - lo <= 8).  Returns the
// digit, or -1 for a key that is not a candidate.
__device__ __forceinline__ int lag_bin(u64 v, int lo, int hi, u64 prefix)
{
    const bool match = hi >= 64 || (v >> hi) == prefix;
    return match ? (int)((v >> lo) & ((1u << (hi - lo)) - 1u)) : -1;
}

// smallest s with (v >> s) < 256: bins of width 2^s cover [0, v]
__device__ __forceinline__ int lag_width_log2(u64 v)
{
    const int nbits = v == 0 ? 0 : 64 - __builtin_clzll(v);
    return nbits > 8 ? nbits - 8 : 0;
}

// WIN: window the first pass around the mean; LCAP: capacity of the
// candidate list (0: every pass reads the registers)
template <int VEC, int K, int WG, bool WIN, int LCAP>
__global__ __launch_bounds__(WG) void k_frontier_lag(const int64_t* __restrict__ d, int64_t T,
                                                     int R, int S, int64_t* __restrict__ lag,
                                                     int64_t* __restrict__ lag_inc)
{
    static_assert(K % VEC == 0 && WG % 64 == 0 && WG / 64 <= 16, "shape");
    constexpr int NW = WG / 64;
    constexpr int NLD = K / VEC;
    // per-wave partials of the block reduction, double-buffered by stage
    // parity: a wave may write stage s+1's while another still reads stage
    // s's (when a boundary needs no radix pass there is no barrier between)
    __shared__ u64 red_max[2][NW], red_min[2][NW], red_c[2][NW], red_s1[2][NW];
    __shared__ double red_s2[2][NW];
    __shared__ uint32_t red_n[2][NW];
    // two histograms used alternately: while wave 0 scans one, the other
    // waves clear the other for the next pass
    __shared__ uint32_t hist[2][kLagWords];
    __shared__ u64 sel[3];     // chosen digit, rank within it, its count (0: none)
    __shared__ u64 found_u;    // the one remaining key, when a digit isolates it
    __shared__ u64 list[LCAP > 0 ? LCAP : 1];  // candidate keys after the first pass
    __shared__ uint32_t list_n;                // fill position of the list

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int64_t t = blockIdx.x;
    if (t >= T) return;  // uniform over the workgroup (the grid is T)
    const int64_t* dt = d + t * (int64_t)S * R;

    bool ok[NLD];
    int idx[NLD];
#pragma unroll
    for (int l = 0; l < NLD; ++l) {
        const int r = (l * WG + tid) * VEC;
        ok[l] = r < R;
        idx[l] = ok[l] ? r : 0;
    }
    // the durations of the next stage, loaded one stage ahead
    int64_t nx[K];
    auto load_stage = [&](int s) {
        const int64_t* row = dt + (int64_t)s * R;
#pragma unroll
        for (int l = 0; l < NLD; ++l) {
            if (VEC == 2) {
                const v2i64 x = __builtin_nontemporal_load(reinterpret_cast<const v2i64*>(row + idx[l]));
                nx[l * VEC] = x.x;
                nx[l * VEC + VEC - 1] = x.y;
            } else {
                nx[l] = __builtin_nontemporal_load(row + idx[l]);
            }
        }
    };
    load_stage(0);

    u64 P[K];
#pragma unroll
    for (int k = 0; k < K; ++k) P[k] = 0;
    for (int i = tid; i < 2 * kLagWords; i += WG) (&hist[0][0])[i] = 0;
    if (tid == 0) list_n = 0;
    int cur = 0;  // the histogram that is clear at the start of a pass
    int64_t L_prev = 0;
    const uint32_t target = (uint32_t)((R - 1) / 2);
    const double inv_r = 1.0 / (double)R;

    for (int s = 0; s < S; ++s) {
#pragma unroll
        for (int k = 0; k < K; ++k) P[k] += ok[k / VEC] ? (u64)nx[k] : 0ull;
        // moments about the wave's first prefix (a slot of lane 0, valid
        // whenever any slot of the wave is), so that a tiny spread on large
        // prefixes does not cancel away
        const u64 cw = lane_bcast<0>(P[0]);
        u64 lmax = 0, lmin = ~0ull, ls1 = 0;
        double ls2 = 0.0;
        uint32_t nw = 0;  // valid prefixes in the wave
#pragma unroll
        for (int k = 0; k < K; ++k) {
            if (WIN) nw += (uint32_t)__popcll(__ballot(ok[k / VEC]));
            if (ok[k / VEC]) {
                lmax = umax64(lmax, P[k]);
                lmin = umin64(lmin, P[k]);
                if (WIN) {
                    const u64 dv = P[k] - cw;
                    ls1 += dv;
                    const double x = (double)(int64_t)dv;
                    ls2 = fma(x, x, ls2);
                }
            }
        }
        if (s + 1 < S) load_stage(s + 1);
        // block max, min (as the max of complements) and moments
        lmax = group_max<64>(lmax);
        lmin = ~group_max<64>(~lmin);
        if (WIN) {
            ls1 = wave_sum_u64(ls1);
            ls2 = wave_sum_f64(ls2);
        }
        const int pb = s & 1;
        if (lane == 63) {
            red_max[pb][wave] = lmax;
            red_min[pb][wave] = lmin;
            if (WIN) {
                red_c[pb][wave] = cw;
                red_s1[pb][wave] = ls1;
                red_s2[pb][wave] = ls2;
                red_n[pb][wave] = nw;
            }
        }
        __syncthreads();
        // every wave combines the partials the same way, lane w taking
        // wave w's (w < NW <= 16: row 0), so the results are uniform
        const bool has = lane < NW;
        const int wl = has ? lane : 0;
        const u64 F = lane_bcast<0>(group_max<16>(has ? red_max[pb][wl] : 0ull));
        const u64 Pmin = ~lane_bcast<0>(group_max<16>(has ? ~red_min[pb][wl] : 0ull));
        // rebase: from here on P holds u = P - Pmin (the minimum is 0)
        const u64 range = F - Pmin;
#pragma unroll
        for (int k = 0; k < K; ++k) P[k] -= Pmin;
        u64 um = 0;  // u of the median (0 when every u is 0)
        if (range != 0) {
            u64 wlo = 0, whi = range;
            if (WIN) {
                // window [wlo, whi] around the mean of u, of half-width sd
                // plus a margin for the rounding of mean and sd
                const u64 pc = red_c[pb][wl];
                const u64 ps1 = has ? red_s1[pb][wl] : 0ull;
                const double ps2 = has ? red_s2[pb][wl] : 0.0;
                const uint32_t pn = has ? red_n[pb][wl] : 0u;
                // sum of u over the block: n (c - Pmin) + S1 per wave (exact)
                const u64 su = lane_bcast<0>(row_sum((u64)pn * (pc - Pmin) + ps1, MoveU64{}));
                const double mu = (double)su * inv_r;
                // sum of squared deviations from the mean, wave by wave:
                // S2 - 2 (mean - c) S1 + n (mean - c)^2, with mean - c = mu - (c - Pmin)
                const double dl = mu - (double)(pc - Pmin);
                const double m2 = lane_bcast_f64<0>(row_sum(
                    has ? ps2 - 2.0 * dl * (double)(int64_t)ps1 + (double)pn * dl * dl : 0.0, MoveF64{}));
                const double var = m2 * inv_r;
                const double sd = var > 0.0 ? sqrt(var) : 0.0;
                const double half = 1.0625 * sd + 16.0;
                const double lo_d = mu - half, hi_d = mu + half;
                if (lo_d > 0.0) wlo = (u64)lo_d;                     // NaN: 0
                if (hi_d < (double)range) whi = (u64)hi_d + 1;       // NaN: range
                if (wlo > whi) {
                    wlo = 0;
                    whi = range;
                }
            }
            // keys v = u - base, held in P for the selection (values under
            // the window wrap to v >= 2^63)
            u64 base = wlo;
#pragma unroll
            for (int k = 0; k < K; ++k) P[k] -= base;
            int lo = lag_width_log2(whi - wlo), hi = lo + 8;
            u64 prefix = 0;
            uint32_t kk = target;
            bool first = true;                // the window pass
            bool window = WIN && base != 0;   // this pass counts the values under the window
            bool in_list = false;
            uint32_t n = 0;  // list length, once in_list
            for (;;) {
                // histogram of the next digit of the candidates (and, in
                // the window pass, the count of values under the window)
                uint32_t* h = hist[cur];
                if (LCAP > 0 && in_list) {
                    for (uint32_t i = tid; i < n; i += WG) lag_hist_add(h, lag_bin(list[i], lo, hi, prefix));
                } else {
                    uint32_t below = 0;
#pragma unroll
                    for (int k = 0; k < K; ++k) {
                        lag_hist_add(h, ok[k / VEC] ? lag_bin(P[k], lo, hi, prefix) : -1);
                        if (WIN && window)
                            below += (uint32_t)__popcll(__ballot(ok[k / VEC] && (int64_t)P[k] < 0));
                    }
                    if (WIN && below != 0 && lane == 0) atomicAdd(&h[kLagBelow], below);
                }
                __syncthreads();
                if (wave == 0) {
                    // scan of the bins, kLagPerLane per lane, behind the
                    // values under the window; the lane whose bins hold the
                    // target rank names the bin
                    uint32_t c[kLagPerLane];
                    const uint32_t* hl = h + lane * (kLagPerLane + 1);  // lag_slot(lane * kLagPerLane)
                    uint32_t part = 0;
#pragma unroll
                    for (int i = 0; i < kLagPerLane; ++i) {
                        c[i] = hl[i];
                        part += c[i];
                    }
                    const uint32_t incl = (WIN ? h[kLagBelow] : 0u) + wave_scan_incl(part);
                    uint32_t cum = incl - part;
                    bool found = false;
                    if (cum <= kk && kk < incl) {
#pragma unroll
                        for (int i = 0; i < kLagPerLane; ++i) {
                            if (!found && kk < cum + c[i]) {
                                found = true;
                                sel[0] = (u64)(lane * kLagPerLane + i);
                                sel[1] = (u64)(kk - cum);
                                sel[2] = (u64)c[i];
                            }
                            cum += c[i];
                        }
                    }
                    // no lane: the target lies outside the window
                    if (__ballot(found) == 0 && lane == 0) sel[2] = 0;
                } else {
                    uint32_t* other = hist[cur ^ 1];
                    for (int i = tid - 64; i < kLagWords; i += WG - 64) other[i] = 0;
                }
                if (NW == 1) {
                    uint32_t* other = hist[cur ^ 1];
                    for (int i = tid; i < kLagWords; i += WG) other[i] = 0;
                }
                __syncthreads();
                // h is cleared during the scan of the next pass (or stage)
                cur ^= 1;
                const uint32_t count = (uint32_t)sel[2];
                if (count == 0) {
                    // the target rank lies outside the window: redo the
                    // pass over [0, range].  Later passes count exactly the
                    // candidates, which hold the target, so they cannot
                    // miss; should one, the loop ends rather than repeat.
                    if (!first) break;
#pragma unroll
                    for (int k = 0; k < K; ++k) P[k] += base;
                    base = 0;
                    lo = lag_width_log2(range);
                    hi = lo + 8;
                    first = window = false;
                    continue;
                }
                first = window = false;
                prefix = (prefix << (hi - lo)) | sel[0];
                kk = (uint32_t)sel[1];
                hi = lo;
                if (hi == 0) break;  // every bit chosen: v == prefix
                lo = lo > 8 ? lo - 8 : 0;
                // the candidates left are the keys with v >> hi == prefix
                if (count == 1) {
                    // one key has the chosen digits: its lane publishes it
                    if (LCAP > 0 && in_list) {
                        for (uint32_t i = tid; i < n; i += WG)
                            if (lag_bin(list[i], lo, hi, prefix) >= 0) found_u = list[i];
                    } else {
#pragma unroll
                        for (int k = 0; k < K; ++k)
                            if (ok[k / VEC] && lag_bin(P[k], lo, hi, prefix) >= 0) found_u = P[k];
                    }
                    __syncthreads();
                    prefix = found_u;
                    break;
                }
                if (LCAP > 0 && !in_list && count <= (uint32_t)LCAP) {
                    // compact the candidates into the list: a wave scan of
                    // the per-lane counts and one atomic per wave for its base
                    uint32_t nc = 0;
#pragma unroll
                    for (int k = 0; k < K; ++k)
                        nc += (ok[k / VEC] && lag_bin(P[k], lo, hi, prefix) >= 0) ? 1u : 0u;
                    const uint32_t incl = wave_scan_incl(nc);
                    const uint32_t total = (uint32_t)__builtin_amdgcn_readlane((int)incl, 63);
                    uint32_t wbase = 0;
                    if (lane == 63 && total != 0) wbase = atomicAdd(&list_n, total);
                    uint32_t pos = (uint32_t)__builtin_amdgcn_readlane((int)wbase, 63) + incl - nc;
#pragma unroll
                    for (int k = 0; k < K; ++k) {
                        if (ok[k / VEC] && lag_bin(P[k], lo, hi, prefix) >= 0) {
                            if (pos < (uint32_t)LCAP) list[pos] = P[k];  // always, as count <= LCAP
                            ++pos;
                        }
                    }
                    __syncthreads();
                    // every wave has taken its base: reset for the next boundary
                    // (its next use follows at least one more barrier)
                    if (tid == 0) list_n = 0;
                    in_list = true;
                    n = count;
                }
            }
            um = base + prefix;
#pragma unroll
            for (int k = 0; k < K; ++k) P[k] += base;  // back to u for the next stage
            // sel, found_u and the list are next written after the next
            // stage's reduction barrier, which every thread passes only
            // after reading them here
        }
        const int64_t L = (int64_t)(range - um);
        if (tid == 0) {
            lag[t * S + s] = L;
            lag_inc[t * S + s] = L - L_prev;
        }
        L_prev = L;
    }
}

struct LagVariant {
    const void* fn;
    int WG;
};

template <int VEC, int K, int WG>
LagVariant lag_variant()
{
    // window pass from 512 slots up (below, its moments cost more than the
    // passes it saves); candidate list: a quarter of the slots, at most
    // 32 KB, none when a lane holds so few values that the registers are as
    // cheap to re-read
    constexpr bool WIN = K * WG >= 512;
    constexpr int LCAP = K <= 2 ? 0 : (K * WG / 4 < 4096 ? K * WG / 4 : 4096);
    return LagVariant{reinterpret_cast<const void*>(&k_frontier_lag<VEC, K, WG, WIN, LCAP>), WG};
}

// One step per workgroup with all R prefixes in registers.
template <int VEC>
LagVariant pick_lag(int R)
{
    if (R <= 128) return lag_variant<VEC, 2, 64>();
    if (R <= 256) return lag_variant<VEC, 4, 64>();
    if (R <= 512) return lag_variant<VEC, 2, 256>();
    if (R <= 1024) return lag_variant<VEC, 4, 256>();
    if (R <= 2048) return lag_variant<VEC, 8, 256>();
    if (R <= 4096) return lag_variant<VEC, 16, 256>();
    if (R <= 8192) return lag_variant<VEC, 16, 512>();
    return lag_variant<VEC, 16, 1024>();  // R <= SF_MAX_R_LAG = 16384
}

}  // namespace sfk

using namespace sfk;

SF_API int sf_frontier_lag(const int64_t* durations, int64_t T, int32_t R, int32_t S,
                           int64_t* out_lag, int64_t* out_lag_inc, sf_stream_t stream)
{
    if (T < 0 || R < 1 || R > SF_MAX_R_LAG || S < 1 || S > SF_MAX_S) return SF_EINVAL;
    if (!fits(T, S, R, 8)) return SF_EINVAL;
    if (T == 0) return SF_OK;
    if (T > INT32_MAX) return SF_EINVAL;  // one workgroup per step
    if (!durations || !out_lag || !out_lag_inc) return SF_EINVAL;
    if (!aligned(durations, 8) || !aligned(out_lag, 8) || !aligned(out_lag_inc, 8))
        return SF_EINVAL;
    const int64_t nd = T * S * (int64_t)R * 8, no = T * S * 8;
    if (!disjoint(durations, nd, out_lag, no) || !disjoint(durations, nd, out_lag_inc, no) ||
        !disjoint(out_lag, no, out_lag_inc, no))
        return SF_EINVAL;
    const bool vec2 = (R % 2 == 0) && aligned(durations, 16);
    const LagVariant v = vec2 ? pick_lag<2>(R) : pick_lag<1>(R);
    int Ri = R, Si = S;
    void* args[] = {(void*)&durations, (void*)&T, (void*)&Ri, (void*)&Si, (void*)&out_lag,
                    (void*)&out_lag_inc};
    return launch(v.fn, dim3((unsigned)T), dim3(v.WG), args, 0, stream);
}
