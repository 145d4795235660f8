// lag.hip -- lag kernel (Sec. 4): L[t,s] = max_r P - median_r P with the lower median
// (rank floor((R-1)/2) in ascending order) and its increment; and, by the
// same selection applied to each stage's durations instead of the prefixes,
// the raw rank spread max_r d - median_r d of Sec. 6.2.
//
// One workgroup per step holds all R prefixes in registers (K per lane), and
// the next stage's durations are loaded while the current boundary is
// resolved.  At each boundary a block reduction gives F = max P and Pmin;
// the prefixes are rebased to u = P - Pmin (so the lag is F - Pmin -
// u(median)), and the median of u is found exactly by radix select.  The
// first pass histograms 256 equal bins fitted to the top bits of F - Pmin;
// later passes take the next 8 bits of the values left, which once few
// enough are compacted into an LDS list so that later passes read only
// them.  A digit that isolates a single value ends the selection, and the
// lane holding that value writes the boundary's outputs.  The barriers
// inside a step order LDS accesses only (lds_barrier), so the next stage's
// loads stay in flight across them (a full barrier waits for every load of
// the wave: measured 11% slower at 4096 ranks).

#include "sf_device.h"
#include "sf_host.h"
#include "sf_select.h"

#include <type_traits>

namespace sfk {

constexpr int kLagWords = kSelWords;

// 32-bit twin of group_max (result valid in the last lane of each group)
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ uint32_t dpp_move32(uint32_t v)
{
    return (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, CTRL, ROW_MASK, 0xF, false);
}

template <int SUB>
__device__ __forceinline__ uint32_t group_max32(uint32_t v)
{
    if (SUB >= 2) v = max(v, dpp_move32<0xB1, 0xF>(v));
    if (SUB >= 4) v = max(v, dpp_move32<0x4E, 0xF>(v));
    if (SUB >= 8) v = max(v, dpp_move32<0x141, 0xF>(v));
    if (SUB >= 16) v = max(v, dpp_move32<0x140, 0xF>(v));
    if (SUB >= 32) v = max(v, dpp_move32<0x142, 0xA>(v));
    if (SUB >= 64) v = max(v, dpp_move32<0x143, 0xC>(v));
    return v;
}

// lane 0's value, in every lane
__device__ __forceinline__ u64 lane0(u64 v) { return lane_value(v, 0); }

// The select's digit and candidate tests on the held values: 64-bit as in
// sf_select.h, and 32-bit for the narrow pass (its values, and so its
// range, stay below 2^32: lo <= 24, hi <= 32, a prefix below 2^(32 - hi)),
// which keeps the shifts and compares in single VALU instructions.
__device__ __forceinline__ bool held_match(u64 u, int hi, u64 prefix) { return sel_match(u, hi, prefix); }
__device__ __forceinline__ int held_bin(u64 u, int lo, int hi, u64 prefix) { return sel_bin(u, lo, hi, prefix); }
__device__ __forceinline__ int held_first_bin(u64 u, int lo) { return sel_first_bin(u, lo); }
__device__ __forceinline__ bool held_match(uint32_t u, int hi, u64 prefix)
{
    return hi >= 32 || (u >> hi) == (uint32_t)prefix;
}
__device__ __forceinline__ int held_bin(uint32_t u, int lo, int hi, u64 prefix)
{
    return held_match(u, hi, prefix) ? (int)((u >> lo) & ((1u << (hi - lo)) - 1u)) : -1;
}
__device__ __forceinline__ int held_first_bin(uint32_t u, int lo) { return (int)(u >> lo); }

// One step per workgroup: at every stage, out[t][s] = max - lower median
// over ranks of the prefixes (PREFIX: the lag, and out_inc gets its
// increment) or of the stage's durations themselves (the raw rank spread;
// out_inc is not written).  LCAP: capacity of the candidate list (0: every
// pass reads the registers).  At least 4 waves per SIMD, so at most 128
// VGPRs: without the cap the raw spread's allocation lands above it.
//
// How a pass's histogram is resolved (SCAN_ALL): wave 0 scans it and
// publishes the digit through LDS, which takes a second barrier per pass,
// while the other waves clear the other of two histograms; or every wave
// scans it itself, with three histograms in rotation (pass p adds into
// hist[p % 3] and clears hist[(p + 1) % 3], last read in pass p - 2's
// scans), one barrier per pass.  Measured on MI355X: the per-wave scans free
// the registers that the raw spread otherwise spills at 4-16 waves per step
// (8-18% faster there), and cost the lag and the one-wave steps 1-7%.
// PUBU: wave 0 takes the chosen bin into wave-uniform registers before lane
// 0 publishes it, instead of the finding lane publishing it; the same work,
// compiled differently (7% faster for the lag with 16 prefixes per lane on
// 1-4 waves, up to 8% slower elsewhere).
//
// NARROW: the values are held in 32 bits.  Steps whose rebased prefixes
// (P - min_r P, rebased at every boundary) and durations stay below 2^32 ns
// (4.29 s; every workload here) need no more, so the values, the loads in
// flight and the reductions take half the registers: at most 64 VGPRs,
// twice the workgroups per CU, which cover each other's barriers.  The stage's loads are consumed in
// chunks so that few hold registers at once.  A step where a duration or a
// rebased prefix reaches 2^32 (detected on the load, by the high word or the
// carry of the 32-bit add) is handed over: once the step is done, its
// out[t][0] is set to kRedo; a second launch of the 64-bit kernel with REDO
// recomputes exactly those steps (every other workgroup of it returns at
// once).  Both compute the same lower median of the same values.
constexpr int64_t kRedo = INT64_MIN;  // outputs are >= 0 under the data contract

template <bool PREFIX, int VEC, int K, int WG, int LCAP, bool PUBU, bool FULL, bool NARROW,
          bool REDO>
__global__ __launch_bounds__(WG) __attribute__((amdgpu_waves_per_eu(NARROW && K <= 16 ? 8 : 4))) void k_median_spread(const int64_t* __restrict__ d, int64_t T,
                                                      int R, int S, int64_t* __restrict__ out,
                                                      int64_t* __restrict__ out_inc)
{
    static_assert(K % VEC == 0 && WG % 64 == 0 && WG / 64 <= 16, "shape");
    static_assert(!NARROW || (VEC == 2 && !REDO), "the narrow pass takes 16-byte loads");
    typedef typename std::conditional<NARROW, uint32_t, u64>::type V;
    constexpr int NW = WG / 64;
    constexpr int NLD = K / VEC;
    constexpr bool SCAN_ALL = !PREFIX && NW > 1;
    constexpr int NH = SCAN_ALL ? 3 : 2;  // histograms
    // per-wave max/min partials, double-buffered by stage parity: a wave
    // may write stage s+1's while another still reads stage s's (when a
    // boundary needs no radix pass there is no barrier between)
    __shared__ u64 red_max[2][NW], red_min[2][NW];
    __shared__ __attribute__((aligned(16))) uint32_t hist[NH][kLagWords];
    __shared__ uint32_t sel[3];  // wave 0's scan: chosen digit, rank within it, its count
    __shared__ V list[LCAP > 0 ? LCAP : 1];  // candidates, once few enough
    __shared__ uint32_t list_n;                // fill position of the list
    __shared__ int64_t lag_sh[2];              // L of the last two stages, by parity

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: LDS slots in SGPRs
    const int64_t t = xcd_block();
    if (t >= T) return;  // uniform over the workgroup (the grid is T)
    if (REDO && out[t * S] != kRedo) return;  // a step the narrow pass resolved
    const int64_t* dt = d + t * (int64_t)S * R;

    bool ok[NLD];
    int idx[NLD];
#pragma unroll
    for (int l = 0; l < NLD; ++l) {
        const int r = (l * WG + tid) * VEC;
        ok[l] = FULL || r < R;
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
    if (!NARROW) load_stage(0);

    V P[K];
#pragma unroll
    for (int k = 0; k < K; ++k) P[k] = 0;
    for (int i = tid; i < NH * kLagWords; i += WG) (&hist[0][0])[i] = 0;
    if (tid == 0) {
        list_n = 0;
        lag_sh[0] = 0;
        lag_sh[1] = 0;
    }
    bool wide_step = false;  // NARROW: some value of this step left 32 bits
    int cur = 0;  // the histogram of the next pass (clear)
    const uint32_t target = (uint32_t)((R - 1) / 2);

    for (int s = 0; s < S; ++s) {
        u64 lmax = 0, lmin = ~0ull;
        if constexpr (NARROW) {
            // the stage's 16-byte loads in CH chunks, each consumed before
            // the next is issued.  The lag's prefixes stay live across
            // stages: at 16 values per lane it takes four loads at a time
            // (with the select's tests in 32 bits this fits the 64-VGPR
            // budget; measured at 16384 ranks 3% faster than two at a time,
            // which the 64-bit tests forced); at 32 values, two at a time
            constexpr int CH = PREFIX ? (K == 16 ? 2 : NLD / 2) : (K <= 32 ? 2 : NLD / 4);
            // the stage row through a buffer resource: its base in SGPRs, a
            // lane's offset in one VGPR (FULL: the same for every load)
            const auto rs = buffer_rsrc(dt + (int64_t)s * R, (uint32_t)R * 8u);
            uint32_t mx = 0, mn = ~0u;
            bool wide = false;  // wave-uniform: some value of the wave left 32 bits
#pragma unroll
            for (int ch = 0; ch < CH; ++ch) {
                uint32_t w = 0;
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
                    // a slot pair past R (re-reading the row's first pair)
                    // keeps 0 and is left out of every reduction and pass
                    const bool okl = ok[ch * (NLD / CH) + l];
#pragma unroll
                    for (int e = 0; e < 2; ++e) {
                        const int k = (ch * (NLD / CH) + l) * 2 + e;
                        const u64 x = (u64)(e == 0 ? xs[l].x : xs[l].y);
                        const uint32_t lo = okl ? (uint32_t)x : 0u;
                        w |= okl ? (uint32_t)(x >> 32) : 0u;
                        if (PREFIX) {
                            const uint32_t np = (uint32_t)P[k] + lo;
                            w |= np < lo ? 1u : 0u;  // carry
                            P[k] = np;
                        } else {
                            P[k] = lo;
                        }
                        mx = max(mx, okl ? (uint32_t)P[k] : 0u);
                        mn = min(mn, okl ? (uint32_t)P[k] : ~0u);
                    }
                }
                wide = wide || __ballot(w != 0) != 0;
                __builtin_amdgcn_sched_barrier(0);
            }
            // a wave holding a value of 2^32 or more reports the maximum
            // ~0, which no 32-bit value reaches
            const u64 wmax = (u64)group_max32<64>(mx);
            const uint32_t nmn = group_max32<64>(~mn);
            lmax = wide ? ~0ull : wmax;
            lmin = (u64)(~nmn);
        } else {
#pragma unroll
            for (int k = 0; k < K; ++k) {
                if (ok[k / VEC]) {
                    P[k] = PREFIX ? P[k] + (u64)nx[k] : (u64)nx[k];
                    lmax = umax64(lmax, P[k]);
                    lmin = umin64(lmin, P[k]);
                }
            }
            if (s + 1 < S) load_stage(s + 1);
            // block max and min (min as the max of complements)
            lmax = group_max<64>(lmax);
            lmin = ~group_max<64>(~lmin);
        }
        const int pb = s & 1;
        if (lane == 63) {
            red_max[pb][wave] = lmax;
            red_min[pb][wave] = lmin;
        }
        lds_barrier();
        // every wave combines the partials the same way, lane w taking
        // wave w's (w < NW <= 16: row 0), so the results are uniform
        const bool has = lane < NW;
        const int wl = has ? lane : 0;
        const u64 F = lane0(group_max<16>(has ? red_max[pb][wl] : 0ull));
        const u64 Pmin = ~lane0(group_max<16>(has ? ~red_min[pb][wl] : 0ull));
        // a value left 32 bits (uniform: every wave read the same
        // partials); the step runs on, on values that no longer matter, and
        // is handed over at its end (an exit here costs the narrow lag 22
        // VGPRs of spills)
        if (NARROW) wide_step = wide_step || (F >> 32) != 0;
        // rebase: from here on P holds u = P - Pmin (the minimum is 0)
        const u64 range = F - Pmin;
#pragma unroll
        for (int k = 0; k < K; ++k) P[k] -= (V)Pmin;
        u64 um = 0;            // u of the median (0 when every u is 0)
        bool written = false;  // the lane holding the median wrote the outputs
        if (range != 0) {
            int lo = sel_first_lo(range), hi = lo + 8;
            u64 prefix = 0;
            uint32_t kk = target;
            bool first = true;     // every value is a candidate
            bool in_list = false;
            uint32_t n = 0;  // list length, once in_list
            for (;;) {
                // histogram of the next digit of the candidates
                uint32_t* h = hist[cur];
                if (SCAN_ALL) {
                    cur = cur == NH - 1 ? 0 : cur + 1;
                    for (int i = tid; i < kLagWords; i += WG) hist[cur][i] = 0;
                }
                if (LCAP > 0 && in_list) {
                    for (uint32_t i = tid; i < n; i += WG) sel_hist_add(h, held_bin(list[i], lo, hi, prefix));
                } else if (first) {
                    // one plain atomic per value (3-4% faster than adding
                    // runs of equal bins among a lane's values at once)
#pragma unroll
                    for (int k = 0; k < K; ++k)
                        if (ok[k / VEC]) atomicAdd(&h[held_first_bin(P[k], lo)], 1u);
                } else {
#pragma unroll
                    for (int k = 0; k < K; ++k)
                        sel_hist_add(h, ok[k / VEC] ? held_bin(P[k], lo, hi, prefix) : -1);
                }
                first = false;
                lds_barrier();
                uint32_t digit, count;
                if (SCAN_ALL) {
                    sel_scan_wave(h, lane, kk, digit, count);
                } else {
                    if (wave == 0 && PUBU) {
                        uint32_t dg, cn;
                        sel_scan_wave(h, lane, kk, dg, cn);
                        if (lane == 0) {
                            sel[0] = dg;
                            sel[1] = kk;
                            sel[2] = cn;
                        }
                    } else if (wave == 0) {
                        const uint4 b4 = sel_lane_bins(h, lane);
                        const uint32_t c[kSelPerLane] = {b4.x, b4.y, b4.z, b4.w};
                        const uint32_t part = c[0] + c[1] + c[2] + c[3];
                        const uint32_t incl = wave_scan_incl(part);
                        uint32_t cum = incl - part;
                        if (cum <= kk && kk < incl) {
                            bool found = false;
#pragma unroll
                            for (int i = 0; i < kSelPerLane; ++i) {
                                if (!found && kk < cum + c[i]) {
                                    found = true;
                                    sel[0] = (uint32_t)(lane * kSelPerLane + i);
                                    sel[1] = kk - cum;
                                    sel[2] = c[i];
                                }
                                cum += c[i];
                            }
                        }
                    } else {
                        uint32_t* other = hist[cur ^ 1];
                        for (int i = tid - 64; i < kLagWords; i += WG - 64) other[i] = 0;
                    }
                    if (NW == 1) {
                        uint32_t* other = hist[cur ^ 1];
                        for (int i = tid; i < kLagWords; i += WG) other[i] = 0;
                    }
                    lds_barrier();
                    // h is cleared during the scan of the next pass (or stage)
                    cur ^= 1;
                    digit = sel[0];
                    kk = sel[1];
                    count = sel[2];
                }
                prefix = (prefix << (hi - lo)) | (u64)digit;
                hi = lo;
                if (hi == 0) break;  // every bit chosen: u == prefix
                lo = lo > 8 ? lo - 8 : 0;
                // the candidates left are the values with u >> hi == prefix
                if (count == 1) {
                    // one value has the chosen digits: its lane writes the
                    // outputs (the previous stage's L is in lag_sh)
                    u64 u = 0;
                    bool holder = false;
                    if (LCAP > 0 && in_list) {
                        for (uint32_t i = tid; i < n; i += WG) {
                            if (held_match(list[i], hi, prefix)) {
                                u = list[i];
                                holder = true;
                            }
                        }
                    } else {
#pragma unroll
                        for (int k = 0; k < K; ++k) {
                            if (ok[k / VEC] && held_match(P[k], hi, prefix)) {
                                u = P[k];
                                holder = true;
                            }
                        }
                    }
                    if (holder) {
                        const int64_t L = (int64_t)(range - u);
                        out[t * S + s] = L;
                        if (PREFIX) out_inc[t * S + s] = L - lag_sh[(s + 1) & 1];
                        lag_sh[s & 1] = L;
                    }
                    written = true;
                    break;
                }
                if (LCAP > 0 && !in_list && count <= (uint32_t)LCAP) {
                    // compact the candidates into the list: a wave scan of
                    // the per-lane counts and one atomic per wave for its base
                    uint32_t cand = 0;  // bit k: P[k] is a candidate
#pragma unroll
                    for (int k = 0; k < K; ++k)
                        cand |= (ok[k / VEC] && held_match(P[k], hi, prefix)) ? (1u << k) : 0u;
                    const uint32_t nc = (uint32_t)__popc(cand);
                    const uint32_t incl2 = wave_scan_incl(nc);
                    const uint32_t total = (uint32_t)__builtin_amdgcn_readlane((int)incl2, 63);
                    uint32_t wbase = 0;
                    if (lane == 63 && total != 0) wbase = atomicAdd(&list_n, total);
                    uint32_t pos = (uint32_t)__builtin_amdgcn_readlane((int)wbase, 63) + incl2 - nc;
#pragma unroll
                    for (int k = 0; k < K; ++k) {
                        if ((cand >> k) & 1u) {
                            if (pos < (uint32_t)LCAP) list[pos] = P[k];  // always, as count <= LCAP
                            ++pos;
                        }
                    }
                    lds_barrier();
                    // every wave has taken its base: reset for the next boundary
                    // (its next use follows at least one more barrier)
                    if (tid == 0) list_n = 0;
                    in_list = true;
                    n = count;
                }
            }
            um = prefix;
            // sel and the list are next written after the next stage's
            // reduction barrier, which every thread passes only after
            // reading them here
        }
        if (!written && tid == 0) {
            const int64_t L = (int64_t)(range - um);
            out[t * S + s] = L;
            if (PREFIX) out_inc[t * S + s] = L - lag_sh[(s + 1) & 1];
            lag_sh[s & 1] = L;
        }
        // lag_sh[s & 1] is read at stage s + 1, after its reduction barrier
    }
    if (NARROW) {
        __syncthreads();  // after every output write of the step (global stores)
        if (wide_step && tid == 0) out[t * S] = kRedo;
    }
}

// More ranks than one workgroup holds in registers as 64-bit values: the
// 64-bit select with the values recomputed from global memory at every pass
// (a prefix from its stage rows, a duration from its row), one workgroup of
// kStreamWG threads per step.  Per boundary: a pass for the max and min,
// then radix passes over u = value - min (256 bins; a digit isolating one
// value ends it; once at most kStreamList values are left they go to an LDS
// list and later passes read only it).  It redoes the steps the 32-bit pass
// hands over (REDO: every other workgroup returns at once); the durations
// of a step are read several times over, from the caches when the step fits
// them.
constexpr int kStreamWG = 1024;
constexpr int kStreamList = 4096;

template <bool PREFIX, bool REDO>
__global__ __launch_bounds__(kStreamWG) void k_median_stream(const int64_t* __restrict__ d,
                                                             int64_t T, int R, int S,
                                                             int64_t* __restrict__ out,
                                                             int64_t* __restrict__ out_inc)
{
    constexpr int NW = kStreamWG / 64;
    __shared__ __attribute__((aligned(16))) uint32_t hist[kSelWords];
    __shared__ u64 red_max[NW], red_min[NW];
    __shared__ uint32_t sel[3];
    __shared__ u64 list[kStreamList];
    __shared__ uint32_t list_n;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int64_t t = blockIdx.x;
    if (t >= T) return;
    if (REDO && out[t * S] != kRedo) return;  // a step the narrow pass resolved
    const int64_t* dt = d + t * (int64_t)S * R;
    for (int i = tid; i < kSelWords; i += kStreamWG) hist[i] = 0;
    int64_t L_prev = 0;
    for (int s = 0; s < S; ++s) {
        auto val = [&](int r) -> u64 {
            if (!PREFIX) return (u64)dt[(int64_t)s * R + r];
            u64 p = 0;
            for (int j = 0; j <= s; ++j) p += (u64)dt[(int64_t)j * R + r];
            return p;
        };
        u64 mx = 0, mn = ~0ull;
        for (int r = tid; r < R; r += kStreamWG) {
            const u64 v = val(r);
            mx = umax64(mx, v);
            mn = umin64(mn, v);
        }
        mx = group_max<64>(mx);
        mn = ~group_max<64>(~mn);
        if (lane == 63) {
            red_max[wave] = mx;
            red_min[wave] = mn;
        }
        __syncthreads();
        u64 F = 0, Pmin = ~0ull;
        for (int i = 0; i < NW; ++i) {
            F = umax64(F, red_max[i]);
            Pmin = umin64(Pmin, red_min[i]);
        }
        const u64 range = F - Pmin;
        u64 um = 0;  // u of the median
        if (range != 0) {
            int lo = sel_first_lo(range), hi = lo + 8;
            u64 prefix = 0;
            uint32_t kk = (uint32_t)((R - 1) / 2);
            bool in_list = false;
            uint32_t n = 0;
            for (;;) {
                if (in_list) {
                    for (uint32_t i = tid; i < n; i += kStreamWG) {
                        const u64 u = list[i];
                        if (sel_match(u, hi, prefix)) atomicAdd(&hist[sel_bin(u, lo, hi, prefix)], 1u);
                    }
                } else {
                    for (int r = tid; r < R; r += kStreamWG) {
                        const u64 u = val(r) - Pmin;
                        if (sel_match(u, hi, prefix)) atomicAdd(&hist[sel_bin(u, lo, hi, prefix)], 1u);
                    }
                }
                __syncthreads();
                if (wave == 0) {
                    uint32_t dg, cn, k2 = kk;
                    sel_scan_wave(hist, lane, k2, dg, cn);
                    if (lane == 0) {
                        sel[0] = dg;
                        sel[1] = k2;
                        sel[2] = cn;
                    }
                }
                __syncthreads();
                const uint32_t digit = sel[0], count = sel[2];
                kk = sel[1];
                for (int i = tid; i < kSelWords; i += kStreamWG) hist[i] = 0;
                if (tid == 0) list_n = 0;
                __syncthreads();  // sel, hist and list_n are rewritten next
                prefix = (prefix << (hi - lo)) | (u64)digit;
                hi = lo;
                if (hi == 0) break;  // every bit chosen
                lo = lo > 8 ? lo - 8 : 0;
                if (count == 1 || (!in_list && count <= (uint32_t)kStreamList)) {
                    // the values left (one, or few enough for the list)
                    if (in_list) {
                        for (uint32_t i = tid; i < n; i += kStreamWG)
                            if (sel_match(list[i], hi, prefix)) red_max[0] = list[i];
                    } else {
                        for (int r = tid; r < R; r += kStreamWG) {
                            const u64 u = val(r) - Pmin;
                            if (sel_match(u, hi, prefix)) {
                                if (count == 1) red_max[0] = u;
                                else list[atomicAdd(&list_n, 1u)] = u;  // < count
                            }
                        }
                    }
                    __syncthreads();
                    if (count == 1) {
                        prefix = red_max[0];
                        __syncthreads();  // red_max is rewritten by the next stage
                        break;
                    }
                    in_list = true;
                    n = count;
                }
            }
            um = prefix;
        }
        if (tid == 0) {
            const int64_t L = (int64_t)(range - um);
            out[t * S + s] = L;
            if (PREFIX) out_inc[t * S + s] = L - L_prev;
        }
        L_prev = (int64_t)(range - um);
        __syncthreads();  // red_max, red_min and the list are rewritten by the next stage
    }
}

struct LagVariant {
    const void* fn;
    int WG;
    const void* redo;  // after a narrow pass: the 64-bit kernel for the steps it handed over
};

template <bool PREFIX, int VEC, int K, int WG, bool FULL, bool NARROW = false, bool REDO = false>
const void* lag_kernel()
{
    // candidate list: a quarter of the slots, at most 4096 values; none when
    // a lane holds so few values that the registers are as cheap to re-read
    constexpr int LCAP = K <= 2 ? 0 : (K * WG / 4 < 4096 ? K * WG / 4 : 4096);
    constexpr bool PUBU = PREFIX && K == 16 && WG <= 256 && !NARROW;
    static_assert(!(PUBU && FULL), "the PUBU shapes keep the rank tests");
    return reinterpret_cast<const void*>(
        &k_median_spread<PREFIX, VEC, K, WG, LCAP, PUBU, FULL, NARROW, REDO>);
}

// FULL: R fills the K * WG slots exactly, so no slot needs a rank test
// (measured on MI355X: 1-4% faster for the raw spread and for the lag at
// 128 and 16384 ranks; 12-13% slower for the lag's PUBU shapes at 1024 and
// 4096 ranks, whose register allocation grows past 96, so those keep the
// tests).  NARROW (32-bit values, two workgroups per CU) for the raw spread
// at 16 values per lane and for the lag where a step holds 8 or more waves
// (measured at 16384 ranks: 32% faster for the raw spread, 18% for the lag;
// at 1024 and 4096 ranks the raw spread 9% and 4% faster, the lag 6% slower,
// so the lag keeps its 64-bit shapes there).
// More than 16384 ranks: up to 32768 the 32-bit pass with 32 values per
// lane (16-byte loads), the streaming 64-bit kernel redoing the steps it
// hands over; beyond that (64 values per lane spill) and with 8-byte loads
// (odd R or a misaligned base) the streaming kernel alone.
template <bool PREFIX, int VEC>
LagVariant lag_wide(int R)
{
    if constexpr (VEC == 2) {
        const void* redo = reinterpret_cast<const void*>(&k_median_stream<PREFIX, true>);
        if (R == 32 * 1024) return LagVariant{lag_kernel<PREFIX, 2, 32, 1024, true, true>(), 1024, redo};
        if (R < 32 * 1024) return LagVariant{lag_kernel<PREFIX, 2, 32, 1024, false, true>(), 1024, redo};
    }
    (void)R;
    return LagVariant{reinterpret_cast<const void*>(&k_median_stream<PREFIX, false>), kStreamWG,
                      nullptr};
}

template <bool PREFIX, int VEC, int K, int WG>
LagVariant lag_shape(int R)
{
    constexpr bool pubu = PREFIX && K == 16 && WG <= 256;
    if constexpr (VEC == 2 && K == 16 && (WG >= 512 || !PREFIX)) {
        if (R == K * WG)
            return LagVariant{lag_kernel<PREFIX, VEC, K, WG, true, true>(), WG,
                              lag_kernel<PREFIX, VEC, K, WG, false, false, true>()};
    }
    if constexpr (!pubu) {
        if (R == K * WG) return LagVariant{lag_kernel<PREFIX, VEC, K, WG, true>(), WG, nullptr};
    }
    return LagVariant{lag_kernel<PREFIX, VEC, K, WG, false>(), WG, nullptr};
}

// One step per workgroup with all R prefixes in registers, as few waves as
// the registers allow: a wave spends less time at barriers than a lane does
// on 4x the prefixes (measured on the 128- to 16384-rank workloads).
template <bool PREFIX, int VEC>
LagVariant pick_lag(int R)
{
    if (R <= 128) return lag_shape<PREFIX, VEC, 2, 64>(R);
    if (R <= 256) return lag_shape<PREFIX, VEC, 4, 64>(R);
    if (R <= 512) return lag_shape<PREFIX, VEC, 8, 64>(R);
    if (R <= 1024) return lag_shape<PREFIX, VEC, 16, 64>(R);
    if (R <= 2048) return lag_shape<PREFIX, VEC, 16, 128>(R);
    if (R <= 4096) return lag_shape<PREFIX, VEC, 16, 256>(R);
    if (R <= 8192) return lag_shape<PREFIX, VEC, 16, 512>(R);
    if (R <= 16384) return lag_shape<PREFIX, VEC, 16, 1024>(R);
    return lag_wide<PREFIX, VEC>(R);  // R <= SF_MAX_R
}

// the narrow pass, then (if it has one) the 64-bit pass over the steps it
// handed over
static int launch_lag(const LagVariant& v, int64_t T, void** args, sf_stream_t stream)
{
    int rc = launch(v.fn, dim3((unsigned)T), dim3(v.WG), args, 0, stream);
    if (rc == SF_OK && v.redo) rc = launch(v.redo, dim3((unsigned)T), dim3(v.WG), args, 0, stream);
    return rc;
}

}  // namespace sfk

using namespace sfk;

SF_API int sf_frontier_lag(const int64_t* durations, int64_t T, int32_t R, int32_t S,
                           int64_t* out_lag, int64_t* out_lag_inc, sf_stream_t stream)
{
    if (T < 0 || R < 1 || R > SF_MAX_R || S < 1) return SF_EINVAL;
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
    const LagVariant v = vec2 ? pick_lag<true, 2>(R) : pick_lag<true, 1>(R);
    int Ri = R, Si = S;
    void* args[] = {(void*)&durations, (void*)&T, (void*)&Ri, (void*)&Si, (void*)&out_lag,
                    (void*)&out_lag_inc};
    return launch_lag(v, T, args, stream);
}

SF_API int sf_rank_spread(const int64_t* durations, int64_t T, int32_t R, int32_t S,
                          int64_t window, int64_t* out_spread, int64_t* out_window_spread,
                          sf_stream_t stream)
{
    if (T < 0 || R < 1 || R > SF_MAX_R || S < 1 || window < 1)
        return SF_EINVAL;
    if (!fits(T, S, R, 8)) return SF_EINVAL;
    if (T == 0) return SF_OK;
    if (T > INT32_MAX) return SF_EINVAL;  // one workgroup per step
    if (!durations || !out_spread || !out_window_spread) return SF_EINVAL;
    if (!aligned(durations, 8) || !aligned(out_spread, 8) || !aligned(out_window_spread, 8))
        return SF_EINVAL;
    const int64_t W = sf_num_windows(T, window);
    const int64_t nd = T * S * (int64_t)R * 8, no = T * S * 8, nw = W * S * 8;
    if (!disjoint(durations, nd, out_spread, no) || !disjoint(durations, nd, out_window_spread, nw) ||
        !disjoint(out_spread, no, out_window_spread, nw))
        return SF_EINVAL;
    const bool vec2 = (R % 2 == 0) && aligned(durations, 16);
    const LagVariant v = vec2 ? pick_lag<false, 2>(R) : pick_lag<false, 1>(R);
    int Ri = R, Si = S;
    int64_t* unused = nullptr;
    void* args[] = {(void*)&durations, (void*)&T, (void*)&Ri, (void*)&Si, (void*)&out_spread,
                    (void*)&unused};
    const int rc = launch_lag(v, T, args, stream);
    if (rc != SF_OK) return rc;
    return launch_window_sum(out_spread, T, S, window, W, out_window_spread, stream);
}
