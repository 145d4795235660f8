// lag.hip -- lag kernel (Sec. 4): L[t,s] = max_r P - median_r P with the lower median
// (rank floor((R-1)/2) in ascending order) and its increment.
//
// One workgroup per step holds all R prefixes in registers (K per lane).  At
// each boundary a block min/max gives F and Pmin; the median of
// u = P - Pmin (< 2^47) is found exactly by radix select on 8-bit digits,
// over only as many passes as the range F - Pmin needs: a 256-bin LDS
// histogram of the digits of the values that still match the selected
// prefix, a scan of the histogram by wave 0, and the bin holding the target
// rank becomes the next digit.  Lanes of a wave whose digit equals the
// wave's first active digit add to the histogram with one aggregated atomic,
// which keeps clustered data (most prefixes share their high digits) from
// serialising on one bin.

#include "sf_device.h"
#include "sf_host.h"

namespace sfk {

constexpr int kLagBins = 256;

template <int VEC, int K, int WG>
__global__ __launch_bounds__(WG) void k_frontier_lag(const int64_t* __restrict__ d, int64_t T,
                                                     int R, int S, int64_t* __restrict__ lag,
                                                     int64_t* __restrict__ lag_inc)
{
    static_assert(K % VEC == 0 && WG % 64 == 0, "shape");
    constexpr int NW = WG / 64;
    constexpr int NLD = K / VEC;
    // block min/max partials, double-buffered by stage parity: a wave may
    // write stage s+1's partial while another still reads stage s's (when
    // a boundary needs no radix pass there is no barrier in between)
    __shared__ u64 red_max[2][NW], red_min[2][NW];
    __shared__ uint32_t hist[kLagBins];
    __shared__ u64 sel[2];

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
    u64 P[K];
#pragma unroll
    for (int k = 0; k < K; ++k) P[k] = 0;
    int64_t L_prev = 0;
    const uint32_t target = (uint32_t)((R - 1) / 2);

    for (int s = 0; s < S; ++s) {
        const int64_t* row = dt + (int64_t)s * R;
        u64 lmax = 0, lmin = ~0ull;
#pragma unroll
        for (int l = 0; l < NLD; ++l) {
            int64_t v[VEC];
            if (VEC == 2) {
                const v2i64 x = __builtin_nontemporal_load(reinterpret_cast<const v2i64*>(row + idx[l]));
                v[0] = x.x;
                v[VEC - 1] = x.y;
            } else {
                v[0] = __builtin_nontemporal_load(row + idx[l]);
            }
#pragma unroll
            for (int e = 0; e < VEC; ++e) {
                const int k = l * VEC + e;
                P[k] += ok[l] ? (u64)v[e] : 0ull;
                if (ok[l]) {
                    lmax = umax64(lmax, P[k]);
                    lmin = umin64(lmin, P[k]);
                }
            }
        }
        // block max and min (min as the max of complements)
        lmax = group_max<64>(lmax);
        lmin = ~group_max<64>(~lmin);
        const int pb = s & 1;
        if (lane == 63) {
            red_max[pb][wave] = lmax;
            red_min[pb][wave] = lmin;
        }
        if (s == 0)
            for (int i = tid; i < kLagBins; i += WG) hist[i] = 0;  // kept zero after every pass
        __syncthreads();
        u64 F = red_max[pb][0], Pmin = red_min[pb][0];
#pragma unroll
        for (int w = 1; w < NW; ++w) {
            F = umax64(F, red_max[pb][w]);
            Pmin = umin64(Pmin, red_min[pb][w]);
        }
        const u64 range = F - Pmin;
        u64 median = F;
        if (range != 0) {
            const int nbits = 64 - __builtin_clzll(range);
            const int passes = (nbits + 7) >> 3;
            u64 prefix = 0;
            uint32_t kk = target;
            for (int p = passes - 1; p >= 0; --p) {
                const int shift = 8 * p;
#pragma unroll
                for (int k = 0; k < K; ++k) {
                    const u64 u = P[k] - Pmin;
                    const bool cand = ok[k / VEC] && (shift + 8 >= 64 || (u >> (shift + 8)) == prefix);
                    const int bin = cand ? (int)((u >> shift) & 0xFF) : -1;
                    const int first = __builtin_amdgcn_readfirstlane(bin);
                    const u64 same = __ballot(bin == first);
                    if (first >= 0 && bin == first) {
                        if (lane == __builtin_ctzll(same))
                            atomicAdd(&hist[first], (uint32_t)__popcll(same));
                    } else if (bin >= 0) {
                        atomicAdd(&hist[bin], 1u);
                    }
                }
                __syncthreads();
                if (wave == 0) {
                    // exclusive scan over 256 bins, 4 per lane
                    uint32_t h[4], part = 0;
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        h[i] = hist[lane * 4 + i];
                        part += h[i];
                    }
                    uint32_t incl = part;
                    for (int off = 1; off < 64; off <<= 1) {
                        const uint32_t o = __shfl_up(incl, off, 64);
                        if (lane >= off) incl += o;
                    }
                    uint32_t cum = incl - part;
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        if (cum <= kk && kk < cum + h[i]) {
                            sel[0] = (u64)(lane * 4 + i);
                            sel[1] = (u64)(kk - cum);
                        }
                        cum += h[i];
                    }
                }
                __syncthreads();
                prefix = (prefix << 8) | sel[0];
                kk = (uint32_t)sel[1];
                for (int i = tid; i < kLagBins; i += WG) hist[i] = 0;
                __syncthreads();
            }
            median = Pmin + prefix;
        }
        const int64_t L = (int64_t)(F - median);
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
    return LagVariant{reinterpret_cast<const void*>(&k_frontier_lag<VEC, K, WG>), WG};
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
