// sf_select.h -- building blocks of the exact radix selects (the lag, the
// raw rank spread and the per-rank window median): 256-bin LDS histograms,
// the digit of a candidate, and a DPP wave scan.
#pragma once

#include "sf_device.h"

namespace sfk {

constexpr int kSelBins = 256;                // bins per histogram (8-bit digits)
constexpr int kSelPerLane = kSelBins / 64;   // bins one lane scans, with one 16-byte read
constexpr int kSelWords = kSelBins;          // words per histogram (16-byte aligned)

// the kSelPerLane bins of lane `lane`, read at once
__device__ __forceinline__ uint4 sel_lane_bins(const uint32_t* h, int lane)
{
    return *reinterpret_cast<const uint4*>(h + lane * kSelPerLane);
}

__device__ __forceinline__ void sel_clear_lane_bins(uint32_t* h, int lane)
{
    *reinterpret_cast<uint4*>(h + lane * kSelPerLane) = make_uint4(0u, 0u, 0u, 0u);
}

// DPP lane move of a 32-bit value in which lanes outside the row/bank masks,
// and lanes whose source lies outside their row, read 0
template <int CTRL, int ROW_MASK = 0xF, int BANK_MASK = 0xF>
__device__ __forceinline__ uint32_t dpp0(uint32_t v)
{
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, ROW_MASK, BANK_MASK, true);
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

// lane L's value, in every lane (L uniform)
__device__ __forceinline__ u64 lane_value(u64 v, int L)
{
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, L);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), L);
    return ((u64)hi << 32) | lo;
}

// Scan of a 256-bin histogram by one wave, kSelPerLane bins per lane: the
// bin that holds the candidate of rank kk (from 0), kk's rank within that
// bin, and the bin's count, in every lane.  The candidates hold rank kk, so
// exactly one lane finds it.
__device__ __forceinline__ void sel_scan_wave(const uint32_t* h, int lane, uint32_t& kk,
                                              uint32_t& digit, uint32_t& count)
{
    const uint4 b4 = sel_lane_bins(h, lane);
    const uint32_t c[kSelPerLane] = {b4.x, b4.y, b4.z, b4.w};
    const uint32_t part = c[0] + c[1] + c[2] + c[3];
    const uint32_t incl = wave_scan_incl(part);
    uint32_t cum = incl - part;
    int fd = -1;
    uint32_t fk = 0, fc = 0;
    if (cum <= kk && kk < incl) {
#pragma unroll
        for (int i = 0; i < kSelPerLane; ++i) {
            if (fd < 0 && kk < cum + c[i]) {
                fd = lane * kSelPerLane + i;
                fk = kk - cum;
                fc = c[i];
            }
            cum += c[i];
        }
    }
    const u64 fm = __ballot(fd >= 0);
    const int src = fm ? __builtin_ctzll(fm) : 0;
    digit = (uint32_t)__builtin_amdgcn_readlane(fd, src);
    kk = (uint32_t)__builtin_amdgcn_readlane((int)fk, src);
    count = (uint32_t)__builtin_amdgcn_readlane((int)fc, src);
}

// Add the active lanes' bins (-1: none) to the histogram.  When every active
// lane has the same bin one lane adds them all, so they do not serialise on
// one word.
__device__ __forceinline__ void sel_hist_add(uint32_t* h, int bin)
{
    const int first = __builtin_amdgcn_readfirstlane(bin);
    if (__ballot(bin != first) == 0) {
        const u64 active = __ballot(1);
        if (first >= 0 && (int)(threadIdx.x & 63) == __builtin_ctzll(active))
            atomicAdd(&h[first], (uint32_t)__popcll(active));
    } else if (bin >= 0) {
        atomicAdd(&h[bin], 1u);
    }
}

// Selection state: the candidates are the values u with u >> hi == prefix,
// and a pass histograms their bits [lo, hi) (hi - lo <= 8).
__device__ __forceinline__ bool sel_match(u64 u, int hi, u64 prefix)
{
    return hi >= 64 || (u >> hi) == prefix;
}

// the digit of a candidate, or -1 for a value that is not one
__device__ __forceinline__ int sel_bin(u64 u, int lo, int hi, u64 prefix)
{
    return sel_match(u, hi, prefix) ? (int)((u >> lo) & ((1u << (hi - lo)) - 1u)) : -1;
}

// the digit in the first pass, where every value u <= range is a candidate
// and 2^(lo + 8) > range (sel_first_lo)
__device__ __forceinline__ int sel_first_bin(u64 u, int lo) { return (int)(uint32_t)(u >> lo); }

// the first pass: 256 bins of width 2^lo cover [0, range] (range > 0)
__device__ __forceinline__ int sel_first_lo(u64 range)
{
    const int nbits = 64 - __builtin_clzll(range);
    return nbits > 8 ? nbits - 8 : 0;
}

}  // namespace sfk
