// median.hip -- per-rank window median, a candidate baseline btilde of Eq. (4)
// (Sec. 4): med[w][s][r] = the lower median over the n steps t of window w of
// d[t][s][r] (the value of rank floor((n-1)/2) in ascending order).
//
// A tile is (window, stage, RPW adjacent ranks).  Persistent workgroups of
// 16 waves walk the tiles; each tile is read once along the rank rows
// (8 * RPW contiguous bytes per step, 256 bytes for windows up to 1024
// steps, in 16-byte loads) into registers while the previous tile is being
// resolved.  Durations in every workload are far below 2^32 ns (4.3 s), so
// the tile is kept in LDS as 32-bit values: its low words, transposed so
// that rank j's column is a run of words with a stride of RPW + 1 (an odd
// stride: a wave reading one column hits distinct banks), while the high
// words are OR-ed together.  Each wave then takes RPW / 16 ranks in turn,
// a column's n values (K per lane, the tile's zero rows past n included as
// values below all others) in registers.
//
// A workgroup walks the windows of one (stage, rank chunk) in order, so a
// column usually has a close guess of its median: the same rank's median in
// the window before (or, in the first window, the median the wave just
// found for a rank 16 below).  Two ballot counts per value then bracket the
// target between g - g/2^e and g + g/2^e, the values inside (about a
// hundred) are listed, and the target is selected among them
// (wave_select_bracket).  Without a guess, or when the bracket misses the
// target, an exact radix select over the whole column finds it: a 256-bin
// histogram of the top 8 bits of the OR of the values, then 8 bits at a time
// of the values left; once at most 64 are left they are compacted, one per
// lane, into the wave's list.  The guess changes which values are listed,
// never the result.  Histograms and lists are private to the wave and a
// wave's LDS operations complete in issue order, so the waves need no
// barrier between them during the selection.
//
// A tile with some value at or above 2^32 (a high word not 0) is resolved
// in 64 bits instead: each wave re-reads its ranks' columns from global
// memory (they were just read, so mostly from the caches) pass by pass.
// Windows longer than the tile rows take the same 64-bit streaming select,
// one wave per (window, stage, rank).

#include "sf_device.h"
#include "sf_host.h"
#include "sf_select.h"

#include <type_traits>

namespace sfk {

// orders this wave's LDS accesses before the ones that follow (a wave's LDS
// operations complete in issue order; this keeps the compiler from moving
// them across)
__device__ __forceinline__ void wave_lds_fence()
{
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    __builtin_amdgcn_wave_barrier();
}

// OR over the 64 lanes, in every lane
__device__ __forceinline__ uint32_t wave_or32(uint32_t v)
{
    v |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, true);
    v |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, true);
    v |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x141, 0xF, 0xF, true);
    v |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x140, 0xF, 0xF, true);
    v |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xA, 0xF, true);
    v |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xC, 0xF, true);
    return (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
}

__device__ __forceinline__ u64 wave_or64(u64 v)
{
    return ((u64)wave_or32((uint32_t)(v >> 32)) << 32) | wave_or32((uint32_t)v);
}

// the position of this lane among the lanes of `mask` below it
__device__ __forceinline__ uint32_t lane_rank(u64 mask)
{
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                     __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

template <typename V>
__device__ __forceinline__ bool sel_match_t(V u, int hi, V prefix)
{
    return hi >= (int)(8 * sizeof(V)) || (u >> hi) == prefix;
}

template <typename V>
__device__ __forceinline__ int sel_first_lo_t(V range)
{
    const int nbits = (int)(8 * sizeof(V)) - (sizeof(V) == 8 ? __builtin_clzll((u64)range)
                                                              : __builtin_clz((uint32_t)range));
    return nbits > 8 ? nbits - 8 : 0;
}

// Exact lower-median select over one wave's KV values per lane, v[k] the
// value of row k * 64 + l of lane l (rows n.. are zeros, which sort at or
// below every duration); the column is read from LDS once, into registers,
// and every pass works on them.  vor is the OR of all the values, kk
// the target's rank among all 64 * KV slots, h the wave's 256-bin histogram
// (zero on entry and on return) and lst the wave's list: 64 entries, then
// one spare word per lane.
template <int KV>
__device__ uint32_t wave_select_regs(const uint32_t (&v)[KV], uint32_t vor, uint32_t kk, int n,
                                    uint32_t* h, uint32_t* lst, int lane)
{
    if (vor == 0) return 0;  // every value is 0
    auto val = [&](int k) { return v[k]; };
    // the first digit: the top 8 bits of the OR of the values, which bounds
    // every value
    int lo = sel_first_lo_t(vor), hi = lo + 8;
    uint32_t prefix = 0;
    bool first = true;     // every value is a candidate
    bool compact = false;  // the values left are one per lane in (c1, ok1)
    uint32_t c1 = 0;
    bool ok1 = false;
    for (;;) {
        if (compact) {
            // one value per lane: a lane without a candidate adds into its
            // own spare word of the list instead of branching
            const bool c = ok1 && sel_match_t(c1, hi, prefix);
            atomicAdd(c ? &h[(c1 >> lo) & ((1u << (hi - lo)) - 1u)] : &lst[64 + lane], 1u);
        } else if (first) {
            // a lane's values come from unrelated steps, so equal
            // neighbouring bins are rare: one plain atomic per value
#pragma unroll 8
            for (int k = 0; k < KV; ++k) atomicAdd(&h[val(k) >> lo], 1u);
        } else {
#pragma unroll 8
            for (int k = 0; k < KV; ++k) {
                const uint32_t x = val(k);
                sel_hist_add(h, sel_match_t(x, hi, prefix) ? (int)((x >> lo) & ((1u << (hi - lo)) - 1u)) : -1);
            }
        }
        first = false;
        wave_lds_fence();
        // scan of the bins, then every lane clears its bins
        uint32_t digit, count;
        sel_scan_wave(h, lane, kk, digit, count);
        sel_clear_lane_bins(h, lane);
        wave_lds_fence();
        prefix = (prefix << (hi - lo)) | digit;
        hi = lo;
        if (hi == 0) return prefix;  // every bit chosen: the median == prefix
        lo = lo > 8 ? lo - 8 : 0;
        if (count == 1) {
            // one value has the chosen digits: its lane hands it over.  The
            // search skips the zero rows: when the one value is such a zero,
            // no lane holds it and lane 0's x = 0 is the answer.
            uint32_t x = 0;
            bool has = false;
            if (compact) {
                has = ok1 && sel_match_t(c1, hi, prefix);
                x = c1;
            } else {
#pragma unroll 8
                for (int k = 0; k < KV; ++k) {
                    const uint32_t y = val(k);
                    if (k * 64 + lane < n && sel_match_t(y, hi, prefix)) {
                        x = y;
                        has = true;
                    }
                }
            }
            const u64 hm = __ballot(has);
            return (uint32_t)__builtin_amdgcn_readlane((int)x, hm ? __builtin_ctzll(hm) : 0);
        }
        if (!compact && count <= 64u) {
            // the values left into the list: each lane marks its candidate
            // slots, a wave scan of the per-lane counts gives each lane its
            // first list position, and every slot is stored, a non-candidate
            // into the lane's spare word (no branch, no per-slot ballot)
            uint32_t cand = 0;
#pragma unroll 8
            for (int k = 0; k < KV; ++k) cand |= sel_match_t(val(k), hi, prefix) ? (1u << k) : 0u;
            const uint32_t nc = (uint32_t)__popc(cand);
            uint32_t pos = wave_scan_incl(nc) - nc;  // < count <= 64 for every candidate
#pragma unroll 4
            for (int k = 0; k < KV; ++k) {
                const bool m = (cand >> k) & 1u;
                lst[m ? pos : 64 + lane] = val(k);
                pos += m ? 1u : 0u;
            }
            wave_lds_fence();
            ok1 = (uint32_t)lane < count;
            c1 = ok1 ? lst[lane] : 0u;
            compact = true;
        }
    }
}

// Exact lower median of the n 64-bit values get(0..n-1), read pass by pass
// (any n): the OR, then one histogram pass per digit, then a search for the
// one value left.  h: the wave's histogram (zero on entry and on return).
template <typename Get>
__device__ u64 wave_select_stream(Get get, int64_t n, uint32_t* h, int lane)
{
    u64 vor = 0;
    for (int64_t i = lane; i < n; i += 64) vor |= get(i);
    vor = wave_or64(vor);
    if (vor == 0) return 0;
    int lo = sel_first_lo_t(vor), hi = lo + 8;
    u64 prefix = 0;
    uint32_t kk = (uint32_t)((n - 1) / 2);
    for (;;) {
        for (int64_t i = lane; i < n; i += 64) {
            const u64 x = get(i);
            if (sel_match_t(x, hi, prefix)) atomicAdd(&h[(uint32_t)((x >> lo) & ((1u << (hi - lo)) - 1u))], 1u);
        }
        wave_lds_fence();
        uint32_t digit, count;
        sel_scan_wave(h, lane, kk, digit, count);
        sel_clear_lane_bins(h, lane);
        wave_lds_fence();
        prefix = (prefix << (hi - lo)) | (u64)digit;
        hi = lo;
        if (hi == 0) return prefix;
        lo = lo > 8 ? lo - 8 : 0;
        if (count == 1) {
            u64 x = 0;
            bool has = false;
            for (int64_t i = lane; i < n; i += 64) {
                const u64 y = get(i);
                if (sel_match_t(y, hi, prefix)) {
                    x = y;
                    has = true;
                }
            }
            const u64 hm = __ballot(has);
            return lane_value(x, hm ? __builtin_ctzll(hm) : 0);
        }
    }
}

constexpr int kMedWaves = 16;            // waves per workgroup
constexpr int kMedWG = 64 * kMedWaves;
constexpr int64_t kMedTileRows = 1024;   // longest window of the tiled kernel
// bracketed values a wave lists in its histogram words: list positions
// start at most kMedListCap, so with the 63 lanes of one ballot they stay
// below kSelWords (past the cap they overwrite each other, and the count,
// then above the cap, rejects the list)
constexpr uint32_t kMedListCap = kSelWords - 64;

// Exact select among at most four values per lane (slot i of lane l is list
// entry l + 64 i; ok: the slot holds a value), every value <= bound (> 0):
// 8-bit histogram passes over the values left, until a digit isolates one
// value or every bit is chosen.  kk: the target's rank among the listed
// values; h: the wave's histogram (zero on entry and on return).
__device__ uint32_t wave_select_list(const uint32_t (&x)[4], const bool (&ok)[4], uint32_t kk,
                                     uint32_t bound, uint32_t* h, int lane)
{
    int lo = sel_first_lo_t(bound), hi = lo + 8;
    uint32_t prefix = 0;
    for (;;) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
            if (ok[i] && sel_match_t(x[i], hi, prefix))
                atomicAdd(&h[(x[i] >> lo) & ((1u << (hi - lo)) - 1u)], 1u);
        wave_lds_fence();
        uint32_t digit, count;
        sel_scan_wave(h, lane, kk, digit, count);
        sel_clear_lane_bins(h, lane);
        wave_lds_fence();
        prefix = (prefix << (hi - lo)) | digit;
        hi = lo;
        if (hi == 0) return prefix;  // every bit chosen
        lo = lo > 8 ? lo - 8 : 0;
        if (count == 1) {
            // one listed value has the chosen digits: its lane hands it over
            uint32_t y = 0;
            bool has = false;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                if (ok[i] && sel_match_t(x[i], hi, prefix)) {
                    y = x[i];
                    has = true;
                }
            }
            const u64 hm = __ballot(has);
            return (uint32_t)__builtin_amdgcn_readlane((int)y, hm ? __builtin_ctzll(hm) : 0);
        }
    }
}

// The lower median of a column started from a guess g of it, with the
// column and kk as for wave_select_regs.  Two counts over the column tell
// whether the target lies in the bracket [g - delta, g + delta), delta =
// g / 2^e; the values inside it (about 100 when the guess is close) are
// listed, offset by the bracket's lower end, in the wave's histogram words
// (every other lane stores into its word of `spare`), and the target is
// selected among them.  Returns false, with h zero, when the target lies
// outside the bracket or the bracket holds more than kMedListCap values:
// the caller then runs the full select.  The guess decides only which
// values are listed, so any guess gives the same median.
template <int KV>
__device__ bool wave_select_bracket(const uint32_t (&v)[KV], uint32_t g, int e, uint32_t kk,
                                    uint32_t* h, uint32_t* spare, int lane, uint32_t& med)
{
    const uint32_t delta = max(g >> e, 1u);
    // lo >= 1 puts the zero rows below the bracket; lo + 2 delta <= 2^32
    // keeps every value below lo out of it after the wrapping subtraction
    if (g <= delta || g > 0xFFFFFFFFu - delta) return false;
    const uint32_t lo = g - delta, w2 = 2u * delta;
    const uint32_t nlo = 0u - lo;  // v < lo exactly when v - lo wraps to >= 2^32 - lo
    uint32_t below = 0, n_in = 0;  // wave-uniform counts
    uint32_t* const dump = spare + lane;  // where a value outside the bracket is stored
#pragma unroll
    for (int k = 0; k < KV; ++k) {
        const uint32_t x = v[k] - lo;
        below += (uint32_t)__popcll(__ballot(x >= nlo));
        const bool in = x < w2;
        const u64 m = __ballot(in);
        const uint32_t r = __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                                     __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
        uint32_t* const at = h + (n_in < kMedListCap ? n_in : kMedListCap) + r;
        n_in += (uint32_t)__popcll(m);
        *(in ? at : dump) = x;  // every lane stores: no branch
    }
    wave_lds_fence();
    const bool hit = below <= kk && kk - below < n_in && n_in <= kMedListCap;
    uint32_t x[4];
    bool ok[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const uint32_t idx = (uint32_t)lane + 64u * (uint32_t)i;
        ok[i] = idx < n_in;
        x[i] = h[idx];
    }
    wave_lds_fence();
    sel_clear_lane_bins(h, lane);
    wave_lds_fence();
    if (!hit) return false;
    med = lo + wave_select_list(x, ok, kk - below, w2 - 1u, h, lane);
    return true;
}

// VEC: int64 elements per load (2: 16-byte loads, even R and a 16-byte
// aligned base); K: values per lane (tile rows 64 * K >= n); RPW: ranks per
// tile (the tile is 64 * K * (RPW + 1) words, about 130 KB).  One workgroup
// per CU: 16 waves of at most 128 VGPRs.
//
// Work units: unit u = q * P + p covers the tile pair p = c * S + s (rank
// chunk c, stage s) over the windows [q * L, min((q + 1) * L, W)).  A
// workgroup takes units blockIdx.x, blockIdx.x + gridDim.x, ... and walks
// each unit's windows in order, so that every median after a unit's first
// window starts from the same rank's median of the window before
// (wave_select_bracket; e sets the bracket width).  Pairs are numbered stage
// fastest, so the units in flight at once spread over every stage row of
// their steps, which the HBM channels serve faster than neighbouring pieces
// of one row (measured on MI355X, plain reads of this walk: 82% of 8 TB/s
// against 76% with the rank chunk fastest).
// C32: units and windows below 2^31 (every workload here), so the cursor
// over them is 32-bit: its divisions and the values kept across a tile fit
// the 128-VGPR budget with 2 spilled VGPRs instead of 7 (1.4% faster at
// 16384 ranks, 2% at 4096)
template <int VEC, int K, int RPW, bool C32>
__global__ __launch_bounds__(kMedWG) __attribute__((amdgpu_waves_per_eu(4))) void k_window_median(
    const int64_t* __restrict__ d, int64_t T, int R, int S, int64_t window, int nchunk, int64_t P,
    int64_t W, int64_t L, int64_t U, int e, int64_t* __restrict__ med)
{
    constexpr int ROWS = 64 * K;     // tile rows (steps), >= n
    constexpr int STRIDE = RPW + 1;  // words per tile row
    constexpr int TPR = RPW / 2;     // threads per tile row, two ranks each
    constexpr int RPS = kMedWG / TPR;  // rows per load sweep
    constexpr int NSW = ROWS / RPS;  // load sweeps
    constexpr int RPWV = RPW / kMedWaves;  // ranks per wave
    static_assert(RPW % (2 * kMedWaves) == 0 && ROWS % RPS == 0 && RPWV <= 64, "shape");
    __shared__ uint32_t tile[ROWS * STRIDE];
    __shared__ __attribute__((aligned(16))) uint32_t hist[kMedWaves][kSelWords];
    __shared__ uint32_t lists[kMedWaves][128];  // 64 entries, then a spare word per lane
    __shared__ uint32_t wide_flag[2];  // by tile parity: some high word is not 0

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: LDS bases in SGPRs
    const int i0 = tid / TPR;          // this thread's first tile row
    const int c = (tid % TPR) * 2;     // its rank pair within a tile row
    uint32_t* h = hist[wave];
    for (int i = lane; i < kSelWords; i += 64) h[i] = 0;  // cleared again by every scan
    if (tid < 2) wide_flag[tid] = 0;

    typedef typename std::conditional<C32, uint32_t, int64_t>::type I;
    struct Cur {
        I u, w, w0, wend;  // unit, window, the unit's windows [w0, wend)
        int s, c;
    };
    const I Pi = (I)P, Li = (I)L, Wi = (I)W;
    auto unit_start = [&](int64_t u64) {
        const I u = (I)u64;
        const I q = u / Pi;
        const I p = u - q * Pi;
        Cur k;
        k.u = u;
        k.w0 = q * Li;
        k.w = k.w0;
        k.wend = k.w0 + Li < Wi ? k.w0 + Li : Wi;
        k.c = (int)(p / (I)S);
        k.s = (int)(p - (I)k.c * (I)S);
        return k;
    };
    auto advance = [&](Cur k) {
        if (++k.w >= k.wend) k = unit_start((int64_t)k.u + gridDim.x);
        return k;
    };
    auto rows_of = [&](const Cur& k) {  // 1 <= n <= ROWS
        const int64_t t0 = (int64_t)k.w * window;
        return (int)((t0 + window < T ? t0 + window : T) - t0);
    };
    const int64_t rstride = (int64_t)RPS * S * R;  // elements between sweeps
    // the next tile in flight: thread (row i0 + j * RPS, pair c) holds ranks
    // r0 + c, r0 + c + 1 of that row
    int64_t x0[NSW], x1[NSW];
    auto load = [&](const Cur& k) {
        const int n = rows_of(k);
        const int r = k.c * RPW + c;
        const int64_t* q = d + (((int64_t)k.w * window + i0) * S + k.s) * (int64_t)R + r;
#pragma unroll
        for (int j = 0; j < NSW; ++j) {
            x0[j] = 0;
            x1[j] = 0;
            if (i0 + j * RPS < n) {
                if (VEC == 2) {
                    if (r < R) {  // R even: r + 1 < R too
                        const v2i64 v = __builtin_nontemporal_load(reinterpret_cast<const v2i64*>(q));
                        x0[j] = v.x;
                        x1[j] = v.y;
                    }
                } else {
                    if (r < R) x0[j] = __builtin_nontemporal_load(q);
                    if (r + 1 < R) x1[j] = __builtin_nontemporal_load(q + 1);
                }
            }
            q += rstride;
        }
    };

    // lane rr of `guess` holds the guess for this wave's rank rr (wave + rr
    // * kMedWaves of the tile): the median just found for it, 0 for none
    uint32_t guess = 0;
    Cur pos = unit_start(blockIdx.x);  // the grid is at most U
    load(pos);
    for (int it = 0; (int64_t)pos.u < U; ++it) {
        const Cur cur = pos;
        const int n = rows_of(cur);
        pos = advance(pos);
        __syncthreads();  // every wave is done with the previous tile's columns and flag
        if (tid == 0) wide_flag[(it + 1) & 1] = 0;  // the previous tile's flag, for the next
        uint32_t hiw = 0;
#pragma unroll
        for (int j = 0; j < NSW; ++j) {
            const int i = i0 + j * RPS;
            tile[i * STRIDE + c] = (uint32_t)x0[j];
            tile[i * STRIDE + c + 1] = (uint32_t)x1[j];
            hiw |= (uint32_t)((u64)x0[j] >> 32) | (uint32_t)((u64)x1[j] >> 32);
        }
        if (__ballot(hiw != 0) != 0 && lane == 0) atomicOr(&wide_flag[it & 1], 1u);
        __syncthreads();
        const bool wide = wide_flag[it & 1] != 0;  // uniform over the workgroup
        const bool more = (int64_t)pos.u < U;
        const bool guessed = cur.w != cur.w0;  // the window before is this unit's
        const int64_t t0 = (int64_t)cur.w * window;
        int64_t* mrow = med + ((int64_t)cur.w * S + cur.s) * (int64_t)R + cur.c * RPW;
        if (!wide) {
            // the next tile's loads fly while this one is resolved
            if (more) load(pos);
            const uint32_t kk = (uint32_t)((n - 1) / 2 + (ROWS - n));
            uint32_t m_prev = 0;
#pragma unroll 1
            for (int rr = 0; rr < RPWV; ++rr) {
                const int j = wave + rr * kMedWaves;  // the tile column
                if (cur.c * RPW + j >= R) break;      // wave-uniform
                const uint32_t* col = tile + lane * STRIDE + j;
                uint32_t v[K];
#pragma unroll
                for (int k = 0; k < K; ++k) v[k] = col[k * 64 * STRIDE];
                // the guess: this rank's median in the window before, else
                // (a unit's first window) the median this wave just found
                // for the rank kMedWaves below
                const uint32_t g = guessed ? (uint32_t)__builtin_amdgcn_readlane((int)guess, rr) : m_prev;
                uint32_t m = 0;
                const bool found = (guessed || rr > 0) &&
                                   wave_select_bracket<K>(v, g, e, kk, h, lists[wave] + 64, lane, m);
                if (!found) {
                    uint32_t vor = 0;
#pragma unroll
                    for (int k = 0; k < K; ++k) vor |= v[k];
                    m = wave_select_regs<K>(v, wave_or32(vor), kk, n, h, lists[wave], lane);
                }
                guess = lane == rr ? m : guess;
                m_prev = m;
                if (lane == 0) mrow[j] = (int64_t)m;
            }
        } else {
            // some value of the tile needs 64 bits: each wave streams its
            // ranks' columns from global memory
#pragma unroll 1
            for (int rr = 0; rr < RPWV; ++rr) {
                const int j = wave + rr * kMedWaves;
                const int r = cur.c * RPW + j;
                if (r >= R) break;
                const int64_t* col = d + (t0 * S + cur.s) * (int64_t)R + r;
                const int64_t cs = (int64_t)S * R;
                const u64 m = wave_select_stream([&](int64_t i) { return (u64)col[i * cs]; }, n, h, lane);
                guess = lane == rr ? ((m >> 32) ? 0u : (uint32_t)m) : guess;
                if (lane == 0) mrow[j] = (int64_t)m;
            }
            if (more) load(pos);
        }
    }
}

// Windows longer than the tile rows: one wave per (window, stage, rank),
// the 64-bit streaming select over the column in global memory.
constexpr int kMedLongWG = 256;

__global__ __launch_bounds__(kMedLongWG) void k_window_median_long(const int64_t* __restrict__ d,
                                                                    int64_t T, int R, int S,
                                                                    int64_t window, int64_t W,
                                                                    int64_t* __restrict__ med)
{
    __shared__ __attribute__((aligned(16))) uint32_t hist[kMedLongWG / 64][kSelWords];
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    uint32_t* h = hist[wave];
    for (int i = lane; i < kSelWords; i += 64) h[i] = 0;
    wave_lds_fence();
    const int64_t total = W * S * (int64_t)R;
    const int64_t waves = (int64_t)gridDim.x * (kMedLongWG / 64);
    for (int64_t id = (int64_t)blockIdx.x * (kMedLongWG / 64) + wave; id < total; id += waves) {
        const int64_t ws = id / R;
        const int r = (int)(id - ws * R);
        const int64_t w = ws / S;
        const int s = (int)(ws - w * S);
        const int64_t t0 = w * window;
        const int64_t n = (t0 + window < T ? t0 + window : T) - t0;
        const int64_t* col = d + (t0 * S + s) * (int64_t)R + r;
        const int64_t cs = (int64_t)S * R;
        const u64 m = wave_select_stream([&](int64_t i) { return (u64)col[i * cs]; }, n, h, lane);
        if (lane == 0) med[id] = (int64_t)m;
    }
}

struct MedianVariant {
    const void* fn;
    int RPW;
};

template <int VEC, int K, int RPW>
MedianVariant median_variant(bool c32)
{
    return MedianVariant{c32 ? reinterpret_cast<const void*>(&k_window_median<VEC, K, RPW, true>)
                             : reinterpret_cast<const void*>(&k_window_median<VEC, K, RPW, false>),
                         RPW};
}

// K values per lane for windows up to 64 K steps; the rank tile widens as
// the window shortens, so that every tile holds about 128 KB of 32-bit
// values (256-byte rows at 1024 steps, 2 KB rows at 128)
template <int VEC>
MedianVariant pick_median(int64_t n, bool c32)
{
    if (n <= 128) return median_variant<VEC, 2, 256>(c32);
    if (n <= 256) return median_variant<VEC, 4, 128>(c32);
    if (n <= 512) return median_variant<VEC, 8, 64>(c32);
    return median_variant<VEC, 16, 32>(c32);  // n <= kMedTileRows
}

}  // namespace sfk

using namespace sfk;

SF_API int sf_window_median(const int64_t* durations, int64_t T, int32_t R, int32_t S,
                            int64_t window, int64_t* out_median, sf_stream_t stream)
{
    if (T < 0 || R < 1 || R > SF_MAX_R || S < 1 || window < 1) return SF_EINVAL;
    if (!fits(T, S, R, 8)) return SF_EINVAL;
    if (T == 0) return SF_OK;
    const int64_t n_max = window < T ? window : T;
    const int64_t W = sf_num_windows(T, window);
    if (!fits(W, S, R, 8)) return SF_EINVAL;
    if (!durations || !out_median) return SF_EINVAL;
    if (!aligned(durations, 8) || !aligned(out_median, 8)) return SF_EINVAL;
    if (!disjoint(durations, T * S * (int64_t)R * 8, out_median, W * S * (int64_t)R * 8))
        return SF_EINVAL;
    int cus = 0;
    if (device_cus(stream, &cus) != SF_OK) return SF_EHIP;
    if (cus < 1) cus = 1;
    if (n_max > kMedTileRows) {
        const int64_t total = W * S * (int64_t)R;
        const int64_t want = (total + kMedLongWG / 64 - 1) / (kMedLongWG / 64);
        const int64_t grid = want < (int64_t)cus * 8 ? want : (int64_t)cus * 8;
        int Ri = R, Si = S;
        int64_t Wl = W;
        void* args[] = {(void*)&durations, (void*)&T, (void*)&Ri, (void*)&Si,
                        (void*)&window, (void*)&Wl, (void*)&out_median};
        return launch(reinterpret_cast<const void*>(&k_window_median_long), dim3((unsigned)grid),
                      dim3(kMedLongWG), args, 0, stream);
    }
    const bool vec2 = (R % 2 == 0) && aligned(durations, 16);
    const int RPW = (vec2 ? pick_median<2>(n_max, false) : pick_median<1>(n_max, false)).RPW;
    const int nchunk = (R + RPW - 1) / RPW;
    const int64_t P = (int64_t)nchunk * S;  // tile pairs (rank chunk, stage)
    // persistent workgroups, at most one per CU (each holds about 150 KB of
    // LDS), over units of L consecutive windows of one pair: the split Q of
    // the windows that minimises the units per workgroup times the unit's
    // cost, counting its first window (no guess, the full select) twice
    int64_t L = W, U = P;
    double best = -1.0;
    const int64_t qmax = W < 4 * (int64_t)cus ? W : 4 * (int64_t)cus;
    for (int64_t q = 1; q <= qmax; ++q) {
        const int64_t l = (W + q - 1) / q;
        if (P > INT64_MAX / ((W + l - 1) / l)) break;
        const int64_t u = P * ((W + l - 1) / l);  // every range non-empty
        const int64_t g = u < cus ? u : cus;
        const double cost = (double)((u + g - 1) / g) * (double)(l + 1);
        if (best < 0.0 || cost < best) {
            best = cost;
            L = l;
            U = u;
        }
    }
    const int64_t grid = U < cus ? U : cus;
    // a 32-bit cursor when the units, and the windows plus a unit's length,
    // stay below 2^31
    const bool c32 = U <= INT32_MAX && W + L <= INT32_MAX;
    const MedianVariant v = vec2 ? pick_median<2>(n_max, c32) : pick_median<1>(n_max, c32);
    // bracket half-width g / 2^e for windows of n_max steps: about 3.7
    // sqrt(n) values inside for a spread of a tenth of the value, so that a
    // guess off by the statistical error of a median still brackets it
    int lg = 0;
    while (((int64_t)2 << lg) <= n_max) ++lg;  // floor(log2(n_max))
    int e = (lg + 1) / 2 + 1;
    if (e < 4) e = 4;
    int Ri = R, Si = S;
    int64_t Wl = W;
    void* args[] = {(void*)&durations, (void*)&T, (void*)&Ri, (void*)&Si, (void*)&window,
                    (void*)&nchunk,    (void*)&P, (void*)&Wl, (void*)&L,  (void*)&U,
                    (void*)&e,         (void*)&out_median};
    return launch(v.fn, dim3((unsigned)grid), dim3(kMedWG), args, 0, stream);
}
