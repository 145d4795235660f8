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
// words are OR-ed together.  Each wave then takes RPW / 16 ranks in turn:
// a column's n values (K per lane, the tile's zero rows past n included as
// values below all others) go to registers, and an exact radix select (a
// 256-bin histogram of the top 8 bits of the OR of the values, then 8 bits
// at a time of the values left) finds the lower median.  Once at most 64
// values are left they are compacted, one per lane, into the wave's list
// (a ballot and a lane count per slot), so later passes handle one value
// per lane.  The histogram and the list are private to the wave and a
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

// VEC: int64 elements per load (2: 16-byte loads, even R and a 16-byte
// aligned base); K: values per lane (tile rows 64 * K >= n); RPW: ranks per
// tile (the tile is 64 * K * (RPW + 1) words, about 130 KB).  One workgroup
// per CU: 16 waves of at most 128 VGPRs.
template <int VEC, int K, int RPW>
__global__ __launch_bounds__(kMedWG) __attribute__((amdgpu_waves_per_eu(4))) void k_window_median(
    const int64_t* __restrict__ d, int64_t T, int R, int S, int64_t window, int nchunk,
    int64_t ntiles, int64_t* __restrict__ med)
{
    constexpr int ROWS = 64 * K;     // tile rows (steps), >= n
    constexpr int STRIDE = RPW + 1;  // words per tile row
    constexpr int TPR = RPW / 2;     // threads per tile row, two ranks each
    constexpr int RPS = kMedWG / TPR;  // rows per load sweep
    constexpr int NSW = ROWS / RPS;  // load sweeps
    constexpr int RPWV = RPW / kMedWaves;  // ranks per wave
    static_assert(RPW % (2 * kMedWaves) == 0 && ROWS % RPS == 0, "shape");
    __shared__ uint32_t tile[ROWS * STRIDE];
    __shared__ __attribute__((aligned(16))) uint32_t hist[kMedWaves][kSelWords];
    __shared__ uint32_t lists[kMedWaves][128];  // 64 entries, then a spare word per lane
    __shared__ uint32_t wide_flag[2];  // by tile parity: some high word is not 0

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int i0 = tid / TPR;          // this thread's first tile row
    const int c = (tid % TPR) * 2;     // its rank pair within a tile row
    uint32_t* h = hist[wave];
    for (int i = lane; i < kSelWords; i += 64) h[i] = 0;  // cleared again by every scan
    if (tid < 2) wide_flag[tid] = 0;

    // tile b -> (window, stage, rank chunk), the chunk fastest so that
    // neighbouring workgroups read neighbouring pieces of the same rows.  A
    // workgroup's tiles advance by gridDim.x: the position is a mixed-radix
    // counter (w, s, chunk) advanced with carries, so that the loop does no
    // 64-bit division.
    struct Pos {
        int64_t w;
        int s, c;
    };
    auto split = [&](int64_t b) {
        const int64_t wsi = b / nchunk;
        return Pos{wsi / S, (int)(wsi % S), (int)(b - wsi * nchunk)};
    };
    const Pos step = split(gridDim.x);
    auto advance = [&](Pos p) {
        p.c += step.c;
        const int cc = p.c >= nchunk;
        p.c -= cc ? nchunk : 0;
        p.s += step.s + cc;
        const int cs = p.s >= S;
        p.s -= cs ? S : 0;
        p.w += step.w + cs;
        return p;
    };
    auto rows_of = [&](const Pos& p) {  // 1 <= n <= ROWS
        const int64_t t0 = p.w * window;
        return (int)((t0 + window < T ? t0 + window : T) - t0);
    };
    const int64_t rstride = (int64_t)RPS * S * R;  // elements between sweeps
    // the next tile in flight: thread (row i0 + j * RPS, pair c) holds ranks
    // r0 + c, r0 + c + 1 of that row
    int64_t x0[NSW], x1[NSW];
    auto load = [&](const Pos& p) {
        const int n = rows_of(p);
        const int r = p.c * RPW + c;
        const int64_t* q = d + ((p.w * window + i0) * S + p.s) * (int64_t)R + r;
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

    int64_t b = blockIdx.x;  // the grid is at most ntiles
    Pos pos = split(b);
    load(pos);
    for (int it = 0; b < ntiles; b += gridDim.x, ++it) {
        const Pos cur = pos;
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
        const bool more = b + gridDim.x < ntiles;
        const int64_t t0 = cur.w * window;
        int64_t* mrow = med + (cur.w * S + cur.s) * (int64_t)R + cur.c * RPW;
        if (!wide) {
            // the next tile's loads fly while this one is resolved
            if (more) load(pos);
            const uint32_t kk = (uint32_t)((n - 1) / 2 + (ROWS - n));
#pragma unroll 1
            for (int rr = 0; rr < RPWV; ++rr) {
                const int j = wave + rr * kMedWaves;  // the tile column
                if (cur.c * RPW + j >= R) break;      // wave-uniform
                const uint32_t* col = tile + lane * STRIDE + j;
                uint32_t v[K];
                uint32_t vor = 0;
#pragma unroll
                for (int k = 0; k < K; ++k) {
                    v[k] = col[k * 64 * STRIDE];
                    vor |= v[k];
                }
                const uint32_t m = wave_select_regs<K>(v, wave_or32(vor), kk, n, h, lists[wave], lane);
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
MedianVariant median_variant()
{
    return MedianVariant{reinterpret_cast<const void*>(&k_window_median<VEC, K, RPW>), RPW};
}

// K values per lane for windows up to 64 K steps; the rank tile widens as
// the window shortens, so that every tile holds about 128 KB of 32-bit
// values (256-byte rows at 1024 steps, 2 KB rows at 128)
template <int VEC>
MedianVariant pick_median(int64_t n)
{
    if (n <= 128) return median_variant<VEC, 2, 256>();
    if (n <= 256) return median_variant<VEC, 4, 128>();
    if (n <= 512) return median_variant<VEC, 8, 64>();
    return median_variant<VEC, 16, 32>();  // n <= kMedTileRows
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
    const MedianVariant v = vec2 ? pick_median<2>(n_max) : pick_median<1>(n_max);
    const int nchunk = (R + v.RPW - 1) / v.RPW;
    int64_t ntiles = W * S * (int64_t)nchunk;
    // persistent workgroups: one per CU (each holds about 150 KB of LDS)
    int64_t grid = cus;
    if (grid > ntiles) grid = ntiles;
    int Ri = R, Si = S;
    void* args[] = {(void*)&durations, (void*)&T,      (void*)&Ri,     (void*)&Si,
                    (void*)&window,    (void*)&nchunk, (void*)&ntiles, (void*)&out_median};
    return launch(v.fn, dim3((unsigned)grid), dim3(kMedWG), args, 0, stream);
}
