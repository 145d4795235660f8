// median.hip -- per-rank window median, a candidate baseline btilde of Eq. (4)
// (Sec. 4): med[w][s][r] = the lower median over the n steps t of window w of
// d[t][s][r] (the value of rank floor((n-1)/2) in ascending order).
//
// A tile is (window, stage, RPW adjacent ranks).  Persistent workgroups walk
// the tiles; each tile is read once along the rank rows (8 * RPW contiguous
// bytes per step, in 16-byte loads) into registers, while the previous tile
// is being resolved, and is then transposed through LDS, where the low and
// high words sit in separate planes with a row stride of RPW + 1 words so
// that a wave reading one rank's column hits distinct banks.  Each wave then
// takes one rank: its n values (K per lane, the tile's zero rows past n
// included as values below all others) go to registers, and an exact radix
// select (a 256-bin histogram of the top 8 bits of the OR of the values,
// then 8 bits at a time of the values left) finds the lower median.  Once
// at most 64 values are left they are compacted, one per lane,
// through the wave's own (already read) tile column, so later passes handle
// one value per lane.  The histogram is private to the wave and a wave's LDS
// operations complete in issue order, so the waves need no barrier between
// them during the selection.

#include "sf_device.h"
#include "sf_host.h"
#include "sf_select.h"

namespace sfk {

// OR over aligned groups of SUB lanes (the DPP pattern of group_max); the
// result is valid in the last lane of each group
template <int SUB>
__device__ __forceinline__ u64 group_or(u64 v)
{
    if (SUB >= 2) v |= dpp_move<0xB1, 0xF>(v);
    if (SUB >= 4) v |= dpp_move<0x4E, 0xF>(v);
    if (SUB >= 8) v |= dpp_move<0x141, 0xF>(v);
    if (SUB >= 16) v |= dpp_move<0x140, 0xF>(v);
    if (SUB >= 32) v |= dpp_move<0x142, 0xA>(v);
    if (SUB >= 64) v |= dpp_move<0x143, 0xC>(v);
    return v;
}

// orders this wave's LDS accesses before the ones that follow (a wave's LDS
// operations complete in issue order; this keeps the compiler from moving
// them across)
__device__ __forceinline__ void wave_lds_fence()
{
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    __builtin_amdgcn_wave_barrier();
}

// At most 64 VGPRs (8 waves per SIMD) for the shapes of windows up to 256
// steps, whose tiles leave LDS for two workgroups per CU: without the cap
// the 256-step shape takes 72 and one workgroup per CU (24% slower).
template <int VEC, int K, int RPW>
__global__ __launch_bounds__(64 * RPW) __attribute__((amdgpu_waves_per_eu(K <= 4 ? 8 : 4))) void k_window_median(const int64_t* __restrict__ d,
                                                            int64_t T, int R, int S,
                                                            int64_t window, int nchunk,
                                                            int64_t ntiles,
                                                            int64_t* __restrict__ med)
{
    constexpr int WG = 64 * RPW;
    constexpr int ROWS = 64 * K;     // tile rows (steps), >= n
    constexpr int STRIDE = RPW + 1;  // words per tile row in each plane
    constexpr int TPR = RPW / 2;     // threads per tile row, two ranks each
    constexpr int RPS = WG / TPR;    // rows per load sweep
    constexpr int NSW = ROWS / RPS;  // load sweeps
    constexpr int LIST = 64;         // values left that are compacted
    static_assert(RPW % 2 == 0 && ROWS % RPS == 0 && ROWS >= LIST, "shape");
    __shared__ uint32_t tlo[ROWS * STRIDE], thi[ROWS * STRIDE];
    __shared__ __attribute__((aligned(16))) uint32_t hist[RPW][kSelWords];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int c = (tid % TPR) * 2;  // this thread's rank pair within a tile row
    uint32_t* h = hist[wave];
    for (int i = lane; i < kSelWords; i += 64) h[i] = 0;  // cleared again by every scan

    // tile b -> (window, stage, rank chunk), the chunk fastest so that
    // neighbouring workgroups read neighbouring pieces of the same rows.  A
    // workgroup's tiles advance by gridDim.x: the position is a mixed-radix
    // counter (w, s, chunk) advanced with carries, so that the loop does no
    // 64-bit division (which costs some 300 scalar instructions per tile in
    // every wave).
    struct Tile {
        int64_t w, t0;
        int s, n, r0;
    };
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
    auto tile = [&](const Pos& p) {
        Tile x;
        x.r0 = p.c * RPW;
        x.s = p.s;
        x.w = p.w;
        x.t0 = x.w * window;
        x.n = (int)((x.t0 + window < T ? x.t0 + window : T) - x.t0);  // 1 <= n <= ROWS
        return x;
    };
    // the next tile in flight: thread (row i, pair c) holds ranks r0 + c, r0 + c + 1
    int64_t x0[NSW], x1[NSW];
    auto load = [&](const Tile& q) {
        const int r = q.r0 + c;
#pragma unroll
        for (int j = 0; j < NSW; ++j) {
            const int i = tid / TPR + j * RPS;
            x0[j] = 0;
            x1[j] = 0;
            if (i < q.n) {
                const int64_t* p = d + ((q.t0 + i) * S + q.s) * (int64_t)R + r;
                if (VEC == 2) {
                    if (r < R) {  // R even: r + 1 < R too
                        const v2i64 v = __builtin_nontemporal_load(reinterpret_cast<const v2i64*>(p));
                        x0[j] = v.x;
                        x1[j] = v.y;
                    }
                } else {
                    if (r < R) x0[j] = __builtin_nontemporal_load(p);
                    if (r + 1 < R) x1[j] = __builtin_nontemporal_load(p + 1);
                }
            }
        }
    };

    int64_t b = blockIdx.x;  // the grid is at most ntiles
    Pos pos = split(b);
    load(tile(pos));
    for (; b < ntiles; b += gridDim.x) {
        const Tile q = tile(pos);
        pos = advance(pos);
        __syncthreads();  // every wave is done with the previous tile's columns
#pragma unroll
        for (int j = 0; j < NSW; ++j) {
            const int i = tid / TPR + j * RPS;
            tlo[i * STRIDE + c] = (uint32_t)x0[j];
            thi[i * STRIDE + c] = (uint32_t)((u64)x0[j] >> 32);
            tlo[i * STRIDE + c + 1] = (uint32_t)x1[j];
            thi[i * STRIDE + c + 1] = (uint32_t)((u64)x1[j] >> 32);
        }
        __syncthreads();
        // this wave's rank: its column to registers.  Rows n.. of the tile
        // hold zeros (the loads leave them 0); durations are >= 0, so the
        // zeros sort at or below every value and the lower median of the n
        // values is the slot of rank (n - 1) / 2 + (ROWS - n) among all
        // ROWS slots: no slot needs a validity test.
        u64 v[K];
#pragma unroll
        for (int k = 0; k < K; ++k) {
            const int i = k * 64 + lane;
            v[k] = ((u64)thi[i * STRIDE + wave] << 32) | tlo[i * STRIDE + wave];
        }
        // the next tile's loads fly while this one is resolved
        if (b + gridDim.x < ntiles) load(tile(pos));
        const int r = q.r0 + wave;
        if (r >= R) continue;  // the barriers are at the top of the loop

        // the first digit: the top 8 bits of the OR of the values, which
        // bounds every value
        u64 vor = 0;
#pragma unroll
        for (int k = 0; k < K; ++k) vor |= v[k];
        vor = lane_value(group_or<64>(vor), 63);
        u64 um = 0;  // the median (0 when every value is 0)
        if (vor != 0) {
            int lo = sel_first_lo(vor), hi = lo + 8;
            u64 prefix = 0;
            uint32_t kk = (uint32_t)((q.n - 1) / 2 + (ROWS - q.n));
            bool first = true;     // every value is a candidate
            bool compact = false;  // the values left are one per lane in (c1, ok1)
            u64 c1 = 0;
            bool ok1 = false;
            for (;;) {
                if (compact) {
                    sel_hist_add(h, ok1 ? sel_bin(c1, lo, hi, prefix) : -1);
                } else if (first) {
                    // a lane's values come from unrelated steps, so equal
                    // neighbouring bins are rare: one plain atomic per value
                    // (2-4% faster than adding runs of equal bins at once)
#pragma unroll
                    for (int k = 0; k < K; ++k) atomicAdd(&h[sel_first_bin(v[k], lo)], 1u);
                } else {
#pragma unroll
                    for (int k = 0; k < K; ++k) sel_hist_add(h, sel_bin(v[k], lo, hi, prefix));
                }
                first = false;
                wave_lds_fence();
                // scan of the bins, then every lane clears its bins
                uint32_t digit, count;
                sel_scan_wave(h, lane, kk, digit, count);
                sel_clear_lane_bins(h, lane);
                wave_lds_fence();
                prefix = (prefix << (hi - lo)) | (u64)digit;
                hi = lo;
                if (hi == 0) break;  // every bit chosen: the median == prefix
                lo = lo > 8 ? lo - 8 : 0;
                if (count == 1) {
                    // one value has the chosen digits: its lane hands it over.
                    // The search skips the zero rows (a mask here keeps the
                    // compiler from holding every slot's match in registers):
                    // when the one value is such a zero, no lane holds it and
                    // lane 0's x = 0 is the answer.
                    u64 x = 0;
                    bool has = false;
                    if (compact) {
                        has = ok1 && sel_match(c1, hi, prefix);
                        x = c1;
                    } else {
#pragma unroll
                        for (int k = 0; k < K; ++k) {
                            if (k * 64 + lane < q.n && sel_match(v[k], hi, prefix)) {
                                x = v[k];
                                has = true;
                            }
                        }
                    }
                    const u64 hm = __ballot(has);
                    prefix = lane_value(x, hm ? __builtin_ctzll(hm) : 0);
                    break;
                }
                if (!compact && count <= (uint32_t)LIST) {
                    // the values left, one per lane, through rows [0, count)
                    // of this wave's tile column (read already)
                    uint32_t cand = 0;  // bit k: v[k] is left
#pragma unroll
                    for (int k = 0; k < K; ++k) cand |= sel_match(v[k], hi, prefix) ? (1u << k) : 0u;
                    const uint32_t nc = (uint32_t)__popc(cand);
                    uint32_t pos = wave_scan_incl(nc) - nc;
#pragma unroll
                    for (int k = 0; k < K; ++k) {
                        if ((cand >> k) & 1u) {
                            if (pos < (uint32_t)LIST) {  // always, as count <= LIST
                                tlo[pos * STRIDE + wave] = (uint32_t)v[k];
                                thi[pos * STRIDE + wave] = (uint32_t)(v[k] >> 32);
                            }
                            ++pos;
                        }
                    }
                    wave_lds_fence();
                    ok1 = (uint32_t)lane < count;
                    c1 = ok1 ? (((u64)thi[lane * STRIDE + wave] << 32) | tlo[lane * STRIDE + wave]) : 0ull;
                    compact = true;
                }
            }
            um = prefix;
        }
        if (lane == 0) med[(q.w * S + q.s) * (int64_t)R + r] = (int64_t)um;
    }
}

struct MedianVariant {
    const void* fn;
    int WG, RPW;
};

template <int VEC, int K, int RPW>
MedianVariant median_variant()
{
    return MedianVariant{reinterpret_cast<const void*>(&k_window_median<VEC, K, RPW>), 64 * RPW, RPW};
}

// K values per lane for windows up to 64 K steps, 16 ranks per workgroup
// (128-byte rows; the 1024-step tile fills 156 KB of LDS)
template <int VEC>
MedianVariant pick_median(int64_t n)
{
    if (n <= 128) return median_variant<VEC, 2, 16>();
    if (n <= 256) return median_variant<VEC, 4, 16>();
    if (n <= 512) return median_variant<VEC, 8, 16>();
    return median_variant<VEC, 16, 16>();  // n <= SF_MAX_WINDOW_MEDIAN = 1024
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
    if (n_max > SF_MAX_WINDOW_MEDIAN) return SF_EINVAL;
    const int64_t W = sf_num_windows(T, window);
    if (!fits(W, S, R, 8)) return SF_EINVAL;
    if (!durations || !out_median) return SF_EINVAL;
    if (!aligned(durations, 8) || !aligned(out_median, 8)) return SF_EINVAL;
    if (!disjoint(durations, T * S * (int64_t)R * 8, out_median, W * S * (int64_t)R * 8))
        return SF_EINVAL;
    const bool vec2 = (R % 2 == 0) && aligned(durations, 16);
    const MedianVariant v = vec2 ? pick_median<2>(n_max) : pick_median<1>(n_max);
    const int nchunk = (R + v.RPW - 1) / v.RPW;
    int64_t ntiles = W * S * (int64_t)nchunk;
    // persistent workgroups: as many as are resident at once on the
    // stream's device
    int cus = 0, per_cu = 0;
    if (device_cus(stream, &cus) != SF_OK ||
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, v.fn, v.WG, 0) != hipSuccess)
        return SF_EHIP;
    int64_t grid = (int64_t)(cus > 0 ? cus : 1) * (per_cu > 0 ? per_cu : 1);
    if (grid > ntiles) grid = ntiles;
    int Ri = R, Si = S;
    void* args[] = {(void*)&durations, (void*)&T,      (void*)&Ri,     (void*)&Si,
                    (void*)&window,    (void*)&nchunk, (void*)&ntiles, (void*)&out_median};
    return launch(v.fn, dim3((unsigned)grid), dim3(v.WG), args, 0, stream);
}
