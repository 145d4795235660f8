// window.hip -- sf_window_summary and sf_num_windows: window sums of the
// advances (Eq. (2) numerators), leader counts and top-2 routing (Sec. 4);
// sf_window_lead_exposed: the exposed time each rank led (every advance
// attributed to its leader, Sec. 3) and the top-2 weighted by it;
// sf_window_leader_switches: leader switches between confident unique
// leaders (Sec. 4 localization evidence); and the generic window sum used
// by sf_exposure_gain.
//
// Window kernels.  One workgroup per (window, stage, rank chunk) builds the
// leader histogram of the window in LDS with LDS atomics and sums the
// advances; one workgroup per window then picks the two largest stages and
// their most frequent leaders.

#include "sf_device.h"
#include "sf_host.h"
#include "sf_select.h"

namespace sfk {

constexpr int kHistChunk = 16384;  // ranks per histogram workgroup (64 KB LDS)

// One workgroup per (window, stage, rank chunk); grid-stride over them.
__global__ __launch_bounds__(kSumWG) void k_window_counts(
    const int64_t* __restrict__ inc, const int32_t* __restrict__ lead, int64_t T, int R, int S,
    int64_t window, int64_t W, int nchunk, int64_t* __restrict__ exposed,
    int32_t* __restrict__ counts)
{
    extern __shared__ int32_t hist[];  // [min(R, kHistChunk)]
    __shared__ int64_t part[kSumWG / 64];
    const int tid = threadIdx.x;
    const int64_t total = W * S * nchunk;
    for (int64_t id = blockIdx.x; id < total; id += gridDim.x) {
        const int c = (int)(id % nchunk);
        const int64_t ws = id / nchunk;
        const int s = (int)(ws % S);
        const int64_t w = ws / S;
        const int lo = c * kHistChunk;
        const int n = min(kHistChunk, R - lo);
        const int64_t t0 = w * window;
        const int64_t t1 = min(t0 + window, T);

        for (int i = tid; i < n; i += kSumWG) hist[i] = 0;
        __syncthreads();
#pragma unroll 4
        for (int64_t t = t0 + tid; t < t1; t += kSumWG) {
            const int64_t r = (int64_t)lead[t * S + s] - lo;
            if (r >= 0 && r < n) atomicAdd(&hist[r], 1);
        }
        if (c == 0) {
            int64_t sum = 0;
#pragma unroll 4
            for (int64_t t = t0 + tid; t < t1; t += kSumWG) sum += inc[t * S + s];
            sum = wave_sum64(sum);
            if ((tid & 63) == 0) part[tid >> 6] = sum;
        }
        __syncthreads();
        if (c == 0 && tid == 0) {
            int64_t sum = 0;
            for (int i = 0; i < kSumWG / 64; ++i) sum += part[i];
            exposed[w * S + s] = sum;
        }
        int32_t* out = counts + (w * S + s) * (int64_t)R + lo;
        for (int i = tid; i < n; i += kSumWG) out[i] = hist[i];
        __syncthreads();  // hist and part are reused by the next id
    }
}

constexpr int kTopWG = 256;

// Block-wide max of a 64-bit key; every thread gets the result.
__device__ __forceinline__ u64 block_max64(u64 v, u64* sh)
{
    for (int off = 32; off > 0; off >>= 1) {
        const u64 o = __shfl_xor(v, off, 64);
        v = umax64(v, o);
    }
    if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = v;
    __syncthreads();
    u64 r = sh[0];
    for (int i = 1; i < kTopWG / 64; ++i) r = umax64(r, sh[i]);
    __syncthreads();
    return r;
}

// Largest lead count of one counts row as a packed (count, lowest rank) key;
// every thread gets the block result.
__device__ __forceinline__ u64 row_modal_key(const int32_t* __restrict__ c, int R, u64* sh)
{
    const int tid = threadIdx.x;
    u64 b0 = 0, b1 = 0, b2 = 0, b3 = 0;
    auto key = [](int32_t cnt, int r) {
        return ((u64)(uint32_t)cnt << 32) | (u64)(0xFFFFFFFFu - (uint32_t)r);
    };
    if ((R & 3) == 0 && (((uintptr_t)c) & 15) == 0) {
        const int4* c4 = reinterpret_cast<const int4*>(c);
        const int n4 = R >> 2;
        // unrolled so that several loads are in flight at once (the loop is
        // bound by load latency)
#pragma unroll 8
        for (int i = tid; i < n4; i += kTopWG) {
            const int4 x = c4[i];
            const int r = i << 2;
            b0 = umax64(b0, key(x.x, r));
            b1 = umax64(b1, key(x.y, r + 1));
            b2 = umax64(b2, key(x.z, r + 2));
            b3 = umax64(b3, key(x.w, r + 3));
        }
    } else {
        for (int r = tid; r < R; r += kTopWG) b0 = umax64(b0, key(c[r], r));
    }
    return block_max64(umax64(umax64(b0, b1), umax64(b2, b3)), sh);
}

// One workgroup per (window, pick k in {0, 1}); grid-stride.  Both
// workgroups of a window choose the two stages (a block pass over the
// window's S totals); each then finds the most frequent leader of its own
// stage.
__global__ __launch_bounds__(kTopWG) void k_window_top2(const int64_t* __restrict__ exposed,
                                                        const int32_t* __restrict__ counts,
                                                        int R, int S, int64_t W,
                                                        int32_t* __restrict__ top2)
{
    __shared__ u64 sh[kTopWG / 64];
    const int tid = threadIdx.x;
    for (int64_t id = blockIdx.x; id < 2 * W; id += gridDim.x) {
        const int64_t w = id >> 1;
        const int k = (int)(id & 1);
        const int64_t* ex = exposed + w * S;
        int pick0 = -1, pick = -1;
        for (int kk = 0; kk <= k; ++kk) {
            // larger exposed total first, then lower stage index
            int64_t be = 0;
            int bs = -1;
            for (int s = tid; s < S; s += kTopWG) {
                if (s == pick0) continue;
                const int64_t e = ex[s];
                if (bs < 0 || e > be) { be = e; bs = s; }
            }
            // two block maxima: the largest total (sign bit flipped, so that
            // unsigned order is signed order), then the lowest stage among
            // the threads holding it; threads without a stage cannot win
            const u64 ekey = bs < 0 ? 0ull : ((u64)be ^ 0x8000000000000000ull);
            const u64 emax = block_max64(ekey, sh);
            const u64 skey = (bs >= 0 && ekey == emax) ? (u64)(0xFFFFFFFFu - (uint32_t)bs) + 1ull : 0ull;
            const u64 smax = block_max64(skey, sh);
            pick = smax ? (int)(0xFFFFFFFFu - (uint32_t)(smax - 1ull)) : -1;
            pick0 = pick;
        }
        int rank = -1;
        if (pick >= 0) {
            const u64 m = row_modal_key(counts + (w * S + pick) * (int64_t)R, R, sh);
            rank = (m >> 32) ? (int)(0xFFFFFFFFu - (uint32_t)(m & 0xFFFFFFFFull)) : -1;
        }
        if (tid == 0) {
            top2[w * 4 + 2 * k] = pick;
            top2[w * 4 + 2 * k + 1] = rank;
        }
    }
}

// Fused frontier pass and window summary for small inputs (few ranks and
// stages, short windows): one workgroup of 1024 threads per window does the
// whole path of Sec. 3 for the window's steps.  Groups of G lanes own a step
// (K ranks per lane, one rank tile, the packed keys and DPP maxima of
// k_frontier), loading a chunk of stage rows at once; the group's last lane
// writes each boundary's advance and leader as soon as the stage is reduced
// and adds them into the window's LDS totals and lead counts; then the
// workgroup writes the counts and picks the top-2.  One launch instead of
// three, for callers bound by launch latency.
constexpr int kFusedMaxR = 256;
constexpr int kFusedMaxS = 64;
constexpr int64_t kFusedMaxWindow = 1024;
constexpr int64_t kFusedMaxSamples = 1 << 20;

constexpr int kFusedWG = 1024;  // threads of the fused kernel: 1024 / G steps per round

// Sum over the 64 lanes, valid in lane 63 (the DPP pattern of group_max,
// with lanes outside a move's rows or sources reading 0)
__device__ __forceinline__ u64 wave_sum64_dpp(u64 v)
{
#define SF_DPP_ADD(CTRL, ROWS)                                                                        \
    {                                                                                                 \
        const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)v, CTRL, ROWS, 0xF, true); \
        const uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)(v >> 32), CTRL, ROWS, 0xF, true); \
        v += ((u64)hi << 32) | lo;                                                                    \
    }
    SF_DPP_ADD(0xB1, 0xF)   // quad_perm [1,0,3,2]
    SF_DPP_ADD(0x4E, 0xF)   // quad_perm [2,3,0,1]
    SF_DPP_ADD(0x141, 0xF)  // row_half_mirror
    SF_DPP_ADD(0x140, 0xF)  // row_mirror
    SF_DPP_ADD(0x142, 0xA)  // row_bcast:15 -> rows 1, 3
    SF_DPP_ADD(0x143, 0xC)  // row_bcast:31 -> rows 2, 3
#undef SF_DPP_ADD
    return v;
}

template <int VEC, int K, int G>
__global__ __launch_bounds__(kFusedWG) void k_frontier_summary(
    const int64_t* __restrict__ d, int64_t T, int R, int S, int64_t window, int64_t W,
    int64_t* __restrict__ inc, int32_t* __restrict__ lead, int64_t* __restrict__ exposed,
    int32_t* __restrict__ counts, int32_t* __restrict__ top2)
{
    static_assert(K % VEC == 0 && G <= 32, "one DPP group per step");
    constexpr int SPW = kFusedWG / G;  // steps per round
    constexpr int NLD = K / VEC;
    constexpr int CH = K >= 8 ? 1 : 16 / K;  // stage rows loaded at once (up to 16 values per lane)
    __shared__ u64 ex_sh[kFusedMaxS];
    __shared__ int32_t cnt_sh[kFusedMaxS * kFusedMaxR];
    const int tid = threadIdx.x;
    const int gl = tid % G;
    const int j = tid / G;
    const bool writer = gl == G - 1;
    const int SR = S * R;
    for (int64_t w = blockIdx.x; w < W; w += gridDim.x) {
        const int64_t t0 = w * window;
        const int64_t t1 = min(t0 + window, T);
        for (int i = tid; i < S; i += kFusedWG) ex_sh[i] = 0;
        for (int i = tid; i < SR; i += kFusedWG) cnt_sh[i] = 0;
        __syncthreads();
        for (int64_t tb = t0; tb < t1; tb += SPW) {
            // a wave whose first step is past the window has nothing to do;
            // in the others every lane runs the stage loop (the wave sums
            // below need all lanes), and a group past the window loads
            // nothing and contributes nothing
            if (tb + (tid & ~63) / G >= t1) continue;
            const bool act = tb + j < t1;
            const int64_t t = act ? tb + j : t0;
            const int64_t* dt = d + t * (int64_t)S * R;
            u64 q[K];
            int idx[NLD];
#pragma unroll
            for (int l = 0; l < NLD; ++l) {
                const int r = (l * G + gl) * VEC;
                const bool ok = r < R;
                // a slot past R re-reads rank 0 with rank field 0: its key
                // stays strictly below rank 0's own
                idx[l] = ok ? r : 0;
#pragma unroll
                for (int e = 0; e < VEC; ++e) q[l * VEC + e] = ok ? (kRankMask - (u64)(r + e)) : 0ull;
            }
            int64_t Fp = 0;
            for (int s0 = 0; s0 < S; s0 += CH) {
                // the chunk's rows are loaded before any is reduced, so their
                // latencies overlap
                int64_t x[CH][K];
#pragma unroll
                for (int c = 0; c < CH; ++c) {
                    const int64_t* row = dt + (int64_t)(s0 + c) * R;
#pragma unroll
                    for (int l = 0; l < NLD; ++l) {
                        if (!act || s0 + c >= S) {
#pragma unroll
                            for (int e = 0; e < VEC; ++e) x[c][l * VEC + e] = 0;
                        } else if (VEC == 2) {
                            const v2i64 v = *reinterpret_cast<const v2i64*>(row + idx[l]);
                            x[c][2 * l] = v.x;
                            x[c][2 * l + 1] = v.y;
                        } else {
                            x[c][l] = row[idx[l]];
                        }
                    }
                }
#pragma unroll
                for (int c = 0; c < CH; ++c) {
                    const int s = s0 + c;
                    if (s >= S) break;
                    u64 m = 0;
#pragma unroll
                    for (int k = 0; k < K; ++k) {
                        q[k] += (u64)x[c][k] << kRankBits;
                        m = umax64(m, q[k]);
                    }
                    m = group_max<G>(m);
                    const int64_t F = (int64_t)(m >> kRankBits);
                    const bool wr = writer && act;
                    if (wr) {
                        const int r = (int)(kRankMask - (m & kRankMask));
                        inc[t * S + s] = F - Fp;
                        lead[t * S + s] = r;
                        atomicAdd(&cnt_sh[s * R + r], 1);
                    }
                    // the window total: the wave's advances summed first,
                    // one LDS atomic per wave (wraps as int64 sums do)
                    const u64 sum = wave_sum64_dpp(wr ? (u64)(F - Fp) : 0ull);
                    if ((tid & 63) == 63) atomicAdd(&ex_sh[s], sum);
                    Fp = F;
                }
            }
        }
        __syncthreads();
        for (int i = tid; i < S; i += kFusedWG) exposed[w * S + i] = (int64_t)ex_sh[i];
        for (int i = tid; i < SR; i += kFusedWG) counts[w * (int64_t)SR + i] = cnt_sh[i];
        if (tid < 64) {
            // wave 0 alone picks the top-2 with DPP wave maxima (no block
            // barriers): the stage of the largest total (a second max takes
            // the lowest stage among the lanes holding it; S <= 64, one stage
            // per lane), then its most frequent leader (R <= 256, four ranks
            // per lane, the lowest rank on equal counts)
            const int lane = tid;
            int sk = -1;
            for (int k = 0; k < 2; ++k) {
                const bool has = lane < S && lane != sk;
                const u64 ekey = has ? (ex_sh[lane] ^ 0x8000000000000000ull) : 0ull;
                const u64 emax = lane_value(group_max<64>(ekey), 63);
                const u64 skey = (has && ekey == emax) ? (u64)(64 - lane) : 0ull;
                const u64 smax = lane_value(group_max<64>(skey), 63);
                const int pick = smax ? (int)(64 - smax) : -1;  // -1 only when S == 1 and k == 1
                u64 best = 0;
                if (pick >= 0) {
                    for (int r = lane; r < R; r += 64) {
                        const u64 key = ((u64)(uint32_t)cnt_sh[pick * R + r] << 32) | (u64)(0xFFFFFFFFu - (uint32_t)r);
                        best = umax64(best, key);
                    }
                }
                const u64 m = lane_value(group_max<64>(best), 63);
                if (lane == 0) {
                    top2[w * 4 + 2 * k] = pick;
                    top2[w * 4 + 2 * k + 1] = (pick >= 0 && (m >> 32)) ? (int)(0xFFFFFFFFu - (uint32_t)(m & 0xFFFFFFFFull)) : -1;
                }
                sk = pick;
            }
        }
        __syncthreads();  // the LDS tables are cleared for the next window
    }
}

template <int VEC>
const void* pick_fused(int R)
{
    if (R <= 8) return reinterpret_cast<const void*>(&k_frontier_summary<VEC, 2, 4>);
    if (R <= 16) return reinterpret_cast<const void*>(&k_frontier_summary<VEC, 2, 8>);
    if (R <= 32) return reinterpret_cast<const void*>(&k_frontier_summary<VEC, 2, 16>);
    if (R <= 64) return reinterpret_cast<const void*>(&k_frontier_summary<VEC, 2, 32>);
    if (R <= 128) return reinterpret_cast<const void*>(&k_frontier_summary<VEC, 4, 32>);
    return reinterpret_cast<const void*>(&k_frontier_summary<VEC, 8, 32>);  // R <= kFusedMaxR
}

// Exposed time led: the same segmented histogram as k_window_counts, with
// every leader weighted by its advance.  One workgroup per (window, stage,
// rank chunk); 64-bit LDS atomics (two's-complement adds, so any int64
// advance sums exactly as in int64).
constexpr int kLeadChunk = 8192;  // ranks per weighted-histogram workgroup (64 KB LDS)

__global__ __launch_bounds__(kSumWG) void k_window_lead_exposed(
    const int64_t* __restrict__ inc, const int32_t* __restrict__ lead, int64_t T, int R, int S,
    int64_t window, int64_t W, int nchunk, int64_t* __restrict__ lead_exposed)
{
    extern __shared__ u64 whist[];  // [min(R, kLeadChunk)]
    const int tid = threadIdx.x;
    const int64_t total = W * S * nchunk;
    for (int64_t id = blockIdx.x; id < total; id += gridDim.x) {
        const int c = (int)(id % nchunk);
        const int64_t ws = id / nchunk;
        const int s = (int)(ws % S);
        const int64_t w = ws / S;
        const int lo = c * kLeadChunk;
        const int n = min(kLeadChunk, R - lo);
        const int64_t t0 = w * window;
        const int64_t t1 = min(t0 + window, T);

        for (int i = tid; i < n; i += kSumWG) whist[i] = 0;
        __syncthreads();
        for (int64_t t = t0 + tid; t < t1; t += kSumWG) {
            const int64_t r = (int64_t)lead[t * S + s] - lo;
            if (r >= 0 && r < n) atomicAdd(&whist[r], (u64)inc[t * S + s]);
        }
        __syncthreads();
        int64_t* out = lead_exposed + (w * S + s) * (int64_t)R + lo;
        for (int i = tid; i < n; i += kSumWG) out[i] = (int64_t)whist[i];
        __syncthreads();  // whist is reused by the next id
    }
}

// One workgroup per (window, pick k in {0, 1}); grid-stride.  The stage
// totals of the window are summed here from the advances, both workgroups
// of a window choose the same two stages, and each then finds the rank that
// led the most exposed time of its own stage: the largest positive entry of
// the row, the lowest rank on ties.  The sums read the window's [steps][S]
// block in order: with S < WG, thread j takes stage j % S at every P-th
// step from step j / S (P = WG / S phases), and the phases are added in LDS
// (int64 sums wrap alike in any order).
constexpr int kLeadTopLdsS = 2048;  // stages whose window totals are staged in LDS (16 KB)

// The two stages of a window with the largest totals (lower stage first on
// ties), from per-thread candidates: each thread passes its best (e1, s1)
// and second (e2, s2) of the stages it summed (s < 0: none); every thread
// gets the picks.  The second overall is the best of some other thread or
// the second of the thread holding the first.
__device__ __forceinline__ void block_top2_stages(int64_t e1, int s1, int64_t e2, int s2, u64* sh,
                                                  int& p1, int& p2)
{
    auto pick = [&](int64_t e, int st) {
        const u64 ekey = st < 0 ? 0ull : ((u64)e ^ 0x8000000000000000ull);
        const u64 emax = block_max64(ekey, sh);
        const u64 skey = (st >= 0 && ekey == emax) ? (u64)(0xFFFFFFFFu - (uint32_t)st) + 1ull : 0ull;
        const u64 smax = block_max64(skey, sh);
        return smax ? (int)(0xFFFFFFFFu - (uint32_t)(smax - 1ull)) : -1;
    };
    p1 = pick(e1, s1);
    const bool mine = s1 >= 0 && s1 == p1;
    p2 = pick(mine ? e2 : e1, mine ? s2 : s1);
}

__global__ __launch_bounds__(kTopWG) void k_window_lead_top2(
    const int64_t* __restrict__ inc, const int64_t* __restrict__ lead_exposed, int64_t T, int R,
    int S, int64_t window, int64_t W, int32_t* __restrict__ top2)
{
    __shared__ int64_t tot[kLeadTopLdsS];
    __shared__ int64_t part[kTopWG];
    __shared__ u64 sh[kTopWG / 64];
    const int tid = threadIdx.x;
    const int P = S < kTopWG ? kTopWG / S : 1;  // phases per stage
    for (int64_t id = blockIdx.x; id < 2 * W; id += gridDim.x) {
        const int64_t w = id >> 1;
        const int k = (int)(id & 1);
        const int64_t t0 = w * window;
        const int64_t t1 = min(t0 + window, T);
        int pick;
        if (S > kLeadTopLdsS) {
            // many stages: each thread sums its own stages and keeps its two
            // largest; two block maxima pick the window's two
            int64_t e1 = 0, e2 = 0;
            int s1 = -1, s2 = -1;
            for (int s = tid; s < S; s += kTopWG) {
                int64_t acc = 0;
                for (int64_t t = t0; t < t1; ++t) acc += inc[t * S + s];
                if (s1 < 0 || acc > e1) {
                    e2 = e1;
                    s2 = s1;
                    e1 = acc;
                    s1 = s;
                } else if (s2 < 0 || acc > e2) {
                    e2 = acc;
                    s2 = s;
                }
            }
            int p1, p2;
            block_top2_stages(e1, s1, e2, s2, sh, p1, p2);
            pick = k == 0 ? p1 : p2;
        } else {
            if (P > 1) {
                int64_t sum = 0;
                if (tid < P * S) {
                    const int s = tid % S, p = tid / S;
#pragma unroll 8
                    for (int64_t t = t0 + p; t < t1; t += P) sum += inc[t * S + s];
                }
                part[tid] = sum;
                __syncthreads();
                for (int s = tid; s < S; s += kTopWG) {
                    int64_t acc = 0;
                    for (int p = 0; p < P; ++p) acc += part[p * S + s];
                    tot[s] = acc;
                }
            } else {
                for (int s = tid; s < S; s += kTopWG) {
                    int64_t acc = 0;
                    for (int64_t t = t0; t < t1; ++t) acc += inc[t * S + s];
                    tot[s] = acc;
                }
            }
            __syncthreads();
            // larger total first, then lower stage index (every thread alike)
            int s1 = 0;
            for (int s = 1; s < S; ++s)
                if (tot[s] > tot[s1]) s1 = s;
            int s2 = -1;
            for (int s = 0; s < S; ++s)
                if (s != s1 && (s2 < 0 || tot[s] > tot[s2])) s2 = s;
            pick = k == 0 ? s1 : s2;
        }

        int rank = -1;
        if (pick >= 0) {
            const int64_t* row = lead_exposed + (w * S + pick) * (int64_t)R;
            int64_t best = 0;
            int br = -1;
            // unrolled so that several loads are in flight at once: the
            // loop is bound by load latency, not bandwidth
#pragma unroll 8
            for (int r = tid; r < R; r += kTopWG) {
                const int64_t v = row[r];
                if (v > best) { best = v; br = r; }
            }
            // the largest positive value (0 when none), then the lowest rank
            // holding it; threads without a positive value cannot win
            const u64 vmax = block_max64((u64)best, sh);
            const u64 rkey = (br >= 0 && (u64)best == vmax) ? (u64)(0xFFFFFFFFu - (uint32_t)br) + 1ull : 0ull;
            const u64 rmax = block_max64(rkey, sh);
            rank = rmax ? (int)(0xFFFFFFFFu - (uint32_t)(rmax - 1ull)) : -1;
        }
        if (tid == 0) {
            top2[w * 4 + 2 * k] = pick;
            top2[w * 4 + 2 * k + 1] = rank;
        }
        __syncthreads();  // tot and part are rewritten by the next id
    }
}

// Leader switches between confident unique leaders: one wave per (window,
// stage), walking the window 64 steps at a time.  A ballot marks the
// qualifying boundaries; each lane takes the leader of the nearest
// qualifying lane below it (or, for the lowest one, the last qualifying
// leader of the previous 64 steps) and a second ballot counts the changes.
// Every count is wave-uniform, so the lanes need no LDS and no barrier.
constexpr int kSwWG = 256;

__global__ __launch_bounds__(kSwWG) void k_window_switches(
    const int32_t* __restrict__ lead, const int64_t* __restrict__ gap,
    const int32_t* __restrict__ ties, int64_t T, int S, int64_t window, int64_t W,
    int64_t min_gap, int32_t* __restrict__ switches, int32_t* __restrict__ eligible)
{
    const int lane = threadIdx.x & 63;
    const int64_t waves = (int64_t)gridDim.x * (kSwWG / 64);
    for (int64_t id = (int64_t)blockIdx.x * (kSwWG / 64) + (threadIdx.x >> 6); id < W * S;
         id += waves) {
        const int64_t w = id / S;
        const int s = (int)(id - w * S);
        const int64_t t0 = w * window;
        const int64_t t1 = min(t0 + window, T);
        int32_t n_sw = 0, n_el = 0;
        int32_t carry = 0;  // the last qualifying leader so far
        bool have = false;  // whether there is one
        for (int64_t tb = t0; tb < t1; tb += 64) {
            const int64_t t = tb + lane;
            bool q = false;
            int32_t ld = 0;
            if (t < t1) {
                const int64_t i = t * S + s;
                ld = lead[i];
                const int64_t g = gap[i];
                q = ties[i] == 1 && (g >= min_gap || g < 0);
            }
            const u64 m = __ballot(q);
            const u64 below = m & ((1ull << lane) - 1ull);
            const int32_t pv = __shfl(ld, below ? 63 - __clzll((long long)below) : 0, 64);
            const bool has_prev = below != 0 || have;
            const int32_t prev = below ? pv : carry;
            n_sw += __popcll(__ballot(q && has_prev && prev != ld));
            n_el += __popcll(m);
            if (m) {
                carry = __shfl(ld, 63 - __clzll((long long)m), 64);
                have = true;
            }
        }
        if (lane == 0) {
            switches[id] = n_sw;
            eligible[id] = n_el;
        }
    }
}

// Segmented sums over windows of the columns of a [T][C] int64 array: one
// workgroup per (window, column); grid-stride.
__global__ __launch_bounds__(kSumWG) void k_window_sum(const int64_t* __restrict__ x, int64_t T,
                                                       int C, int64_t window, int64_t W,
                                                       int64_t* __restrict__ out)
{
    __shared__ int64_t part[kSumWG / 64];
    const int tid = threadIdx.x;
    for (int64_t id = blockIdx.x; id < W * C; id += gridDim.x) {
        const int64_t w = id / C;
        const int c = (int)(id - w * C);
        const int64_t t0 = w * window;
        const int64_t t1 = min(t0 + window, T);
        int64_t sum = 0;
        for (int64_t t = t0 + tid; t < t1; t += kSumWG) sum += x[t * C + c];
        sum = wave_sum64(sum);
        if ((tid & 63) == 0) part[tid >> 6] = sum;
        __syncthreads();
        if (tid == 0) {
            int64_t acc = 0;
            for (int i = 0; i < kSumWG / 64; ++i) acc += part[i];
            out[w * C + c] = acc;
        }
        __syncthreads();
    }
}

int launch_window_sum(const int64_t* x, int64_t T, int C, int64_t window, int64_t W,
                      int64_t* out, sf_stream_t stream)
{
    const int64_t items = W * C;
    void* args[] = {(void*)&x, (void*)&T, (void*)&C, (void*)&window, (void*)&W, (void*)&out};
    return launch(reinterpret_cast<const void*>(&k_window_sum),
                  dim3((unsigned)(items < 1048576 ? items : 1048576)), dim3(kSumWG), args, 0, stream);
}

}  // namespace sfk

using namespace sfk;

SF_API int64_t sf_num_windows(int64_t T, int64_t window)
{
    if (T < 0 || window < 1) return -1;
    return T / window + (T % window != 0);
}

SF_API int sf_window_summary(const int64_t* increment, const int32_t* leader, int64_t T,
                             int32_t R, int32_t S, int64_t window, int64_t* out_stage_exposed,
                             int32_t* out_lead_counts, int32_t* out_top2, sf_stream_t stream)
{
    if (T < 0 || R < 1 || R > SF_MAX_R || S < 1 || window < 1) return SF_EINVAL;
    if (!fits(T, S, 1, 8)) return SF_EINVAL;
    if (T == 0) return SF_OK;
    const int64_t W = sf_num_windows(T, window);
    if (!fits(W, S, R, 4)) return SF_EINVAL;
    if (!increment || !leader || !out_stage_exposed || !out_lead_counts || !out_top2)
        return SF_EINVAL;
    if (!aligned(increment, 8) || !aligned(leader, 4) || !aligned(out_stage_exposed, 8) ||
        !aligned(out_lead_counts, 4) || !aligned(out_top2, 4))
        return SF_EINVAL;
    const void* bufs[5] = {increment, leader, out_stage_exposed, out_lead_counts, out_top2};
    const int64_t sizes[5] = {T * S * 8, T * S * 4, W * S * 8, W * S * (int64_t)R * 4, W * 16};
    for (int a = 0; a < 5; ++a)
        for (int b = (a < 2 ? 2 : a + 1); b < 5; ++b)
            if (!disjoint(bufs[a], sizes[a], bufs[b], sizes[b])) return SF_EINVAL;

    const int nchunk = (R + kHistChunk - 1) / kHistChunk;
    const int64_t items = W * S * nchunk;
    const unsigned g1 = (unsigned)(items < 1048576 ? items : 1048576);
    const size_t lds = (size_t)(R < kHistChunk ? R : kHistChunk) * sizeof(int32_t);
    int Ri = R, Si = S;
    int64_t Wl = W;
    void* a1[] = {(void*)&increment, (void*)&leader, (void*)&T, (void*)&Ri, (void*)&Si,
                  (void*)&window, (void*)&Wl, (void*)&nchunk, (void*)&out_stage_exposed,
                  (void*)&out_lead_counts};
    int rc = launch(reinterpret_cast<const void*>(&k_window_counts), dim3(g1), dim3(kSumWG), a1,
                    lds, stream);
    if (rc != SF_OK) return rc;
    const unsigned g2 = (unsigned)(2 * W < 65536 ? 2 * W : 65536);
    void* a2[] = {(void*)&out_stage_exposed, (void*)&out_lead_counts, (void*)&Ri, (void*)&Si,
                  (void*)&Wl, (void*)&out_top2};
    return launch(reinterpret_cast<const void*>(&k_window_top2), dim3(g2), dim3(kTopWG), a2, 0,
                  stream);
}

SF_API int sf_window_lead_exposed(const int64_t* increment, const int32_t* leader, int64_t T,
                                  int32_t R, int32_t S, int64_t window, int64_t* out_lead_exposed,
                                  int32_t* out_top2, sf_stream_t stream)
{
    if (T < 0 || R < 1 || R > SF_MAX_R || S < 1 || window < 1) return SF_EINVAL;
    if (!fits(T, S, 1, 8)) return SF_EINVAL;
    if (T == 0) return SF_OK;
    const int64_t W = sf_num_windows(T, window);
    if (!fits(W, S, R, 8)) return SF_EINVAL;
    if (!increment || !leader || !out_lead_exposed || !out_top2) return SF_EINVAL;
    if (!aligned(increment, 8) || !aligned(leader, 4) || !aligned(out_lead_exposed, 8) ||
        !aligned(out_top2, 4))
        return SF_EINVAL;
    const void* bufs[4] = {increment, leader, out_lead_exposed, out_top2};
    const int64_t sizes[4] = {T * S * 8, T * S * 4, W * S * (int64_t)R * 8, W * 16};
    for (int a = 0; a < 4; ++a)
        for (int b = (a < 2 ? 2 : a + 1); b < 4; ++b)
            if (!disjoint(bufs[a], sizes[a], bufs[b], sizes[b])) return SF_EINVAL;

    const int nchunk = (R + kLeadChunk - 1) / kLeadChunk;
    const int64_t items = W * S * nchunk;
    const unsigned g1 = (unsigned)(items < 1048576 ? items : 1048576);
    const size_t lds = (size_t)(R < kLeadChunk ? R : kLeadChunk) * sizeof(u64);
    int Ri = R, Si = S;
    int64_t Wl = W;
    void* a1[] = {(void*)&increment, (void*)&leader, (void*)&T, (void*)&Ri, (void*)&Si,
                  (void*)&window, (void*)&Wl, (void*)&nchunk, (void*)&out_lead_exposed};
    int rc = launch(reinterpret_cast<const void*>(&k_window_lead_exposed), dim3(g1), dim3(kSumWG),
                    a1, lds, stream);
    if (rc != SF_OK) return rc;
    const unsigned g2 = (unsigned)(2 * W < 65536 ? 2 * W : 65536);
    const int64_t* le = out_lead_exposed;
    void* a2[] = {(void*)&increment, (void*)&le, (void*)&T, (void*)&Ri, (void*)&Si,
                  (void*)&window, (void*)&Wl, (void*)&out_top2};
    return launch(reinterpret_cast<const void*>(&k_window_lead_top2), dim3(g2), dim3(kTopWG), a2, 0,
                  stream);
}

SF_API int sf_window_leader_switches(const int32_t* leader, const int64_t* gap,
                                     const int32_t* ties, int64_t T, int32_t S, int64_t window,
                                     int64_t min_gap, int32_t* out_switches,
                                     int32_t* out_eligible, sf_stream_t stream)
{
    if (T < 0 || S < 1 || window < 1) return SF_EINVAL;
    if (!fits(T, S, 1, 8)) return SF_EINVAL;
    if (T == 0) return SF_OK;
    if ((window < T ? window : T) > INT32_MAX) return SF_EINVAL;  // int32 counts
    const int64_t W = sf_num_windows(T, window);
    if (!leader || !gap || !ties || !out_switches || !out_eligible) return SF_EINVAL;
    if (!aligned(leader, 4) || !aligned(gap, 8) || !aligned(ties, 4) || !aligned(out_switches, 4) ||
        !aligned(out_eligible, 4))
        return SF_EINVAL;
    const void* bufs[5] = {leader, gap, ties, out_switches, out_eligible};
    const int64_t sizes[5] = {T * S * 4, T * S * 8, T * S * 4, W * S * 4, W * S * 4};
    for (int a = 0; a < 5; ++a)
        for (int b = (a < 3 ? 3 : a + 1); b < 5; ++b)
            if (!disjoint(bufs[a], sizes[a], bufs[b], sizes[b])) return SF_EINVAL;

    const int64_t blocks = (W * S + kSwWG / 64 - 1) / (kSwWG / 64);
    const unsigned g = (unsigned)(blocks < 65536 ? blocks : 65536);
    int Si = S;
    int64_t Wl = W;
    void* a[] = {(void*)&leader, (void*)&gap, (void*)&ties, (void*)&T, (void*)&Si, (void*)&window,
                 (void*)&Wl, (void*)&min_gap, (void*)&out_switches, (void*)&out_eligible};
    return launch(reinterpret_cast<const void*>(&k_window_switches), dim3(g), dim3(kSwWG), a, 0,
                  stream);
}

SF_API int sf_frontier_summary(const int64_t* durations, int64_t T, int32_t R, int32_t S,
                               int64_t window, int64_t* out_increment, int32_t* out_leader,
                               int64_t* out_stage_exposed, int32_t* out_lead_counts,
                               int32_t* out_top2, sf_stream_t stream)
{
    if (T < 0 || R < 1 || R > SF_MAX_R || S < 1 || window < 1) return SF_EINVAL;
    if (!fits(T, S, R, 8)) return SF_EINVAL;
    if (T == 0) return SF_OK;
    const int64_t W = sf_num_windows(T, window);
    if (!fits(W, S, R, 4)) return SF_EINVAL;
    const void* bufs[6] = {durations, out_increment, out_leader, out_stage_exposed,
                           out_lead_counts, out_top2};
    const int64_t sizes[6] = {T * S * (int64_t)R * 8, T * S * 8, T * S * 4, W * S * 8,
                              W * S * (int64_t)R * 4, W * 16};
    const uintptr_t align[6] = {8, 8, 4, 8, 4, 4};
    for (int a = 0; a < 6; ++a)
        if (!bufs[a] || !aligned(bufs[a], align[a])) return SF_EINVAL;
    for (int a = 0; a < 6; ++a)
        for (int b = a + 1; b < 6; ++b)
            if (!disjoint(bufs[a], sizes[a], bufs[b], sizes[b])) return SF_EINVAL;
    const int64_t n_max = window < T ? window : T;
    if (R <= kFusedMaxR && S <= kFusedMaxS && n_max <= kFusedMaxWindow &&
        T * S * (int64_t)R <= kFusedMaxSamples) {
        const bool vec2 = (R % 2 == 0) && aligned(durations, 16);
        const void* fn = vec2 ? pick_fused<2>(R) : pick_fused<1>(R);
        int Ri = R, Si = S;
        int64_t Wl = W;
        void* args[] = {(void*)&durations,         (void*)&T,               (void*)&Ri,
                        (void*)&Si,                (void*)&window,          (void*)&Wl,
                        (void*)&out_increment,     (void*)&out_leader,      (void*)&out_stage_exposed,
                        (void*)&out_lead_counts,   (void*)&out_top2};
        return launch(fn, dim3((unsigned)(W < 65536 ? W : 65536)), dim3(kFusedWG), args, 0, stream);
    }
    const int rc = sf_frontier(durations, T, R, S, out_increment, out_leader, stream);
    if (rc != SF_OK) return rc;
    return sf_window_summary(out_increment, out_leader, T, R, S, window, out_stage_exposed,
                             out_lead_counts, out_top2, stream);
}
