// stagefrontier.hip -- HIP kernels for gfx950 (MI355X) and the C ABI of
// libstagefrontier: StageFrontier frontier accounting (Sec. 3, Eq. (1) and
// Eq. (2); top-2 routing of Sec. 4).
//
// Data layout in HBM: durations [T][S][R] int64 (rank fastest), per-step
// outputs [T][S], window outputs [W][S], [W][S][R] and [W][2][2].
//
// Frontier kernel.  Every step is independent (Sec. 3 streams one step at a
// time), so the grid walks the step axis; inside a step, a group of G lanes
// owns the step and each lane owns K ranks of a tile of G*K ranks.  The lane
// keeps the running prefix of each of its ranks in registers as a packed key
//     q = (P << 16) | (0xFFFF - r)
// so that an unsigned 64-bit max over keys yields the largest prefix and, on
// equal prefixes, the lowest rank.  Adding a duration shifted left by 16
// advances P without touching the rank field, so the key is built once per
// rank and then only added to.  Per stage, a lane takes the max of its K
// keys, the group reduces with DPP lane moves (quad_perm, row mirrors,
// row broadcasts: no LDS traffic), and the last lane of each 64-lane (or
// smaller) sub-group stores the partial max in LDS.  After the last stage
// the workgroup decodes F and the leader per (step, stage), takes the
// advance F[s] - F[s-1] and writes [T][S] rows with contiguous stores.
// Durations are read exactly once, with 16-byte loads when R is even.
//
// Window kernels.  One workgroup per (window, stage, rank chunk) builds the
// leader histogram of the window in LDS with LDS atomics and sums the
// advances; one workgroup per window then picks the two largest stages and
// their most frequent leaders.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "stagefrontier.h"

#define SF_API extern "C" __attribute__((visibility("default")))

namespace {

typedef unsigned long long u64;
typedef long long v2i64 __attribute__((ext_vector_type(2)));

constexpr int kRankBits = 16;
constexpr u64 kRankMask = 0xFFFFull;

__device__ __forceinline__ u64 umax64(u64 a, u64 b) { return a > b ? a : b; }

// One DPP lane move of a 64-bit value.  Lanes outside ROW_MASK, and lanes
// whose source is out of range, keep their own value, which is neutral for
// a max.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ u64 dpp_move(u64 v)
{
    const int lo = (int)(uint32_t)v;
    const int hi = (int)(uint32_t)(v >> 32);
    const uint32_t nlo = (uint32_t)__builtin_amdgcn_update_dpp(lo, lo, CTRL, ROW_MASK, 0xF, false);
    const uint32_t nhi = (uint32_t)__builtin_amdgcn_update_dpp(hi, hi, CTRL, ROW_MASK, 0xF, false);
    return ((u64)nhi << 32) | nlo;
}

// Max over aligned groups of SUB lanes (SUB a power of two <= 64).  The
// result is valid in the last lane of each group (in every lane of the
// group for SUB <= 16).
template <int SUB>
__device__ __forceinline__ u64 group_max(u64 v)
{
    if (SUB >= 2) v = umax64(v, dpp_move<0xB1, 0xF>(v));   // quad_perm [1,0,3,2]
    if (SUB >= 4) v = umax64(v, dpp_move<0x4E, 0xF>(v));   // quad_perm [2,3,0,1]
    if (SUB >= 8) v = umax64(v, dpp_move<0x141, 0xF>(v));  // row_half_mirror
    if (SUB >= 16) v = umax64(v, dpp_move<0x140, 0xF>(v)); // row_mirror
    if (SUB >= 32) v = umax64(v, dpp_move<0x142, 0xA>(v)); // row_bcast:15 -> rows 1, 3
    if (SUB >= 64) v = umax64(v, dpp_move<0x143, 0xC>(v)); // row_bcast:31 -> rows 2, 3
    return v;
}

// ---------------------------------------------------------------------------
// frontier kernel

// VEC: int64 elements per load (2: 16-byte loads, needs even R and a 16-byte
//      aligned base); K: ranks per lane per tile; G: lanes per step;
// WG:  threads per workgroup (WG / G steps per workgroup).
template <int VEC, int K, int G, int WG>
__global__ __launch_bounds__(WG) void k_frontier(const int64_t* __restrict__ d, int64_t T,
                                                 int R, int S, int64_t* __restrict__ inc,
                                                 int32_t* __restrict__ lead)
{
    static_assert(K % VEC == 0, "K must be a multiple of VEC");
    static_assert(WG % G == 0 || G == WG, "a workgroup holds whole steps");
    constexpr int SUB = G < 64 ? G : 64;  // lanes per DPP reduction group
    constexpr int SPW = WG / G;           // steps per workgroup
    constexpr int SPS = G / SUB;          // LDS slots per step
    constexpr int NLD = K / VEC;          // loads per lane per stage row
    constexpr int RT = G * K;             // ranks per tile

    extern __shared__ u64 tab[];          // [WG / SUB][S] partial maxima

    const int tid = threadIdx.x;
    const int gl = tid % G;
    const int j = tid / G;
    const int slot = tid / SUB;
    const bool writer = (tid % SUB) == SUB - 1;
    const int64_t t = (int64_t)blockIdx.x * SPW + j;

    if (t < T) {  // uniform over the step group
        const int64_t* dt = d + t * (int64_t)S * R;
        for (int r0 = 0; r0 < R; r0 += RT) {
            u64 q[K];
            bool ok[NLD];
#pragma unroll
            for (int l = 0; l < NLD; ++l) {
                const int r = r0 + (l * G + gl) * VEC;
                ok[l] = r < R;
#pragma unroll
                for (int e = 0; e < VEC; ++e)
                    q[l * VEC + e] = ok[l] ? (kRankMask - (u64)(r + e)) : 0ull;
            }
            int64_t v[K];
            auto load_row = [&](int s) {
                const int64_t* row = dt + (int64_t)s * R + r0;
                // A lane slot past R reads the tile's first rank instead (in
                // bounds, no branch).  Its key starts with rank field 0, so it
                // tracks that rank's prefix with a key strictly below the
                // rank's own key and can never be the maximum.
#pragma unroll
                for (int l = 0; l < NLD; ++l) {
                    const int idx = ok[l] ? (l * G + gl) * VEC : 0;
                    if (VEC == 2) {
                        const v2i64 x = __builtin_nontemporal_load(reinterpret_cast<const v2i64*>(row + idx));
                        v[2 * l] = x.x;
                        v[2 * l + 1] = x.y;
                    } else {
                        v[l] = __builtin_nontemporal_load(row + idx);
                    }
                }
            };
            load_row(0);
            for (int s = 0; s < S; ++s) {
                u64 m = 0;
#pragma unroll
                for (int k = 0; k < K; ++k) {
                    q[k] += (u64)v[k] << kRankBits;
                    m = umax64(m, q[k]);
                }
                if (s + 1 < S) load_row(s + 1);
                m = group_max<SUB>(m);
                if (writer) {
                    u64* p = &tab[slot * S + s];
                    *p = (r0 == 0) ? m : umax64(*p, m);
                }
            }
        }
    }
    __syncthreads();

    // decode F and the leader per (step, stage); rows of out are contiguous
    const int64_t tb = (int64_t)blockIdx.x * SPW;
    for (int i = tid; i < SPW * S; i += WG) {
        const int jj = i / S;
        const int s = i - jj * S;
        const int64_t tt = tb + jj;
        if (tt >= T) break;
        u64 key = 0, kprev = 0;
#pragma unroll
        for (int qd = 0; qd < SPS; ++qd) {
            key = umax64(key, tab[(jj * SPS + qd) * S + s]);
            if (s > 0) kprev = umax64(kprev, tab[(jj * SPS + qd) * S + s - 1]);
        }
        const int64_t F = (int64_t)(key >> kRankBits);
        const int64_t Fp = (int64_t)(kprev >> kRankBits);
        inc[tt * S + s] = F - Fp;
        lead[tt * S + s] = (int32_t)(kRankMask - (key & kRankMask));
    }
}

struct FrontierVariant {
    const void* fn;
    int K, G, WG;
    int per_cu;  // resident workgroups per CU to allow (0: no cap)
};

template <int VEC, int K, int G, int WG>
FrontierVariant variant(int per_cu)
{
    return FrontierVariant{reinterpret_cast<const void*>(&k_frontier<VEC, K, G, WG>), K, G, WG,
                           per_cu};
}

// Launch shape by rank count, measured on MI355X over R = 16 .. 16384.
// Wide per-lane tiles (K = 32 ranks, about 250 VGPRs) and few resident
// workgroups per CU read HBM fastest for large R: fewer concurrent step
// streams, each with up to 32 KB of loads in flight per wave.  A tile wider
// than R costs no HBM traffic (lane slots past R re-read a cached rank).
template <int VEC>
FrontierVariant pick_frontier(int R)
{
    if (R <= 8) return variant<VEC, 2, 4, 64>(0);
    if (R <= 16) return variant<VEC, 2, 8, 128>(0);
    if (R <= 32) return variant<VEC, 4, 8, 128>(0);
    if (R <= 64) return variant<VEC, 4, 16, 256>(6);
    if (R <= 128) return variant<VEC, 8, 32, 256>(6);
    if (R <= 256) return variant<VEC, 16, 32, 256>(4);
    if (R <= 512) return variant<VEC, 4, 256, 256>(0);
    if (R <= 1024) return variant<VEC, 32, 64, 256>(6);
    if (R <= 2048) return variant<VEC, 8, 512, 512>(0);
    if (R <= 4096) return variant<VEC, 32, 256, 256>(0);
    return variant<VEC, 32, 64, 64>(3);
}

// LDS on one gfx950 CU.  Asking for LDS_PER_CU / n bytes per workgroup caps
// residency at n workgroups per CU.
constexpr size_t kLdsPerCu = 160 * 1024;
constexpr size_t kLdsMaxPerWg = 64 * 1024;

size_t lds_request(size_t need, int per_cu)
{
    if (per_cu <= 0) return need;
    size_t cap = (kLdsPerCu / (size_t)per_cu) & ~(size_t)1023;
    if (cap > kLdsMaxPerWg) cap = kLdsMaxPerWg;
    return need > cap ? need : cap;
}

// ---------------------------------------------------------------------------
// window kernels

constexpr int kHistChunk = 16384;  // ranks per histogram workgroup (64 KB LDS)
constexpr int kSumWG = 256;

__device__ __forceinline__ int64_t wave_sum64(int64_t v)
{
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
    return v;
}

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
        for (int64_t t = t0 + tid; t < t1; t += kSumWG) {
            const int64_t r = (int64_t)lead[t * S + s] - lo;
            if (r >= 0 && r < n) atomicAdd(&hist[r], 1);
        }
        if (c == 0) {
            int64_t sum = 0;
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
// workgroups of a window choose the two stages (cheap: S <= SF_MAX_S); each
// then finds the most frequent leader of its own stage.
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

// ---------------------------------------------------------------------------
// evidence kernel: the frontier pass plus, per boundary, the runner-up gap and
// the tie-set size (localization evidence, Sec. 4) and max_r d / sum_r d
// (the per-stage terms of the max and mean baselines, Props. 1 and 2).
//
// One workgroup per step (WG = 64 or 128 threads).  Each lane accumulates,
// over its ranks of a tile, the two largest packed keys, the number of its
// ranks whose prefix equals that of its largest key, and the max and sum of
// the stage's durations.  The wave reduces these with DPP lane moves.  Sums
// and counts are not idempotent, so every move used gives each receiving lane
// a distinct partner; lanes a row broadcast does not reach hold partial
// values that are never read.  The full result is in lane 63.

struct EvAcc {
    u64 k1, k2;      // largest and second-largest packed key
    int64_t smax;    // max of d over ranks
    int64_t ssum;    // sum of d over ranks
    uint32_t c;      // ranks whose prefix equals that of k1
};

__device__ __forceinline__ u64 umin64(u64 a, u64 b) { return a < b ? a : b; }

__device__ __forceinline__ void ev_merge(EvAcc& a, const EvAcc& b)
{
    const u64 pa = a.k1 >> kRankBits, pb = b.k1 >> kRankBits;
    a.c = pa > pb ? a.c : (pb > pa ? b.c : a.c + b.c);
    a.k2 = umax64(umin64(a.k1, b.k1), umax64(a.k2, b.k2));
    a.k1 = umax64(a.k1, b.k1);
    a.smax = a.smax > b.smax ? a.smax : b.smax;
    a.ssum += b.ssum;
}

template <int CTRL, int ROW_MASK>
__device__ __forceinline__ EvAcc ev_move(const EvAcc& a)
{
    EvAcc b;
    b.k1 = dpp_move<CTRL, ROW_MASK>(a.k1);
    b.k2 = dpp_move<CTRL, ROW_MASK>(a.k2);
    b.smax = (int64_t)dpp_move<CTRL, ROW_MASK>((u64)a.smax);
    b.ssum = (int64_t)dpp_move<CTRL, ROW_MASK>((u64)a.ssum);
    b.c = (uint32_t)__builtin_amdgcn_update_dpp((int)a.c, (int)a.c, CTRL, ROW_MASK, 0xF, false);
    return b;
}

// Merge over aligned groups of SUB lanes (a power of two <= 64); the result
// is valid in the last lane of each group.
template <int SUB>
__device__ __forceinline__ EvAcc ev_group_reduce(EvAcc a)
{
    if (SUB >= 2) ev_merge(a, ev_move<0xB1, 0xF>(a));   // quad_perm [1,0,3,2]: lane ^ 1
    if (SUB >= 4) ev_merge(a, ev_move<0x4E, 0xF>(a));   // quad_perm [2,3,0,1]: lane ^ 2
    if (SUB >= 8) ev_merge(a, ev_move<0x141, 0xF>(a));  // row_half_mirror: other quad of 8
    if (SUB >= 16) ev_merge(a, ev_move<0x140, 0xF>(a)); // row_mirror: other half of the row
    if (SUB >= 32) ev_merge(a, ev_move<0x142, 0xA>(a)); // row_bcast:15: row 0 -> 1, row 2 -> 3
    if (SUB >= 64) ev_merge(a, ev_move<0x143, 0xC>(a)); // row_bcast:31: rows 0-1 -> row 3
    return a;
}

__device__ __forceinline__ void ev_store(int64_t i, const EvAcc& a, u64 kprev, int R,
                                         int64_t* inc, int32_t* lead, int64_t* gap,
                                         int32_t* ties, int64_t* stage_max, int64_t* stage_sum)
{
    const int64_t F = (int64_t)(a.k1 >> kRankBits);
    inc[i] = F - (int64_t)(kprev >> kRankBits);
    lead[i] = (int32_t)(kRankMask - (a.k1 & kRankMask));
    gap[i] = R > 1 ? F - (int64_t)(a.k2 >> kRankBits) : -1;
    ties[i] = (int32_t)a.c;
    stage_max[i] = a.smax;
    stage_sum[i] = a.ssum;
}

// Same step/lane layout as k_frontier: G lanes per step, K ranks per lane,
// WG / G steps per workgroup.  When one group of at most 64 lanes covers all
// R ranks of its step, the group's last lane writes each boundary's outputs
// as soon as the stage is reduced; otherwise partial results go through LDS
// (5 arrays of [WG / min(G, 64)][S]) and the workgroup writes them at the end.
template <int VEC, int K, int G, int WG>
__global__ __launch_bounds__(WG) void k_frontier_evidence(
    const int64_t* __restrict__ d, int64_t T, int R, int S, int64_t* __restrict__ inc,
    int32_t* __restrict__ lead, int64_t* __restrict__ gap, int32_t* __restrict__ ties,
    int64_t* __restrict__ stage_max, int64_t* __restrict__ stage_sum)
{
    static_assert(K % VEC == 0 && (WG % G == 0 || G == WG), "shape");
    constexpr int SUB = G < 64 ? G : 64;
    constexpr int SPW = WG / G;
    constexpr int SPS = G / SUB;
    constexpr int NSLOT = WG / SUB;
    constexpr int NLD = K / VEC;
    constexpr int RT = G * K;

    extern __shared__ u64 evtab[];
    u64* t_k1 = evtab;
    u64* t_k2 = t_k1 + NSLOT * S;
    u64* t_c = t_k2 + NSLOT * S;
    u64* t_max = t_c + NSLOT * S;
    u64* t_sum = t_max + NSLOT * S;

    const bool direct = SPS == 1 && R <= RT;  // uniform over the launch
    const int tid = threadIdx.x;
    const int gl = tid % G;
    const int slot = tid / SUB;
    const bool writer = (tid % SUB) == SUB - 1;
    const int64_t tb = (int64_t)blockIdx.x * SPW;
    const int64_t t = tb + tid / G;

    if (t < T) {  // uniform over the step group
        const int64_t* dt = d + t * (int64_t)S * R;
        for (int r0 = 0; r0 < R; r0 += RT) {
            u64 q[K];
            bool ok[NLD];
#pragma unroll
            for (int l = 0; l < NLD; ++l) {
                const int r = r0 + (l * G + gl) * VEC;
                ok[l] = r < R;
#pragma unroll
                for (int e = 0; e < VEC; ++e)
                    q[l * VEC + e] = ok[l] ? (kRankMask - (u64)(r + e)) : 0ull;
            }
            int64_t v[K];
            auto load_row = [&](int s) {
                const int64_t* row = dt + (int64_t)s * R + r0;
#pragma unroll
                for (int l = 0; l < NLD; ++l) {
                    const int idx = ok[l] ? (l * G + gl) * VEC : 0;
                    if (VEC == 2) {
                        const v2i64 x = __builtin_nontemporal_load(reinterpret_cast<const v2i64*>(row + idx));
                        v[2 * l] = x.x;
                        v[2 * l + 1] = x.y;
                    } else {
                        v[l] = __builtin_nontemporal_load(row + idx);
                    }
                }
            };
            load_row(0);
            u64 kprev = 0;
            for (int s = 0; s < S; ++s) {
                EvAcc a;
                a.k1 = 0;
                a.k2 = 0;
                a.smax = 0;
                a.ssum = 0;
                a.c = 0;
#pragma unroll
                for (int k = 0; k < K; ++k) {
                    // slots past R carry no rank: their duration counts as 0
                    // and their key stays 0, below every real key
                    const int64_t dv = ok[k / VEC] ? v[k] : 0;
                    q[k] += (u64)dv << kRankBits;
                    a.k2 = umax64(a.k2, umin64(a.k1, q[k]));
                    a.k1 = umax64(a.k1, q[k]);
                    a.smax = a.smax > dv ? a.smax : dv;
                    a.ssum += dv;
                }
#pragma unroll
                for (int k = 0; k < K; ++k)
                    a.c += (ok[k / VEC] && ((q[k] ^ a.k1) >> kRankBits) == 0) ? 1u : 0u;
                if (s + 1 < S) load_row(s + 1);
                a = ev_group_reduce<SUB>(a);
                if (writer) {
                    if (direct) {
                        ev_store(t * S + s, a, kprev, R, inc, lead, gap, ties, stage_max, stage_sum);
                        kprev = a.k1;
                    } else {
                        const int i = slot * S + s;
                        if (r0 > 0) {
                            EvAcc b;
                            b.k1 = t_k1[i];
                            b.k2 = t_k2[i];
                            b.c = (uint32_t)t_c[i];
                            b.smax = (int64_t)t_max[i];
                            b.ssum = (int64_t)t_sum[i];
                            ev_merge(a, b);
                        }
                        t_k1[i] = a.k1;
                        t_k2[i] = a.k2;
                        t_c[i] = a.c;
                        t_max[i] = (u64)a.smax;
                        t_sum[i] = (u64)a.ssum;
                    }
                }
            }
        }
    }
    if (direct) return;
    __syncthreads();

    for (int i = tid; i < SPW * S; i += WG) {
        const int jj = i / S;
        const int s = i - jj * S;
        const int64_t tt = tb + jj;
        if (tt >= T) break;
        EvAcc a, p;
        const int i0 = jj * SPS * S + s;
        a.k1 = t_k1[i0];
        a.k2 = t_k2[i0];
        a.c = (uint32_t)t_c[i0];
        a.smax = (int64_t)t_max[i0];
        a.ssum = (int64_t)t_sum[i0];
        u64 kp = s > 0 ? t_k1[i0 - 1] : 0;
#pragma unroll
        for (int qd = 1; qd < SPS; ++qd) {
            const int iq = (jj * SPS + qd) * S + s;
            p.k1 = t_k1[iq];
            p.k2 = t_k2[iq];
            p.c = (uint32_t)t_c[iq];
            p.smax = (int64_t)t_max[iq];
            p.ssum = (int64_t)t_sum[iq];
            ev_merge(a, p);
            if (s > 0) kp = umax64(kp, t_k1[iq - 1]);
        }
        ev_store(tt * S + s, a, kp, R, inc, lead, gap, ties, stage_max, stage_sum);
    }
}

struct EvidenceVariant {
    const void* fn;
    int K, G, WG;
    int per_cu;  // resident workgroups per CU to allow (0: no cap)
};

template <int VEC, int K, int G, int WG>
EvidenceVariant ev_variant(int per_cu)
{
    return EvidenceVariant{reinterpret_cast<const void*>(&k_frontier_evidence<VEC, K, G, WG>), K,
                           G, WG, per_cu};
}

// LDS bytes a variant needs: none when one group of <= 64 lanes covers the
// step's ranks, else 5 arrays of [WG / min(G, 64)][S] u64.
size_t ev_lds_need(const EvidenceVariant& v, int R, int S)
{
    const int sub = v.G < 64 ? v.G : 64;
    if (v.G <= 64 && R <= v.G * v.K) return 0;
    return (size_t)5 * (v.WG / sub) * S * 8;
}

// Launch shape by rank count, measured on MI355X; a shape whose LDS would
// exceed 64 KB at this S falls back to two 64-lane slots per step
// (80 * S bytes, at most 40 KB).
template <int VEC>
EvidenceVariant pick_evidence(int R, int S)
{
    EvidenceVariant v;
    if (R <= 8) v = ev_variant<VEC, 2, 4, 64>(0);
    else if (R <= 16) v = ev_variant<VEC, 2, 8, 64>(0);
    else if (R <= 32) v = ev_variant<VEC, 4, 8, 64>(0);
    else if (R <= 64) v = ev_variant<VEC, 4, 16, 64>(0);
    else if (R <= 128) v = ev_variant<VEC, 8, 16, 256>(8);
    else if (R <= 256) v = ev_variant<VEC, 8, 16, 256>(8);
    else if (R <= 512) v = ev_variant<VEC, 16, 32, 64>(0);
    else if (R <= 1024) v = ev_variant<VEC, 16, 32, 64>(8);
    else if (R <= 4096) v = ev_variant<VEC, 16, 256, 256>(2);
    else v = ev_variant<VEC, 32, 256, 256>(0);
    if (ev_lds_need(v, R, S) > kLdsMaxPerWg) v = ev_variant<VEC, 16, 128, 128>(0);
    return v;
}

// ---------------------------------------------------------------------------
// ingest kernel: gathered per-rank buffers -> [T][S][R] with the Appendix A
// closure (residual stage last, overlap error aside).
//
// A workgroup owns RB ranks x TB steps.  Reading: each wave takes whole
// ranks and streams the rank's TB*K contiguous explicit durations into an
// LDS row (rows padded to an odd length, so that the column reads below hit
// distinct banks).  Closure: one thread per (step, rank) sums its K values
// and forms the residual max(0, e) and the overlap max(0, -e).  Writing: each
// wave writes whole [t][s] rows of RB ranks with contiguous stores.  Every
// index comes from the loop structure or from a power-of-two RB; nothing is
// divided by a runtime value per element.

constexpr int kIngestWG = 256;

struct IngestTile {
    const void* fn;
    int RB, TB, segp;
    size_t lds;
};

template <int RB, bool BATCH>
__global__ __launch_bounds__(kIngestWG) void k_ingest(const int64_t* __restrict__ x,
                                                      const int64_t* __restrict__ w, int64_t T,
                                                      int R, int K, int TB, int segp,
                                                      int64_t* __restrict__ d,
                                                      int64_t* __restrict__ o)
{
    static_assert(RB <= 64 && (64 % RB) == 0, "RB divides a wave");
    constexpr int ROWS_PER_WAVE = 64 / RB;
    extern __shared__ int64_t tile[];  // [RB][segp] explicit, then res/ovl [TB][RB] each
    int64_t* res = tile + (size_t)RB * segp;
    int64_t* ovl = res + (size_t)TB * RB;
    const int S = K + 1;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int nwave = kIngestWG / 64;
    const int64_t nrb = (R + RB - 1) / RB;
    const int64_t ntb = (T + TB - 1) / TB;
    for (int64_t blk = blockIdx.x; blk < nrb * ntb; blk += gridDim.x) {
        const int r0 = (int)(blk % nrb) * RB;
        const int64_t t0 = (blk / nrb) * TB;
        const int rn = min(RB, R - r0);
        const int tn = (int)min((int64_t)TB, T - t0);
        const int seg = tn * K;
        if (BATCH) {
            // seg <= 64: lane e of wave q reads element e of ranks
            // q, q + nwave, ... ; all RB / nwave loads are issued before any
            // is stored, so each lane keeps them in flight together
            constexpr int PER = RB / 4;
            int64_t v[PER];
#pragma unroll
            for (int m = 0; m < PER; ++m) {
                const int j = wave + m * nwave;
                const bool ok = lane < seg && j < rn;
                const int64_t* src = x + ((int64_t)(r0 + (ok ? j : 0)) * T + t0) * K;
                v[m] = ok ? src[lane] : 0;
            }
#pragma unroll
            for (int m = 0; m < PER; ++m) {
                const int j = wave + m * nwave;
                if (lane < seg && j < rn) tile[j * segp + lane] = v[m];
            }
        } else {
            // one wave per rank, lanes along the rank's contiguous segment
            for (int j = wave; j < rn; j += nwave) {
                const int64_t* src = x + ((int64_t)(r0 + j) * T + t0) * K;
                for (int e = lane; e < seg; e += 64) tile[j * segp + e] = src[e];
            }
        }
        for (int i = tid; i < tn * RB; i += kIngestWG) {
            const int tl = i / RB;  // RB is a power of two
            const int j = i & (RB - 1);
            if (j < rn) res[i] = w[(int64_t)(r0 + j) * T + t0 + tl];
        }
        __syncthreads();
        // closure per (step, rank): res holds w on entry
        for (int i = tid; i < tn * RB; i += kIngestWG) {
            const int tl = i / RB;
            const int j = i & (RB - 1);
            if (j >= rn) continue;
            const int64_t* row = tile + j * segp + tl * K;
            int64_t sum = 0;
            for (int k = 0; k < K; ++k) sum += row[k];
            const int64_t e = res[i] - sum;
            res[i] = e > 0 ? e : 0;
            ovl[i] = e < 0 ? -e : 0;
        }
        __syncthreads();
        // write: each wave writes ROWS_PER_WAVE [t][s] rows of RB ranks at once
        const int sub = lane / RB;
        const int j = lane & (RB - 1);
        const int nrows = tn * S;
        constexpr int UW = 4;  // rows per wave in flight
        for (int row0 = wave * ROWS_PER_WAVE; row0 < nrows; row0 += UW * nwave * ROWS_PER_WAVE) {
            int64_t v[UW];
            int64_t* dst[UW];
#pragma unroll
            for (int u = 0; u < UW; ++u) {
                const int row = row0 + u * nwave * ROWS_PER_WAVE + sub;
                dst[u] = nullptr;
                v[u] = 0;
                if (row < nrows && j < rn) {
                    const int tl = row / S;
                    const int s = row - tl * S;
                    v[u] = s < K ? tile[j * segp + tl * K + s] : res[tl * RB + j];
                    dst[u] = d + ((t0 + tl) * S + s) * (int64_t)R + r0 + j;
                }
            }
#pragma unroll
            for (int u = 0; u < UW; ++u)
                if (dst[u]) *dst[u] = v[u];
        }
        for (int i = tid; i < tn * RB; i += kIngestWG) {
            const int tl = i / RB;
            const int jj = i & (RB - 1);
            if (jj < rn) o[(t0 + tl) * (int64_t)R + r0 + jj] = ovl[i];
        }
        __syncthreads();  // the tile is reused by the next block
    }
}

template <int RB, bool BATCH>
IngestTile ingest_variant(int K, int64_t T)
{
    // LDS budget 48 KB: RB rows of TB*K (+ padding) plus two [TB][RB] arrays;
    // the batched read also needs TB*K <= 64
    const int64_t per_step = (int64_t)RB * K * 8 + 2 * (int64_t)RB * 8;
    int64_t tb = (48 * 1024 - (int64_t)RB * 16) / per_step;
    if (BATCH && K > 0 && tb > 64 / K) tb = 64 / K;
    if (tb < 1) tb = 1;
    if (tb > T) tb = T;
    int segp = (int)tb * K + 1;
    if ((segp & 1) == 0) segp += 1;
    IngestTile g;
    g.fn = reinterpret_cast<const void*>(&k_ingest<RB, BATCH>);
    g.RB = RB;
    g.TB = (int)tb;
    g.segp = segp;
    g.lds = (size_t)RB * segp * 8 + 2 * (size_t)tb * RB * 8;
    return g;
}

IngestTile pick_ingest(int K, int64_t T)
{
    if (K <= 64) return ingest_variant<64, true>(K, T);
    if (K <= 256) return ingest_variant<16, false>(K, T);
    return ingest_variant<8, false>(K, T);
}

// ---------------------------------------------------------------------------
// routing-set kernel (Sec. 4): per window, stages by exposed total
// (descending, lower stage first) and the smallest leading prefix whose
// exposed sum reaches tau_num / tau_den of the window total, compared
// exactly in 128-bit integers.  One workgroup per window.

constexpr int kRouteWG = 256;

__global__ __launch_bounds__(kRouteWG) void k_route(const int64_t* __restrict__ exposed,
                                                    int64_t W, int S, int64_t tau_num,
                                                    int64_t tau_den, int32_t* __restrict__ order,
                                                    int32_t* __restrict__ size)
{
    __shared__ int64_t ex[SF_MAX_S];
    __shared__ int64_t sorted_ex[SF_MAX_S];
    const int tid = threadIdx.x;
    for (int64_t win = blockIdx.x; win < W; win += gridDim.x) {
        for (int s = tid; s < S; s += kRouteWG) ex[s] = exposed[win * S + s];
        __syncthreads();
        // position of stage s = number of stages that come before it
        for (int s = tid; s < S; s += kRouteWG) {
            const int64_t e = ex[s];
            int pos = 0;
            for (int u = 0; u < S; ++u) pos += (ex[u] > e || (ex[u] == e && u < s)) ? 1 : 0;
            order[win * S + pos] = s;
            sorted_ex[pos] = e;
        }
        __syncthreads();
        // wave 0 scans the sorted totals: each lane sums a contiguous part,
        // an exclusive scan over lanes gives each part's starting sum, and
        // each lane finds the first prefix in its part that reaches tau
        if (tid < 64) {
            const int per = (S + 63) / 64;
            const int b = tid * per;
            const int e = min(S, b + per);
            __int128 part = 0;
            for (int i = b; i < e; ++i) part += sorted_ex[i];
            // exclusive scan of the 64 lane parts (two 64-bit halves per step)
            __int128 incl = part;
            for (int off = 1; off < 64; off <<= 1) {
                const uint64_t lo = (uint64_t)incl, hi = (uint64_t)(incl >> 64);
                const uint64_t olo = __shfl_up(lo, off, 64), ohi = __shfl_up(hi, off, 64);
                if (tid >= off) incl += (__int128)(((unsigned __int128)ohi << 64) | olo);
            }
            const uint64_t tlo = __shfl((uint64_t)incl, 63, 64);
            const uint64_t thi = __shfl((uint64_t)(incl >> 64), 63, 64);
            const __int128 total = (__int128)(((unsigned __int128)thi << 64) | tlo);
            const __int128 need = (__int128)tau_num * total;
            __int128 cum = incl - part;  // exposed sum of the stages before b
            int k = S + 1;               // "not reached in this lane's part"
            if (b == 0 && (__int128)tau_den * 0 >= need) k = 0;
            for (int i = b; i < e && k > S; ++i) {
                cum += sorted_ex[i];
                if ((__int128)tau_den * cum >= need) k = i + 1;
            }
            for (int off = 32; off > 0; off >>= 1) k = min(k, __shfl_xor(k, off, 64));
            if (tid == 0) size[win] = k > S ? S : k;
        }
        __syncthreads();
    }
}

// ---------------------------------------------------------------------------
// direct-exposure gain, Eq. (4).  Replacing stage s of every rank by
// b = min(d, btilde) changes the last frontier F[t,S] = max_r P[t,r,S] only
// through the rank totals: F^(s<-b)[t,S] = max_r (P[t,r,S] - delta[r,s]) with
// delta = max(0, d - btilde).  Step group layout as in k_frontier; each lane
// keeps its ranks' totals and the deltas of all stages in registers (the
// stage loop is unrolled to SMAX, rows past S re-read row 0 and are
// ignored), then every stage's candidate max and the plain max go through
// the idempotent DPP max, so lane slots past R (which re-read rank r0) need
// no masking.  Partial maxima of several tiles or groups meet in LDS.

template <int VEC, int K, int G, int WG, int SMAX>
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

    __shared__ u64 tab[(WG / SUB) * NCOL];

    const int tid = threadIdx.x;
    const int gl = tid % G;
    const int slot = tid / SUB;
    const bool writer = (tid % SUB) == SUB - 1;
    const int64_t tb = (int64_t)blockIdx.x * SPW;
    const int64_t t = tb + tid / G;

    if (t < T) {
        const int64_t* dt = d + t * (int64_t)S * R;
        const int64_t* bw = btilde + (t / window) * (int64_t)S * R;
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
            fmax = group_max<SUB>(fmax);
            if (writer) {
                u64* p = &tab[slot * NCOL + SMAX];
                *p = (r0 == 0) ? fmax : umax64(*p, fmax);
            }
#pragma unroll
            for (int s = 0; s < SMAX; ++s) {
                if (s < S) {
                    u64 m = 0;
#pragma unroll
                    for (int k = 0; k < K; ++k) m = umax64(m, (u64)(tot[k] - dl[k][s]));
                    m = group_max<SUB>(m);
                    if (writer) {
                        u64* p = &tab[slot * NCOL + s];
                        *p = (r0 == 0) ? m : umax64(*p, m);
                    }
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

struct GainVariant {
    const void* fn;
    int G, WG;
};

template <int VEC, int K, int G, int WG, int SMAX>
GainVariant gain_variant()
{
    return GainVariant{reinterpret_cast<const void*>(&k_exposure_gain<VEC, K, G, WG, SMAX>), G, WG};
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
    return gain_variant<VEC, K, 256, 256, SMAX>();
}

GainVariant pick_gain(int R, int S, bool vec2)
{
    if (S <= 8) return vec2 ? pick_gain_g<2, 2, 8>(R) : pick_gain_g<1, 2, 8>(R);
    if (S <= 16) return vec2 ? pick_gain_g<2, 2, 16>(R) : pick_gain_g<1, 2, 16>(R);
    if (S <= 32) return vec2 ? pick_gain_g<2, 2, 32>(R) : pick_gain_g<1, 2, 32>(R);
    return pick_gain_g<1, 1, 64>(R);
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

// ---------------------------------------------------------------------------
// lag kernel (Sec. 4): L[t,s] = max_r P - median_r P with the lower median
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

// ---------------------------------------------------------------------------
// host helpers

bool disjoint(const void* a, int64_t na, const void* b, int64_t nb)
{
    const uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
    return x + (uintptr_t)na <= y || y + (uintptr_t)nb <= x;
}

bool aligned(const void* p, uintptr_t a) { return ((uintptr_t)p & (a - 1)) == 0; }

// true if n1 * n2 * n3 * bytes fits in int64
bool fits(int64_t n1, int64_t n2, int64_t n3, int64_t bytes)
{
    const int64_t lim = INT64_MAX;
    if (n1 == 0) return true;
    return n1 <= lim / n2 / n3 / bytes;
}

int launch(const void* fn, dim3 grid, dim3 block, void** args, size_t lds, sf_stream_t stream)
{
    const hipError_t e = hipLaunchKernel(fn, grid, block, args, lds, (hipStream_t)stream);
    return e == hipSuccess ? SF_OK : SF_EHIP;
}

}  // namespace

// ---------------------------------------------------------------------------
// C ABI

SF_API int sf_frontier(const int64_t* durations, int64_t T, int32_t R, int32_t S,
                       int64_t* out_increment, int32_t* out_leader, sf_stream_t stream)
{
    if (T < 0 || R < 1 || R > SF_MAX_R || S < 1 || S > SF_MAX_S) return SF_EINVAL;
    if (!fits(T, S, R, 8)) return SF_EINVAL;
    if (T == 0) return SF_OK;
    if (!durations || !out_increment || !out_leader) return SF_EINVAL;
    if (!aligned(durations, 8) || !aligned(out_increment, 8) || !aligned(out_leader, 4))
        return SF_EINVAL;
    const int64_t nd = T * S * (int64_t)R * 8, ni = T * S * 8, nl = T * S * 4;
    if (!disjoint(durations, nd, out_increment, ni) || !disjoint(durations, nd, out_leader, nl) ||
        !disjoint(out_increment, ni, out_leader, nl))
        return SF_EINVAL;

    const bool vec2 = (R % 2 == 0) && aligned(durations, 16);
    const FrontierVariant v = vec2 ? pick_frontier<2>(R) : pick_frontier<1>(R);
    const int spw = v.WG / v.G;
    const int sub = v.G < 64 ? v.G : 64;
    const int64_t blocks = (T + spw - 1) / spw;
    if (blocks > INT32_MAX) return SF_EINVAL;
    const size_t lds = lds_request((size_t)(v.WG / sub) * S * sizeof(u64), v.per_cu);
    int Ri = R, Si = S;
    void* args[] = {(void*)&durations, (void*)&T, (void*)&Ri, (void*)&Si, (void*)&out_increment,
                    (void*)&out_leader};
    return launch(v.fn, dim3((unsigned)blocks), dim3(v.WG), args, lds, stream);
}

SF_API int sf_frontier_evidence(const int64_t* durations, int64_t T, int32_t R, int32_t S,
                                int64_t* out_increment, int32_t* out_leader, int64_t* out_gap,
                                int32_t* out_ties, int64_t* out_stage_max,
                                int64_t* out_stage_sum, sf_stream_t stream)
{
    if (T < 0 || R < 1 || R > SF_MAX_R || S < 1 || S > SF_MAX_S) return SF_EINVAL;
    if (!fits(T, S, R, 8)) return SF_EINVAL;
    if (T == 0) return SF_OK;
    if (T > INT32_MAX) return SF_EINVAL;
    const void* bufs[7] = {durations, out_increment, out_leader, out_gap,
                           out_ties, out_stage_max, out_stage_sum};
    const uintptr_t align[7] = {8, 8, 4, 8, 4, 8, 8};
    const int64_t ts = T * S;
    const int64_t sizes[7] = {ts * R * 8, ts * 8, ts * 4, ts * 8, ts * 4, ts * 8, ts * 8};
    for (int a = 0; a < 7; ++a)
        if (!bufs[a] || !aligned(bufs[a], align[a])) return SF_EINVAL;
    for (int a = 0; a < 7; ++a)
        for (int b = (a < 1 ? 1 : a + 1); b < 7; ++b)
            if (!disjoint(bufs[a], sizes[a], bufs[b], sizes[b])) return SF_EINVAL;

    const bool vec2 = (R % 2 == 0) && aligned(durations, 16);
    const EvidenceVariant v = vec2 ? pick_evidence<2>(R, S) : pick_evidence<1>(R, S);
    const int spw = v.WG / v.G;
    const size_t lds = lds_request(ev_lds_need(v, R, S), v.per_cu);
    const int64_t blocks = (T + spw - 1) / spw;
    int Ri = R, Si = S;
    void* args[] = {(void*)&durations, (void*)&T, (void*)&Ri, (void*)&Si,
                    (void*)&out_increment, (void*)&out_leader, (void*)&out_gap,
                    (void*)&out_ties, (void*)&out_stage_max, (void*)&out_stage_sum};
    return launch(v.fn, dim3((unsigned)blocks), dim3(v.WG), args, lds, stream);
}

SF_API int sf_ingest(const int64_t* stages, const int64_t* wall, int64_t T, int32_t R,
                     int32_t K, int64_t* out_durations, int64_t* out_overlap,
                     sf_stream_t stream)
{
    if (T < 0 || R < 1 || R > SF_MAX_R || K < 0 || K + 1 > SF_MAX_S) return SF_EINVAL;
    if (!fits(T, K + 2, R, 8)) return SF_EINVAL;
    if (T == 0) return SF_OK;
    const int64_t S = K + 1;
    const void* bufs[4] = {stages, wall, out_durations, out_overlap};
    const int64_t sizes[4] = {(int64_t)R * T * K * 8, (int64_t)R * T * 8, T * S * (int64_t)R * 8,
                              T * (int64_t)R * 8};
    for (int a = 0; a < 4; ++a)
        if ((!bufs[a] && sizes[a] > 0) || !aligned(bufs[a], 8)) return SF_EINVAL;
    for (int a = 0; a < 4; ++a)
        for (int b = (a < 2 ? 2 : a + 1); b < 4; ++b)
            if (sizes[a] > 0 && sizes[b] > 0 && !disjoint(bufs[a], sizes[a], bufs[b], sizes[b]))
                return SF_EINVAL;
    const IngestTile g = pick_ingest(K, T);
    const int64_t nblk = ((R + g.RB - 1) / g.RB) * ((T + g.TB - 1) / g.TB);
    const unsigned grid = (unsigned)(nblk < (1 << 20) ? nblk : (1 << 20));
    int Ri = R, Ki = K, TB = g.TB, segp = g.segp;
    void* args[] = {(void*)&stages, (void*)&wall, (void*)&T, (void*)&Ri, (void*)&Ki,
                    (void*)&TB, (void*)&segp, (void*)&out_durations, (void*)&out_overlap};
    return launch(g.fn, dim3(grid), dim3(kIngestWG), args, g.lds, stream);
}

SF_API int sf_route(const int64_t* stage_exposed, int64_t W, int32_t S, int64_t tau_num,
                    int64_t tau_den, int32_t* out_order, int32_t* out_size, sf_stream_t stream)
{
    if (W < 0 || S < 1 || S > SF_MAX_S || tau_den < 1 || tau_num < 0 || tau_num > tau_den ||
        tau_den > INT32_MAX)
        return SF_EINVAL;
    if (!fits(W, S, 1, 8)) return SF_EINVAL;
    if (W == 0) return SF_OK;
    if (!stage_exposed || !out_order || !out_size) return SF_EINVAL;
    if (!aligned(stage_exposed, 8) || !aligned(out_order, 4) || !aligned(out_size, 4))
        return SF_EINVAL;
    const int64_t ne = W * S * 8, no = W * S * 4, ns = W * 4;
    if (!disjoint(stage_exposed, ne, out_order, no) || !disjoint(stage_exposed, ne, out_size, ns) ||
        !disjoint(out_order, no, out_size, ns))
        return SF_EINVAL;
    const unsigned grid = (unsigned)(W < 65536 ? W : 65536);
    int Si = S;
    void* args[] = {(void*)&stage_exposed, (void*)&W, (void*)&Si, (void*)&tau_num, (void*)&tau_den,
                    (void*)&out_order, (void*)&out_size};
    return launch(reinterpret_cast<const void*>(&k_route), dim3(grid), dim3(kRouteWG), args, 0,
                  stream);
}

SF_API int sf_exposure_gain(const int64_t* durations, const int64_t* baseline, int64_t T,
                            int32_t R, int32_t S, int64_t window, int64_t* out_gain,
                            int64_t* out_makespan, int64_t* out_window_gain,
                            int64_t* out_window_makespan, sf_stream_t stream)
{
    if (T < 0 || R < 1 || R > SF_MAX_R || S < 1 || S > SF_MAX_S_GAIN || window < 1)
        return SF_EINVAL;
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
    const GainVariant v = pick_gain(R, S, vec2);
    const int spw = v.WG / v.G;
    const int64_t blocks = (T + spw - 1) / spw;
    if (blocks > INT32_MAX) return SF_EINVAL;
    int Ri = R, Si = S;
    void* a1[] = {(void*)&durations, (void*)&baseline, (void*)&T, (void*)&Ri, (void*)&Si,
                  (void*)&window, (void*)&out_gain, (void*)&out_makespan};
    int rc = launch(v.fn, dim3((unsigned)blocks), dim3(v.WG), a1, 0, stream);
    if (rc != SF_OK) return rc;
    int64_t Wl = W;
    const int64_t items = W * S;
    void* a2[] = {(void*)&out_gain, (void*)&T, (void*)&Si, (void*)&window, (void*)&Wl,
                  (void*)&out_window_gain};
    rc = launch(reinterpret_cast<const void*>(&k_window_sum),
                dim3((unsigned)(items < 1048576 ? items : 1048576)), dim3(kSumWG), a2, 0, stream);
    if (rc != SF_OK) return rc;
    int one = 1;
    void* a3[] = {(void*)&out_makespan, (void*)&T, (void*)&one, (void*)&window, (void*)&Wl,
                  (void*)&out_window_makespan};
    return launch(reinterpret_cast<const void*>(&k_window_sum),
                  dim3((unsigned)(W < 1048576 ? W : 1048576)), dim3(kSumWG), a3, 0, stream);
}

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

SF_API int64_t sf_num_windows(int64_t T, int64_t window)
{
    if (T < 0 || window < 1) return -1;
    return T / window + (T % window != 0);
}

SF_API int sf_window_summary(const int64_t* increment, const int32_t* leader, int64_t T,
                             int32_t R, int32_t S, int64_t window, int64_t* out_stage_exposed,
                             int32_t* out_lead_counts, int32_t* out_top2, sf_stream_t stream)
{
    if (T < 0 || R < 1 || R > SF_MAX_R || S < 1 || S > SF_MAX_S || window < 1) return SF_EINVAL;
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

SF_API const char* sf_strerror(int status)
{
    switch (status) {
    case SF_OK: return "success";
    case SF_EINVAL: return "invalid argument";
    case SF_ERANGE: return "value out of range";
    case SF_EHIP: return "HIP kernel launch failed";
    default: return "unknown status";
    }
}

SF_API const char* sf_version(void) { return "libstagefrontier 0.1.0 (gfx950)"; }
