// frontier.hip -- sf_frontier: per-step frontier advances and leaders
// (Sec. 3, Eq. (1)) on gfx950.
//
// Data layout in HBM: durations [T][S][R] int64 (rank fastest), outputs
// [T][S].
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
// Stage counts beyond what LDS holds (the gradient-accumulation expansion of
// Sec. 3 multiplies S by the number of micro-steps) take the GTAB variant:
// one group of at most 64 lanes owns a step, and its last lane keeps the
// step's per-stage partial maxima in the step's own out_increment row (the
// caller's output, so no extra memory); after the last tile the workgroup
// decodes those rows in place, chunk by chunk from the end, each chunk read
// before any of it is written.
//
// The checked variant also verifies the data contract on the way: every
// duration in [0, 2^47) (its high word below 2^15) and every prefix below
// 2^47 (the top bit of every key clear: while all durations are below 2^47
// a prefix that first reaches 2^47 is still below 2^48, so its key's top bit
// is set at that stage).  A wave that sees a violation ORs SF_ERANGE into the
// caller's status word.
//

#include "sf_device.h"
#include "sf_host.h"

namespace sfk {

// VEC: int64 elements per load (2: 16-byte loads, needs even R and a 16-byte
//      aligned base); K: ranks per lane per tile; G: lanes per step;
// WG:  threads per workgroup (WG / G steps per workgroup); CHECK: verify the
//      data contract into *status; GTAB: partial maxima in the out_increment
//      rows instead of LDS (any S; G <= 64).
template <int VEC, int K, int G, int WG, bool CHECK, bool GTAB>
__global__ __launch_bounds__(WG) void k_frontier(const int64_t* __restrict__ d, int64_t T,
                                                 int R, int S, int64_t* __restrict__ inc,
                                                 int32_t* __restrict__ lead,
                                                 uint32_t* __restrict__ status)
{
    static_assert(K % VEC == 0, "K must be a multiple of VEC");
    static_assert(WG % G == 0 || G == WG, "a workgroup holds whole steps");
    static_assert(!GTAB || G <= 64, "GTAB: one writer lane per step");
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
    const int64_t lb = xcd_block();  // XCD-contiguous step runs
    const int64_t t = lb * SPW + j;
    uint32_t dhi = 0, khi = 0;  // CHECK: OR of the durations' and the keys' high words

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
                    if (CHECK) dhi |= (uint32_t)((u64)v[k] >> 32);
                }
                if (CHECK) khi |= (uint32_t)(m >> 32);
                if (s + 1 < S) load_row(s + 1);
                m = group_max<SUB>(m);
                if (writer) {
                    // GTAB: the step's own out_increment row, read back by
                    // the same lane only until the decode below
                    u64* p = GTAB ? reinterpret_cast<u64*>(inc) + t * S + s : &tab[slot * S + s];
                    *p = (r0 == 0) ? m : umax64(*p, m);
                }
            }
        }
    }
    if (CHECK) {
        const u64 bad = __ballot((dhi >> 15) != 0 || (khi >> 31) != 0);
        if (bad != 0 && (tid & 63) == __builtin_ctzll(bad)) atomicOr(status, (uint32_t)SF_ERANGE);
    }
    __syncthreads();

    const int64_t tb = lb * SPW;
    if constexpr (GTAB) {
        // the workgroup's steps are contiguous rows of out_increment holding
        // keys: decode them in place in chunks of WG entries, the last chunk
        // first.  A chunk reads its keys and the key before each (which lies
        // in the same chunk or the one below, not yet decoded), waits for
        // every thread's reads, then writes.
        const int64_t steps = T - tb < SPW ? T - tb : SPW;
        const int64_t n = steps * S;
        u64* g = reinterpret_cast<u64*>(inc) + tb * S;
        for (int64_t c = (n - 1) / WG; c >= 0; --c) {
            const int64_t i = c * WG + tid;
            const bool ok = i < n;
            u64 key = 0, kprev = 0;
            if (ok) {
                key = g[i];
                if (i % S != 0) kprev = g[i - 1];
            }
            __syncthreads();
            if (ok) {
                inc[tb * S + i] = (int64_t)(key >> kRankBits) - (int64_t)(kprev >> kRankBits);
                lead[tb * S + i] = (int32_t)(kRankMask - (key & kRankMask));
            }
        }
        return;
    }

    // decode F and the leader per (step, stage); rows of out are contiguous
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

template <int VEC, bool CHECK, int K, int G, int WG, bool GTAB = false>
FrontierVariant variant(int per_cu)
{
    return FrontierVariant{reinterpret_cast<const void*>(&k_frontier<VEC, K, G, WG, CHECK, GTAB>),
                           K, G, WG, per_cu};
}

// Launch shape by rank count, measured on MI355X over R = 16 .. 16384.
// Wide per-lane tiles (K = 32 ranks, about 250 VGPRs) and few resident
// workgroups per CU read HBM fastest for large R: fewer concurrent step
// streams, each with up to 32 KB of loads in flight per wave.  A tile wider
// than R costs no HBM traffic (lane slots past R re-read a cached rank).
template <int VEC, bool CHECK>
FrontierVariant pick_frontier(int R)
{
    if (R <= 8) return variant<VEC, CHECK, 2, 4, 64>(0);
    if (R <= 16) return variant<VEC, CHECK, 2, 8, 128>(0);
    if (R <= 32) return variant<VEC, CHECK, 4, 8, 128>(0);
    if (R <= 64) return variant<VEC, CHECK, 4, 16, 256>(6);
    if (R <= 128) return variant<VEC, CHECK, 8, 32, 256>(6);
    if (R <= 256) return variant<VEC, CHECK, 16, 32, 256>(4);
    if (R <= 512) return variant<VEC, CHECK, 4, 256, 256>(0);
    if (R <= 1024) return variant<VEC, CHECK, 32, 64, 256>(6);
    if (R <= 2048) return variant<VEC, CHECK, 8, 512, 512>(0);
    if (R <= 4096) return variant<VEC, CHECK, 32, 256, 256>(0);
    return variant<VEC, CHECK, 32, 64, 64>(3);
}

// Stage counts whose LDS table would exceed what a workgroup may hold: the
// shapes with one group of at most 64 lanes per step, with the table in the
// out_increment rows.
template <int VEC, bool CHECK>
FrontierVariant pick_frontier_gtab(int R)
{
    if (R <= 8) return variant<VEC, CHECK, 2, 4, 64, true>(0);
    if (R <= 16) return variant<VEC, CHECK, 2, 8, 128, true>(0);
    if (R <= 32) return variant<VEC, CHECK, 4, 8, 128, true>(0);
    if (R <= 64) return variant<VEC, CHECK, 4, 16, 256, true>(6);
    if (R <= 128) return variant<VEC, CHECK, 8, 32, 256, true>(6);
    if (R <= 256) return variant<VEC, CHECK, 16, 32, 256, true>(4);
    return variant<VEC, CHECK, 32, 64, 64, true>(3);
}

// Largest S whose LDS table of partial maxima (16 slots of S keys in the
// widest-slot shapes) fits the 64 KB a workgroup is given.
constexpr int kFrontierLdsS = 512;

static int frontier_launch(const int64_t* durations, int64_t T, int32_t R, int32_t S,
                           int64_t* out_increment, int32_t* out_leader, uint32_t* status,
                           sf_stream_t stream)
{
    if (T < 0 || R < 1 || R > SF_MAX_R || S < 1) return SF_EINVAL;
    if (!fits(T, S, R, 8)) return SF_EINVAL;
    if (T == 0) return SF_OK;
    if (!durations || !out_increment || !out_leader) return SF_EINVAL;
    if (!aligned(durations, 8) || !aligned(out_increment, 8) || !aligned(out_leader, 4))
        return SF_EINVAL;
    const int64_t nd = T * S * (int64_t)R * 8, ni = T * S * 8, nl = T * S * 4;
    if (!disjoint(durations, nd, out_increment, ni) || !disjoint(durations, nd, out_leader, nl) ||
        !disjoint(out_increment, ni, out_leader, nl))
        return SF_EINVAL;
    if (status && (!aligned(status, 4) || !disjoint(status, 4, durations, nd) ||
                   !disjoint(status, 4, out_increment, ni) || !disjoint(status, 4, out_leader, nl)))
        return SF_EINVAL;

    const bool vec2 = (R % 2 == 0) && aligned(durations, 16);
    const bool gtab = S > kFrontierLdsS;
    FrontierVariant v;
    if (gtab)
        v = status ? (vec2 ? pick_frontier_gtab<2, true>(R) : pick_frontier_gtab<1, true>(R))
                   : (vec2 ? pick_frontier_gtab<2, false>(R) : pick_frontier_gtab<1, false>(R));
    else
        v = status ? (vec2 ? pick_frontier<2, true>(R) : pick_frontier<1, true>(R))
                   : (vec2 ? pick_frontier<2, false>(R) : pick_frontier<1, false>(R));
    const int spw = v.WG / v.G;
    const int sub = v.G < 64 ? v.G : 64;
    const int64_t blocks = (T + spw - 1) / spw;
    if (blocks > INT32_MAX) return SF_EINVAL;
    const size_t lds = lds_request(gtab ? 0 : (size_t)(v.WG / sub) * S * sizeof(u64), v.per_cu);
    int Ri = R, Si = S;
    void* args[] = {(void*)&durations,     (void*)&T,          (void*)&Ri,    (void*)&Si,
                    (void*)&out_increment, (void*)&out_leader, (void*)&status};
    return launch(v.fn, dim3((unsigned)blocks), dim3(v.WG), args, lds, stream);
}

}  // namespace sfk

using namespace sfk;

SF_API int sf_frontier(const int64_t* durations, int64_t T, int32_t R, int32_t S,
                       int64_t* out_increment, int32_t* out_leader, sf_stream_t stream)
{
    return frontier_launch(durations, T, R, S, out_increment, out_leader, nullptr, stream);
}

SF_API int sf_frontier_checked(const int64_t* durations, int64_t T, int32_t R, int32_t S,
                               int64_t* out_increment, int32_t* out_leader, uint32_t* status,
                               sf_stream_t stream)
{
    if (!status) return SF_EINVAL;
    return frontier_launch(durations, T, R, S, out_increment, out_leader, status, stream);
}
