// evidence.hip -- evidence kernel: the frontier pass plus, per boundary, the runner-up gap and
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

#include "sf_device.h"
#include "sf_host.h"

namespace sfk {

struct EvAcc {
    u64 k1, k2;      // largest and second-largest packed key
    int64_t smax;    // max of d over ranks
    int64_t ssum;    // sum of d over ranks
    uint32_t c;      // ranks whose prefix equals that of k1
};

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
// GTAB (stage counts past what LDS holds; G <= 64): the group's last lane
// keeps the partial results of its step in the step's own output rows (the
// largest key in out_increment, the runner-up key in out_gap, the tie count,
// max and sum in their final rows), and after the last tile the workgroup
// decodes the increment, leader and gap in place, chunk by chunk from the
// end, each chunk read before any of it is written.
template <int VEC, int K, int G, int WG, bool GTAB>
__global__ __launch_bounds__(WG) void k_frontier_evidence(
    const int64_t* __restrict__ d, int64_t T, int R, int S, int64_t* __restrict__ inc,
    int32_t* __restrict__ lead, int64_t* __restrict__ gap, int32_t* __restrict__ ties,
    int64_t* __restrict__ stage_max, int64_t* __restrict__ stage_sum)
{
    static_assert(K % VEC == 0 && (WG % G == 0 || G == WG), "shape");
    static_assert(!GTAB || G <= 64, "GTAB: one writer lane per step");
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
    const int64_t tb = xcd_block() * SPW;
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
                    } else if (GTAB) {
                        // the step's own output rows, read back by this lane
                        // only until the decode below
                        const int64_t i = t * S + s;
                        if (r0 > 0) {
                            EvAcc b;
                            b.k1 = (u64)inc[i];
                            b.k2 = (u64)gap[i];
                            b.c = (uint32_t)ties[i];
                            b.smax = stage_max[i];
                            b.ssum = stage_sum[i];
                            ev_merge(a, b);
                        }
                        inc[i] = (int64_t)a.k1;
                        gap[i] = (int64_t)a.k2;
                        ties[i] = (int32_t)a.c;
                        stage_max[i] = a.smax;
                        stage_sum[i] = a.ssum;
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

    if constexpr (GTAB) {
        // the workgroup's steps are contiguous rows; a chunk of WG entries
        // reads its keys and the key before each (in the same chunk or the
        // one below, not yet decoded), waits for every thread's reads, then
        // writes.  The tie count, max and sum are final already.
        const int64_t steps = T - tb < SPW ? T - tb : SPW;
        const int64_t n = steps * S;
        const int64_t base = tb * S;
        for (int64_t c = (n - 1) / WG; c >= 0; --c) {
            const int64_t i = c * WG + tid;
            const bool ok = i < n;
            u64 key = 0, kprev = 0, key2 = 0;
            if (ok) {
                key = (u64)inc[base + i];
                key2 = (u64)gap[base + i];
                if (i % S != 0) kprev = (u64)inc[base + i - 1];
            }
            __syncthreads();
            if (ok) {
                const int64_t F = (int64_t)(key >> kRankBits);
                inc[base + i] = F - (int64_t)(kprev >> kRankBits);
                lead[base + i] = (int32_t)(kRankMask - (key & kRankMask));
                gap[base + i] = R > 1 ? F - (int64_t)(key2 >> kRankBits) : -1;
            }
        }
        return;
    }

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

template <int VEC, int K, int G, int WG, bool GTAB = false>
EvidenceVariant ev_variant(int per_cu)
{
    return EvidenceVariant{reinterpret_cast<const void*>(&k_frontier_evidence<VEC, K, G, WG, GTAB>),
                           K, G, WG, per_cu};
}

// LDS bytes a variant needs: none when one group of <= 64 lanes covers the
// step's ranks or the partial results live in the output rows, else 5
// arrays of [WG / min(G, 64)][S] u64.
size_t ev_lds_need(const EvidenceVariant& v, int R, int S, bool gtab)
{
    const int sub = v.G < 64 ? v.G : 64;
    if (gtab || (v.G <= 64 && R <= v.G * v.K)) return 0;
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
    if (ev_lds_need(v, R, S, false) > kLdsMaxPerWg) v = ev_variant<VEC, 16, 128, 128>(0);
    return v;
}

// Stage counts whose LDS table would not fit even the two-slot fallback
// (more than 819 stages): one group of at most 64 lanes per step, the
// partial results in the output rows.
template <int VEC>
EvidenceVariant pick_evidence_gtab(int R)
{
    if (R <= 8) return ev_variant<VEC, 2, 4, 64, true>(0);
    if (R <= 16) return ev_variant<VEC, 2, 8, 64, true>(0);
    if (R <= 32) return ev_variant<VEC, 4, 8, 64, true>(0);
    if (R <= 64) return ev_variant<VEC, 4, 16, 64, true>(0);
    if (R <= 512) return ev_variant<VEC, 16, 32, 64, true>(0);
    return ev_variant<VEC, 16, 64, 64, true>(0);
}

}  // namespace sfk

using namespace sfk;

SF_API int sf_frontier_evidence(const int64_t* durations, int64_t T, int32_t R, int32_t S,
                                int64_t* out_increment, int32_t* out_leader, int64_t* out_gap,
                                int32_t* out_ties, int64_t* out_stage_max,
                                int64_t* out_stage_sum, sf_stream_t stream)
{
    if (T < 0 || R < 1 || R > SF_MAX_R || S < 1) return SF_EINVAL;
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
    EvidenceVariant v = vec2 ? pick_evidence<2>(R, S) : pick_evidence<1>(R, S);
    const bool gtab = ev_lds_need(v, R, S, false) > kLdsMaxPerWg;
    if (gtab) v = vec2 ? pick_evidence_gtab<2>(R) : pick_evidence_gtab<1>(R);
    const int spw = v.WG / v.G;
    const size_t lds = lds_request(ev_lds_need(v, R, S, gtab), v.per_cu);
    const int64_t blocks = (T + spw - 1) / spw;
    int Ri = R, Si = S;
    void* args[] = {(void*)&durations, (void*)&T, (void*)&Ri, (void*)&Si,
                    (void*)&out_increment, (void*)&out_leader, (void*)&out_gap,
                    (void*)&out_ties, (void*)&out_stage_max, (void*)&out_stage_sum};
    return launch(v.fn, dim3((unsigned)blocks), dim3(v.WG), args, lds, stream);
}
