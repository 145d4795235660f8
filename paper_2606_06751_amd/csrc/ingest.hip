// ingest.hip -- ingest kernel: gathered per-rank buffers -> [T][S][R] with the Appendix A
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

#include "sf_device.h"
#include "sf_host.h"

namespace sfk {

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
        // write: each wave writes ROWS_PER_WAVE [t][s] rows of RB ranks at
        // once, with non-temporal stores (the output is written once and not
        // read again here: measured 2-6% faster than plain stores on the
        // four large workloads; non-temporal loads of the input, read
        // through L2 in 512-byte pieces, measured 8-29% slower)
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
                if (dst[u]) __builtin_nontemporal_store(v[u], dst[u]);
        }
        for (int i = tid; i < tn * RB; i += kIngestWG) {
            const int tl = i / RB;
            const int jj = i & (RB - 1);
            if (jj < rn) __builtin_nontemporal_store(ovl[i], &o[(t0 + tl) * (int64_t)R + r0 + jj]);
        }
        __syncthreads();  // the tile is reused by the next block
    }
}

// More explicit stages than a rank's segment of one step fits in LDS
// (K + 1 > kIngestTiledS): one thread per (step, rank), walking the rank's
// K contiguous values of the step, writing each to its [t][s] row (the
// threads of a wave cover 64 adjacent ranks, so every store is coalesced)
// and summing them for the closure.  Each lane's reads run along its own
// row, so the cache lines of a row are fetched once and used for the next
// values.
constexpr int kIngestTiledS = 512;

__global__ __launch_bounds__(kIngestWG) void k_ingest_wide(const int64_t* __restrict__ x,
                                                           const int64_t* __restrict__ w,
                                                           int64_t T, int R, int K,
                                                           int64_t* __restrict__ d,
                                                           int64_t* __restrict__ o)
{
    const int64_t nrc = (R + kIngestWG - 1) / kIngestWG;
    const int64_t S = (int64_t)K + 1;
    for (int64_t blk = blockIdx.x; blk < nrc * T; blk += gridDim.x) {
        const int64_t t = blk / nrc;
        const int r = (int)(blk - t * nrc) * kIngestWG + (int)threadIdx.x;
        if (r >= R) continue;
        const int64_t* src = x + ((int64_t)r * T + t) * K;
        int64_t* dst = d + t * S * R + r;
        int64_t sum = 0;
        for (int k = 0; k < K; ++k) {
            const int64_t v = src[k];
            __builtin_nontemporal_store(v, dst + (int64_t)k * R);
            sum += v;
        }
        const int64_t e = w[(int64_t)r * T + t] - sum;
        __builtin_nontemporal_store(e > 0 ? e : (int64_t)0, dst + (int64_t)K * R);
        __builtin_nontemporal_store(e < 0 ? -e : (int64_t)0, &o[t * R + r]);
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

}  // namespace sfk

using namespace sfk;

SF_API int sf_ingest(const int64_t* stages, const int64_t* wall, int64_t T, int32_t R,
                     int32_t K, int64_t* out_durations, int64_t* out_overlap,
                     sf_stream_t stream)
{
    if (T < 0 || R < 1 || R > SF_MAX_R || K < 0 || K > INT32_MAX - 2) return SF_EINVAL;
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
    if (S > kIngestTiledS) {
        const int64_t nblk = ((R + kIngestWG - 1) / kIngestWG) * T;
        const unsigned grid = (unsigned)(nblk < (1 << 20) ? nblk : (1 << 20));
        int Ri = R, Ki = K;
        void* args[] = {(void*)&stages, (void*)&wall,          (void*)&T,          (void*)&Ri,
                        (void*)&Ki,     (void*)&out_durations, (void*)&out_overlap};
        return launch(reinterpret_cast<const void*>(&k_ingest_wide), dim3(grid), dim3(kIngestWG),
                      args, 0, stream);
    }
    const IngestTile g = pick_ingest(K, T);
    const int64_t nblk = ((R + g.RB - 1) / g.RB) * ((T + g.TB - 1) / g.TB);
    const unsigned grid = (unsigned)(nblk < (1 << 20) ? nblk : (1 << 20));
    int Ri = R, Ki = K, TB = g.TB, segp = g.segp;
    void* args[] = {(void*)&stages, (void*)&wall, (void*)&T, (void*)&Ri, (void*)&Ki,
                    (void*)&TB, (void*)&segp, (void*)&out_durations, (void*)&out_overlap};
    return launch(g.fn, dim3(grid), dim3(kIngestWG), args, g.lds, stream);
}
