// route.hip -- routing-set kernel (Sec. 4): per window, stages by exposed total
// (descending, lower stage first) and the smallest leading prefix whose
// exposed sum reaches tau_num / tau_den of the window total, compared
// exactly in 128-bit integers.  One workgroup per window.

#include "sf_device.h"
#include "sf_host.h"

namespace sfk {

constexpr int kRouteWG = 256;
constexpr int kRouteLdsS = 4096;  // stages staged in LDS (two rows of 8-byte totals, 64 KB)

// LDS: the window's totals and their sorted copy are staged in LDS (S <=
// kRouteLdsS); otherwise they are read from global memory, the sorted copy
// through the order just written.
template <bool LDS>
__global__ __launch_bounds__(kRouteWG) void k_route(const int64_t* __restrict__ exposed,
                                                    int64_t W, int S, int64_t tau_num,
                                                    int64_t tau_den, int32_t* __restrict__ order,
                                                    int32_t* __restrict__ size)
{
    extern __shared__ int64_t rsh[];  // LDS: [2][S]
    const int tid = threadIdx.x;
    for (int64_t win = blockIdx.x; win < W; win += gridDim.x) {
        const int64_t* exg = exposed + win * S;
        int32_t* ord = order + win * S;
        if (LDS) {
            for (int s = tid; s < S; s += kRouteWG) rsh[s] = exg[s];
            __syncthreads();
        }
        const int64_t* ex = LDS ? rsh : exg;
        // position of stage s = number of stages that come before it
        for (int s = tid; s < S; s += kRouteWG) {
            const int64_t e = ex[s];
            int pos = 0;
            for (int u = 0; u < S; ++u) pos += (ex[u] > e || (ex[u] == e && u < s)) ? 1 : 0;
            ord[pos] = s;
            if (LDS) rsh[S + pos] = e;
        }
        __syncthreads();
        auto sorted_ex = [&](int i) { return LDS ? rsh[S + i] : exg[ord[i]]; };
        // wave 0 scans the sorted totals: each lane sums a contiguous part,
        // an exclusive scan over lanes gives each part's starting sum, and
        // each lane finds the first prefix in its part that reaches tau
        if (tid < 64) {
            const int per = (S + 63) / 64;
            const int b = tid * per;
            const int e = min(S, b + per);
            __int128 part = 0;
            for (int i = b; i < e; ++i) part += sorted_ex(i);
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
                cum += sorted_ex(i);
                if ((__int128)tau_den * cum >= need) k = i + 1;
            }
            for (int off = 32; off > 0; off >>= 1) k = min(k, __shfl_xor(k, off, 64));
            if (tid == 0) size[win] = k > S ? S : k;
        }
        __syncthreads();
    }
}

}  // namespace sfk

using namespace sfk;

SF_API int sf_route(const int64_t* stage_exposed, int64_t W, int32_t S, int64_t tau_num,
                    int64_t tau_den, int32_t* out_order, int32_t* out_size, sf_stream_t stream)
{
    if (W < 0 || S < 1 || tau_den < 1 || tau_num < 0 || tau_num > tau_den ||
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
    if (S <= kRouteLdsS)
        return launch(reinterpret_cast<const void*>(&k_route<true>), dim3(grid), dim3(kRouteWG),
                      args, (size_t)2 * S * sizeof(int64_t), stream);
    return launch(reinterpret_cast<const void*>(&k_route<false>), dim3(grid), dim3(kRouteWG), args,
                  0, stream);
}
