// route.hip -- routing-set kernel (Sec. 4): per window, stages by exposed total
// (descending, lower stage first) and the smallest leading prefix whose
// exposed sum reaches tau_num / tau_den of the window total, compared
// exactly in 128-bit integers.  One workgroup per window.

#include "sf_device.h"
#include "sf_host.h"

namespace sfk {

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

}  // namespace sfk

using namespace sfk;

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
