// calib.hip -- plain-read calibration: the XOR of the 64-bit words of every
// 256 KB piece of a device buffer.  It reads each byte once with the same
// 16-byte non-temporal loads as the frontier pass and does no other work,
// so its rate is the device's practical read ceiling, the yardstick for the
// HBM-bound kernels (the frontier pass reads its input exactly once).
//
// One workgroup of 256 threads per piece, 16 loads in flight per thread.
// Measured on MI355X over a 15.7 GB buffer: reads that write nothing reach
// 7.2-7.3 TB/s with 32 KB-256 KB contiguous pieces per workgroup; one word
// written per piece costs 4% at 64 KB pieces, 1% at 256 KB (scattered 8-byte
// stores interrupt the read stream).  A persistent grid striding over the
// pieces read at 5.6-6.8 TB/s, and folding the pieces into one word with
// device-scope atomics on one address costs about 10 ns per atomic,
// serialised.  Hence one result word per 256 KB piece, which the caller
// folds if it wants one.

#include "sf_device.h"
#include "sf_host.h"

namespace sfk {

typedef u64 v2u64 __attribute__((ext_vector_type(2)));

constexpr int kCalWG = 256;
constexpr int kCalU = 16;
constexpr int64_t kCalVec = SF_XOR_PIECE_BYTES / 16;  // 16-byte vectors per piece
static_assert(SF_XOR_PIECE_BYTES % (16 * kCalWG * kCalU) == 0, "piece = whole load rounds");

__global__ __launch_bounds__(kCalWG) void k_read_xor(const v2u64* __restrict__ p, int64_t nvec,
                                                     const u64* __restrict__ tail,
                                                     u64* __restrict__ out)
{
    __shared__ u64 part[kCalWG / 64];
    const int64_t b0 = (int64_t)blockIdx.x * kCalVec;
    const int64_t e = b0 + kCalVec < nvec ? b0 + kCalVec : nvec;
    u64 acc = 0;
    int64_t i = b0 + threadIdx.x;
    for (; i + (kCalU - 1) * kCalWG < e; i += kCalU * kCalWG) {
        v2u64 x[kCalU];
#pragma unroll
        for (int u = 0; u < kCalU; ++u) x[u] = __builtin_nontemporal_load(p + i + u * kCalWG);
#pragma unroll
        for (int u = 0; u < kCalU; ++u) acc ^= x[u].x ^ x[u].y;
    }
    for (; i < e; i += kCalWG) {
        const v2u64 x = __builtin_nontemporal_load(p + i);
        acc ^= x.x ^ x.y;
    }
    // a lone last word (odd word count) belongs to the last piece
    if (tail && blockIdx.x == gridDim.x - 1 && threadIdx.x == 0) acc ^= *tail;
    for (int off = 32; off > 0; off >>= 1) acc ^= __shfl_xor(acc, off, 64);
    if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = acc;
    __syncthreads();
    if (threadIdx.x == 0) {
        u64 v = 0;
#pragma unroll
        for (int w = 0; w < kCalWG / 64; ++w) v ^= part[w];
        out[blockIdx.x] = v;
    }
}

}  // namespace sfk

using namespace sfk;

SF_API int64_t sf_read_xor_pieces(int64_t bytes)
{
    if (bytes < 0) return -1;
    return (bytes + SF_XOR_PIECE_BYTES - 1) / SF_XOR_PIECE_BYTES;
}

SF_API int sf_read_xor(const void* buf, int64_t bytes, uint64_t* out_xor, sf_stream_t stream)
{
    if (bytes < 0 || bytes % 8 != 0) return SF_EINVAL;
    if (bytes == 0) return SF_OK;
    if (!buf || !aligned(buf, 16) || !out_xor || !aligned(out_xor, 8)) return SF_EINVAL;
    const int64_t pieces = sf_read_xor_pieces(bytes);
    if (pieces > INT32_MAX || !disjoint(buf, bytes, out_xor, pieces * 8)) return SF_EINVAL;
    const int64_t nvec = bytes / 16;
    const u64* tail = (bytes % 16) ? reinterpret_cast<const u64*>(buf) + 2 * nvec : nullptr;
    const v2u64* p = reinterpret_cast<const v2u64*>(buf);
    u64* out = reinterpret_cast<u64*>(out_xor);
    void* args[] = {(void*)&p, (void*)&nvec, (void*)&tail, (void*)&out};
    return launch(reinterpret_cast<const void*>(&k_read_xor), dim3((unsigned)pieces),
                  dim3(kCalWG), args, 0, stream);
}
