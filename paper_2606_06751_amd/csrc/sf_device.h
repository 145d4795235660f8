// sf_device.h -- device-side building blocks shared by the libstagefrontier
// kernels (gfx950, wave64): the packed (prefix, rank) key, DPP lane moves and
// the wave reductions built on them.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sfk {

typedef unsigned long long u64;
typedef long long v2i64 __attribute__((ext_vector_type(2)));

constexpr int kRankBits = 16;
constexpr u64 kRankMask = 0xFFFFull;

__device__ __forceinline__ u64 umax64(u64 a, u64 b) { return a > b ? a : b; }

// Workgroups are dispatched round-robin over the 8 XCDs of the chip, each
// with its own L2.  xcd_block() renumbers them so that each XCD takes one
// contiguous run of block indices: output rows of neighbouring steps, which
// share cache lines, are then written from one L2 instead of two (measured
// on MI355X: 1-3% faster frontier passes at 128-4096 ranks).  A bijection
// on [0, gridDim.x) for any grid size.
__device__ __forceinline__ int64_t xcd_block()
{
    const int64_t n = gridDim.x, b = blockIdx.x;
    const int64_t x = b & 7, i = b >> 3;
    const int64_t per = n >> 3, extra = n & 7;
    return x * per + (x < extra ? x : extra) + i;
}

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

__device__ __forceinline__ u64 umin64(u64 a, u64 b) { return a < b ? a : b; }

// A workgroup barrier that orders LDS accesses only: waves wait for their
// own LDS operations, not for their global loads in flight, so a load issued
// before it (the next stage's rows) keeps flying across it.  __syncthreads()
// would wait for those loads too.  Not for communication through global
// memory.
__device__ __forceinline__ void lds_barrier()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// A raw buffer resource over `bytes` bytes at `base` (gfx950 word 3: raw,
// 32-bit untyped), so that loads take the base from SGPRs, a lane's byte
// offset from one VGPR and a wave-uniform byte offset from an SGPR.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void* base, uint32_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, (int)bytes, 0x00020000);
}

// 16 bytes at base + voff + soff, non-temporal (aux bit 1)
__device__ __forceinline__ v2i64 buffer_load16_nt(__amdgpu_buffer_rsrc_t rs, uint32_t voff, uint32_t soff)
{
    return __builtin_bit_cast(v2i64, __builtin_amdgcn_raw_buffer_load_b128(rs, (int)voff, (int)soff, 2));
}

constexpr int kSumWG = 256;  // threads of the window reduction kernels

__device__ __forceinline__ int64_t wave_sum64(int64_t v)
{
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
    return v;
}

}  // namespace sfk
