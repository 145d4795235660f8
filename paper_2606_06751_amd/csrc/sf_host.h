// sf_host.h -- host-side helpers shared by the libstagefrontier entry points:
// argument checks, kernel launch, LDS sizing.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "stagefrontier.h"

#define SF_API extern "C" __attribute__((visibility("default")))

namespace sfk {

static inline bool disjoint(const void* a, int64_t na, const void* b, int64_t nb)
{
    const uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
    return x + (uintptr_t)na <= y || y + (uintptr_t)nb <= x;
}

static inline bool aligned(const void* p, uintptr_t a) { return ((uintptr_t)p & (a - 1)) == 0; }

// true if n1 * n2 * n3 * bytes fits in int64
static inline bool fits(int64_t n1, int64_t n2, int64_t n3, int64_t bytes)
{
    const int64_t lim = INT64_MAX;
    if (n1 == 0) return true;
    return n1 <= lim / n2 / n3 / bytes;
}

static inline int launch(const void* fn, dim3 grid, dim3 block, void** args, size_t lds, sf_stream_t stream)
{
    const hipError_t e = hipLaunchKernel(fn, grid, block, args, lds, (hipStream_t)stream);
    return e == hipSuccess ? SF_OK : SF_EHIP;
}

// LDS on one gfx950 CU.  Asking for LDS_PER_CU / n bytes per workgroup caps
// residency at n workgroups per CU.
constexpr size_t kLdsPerCu = 160 * 1024;
constexpr size_t kLdsMaxPerWg = 64 * 1024;

static inline size_t lds_request(size_t need, int per_cu)
{
    if (per_cu <= 0) return need;
    size_t cap = (kLdsPerCu / (size_t)per_cu) & ~(size_t)1023;
    if (cap > kLdsMaxPerWg) cap = kLdsMaxPerWg;
    return need > cap ? need : cap;
}

// Compute units of the device that `stream` belongs to (the current device
// for the NULL stream).
static inline int device_cus(sf_stream_t stream, int* cus)
{
    hipDevice_t dev = 0;
    const hipError_t de = stream ? hipStreamGetDevice((hipStream_t)stream, &dev) : hipGetDevice(&dev);
    if (de != hipSuccess ||
        hipDeviceGetAttribute(cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
        return SF_EHIP;
    return SF_OK;
}

// Window sums of the columns of a [T][C] int64 array into [W][C]
// (window.hip).
int launch_window_sum(const int64_t* x, int64_t T, int C, int64_t window, int64_t W,
                      int64_t* out, sf_stream_t stream);

}  // namespace sfk
