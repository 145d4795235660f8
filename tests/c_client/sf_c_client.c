/*
 * sf_c_client.c -- a plain C99 host program that drives libstagefrontier
 * through its C ABI alone: no C++, no Python, no torch.  It allocates
 * device memory with the HIP runtime, runs the hot path (sf_frontier on a
 * stream of its own, then sf_window_summary on the NULL stream), and writes
 * the results to a file; the GPU tests compare them with the CPU oracle.
 *
 *   sf_c_client IN OUT T R S WINDOW
 *
 * IN   raw little-endian int64 durations [T][S][R].
 * OUT  raw results, back to back: increment [T][S] int64, leader [T][S]
 *      int32, stage_exposed [W][S] int64, lead_counts [W][S][R] int32,
 *      top2 [W][2][2] int32, with W = sf_num_windows(T, WINDOW).
 *
 * stdout: the library version and one "name value" line per host-side
 * check of the argument validation (statuses that need no device work).
 * Exit status 0 on success, 1 on any failure (with a message on stderr).
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include <hip/hip_runtime_api.h>

#include "stagefrontier.h"

#define HIP_OK(call)                                                                  \
    do {                                                                              \
        hipError_t e_ = (call);                                                       \
        if (e_ != hipSuccess) {                                                       \
            fprintf(stderr, "%s failed: %s\n", #call, hipGetErrorString(e_));         \
            return 1;                                                                 \
        }                                                                             \
    } while (0)

#define SF_OK_OR_FAIL(call)                                                           \
    do {                                                                              \
        int s_ = (call);                                                              \
        if (s_ != SF_OK) {                                                            \
            fprintf(stderr, "%s returned %d (%s)\n", #call, s_, sf_strerror(s_));     \
            return 1;                                                                 \
        }                                                                             \
    } while (0)

static void* read_file(const char* path, size_t bytes)
{
    FILE* f = fopen(path, "rb");
    void* p;
    if (!f) return NULL;
    p = malloc(bytes ? bytes : 1);
    if (p && bytes && fread(p, 1, bytes, f) != bytes) {
        free(p);
        p = NULL;
    }
    fclose(f);
    return p;
}

int main(int argc, char** argv)
{
    int64_t T, W, window;
    int32_t R, S;
    size_t nd, ni, nl, ne, nc, nt;
    int64_t* hd;
    void* hout;
    int64_t *dd, *dinc, *dex;
    int32_t *dlead, *dcnt, *dtop;
    hipStream_t stream;
    FILE* f;

    if (argc != 7) {
        fprintf(stderr, "usage: %s IN OUT T R S WINDOW\n", argv[0]);
        return 1;
    }
    T = strtoll(argv[3], NULL, 10);
    R = (int32_t)strtol(argv[4], NULL, 10);
    S = (int32_t)strtol(argv[5], NULL, 10);
    window = strtoll(argv[6], NULL, 10);
    W = sf_num_windows(T, window);
    if (T < 1 || R < 1 || S < 1 || W < 1) {
        fprintf(stderr, "bad sizes\n");
        return 1;
    }
    printf("version %s\n", sf_version());

    /* host-side validation: every one of these returns before any launch */
    printf("frontier_r0 %d\n", sf_frontier(NULL, T, 0, S, NULL, NULL, NULL));
    printf("frontier_null %d\n", sf_frontier(NULL, T, R, S, NULL, NULL, NULL));
    printf("frontier_r_too_big %d\n", sf_frontier(NULL, T, SF_MAX_R + 1, S, NULL, NULL, NULL));
    printf("summary_window0 %d\n", sf_window_summary(NULL, NULL, T, R, S, 0, NULL, NULL, NULL, NULL));
    printf("frontier_t0 %d\n", sf_frontier(NULL, 0, R, S, NULL, NULL, NULL));
    printf("num_windows %lld\n", (long long)W);
    printf("strerror_einval %s\n", sf_strerror(SF_EINVAL));

    nd = (size_t)T * (size_t)S * (size_t)R * 8u;
    ni = (size_t)T * (size_t)S * 8u;
    nl = (size_t)T * (size_t)S * 4u;
    ne = (size_t)W * (size_t)S * 8u;
    nc = (size_t)W * (size_t)S * (size_t)R * 4u;
    nt = (size_t)W * 16u;
    hd = (int64_t*)read_file(argv[1], nd);
    if (!hd) {
        fprintf(stderr, "cannot read %s (%zu bytes)\n", argv[1], nd);
        return 1;
    }

    HIP_OK(hipMalloc((void**)&dd, nd));
    HIP_OK(hipMalloc((void**)&dinc, ni));
    HIP_OK(hipMalloc((void**)&dlead, nl));
    HIP_OK(hipMalloc((void**)&dex, ne));
    HIP_OK(hipMalloc((void**)&dcnt, nc));
    HIP_OK(hipMalloc((void**)&dtop, nt));
    HIP_OK(hipStreamCreate(&stream));
    HIP_OK(hipMemcpy(dd, hd, nd, hipMemcpyHostToDevice));

    SF_OK_OR_FAIL(sf_frontier(dd, T, R, S, dinc, dlead, (sf_stream_t)stream));
    HIP_OK(hipStreamSynchronize(stream));
    SF_OK_OR_FAIL(sf_window_summary(dinc, dlead, T, R, S, window, dex, dcnt, dtop, NULL));
    HIP_OK(hipDeviceSynchronize());

    hout = malloc(ni + nl + ne + nc + nt);
    if (!hout) {
        fprintf(stderr, "out of host memory\n");
        return 1;
    }
    HIP_OK(hipMemcpy((char*)hout, dinc, ni, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy((char*)hout + ni, dlead, nl, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy((char*)hout + ni + nl, dex, ne, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy((char*)hout + ni + nl + ne, dcnt, nc, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy((char*)hout + ni + nl + ne + nc, dtop, nt, hipMemcpyDeviceToHost));

    f = fopen(argv[2], "wb");
    if (!f || fwrite(hout, 1, ni + nl + ne + nc + nt, f) != ni + nl + ne + nc + nt) {
        fprintf(stderr, "cannot write %s\n", argv[2]);
        return 1;
    }
    fclose(f);

    HIP_OK(hipStreamDestroy(stream));
    HIP_OK(hipFree(dd));
    HIP_OK(hipFree(dinc));
    HIP_OK(hipFree(dlead));
    HIP_OK(hipFree(dex));
    HIP_OK(hipFree(dcnt));
    HIP_OK(hipFree(dtop));
    free(hd);
    free(hout);
    printf("done\n");
    return 0;
}
