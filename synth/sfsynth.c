/*
 * sfsynth.c -- seeded, counter-based generator of synthetic stage-duration
 * matrices d[t][s][r] (int64 ns, layout [T][S][R], rank fastest).
 *
 * This file holds no part of the accounting method: it only draws numbers.
 * Every sample is a pure function of (seed, t, s, r), so any step range can
 * be generated on its own and chunks concatenate to the full matrix.
 *
 * Random bits: SplitMix64 (Steele, Lea and Flood, "Fast splittable
 * pseudorandom number generators", OOPSLA 2014): the i-th output of the
 * sequence seeded with k is fmix(k + (i + 1) * GAMMA), where fmix is the
 * published 64-bit finaliser with constants 0xbf58476d1ce4e5b9 and
 * 0x94d049bb133111eb and GAMMA = 0x9e3779b97f4a7c15.
 *
 * Lognormal stage durations: inverse-transform sampling (Devroye,
 * "Non-Uniform Random Variate Generation", 1986, ch. II.2) through a
 * per-stage table of 2^QBITS + 1 quantile nodes of the target lognormal,
 * computed by the caller in float64 and rounded to integer ns, with linear
 * interpolation between nodes in integer arithmetic.  Integer-only sampling
 * keeps the bytes identical on every machine.
 */
#include <stdint.h>

#define GAMMA 0x9e3779b97f4a7c15ULL

static inline uint64_t fmix(uint64_t z)
{
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ULL;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebULL;
    return z ^ (z >> 31);
}

/* i-th output of the SplitMix64 sequence seeded with k */
static inline uint64_t splitmix_at(uint64_t k, uint64_t i)
{
    return fmix(k + (i + 1) * GAMMA);
}

/* Exported so that tests can check the generator against the published
 * reference outputs of SplitMix64. */
uint64_t sfs_splitmix64_at(uint64_t k, uint64_t i) { return splitmix_at(k, i); }

/*
 * Fill out[(t - t0)][s][r] for t in [t0, t1).
 *
 *   table      [S][2^qbits + 1] quantile nodes (ns), nondecreasing per stage
 *   key_base   SplitMix64 key of the base draw
 *   key_tail   key of the heavy-tail draw (used when tail_thresh > 0)
 *   tail_thresh  a sample is multiplied by tail_mult when its tail draw is
 *                below this threshold (probability tail_thresh / 2^64)
 *   straggler  rank whose samples get + v * strag_num / strag_den (or -1)
 *   groups, group_off  rank role groups g = groups * r / R and an additive
 *                offset group_off[g][s] (groups == 0: none)
 *
 * Order per sample: base draw, + role offset, x tail_mult, + straggler.
 */
void sfs_generate(int64_t t0, int64_t t1, int32_t R, int32_t S,
                  const int64_t* table, int32_t qbits,
                  uint64_t key_base, uint64_t key_tail, uint64_t tail_thresh,
                  int64_t tail_mult, int32_t straggler, int64_t strag_num,
                  int64_t strag_den, int32_t groups, const int64_t* group_off,
                  int64_t* out, int32_t nthreads)
{
    const int64_t nodes = ((int64_t)1 << qbits) + 1;
#pragma omp parallel for schedule(static) num_threads(nthreads)
    for (int64_t t = t0; t < t1; ++t) {
        for (int32_t s = 0; s < S; ++s) {
            const int64_t* tab = table + (int64_t)s * nodes;
            int64_t* row = out + ((t - t0) * S + s) * (int64_t)R;
            const uint64_t ctr0 = ((uint64_t)t * (uint64_t)S + (uint64_t)s) * (uint64_t)R;
            for (int32_t r = 0; r < R; ++r) {
                uint64_t h = splitmix_at(key_base, ctr0 + (uint64_t)r);
                uint64_t idx = h >> (64 - qbits);
                uint64_t frac = (h >> (32 - qbits)) & 0xFFFFFFFFULL;
                int64_t lo = tab[idx], hi = tab[idx + 1];
                int64_t v = lo + (int64_t)(((unsigned __int128)(uint64_t)(hi - lo) * frac) >> 32);
                if (groups > 0) {
                    int32_t g = (int32_t)(((int64_t)groups * r) / R);
                    v += group_off[(int64_t)g * S + s];
                }
                if (tail_thresh && splitmix_at(key_tail, ctr0 + (uint64_t)r) < tail_thresh)
                    v *= tail_mult;
                if (r == straggler) v += v * strag_num / strag_den;
                row[r] = v;
            }
        }
    }
}
