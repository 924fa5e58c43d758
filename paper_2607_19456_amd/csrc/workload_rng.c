/*
 * workload_rng.c -- seeded N(0,1) float32 generator for synthetic workloads.
 *
 * Holds no part of the attention arithmetic: it only turns (seed, stream,
 * index) into normally distributed numbers, so that the HIP path and the
 * CPU reference can be fed the very same bytes at any size quickly.
 *
 * Uniform bits: Philox4x32-10, the counter-based generator of Salmon,
 * Moraes, Dror and Shaw, "Parallel random numbers: as easy as 1, 2, 3"
 * (SC'11): a 128-bit counter (index, stream, 0, 0) and a 64-bit key
 * (seed) go through ten rounds of two 32x32->64 multiplies with the
 * published constants; the key is bumped by the published Weyl increments
 * between rounds.
 * Normals: Box-Muller in double precision on pairs of 32-bit words,
 * u1 in (0, 1], u2 in [0, 1), rounded to float32.  Element i of a stream
 * depends only on (seed, stream, i), so any thread split gives identical
 * output.
 */
#include <math.h>
#include <stdint.h>

#ifndef M_PI
#define M_PI 3.14159265358979323846
#endif

#define PHILOX_M0 0xD2511F53u
#define PHILOX_M1 0xCD9E8D57u
#define PHILOX_W0 0x9E3779B9u
#define PHILOX_W1 0xBB67AE85u

static void philox4x32_10(uint32_t ctr[4], uint32_t k0, uint32_t k1)
{
    for (int r = 0; r < 10; ++r) {
        const uint64_t p0 = (uint64_t)PHILOX_M0 * ctr[0];
        const uint64_t p1 = (uint64_t)PHILOX_M1 * ctr[2];
        const uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        const uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        const uint32_t n0 = hi1 ^ ctr[1] ^ k0;
        const uint32_t n1 = lo1;
        const uint32_t n2 = hi0 ^ ctr[3] ^ k1;
        const uint32_t n3 = lo0;
        ctr[0] = n0; ctr[1] = n1; ctr[2] = n2; ctr[3] = n3;
        k0 += PHILOX_W0;
        k1 += PHILOX_W1;
    }
}

/* Four normals from one Philox block: counter (block, stream, 0, 0). */
static void normals4(uint64_t seed, uint32_t stream, uint64_t block, double z[4])
{
    uint32_t c[4] = {(uint32_t)block, stream, (uint32_t)(block >> 32), 0u};
    philox4x32_10(c, (uint32_t)seed, (uint32_t)(seed >> 32));
    for (int p = 0; p < 2; ++p) {
        const double u1 = ((double)c[2 * p] + 1.0) * (1.0 / 4294967296.0);
        const double u2 = (double)c[2 * p + 1] * (1.0 / 4294967296.0);
        const double r = sqrt(-2.0 * log(u1));
        const double t = 2.0 * M_PI * u2;
        z[2 * p] = r * cos(t);
        z[2 * p + 1] = r * sin(t);
    }
}

/* out[i] = N(0,1) sample (offset + i) of (seed, stream), i in [0, count). */
void workload_normal_f32(uint64_t seed, uint32_t stream, int64_t offset,
                         float *out, int64_t count, int threads)
{
    if (count <= 0 || offset < 0) return;
    const int64_t first = offset / 4;
    const int64_t last = (offset + count - 1) / 4;
#pragma omp parallel for schedule(static) num_threads(threads > 0 ? threads : 1)
    for (int64_t blk = first; blk <= last; ++blk) {
        double z[4];
        normals4(seed, stream, (uint64_t)blk, z);
        for (int k = 0; k < 4; ++k) {
            const int64_t i = blk * 4 + k - offset;
            if (i >= 0 && i < count) out[i] = (float)z[k];
        }
    }
}

/* Raw Philox block, exposed so a test can check the published test vectors. */
void workload_philox4x32_10(const uint32_t ctr_in[4], const uint32_t key[2],
                            uint32_t out[4])
{
    uint32_t c[4] = {ctr_in[0], ctr_in[1], ctr_in[2], ctr_in[3]};
    philox4x32_10(c, key[0], key[1]);
    for (int k = 0; k < 4; ++k) out[k] = c[k];
}
