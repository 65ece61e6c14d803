/*
 * gen.c -- seeded synthetic inputs for the sharded-commit workloads.
 *
 * Holds none of the commit's or the digest's arithmetic: it only draws
 * bit-reproducible pseudo-random binary32 arrays.  Both the GPU runs and the
 * CPU oracle take their inputs from here (generated on the host, then copied
 * to the device), so neither side produces the other's inputs.
 *
 * Generator: Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel random
 * numbers: as easy as 1, 2, 3", SC 2011) keyed by the seed, with counter
 * (lo32(index), hi32(index), lo32(step), array id).  One call gives 128 bits =
 * eight 16-bit uniforms u_j; their centred sum  s = sum_j u_j - 262140  is an
 * Irwin-Hall(8) approximation of a normal with standard deviation
 * 65536*sqrt(2/3)*sqrt(1 - 2^-32).  The value is  f32(s) * f32(scale), exact
 * integer work until one binary32 multiply, so any host reproduces it bit for
 * bit.  Since |s| <= 262140 the result is never a denormal, and s = 0 gives +0.
 * Every element is a pure function of (seed, array id, step, global index), so
 * any shard of a larger flat vector, and any chunking, draws the same values.
 */
#include <stdint.h>
#include <string.h>

#define PHILOX_M0 0xD2511F53u
#define PHILOX_M1 0xCD9E8D57u
#define PHILOX_W0 0x9E3779B9u
#define PHILOX_W1 0xBB67AE85u

void gen_philox4x32_10(const uint32_t ctr_in[4], const uint32_t key_in[2], uint32_t out[4]) {
    uint32_t c0 = ctr_in[0], c1 = ctr_in[1], c2 = ctr_in[2], c3 = ctr_in[3];
    uint32_t k0 = key_in[0], k1 = key_in[1];
    for (int r = 0; r < 10; r++) {
        const uint64_t prod0 = (uint64_t)PHILOX_M0 * c0;
        const uint64_t prod1 = (uint64_t)PHILOX_M1 * c2;
        const uint32_t hi0 = (uint32_t)(prod0 >> 32), lo0 = (uint32_t)prod0;
        const uint32_t hi1 = (uint32_t)(prod1 >> 32), lo1 = (uint32_t)prod1;
        const uint32_t n0 = hi1 ^ c1 ^ k0;
        const uint32_t n2 = hi0 ^ c3 ^ k1;
        c0 = n0;
        c1 = lo1;
        c2 = n2;
        c3 = lo0;
        k0 += PHILOX_W0;
        k1 += PHILOX_W1;
    }
    out[0] = c0;
    out[1] = c1;
    out[2] = c2;
    out[3] = c3;
}

static inline int32_t centred_sum(uint64_t seed, uint32_t array_id, uint64_t step, uint64_t index) {
    const uint32_t ctr[4] = {(uint32_t)index, (uint32_t)(index >> 32), (uint32_t)step, array_id};
    const uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    uint32_t w[4];
    gen_philox4x32_10(ctr, key, w);
    int32_t s = 0;
    for (int j = 0; j < 4; j++) {
        s += (int32_t)(w[j] & 0xFFFFu) + (int32_t)(w[j] >> 16);
    }
    return s - 262140;
}

/*
 * Fill out[0..n) with the values of global indices first_index .. first_index+n-1.
 * kind 0: normal-like, sd = sd_scale-defined;  kind 1: its absolute value;
 * kind 2: all +0.  scale is the binary32 multiplier (sigma / sd of the sum).
 * Threads: OpenMP over the index range when built with -fopenmp.
 */
void gen_fill(float* out, uint64_t n, uint64_t first_index, uint64_t seed, uint32_t array_id,
              uint64_t step, int kind, float scale) {
    if (kind == 2) {
        memset(out, 0, n * sizeof(float));
        return;
    }
    const int64_t nn = (int64_t)n;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < nn; i++) {
        const int32_t s = centred_sum(seed, array_id, step, first_index + (uint64_t)i);
        float x = (float)s * scale;
        if (kind == 1 && x < 0.0f) {
            x = -x;
        }
        out[i] = x;
    }
}

int gen_num_threads(void) {
#ifdef _OPENMP
    extern int omp_get_max_threads(void);
    return omp_get_max_threads();
#else
    return 1;
#endif
}
