/*
 * Exhaustive check of a binary32 -> bfloat16 rounding routine against an
 * independent method: for every one of the 2^32 bit patterns, take the two
 * bfloat16 neighbours of the value (truncation toward zero and the next one
 * out), measure both distances in double (exact: every binary32 and every
 * bfloat16 value is a double, and so are their differences here), and pick the
 * nearer, ties to the even last bit.  The neighbour past the largest finite
 * bfloat16 is 2^128, which rounds to infinity as IEEE 754 prescribes.
 * NaN inputs must give a quiet NaN of the same sign.
 *
 * Usage: bf16_nearest <path to a shared library exporting
 *        uint16_t <symbol>(uint32_t)> <symbol>
 * Prints the number of mismatching patterns and the first few.
 */
#include <dlfcn.h>
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

typedef uint16_t (*round_fn)(uint32_t);

static double value_of_f32_bits(uint32_t u) {
    float f;
    memcpy(&f, &u, 4);
    return (double)f;
}

static uint16_t expected(uint32_t u) {
    const uint32_t sign = u & 0x80000000u;
    const uint32_t mag = u & 0x7FFFFFFFu;
    if (mag > 0x7F800000u) return 0; /* NaN: checked separately */
    if (mag == 0x7F800000u) return (uint16_t)(u >> 16);
    const uint32_t down = mag & 0xFFFF0000u;
    const uint32_t up = down + 0x10000u;
    const double x = fabs(value_of_f32_bits(u));
    const double lo = value_of_f32_bits(down);
    const double hi = (up >= 0x7F800000u) ? ldexp(1.0, 128) : value_of_f32_bits(up);
    const double dl = x - lo, dh = hi - x;
    uint32_t pick;
    if (dl < dh) pick = down;
    else if (dh < dl) pick = up;
    else pick = ((down >> 16) & 1u) ? up : down;
    return (uint16_t)((pick | sign) >> 16);
}

int main(int argc, char** argv) {
    if (argc != 3) { fprintf(stderr, "usage: %s lib symbol\n", argv[0]); return 2; }
    void* h = dlopen(argv[1], RTLD_NOW);
    if (!h) { fprintf(stderr, "%s\n", dlerror()); return 2; }
    round_fn fn = (round_fn)dlsym(h, argv[2]);
    if (!fn) { fprintf(stderr, "%s\n", dlerror()); return 2; }
    unsigned long long bad = 0;
    unsigned long long nan_seen = 0;
#pragma omp parallel for schedule(static) reduction(+:bad, nan_seen)
    for (long long k = 0; k < (1LL << 32); k++) {
        const uint32_t u = (uint32_t)k;
        const uint16_t got = fn(u);
        if ((u & 0x7FFFFFFFu) > 0x7F800000u) {
            nan_seen++;
            const int is_nan = ((got & 0x7F80u) == 0x7F80u) && (got & 0x007Fu);
            const int quiet = (got & 0x0040u) != 0;
            const int same_sign = (got >> 15) == (u >> 31);
            if (!(is_nan && quiet && same_sign)) bad++;
            continue;
        }
        if (got != expected(u)) {
            bad++;
        }
    }
    printf("%llu %llu\n", bad, nan_seen);
    return 0;
}
