/* Exhaustive check of the square-root selection the BF16-state commit uses
 * for second moments in [2^-96, +inf): given a hardware root s within one
 * ulp of sqrt(x), the root is s_dn = s - 1 ulp when fma(-s_dn, s, x) <= 0,
 * s_up = s + 1 ulp when fma(-s_up, s, x) > 0, else s (bit patterns +-1).
 * For every binary32 x in the range and each of the three hardware results
 * the one-ulp bound allows (the correctly rounded root and its two
 * neighbours), the selection must give the correctly rounded root.  The
 * reference root is the correctly rounded sqrtf of the C library (IEEE
 * binary32).  Prints the number of inputs checked and of failures; exit
 * status 0 only if there are none. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

static float from_bits(uint32_t u) { float f; memcpy(&f, &u, 4); return f; }
static uint32_t to_bits(float f) { uint32_t u; memcpy(&u, &f, 4); return u; }

static float select_root(float s, float x) {
    const float s_dn = from_bits(to_bits(s) - 1u);
    const float s_up = from_bits(to_bits(s) + 1u);
    const float r_dn = fmaf(-s_dn, s, x);
    const float r_up = fmaf(-s_up, s, x);
    const float t = r_dn <= 0.0f ? s_dn : s;
    return r_up > 0.0f ? s_up : t;
}

int main(void) {
    const uint32_t lo = 0x0F800000u, hi = 0x7F800000u; /* [2^-96, +inf) */
    unsigned long long checked = 0, bad = 0;
#pragma omp parallel for reduction(+ : checked, bad) schedule(static)
    for (long long k = lo; k < (long long)hi; ++k) {
        const float x = from_bits((uint32_t)k);
        const float want = sqrtf(x);
        const uint32_t w = to_bits(want);
        for (int d = -1; d <= 1; ++d) {
            const float s = from_bits(w + (uint32_t)d);
            if (to_bits(select_root(s, x)) != w) ++bad;
        }
        ++checked;
    }
    printf("%llu %llu\n", checked, bad);
    return bad == 0 ? 0 : 1;
}
