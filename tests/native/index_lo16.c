/* Check of the short first mixing round the digesting kernels use for
 * 16-bit words (BF16 state, the bf16 working copy).  For a word w < 2^16 at
 * flat index i = hi:lo (tag k) the digest hashes z = (w ^ i) + gamma_k with
 * the splitmix64 mix.  When every index of a tile shares bits 16..63, x =
 * w ^ lo = A + v with A = lo & 0xFFFF0000 and v < 2^16, and with
 * B = A + lo32(gamma) = c0 * 2^32 + B_lo the short form takes
 *   z_lo = x + lo32(gamma),  lo1 = z_lo ^ U,  U = (z_hi << 2) | (B_lo >> 30),
 *   z_hi = hi + hi32(gamma) + (k << 24) + c0,  H = z_hi ^ (z_hi >> 30),
 *   z1 = lo1 * CLO + ((lo1 * CHI + H * CLO) << 32)   (mod 2^64)
 * whenever B_lo <= 0xFFFF0000 and (B_lo mod 2^30) <= 0x3FFF0000.
 * Checked here: for every A (all 2^16 values of bits 16..31) that passes the
 * two conditions and every v (all 2^16), at one high half and tag, z1 equals
 * the first mixing round of the definition; at a spread of other high halves
 * and all four tags on sampled (A, v); and exactly four values of A fail the
 * conditions.  Prints: pairs checked, mismatches, failing A values; exit
 * status 0 only if there are no mismatches. */
#include <stdint.h>
#include <stdio.h>

static const uint64_t GAMMA = 0x9E3779B97F4A7C15ull;
static const uint64_t C1 = 0xBF58476D1CE4E5B9ull;

/* first mixing round of splitmix64, as defined: z ^ (z >> 30), times C1 */
static uint64_t round1_plain(uint64_t z) { return (z ^ (z >> 30)) * C1; }

static int passes(uint32_t a) {
    const uint32_t b_lo = a + (uint32_t)GAMMA;
    return b_lo <= 0xFFFF0000u && (b_lo & 0x3FFFFFFFu) <= 0x3FFF0000u;
}

static uint64_t round1_short(uint32_t hi, uint32_t k, uint32_t a, uint32_t x) {
    const uint64_t b = (uint64_t)a + (uint32_t)GAMMA;
    const uint32_t c0 = (uint32_t)(b >> 32), t = (uint32_t)b >> 30;
    const uint32_t z_hi = hi + (uint32_t)(GAMMA >> 32) + (k << 24) + c0;
    const uint32_t h = z_hi ^ (z_hi >> 30);
    const uint32_t u = (z_hi << 2) | t;
    const uint32_t lo1 = (x + (uint32_t)GAMMA) ^ u;
    const uint32_t clo = (uint32_t)C1, chi = (uint32_t)(C1 >> 32);
    const uint64_t prod = (uint64_t)lo1 * clo + ((uint64_t)(h * clo) << 32);
    return prod + ((uint64_t)(lo1 * chi) << 32);
}

static uint64_t splitmix_state(uint32_t hi, uint32_t k, uint32_t a, uint32_t v) {
    /* w ^ i with i = hi:(a + l) and w such that x = w ^ lo = a + v: the state
     * depends only on x, so x = a + v stands for every (w, l) pair giving it */
    const uint64_t x = (uint64_t)hi << 32 | (uint64_t)(a + v);
    return x + GAMMA + ((uint64_t)k << 56);
}

int main(void) {
    unsigned long long checked = 0, bad = 0;
    int failing = 0;
    for (uint32_t ah = 0; ah < 65536; ++ah) failing += !passes(ah << 16);
#pragma omp parallel for reduction(+ : checked, bad) schedule(dynamic, 64)
    for (int ah = 0; ah < 65536; ++ah) {
        const uint32_t a = (uint32_t)ah << 16;
        if (!passes(a)) continue;
        for (uint32_t v = 0; v < 65536; ++v) {
            const uint32_t hi = 0x00ABCDEFu;
            if (round1_short(hi, 0, a, a + v) != round1_plain(splitmix_state(hi, 0, a, v))) ++bad;
            ++checked;
        }
        /* other high halves (up to the 2^56 index limit) and every tag */
        uint64_t s = 0x9E3779B97F4A7C15ull * (uint64_t)(ah + 1);
        for (int r = 0; r < 64; ++r) {
            s ^= s << 13; s ^= s >> 7; s ^= s << 17;
            const uint32_t hi = (uint32_t)(s >> 40);          /* < 2^24 */
            const uint32_t v = (uint32_t)s & 0xFFFFu;
            for (uint32_t k = 0; k < 4; ++k) {
                if (round1_short(hi, k, a, a + v) != round1_plain(splitmix_state(hi, k, a, v))) ++bad;
                ++checked;
            }
        }
    }
    printf("%llu %llu %d\n", checked, bad, failing);
    return bad != 0;
}
