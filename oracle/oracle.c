/*
 * oracle.c -- the plain CPU definition of the sharded AdamW commit and the
 * state digest.  TEST INFRASTRUCTURE ONLY: see oracle.h.  Single-threaded,
 * one element at a time, one rounding per statement, written for a reader to
 * check by eye rather than for speed.
 */
#include "oracle.h"

#include <math.h>
#include <string.h>

static uint32_t f32_bits(float x) {
    uint32_t u;
    memcpy(&u, &x, sizeof u);
    return u;
}

/* ------------------------------------------------------------------------ */
/* splitmix64 (Steele, Lea, Flood, "Fast splittable pseudorandom number       */
/* generators", OOPSLA 2014, with the mixing constants of Vigna's public      */
/* reference splitmix64.c).  The generator adds the golden gamma to its state */
/* and returns the mix of the new state; the digest applies that to one word. */
/* All arithmetic wraps mod 2^64.                                             */
/* ------------------------------------------------------------------------ */
uint64_t oracle_splitmix64(uint64_t x) {
    uint64_t z = x + 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

/* ------------------------------------------------------------------------ */
/* bfloat16 working copy (the paper keeps BF16 working state, Sec. IV-A).     */
/* bf16 keeps the sign, the 8 exponent bits and the top 7 mantissa bits of a  */
/* binary32 value.  Round to nearest, ties to even, on the 16 dropped bits:   */
/*   dropped above one half       -> round the magnitude up                   */
/*   dropped exactly one half     -> round up only if the kept part is odd    */
/*   dropped below one half       -> truncate                                 */
/* A carry out of the mantissa moves to the next binade, and out of the       */
/* largest finite binade to infinity, exactly as IEEE rounding requires.      */
/* NaN keeps its sign and top payload bits and is made quiet.                 */
/* ------------------------------------------------------------------------ */
uint16_t oracle_bf16_rne(uint32_t u) {
    const uint32_t exponent = (u >> 23) & 0xFFu;
    const uint32_t mantissa = u & 0x007FFFFFu;
    if (exponent == 0xFFu && mantissa != 0u) {
        return (uint16_t)((u >> 16) | 0x0040u);
    }
    uint32_t kept = u >> 16;
    const uint32_t dropped = u & 0xFFFFu;
    const uint32_t half = 0x8000u;
    if (dropped > half || (dropped == half && (kept & 1u) != 0u)) {
        kept = kept + 1u;
    }
    return (uint16_t)kept;
}

void oracle_bf16_rne_array(const uint32_t* in, uint16_t* out, uint64_t n) {
    for (uint64_t i = 0; i < n; i++) {
        out[i] = oracle_bf16_rne(in[i]);
    }
}

/* ------------------------------------------------------------------------ */
/* Per-step scalars.  The optimizer step counter tau_opt is part of the       */
/* preserved state (Sec. III-A, eq. 2); t is its value after the increment.   */
/* beta^t is formed by t successive double multiplications starting from 1.   */
/* (Once neither product changes any more, further multiplications cannot     */
/* change it either, so the loop may stop there.)                             */
/* ------------------------------------------------------------------------ */
void oracle_make_scalars(const oracle_hyper* h, uint64_t step, oracle_scalars* out) {
    const double lr = (double)h->lr;
    const double b1 = (double)h->beta1;
    const double b2 = (double)h->beta2;
    const double wd = (double)h->weight_decay;

    double b1_pow = 1.0;
    double b2_pow = 1.0;
    for (uint64_t t = 0; t < step; t++) {
        const double n1 = b1_pow * b1;
        const double n2 = b2_pow * b2;
        const int unchanged = (n1 == b1_pow) && (n2 == b2_pow);
        b1_pow = n1;
        b2_pow = n2;
        if (unchanged) {
            break;
        }
    }

    out->beta1 = h->beta1;
    out->beta2 = h->beta2;
    out->eps = h->eps;
    out->decay = (float)(1.0 - lr * wd);
    out->omb1 = (float)(1.0 - b1);
    out->omb2 = (float)(1.0 - b2);
    out->step_size = (float)(lr / (1.0 - b1_pow));
    out->rs_bc2 = (float)(1.0 / sqrt(1.0 - b2_pow));
}

/* ------------------------------------------------------------------------ */
/* AdamW on the local flat shard: the update that makes W, M, V "committed"  */
/* (Sec. I; Sec. III-A action L1).  Decoupled weight decay on the pre-update  */
/* weight, bias-corrected moments, eps added after the bias-corrected root.   */
/* Each statement is one binary32 operation with one RNE rounding.            */
/* ------------------------------------------------------------------------ */
static void adamw_element(float* p, float grad, float* m, float* v, const oracle_scalars* sc) {
    const float w = *p;
    const float m_prev = *m;
    const float v_prev = *v;

    const float w_decayed = w * sc->decay;

    const float m_keep = sc->beta1 * m_prev;
    const float m_push = sc->omb1 * grad;
    const float m_next = m_keep + m_push;

    const float grad_sq = grad * grad;
    const float v_keep = sc->beta2 * v_prev;
    const float v_push = sc->omb2 * grad_sq;
    const float v_next = v_keep + v_push;

    const float root = sqrtf(v_next);
    const float root_hat = root * sc->rs_bc2;
    const float denom = root_hat + sc->eps;
    const float ratio = m_next / denom;
    const float delta = sc->step_size * ratio;
    const float w_next = w_decayed - delta;

    *p = w_next;
    *m = m_next;
    *v = v_next;
}

void oracle_adamw_commit(float* p, const float* g, float* m, float* v,
                         uint16_t* bf16, uint64_t n, const oracle_scalars* sc) {
    for (uint64_t i = 0; i < n; i++) {
        adamw_element(&p[i], g[i], &m[i], &v[i], sc);
        bf16[i] = oracle_bf16_rne(f32_bits(p[i]));
    }
}

/* ------------------------------------------------------------------------ */
/* BF16 state, the paper's own precision for weights and moments (Sec. IV-A): */
/* widen each word exactly, apply the same binary32 update, round p', m', v'  */
/* back with the RNE rule above.                                               */
/* ------------------------------------------------------------------------ */
static float widen_bf16(uint16_t b) {
    const uint32_t u = (uint32_t)b << 16;
    float x;
    memcpy(&x, &u, sizeof x);
    return x;
}

void oracle_adamw_commit_bf16(uint16_t* p, const uint16_t* g, uint16_t* m, uint16_t* v,
                              uint64_t n, const oracle_scalars* sc) {
    for (uint64_t i = 0; i < n; i++) {
        float w = widen_bf16(p[i]);
        float mm = widen_bf16(m[i]);
        float vv = widen_bf16(v[i]);
        adamw_element(&w, widen_bf16(g[i]), &mm, &vv, sc);
        p[i] = oracle_bf16_rne(f32_bits(w));
        m[i] = oracle_bf16_rne(f32_bits(mm));
        v[i] = oracle_bf16_rne(f32_bits(vv));
    }
}

uint64_t oracle_state_digest_bf16(const uint16_t* p, const uint16_t* m, const uint16_t* v,
                                  uint64_t n, uint64_t first_index) {
    uint64_t sum = 0;
    for (uint64_t i = 0; i < n; i++) {
        const uint64_t index = first_index + i;
        sum += oracle_splitmix64((uint64_t)p[i] ^ (index | (0ull << 56)));
        sum += oracle_splitmix64((uint64_t)m[i] ^ (index | (1ull << 56)));
        sum += oracle_splitmix64((uint64_t)v[i] ^ (index | (2ull << 56)));
    }
    return sum;
}

/* ------------------------------------------------------------------------ */
/* State digest: the identity of a committed frontier.  The paper checks     */
/* that every rank's W, M, V match bitwise (abstract; Sec. IV-G); this digest */
/* names that state in 64 bits.  Word = the 32 bits of one element, zero     */
/* extended; it is XORed with the element's global flat index, whose bits    */
/* 56..63 carry the array tag (0 = W, 1 = M, 2 = V, 3 = bf16 copy).  The     */
/* splitmix64 values are summed mod 2^64, so any partition of the index      */
/* range, in any order, gives the same sum.                                  */
/* ------------------------------------------------------------------------ */
uint64_t oracle_state_digest(const float* p, const float* m, const float* v,
                             uint64_t n, uint64_t first_index) {
    uint64_t sum = 0;
    for (uint64_t i = 0; i < n; i++) {
        const uint64_t index = first_index + i;
        sum += oracle_splitmix64((uint64_t)f32_bits(p[i]) ^ (index | (0ull << 56)));
        sum += oracle_splitmix64((uint64_t)f32_bits(m[i]) ^ (index | (1ull << 56)));
        sum += oracle_splitmix64((uint64_t)f32_bits(v[i]) ^ (index | (2ull << 56)));
    }
    return sum;
}

uint64_t oracle_bf16_digest(const uint16_t* b, uint64_t n, uint64_t first_index) {
    uint64_t sum = 0;
    for (uint64_t i = 0; i < n; i++) {
        const uint64_t index = first_index + i;
        sum += oracle_splitmix64((uint64_t)b[i] ^ (index | (3ull << 56)));
    }
    return sum;
}

uint64_t oracle_commit_and_digest(float* p, const float* g, float* m, float* v,
                                  uint16_t* bf16, uint64_t n, uint64_t first_index,
                                  const oracle_hyper* h, uint64_t step) {
    oracle_scalars sc;
    oracle_make_scalars(h, step, &sc);
    oracle_adamw_commit(p, g, m, v, bf16, n, &sc);
    return oracle_state_digest(p, m, v, n, first_index);
}

/* ------------------------------------------------------------------------ */
/* The quiescent boundary: gradients zeroed once the update has committed     */
/* (Sec. I; Sec. III-C, phase 2), and the guard that checks it.              */
/* ------------------------------------------------------------------------ */
void oracle_zero_grad(float* g, uint64_t n) {
    for (uint64_t i = 0; i < n; i++) {
        g[i] = 0.0f;
    }
}

uint64_t oracle_count_outstanding(const float* g, uint64_t n) {
    uint64_t count = 0;
    for (uint64_t i = 0; i < n; i++) {
        if (f32_bits(g[i]) != 0u) {
            count++;
        }
    }
    return count;
}
