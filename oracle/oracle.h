/*
 * oracle.h -- plain, slow, single-threaded CPU definition of the sharded
 * AdamW commit and of the 64-bit state digest.
 *
 * TEST INFRASTRUCTURE ONLY.  This code exists to check the GPU library; it is
 * never part of the product path.  Only the test suite, the smoke check and
 * the CPU-baseline leg of the benchmark may load it.  It shares no source,
 * header, helper or constant table with the GPU library.
 *
 * What it follows (the paper names the optimizer and the state but prints no
 * formula, constant or rounding for it):
 *   - the preserved application state is the sharded weights W and the AdamW
 *     first/second moments M, V plus the step counter (Sec. III-A, eq. 2);
 *   - state is "committed" once the optimizer update has been applied
 *     (Sec. I, Sec. III-A, action L1);
 *   - recovered ranks must hold bit-identical W, M, V (abstract; Sec. IV-G).
 * The arithmetic below is the reading this project fixes where the paper is
 * silent (decoupled weight decay on the pre-update weight, bias correction by
 * beta^t computed with t double multiplications, one fp32 rounding per scalar,
 * binary32 round-to-nearest-even per operation with no fused multiply-add,
 * RNE bf16 working copy, splitmix64 sum digest).  Every such reading is listed
 * in the design notes of the repository.
 *
 * Build: gcc -O2 -std=c11 -ffp-contract=off -fno-fast-math -fno-math-errno.
 * On x86-64 float arithmetic is SSE binary32 (no excess precision), sqrtf is
 * the correctly rounded square root and '/' the correctly rounded division.
 */
#ifndef PACT_ORACLE_H
#define PACT_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* The five user hyperparameters of AdamW, as binary32. */
typedef struct oracle_hyper {
    float lr;
    float beta1;
    float beta2;
    float eps;
    float weight_decay;
} oracle_hyper;

/* The per-call scalars the element loop uses.  beta1, beta2 and eps are the
 * user's binary32 values unchanged; the other five are derived in double and
 * rounded once to binary32. */
typedef struct oracle_scalars {
    float beta1;
    float beta2;
    float eps;
    float decay;      /* f32(1 - lr*wd)               */
    float omb1;       /* f32(1 - beta1)               */
    float omb2;       /* f32(1 - beta2)               */
    float step_size;  /* f32(lr / (1 - beta1^t))      */
    float rs_bc2;     /* f32(1 / sqrt(1 - beta2^t))   */
} oracle_scalars;

/* splitmix64 output for generator state x: mix(x + golden gamma). */
uint64_t oracle_splitmix64(uint64_t x);

/* Round-to-nearest-even binary32 -> bfloat16 (upper 16 bits). */
uint16_t oracle_bf16_rne(uint32_t f32_bits);
void oracle_bf16_rne_array(const uint32_t* in, uint16_t* out, uint64_t n);

/* Scalars for step t >= 1. */
void oracle_make_scalars(const oracle_hyper* h, uint64_t step, oracle_scalars* out);

/* One AdamW commit over n elements, in place on p, m, v; writes bf16 = RNE(p'). */
void oracle_adamw_commit(float* p, const float* g, float* m, float* v,
                         uint16_t* bf16, uint64_t n, const oracle_scalars* sc);

/* Digest of (p, m, v): sum over k in {0,1,2}, i < n of
 * splitmix64(zext(bits(X_k[i])) ^ ((first_index + i) | k << 56)), mod 2^64. */
uint64_t oracle_state_digest(const float* p, const float* m, const float* v,
                             uint64_t n, uint64_t first_index);

/* Digest of the bf16 copy, tag 3, 16-bit words zero-extended. */
uint64_t oracle_bf16_digest(const uint16_t* b, uint64_t n, uint64_t first_index);

/* BF16 state (the paper's precision: BF16 weights and moments, Sec. IV-A).
 * Each bf16 word is widened exactly to binary32 (bits << 16), the same
 * binary32 update as oracle_adamw_commit is applied, and p', m', v' are
 * rounded back to bf16 with oracle_bf16_rne. */
void oracle_adamw_commit_bf16(uint16_t* p, const uint16_t* g, uint16_t* m, uint16_t* v,
                              uint64_t n, const oracle_scalars* sc);

/* Digest of BF16 state: the same sum with the 16-bit words, tags 0, 1, 2. */
uint64_t oracle_state_digest_bf16(const uint16_t* p, const uint16_t* m, const uint16_t* v,
                                  uint64_t n, uint64_t first_index);

/* The committed boundary also has the flat gradients zeroed (Sec. I;
 * Sec. III-C, phase 2): every element of g becomes +0.0. */
void oracle_zero_grad(float* g, uint64_t n);

/* Boundary guard: gradient elements whose 32-bit pattern is not all zero
 * (an outstanding gradient; -0.0 counts). */
uint64_t oracle_count_outstanding(const float* g, uint64_t n);

/* Commit followed by the digest of the committed state: the whole hot path. */
uint64_t oracle_commit_and_digest(float* p, const float* g, float* m, float* v,
                                  uint16_t* bf16, uint64_t n, uint64_t first_index,
                                  const oracle_hyper* h, uint64_t step);

#ifdef __cplusplus
}
#endif

#endif
