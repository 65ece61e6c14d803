/*
 * c_caller.c -- a plain C program that drives libpactshard through its C ABI
 * alone: device memory and a stream from the HIP runtime, no Python, no torch.
 * Test infrastructure (it links the CPU oracle to check the results).
 *
 *   c_caller N GLOBAL_OFFSET STEP SEED
 *
 * Draws a warm shard of N elements (seeded generator), commits it twice on
 * the GPU (steps STEP and STEP+1, a fresh gradient each time), then takes the
 * standalone state digest and the bf16 digest, and compares every output bit
 * for bit with the oracle on the same host arrays.  Also checks that an
 * argument error (step 0) is reported before anything is enqueued and leaves
 * the shard untouched.  Prints one line and exits 0 on agreement, 1 on a
 * mismatch, 2 on a HIP or library error.
 */
#include <hip/hip_runtime_api.h>
#include <inttypes.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "oracle.h"
#include "pactshard.h"

/* workloads/gen.c */
void gen_fill(float* out, uint64_t n, uint64_t first_index, uint64_t seed, uint32_t array_id, uint64_t step,
              int kind, float scale);

/* standard deviation of the generator's centred sum of eight 16-bit uniforms */
#define SUM_SD 53509.98f

#define HIP_CHECK(call)                                                                    \
    do {                                                                                   \
        hipError_t e_ = (call);                                                            \
        if (e_ != hipSuccess) {                                                            \
            fprintf(stderr, "c_caller: %s failed: %s\n", #call, hipGetErrorString(e_));    \
            exit(2);                                                                       \
        }                                                                                  \
    } while (0)

#define PACT_CHECK(call)                                                                   \
    do {                                                                                   \
        int rc_ = (call);                                                                  \
        if (rc_ != PACT_OK) {                                                              \
            fprintf(stderr, "c_caller: %s returned %d (%s)\n", #call, rc_, pact_strerror(rc_)); \
            exit(2);                                                                       \
        }                                                                                  \
    } while (0)

static int same_bits(const void* a, const void* b, size_t bytes, const char* what) {
    if (memcmp(a, b, bytes) != 0) {
        fprintf(stderr, "c_caller: %s differs from the oracle\n", what);
        return 0;
    }
    return 1;
}

int main(int argc, char** argv) {
    if (argc != 5) {
        fprintf(stderr, "usage: c_caller N GLOBAL_OFFSET STEP SEED\n");
        return 2;
    }
    const uint64_t n = strtoull(argv[1], NULL, 10);
    const uint64_t goff = strtoull(argv[2], NULL, 10);
    const uint64_t step0 = strtoull(argv[3], NULL, 10);
    const uint64_t seed = strtoull(argv[4], NULL, 10);
    if (n == 0 || step0 == 0) {
        fprintf(stderr, "c_caller: N and STEP must be positive\n");
        return 2;
    }

    /* host state: a warm shard, the same arrays for both sides */
    float* p = malloc(n * 4);
    float* g = malloc(n * 4);
    float* m = malloc(n * 4);
    float* v = malloc(n * 4);
    float* back = malloc(n * 4);
    uint16_t* bf = malloc(n * 2);
    uint16_t* bf_back = malloc(n * 2);
    if (!p || !g || !m || !v || !back || !bf || !bf_back) {
        fprintf(stderr, "c_caller: out of host memory\n");
        return 2;
    }
    gen_fill(p, n, goff, seed, 0, 0, 0, 0.02f / SUM_SD);
    gen_fill(m, n, goff, seed, 2, 0, 0, 1e-4f / SUM_SD);
    gen_fill(v, n, goff, seed, 3, 0, 1, 1e-7f / SUM_SD);

    /* device state, owned by this program: one pool, the five arrays placed
     * by the library's rule */
    float *dp, *dg, *dm, *dv;
    uint16_t* db;
    uint64_t *dslot, *dbslot;
    void* ws;
    char* pool;
    hipStream_t stream;
    pact_arena_layout plan;
    PACT_CHECK(pact_arena_plan(n, 0, &plan));
    if (plan.offset[1] < n * 4 || plan.offset[4] + n * 2 > plan.pool_bytes || plan.offset[0] != 0) {
        fprintf(stderr, "c_caller: placement plan does not hold the arrays\n");
        return 2;
    }
    HIP_CHECK(hipStreamCreate(&stream));
    HIP_CHECK(hipMalloc((void**)&pool, plan.pool_bytes));
    dp = (float*)(pool + plan.offset[0]);
    dg = (float*)(pool + plan.offset[1]);
    dm = (float*)(pool + plan.offset[2]);
    dv = (float*)(pool + plan.offset[3]);
    db = (uint16_t*)(pool + plan.offset[4]);
    HIP_CHECK(hipMalloc((void**)&dslot, 8));
    HIP_CHECK(hipMalloc((void**)&dbslot, 8));
    HIP_CHECK(hipMemcpy(dp, p, n * 4, hipMemcpyHostToDevice));
    HIP_CHECK(hipMemcpy(dm, m, n * 4, hipMemcpyHostToDevice));
    HIP_CHECK(hipMemcpy(dv, v, n * 4, hipMemcpyHostToDevice));

    pact_shard s;
    memset(&s, 0, sizeof s);
    s.param = dp;
    s.grad = dg;
    s.exp_avg = dm;
    s.exp_avg_sq = dv;
    s.param_bf16 = db;
    s.numel = n;
    s.global_offset = goff;
    s.digest_dev = dslot;
    s.stream = stream;
    const int64_t ws_bytes = pact_workspace_bytes(&s);
    if (ws_bytes <= 0 || pact_digest_slots(&s) != 1) {
        fprintf(stderr, "c_caller: unexpected workspace size or slot count\n");
        return 2;
    }
    HIP_CHECK(hipMalloc(&ws, (size_t)ws_bytes));
    s.workspace = ws;
    s.workspace_bytes = (uint64_t)ws_bytes;

    const pact_hyper hyper = {3e-4f, 0.9f, 0.95f, 1e-8f, 0.1f};
    const oracle_hyper ohyper = {3e-4f, 0.9f, 0.95f, 1e-8f, 0.1f};
    int ok = 1;
    uint64_t d_gpu = 0, d_ref = 0;

    /* an argument error is found before anything is enqueued */
    if (pact_adamw_commit(&s, 0, &hyper) != PACT_EINVAL) {
        fprintf(stderr, "c_caller: step 0 was not rejected\n");
        ok = 0;
    }

    for (uint64_t step = step0; step < step0 + 2 && ok; ++step) {
        gen_fill(g, n, goff, seed, 1, step, 0, 1e-3f / SUM_SD);
        HIP_CHECK(hipMemcpy(dg, g, n * 4, hipMemcpyHostToDevice));
        PACT_CHECK(pact_adamw_commit(&s, step, &hyper));
        HIP_CHECK(hipStreamSynchronize(stream));
        d_ref = oracle_commit_and_digest(p, g, m, v, bf, n, goff, &ohyper, step);
        HIP_CHECK(hipMemcpy(&d_gpu, dslot, 8, hipMemcpyDeviceToHost));
        if (d_gpu != d_ref) {
            fprintf(stderr, "c_caller: step %" PRIu64 " digest 0x%016" PRIx64 ", oracle 0x%016" PRIx64 "\n", step,
                    d_gpu, d_ref);
            ok = 0;
        }
        HIP_CHECK(hipMemcpy(back, dp, n * 4, hipMemcpyDeviceToHost));
        ok &= same_bits(back, p, n * 4, "param");
        HIP_CHECK(hipMemcpy(back, dm, n * 4, hipMemcpyDeviceToHost));
        ok &= same_bits(back, m, n * 4, "exp_avg");
        HIP_CHECK(hipMemcpy(back, dv, n * 4, hipMemcpyDeviceToHost));
        ok &= same_bits(back, v, n * 4, "exp_avg_sq");
        HIP_CHECK(hipMemcpy(bf_back, db, n * 2, hipMemcpyDeviceToHost));
        ok &= same_bits(bf_back, bf, n * 2, "param_bf16");
    }

    /* the standalone digests of the committed state and of the bf16 copy */
    uint64_t d_state = 0, d_bf16 = 0;
    PACT_CHECK(pact_shard_digest(&s));
    PACT_CHECK(pact_bf16_digest(&s, dbslot));
    HIP_CHECK(hipStreamSynchronize(stream));
    HIP_CHECK(hipMemcpy(&d_state, dslot, 8, hipMemcpyDeviceToHost));
    HIP_CHECK(hipMemcpy(&d_bf16, dbslot, 8, hipMemcpyDeviceToHost));
    if (d_state != oracle_state_digest(p, m, v, n, goff)) {
        fprintf(stderr, "c_caller: state digest differs from the oracle\n");
        ok = 0;
    }
    if (d_bf16 != oracle_bf16_digest(bf, n, goff)) {
        fprintf(stderr, "c_caller: bf16 digest differs from the oracle\n");
        ok = 0;
    }

    HIP_CHECK(hipFree(ws));
    HIP_CHECK(hipFree(dbslot));
    HIP_CHECK(hipFree(dslot));
    HIP_CHECK(hipFree(pool));
    HIP_CHECK(hipStreamDestroy(stream));
    free(p);
    free(g);
    free(m);
    free(v);
    free(back);
    free(bf);
    free(bf_back);

    printf("c_caller %s: n=%" PRIu64 " offset=%" PRIu64 " steps=%" PRIu64 "..%" PRIu64
           " digest=0x%016" PRIx64 " bf16_digest=0x%016" PRIx64 "\n",
           ok ? "ok" : "MISMATCH", n, goff, step0, step0 + 1, d_state, d_bf16);
    return ok ? 0 : 1;
}
