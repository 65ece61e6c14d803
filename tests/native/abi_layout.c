/* Prints the size and field offsets of every struct in pactshard.h as JSON,
 * compiled as strict C99: the header must be plain C, and the Python
 * binding's ctypes mirrors must agree with it field for field. */
#include <stddef.h>
#include <stdio.h>

#include "pactshard.h"

#define F(T, f) printf("%s\"%s\": %zu", first ? "" : ", ", #f, offsetof(T, f)), first = 0
#define OPEN(T) printf("%s\"%s\": {\"sizeof\": %zu, \"fields\": {", nstruct++ ? ", " : "", #T, sizeof(T)), first = 1
#define CLOSE() printf("}}")

int main(void) {
    int first = 1, nstruct = 0;
    printf("{");
    OPEN(pact_hyper);
    F(pact_hyper, lr); F(pact_hyper, beta1); F(pact_hyper, beta2); F(pact_hyper, eps);
    F(pact_hyper, weight_decay);
    CLOSE();
    OPEN(pact_segment);
    F(pact_segment, offset); F(pact_segment, length); F(pact_segment, hyper_index); F(pact_segment, reserved);
    CLOSE();
    OPEN(pact_shard);
    F(pact_shard, param); F(pact_shard, grad); F(pact_shard, exp_avg); F(pact_shard, exp_avg_sq);
    F(pact_shard, param_bf16); F(pact_shard, numel); F(pact_shard, global_offset); F(pact_shard, segs);
    F(pact_shard, num_segs); F(pact_shard, num_hypers); F(pact_shard, hypers); F(pact_shard, digest_dev);
    F(pact_shard, workspace); F(pact_shard, workspace_bytes); F(pact_shard, stream);
    CLOSE();
    OPEN(pact_shard_bf16);
    F(pact_shard_bf16, param); F(pact_shard_bf16, grad); F(pact_shard_bf16, exp_avg); F(pact_shard_bf16, exp_avg_sq);
    F(pact_shard_bf16, numel); F(pact_shard_bf16, global_offset); F(pact_shard_bf16, segs);
    F(pact_shard_bf16, num_segs); F(pact_shard_bf16, num_hypers); F(pact_shard_bf16, hypers);
    F(pact_shard_bf16, digest_dev); F(pact_shard_bf16, workspace); F(pact_shard_bf16, workspace_bytes);
    F(pact_shard_bf16, stream);
    CLOSE();
    OPEN(pact_arena_layout);
    F(pact_arena_layout, pool_bytes); F(pact_arena_layout, spacing); F(pact_arena_layout, offset);
    CLOSE();
    printf(", \"codes\": {\"PACT_ARENA_SPACING\": %llu, \"PACT_ARENA_PACK_BELOW\": %llu, ",
           (unsigned long long)PACT_ARENA_SPACING, (unsigned long long)PACT_ARENA_PACK_BELOW);
    printf("\"PACT_OK\": %d, \"PACT_EINVAL\": %d, \"PACT_EALIGN\": %d, \"PACT_EOVERLAP\": %d, "
           "\"PACT_ERANGE\": %d, \"PACT_EHIP\": %d, \"PACT_ESCRATCH\": %d, \"PACT_COMMIT_ZERO_GRAD\": %u, "
           "\"PACT_COMMIT_WORKSPACE_CLEAN\": %u, \"PACT_STATIC_MAX_SEGMENTS\": %d}}\n",
           PACT_OK, PACT_EINVAL, PACT_EALIGN, PACT_EOVERLAP, PACT_ERANGE, PACT_EHIP, PACT_ESCRATCH,
           PACT_COMMIT_ZERO_GRAD, PACT_COMMIT_WORKSPACE_CLEAN, PACT_STATIC_MAX_SEGMENTS);
    return 0;
}
