/*
 * pactshard.h -- C ABI of libpactshard: the per-rank sharded AdamW commit and
 * the 64-bit state digest, for AMD Instinct MI355X (gfx950).
 *
 * What the calls compute.  The preserved training state of a rank is its
 * shard of the weights W, the AdamW moments M and V, and the optimizer step
 * counter (Sec. III-A, eq. 2).  In-memory recovery keeps that state in device
 * memory once the optimizer update has committed (Sec. I; Sec. III-A, action
 * L1), and every rank must then hold it bit-identically (abstract; Sec. IV-G).
 * pact_adamw_commit applies that update to one flat shard; pact_shard_digest
 * names the committed state in 64 bits so ranks can compare it cheaply.
 *
 * Arithmetic (the paper prints no formula; this is the library's contract).
 * Per call, per segment, in double and rounded once to binary32:
 *   decay = 1 - lr*wd, omb1 = 1 - beta1, omb2 = 1 - beta2,
 *   step_size = lr / (1 - beta1^t), rs_bc2 = 1 / sqrt(1 - beta2^t),
 * with beta^t formed by t successive double multiplications.  Per element,
 * each operation one binary32 round-to-nearest-even, no fused multiply-add:
 *   p1 = p*decay;  m' = beta1*m + omb1*g;  v' = beta2*v + omb2*(g*g);
 *   den = sqrt(v')*rs_bc2 + eps;  p' = p1 - step_size*(m'/den)
 * with IEEE-correct sqrt and division and fp32 denormals kept.  The bf16 copy
 * is round-to-nearest-even of p' (NaN: quiet, sign and top payload kept).
 *
 * Digest.  D = sum over k in {0:p', 1:m', 2:v'} and shard elements i of
 *   splitmix64( zext64(bits32(X_k[i])) XOR ((global_offset + i) | k << 56) )
 * mod 2^64, where splitmix64(x) is the generator output for state x (add the
 * golden gamma 0x9E3779B97F4A7C15, then the standard 30/27/31 mix).  The sum
 * wraps, so D does not depend on how the index range is partitioned: digests
 * of disjoint shards, segments or ranks add up to the digest of their union.
 * The bf16 digest uses tag k = 3 on the zero-extended 16-bit words.
 *
 * Memory and ownership.  Every buffer belongs to the caller; the library
 * allocates nothing.  All array pointers are device pointers (HBM).
 * param, exp_avg, exp_avg_sq are read and overwritten in place; grad is
 * read (and overwritten with +0.0 only by a commit asked to zero it);
 * param_bf16 is only written.  The five arrays must not overlap each
 * other or digest_dev.  fp32 arrays need 4-byte and bf16 2-byte alignment;
 * a segment whose start is 16-byte aligned in all four fp32 arrays and 8-byte
 * aligned in the bf16 array runs the vector path, any other segment the
 * element-wise path, with identical results.
 *
 * Segments (at most 2^24).  segs == NULL: the shard is one segment [0, numel) updated with
 * *hyper, and digest_dev[0] receives D.  Otherwise segs[0..num_segs) lists
 * disjoint ranges (offset, length, hyper_index) in increasing offset order
 * inside [0, numel); elements outside every segment (padding) are neither
 * read, written nor digested; hypers[hyper_index] applies per segment and
 * `hyper` is ignored; digest_dev[0..num_segs) receive the per-segment digests
 * and digest_dev[num_segs] their sum.  pact_digest_slots() gives the count.
 *
 * Workspace.  Optional caller-owned device scratch for the digest's partial
 * sums; see pact_workspace_bytes().
 *
 * Streams and completion.  Every call only enqueues work on `stream` (a
 * hipStream_t; NULL is the default stream) and returns; the digest slots
 * hold their value once the stream has reached that point.  Calls on one
 * stream are ordered; concurrent calls on different streams must not touch
 * the same buffers.  A call enqueues kernel launches only (no memset, no
 * allocation, no host synchronisation), so it can be captured into a HIP
 * graph; pointers, segment table, step and hyperparameters are taken at call
 * time, so every replay of such a graph repeats the captured step on the
 * same buffers.
 *
 * Errors.  0 on success, a negative PACT_E* code otherwise.  Argument errors
 * are found before anything is enqueued and leave every buffer untouched.
 * PACT_EHIP means a launch failed after validation: the shard may be partly
 * updated and must be treated as uncommitted (the caller falls back to
 * restart from a checkpoint, the paper's L2 action, Sec. III-A).
 */
#ifndef PACTSHARD_H
#define PACTSHARD_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define PACT_OK 0
#define PACT_EINVAL (-1)   /* null pointer, bad size, bad hyperparameter or segment table, step == 0 */
#define PACT_EALIGN (-2)   /* misaligned pointer */
#define PACT_EOVERLAP (-3) /* two buffers overlap */
#define PACT_ERANGE (-4)   /* an index reaches 2^56 (the tag bits): global_offset + numel > 2^56; or the
                            * shard needs more than 2^24 - 1 tiles of 4096 elements (one launch grid) */
#define PACT_EHIP (-5)     /* a HIP call failed; see pact_last_hip_error() */
#define PACT_ESCRATCH (-6) /* pact_adamw_commit_static: more segments than its static scratch holds */

/* AdamW hyperparameters.  Valid: lr >= 0, 0 <= beta1 < 1, 0 <= beta2 < 1,
 * eps > 0, weight_decay >= 0, all finite. */
typedef struct pact_hyper {
    float lr;
    float beta1;
    float beta2;
    float eps;
    float weight_decay;
} pact_hyper;

/* One tensor of a multi-tensor flat shard, in shard elements. */
typedef struct pact_segment {
    uint64_t offset;
    uint64_t length;
    uint32_t hyper_index;
    uint32_t reserved; /* must be 0 */
} pact_segment;

/* One rank's flat shard.  Host struct; array pointers are device pointers,
 * segs and hypers are host pointers read during the call only. */
typedef struct pact_shard {
    float* param;            /* W: fp32 master weights, numel elements          */
    float* grad;             /* fp32 gradient, numel elements; written only by  */
                             /* PACT_COMMIT_ZERO_GRAD, read-only otherwise      */
    float* exp_avg;          /* M: fp32 first moment                            */
    float* exp_avg_sq;       /* V: fp32 second moment                           */
    uint16_t* param_bf16;    /* bf16 working copy of W (bit patterns)           */
    uint64_t numel;          /* elements in the shard, padding included         */
    uint64_t global_offset;  /* flat index of element 0 in the full vector      */
    const pact_segment* segs;/* NULL or num_segs entries                        */
    uint32_t num_segs;
    uint32_t num_hypers;
    const pact_hyper* hypers;/* num_hypers entries when segs != NULL            */
    uint64_t* digest_dev;    /* device, pact_digest_slots() uint64 slots        */
    void* workspace;         /* device scratch or NULL, see pact_workspace_bytes */
    uint64_t workspace_bytes;/* size of workspace in bytes                      */
    void* stream;            /* hipStream_t                                     */
} pact_shard;

/* Number of uint64 digest slots a call on this shard writes: 1 without
 * segments, num_segs + 1 with them; negative error code if s is NULL. */
int64_t pact_digest_slots(const pact_shard* s);

/* Bytes of device workspace that lets a call spread its digest partial sums
 * over several memory locations (16 lanes, 256 bytes apart, per digest slot)
 * instead of funnelling one 64-bit atomic per 4096-element tile into a single
 * address, which serializes on large shards.  The caller allocates it (8-byte
 * aligned, disjoint from every other buffer) and may reuse it for any later
 * call on the same stream.  Its contents on entry do not matter (the call
 * clears the part it uses first, unless told with PACT_COMMIT_WORKSPACE_CLEAN
 * that it is clear already), and every call that returns PACT_OK leaves that
 * part zero again once the stream has run it.  workspace == NULL is valid:
 * the call is then correct but slower.  A non-NULL workspace with
 * workspace_bytes below this figure is PACT_EINVAL.  Negative error code if s
 * is NULL. */
int64_t pact_workspace_bytes(const pact_shard* s);

/* The fused commit (Sec. III-A: the update after which W, M, V count as
 * committed): reads p, g, m, v once, writes p', m', v' in place and the bf16
 * copy, and accumulates the digest of (p', m', v') in the same pass.
 * step = the optimizer step t >= 1 after its increment. */
int pact_adamw_commit(const pact_shard* s, uint64_t step, const pact_hyper* hyper);

/* Options of pact_adamw_commit_ex. */
#define PACT_COMMIT_ZERO_GRAD 1u       /* the same pass writes +0.0 into every committed grad element */
#define PACT_COMMIT_WORKSPACE_CLEAN 2u /* the workspace is already clear: skip clearing it */

/* The commit with options; flags = 0 is exactly pact_adamw_commit.
 * PACT_COMMIT_ZERO_GRAD: after reading g, the same pass writes +0.0 into
 * every committed element of `grad` (4 more bytes per element, 34 in all),
 * so that one call leaves the shard at the boundary the paper admits for
 * in-memory recovery: update committed and flat gradients zeroed (Sec. I;
 * Sec. III-C, phase 2).  `grad` must then be writable device memory.
 * PACT_COMMIT_WORKSPACE_CLEAN: the caller vouches that the workspace is clear
 * (zero-filled before its first use, and touched since then only by calls on
 * this stream that returned PACT_OK), so the call skips the launch that
 * clears it; a workspace in any other state gives a wrong digest.  Without a
 * workspace the flag has no effect.  Unknown flag bits are PACT_EINVAL. */
int pact_adamw_commit_ex(const pact_shard* s, uint64_t step, const pact_hyper* hyper, uint32_t flags);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * pact_adamw_commit_ex with the digest partial sums kept in a static device
 * array inside the library instead of a caller workspace.  The array holds
 * the lanes of at most PACT_STATIC_MAX_SEGMENTS result slots (2 MiB); each
 * GPU the library runs on holds its own copy until the process ends.
 * Inputs and outputs are the caller's, as for pact_adamw_commit_ex;
 * s->workspace must be NULL.  flags: 0 or PACT_COMMIT_ZERO_GRAD.  A shard
 * with more than PACT_STATIC_MAX_SEGMENTS segments is PACT_ESCRATCH, found
 * before anything is enqueued.  The call allocates nothing and calls no
 * allocating routine; the first call on a device looks up the address of
 * that device's copy (hipGetSymbolAddress, on the device of `stream`), so
 * a caller that captures should make one call on each device beforehand.
 * Every call on a GPU shares that GPU's array: each call clears the part it
 * uses with a kernel before its tiles run, and calls that overlap in time
 * on one GPU (concurrent streams, or host threads) race and give wrong
 * digests. */
#define PACT_STATIC_MAX_SEGMENTS 512
int pact_adamw_commit_static(const pact_shard* s, uint64_t step, const pact_hyper* hyper, uint32_t flags);

/* Boundary guard for zero outstanding gradients (Sec. III-C, phase 2):
 * counts the elements of `grad` whose 32-bit pattern is not all zero (-0.0
 * counts as outstanding), per segment and in total, into dev_out
 * (pact_digest_slots() uint64 slots, device memory).  param, exp_avg,
 * exp_avg_sq and param_bf16 are not read and may be NULL. */
int pact_grad_guard(const pact_shard* s, uint64_t* dev_out);

/* Digest of the current (p, m, v) without updating them (the bitwise state
 * check of Sec. IV-G, as a 64-bit identity).  grad and param_bf16 are not
 * read and may be NULL. */
int pact_shard_digest(const pact_shard* s);

/* Digest (tag 3) of the bf16 copy into dev_out (pact_digest_slots() slots,
 * device memory); param, grad, exp_avg, exp_avg_sq are not read and may be
 * NULL.  A verification aid: the bf16 copy is a function of p'. */
int pact_bf16_digest(const pact_shard* s, uint64_t* dev_out);

/* One rank's flat shard held in BF16, the paper's own precision for weights
 * and AdamW moments (Sec. IV-A): the fields of pact_shard with 16-bit
 * arrays (bf16 bit patterns) and no separate working copy.  fp32 rules apply
 * with 2-byte alignment; a segment whose start is 16-byte aligned in all four
 * arrays runs the vector path. */
typedef struct pact_shard_bf16 {
    uint16_t* param;          /* W, bf16, numel elements                       */
    const uint16_t* grad;     /* bf16 gradient                                 */
    uint16_t* exp_avg;        /* M, bf16                                       */
    uint16_t* exp_avg_sq;     /* V, bf16                                       */
    uint64_t numel;
    uint64_t global_offset;
    const pact_segment* segs;
    uint32_t num_segs;
    uint32_t num_hypers;
    const pact_hyper* hypers;
    uint64_t* digest_dev;
    void* workspace;
    uint64_t workspace_bytes;
    void* stream;
} pact_shard_bf16;

/* The commit on BF16 state: each bf16 word of p, g, m, v is widened exactly
 * to binary32, the binary32 update above is applied unchanged, and p', m',
 * v' are rounded back to bf16 (round to nearest even), in place.  Reads 8 and
 * writes 6 bytes per element; the digest of (p', m', v') uses the 16-bit
 * words zero-extended, with the same indices and tags 0, 1, 2. */
int pact_adamw_commit_bf16(const pact_shard_bf16* s, uint64_t step, const pact_hyper* hyper);

/* Digest of the current BF16 (p, m, v); grad is not read and may be NULL. */
int pact_shard_digest_bf16(const pact_shard_bf16* s);

/* Slot count and workspace size for a BF16 shard (as for pact_shard). */
int64_t pact_digest_slots_bf16(const pact_shard_bf16* s);
int64_t pact_workspace_bytes_bf16(const pact_shard_bf16* s);

/* Placement of one shard's five arrays in one device pool.  On MI355X the
 * commit's eight concurrent streams (reads of p, g, m, v; writes of p', m',
 * v' and the bf16 copy) reach about 6.4-6.5 TB/s (80-81% of the 8 TB/s
 * peak) when the arrays sit in separate regions of HBM some tens of GB
 * apart, and about 5.6-5.7 TB/s (70-71%) when they sit within a few GB of
 * each other -- the case of five back-to-back allocations.  The kernels are
 * the same; the difference is the memory system's.  pact_arena_plan gives
 * the library's placement rule as byte offsets into one pool the caller
 * allocates (one hipMalloc of pool_bytes, 2 MiB aligned):
 *   fp32 array k (0 param, 1 grad, 2 exp_avg, 3 exp_avg_sq) at k * spacing,
 *   the bf16 copy at 4 * spacing, pool_bytes = 4 * spacing + its size;
 * spacing = the requested one (at least one fp32 array, rounded up to
 * 2 MiB), or with spacing == 0 the default: PACT_ARENA_SPACING when the
 * five arrays together exceed PACT_ARENA_PACK_BELOW bytes, else the arrays
 * back to back (a shard that small stays in the 256 MB on-chip cache and
 * placement does not matter).  With the default spacing the pool reserves
 * about 176 GiB for any shard above that size; the gaps after each fp32
 * array (offset[k] + array bytes .. offset[k+1]) hold nothing of the shard
 * and are free for the caller's other buffers.  Pure host arithmetic: no HIP
 * call, no allocation.  PACT_EINVAL if out is NULL, PACT_ERANGE if the pool
 * does not fit 64 bits. */
#define PACT_ARENA_SPACING (44ull << 30)
#define PACT_ARENA_PACK_BELOW (512ull << 20)
typedef struct pact_arena_layout {
    uint64_t pool_bytes;  /* bytes to allocate for the pool                        */
    uint64_t spacing;     /* bytes between the starts of consecutive fp32 arrays    */
    uint64_t offset[5];   /* byte offsets of param, grad, exp_avg, exp_avg_sq, bf16 */
} pact_arena_layout;
int pact_arena_plan(uint64_t numel, uint64_t spacing, pact_arena_layout* out);

/* Measurement support, not part of the commit: streams the same bytes as a
 * commit (reads 4 fp32 arrays, writes 3 fp32 arrays and one 16-bit array,
 * 30 bytes per element) with no arithmetic beyond one add, so its rate is
 * the practical HBM ceiling of that access pattern.  out_* may alias in_*
 * element for element (in-place), as in a commit. */
int pact_stream_probe(const float* in0, const float* in1, const float* in2, const float* in3,
                      float* out0, float* out2, float* out3, uint16_t* out_half,
                      uint64_t n, void* stream);

/* The same probe from a persistent grid of `workgroups` workgroups of 256
 * threads, each striding over the 4096-element tiles (workgroups == 0: one
 * workgroup per tile, exactly pact_stream_probe).  Measurement support: it
 * compares the grid-stride launch shape with the one the kernels use. */
int pact_stream_probe_grid(const float* in0, const float* in1, const float* in2, const float* in3,
                           float* out0, float* out2, float* out3, uint16_t* out_half,
                           uint64_t n, uint32_t workgroups, void* stream);

/* Static text for a PACT_E* code. */
const char* pact_strerror(int code);

/* The hipError_t of the last failed HIP call on this thread (0 if none). */
int pact_last_hip_error(void);

/* Library version, major * 10000 + minor * 100 + patch. */
int pact_version(void);

#ifdef __cplusplus
}
#endif

#endif /* PACTSHARD_H */
