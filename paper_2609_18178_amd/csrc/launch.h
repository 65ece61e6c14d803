// launch.h -- internal interface between the host validation layer
// (pactshard.hip) and the gfx950 kernels (kernels.hip).  Not installed.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pact {

// Segments handled by one kernel launch; longer tables take several launches.
// The batch travels in the kernel-argument segment (about 2 KB), so no device
// table has to be allocated or copied.
constexpr int kSegsPerLaunch = 32;

// Threads per workgroup (4 waves of 64) and fp32 elements one thread moves
// per tile: four 16-byte vectors per array.
constexpr int kBlock = 256;
constexpr int kVec = 4;
constexpr int kUnroll = 4;
constexpr int kTile = kBlock * kVec * kUnroll;  // 4096 elements per tile

// Digest partial sums: each result slot owns kLanes workspace words,
// kLaneStride words (256 bytes) apart; workgroup w adds into lane w % kLanes.
constexpr int kLanes = 16;
constexpr int kLaneStride = 32;

// Per-segment binary32 scalars of one step.
struct StepScalars {
    float beta1, beta2, eps, decay, omb1, omb2, step_size, rs_bc2;
};

// One launch's slice of the segment table.  Tiles never straddle segments:
// segment s owns tiles [tile_begin[s], tile_begin[s+1]).
struct Batch {
    uint32_t nseg;
    uint32_t slot0;        // result slot of this batch's first segment
    uint32_t per_segment;  // nonzero: one result slot per segment, else one in all
    uint64_t tile_begin[kSegsPerLaunch + 1];
    uint64_t elem_begin[kSegsPerLaunch];  // shard-relative first element
    uint64_t elem_count[kSegsPerLaunch];
    uint32_t vec_ok[kSegsPerLaunch];      // 16-B (fp32) / 8-B (bf16) aligned start
    StepScalars sc[kSegsPerLaunch];
};

struct Arrays {
    float* p;
    const float* g;
    float* g_zero;      // the grad array, written only by Mode::CommitZeroGrad
    float* m;
    float* v;
    uint16_t* b;
    uint64_t goff;      // global flat index of shard element 0
    uint64_t* digest;   // result slots
    uint64_t* lanes;    // workspace lanes, or null: atomics go to the result slots
};

// The same arrays for a shard held in BF16 (no separate working copy).
struct ArraysBf16 {
    uint16_t* p;
    const uint16_t* g;
    uint16_t* m;
    uint16_t* v;
    uint64_t goff;
    uint64_t* digest;
    uint64_t* lanes;
};

enum class Mode : int {
    Commit = 0,
    StateDigest = 1,
    Bf16Digest = 2,
    CommitZeroGrad = 3,
    GradGuard = 4,
    CommitBf16State = 5,
    DigestBf16State = 6,
};

// Enqueue the clearing of what the tile kernels accumulate into: the
// nres * kLanes lane words when `lanes` is given, else the nslots digest slots.
hipError_t launch_clear(uint64_t* digest, uint64_t* lanes, uint32_t nres, uint32_t nslots, hipStream_t stream);

// Enqueue one batch in the given mode: one workgroup per tile, so `grid` is
// the batch's tile count.
hipError_t launch_batch(Mode mode, const Arrays& a, const Batch& b, uint32_t grid, hipStream_t stream);

// Enqueue one batch of a BF16-state mode (CommitBf16State, DigestBf16State).
hipError_t launch_batch_bf16(Mode mode, const ArraysBf16& a, const Batch& b, uint32_t grid, hipStream_t stream);

// Enqueue the final sums: digest[r] = sum of r's lanes (when `lanes` is
// given) for r < nres, and, with per-segment results, digest[nres] = their sum.
hipError_t launch_finish(uint64_t* digest, uint64_t* lanes, uint32_t nres, bool per_segment, hipStream_t stream);

// Enqueue the 30-byte/element stream probe (n a multiple of kVec): one
// workgroup per tile when workgroups == 0, else a persistent grid of that
// many workgroups striding over the tiles.
hipError_t launch_probe(const float* i0, const float* i1, const float* i2, const float* i3,
                        float* o0, float* o2, float* o3, uint16_t* oh, uint64_t n, uint32_t workgroups,
                        hipStream_t stream);

}  // namespace pact
