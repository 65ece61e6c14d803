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
// per tile: two 16-byte vectors per array.
constexpr int kBlock = 256;
constexpr int kVec = 4;
constexpr int kUnroll = 2;
constexpr int kTile = kBlock * kVec * kUnroll;  // 2048 elements per tile

// Per-segment binary32 scalars of one step.
struct StepScalars {
    float beta1, beta2, eps, decay, omb1, omb2, step_size, rs_bc2;
};

// One launch's slice of the segment table.  Tiles never straddle segments:
// segment s owns tiles [tile_begin[s], tile_begin[s+1]).
struct Batch {
    uint32_t nseg;
    uint32_t slot0;        // digest slot of this batch's first segment
    uint32_t total_slot;   // slot of the sum over all segments
    uint32_t per_segment;  // nonzero: also write per-segment slots
    uint64_t tile_begin[kSegsPerLaunch + 1];
    uint64_t elem_begin[kSegsPerLaunch];  // shard-relative first element
    uint64_t elem_count[kSegsPerLaunch];
    uint32_t vec_ok[kSegsPerLaunch];      // 16-B (fp32) / 8-B (bf16) aligned start
    StepScalars sc[kSegsPerLaunch];
};

struct Arrays {
    float* p;
    const float* g;
    float* m;
    float* v;
    uint16_t* b;
    uint64_t goff;      // global flat index of shard element 0
    uint64_t* digest;   // slots
};

enum class Mode : int { Commit = 0, StateDigest = 1, Bf16Digest = 2 };

// Enqueue: zero `nslots` digest slots.
hipError_t launch_zero(uint64_t* slots, uint32_t nslots, hipStream_t stream);

// Enqueue one batch in the given mode on `grid` workgroups.
hipError_t launch_batch(Mode mode, const Arrays& a, const Batch& b, uint32_t grid, hipStream_t stream);

// Enqueue the 30-byte/element stream probe.
hipError_t launch_probe(const float* i0, const float* i1, const float* i2, const float* i3,
                        float* o0, float* o2, float* o3, uint16_t* oh, uint64_t n,
                        uint32_t grid, hipStream_t stream);

}  // namespace pact
