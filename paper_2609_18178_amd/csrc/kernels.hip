// kernels.hip -- gfx950 kernels of libpactshard.
//
// One persistent, grid-stride kernel serves the three modes (commit, state
// digest, bf16 digest).  Work is cut into tiles of kTile elements that never
// straddle a segment; workgroup w takes tiles w, w + grid, w + 2*grid, ... so
// at any moment the whole chip streams one contiguous window of each array.
// A full, aligned tile moves two 16-byte vectors per array per thread
// (global_load_dwordx4 / global_store_dwordx4, bf16 as dwordx2); a ragged
// tail or a misaligned segment goes element by element.
//
// The digest is accumulated per thread in a 64-bit register (wrapping add),
// reduced across the wave with shuffles and across the workgroup's four
// waves through LDS, and added to the caller's slot with one 64-bit atomic
// per workgroup (per segment when per-segment digests are asked for).
// Wrapping addition is associative and commutative, so the order in which
// workgroups arrive cannot change the result.
//
// Arithmetic is the library contract in pactshard.h: one IEEE binary32
// rounding per operation, no contraction or reassociation (the translation
// unit is built with -ffp-contract=off and without fast-math), correctly
// rounded sqrt and division, fp32 denormals kept.
#include "launch.h"

// No fused multiply-add anywhere in this file, whatever the command line says.
#pragma clang fp contract(off)

namespace pact {
namespace {

// ---------------------------------------------------------------------------
// digest word hash: splitmix64 generator output for state x
// ---------------------------------------------------------------------------
constexpr uint64_t kGamma = 0x9E3779B97F4A7C15ull;
constexpr uint64_t kMul1 = 0xBF58476D1CE4E5B9ull;
constexpr uint64_t kMul2 = 0x94D049BB133111EBull;
constexpr uint64_t kTagM = 1ull << 56;
constexpr uint64_t kTagV = 2ull << 56;
constexpr uint64_t kTagB = 3ull << 56;

__device__ __forceinline__ uint64_t hash_word(uint32_t word, uint64_t tagged_index) {
    uint64_t z = ((uint64_t)word ^ tagged_index) + kGamma;
    z = (z ^ (z >> 30)) * kMul1;
    z = (z ^ (z >> 27)) * kMul2;
    return z ^ (z >> 31);
}

// ---------------------------------------------------------------------------
// AdamW on one element, in the contract's order.  With -ffp-contract=off and
// no fast-math flags every +, -, * below is one IEEE binary32 operation
// rounded to nearest even, '/' is the correctly rounded division, and
// __builtin_sqrtf is lowered to the correctly rounded square root (the
// -fhip-fp32-correctly-rounded-divide-sqrt default).  HIP's __fsqrt_rn is
// NOT used: unless OCML_BASIC_ROUNDED_OPERATIONS is defined it maps to the
// hardware's approximate v_sqrt_f32.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void adamw(float& p, float g, float& m, float& v, const StepScalars& s) {
    const float p_dec = p * s.decay;
    const float m_keep = s.beta1 * m;
    const float m_push = s.omb1 * g;
    const float m_new = m_keep + m_push;
    const float g_sq = g * g;
    const float v_keep = s.beta2 * v;
    const float v_push = s.omb2 * g_sq;
    const float v_new = v_keep + v_push;
    const float root = __builtin_sqrtf(v_new);
    const float den = root * s.rs_bc2 + s.eps;
    const float ratio = m_new / den;
    const float step = s.step_size * ratio;
    p = p_dec - step;
    m = m_new;
    v = v_new;
}

// binary32 -> bfloat16, round to nearest even; NaN stays a quiet NaN.
__device__ __forceinline__ uint32_t to_bf16(float x) {
    const uint32_t u = __float_as_uint(x);
    const uint32_t rounded = (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
    return ((u & 0x7FFFFFFFu) > 0x7F800000u) ? ((u >> 16) | 0x0040u) : rounded;
}

// ---------------------------------------------------------------------------
// workgroup sum of a 64-bit value; result valid in thread 0
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint64_t block_sum(uint64_t x, uint64_t* lds) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        x += __shfl_xor(x, off, 64);
    }
    const int wave = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) {
        lds[wave] = x;
    }
    __syncthreads();
    uint64_t r = 0;
    if (threadIdx.x == 0) {
#pragma unroll
        for (int w = 0; w < kBlock / 64; ++w) {
            r += lds[w];
        }
    }
    __syncthreads();
    return r;
}

// ---------------------------------------------------------------------------
// one element, element-wise path
// ---------------------------------------------------------------------------
template <Mode M>
__device__ __forceinline__ uint64_t do_scalar(const Arrays& a, uint64_t e, const StepScalars& sc) {
    const uint64_t idx = a.goff + e;
    if constexpr (M == Mode::Bf16Digest) {
        return hash_word(a.b[e], idx | kTagB);
    } else {
        float p = a.p[e];
        float m = a.m[e];
        float v = a.v[e];
        if constexpr (M == Mode::Commit) {
            adamw(p, a.g[e], m, v, sc);
            a.p[e] = p;
            a.m[e] = m;
            a.v[e] = v;
            a.b[e] = (uint16_t)to_bf16(p);
        }
        return hash_word(__float_as_uint(p), idx) + hash_word(__float_as_uint(m), idx | kTagM) +
               hash_word(__float_as_uint(v), idx | kTagV);
    }
}

// ---------------------------------------------------------------------------
// one full aligned tile, vector path: kUnroll x 16-byte vectors per array
// ---------------------------------------------------------------------------
template <Mode M>
__device__ __forceinline__ uint64_t do_tile_vec(const Arrays& a, uint64_t e0, const StepScalars& sc) {
    uint64_t acc = 0;
    if constexpr (M == Mode::Bf16Digest) {
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const uint64_t e = e0 + (uint64_t)(u * kBlock * kVec) + threadIdx.x * kVec;
            const uint2 w = *reinterpret_cast<const uint2*>(a.b + e);
            const uint64_t idx = a.goff + e;
            acc += hash_word(w.x & 0xFFFFu, idx | kTagB) + hash_word(w.x >> 16, (idx + 1) | kTagB) +
                   hash_word(w.y & 0xFFFFu, (idx + 2) | kTagB) + hash_word(w.y >> 16, (idx + 3) | kTagB);
        }
        return acc;
    } else {
        float4 P[kUnroll], G[kUnroll], Mo[kUnroll], V[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const uint64_t e = e0 + (uint64_t)(u * kBlock * kVec) + threadIdx.x * kVec;
            P[u] = *reinterpret_cast<const float4*>(a.p + e);
            Mo[u] = *reinterpret_cast<const float4*>(a.m + e);
            V[u] = *reinterpret_cast<const float4*>(a.v + e);
            if constexpr (M == Mode::Commit) {
                G[u] = *reinterpret_cast<const float4*>(a.g + e);
            }
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const uint64_t e = e0 + (uint64_t)(u * kBlock * kVec) + threadIdx.x * kVec;
            if constexpr (M == Mode::Commit) {
                adamw(P[u].x, G[u].x, Mo[u].x, V[u].x, sc);
                adamw(P[u].y, G[u].y, Mo[u].y, V[u].y, sc);
                adamw(P[u].z, G[u].z, Mo[u].z, V[u].z, sc);
                adamw(P[u].w, G[u].w, Mo[u].w, V[u].w, sc);
                *reinterpret_cast<float4*>(a.p + e) = P[u];
                *reinterpret_cast<float4*>(a.m + e) = Mo[u];
                *reinterpret_cast<float4*>(a.v + e) = V[u];
                uint2 h;
                h.x = to_bf16(P[u].x) | (to_bf16(P[u].y) << 16);
                h.y = to_bf16(P[u].z) | (to_bf16(P[u].w) << 16);
                *reinterpret_cast<uint2*>(a.b + e) = h;
            }
            const uint64_t idx = a.goff + e;
            const float pv[4] = {P[u].x, P[u].y, P[u].z, P[u].w};
            const float mv[4] = {Mo[u].x, Mo[u].y, Mo[u].z, Mo[u].w};
            const float vv[4] = {V[u].x, V[u].y, V[u].z, V[u].w};
#pragma unroll
            for (int j = 0; j < kVec; ++j) {
                const uint64_t i = idx + j;
                acc += hash_word(__float_as_uint(pv[j]), i) + hash_word(__float_as_uint(mv[j]), i | kTagM) +
                       hash_word(__float_as_uint(vv[j]), i | kTagV);
            }
        }
        return acc;
    }
}

template <Mode M>
__global__ __launch_bounds__(kBlock) void shard_kernel(Arrays a, Batch bt) {
    __shared__ uint64_t lds[kBlock / 64];
    const uint64_t ntiles = bt.tile_begin[bt.nseg];
    uint32_t seg = 0;
    uint64_t seg_acc = 0;  // this thread's share of the current segment
    uint64_t all_acc = 0;  // this thread's share of the launch's segments

    for (uint64_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
        // tile and seg are uniform across the workgroup
        while (tile >= bt.tile_begin[seg + 1]) {
            if (bt.per_segment) {
                const uint64_t s = block_sum(seg_acc, lds);
                if (threadIdx.x == 0 && s != 0) {
                    atomicAdd(reinterpret_cast<unsigned long long*>(a.digest + bt.slot0 + seg),
                              (unsigned long long)s);
                }
            }
            all_acc += seg_acc;
            seg_acc = 0;
            ++seg;
        }
        const StepScalars sc = bt.sc[seg];
        const uint64_t seg_first = bt.elem_begin[seg];
        const uint64_t seg_end = seg_first + bt.elem_count[seg];
        const uint64_t e0 = seg_first + (tile - bt.tile_begin[seg]) * (uint64_t)kTile;
        if (bt.vec_ok[seg] && e0 + kTile <= seg_end) {
            seg_acc += do_tile_vec<M>(a, e0, sc);
        } else {
            const uint64_t e1 = (e0 + kTile < seg_end) ? e0 + kTile : seg_end;
            for (uint64_t e = e0 + threadIdx.x; e < e1; e += kBlock) {
                seg_acc += do_scalar<M>(a, e, sc);
            }
        }
    }
    // flush the last segment this workgroup touched and the launch total
    if (bt.per_segment) {
        const uint64_t s = block_sum(seg_acc, lds);
        if (threadIdx.x == 0 && s != 0) {
            atomicAdd(reinterpret_cast<unsigned long long*>(a.digest + bt.slot0 + seg), (unsigned long long)s);
        }
    }
    all_acc += seg_acc;
    const uint64_t t = block_sum(all_acc, lds);
    if (threadIdx.x == 0 && t != 0) {
        atomicAdd(reinterpret_cast<unsigned long long*>(a.digest + bt.total_slot), (unsigned long long)t);
    }
}

__global__ void zero_kernel(uint64_t* slots, uint32_t n) {
    for (uint32_t i = threadIdx.x; i < n; i += blockDim.x) {
        slots[i] = 0;
    }
}

// 30 bytes per element, no arithmetic beyond one add: the ceiling of the
// commit's access pattern.
// The outputs may alias the inputs element for element (in place).
__global__ __launch_bounds__(kBlock) void probe_kernel(const float* i0, const float* i1, const float* i2,
                                                       const float* i3, float* o0, float* o2, float* o3,
                                                       uint16_t* oh, uint64_t nvec) {
    const uint64_t stride = (uint64_t)gridDim.x * kBlock;
    for (uint64_t k = (uint64_t)blockIdx.x * kBlock + threadIdx.x; k < nvec; k += stride) {
        const float4 a = reinterpret_cast<const float4*>(i0)[k];
        const float4 b = reinterpret_cast<const float4*>(i1)[k];
        const float4 c = reinterpret_cast<const float4*>(i2)[k];
        const float4 d = reinterpret_cast<const float4*>(i3)[k];
        float4 s;
        s.x = a.x + b.x;
        s.y = a.y + b.y;
        s.z = a.z + b.z;
        s.w = a.w + b.w;
        reinterpret_cast<float4*>(o0)[k] = s;
        reinterpret_cast<float4*>(o2)[k] = c;
        reinterpret_cast<float4*>(o3)[k] = d;
        uint2 h;
        h.x = (__float_as_uint(s.x) >> 16) | (__float_as_uint(s.y) & 0xFFFF0000u);
        h.y = (__float_as_uint(s.z) >> 16) | (__float_as_uint(s.w) & 0xFFFF0000u);
        reinterpret_cast<uint2*>(oh)[k] = h;
    }
}

}  // namespace

hipError_t launch_zero(uint64_t* slots, uint32_t nslots, hipStream_t stream) {
    hipLaunchKernelGGL(zero_kernel, dim3(1), dim3(256), 0, stream, slots, nslots);
    return hipGetLastError();
}

hipError_t launch_batch(Mode mode, const Arrays& a, const Batch& b, uint32_t grid, hipStream_t stream) {
    switch (mode) {
        case Mode::Commit:
            hipLaunchKernelGGL(shard_kernel<Mode::Commit>, dim3(grid), dim3(kBlock), 0, stream, a, b);
            break;
        case Mode::StateDigest:
            hipLaunchKernelGGL(shard_kernel<Mode::StateDigest>, dim3(grid), dim3(kBlock), 0, stream, a, b);
            break;
        case Mode::Bf16Digest:
            hipLaunchKernelGGL(shard_kernel<Mode::Bf16Digest>, dim3(grid), dim3(kBlock), 0, stream, a, b);
            break;
    }
    return hipGetLastError();
}

hipError_t launch_probe(const float* i0, const float* i1, const float* i2, const float* i3,
                        float* o0, float* o2, float* o3, uint16_t* oh, uint64_t n,
                        uint32_t grid, hipStream_t stream) {
    hipLaunchKernelGGL(probe_kernel, dim3(grid), dim3(kBlock), 0, stream, i0, i1, i2, i3, o0, o2, o3, oh,
                       n / kVec);
    return hipGetLastError();
}

}  // namespace pact
