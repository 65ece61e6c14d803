// kernels.hip -- gfx950 kernels of libpactshard.
//
// One tile kernel serves every mode on binary32 state (commit, commit that
// also zeroes the gradient, state digest, bf16 digest, gradient guard) and a
// twin serves state held in BF16 (commit, state digest).
// Work is cut into tiles of kTile elements that never straddle a segment, and
// each workgroup takes exactly one tile (the hardware dispatcher then keeps
// every CU full and balances the tail by itself; a persistent grid measured
// slower on this pattern).  A full, aligned tile moves, per thread and per
// binary32 array, four 16-byte vectors with buffer_load/store_dwordx4, and four
// 8-byte ones into the bf16 working copy (dwordx2); on BF16 state, two 16-byte
// vectors of eight elements per array.  All of it is marked non-temporal; a
// ragged tail or a misaligned segment goes element by element.
//
// The digest is accumulated per thread in a 64-bit register (wrapping add),
// summed over the workgroup with 64-bit LDS atomics (one word per wave, the
// four words added by thread 0), and added with one 64-bit atomic per
// workgroup into one of kLanes workspace words of its result slot (256 bytes
// apart, so the atomics of neighbouring workgroups do not queue on one
// address); a final
// one-workgroup kernel sums the lanes and sets them back to zero, so a call
// that is told its workspace is clear can skip clearing it.  Without a
// workspace the atomics go to the result slot itself.  Wrapping addition is
// associative and commutative, so the order in which workgroups arrive
// cannot change the result.
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
constexpr uint32_t kTagP = 0, kTagM = 1, kTagV = 2, kTagB = 3;  // array tags (bits 56..63 of the index)

// Low 64 bits of z * C for a constant C = CHI:CLO.  With z = hi:lo,
//   z * C mod 2^64 = lo*CLO + ((hi*CLO + lo*CHI) << 32)
// and only the low 32 bits of the cross term hi*CLO + lo*CHI matter:
//   t     = lo * CHI              v_mul_lo_u32
//   cross = hi * CLO + t          v_mad_u64_u32 (t zero-extended; low half used)
//   prod  = lo * CLO              v_mad_u64_u32 (full 64-bit product)
//   res   = prod + (cross << 32)  v_add_u32 on the high half
// Three VOP3 instructions and one VOP2 add.  On gfx950 a VOP3 instruction
// issues at about half the rate of a VOP2 one, and the hash is most of the
// VALU work of every digesting kernel, so the cheaper add in place of a
// 64-bit shift or a fourth multiply counts.  The compiler's own lowering
// takes four multiply-class instructions plus register moves.  VALU-only
// inline assembly (the carry-out operand lands in a scalar register pair the
// result ignores).
template <uint32_t CLO, uint32_t CHI>
__device__ __forceinline__ uint64_t mul_const64(uint64_t z) {
    const uint32_t lo = (uint32_t)z;
    const uint32_t hi = (uint32_t)(z >> 32);
    const uint32_t t = lo * CHI;
    uint64_t cross, prod, carry0, carry1;
    asm("v_mad_u64_u32 %0, %1, %2, %3, %4" : "=v"(cross), "=s"(carry0) : "v"(hi), "s"(CLO), "v"((uint64_t)t));
    asm("v_mad_u64_u32 %0, %1, %2, %3, 0" : "=v"(prod), "=s"(carry1) : "v"(lo), "s"(CLO));
    uint32_t res_hi;
    asm("v_add_u32_e32 %0, %1, %2" : "=v"(res_hi) : "v"((uint32_t)(prod >> 32)), "v"((uint32_t)cross));
    return ((uint64_t)res_hi << 32) | (uint32_t)prod;
}

// The mixing function applied after the generator's first addition.
__device__ __forceinline__ uint64_t splitmix_mix(uint64_t z) {
    z = mul_const64<(uint32_t)kMul1, (uint32_t)(kMul1 >> 32)>(z ^ (z >> 30));
    z = mul_const64<(uint32_t)kMul2, (uint32_t)(kMul2 >> 32)>(z ^ (z >> 27));
    return z ^ (z >> 31);
}

// splitmix64 of  word ^ (index | Tag << 56)  for a word of array Tag at flat
// index `index`.  Indices stay below 2^56 (the host rejects larger ones) and
// a word has 32 bits, so the tag bits meet only zeros on both sides:
//   word ^ (index | Tag << 56) = (word ^ index) + (Tag << 56)
// and the tag folds into the constant the generator adds first,
//   z = (word ^ index) + (gamma + (Tag << 56))  mod 2^64.
template <uint32_t Tag>
__device__ __forceinline__ uint64_t hash_word(uint32_t word, uint64_t index) {
    static_assert(Tag < 4, "array tags 0..3");
    constexpr uint64_t kAdd = kGamma + ((uint64_t)Tag << 56);
    return splitmix_mix(((uint64_t)word ^ index) + kAdd);
}

// The indices of the digest words of one vector tile, as seen by one lane:
// word `off` of the lane sits at flat index first + off.
//
// IndexAny: plain 64-bit indices, valid for every tile.
struct IndexAny {
    uint64_t first;  // index of the lane's first word
    __device__ __forceinline__ IndexAny(uint64_t tile_first, uint32_t lane_off) : first(tile_first + lane_off) {}
    template <uint32_t Tag>
    __device__ __forceinline__ uint64_t hash(uint32_t word, uint32_t off) const {
        return hash_word<Tag>(word, first + off);
    }
};

// The rest of the mix once the first round's product is known as
// prod + (cross << 32) (prod the full 64-bit product of the low halves with
// the first round's addend folded in, cross the low half of the cross
// term): the high half takes cross with one VOP2 add, then the second
// xor-shift and multiply and the final xor-shift.
__device__ __forceinline__ uint64_t mix_after_first_round(uint64_t prod, uint32_t cross) {
    uint32_t res_hi;
    asm("v_add_u32_e32 %0, %1, %2" : "=v"(res_hi) : "v"((uint32_t)(prod >> 32)), "v"(cross));
    uint64_t z = ((uint64_t)res_hi << 32) | (uint32_t)prod;
    z = z ^ (z >> 27);
    {
        constexpr uint32_t c2lo = (uint32_t)kMul2, c2hi = (uint32_t)(kMul2 >> 32);
        const uint32_t zl = (uint32_t)z, zh = (uint32_t)(z >> 32);
        const uint32_t t = zl * c2hi;
        uint64_t cr, pr, cy0, cy1;
        asm("v_mad_u64_u32 %0, %1, %2, %3, %4" : "=v"(cr), "=s"(cy0) : "v"(zh), "s"(c2lo), "v"(((uint64_t)zh << 32) | t));
        asm("v_mad_u64_u32 %0, %1, %2, %3, 0" : "=v"(pr), "=s"(cy1) : "v"(zl), "s"(c2lo));
        uint32_t rh;
        asm("v_add_u32_e32 %0, %1, %2" : "=v"(rh) : "v"((uint32_t)(pr >> 32)), "v"((uint32_t)cr));
        z = ((uint64_t)rh << 32) | (uint32_t)pr;
    }
    return z ^ (z >> 31);
}

// (h ^ (h >> 30)) * c mod 2^32 of wave-uniform h and c, on the scalar unit
// (left to itself the compiler forms such per-tile constants with VALU
// instructions, because their uses want VGPRs).
__device__ __forceinline__ uint32_t scalar_xorshift30_mul(uint32_t h, uint32_t c) {
    uint32_t r;
    asm("s_lshr_b32 %0, %1, 30\n\ts_xor_b32 %0, %0, %1\n\ts_mul_i32 %0, %0, %2" : "=&s"(r) : "s"(h), "s"(c) : "scc");
    return r;
}

// IndexHi32: for a tile whose indices all share their upper 32 bits `hi`
// (every tile but one that crosses a multiple of 2^32).  With index = hi:lo
// the word only meets the low half, so
//   z = (word ^ index) + gamma_k = zext(x) + G_k,   x = word ^ lo,
// where gamma_k = gamma + (k << 56) is the tagged constant above and
// G_k = (hi << 32) + gamma_k is one wave-uniform 64-bit value per tag.  Its
// low half is gamma's (the same for every tile and tag), so z's halves are
//   z_lo = x + G_lo (carry c),   z_hi = G_hi + c,
// and z_hi takes one of two values.  The first mixing round then reads the
// carry instead of a 64-bit value:
//   z ^ (z >> 30):  lo1 = z_lo ^ alignbit(z_hi, z_lo, 30),
//                   hi1 = z_hi ^ (z_hi >> 30), one of H_0, H_1 (c = 0, 1);
//   times C1 = CHI:CLO, low 64 bits: lo1 * CLO + ((lo1 * CHI + hi1 * CLO) << 32),
// and hi1 * CLO is one of K_0, K_1 = H_c * CLO mod 2^32.  So the product is
//   prod  = lo1 * CLO + (K_0 << 32)          v_mad_u64_u32, scalar addend
//   cross = lo1 * CHI + (c ? K_1 - K_0 : 0)  v_mad_u64_u32, low half used
//   z1    = prod + (cross << 32)             v_add_u32 on the high half
// with the carry, z_hi and the select taken by three VOP2 instructions that
// share the carry in VCC.  Against the plain round this trades a 64-bit
// shift, a multiply and the 64-bit index add (five VOP3 instructions) for
// three VOP3 and two more VOP2 ones; the later rounds are unchanged.
struct IndexHi32 {
    static constexpr uint32_t kGammaLo = (uint32_t)kGamma;
    uint32_t lo;        // low half of the lane's first index
    uint32_t ghi[4];    // G_hi per tag
    uint32_t kdiff[4];  // K_1 - K_0 per tag
    uint64_t k0hi[4];   // K_0 << 32 per tag
    __device__ __forceinline__ IndexHi32(uint64_t tile_first, uint32_t lane_off)
        : lo((uint32_t)tile_first + lane_off) {
        constexpr uint32_t clo = (uint32_t)kMul1;
        const uint64_t high = tile_first & 0xFFFFFFFF00000000ull;
#pragma unroll
        for (uint32_t k = 0; k < 4; ++k) {
            const uint32_t h = (uint32_t)((high + kGamma + ((uint64_t)k << 56)) >> 32);
            const uint32_t h1 = h + 1u;
            // wave-uniform per tile: scalar unit, then one copy into VGPRs
            const uint32_t k0 = scalar_xorshift30_mul(h, clo);
            const uint32_t k1 = scalar_xorshift30_mul(h1, clo);
            ghi[k] = h;
            kdiff[k] = k1 - k0;
            k0hi[k] = (uint64_t)k0 << 32;
        }
    }
    template <uint32_t Tag>
    __device__ __forceinline__ uint64_t hash(uint32_t word, uint32_t off) const {
        static_assert(Tag < 4, "array tags 0..3");
        constexpr uint32_t clo = (uint32_t)kMul1, chi = (uint32_t)(kMul1 >> 32);
        const uint32_t x = word ^ (lo + off);
        uint32_t zlo, zhi, ksel;
        // VCC carries c from the add to the select and to z_hi; a VALU write
        // of VCC needs two wait states before a VALU reads it as a lane mask.
        asm("v_add_co_u32_e32 %0, vcc, %3, %4\n\t"
            "s_nop 1\n\t"
            "v_cndmask_b32_e32 %1, 0, %5, vcc\n\t"
            "v_addc_co_u32_e32 %2, vcc, 0, %6, vcc"
            : "=&v"(zlo), "=&v"(ksel), "=v"(zhi)
            : "s"(kGammaLo), "v"(x), "v"(kdiff[Tag]), "v"(ghi[Tag])
            : "vcc");
        const uint32_t lo1 = zlo ^ __builtin_amdgcn_alignbit(zhi, zlo, 30);
        uint64_t prod, cross, carry0, carry1;
        asm("v_mad_u64_u32 %0, %1, %2, %3, %4" : "=v"(prod), "=s"(carry0) : "v"(lo1), "v"(clo), "s"(k0hi[Tag]));
        // Only cross's low half is used, so the addend's high half may hold
        // anything: z_hi, which sits beside the select in the register pair.
        asm("v_mad_u64_u32 %0, %1, %2, %3, %4"
            : "=v"(cross), "=s"(carry1)
            : "v"(lo1), "s"(chi), "v"(((uint64_t)zhi << 32) | ksel));
        return mix_after_first_round(prod, (uint32_t)cross);
    }
};

// IndexLo16: for a tile of 16-bit words (BF16 state, the bf16 working copy)
// whose indices all share bits 16..63.  There x = word ^ lo = A + v with
// A = lo & 0xFFFF0000 the same for the whole tile and v < 2^16, so with
// B = A + G_lo = c0 * 2^32 + B_lo (wave-uniform):
//   z_lo = x + G_lo = B_lo + v,   z_hi = G_hi + c0,
// provided B_lo + v never carries out of 32 bits (B_lo <= 0xFFFF0000).  If
// moreover no carry reaches bit 30 ((B_lo mod 2^30) <= 0x3FFF0000), the top
// two bits of z_lo are those of B_lo, T = B_lo >> 30, so the first mixing
// round is
//   lo1 = z_lo ^ (T | z_hi << 2) = (x + G_lo) ^ U_k,   hi1 = H_k,
//   z1  = lo1 * CLO + ((lo1 * CHI + H_k * CLO) << 32),
// with U_k, H_k and K_k = H_k * CLO wave-uniform per tag: an add, an xor, a
// multiply-add with the scalar addend K_k << 32, a multiply and an add, two
// VOP3 instructions against three (and three fewer VALU instructions) in
// IndexHi32, and no carry to pass.  The two checks fail only for A in
// {0x00B50000, 0x40B50000, 0x80B50000, 0xC0B50000}; such a tile, and one that
// crosses a multiple of 2^16, takes IndexHi32 or IndexAny.
struct IndexLo16 {
    static constexpr uint32_t kGammaLo = (uint32_t)kGamma;
    uint32_t lo;       // low half of the lane's first index
    uint32_t u[4];     // U_k per tag
    uint64_t khi[4];   // K_k << 32 per tag
    // Whether the tile of kTile indices from `first` on may take this form
    // (wave-uniform).
    static __device__ __forceinline__ bool applies(uint64_t first) {
        if ((first >> 16) != ((first + kTile - 1) >> 16)) {
            return false;
        }
        const uint32_t b_lo = ((uint32_t)first & 0xFFFF0000u) + kGammaLo;
        return b_lo <= 0xFFFF0000u && (b_lo & 0x3FFFFFFFu) <= 0x3FFF0000u;
    }
    __device__ __forceinline__ IndexLo16(uint64_t tile_first, uint32_t lane_off)
        : lo((uint32_t)tile_first + lane_off) {
        constexpr uint32_t clo = (uint32_t)kMul1;
        const uint64_t b = (uint64_t)((uint32_t)tile_first & 0xFFFF0000u) + kGammaLo;
        const uint32_t c0 = (uint32_t)(b >> 32);
        const uint32_t t = (uint32_t)b >> 30;
        const uint32_t hi = (uint32_t)(tile_first >> 32);
#pragma unroll
        for (uint32_t k = 0; k < 4; ++k) {
            const uint32_t zhi = hi + (uint32_t)(kGamma >> 32) + (k << 24) + c0;
            u[k] = (zhi << 2) | t;
            khi[k] = (uint64_t)scalar_xorshift30_mul(zhi, clo) << 32;
        }
    }
    template <uint32_t Tag>
    __device__ __forceinline__ uint64_t hash(uint32_t word, uint32_t off) const {
        static_assert(Tag < 4, "array tags 0..3");
        constexpr uint32_t clo = (uint32_t)kMul1, chi = (uint32_t)(kMul1 >> 32);
        const uint32_t x = word ^ (lo + off);
        uint32_t zlo;
        asm("v_add_u32_e32 %0, %1, %2" : "=v"(zlo) : "s"(kGammaLo), "v"(x));
        const uint32_t lo1 = zlo ^ u[Tag];
        uint64_t prod, carry0;
        asm("v_mad_u64_u32 %0, %1, %2, %3, %4" : "=v"(prod), "=s"(carry0) : "v"(lo1), "v"(clo), "s"(khi[Tag]));
        return mix_after_first_round(prod, lo1 * chi);
    }
};

// Whether the `count` indices from `first` on share their upper 32 bits.
__device__ __forceinline__ bool same_high_half(uint64_t first, uint64_t count) {
    return (first >> 32) == ((first + count - 1) >> 32);
}

// ---------------------------------------------------------------------------
// AdamW on one element, in the contract's order.  With -ffp-contract=off and
// no fast-math flags every +, -, * below is one IEEE binary32 operation
// rounded to nearest even, '/' is the correctly rounded division, and
// __builtin_sqrtf is lowered to the correctly rounded square root (the
// -fhip-fp32-correctly-rounded-divide-sqrt default).  HIP's __fsqrt_rn is
// NOT used: unless OCML_BASIC_ROUNDED_OPERATIONS is defined it maps to the
// hardware's approximate v_sqrt_f32.  The update is split in two: the
// moments, then the bias-corrected step, so that a tile can pick the form of
// the square root once for all its elements (see sqrt_rn_in_range).
// ---------------------------------------------------------------------------
__device__ __forceinline__ void adamw_moments(float& p, float g, float& m, float& v, const StepScalars& s) {
    const float p_dec = p * s.decay;
    const float m_keep = s.beta1 * m;
    const float m_push = s.omb1 * g;
    const float m_new = m_keep + m_push;
    const float g_sq = g * g;
    const float v_keep = s.beta2 * v;
    const float v_push = s.omb2 * g_sq;
    const float v_new = v_keep + v_push;
    p = p_dec;
    m = m_new;
    v = v_new;
}

// Correctly rounded square root of x in [2^-96, +inf).  The hardware root
// s = v_sqrt_f32(x) is within one ulp of sqrt(x) there (so is the compiler's
// full sequence built on it), so the correctly rounded root is s or one of
// its neighbours s_dn, s_up (bit patterns minus and plus one), and two exact
// residuals decide which (the rounding test for square roots by fused
// multiply-add, as in Markstein's and Goldschmidt-style refinements):
//   x <= s_dn * s  => sqrt(x) lies below the midpoint of s_dn and s
//                     (the geometric mean is below the arithmetic one);
//   x >  s * s_up  => sqrt(x) lies above the midpoint of s and s_up: the
//                     squared midpoint exceeds s * s_up by ulp^2 / 4, and
//                     no binary32 x falls in that gap (x's grid near s^2 is
//                     at least 2^22 of those units);
//   otherwise s.
// The residuals x - s_dn*s and x - s_up*s are computed by one FMA each; for
// x >= 2^-96 they are multiples of 2^-142, so their signs come out exact
// (denormals are kept).  The compiler's full sequence adds a rescaling of
// inputs below 2^-96 and a class test for 0 and infinity; a tile whose
// inputs all lie in [2^-96, +inf) takes this form (a wave-uniform branch),
// any other tile the full one, with the same bits.
__device__ __forceinline__ bool sqrt_rn_in_range(float x) {
    return (__float_as_uint(x) - 0x0F800000u) < (0x7F800000u - 0x0F800000u);
}

__device__ __forceinline__ float sqrt_rn_in_range_root(float x) {
    const float s = __builtin_amdgcn_sqrtf(x);
    const float s_dn = __uint_as_float(__float_as_uint(s) - 1u);
    const float s_up = __uint_as_float(__float_as_uint(s) + 1u);
    const float r_dn = __builtin_fmaf(-s_dn, s, x);
    const float r_up = __builtin_fmaf(-s_up, s, x);
    const float t = r_dn <= 0.0f ? s_dn : s;
    return r_up > 0.0f ? s_up : t;
}

template <bool InRange>
__device__ __forceinline__ float adamw_step(float p_dec, float m_new, float v_new, const StepScalars& s) {
    const float root = InRange ? sqrt_rn_in_range_root(v_new) : __builtin_sqrtf(v_new);
    const float den = root * s.rs_bc2 + s.eps;
    const float ratio = m_new / den;
    const float step = s.step_size * ratio;
    return p_dec - step;
}

__device__ __forceinline__ void adamw(float& p, float g, float& m, float& v, const StepScalars& s) {
    adamw_moments(p, g, m, v, s);
    p = adamw_step<false>(p, m, v, s);
}

// The bias-corrected steps of all n elements of a lane's share of a tile
// (p holds p*decay, m and v the new moments), with the short square root
// when every v of the wave is in its range.
template <int N>
__device__ __forceinline__ void adamw_steps(float (&p)[N], const float (&m)[N], const float (&v)[N],
                                            const StepScalars& s) {
    bool in_range = true;
#pragma unroll
    for (int i = 0; i < N; ++i) in_range = in_range && sqrt_rn_in_range(v[i]);
    if (__builtin_amdgcn_ballot_w64(!in_range) == 0) {
#pragma unroll
        for (int i = 0; i < N; ++i) p[i] = adamw_step<true>(p[i], m[i], v[i], s);
    } else {
#pragma unroll
        for (int i = 0; i < N; ++i) p[i] = adamw_step<false>(p[i], m[i], v[i], s);
    }
}

// binary32 -> bfloat16, round to nearest even; NaN stays a quiet NaN with
// its sign and top payload bits.  The rule, on the bits u of x:
//   NaN:       (u >> 16) | 0x0040
//   otherwise: (u + 0x7FFF + ((u >> 16) & 1)) >> 16
// gfx950's v_cvt_pk_bf16_f32 computes exactly this, two values per
// instruction, so the kernels use it: a GPU test sends all 2^32 patterns
// through the commit as weights (p' = p * 1 - 0) and compares the bf16 copy
// with this rule applied to the GPU's own p', NaNs included.
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t to_bf16x2(float lo, float hi) {
    const f32x2_t f = {lo, hi};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2_t));
}

__device__ __forceinline__ uint32_t to_bf16(float x) { return to_bf16x2(x, 0.0f) & 0xFFFFu; }

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
    return r;
}

// ---------------------------------------------------------------------------
// HBM access: raw buffer instructions on a per-tile resource (base address in
// scalar registers, 32-bit byte offset per lane), with the non-temporal cache
// policy on loads and stores -- every byte is touched exactly once.
// ---------------------------------------------------------------------------
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kRsrcWord3 = 0x00020000;  // raw, untyped buffer (gfx9 family)
constexpr int kNonTemporal = 2;         // cache-policy 'nt' bit

__device__ __forceinline__ __amdgpu_buffer_rsrc_t tile_rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, kRsrcWord3);
}

// The whole byte offset travels in the per-lane VGPR offset and the scalar
// offset field stays the literal 0.  That matters for stores wider than 8
// bytes: their data VGPRs must not be overwritten by the very next VALU
// instruction (one wait state), and the compiler only guards that hazard
// when the scalar offset is not a register.  With a register scalar offset a
// following VALU write was seen to corrupt the first dword of the stored
// vector.
__device__ __forceinline__ u32x4 load16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, kNonTemporal);
}
__device__ __forceinline__ void store16(u32x4 x, __amdgpu_buffer_rsrc_t r, uint32_t off) {
    __builtin_amdgcn_raw_buffer_store_b128(x, r, (int)off, 0, kNonTemporal);
}
__device__ __forceinline__ u32x2 load8(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_amdgcn_raw_buffer_load_b64(r, (int)off, 0, kNonTemporal);
}
__device__ __forceinline__ void store8(u32x2 x, __amdgpu_buffer_rsrc_t r, uint32_t off) {
    __builtin_amdgcn_raw_buffer_store_b64(x, r, (int)off, 0, kNonTemporal);
}

// ---------------------------------------------------------------------------
// one element, element-wise path (ragged tails, misaligned segments)
// ---------------------------------------------------------------------------
template <Mode M>
constexpr bool kCommits = (M == Mode::Commit || M == Mode::CommitZeroGrad);

// Modes whose digest words have 16 bits (the short IndexLo16 form applies).
template <Mode M>
constexpr bool kWords16 = (M == Mode::Bf16Digest || M == Mode::CommitBf16State || M == Mode::DigestBf16State);

template <Mode M>
__device__ __forceinline__ uint64_t do_scalar(const Arrays& a, uint64_t e, const StepScalars& sc) {
    const uint64_t idx = a.goff + e;
    if constexpr (M == Mode::Bf16Digest) {
        return hash_word<kTagB>(a.b[e], idx);
    } else if constexpr (M == Mode::GradGuard) {
        return __float_as_uint(a.g[e]) != 0u ? 1u : 0u;
    } else {
        float p = a.p[e];
        float m = a.m[e];
        float v = a.v[e];
        if constexpr (kCommits<M>) {
            adamw(p, a.g[e], m, v, sc);
            a.p[e] = p;
            a.m[e] = m;
            a.v[e] = v;
            a.b[e] = (uint16_t)to_bf16(p);
            if constexpr (M == Mode::CommitZeroGrad) {
                a.g_zero[e] = 0.0f;
            }
        }
        return hash_word<kTagP>(__float_as_uint(p), idx) + hash_word<kTagM>(__float_as_uint(m), idx) +
               hash_word<kTagV>(__float_as_uint(v), idx);
    }
}

// ---------------------------------------------------------------------------
// one full tile whose start is 16-byte aligned in every fp32 array (8-byte in
// the bf16 array): kUnroll rows of kBlock 16-byte vectors per array.  Row u,
// lane t holds elements e0 + u*kBlock*4 + 4t .. +3.
// ---------------------------------------------------------------------------
template <Mode M, typename Ix>
__device__ __forceinline__ uint64_t do_tile_vec(const Arrays& a, uint64_t e0, const StepScalars& sc) {
    constexpr uint32_t kRow32 = kBlock * kVec * 4;  // bytes of one fp32 row
    constexpr uint32_t kRow16 = kBlock * kVec * 2;  // bytes of one bf16 row
    const uint32_t lane32 = threadIdx.x * kVec * 4;
    const uint32_t lane16 = threadIdx.x * kVec * 2;
    const Ix ix(a.goff + e0, threadIdx.x * kVec);  // word k of this lane: index + k
    uint64_t acc = 0;
    if constexpr (M == Mode::GradGuard) {
        const auto rg = tile_rsrc(a.g + e0, kTile * 4);
        u32x4 G[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            G[u] = load16(rg, lane32 + u * kRow32);
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
#pragma unroll
            for (int j = 0; j < kVec; ++j) {
                acc += G[u][j] != 0u ? 1u : 0u;
            }
        }
        return acc;
    } else if constexpr (M == Mode::Bf16Digest) {
        const auto rb = tile_rsrc(a.b + e0, kTile * 2);
        u32x2 W[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            W[u] = load8(rb, lane16 + u * kRow16);
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const uint32_t o = u * kBlock * kVec;
            acc += ix.template hash<kTagB>(W[u].x & 0xFFFFu, o) + ix.template hash<kTagB>(W[u].x >> 16, o + 1) +
                   ix.template hash<kTagB>(W[u].y & 0xFFFFu, o + 2) + ix.template hash<kTagB>(W[u].y >> 16, o + 3);
        }
        return acc;
    } else {
        const auto rp = tile_rsrc(a.p + e0, kTile * 4);
        const auto rm = tile_rsrc(a.m + e0, kTile * 4);
        const auto rv = tile_rsrc(a.v + e0, kTile * 4);
        u32x4 P[kUnroll], G[kUnroll], Mo[kUnroll], V[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            P[u] = load16(rp, lane32 + u * kRow32);
            Mo[u] = load16(rm, lane32 + u * kRow32);
            V[u] = load16(rv, lane32 + u * kRow32);
        }
        if constexpr (kCommits<M>) {
            const auto rg = tile_rsrc(a.g + e0, kTile * 4);
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) {
                G[u] = load16(rg, lane32 + u * kRow32);
            }
            if constexpr (M == Mode::CommitZeroGrad) {
                const u32x4 zero = {0u, 0u, 0u, 0u};
#pragma unroll
                for (int u = 0; u < kUnroll; ++u) {
                    store16(zero, rg, lane32 + u * kRow32);
                }
            }
            const auto rb = tile_rsrc(a.b + e0, kTile * 2);
            // Bound by HBM: each row is updated and stored as soon as it is
            // ready, with the full square root (the short in-range form of the
            // BF16-state commit measured no faster here).
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) {
                float p[4], m[4], v[4];
#pragma unroll
                for (int j = 0; j < kVec; ++j) {
                    p[j] = __uint_as_float(P[u][j]);
                    m[j] = __uint_as_float(Mo[u][j]);
                    v[j] = __uint_as_float(V[u][j]);
                    adamw(p[j], __uint_as_float(G[u][j]), m[j], v[j], sc);
                    P[u][j] = __float_as_uint(p[j]);
                    Mo[u][j] = __float_as_uint(m[j]);
                    V[u][j] = __float_as_uint(v[j]);
                }
                store16(P[u], rp, lane32 + u * kRow32);
                store16(Mo[u], rm, lane32 + u * kRow32);
                store16(V[u], rv, lane32 + u * kRow32);
                u32x2 h;
                h.x = to_bf16x2(p[0], p[1]);
                h.y = to_bf16x2(p[2], p[3]);
                store8(h, rb, lane16 + u * kRow16);
            }
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
#pragma unroll
            for (int j = 0; j < kVec; ++j) {
                const uint32_t o = u * kBlock * kVec + j;
                acc += ix.template hash<kTagP>(P[u][j], o) + ix.template hash<kTagM>(Mo[u][j], o) +
                       ix.template hash<kTagV>(V[u][j], o);
            }
        }
        return acc;
    }
}

// ---------------------------------------------------------------------------
// BF16 state: a tile is kTile / (kBlock * 8) rows of kBlock 16-byte vectors
// (eight bf16 words each) per array; element 2j of a vector is the low half
// of its word j.
// ---------------------------------------------------------------------------
__device__ __forceinline__ float widen_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float widen_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

template <Mode M>
__device__ __forceinline__ uint64_t do_scalar(const ArraysBf16& a, uint64_t e, const StepScalars& sc) {
    const uint64_t idx = a.goff + e;
    uint32_t p = a.p[e];
    uint32_t m = a.m[e];
    uint32_t v = a.v[e];
    if constexpr (M == Mode::CommitBf16State) {
        float pf = widen_lo(p), mf = widen_lo(m), vf = widen_lo(v);
        adamw(pf, widen_lo(a.g[e]), mf, vf, sc);
        p = to_bf16(pf);
        m = to_bf16(mf);
        v = to_bf16(vf);
        a.p[e] = (uint16_t)p;
        a.m[e] = (uint16_t)m;
        a.v[e] = (uint16_t)v;
    }
    return hash_word<kTagP>(p, idx) + hash_word<kTagM>(m, idx) + hash_word<kTagV>(v, idx);
}

template <Mode M, typename Ix>
__device__ __forceinline__ uint64_t do_tile_vec(const ArraysBf16& a, uint64_t e0, const StepScalars& sc) {
    constexpr int kRows = kTile / (kBlock * 8);
    constexpr uint32_t kRowBytes = kBlock * 16;
    const uint32_t lane = threadIdx.x * 16;
    const Ix ix(a.goff + e0, threadIdx.x * 8);  // word k of this lane: index + k
    const auto rp = tile_rsrc(a.p + e0, kTile * 2);
    const auto rm = tile_rsrc(a.m + e0, kTile * 2);
    const auto rv = tile_rsrc(a.v + e0, kTile * 2);
    u32x4 P[kRows], G[kRows], Mo[kRows], V[kRows];
#pragma unroll
    for (int r = 0; r < kRows; ++r) {
        P[r] = load16(rp, lane + r * kRowBytes);
        Mo[r] = load16(rm, lane + r * kRowBytes);
        V[r] = load16(rv, lane + r * kRowBytes);
    }
    if constexpr (M == Mode::CommitBf16State) {
        const auto rg = tile_rsrc(a.g + e0, kTile * 2);
#pragma unroll
        for (int r = 0; r < kRows; ++r) {
            G[r] = load16(rg, lane + r * kRowBytes);
        }
        constexpr int kN = kRows * 8;
        float p[kN], m[kN], v[kN];
#pragma unroll
        for (int r = 0; r < kRows; ++r) {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int i = r * 8 + 2 * j;
                p[i] = widen_lo(P[r][j]);
                p[i + 1] = widen_hi(P[r][j]);
                m[i] = widen_lo(Mo[r][j]);
                m[i + 1] = widen_hi(Mo[r][j]);
                v[i] = widen_lo(V[r][j]);
                v[i + 1] = widen_hi(V[r][j]);
                adamw_moments(p[i], widen_lo(G[r][j]), m[i], v[i], sc);
                adamw_moments(p[i + 1], widen_hi(G[r][j]), m[i + 1], v[i + 1], sc);
            }
        }
        adamw_steps<kN>(p, m, v, sc);
#pragma unroll
        for (int r = 0; r < kRows; ++r) {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int i = r * 8 + 2 * j;
                P[r][j] = to_bf16x2(p[i], p[i + 1]);
                Mo[r][j] = to_bf16x2(m[i], m[i + 1]);
                V[r][j] = to_bf16x2(v[i], v[i + 1]);
            }
            store16(P[r], rp, lane + r * kRowBytes);
            store16(Mo[r], rm, lane + r * kRowBytes);
            store16(V[r], rv, lane + r * kRowBytes);
        }
    }
    uint64_t acc = 0;
#pragma unroll
    for (int r = 0; r < kRows; ++r) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const uint32_t o = r * kBlock * 8 + 2 * j;
            acc += ix.template hash<kTagP>(P[r][j] & 0xFFFFu, o) + ix.template hash<kTagP>(P[r][j] >> 16, o + 1) +
                   ix.template hash<kTagM>(Mo[r][j] & 0xFFFFu, o) + ix.template hash<kTagM>(Mo[r][j] >> 16, o + 1) +
                   ix.template hash<kTagV>(V[r][j] & 0xFFFFu, o) + ix.template hash<kTagV>(V[r][j] >> 16, o + 1);
        }
    }
    return acc;
}

// ---------------------------------------------------------------------------
// One workgroup per tile.  The tile's segment is found by binary search over
// the batch's tile prefix (kernel arguments, scalar loads); the tile's digest
// share is summed over the workgroup in LDS and added with one 64-bit atomic.
// ---------------------------------------------------------------------------
template <Mode M, typename A>
__device__ __forceinline__ void tile_body(const A& a, const Batch& bt, uint64_t* lds) {
    const uint64_t tile = blockIdx.x;
    uint32_t lo = 0, hi = bt.nseg;  // largest lo with tile_begin[lo] <= tile
    while (hi - lo > 1) {
        const uint32_t mid = (lo + hi) >> 1;
        if (tile >= bt.tile_begin[mid]) {
            lo = mid;
        } else {
            hi = mid;
        }
    }
    const uint32_t seg = lo;
    const StepScalars sc = bt.sc[seg];
    const uint64_t seg_first = bt.elem_begin[seg];
    const uint64_t seg_end = seg_first + bt.elem_count[seg];
    const uint64_t e0 = seg_first + (tile - bt.tile_begin[seg]) * (uint64_t)kTile;
    // This wave's word of the workgroup sum starts at zero (LDS operations of
    // one wave are carried out in the order it issues them, so the clearing
    // comes before the wave's own additions below).
    uint64_t* const wave_sum = lds + (threadIdx.x >> 6);
    if ((threadIdx.x & 63) == 0) {
        __hip_atomic_store(wave_sum, (uint64_t)0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    }
    uint64_t acc = 0;
    if (bt.vec_ok[seg] && e0 + kTile <= seg_end) {
        // The short index form for tiles that do not cross a multiple of
        // 2^32 (a uniform branch: at most one tile in 2^20 takes the other);
        // the binary32 commits are bound by HBM, not by VALU issue, and keep
        // the plain form (the short one measured 0.3% slower there, with one
        // more wave per SIMD resident).
        if (kWords16<M> && IndexLo16::applies(a.goff + e0)) {
            acc = do_tile_vec<M, IndexLo16>(a, e0, sc);
        } else if (!kCommits<M> && same_high_half(a.goff + e0, kTile)) {
            acc = do_tile_vec<M, IndexHi32>(a, e0, sc);
        } else {
            acc = do_tile_vec<M, IndexAny>(a, e0, sc);
        }
    } else {
        const uint64_t e1 = (e0 + kTile < seg_end) ? e0 + kTile : seg_end;
        for (uint64_t e = e0 + threadIdx.x; e < e1; e += kBlock) {
            acc += do_scalar<M>(a, e, sc);
        }
    }
    // Workgroup sum: every lane adds its share into its wave's LDS word with
    // one 64-bit LDS atomic (no VALU work: a shuffle tree costs about fifty
    // VALU instructions per lane, a few percent of a digesting kernel), then
    // thread 0 adds the four words.
    __hip_atomic_fetch_add(wave_sum, acc, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    __syncthreads();
    uint64_t s = 0;
    if (threadIdx.x == 0) {
#pragma unroll
        for (int w = 0; w < kBlock / 64; ++w) {
            s += lds[w];
        }
    }
    if (threadIdx.x == 0 && s != 0) {
        const uint64_t r = bt.per_segment ? bt.slot0 + seg : 0;
        uint64_t* dst = a.lanes ? a.lanes + (r * kLanes + (blockIdx.x & (kLanes - 1))) * kLaneStride : a.digest + r;
        atomicAdd(reinterpret_cast<unsigned long long*>(dst), (unsigned long long)s);
    }
}

// Waves per SIMD a kernel must be able to keep resident (caps its VGPRs).
// The two standalone digests are bound by VALU issue and keep the full
// eight waves per SIMD (the short index form would otherwise take the state
// digest to 66 VGPRs and seven waves).  The BF16-state commit, which holds
// the moments of all its elements before the square roots, needs at least
// five; it takes 79 VGPRs, six waves (capped at seven it spills).
template <Mode M>
constexpr unsigned kMinWavesPerSimd = (M == Mode::StateDigest || M == Mode::DigestBf16State) ? 8u
                                      : (M == Mode::CommitBf16State)                         ? 5u
                                                                                             : 1u;

template <Mode M>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(kMinWavesPerSimd<M>)))
void tile_kernel(Arrays a, Batch bt) {
    __shared__ uint64_t lds[kBlock / 64];
    tile_body<M>(a, bt, lds);
}

template <Mode M>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(kMinWavesPerSimd<M>)))
void tile_kernel_bf16(ArraysBf16 a, Batch bt) {
    __shared__ uint64_t lds[kBlock / 64];
    tile_body<M>(a, bt, lds);
}

__global__ __launch_bounds__(kBlock) void clear_kernel(uint64_t* digest, uint64_t* lanes, uint32_t nres,
                                                       uint32_t nslots) {
    if (lanes) {
        const uint32_t n = nres * kLanes;
        for (uint32_t i = threadIdx.x; i < n; i += kBlock) {
            lanes[(uint64_t)i * kLaneStride] = 0;
        }
    } else {
        for (uint32_t i = threadIdx.x; i < nslots; i += kBlock) {
            digest[i] = 0;
        }
    }
}

// digest[r] = sum of r's lanes for r < nres (when lanes are used); with
// per-segment results also digest[nres] = sum of digest[0..nres).  Each lane
// is set back to zero once read, so a call always leaves its workspace lanes
// at zero and the next call may skip clearing them.
__global__ __launch_bounds__(kBlock) void finish_kernel(uint64_t* digest, uint64_t* lanes, uint32_t nres,
                                                        uint32_t per_segment) {
    __shared__ uint64_t lds[kBlock / 64];
    uint64_t total = 0;
    for (uint32_t r = threadIdx.x; r < nres; r += kBlock) {
        uint64_t x;
        if (lanes) {
            x = 0;
            for (int l = 0; l < kLanes; ++l) {
                uint64_t* lane = lanes + ((uint64_t)r * kLanes + l) * kLaneStride;
                x += *lane;
                *lane = 0;
            }
            digest[r] = x;
        } else {
            x = digest[r];
        }
        total += x;
    }
    if (per_segment) {
        const uint64_t t = block_sum(total, lds);
        if (threadIdx.x == 0) {
            digest[nres] = t;
        }
    }
}

// 30 bytes per element with no arithmetic beyond one add, through the same
// instructions and tile shape as the commit: the ceiling of the commit's
// access pattern.  The outputs may alias the inputs element for element (in
// place).  n is a multiple of 4; the last tile's resources end at n, and a
// vector beyond it is dropped by the buffer range check.
__device__ __forceinline__ void probe_tile(const float* i0, const float* i1, const float* i2, const float* i3,
                                           float* o0, float* o2, float* o3, uint16_t* oh, uint64_t n,
                                           uint64_t tile) {
    constexpr uint32_t kRow32 = kBlock * kVec * 4;
    constexpr uint32_t kRow16 = kBlock * kVec * 2;
    const uint64_t e0 = tile * kTile;
    const uint64_t left = n - e0;
    const uint32_t cnt = left < (uint64_t)kTile ? (uint32_t)left : (uint32_t)kTile;
    const auto r0 = tile_rsrc(i0 + e0, cnt * 4), r1 = tile_rsrc(i1 + e0, cnt * 4);
    const auto r2 = tile_rsrc(i2 + e0, cnt * 4), r3 = tile_rsrc(i3 + e0, cnt * 4);
    const auto w0 = tile_rsrc(o0 + e0, cnt * 4), w2 = tile_rsrc(o2 + e0, cnt * 4);
    const auto w3 = tile_rsrc(o3 + e0, cnt * 4), wh = tile_rsrc(oh + e0, cnt * 2);
    const uint32_t lane32 = threadIdx.x * kVec * 4, lane16 = threadIdx.x * kVec * 2;
    u32x4 A[kUnroll], B[kUnroll], C[kUnroll], D[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
        A[u] = load16(r0, lane32 + u * kRow32);
        B[u] = load16(r1, lane32 + u * kRow32);
        C[u] = load16(r2, lane32 + u * kRow32);
        D[u] = load16(r3, lane32 + u * kRow32);
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
        u32x4 s;
#pragma unroll
        for (int j = 0; j < kVec; ++j) {
            s[j] = __float_as_uint(__uint_as_float(A[u][j]) + __uint_as_float(B[u][j]));
        }
        store16(s, w0, lane32 + u * kRow32);
        store16(C[u], w2, lane32 + u * kRow32);
        store16(D[u], w3, lane32 + u * kRow32);
        u32x2 h;
        h.x = (s.x >> 16) | (s.y & 0xFFFF0000u);
        h.y = (s.z >> 16) | (s.w & 0xFFFF0000u);
        store8(h, wh, lane16 + u * kRow16);
    }
}

// One workgroup per tile, as the commit launches.
__global__ __launch_bounds__(kBlock) void probe_kernel(const float* i0, const float* i1, const float* i2,
                                                       const float* i3, float* o0, float* o2, float* o3,
                                                       uint16_t* oh, uint64_t n) {
    probe_tile(i0, i1, i2, i3, o0, o2, o3, oh, n, blockIdx.x);
}

// The same work from a persistent grid: workgroup b takes tiles b, b + grid,
// b + 2 grid, ... (the grid-stride shape), for comparison with one
// workgroup per tile.
__global__ __launch_bounds__(kBlock) void probe_persistent_kernel(const float* i0, const float* i1,
                                                                  const float* i2, const float* i3, float* o0,
                                                                  float* o2, float* o3, uint16_t* oh, uint64_t n) {
    const uint64_t tiles = (n + kTile - 1) / kTile;
    for (uint64_t t = blockIdx.x; t < tiles; t += gridDim.x) {
        probe_tile(i0, i1, i2, i3, o0, o2, o3, oh, n, t);
    }
}

}  // namespace

hipError_t launch_clear(uint64_t* digest, uint64_t* lanes, uint32_t nres, uint32_t nslots, hipStream_t stream) {
    hipLaunchKernelGGL(clear_kernel, dim3(1), dim3(kBlock), 0, stream, digest, lanes, nres, nslots);
    return hipGetLastError();
}

hipError_t launch_batch(Mode mode, const Arrays& a, const Batch& b, uint32_t grid, hipStream_t stream) {
    switch (mode) {
        case Mode::Commit:
            hipLaunchKernelGGL(tile_kernel<Mode::Commit>, dim3(grid), dim3(kBlock), 0, stream, a, b);
            break;
        case Mode::StateDigest:
            hipLaunchKernelGGL(tile_kernel<Mode::StateDigest>, dim3(grid), dim3(kBlock), 0, stream, a, b);
            break;
        case Mode::Bf16Digest:
            hipLaunchKernelGGL(tile_kernel<Mode::Bf16Digest>, dim3(grid), dim3(kBlock), 0, stream, a, b);
            break;
        case Mode::CommitZeroGrad:
            hipLaunchKernelGGL(tile_kernel<Mode::CommitZeroGrad>, dim3(grid), dim3(kBlock), 0, stream, a, b);
            break;
        case Mode::GradGuard:
            hipLaunchKernelGGL(tile_kernel<Mode::GradGuard>, dim3(grid), dim3(kBlock), 0, stream, a, b);
            break;
        default:
            return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_batch_bf16(Mode mode, const ArraysBf16& a, const Batch& b, uint32_t grid, hipStream_t stream) {
    switch (mode) {
        case Mode::CommitBf16State:
            hipLaunchKernelGGL(tile_kernel_bf16<Mode::CommitBf16State>, dim3(grid), dim3(kBlock), 0, stream, a, b);
            break;
        case Mode::DigestBf16State:
            hipLaunchKernelGGL(tile_kernel_bf16<Mode::DigestBf16State>, dim3(grid), dim3(kBlock), 0, stream, a, b);
            break;
        default:
            return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_finish(uint64_t* digest, uint64_t* lanes, uint32_t nres, bool per_segment, hipStream_t stream) {
    hipLaunchKernelGGL(finish_kernel, dim3(1), dim3(kBlock), 0, stream, digest, lanes, nres, per_segment ? 1u : 0u);
    return hipGetLastError();
}

hipError_t launch_probe(const float* i0, const float* i1, const float* i2, const float* i3,
                        float* o0, float* o2, float* o3, uint16_t* oh, uint64_t n, uint32_t workgroups,
                        hipStream_t stream) {
    if (workgroups == 0) {
        const uint64_t tiles = (n + kTile - 1) / kTile;
        hipLaunchKernelGGL(probe_kernel, dim3((uint32_t)tiles), dim3(kBlock), 0, stream, i0, i1, i2, i3, o0, o2,
                           o3, oh, n);
    } else {
        hipLaunchKernelGGL(probe_persistent_kernel, dim3(workgroups), dim3(kBlock), 0, stream, i0, i1, i2, i3, o0,
                           o2, o3, oh, n);
    }
    return hipGetLastError();
}

}  // namespace pact
