// Device helpers shared by the kernel files: element formats, 16-byte chunk
// access, the counter-based RNG, wave reductions and TIES's sign election
// with the disjoint mean.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace mp {

// ---------------------------------------------------------------- formats
// A "chunk" is 16 bytes: 4 fp32 or 8 bf16 elements.  Every tensor starts
// 16-byte aligned (numel is a multiple of the chunk width), and blocks are a
// multiple of the chunk width long, so a chunk never straddles two blocks.

template <int DT>
struct Fmt;

template <>
struct Fmt<0> {  // fp32
    static constexpr int V = 4;
    static constexpr int esize = 4;
    __device__ static inline void unpack(const uint4& c, float* f)
    {
        f[0] = __uint_as_float(c.x);
        f[1] = __uint_as_float(c.y);
        f[2] = __uint_as_float(c.z);
        f[3] = __uint_as_float(c.w);
    }
    __device__ static inline uint4 pack(const float* f)
    {
        return make_uint4(__float_as_uint(f[0]), __float_as_uint(f[1]), __float_as_uint(f[2]),
                          __float_as_uint(f[3]));
    }
};

// bfloat16 -> fp32 is exact (the 16 high bits of the fp32 pattern).
// fp32 -> bfloat16 rounds to nearest, ties to even (inputs are finite).

template <>
struct Fmt<1> {  // bf16
    static constexpr int V = 8;
    static constexpr int esize = 2;
    __device__ static inline void unpack(const uint4& c, float* f)
    {
        f[0] = __uint_as_float(c.x << 16);
        f[1] = __uint_as_float(c.x & 0xffff0000u);
        f[2] = __uint_as_float(c.y << 16);
        f[3] = __uint_as_float(c.y & 0xffff0000u);
        f[4] = __uint_as_float(c.z << 16);
        f[5] = __uint_as_float(c.z & 0xffff0000u);
        f[6] = __uint_as_float(c.w << 16);
        f[7] = __uint_as_float(c.w & 0xffff0000u);
    }
    // Hardware conversion (v_cvt_pk_bf16_f32, round to nearest even).  On
    // gfx950 it gives (u + 0x7fff + ((u >> 16) & 1)) >> 16 of the fp32
    // pattern u for every finite input (checked exhaustively, both halves).
    __device__ static inline uint32_t pack2(float a, float b)
    {
        typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
        const bf16x2 v = {(__bf16)a, (__bf16)b};
        return __builtin_bit_cast(uint32_t, v);
    }
    __device__ static inline uint4 pack(const float* f)
    {
        return make_uint4(pack2(f[0], f[1]), pack2(f[2], f[3]), pack2(f[4], f[5]), pack2(f[6], f[7]));
    }
};

__device__ static inline const uint4* chunk_ptr(const void* base, uint64_t elem_off, int esize)
{
    return reinterpret_cast<const uint4*>(static_cast<const char*>(base) + elem_off * (uint64_t)esize);
}

// A block of one checkpoint as a buffer resource: a wave-uniform base
// address and the block's byte length.  Loads then take one 32-bit offset
// register, which the base, every expert and the output of a block share;
// a load past the length returns zeros without touching memory and a store
// past it is dropped, so lanes beyond the end of a short block need no
// branch.  Third descriptor word: raw 32-bit data (the gfx9 encoding).
__device__ inline __amdgpu_buffer_rsrc_t block_rsrc(const void* p, uint32_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
__device__ inline uint4 bld16(__amdgpu_buffer_rsrc_t r, uint32_t off)
{
    const u32x4_t v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
    return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ inline void bst16(__amdgpu_buffer_rsrc_t r, uint32_t off, uint4 v)
{
    const u32x4_t w = {v.x, v.y, v.z, v.w};
    __builtin_amdgcn_raw_buffer_store_b128(w, r, off, 0, 0);
}

// Streaming accesses: data a kernel touches once (expert and base blocks,
// merged output) carry the non-temporal cache policy (the "nt" bit, cache
// policy 2 of the buffer and global instructions), so that they do not
// displace lines that are reused.  Measured on the headline family, it took
// the threshold merges from 1.69 / 2.07 / 2.95 ms to 1.62 / 1.95 / 2.74 ms at
// B = 25/50/100%.
__device__ inline uint4 bld16s(__amdgpu_buffer_rsrc_t r, uint32_t off)
{
    const u32x4_t v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 2);
    return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ inline void bst16s(__amdgpu_buffer_rsrc_t r, uint32_t off, uint4 v)
{
    const u32x4_t w = {v.x, v.y, v.z, v.w};
    __builtin_amdgcn_raw_buffer_store_b128(w, r, off, 0, 2);
}
__device__ inline uint4 ld16s(const uint4* p)
{
    const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ inline void st16s(uint4* p, uint4 v)
{
    const u32x4_t w = {v.x, v.y, v.z, v.w};
    __builtin_nontemporal_store(w, reinterpret_cast<u32x4_t*>(p));
}

// ---------------------------------------------------------------- Philox4x32-10
// Salmon, Moraes, Dror, Shaw, "Parallel Random Numbers: As Easy as 1, 2, 3"
// (SC 2011): ten rounds of two 32x32->64 multiplies with the Weyl-bumped key.
// a ^ b ^ k with k wave-uniform, as one CDNA4 three-input bitwise op (truth
// table 0x96 is the odd-parity function of its inputs).  Left to itself the
// compiler issues two v_xor_b32 here, and Philox's rounds are most of the
// VALU work of the DARE kernels.
__device__ static inline uint32_t xor3_u32(uint32_t a, uint32_t b, uint32_t k)
{
    uint32_t r;
    asm("v_bitop3_b32 %0, %1, %2, %3 bitop3:0x96" : "=v"(r) : "v"(a), "v"(b), "s"(k));
    return r;
}

__device__ static inline uint4 philox4x32_10(uint4 c, uint32_t k0, uint32_t k1)
{
    constexpr uint32_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u;
    constexpr uint32_t W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        // full 32x32 -> 64-bit products (one v_mad_u64_u32 each)
        const uint64_t p0 = (uint64_t)M0 * c.x;
        const uint64_t p1 = (uint64_t)M1 * c.z;
        const uint32_t lo0 = (uint32_t)p0, hi0 = (uint32_t)(p0 >> 32);
        const uint32_t lo1 = (uint32_t)p1, hi1 = (uint32_t)(p1 >> 32);
        c = make_uint4(xor3_u32(hi1, c.y, k0), lo1, xor3_u32(hi0, c.w, k1), lo0);
        k0 += W0;
        k1 += W1;
    }
    return c;
}

// ---------------------------------------------------------------- wave64 cross-lane helpers
// DPP row shifts / row broadcasts (GCN/CDNA wave64), no LDS round trip.
template <int CTRL, int ROW_MASK, int BANK_MASK, bool BOUND_CTRL>
__device__ static inline uint32_t dpp_u32(uint32_t v)
{
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, ROW_MASK, BANK_MASK, BOUND_CTRL);
}

// Inclusive prefix sum over the 64 lanes of a wave (lane 0 first).
__device__ static inline uint32_t wave_incl_sum(uint32_t v)
{
    uint32_t s = v;
    s += dpp_u32<0x111, 0xf, 0xf, true>(v);   // row_shr:1
    s += dpp_u32<0x112, 0xf, 0xf, true>(v);   // row_shr:2
    s += dpp_u32<0x113, 0xf, 0xf, true>(v);   // row_shr:3
    s += dpp_u32<0x114, 0xf, 0xe, false>(s);  // row_shr:4, banks 1-3
    s += dpp_u32<0x118, 0xf, 0xc, false>(s);  // row_shr:8, banks 2-3
    s += dpp_u32<0x142, 0xa, 0xf, false>(s);  // row_bcast:15 into rows 1, 3
    s += dpp_u32<0x143, 0xc, 0xf, false>(s);  // row_bcast:31 into rows 2, 3
    return s;
}

// Maximum over the 64 lanes of a wave, returned as a wave-uniform value.
__device__ static inline uint32_t wave_max_u32(uint32_t v)
{
    v = max(v, dpp_u32<0xb1, 0xf, 0xf, true>(v));   // quad_perm [1,0,3,2]
    v = max(v, dpp_u32<0x4e, 0xf, 0xf, true>(v));   // quad_perm [2,3,0,1]
    v = max(v, dpp_u32<0x141, 0xf, 0xf, true>(v));  // row_half_mirror
    v = max(v, dpp_u32<0x140, 0xf, 0xf, true>(v));  // row_mirror
    v = max(v, dpp_u32<0x142, 0xa, 0xf, false>(v)); // row_bcast:15
    v = max(v, dpp_u32<0x143, 0xc, 0xf, false>(v)); // row_bcast:31
    return (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
}

// Bitwise OR over the 64 lanes of a wave, returned as a wave-uniform value.
__device__ static inline uint32_t wave_or_u32(uint32_t v)
{
    v |= dpp_u32<0xb1, 0xf, 0xf, true>(v);   // quad_perm [1,0,3,2]
    v |= dpp_u32<0x4e, 0xf, 0xf, true>(v);   // quad_perm [2,3,0,1]
    v |= dpp_u32<0x141, 0xf, 0xf, true>(v);  // row_half_mirror
    v |= dpp_u32<0x140, 0xf, 0xf, true>(v);  // row_mirror
    v |= dpp_u32<0x142, 0xa, 0xf, false>(v); // row_bcast:15
    v |= dpp_u32<0x143, 0xc, 0xf, false>(v); // row_bcast:31
    return (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
}

__device__ static inline uint32_t uniform_u32(uint32_t v)
{
    return (uint32_t)__builtin_amdgcn_readfirstlane((int)v);
}

// ---------------------------------------------------------------- TIES sign election
// TIES's sign election and disjoint mean (Appendix A.1) over a lane's E
// elements: ps and ns hold the sums of the kept positive and negative deltas
// (added in increasing expert order), cpn their counts (positive in the low,
// negative in the high half, at most 32 each).  The sign whose rounded mass
// is larger in magnitude is elected; acc receives the elected sum divided by
// its count, correctly rounded, or 0 where no sign is elected (equal masses,
// nothing kept).  Every lane of the wave calls it together (it reads other
// lanes' registers); lane is the caller's index in the wave.
template <int E>
__device__ inline void ties_elect_mean(const float (&ps)[E], const float (&ns)[E], const uint32_t (&cpn)[E],
                                       float (&acc)[E], int lane)
{
    // elect by comparing the rounded masses P and -N; mean of the
    // agreeing entries (branch-free: every lane runs the same instructions)
    uint32_t den[E];
    uint32_t oddm = 0u;
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const bool up = ps[e] > -ns[e];
        const bool dn = ps[e] < -ns[e];
        acc[e] = up ? ps[e] : (dn ? ns[e] : 0.0f);  // never NaN: a NaN mass elects nothing
        // the elected sign's count (low half: positive, high half:
        // negative); with no elected sign acc is 0 and any count >= 1 gives 0
        den[e] = max(__builtin_amdgcn_ubfe(cpn[e], dn ? 16u : 0u, 16u), 1u);
        oddm |= den[e] & (den[e] - 1u);
    }
    const bool odd = oddm != 0u;
    bool tiny = false;
    if (__any(odd)) {
#pragma unroll
        for (int e = 0; e < E; ++e)
            tiny |= (fabsf(acc[e]) < 0x1p-100f) & (acc[e] != 0.0f);
    }
    if (!__any(odd)) {
        // counts that are powers of two divide by exact scaling, one
        // rounding of the quotient
#pragma unroll
        for (int e = 0; e < E; ++e)
            acc[e] = __builtin_amdgcn_ldexpf(acc[e], -(int)__builtin_ctz(den[e]));
    } else if (!__any(tiny)) {
        // The correctly rounded quotient acc / den (1 <= den <= 32)
        // without a division.  Lane j holds h + l, two terms of 1/j:
        // h <= 1/j within an ulp, l = max(fl32((1 - j h) h), 2^-126) > 0
        // (the residual 1 - j h is exact), |h + l - 1/j| < 2^-44 / j.  Then
        // fma(a, h, a l) lies within 2^-43 of a / den (relative).  When
        // a / den is a normal number, every rounding boundary (a midpoint
        // between neighbouring floats, which a / den never equals) lies
        // at least 2^-25 / den >= 2^-30 (relative) away from it, so both
        // round to the same value.  |a| >= 2^-100 keeps a / den and a l
        // clear of the subnormal range (smaller masses divide); l > 0,
        // so an infinite mass gives a l of its own sign and stays
        // infinite.
        const float fj = (float)(lane > 0 ? lane : 1);
        float h = __builtin_amdgcn_rcpf(fj);
        float r = fmaf(-fj, h, 1.0f);
        if (r < 0.0f) {  // the hardware reciprocal rounded up: one ulp down
            h = __uint_as_float(__float_as_uint(h) - 1u);
            r = fmaf(-fj, h, 1.0f);
        }
        const float l = fmaxf(r * h, 0x1p-126f);
#pragma unroll
        for (int e = 0; e < E; ++e) {
            const int src = (int)(den[e] << 2);
            const float he = __int_as_float(__builtin_amdgcn_ds_bpermute(src, __float_as_int(h)));
            const float le = __int_as_float(__builtin_amdgcn_ds_bpermute(src, __float_as_int(l)));
            acc[e] = fmaf(acc[e], he, acc[e] * le);
        }
    } else {
#pragma unroll
        for (int e = 0; e < E; ++e)
            acc[e] = acc[e] / (float)den[e];
    }
}

// SplitMix64 output function: the value SplitMix64 returns when its state
// before the step is x (Steele, Lea, Flood 2014).
__device__ static inline unsigned long long mix64(unsigned long long x)
{
    unsigned long long z = x + 0x9e3779b97f4a7c15ull;
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
    return z ^ (z >> 31);
}

}  // namespace mp
