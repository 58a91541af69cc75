// Helpers for the gfx950 bf16 matrix-core kernels (v_mfma_f32_16x16x32_bf16).
//
// Operand layouts used throughout: for a 16x16 result tile, lane
// (g = lane / 16, n = lane % 16) holds rows 4g + {0..3} of column n.  A
// 32-long contraction takes, in lane group g, the eight k-indices
// {4g .. 4g+3} and {16 + 4g .. 16 + 4g + 3} (element e < 4 and e >= 4 of the
// 8-wide operand), for both the A operand (row m = lane % 16) and the B
// operand (column n = lane % 16).  Any fixed assignment of k-indices to
// operand elements gives the same product as long as A and B agree; this one
// lets two stacked 16-row result tiles feed the next contraction directly.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mesa {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f32x4 mfma16(const bf16x8& a, const bf16x8& b, const f32x4& c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 pack8(const f32x4& lo, const f32x4& hi)
{
    bf16x8 r;
    r[0] = (__bf16)lo[0];
    r[1] = (__bf16)lo[1];
    r[2] = (__bf16)lo[2];
    r[3] = (__bf16)lo[3];
    r[4] = (__bf16)hi[0];
    r[5] = (__bf16)hi[1];
    r[6] = (__bf16)hi[2];
    r[7] = (__bf16)hi[3];
    return r;
}

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// Two fp32 rounded to bf16 (nearest even), packed as a | b << 16 (one conversion).
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b)
{
    const bf16x2 r = {(__bf16)a, (__bf16)b};
    return __builtin_bit_cast(uint32_t, r);
}

// Four fp32 rounded to bf16, as two 32-bit words (half of an 8-wide operand).
__device__ __forceinline__ uint2 pack4(const f32x4& v)
{
    const bf16x8 r = pack8(v, v);
    const uint4 u = __builtin_bit_cast(uint4, r);
    return make_uint2(u.x, u.y);
}

// Split of two fp32 values into bf16 high parts hi = bf16(x) (nearest even) and low
// parts lo = bf16(x - hi), each pair packed as a | b << 16: hi + lo carries x to
// ~2^-16 relative, so a product of two split operands, hi*hi + hi*lo + lo*hi with fp32
// accumulation, is accurate to that order.  The high parts are widened back to fp32
// from the packed word (a shift and a mask) rather than converted again.
__device__ __forceinline__ void split2(float x0, float x1, uint32_t& hi, uint32_t& lo)
{
    hi = pack_bf16x2(x0, x1);
    lo = pack_bf16x2(x0 - __uint_as_float(hi << 16), x1 - __uint_as_float(hi & 0xffff0000u));
}

// The split of the 8 values of one 8-wide operand (a -> elements 0..3, b -> 4..7).
__device__ __forceinline__ void split8(const f32x4& a, const f32x4& b, bf16x8& hi, bf16x8& lo)
{
    uint32_t h[4], l[4];
    split2(a[0], a[1], h[0], l[0]);
    split2(a[2], a[3], h[1], l[1]);
    split2(b[0], b[1], h[2], l[2]);
    split2(b[2], b[3], h[3], l[3]);
    hi = __builtin_bit_cast(bf16x8, make_uint4(h[0], h[1], h[2], h[3]));
    lo = __builtin_bit_cast(bf16x8, make_uint4(l[0], l[1], l[2], l[3]));
}

// 8 bf16 from LDS: base[0..3] and base[16..19] (the k-index map above).
__device__ __forceinline__ bf16x8 lds_frag(const uint16_t* base)
{
    const uint2 lo = *reinterpret_cast<const uint2*>(base);
    const uint2 hi = *reinterpret_cast<const uint2*>(base + 16);
    return __builtin_bit_cast(bf16x8, make_uint4(lo.x, lo.y, hi.x, hi.y));
}

// 16 bytes into an LDS row that is only 8-byte aligned, as two 8-byte stores.
__device__ __forceinline__ void put8x2(uint16_t* dst, const uint4& x)
{
    reinterpret_cast<uint2*>(dst)[0] = make_uint2(x.x, x.y);
    reinterpret_cast<uint2*>(dst)[1] = make_uint2(x.z, x.w);
}

// 8 fp32 from global memory, base[0..3] and base[16..19], rounded to bf16.
__device__ __forceinline__ bf16x8 gmem_frag(const float* base)
{
    const f32x4 lo = *reinterpret_cast<const f32x4*>(base);
    const f32x4 hi = *reinterpret_cast<const f32x4*>(base + 16);
    return pack8(lo, hi);
}

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t bits16) { return __uint_as_float(bits16 << 16); }

__device__ __forceinline__ uint16_t bf16_bits(__bf16 x) { return __builtin_bit_cast(uint16_t, x); }

// Transposed staging of two consecutive tokens (2p, 2p+1), 8 features each
// (bf16 bits in a and b), into a feature-major LDS tile of 32-bit words:
// word [(f0 + q) * ld32 + p] = (token 2p, token 2p+1) of feature f0 + q.
// Lanes with consecutive p write consecutive words, so a wave's stores do not
// collide in LDS banks.
__device__ __forceinline__ void stage_token_pair(uint32_t* dst32, int ld32, int f0, int p, const uint4& a,
                                                 const uint4& b)
{
    const uint32_t wa[4] = {a.x, a.y, a.z, a.w};
    const uint32_t wb[4] = {b.x, b.y, b.z, b.w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        dst32[(f0 + 2 * q) * ld32 + p] = (wa[q] & 0xffffu) | (wb[q] << 16);
        dst32[(f0 + 2 * q + 1) * ld32 + p] = (wa[q] >> 16) | (wb[q] & 0xffff0000u);
    }
}

// Direct global -> LDS load of one wave (gfx950 global_load_lds_dwordx4): lane l's
// 16 bytes at src land at lds + 16 l; lds must be the same in every lane.  The data
// is complete once the issuing wave's vector memory count has drained.  The builtin
// exists for the device pass only: in the host pass a kernel that names it would
// lose its launch stub, and the host never runs this code.
__device__ __forceinline__ void load_lds16(const void* src, void* lds)
{
#if defined(__HIP_DEVICE_COMPILE__)
    __builtin_amdgcn_global_load_lds(src, lds, 16, 0, 0);
#else
    (void)src;
    (void)lds;
#endif
}

// s_waitcnt operand that waits for the vector memory count to reach 0 and leaves
// the export and LDS/scalar counts alone (GFX9 encoding).
constexpr int kWaitVmcnt0 = 0x0F70;

}  // namespace mesa
