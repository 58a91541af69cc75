// Device-side helpers shared by the libmesa kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mesa {

constexpr int kWave = 64;

// bf16 values travel as raw 16-bit patterns; widening to fp32 is exact.
struct bf16_t {
    uint16_t bits;
};

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16_t x) { return __uint_as_float(uint32_t(x.bits) << 16); }

// Cross-lane data movement without LDS: DPP moves within 16-lane rows, and the
// gfx950 permlane swaps between rows.  DPP control codes (GFX9 encoding).
constexpr int kDppQuadSwap1 = 0xB1;  // quad_perm [1,0,3,2]
constexpr int kDppQuadSwap2 = 0x4E;  // quad_perm [2,3,0,1]
constexpr int kDppRowShr1 = 0x111;
constexpr int kDppRowShr2 = 0x112;
constexpr int kDppRowShr4 = 0x114;
constexpr int kDppRowShr8 = 0x118;
constexpr int kDppRowRor4 = 0x124;
constexpr int kDppRowRor8 = 0x128;
constexpr int kDppRowBcast15 = 0x142;  // last lane of a row to the whole next row
constexpr int kDppRowBcast31 = 0x143;  // lane 31 to rows 2 and 3

template <int Ctrl, int RowMask = 0xF>
__device__ __forceinline__ float dpp_f32(float old, float src)
{
    return __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(old), __float_as_int(src), Ctrl, RowMask, 0xF, false));
}

template <int Ctrl, int RowMask = 0xF>
__device__ __forceinline__ int dpp_i32(int old, int src)
{
    return __builtin_amdgcn_update_dpp(old, src, Ctrl, RowMask, 0xF, false);
}

// Sum over the four 16-lane rows: every lane receives the sum of its column position.
__device__ __forceinline__ float row_pair_sums(float v)
{
    const auto s16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = __uint_as_float(s16[0]) + __uint_as_float(s16[1]);
    const auto s32 = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(s32[0]) + __uint_as_float(s32[1]);
}

// Sum over all 64 lanes of a wave; every lane receives the total.
__device__ __forceinline__ float wave_sum(float x)
{
    x += dpp_f32<kDppQuadSwap1>(x, x);
    x += dpp_f32<kDppQuadSwap2>(x, x);
    x += dpp_f32<kDppRowRor4>(x, x);
    x += dpp_f32<kDppRowRor8>(x, x);
    return row_pair_sums(x);
}

// Inclusive prefix sum / prefix max over the 64 lanes of a wave.
__device__ __forceinline__ float wave_scan_add(float x)
{
    x += dpp_f32<kDppRowShr1>(0.0f, x);
    x += dpp_f32<kDppRowShr2>(0.0f, x);
    x += dpp_f32<kDppRowShr4>(0.0f, x);
    x += dpp_f32<kDppRowShr8>(0.0f, x);
    x += dpp_f32<kDppRowBcast15, 0xA>(0.0f, x);
    x += dpp_f32<kDppRowBcast31, 0xC>(0.0f, x);
    return x;
}

__device__ __forceinline__ int wave_scan_max(int x)
{
    x = max(x, dpp_i32<kDppRowShr1>(-1, x));
    x = max(x, dpp_i32<kDppRowShr2>(-1, x));
    x = max(x, dpp_i32<kDppRowShr4>(-1, x));
    x = max(x, dpp_i32<kDppRowShr8>(-1, x));
    x = max(x, dpp_i32<kDppRowBcast15, 0xA>(-1, x));
    x = max(x, dpp_i32<kDppRowBcast31, 0xC>(-1, x));
    return x;
}

// Value of lane `l` (a wave-uniform index) in every lane.
__device__ __forceinline__ float lane_value(float x, int l) { return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), l)); }
__device__ __forceinline__ int lane_value(int x, int l) { return __builtin_amdgcn_readlane(x, l); }
// x of lane src (0..63, per lane) through ds_bpermute.  HIP's __shfl also forms
// (lane & ~63) + src for its width argument, a per-lane value that the compiler keeps live
// (in the larger kernels, in a spill slot).
__device__ __forceinline__ float shfl_lane(float x, int src)
{
    return __int_as_float(__builtin_amdgcn_ds_bpermute(src << 2, __float_as_int(x)));
}

// Gate log-cumsums of one chunk (Sec. 2: zeta_{t,s} = prod_{s<i<=t} gamma_i).
// Called by the 64 lanes of ONE wave, for C <= 64 tokens starting at `gamma`
// (tokens at or beyond `valid` count as gamma = 1, i.e. absent).  For in-chunk
// token j it stores
//     lg[j] = sum_{s <= j, gamma_s > 0} log gamma_s
//     zl[j] = max{ s <= j : gamma_s == 0 }, or -1,
// from which, for i <= j,
//     prod_{s=i+1..j} gamma_s = (zl[j] > i) ? 0 : exp(lg[j] - lg[i])
//     prod_{s=0..j}   gamma_s = (zl[j] >= 0) ? 0 : exp(lg[j]).
// A zero gate therefore resets memory exactly instead of producing log(0).
__device__ __forceinline__ void chunk_log_decays(const float* gamma, int valid, float* lg, int* zl)
{
    const int lane = threadIdx.x & (kWave - 1);
    const float g = lane < valid ? gamma[lane] : 1.0f;
    const float s = wave_scan_add(g > 0.0f ? logf(g) : 0.0f);
    const int z = wave_scan_max((lane < valid && !(g > 0.0f)) ? lane : -1);
    lg[lane] = s;
    zl[lane] = z;
}

// prod_{s=i+1..j} gamma_s for in-chunk tokens i <= j (1 when i == j), 0 for i > j.
__device__ __forceinline__ float decay_between(const float* lg, const int* zl, int i, int j)
{
    if (i > j || zl[j] > i) return 0.0f;
    return expf(lg[j] - lg[i]);
}

// prod_{s=0..j} gamma_s: the decay from the chunk's entering state to token j.
__device__ __forceinline__ float decay_from_start(const float* lg, const int* zl, int j)
{
    return zl[j] >= 0 ? 0.0f : expf(lg[j]);
}

// Smallest normal fp32 number (2^-126).  The CG loops stop a column once p^T A p or
// |r|^2 falls below it (alpha would need the reciprocal of a subnormal, and the
// recursively updated residual goes on shrinking long after the true one stops
// improving); each column solves for q scaled by a power of two that brings |q|^2 into
// [1/2, 2), so the threshold is relative to |q|^2 and no rounding changes.
constexpr float kMinNormal = 1.17549435e-38f;

// log2 of the power-of-two scale that brings |q|^2 = qq into [1/2, 2) (0 for qq = 0)
__device__ __forceinline__ int cg_scale_shift(float qq) { return __builtin_amdgcn_frexp_expf(qq) >> 1; }

// Workgroups are dealt to the 8 XCDs round-robin (block b runs on XCD b % 8),
// and each XCD has its own L2.  This maps the hardware block index to a logical
// one so that logically consecutive workgroups share an XCD: workgroups that
// read the same inputs then hit one L2 instead of fetching them eight times.
constexpr int kNumXcd = 8;
__device__ __forceinline__ int xcd_major_block(int b, int n)
{
    const int per = n / kNumXcd, rem = n % kNumXcd;
    const int x = b % kNumXcd, local = b / kNumXcd;
    return x * per + min(x, rem) + local;
}

// A global load from a base address that every lane shares, at a 32-bit byte offset of the
// lane's own: the address is an SGPR base plus a 32-bit VGPR offset.  The empty asm makes
// the offset opaque, so it is formed next to its load; otherwise the compiler may form the
// offsets of loads that repeat (a tile fetched in several phases) once, as 64-bit
// addresses, and hold them across the kernel, which spilled in the backward gradient
// kernel (and each reload of a spilled address waited for every load in flight).
template <typename T>
__device__ __forceinline__ T load_at(const void* base, uint32_t byte_off)
{
    asm volatile("" : "+v"(byte_off));
    return *reinterpret_cast<const T*>(static_cast<const char*>(base) + byte_off);
}

}  // namespace mesa
