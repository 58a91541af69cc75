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

// Sum over all 64 lanes of a wave; every lane receives the total.
__device__ __forceinline__ float wave_sum(float x)
{
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) x += __shfl_xor(x, off, kWave);
    return x;
}

// Gate log-cumsums of one chunk (Sec. 3: zeta_{t,s} = prod_{s<i<=t} gamma_i).
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
    float s = g > 0.0f ? logf(g) : 0.0f;
    int z = (lane < valid && !(g > 0.0f)) ? lane : -1;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        const float so = __shfl_up(s, off, kWave);
        const int zo = __shfl_up(z, off, kWave);
        if (lane >= off) {
            s += so;
            z = max(z, zo);
        }
    }
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

}  // namespace mesa
