// Backward pass of the Mesa layer (App. D, "Mesa layer backward pass"), fp32.
//
// Given e_t = dL/do_t and the forward's solutions q*_t, the gradients are
//   e*_t = (H_t + Lambda)^{-1} G_t^T e_t              dL/dq_t = e*_t
//   dL/dLambda_a = -sum_t q*_{t,a} e*_{t,a}
// and, with the state adjoints DG_s = sum_{t>=s} zeta_{t,s} e_t q*_t^T and
// DH_s = -sum_{t>=s} zeta_{t,s} e*_t q*_t^T,
//   dL/dv_s = beta_s DG_s k_s,   dL/dk_s = beta_s (DG_s^T v_s + (DH_s + DH_s^T) k_s),
//   dL/dbeta_s = v_s^T DG_s k_s + k_s^T DH_s k_s,
//   dL/dgamma_s = <DG_s, G_{s-1}> + <DH_s, H_{s-1}>.
// (The paper's sums written with the input gate; the value term of dL/dk_s is
// q*_t e_t^T v_s, what differentiating e_t^T G_t q*_t gives.)
//
// Chunkwise, with E the last token of chunk n, the adjoints split into the part of
// the chunk's own tokens and the adjoint arriving from later chunks,
//   A^G_n = sum_{t>E} zeta_{t,E} e_t q*_t^T,   S^H_n = -sum_{t>E} zeta_{t,E} (e*_t q*_t^T + q*_t e*_t^T)
// (the symmetric part of the H adjoint is all the gradients need, since H is
// symmetric), scanned backwards as X_{n-1} = D_n X_n + sum_{j in n} zeta_{j,c-1} Y_j
// (the time reverse of the forward chunk scan).  Within a chunk every term is a
// C x C gram matrix of the chunk's tokens (gate-masked as in App. D) plus products
// with the four d x d matrices A^G_n, S^H_n, G_c, H_c; dL/dgamma uses the paper's
// trace rewriting, whose cross term is the diagonal of Z* Q Z.
//
// Launches (one stream): the forward chunk-state scan (fp32 states), the right-hand
// sides u_t = G_t^T e_t, the chunked CG solve of (H_t + Lambda) e*_t = u_t, the
// reverse adjoint scan, the per-chunk gradients, and the Lambda reduction.  Every
// product over tokens or features is a dense contraction of fp32 operands and runs
// on the matrix cores in fp32 (v_mfma_f32_16x16x4f32: exact fp32 products, fp32
// accumulation), 16 x 16 output tiles per wave.
#include <type_traits>

#include "mesa_device.hpp"
#include "mesa_kernels.hpp"
#include "mesa_mfma.hpp"

namespace mesa {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kC = 64;       // tokens per chunk of the backward
constexpr int kLdT = 132;    // row stride of [token][feature] tiles (16-byte aligned rows)
constexpr int kLdC = 68;     // row stride of [token][token] matrices (16-byte aligned rows)

// One 16 x 16 output tile += A (16 x K) B (K x 16) on the matrix cores, fp32:
// A(m, k) = A[m * AM + k * AK], B(k, n) = B[k * BK + n * BN].  With
// v_mfma_f32_16x16x4f32 lane l supplies one A(l % 16, k) and one B(k, l % 16) per step;
// element i of the result holds row 4 (l / 16) + i, column l % 16.  Step s of lane group
// sl = l / 16 contracts k = 16 (s / 4) + 4 sl + s % 4 (any assignment of the K indices to
// (step, group) gives the same product as long as A and B agree): a lane's four
// consecutive steps take four consecutive k, so an operand whose k runs along a row (stride
// 1, rows 16-byte aligned) comes in one 16-byte load per four steps.
template <int K, int M, int S>
__device__ __forceinline__ void load_opnd(const float* X, float (&v)[K / 4], int k0 = 0)
{
    static_assert(K % 16 == 0 && (S != 1 || M % 4 == 0), "16-byte operand rows");
    const int lane = threadIdx.x % kWave, r = lane % 16, sl = lane / 16;
    // all loads first (one round trip for the whole contraction); steps below k0 skipped
#pragma unroll
    for (int j = 0; j < K / 16; ++j) {
        if (16 * j + 16 <= k0) continue;
        if constexpr (S == 1) {
            const float4 f = *reinterpret_cast<const float4*>(X + r * M + 16 * j + 4 * sl);
            v[4 * j] = f.x;
            v[4 * j + 1] = f.y;
            v[4 * j + 2] = f.z;
            v[4 * j + 3] = f.w;
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) v[4 * j + e] = X[(16 * j + 4 * sl + e) * S + r * M];
        }
    }
}

template <int K>
__device__ __forceinline__ f32x4 mma_steps(const float (&av)[K / 4], const float (&bv)[K / 4], f32x4 acc, int k0 = 0)
{
#pragma unroll
    for (int i = 0; i < K / 4; ++i)
        if (16 * (i / 4) + 16 > k0) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av[i], bv[i], acc, 0, 0, 0);
    return acc;
}

template <int K, int AM, int AK, int BK, int BN>
__device__ __forceinline__ f32x4 mma16(const float* A, const float* B, f32x4 acc)
{
    float av[K / 4], bv[K / 4];
    load_opnd<K, AM, AK>(A, av);
    load_opnd<K, BN, BK>(B, bv);
    return mma_steps<K>(av, bv, acc);
}

// mma16 over contraction indices k0 .. K - 1 only (k0 a multiple of 16): for products
// with a causally masked matrix whose entries below k0 are zero.  The skipped steps are
// resolved at compile time wherever k0 is a constant of an unrolled loop.
template <int K, int AM, int AK, int BK, int BN>
__device__ __forceinline__ f32x4 mma16_from(const float* A, const float* B, int k0, f32x4 acc)
{
    float av[K / 4], bv[K / 4];
    load_opnd<K, AM, AK>(A, av, k0);
    load_opnd<K, BN, BK>(B, bv, k0);
    return mma_steps<K>(av, bv, acc, k0);
}

// The same product split in two: the B operand values of one tile (a global matrix,
// loaded one tile ahead so its latency overlaps the previous tile's products), then
// the products with A read from LDS.
template <int K, int BK, int BN>
__device__ __forceinline__ void load_b(const float* B, float (&bv)[K / 4])
{
    load_opnd<K, BN, BK>(B, bv);
}
template <int K, int AM, int AK>
__device__ __forceinline__ f32x4 mma16_b(const float* A, const float (&bv)[K / 4], f32x4 acc)
{
    float av[K / 4];
    load_opnd<K, AM, AK>(A, av);
    return mma_steps<K>(av, bv, acc);
}

constexpr f32x4 kZero4 = {0.0f, 0.0f, 0.0f, 0.0f};

// bf16 matrix-core products of the bf16 route (v_mfma_f32_16x16x32_bf16): in step b
// lane (g = l / 16, m = l % 16) supplies A(m, k) and B(k, m) for the eight k = 32 b + 4g +
// {0..3} and 32 b + 16 + 4g + {0..3}; the result tile has the layout of the fp32
// products above.  An fp32 operand enters split into bf16 high and low parts (x = hi +
// lo to ~2^-16 relative): a product of two split operands takes hi*hi + hi*lo + lo*hi, a
// product with an operand that is exact in bf16 (the route's keys and values) x*hi + x*lo.
// Operand values are held as fp32, [D / 32][8] per lane.

// Row operand from global memory: v[b] = row[32 b + 4g .. +3], row[32 b + 16 + 4g .. +3] of
// the row that starts at base + off (16-byte aligned rows).
template <int D>
__device__ __forceinline__ void load_row8(const float* base, int off, float (&v)[D / 32][8])
{
    const int g = (threadIdx.x % kWave) / 16;
#pragma unroll
    for (int b = 0; b < D / 32; ++b) {
        const float4 x = load_at<float4>(base, 4u * (off + 32 * b + 4 * g));
        const float4 y = load_at<float4>(base, 4u * (off + 32 * b + 16 + 4 * g));
        v[b][0] = x.x;
        v[b][1] = x.y;
        v[b][2] = x.z;
        v[b][3] = x.w;
        v[b][4] = y.x;
        v[b][5] = y.y;
        v[b][6] = y.z;
        v[b][7] = y.w;
    }
}
// The same from a row of an LDS tile.
template <int D>
__device__ __forceinline__ void lds_row8(const float* row, float (&v)[D / 32][8])
{
    const int g = (threadIdx.x % kWave) / 16;
#pragma unroll
    for (int b = 0; b < D / 32; ++b) {
        const float4 x = *reinterpret_cast<const float4*>(row + 32 * b + 4 * g);
        const float4 y = *reinterpret_cast<const float4*>(row + 32 * b + 16 + 4 * g);
        v[b][0] = x.x;
        v[b][1] = x.y;
        v[b][2] = x.z;
        v[b][3] = x.w;
        v[b][4] = y.x;
        v[b][5] = y.y;
        v[b][6] = y.z;
        v[b][7] = y.w;
    }
}
// Column operand of a row-major matrix: v[b][e] = base[k(b, e) * ld + col] for the lane's k.
template <int D>
__device__ __forceinline__ void load_col8(const float* base, int col, int ld, float (&v)[D / 32][8])
{
    const int g = (threadIdx.x % kWave) / 16;
#pragma unroll
    for (int b = 0; b < D / 32; ++b)
#pragma unroll
        for (int e = 0; e < 8; ++e)
            v[b][e] = load_at<float>(base, 4u * ((32 * b + (e < 4 ? 4 * g + e : 16 + 4 * g + e - 4)) * ld + col));
}
// The split operand of every step, hi[b] and lo[b].
template <int D>
__device__ __forceinline__ void split_steps(const float (&v)[D / 32][8], bf16x8 (&hi)[D / 32], bf16x8 (&lo)[D / 32])
{
#pragma unroll
    for (int b = 0; b < D / 32; ++b)
        split8(f32x4{v[b][0], v[b][1], v[b][2], v[b][3]}, f32x4{v[b][4], v[b][5], v[b][6], v[b][7]}, hi[b], lo[b]);
}
// The A values of step b from a row: row[32 b + 4g .. +3], row[32 b + 16 + 4g .. +3].
__device__ __forceinline__ void row_step(const float* row, int b, f32x4& x, f32x4& y)
{
    const int g = (threadIdx.x % kWave) / 16;
    x = *reinterpret_cast<const f32x4*>(row + 32 * b + 4 * g);
    y = *reinterpret_cast<const f32x4*>(row + 32 * b + 16 + 4 * g);
}
// acc += A B, A from the rows of an LDS tile holding values exact in bf16, B split
template <int D>
__device__ __forceinline__ f32x4 mma_xs(const float* arow, const bf16x8 (&bhi)[D / 32], const bf16x8 (&blo)[D / 32],
                                        f32x4 acc)
{
#pragma unroll
    for (int b = 0; b < D / 32; ++b) {
        f32x4 x0, x1;
        row_step(arow, b, x0, x1);
        const bf16x8 x = pack8(x0, x1);
        acc = mfma16(x, bhi[b], acc);
        acc = mfma16(x, blo[b], acc);
    }
    return acc;
}
// acc += A B, A from the rows of a bf16 LDS tile (exact), B split
template <int D>
__device__ __forceinline__ f32x4 mma_bs(const uint16_t* arow, const bf16x8 (&bhi)[D / 32], const bf16x8 (&blo)[D / 32],
                                        f32x4 acc)
{
    const int g = (threadIdx.x % kWave) / 16;
#pragma unroll
    for (int b = 0; b < D / 32; ++b) {
        const bf16x8 x = lds_frag(arow + 32 * b + 4 * g);
        acc = mfma16(x, bhi[b], acc);
        acc = mfma16(x, blo[b], acc);
    }
    return acc;
}
// acc += A B with both split (A from the rows of an fp32 LDS tile)
template <int D>
__device__ __forceinline__ f32x4 mma_ss(const float* arow, const bf16x8 (&bhi)[D / 32], const bf16x8 (&blo)[D / 32],
                                        f32x4 acc)
{
#pragma unroll
    for (int b = 0; b < D / 32; ++b) {
        f32x4 x0, x1;
        row_step(arow, b, x0, x1);
        bf16x8 ahi, alo;
        split8(x0, x1, ahi, alo);
        acc = mfma16(ahi, bhi[b], acc);
        acc = mfma16(ahi, blo[b], acc);
        acc = mfma16(alo, bhi[b], acc);
    }
    return acc;
}
// sum over the lane's elements of (hi + lo) y: a Frobenius product with the split
// values standing for the fp32 ones (to ~2^-16 relative)
template <int D>
__device__ __forceinline__ float dot_split(const bf16x8 (&hi)[D / 32], const bf16x8 (&lo)[D / 32], const float (&y)[D / 32][8])
{
    float s = 0.0f;
#pragma unroll
    for (int b = 0; b < D / 32; ++b)
#pragma unroll
        for (int e = 0; e < 8; ++e) s = fmaf((float)hi[b][e] + (float)lo[b][e], y[b][e], s);
    return s;
}

// Sum over the 16 lanes of a lane row (the columns of a result tile); every lane of
// the row receives it.
__device__ __forceinline__ float row16_sum(float x)
{
    x += dpp_f32<kDppQuadSwap1>(x, x);
    x += dpp_f32<kDppQuadSwap2>(x, x);
    x += dpp_f32<kDppRowRor4>(x, x);
    x += dpp_f32<kDppRowRor8>(x, x);
    return x;
}

// [token][feature] tile of a chunk (rows past `valid` zero) into LDS rows of `ld` floats:
// 16-byte global loads (4 fp32 or 8 bf16), every load of the thread issued before the
// first store.  Rows past the end re-read the last valid token and are zeroed.
template <int D, int LD = kLdT>
__device__ __forceinline__ void load_tile(float* dst, const float* src, int64_t tok0, int valid)
{
    constexpr int V = kC * D / 4 / kThreads;  // float4 per thread
    float4 x[V];
#pragma unroll
    for (int m = 0; m < V; ++m) {
        const int e = threadIdx.x + kThreads * m, i = e / (D / 4), f = 4 * (e % (D / 4));
        x[m] = *reinterpret_cast<const float4*>(src + (tok0 + min(i, valid - 1)) * D + f);
    }
#pragma unroll
    for (int m = 0; m < V; ++m) {
        const int e = threadIdx.x + kThreads * m, i = e / (D / 4), f = 4 * (e % (D / 4));
        const bool ok = i < valid;
        float* o = dst + i * LD + f;
        o[0] = ok ? x[m].x : 0.0f;
        o[1] = ok ? x[m].y : 0.0f;
        o[2] = ok ? x[m].z : 0.0f;
        o[3] = ok ? x[m].w : 0.0f;
    }
}
template <int D, int LD = kLdT>
__device__ __forceinline__ void load_tile(float* dst, const bf16_t* src, int64_t tok0, int valid)
{
    constexpr int V = kC * D / 8 / kThreads;  // 8-element loads per thread
    uint4 x[V];
#pragma unroll
    for (int m = 0; m < V; ++m) {
        const int e = threadIdx.x + kThreads * m, i = e / (D / 8), f = 8 * (e % (D / 8));
        x[m] = *reinterpret_cast<const uint4*>(src + (tok0 + min(i, valid - 1)) * D + f);
    }
#pragma unroll
    for (int m = 0; m < V; ++m) {
        const int e = threadIdx.x + kThreads * m, i = e / (D / 8), f = 8 * (e % (D / 8));
        const bool ok = i < valid;
        const uint32_t w4[4] = {x[m].x, x[m].y, x[m].z, x[m].w};
        float* o = dst + i * LD + f;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            o[2 * q] = ok ? __uint_as_float(w4[q] << 16) : 0.0f;
            o[2 * q + 1] = ok ? __uint_as_float(w4[q] & 0xffff0000u) : 0.0f;
        }
    }
}

// The same tile in two steps, so its global loads can be in flight while the previous
// phase computes: fetch issues the 16-byte loads into registers, put (after the LDS
// tile is free) zeroes rows past `valid` and stores it.
template <int D, typename T, int NT = kThreads>
struct Tile;
template <int D, int NT>
struct Tile<D, float, NT> {
    static constexpr int V = kC * D / 4 / NT;
    float4 x[V];
    __device__ __forceinline__ void fetch(const float* src, int64_t tok0, int valid)
    {
#pragma unroll
        for (int m = 0; m < V; ++m) {
            const int e = threadIdx.x + NT * m, i = e / (D / 4), f = 4 * (e % (D / 4));
            x[m] = load_at<float4>(src + tok0 * D, 4u * (min(i, valid - 1) * D + f));
        }
    }
    __device__ __forceinline__ void put(float* dst, int valid) const
    {
#pragma unroll
        for (int m = 0; m < V; ++m) {
            const int e = threadIdx.x + NT * m, i = e / (D / 4), f = 4 * (e % (D / 4));
            const bool ok = i < valid;
            float* o = dst + i * kLdT + f;
            o[0] = ok ? x[m].x : 0.0f;
            o[1] = ok ? x[m].y : 0.0f;
            o[2] = ok ? x[m].z : 0.0f;
            o[3] = ok ? x[m].w : 0.0f;
        }
    }
};
template <int D, int NT>
struct Tile<D, bf16_t, NT> {
    static constexpr int V = kC * D / 8 / NT;
    uint4 x[V];
    // the tile as bf16, rows of `ld` elements (8-byte aligned), rows past `valid` zero
    __device__ __forceinline__ void put_bf16(uint16_t* dst, int ld, int valid) const
    {
#pragma unroll
        for (int m = 0; m < V; ++m) {
            const int e = threadIdx.x + NT * m, i = e / (D / 8), f = 8 * (e % (D / 8));
            const uint4 v = i < valid ? x[m] : make_uint4(0u, 0u, 0u, 0u);
            uint2* o = reinterpret_cast<uint2*>(dst + i * ld + f);
            o[0] = make_uint2(v.x, v.y);
            o[1] = make_uint2(v.z, v.w);
        }
    }
    __device__ __forceinline__ void fetch(const bf16_t* src, int64_t tok0, int valid)
    {
#pragma unroll
        for (int m = 0; m < V; ++m) {
            const int e = threadIdx.x + NT * m, i = e / (D / 8), f = 8 * (e % (D / 8));
            x[m] = load_at<uint4>(src + tok0 * D, 2u * (min(i, valid - 1) * D + f));
        }
    }
    __device__ __forceinline__ void put(float* dst, int valid) const
    {
#pragma unroll
        for (int m = 0; m < V; ++m) {
            const int e = threadIdx.x + NT * m, i = e / (D / 8), f = 8 * (e % (D / 8));
            const bool ok = i < valid;
            const uint32_t w4[4] = {x[m].x, x[m].y, x[m].z, x[m].w};
            float* o = dst + i * kLdT + f;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                o[2 * q] = ok ? __uint_as_float(w4[q] << 16) : 0.0f;
                o[2 * q + 1] = ok ? __uint_as_float(w4[q] & 0xffff0000u) : 0.0f;
            }
        }
    }
};

// ---------------------------------------------------------------- u = G^T e
// u_t = zeta_{t,c-1} G_c^T e_t + sum_{i<=t} zeta_{t,i} beta_i (v_i . e_t) k_i for
// the tokens of one chunk (the GLA form of App. D with the roles of k and v swapped).
// Wave w owns tokens t = 16w .. 16w+15, as the columns of transposed products:
// S^T = V E^T (rows i, the gate weights applied in place) stays in the result
// registers and is the B operand of K^T S^T (in the product for element r of row
// tile it, k-slot g stands for token i = 16 it + 4 g + r, exactly the element lane
// (g, n) holds), and u^T = zeta ⊙ (G_c^T E^T) + K^T S^T comes out as [feature][token]
// tiles, four consecutive features of one token per lane.  No C x C matrix goes
// through LDS, so two workgroups share a compute unit.  On the bf16 route the three
// products run on the bf16 matrix cores with split operands: V E^T and K^T S^T with E and
// S^T split (values and keys are exact in bf16, two passes per 32-long step), G_c^T E^T
// with both split (three passes).
template <typename Tin, int DK, int DV>
__global__ __launch_bounds__(kThreads) void bwd_rhs_kernel(BwdArgs a)
{
    const ForwardShape s = a.s;
    const int nc = s.n_chunks;
    const int n = blockIdx.x % nc;
    const int64_t bh = blockIdx.x / nc;
    const int64_t t0 = int64_t(n) * kC;
    const int valid = int(min<int64_t>(kC, s.seq_len - t0));
    const int64_t tok0 = bh * s.seq_len + t0;
    const int tid = threadIdx.x;
    const int w = __builtin_amdgcn_readfirstlane(tid / kWave), lane = tid % kWave, g = lane / 16, ln = lane % 16;
    const int t = 16 * w + ln;  // this lane's token (column of the transposed products)

    __shared__ __attribute__((aligned(16))) float sE[kC * kLdT];   // e_t [t][a]
    __shared__ __attribute__((aligned(16))) float sX[kC * kLdT];   // v_i, then k_i
    __shared__ float sLg[kC];
    __shared__ int sZl[kC];

    load_tile<DV>(sX, static_cast<const Tin*>(a.v), tok0, valid);
    load_tile<DV>(sE, a.dout, tok0, valid);
    if (tid < kWave) chunk_log_decays(a.gamma + tok0, valid, sLg, sZl);
    Tile<DK, Tin> tk;  // the keys, in flight during the value products
    tk.fetch(static_cast<const Tin*>(a.k), tok0, valid);
    __syncthreads();
    // S^T[i][t] = beta_i zeta_{t,i} (v_i . e_t) for i <= t (0 otherwise and past the end);
    // row tiles it > w lie wholly above this wave's tokens and are zero
    constexpr bool kSplit = std::is_same<Tin, bf16_t>::value;
    f32x4 sT[kC / 16];
    bf16x8 ehi[DV / 32], elo[DV / 32];  // bf16 route: e_t, this lane's token, split
    if constexpr (kSplit) {
        float ev[DV / 32][8];
        lds_row8<DV>(sE + (16 * w + ln) * kLdT, ev);
        split_steps<DV>(ev, ehi, elo);
    }
#pragma unroll
    for (int it = 0; it < kC / 16; ++it) {
        if (it > w) {
            sT[it] = kZero4;
            continue;
        }
        f32x4 ve;
        if constexpr (kSplit)
            ve = mma_xs<DV>(sX + (16 * it + ln) * kLdT, ehi, elo, kZero4);
        else
            ve = mma16<DV, kLdT, 1, 1, kLdT>(sX + 16 * it * kLdT, sE + 16 * w * kLdT, kZero4);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int i = 16 * it + 4 * g + r;
            sT[it][r] = (i <= t && i < valid) ? a.beta[tok0 + i] * decay_between(sLg, sZl, i, t) * ve[r] : 0.0f;
        }
    }
    // E^T as the B operand of every G_c^T E^T tile: B(k = a, n = t) = e_t[a] (fp32 route;
    // the bf16 route has it split in ehi, elo)
    float eb[DV / 4];
    if constexpr (!kSplit) {
#pragma unroll
        for (int i = 0; i < DV / 4; ++i) eb[i] = sE[t * kLdT + 4 * i + g];
    }
    // bf16 route: S^T as the B operand of K^T S^T, step s = token tiles 2s, 2s + 1 (the
    // k-slots of lane group g are exactly the tokens this lane holds), split
    bf16x8 shi[2], slo[2];
    if constexpr (kSplit) {
#pragma unroll
        for (int u = 0; u < 2; ++u) split8(sT[2 * u], sT[2 * u + 1], shi[u], slo[u]);
    }
    __syncthreads();
    tk.put(sX, valid);
    __syncthreads();
    const float zs = decay_from_start(sLg, sZl, t);
    // A operand of G_c^T E^T for feature tile bt: A(m = b, k = a) = G_c[a][16 bt + m], one
    // tile ahead
    const float* Gc = a.Gs + (bh * nc + n) * int64_t(DV) * DK;
    auto load_ga = [&](int bt, float (&ga)[DV / 4]) {
        if constexpr (kSplit) {
            // the bf16 k-map: step b takes a = 32 b + 4g + {0..3} and 32 b + 16 + 4g + {0..3}
            load_col8<DV>(Gc, 16 * bt + ln, DK, reinterpret_cast<float (&)[DV / 32][8]>(ga));
        } else {
#pragma unroll
            for (int i = 0; i < DV / 4; ++i) ga[i] = Gc[(4 * i + g) * DK + 16 * bt + ln];
        }
    };
    float ga[2][DV / 4];
    load_ga(0, ga[0]);
#pragma unroll
    for (int bt = 0; bt < DK / 16; ++bt) {
        if (bt + 1 < DK / 16) load_ga(bt + 1, ga[(bt + 1) % 2]);
        f32x4 eg = kZero4;
        if constexpr (kSplit) {
            bf16x8 ghi[DV / 32], glo[DV / 32];
            split_steps<DV>(reinterpret_cast<const float (&)[DV / 32][8]>(ga[bt % 2]), ghi, glo);
#pragma unroll
            for (int b = 0; b < DV / 32; ++b) {
                eg = mfma16(ghi[b], ehi[b], eg);
                eg = mfma16(ghi[b], elo[b], eg);
                eg = mfma16(glo[b], ehi[b], eg);
            }
        } else {
#pragma unroll
            for (int i = 0; i < DV / 4; ++i) eg = __builtin_amdgcn_mfma_f32_16x16x4f32(ga[bt % 2][i], eb[i], eg, 0, 0, 0);
        }
        // K^T S^T: A(m = b, k = i) = k_i[16 bt + m] with i = 16 it + 4 g + r (the zero
        // tiles it > w skipped)
        f32x4 sk = kZero4;
        if constexpr (kSplit) {
            // step u: tokens 32u + 4g + e and 32u + 16 + 4g + e (exact in bf16)
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                if (2 * u > w) continue;
                f32x4 k0, k1;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    k0[e] = sX[(32 * u + 4 * g + e) * kLdT + 16 * bt + ln];
                    k1[e] = sX[(32 * u + 16 + 4 * g + e) * kLdT + 16 * bt + ln];
                }
                const bf16x8 kb = pack8(k0, k1);
                sk = mfma16(kb, shi[u], sk);
                sk = mfma16(kb, slo[u], sk);
            }
        } else {
            float ka[kC / 4];
#pragma unroll
            for (int it = 0; it < kC / 16; ++it) {
                if (it > w) continue;
#pragma unroll
                for (int r = 0; r < 4; ++r) ka[4 * it + r] = sX[(16 * it + 4 * g + r) * kLdT + 16 * bt + ln];
            }
#pragma unroll
            for (int it = 0; it < kC / 16; ++it) {
                if (it > w) continue;
#pragma unroll
                for (int r = 0; r < 4; ++r) sk = __builtin_amdgcn_mfma_f32_16x16x4f32(ka[4 * it + r], sT[it][r], sk, 0, 0, 0);
            }
        }
        // lane (g, n): u_t[16 bt + 4g + r], r = 0..3
        if (t < valid) {
            const f32x4 u = zs * eg + sk;
            const int64_t o = (tok0 + t) * DK + 16 * bt + 4 * g;
            if (a.u16)
                *reinterpret_cast<uint2*>(a.u16 + o) = make_uint2(pack_bf16x2(u[0], u[1]), pack_bf16x2(u[2], u[3]));  // nearest even
            else
                *reinterpret_cast<float4*>(a.u + o) = make_float4(u[0], u[1], u[2], u[3]);
        }
    }
}

// ---------------------------------------------------------------- adjoint scan
// One workgroup owns 64 rows of S^H (d_k x d_k) or of A^G (d_v x d_k) of one
// sequence and walks the chunks from last to first; wave w keeps rows 16w .. +15 of
// the slice as d_k / 16 result tiles in registers and adds each chunk's rank-64
// update on the matrix cores.  The gate weight zeta_{j,c-1} is folded into the row
// operands as they are staged.
// Few long sequences walk in segments, in time reverse of the forward scan's: a first
// launch computes each later segment's contribution from a zero state, T_s, and its decay
// D_s; the second starts segment s from E_s = sum_{t>s} (D_{s+1} ... D_{t-1}) T_t.
// On the bf16 route (SPLIT) the rank-64 products run on the bf16 matrix cores with both
// operands split into high and low parts (hi*hi + hi*lo + lo*hi, ~2^-16 relative; the
// fp32 route keeps exact fp32 products): the operands are staged transposed, one bf16
// plane each for the high and low parts, two tokens per 32-bit word.
constexpr int kAdjRows = 64;
constexpr int kLdX = 144;   // row stride of the [token][column] operands (16 banks apart)
constexpr int kLdR = 80;    // row stride of the [token][row] operands
// Row stride in 32-bit words of the split [feature][token] planes.  An 8-byte LDS read
// serves 16 lanes at a time from 32 four-byte banks; the 16 rows of an operand fragment then
// start 2 banks apart (34 = 2 mod 32) and fill the banks once.  With 36 (4 apart) rows 8
// apart shared banks and every fragment read took twice its cycles (14.2k of ~160k cycles
// per wave were bank-conflict stalls at d = 128; 0.4k with 34).
constexpr int kLdP = 34;

struct AdjSeg {
    int len;      // chunks per segment (the last may be shorter)
    int total;    // segments of a sequence
    int first;    // first segment this launch walks
    int count;    // segments this launch walks
    bool totals;  // write T_s and D_s instead of the per-chunk adjoints
    float* tot;   // [B*H, total, d_k (d_k + d_v)]: T_s of S^H then of A^G (chunk layout)
    float* dec;   // [B*H, total]: D_s
};

template <int DK, int DV, bool SPLIT>
__global__ __launch_bounds__(kThreads, 2) void bwd_adjoint_kernel(BwdArgs a, AdjSeg sg)
{
    constexpr int NCT = DK / 16;                  // column tiles
    constexpr int NTH = DK / kAdjRows;            // row slices of S^H
    constexpr int NTILE = NTH + DV / kAdjRows;    // then row slices of A^G
    const ForwardShape s = a.s;
    const int nc = s.n_chunks;
    const int blk = xcd_major_block(blockIdx.x, gridDim.x);
    const int tile = blk % NTILE;
    const int seg = sg.first + (blk / NTILE) % sg.count;
    const int64_t bh = blk / NTILE / sg.count;
    const int nbeg = seg * sg.len, nend = min(nbeg + sg.len, nc);  // this segment's chunks
    const bool isG = tile >= NTH;
    const int r0 = (isG ? tile - NTH : tile) * kAdjRows;
    const int nrow = isG ? DV : DK;
    const int tid = threadIdx.x;
    const int w = tid / kWave, lane = tid % kWave, g = lane / 16, ln = lane % 16;
    constexpr int64_t kSegElems = int64_t(DK) * (DK + DV);
    // this thread's elements of segment t's total: rows r0 + 16w + 4g + r, columns 16 ct + ln
    auto seg_tile = [&](int t) { return sg.tot + (bh * sg.total + t) * kSegElems + (isG ? DK * DK : 0) +
                                        int64_t(r0 + 16 * w + 4 * g) * DK + ln; };

    // One pass per rank-64 product: the token tile goes to sX, the weighted row slice to
    // sYr.  A^G has one pass per chunk (q*, zeta e), S^H two (q*, -zeta e*) and (e*, -zeta q*).
    // The inputs of the next pass are fetched into registers while this one multiplies.
    // fp32: token tile [j][c] (sX) and weighted row slice [j][r] (rows r0.., sYr);
    // SPLIT: the same transposed as bf16 planes, [c][j] and [r][j], high then low parts
    constexpr int kFloats = SPLIT ? 2 * (DK + kAdjRows) * kLdP : kC * (kLdX + kLdR);
    __shared__ __attribute__((aligned(16))) float sBuf[kFloats];
    float* const sX = sBuf;
    float* const sYr = sBuf + kC * kLdX;
    uint32_t* const pXh = reinterpret_cast<uint32_t*>(sBuf);
    uint32_t* const pXl = pXh + DK * kLdP;
    uint32_t* const pYh = pXl + DK * kLdP;
    uint32_t* const pYl = pYh + kAdjRows * kLdP;
    __shared__ float sW[kC];
    __shared__ float sLg[kC];
    __shared__ int sZl[kC];

    f32x4 st[NCT];
#pragma unroll
    for (int ct = 0; ct < NCT; ++ct) st[ct] = kZero4;
    if (!sg.totals) {
        // the adjoint arriving from the later segments
        float c = 1.0f;
        for (int t = seg + 1; t < sg.total; ++t) {
            const float* tb = seg_tile(t);
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
                for (int r = 0; r < 4; ++r) st[ct][r] += c * tb[r * DK + 16 * ct];
            c *= sg.dec[bh * sg.total + t];
        }
    }
    constexpr int VT = kC * DK / 4 / kThreads;        // tile: 16-byte pieces per thread
    constexpr int VR = kC * kAdjRows / 4 / kThreads;  // row slice: 16-byte pieces per thread
    struct PassRegs {
        float4 t[VT], r[VR];
    };
    // The thread's 16-byte pieces: piece m is token j, columns (rows) f .. f + 3.  SPLIT
    // pairs the pieces, tokens 2q and 2q + 1 at the same columns, so a column's two values
    // form one 32-bit word of the transposed planes; consecutive lanes take consecutive
    // token pairs, so a wave's stores of one column fall in distinct banks.  SPLIT also
    // starts the tile's columns at r0 (mod d_k), so that pieces 0 .. 3 hold this workgroup's
    // row slice r0 .. r0 + 63 (S^H takes its row operand from them).
    auto tile_piece = [&](int m, int& j, int& f) {
        const int e = tid + kThreads * (SPLIT ? m / 2 : m);
        j = SPLIT ? 2 * (e % (kC / 2)) + m % 2 : e / (DK / 4);
        f = SPLIT ? (4 * (e / (kC / 2)) + r0) % DK : 4 * (e % (DK / 4));
    };
    auto row_piece = [&](int m, int& j, int& r) {
        const int e = tid + kThreads * (SPLIT ? m / 2 : m);
        j = SPLIT ? 2 * (e % (kC / 2)) + m % 2 : e / (kAdjRows / 4);
        r = 4 * (SPLIT ? e / (kC / 2) : e % (kAdjRows / 4));
    };
    // pass p of chunk n: tokens past the end re-read the last valid one (zeroed in put)
    auto fetch = [&](int n, int p, PassRegs& R) {
        const int64_t t0 = int64_t(n) * kC;
        const int valid = int(min<int64_t>(kC, s.seq_len - t0));
        const int64_t tok0 = bh * s.seq_len + t0;
        const float* ts = (isG || p == 0) ? a.qstar : a.estar;
        const float* rs = isG ? a.dout : (p == 0 ? a.estar : a.qstar);
        const int rd = isG ? DV : DK;
#pragma unroll
        for (int m = 0; m < VT; ++m) {
            int j, f;
            tile_piece(m, j, f);
            R.t[m] = *reinterpret_cast<const float4*>(ts + (tok0 + min(j, valid - 1)) * DK + f);
        }
#pragma unroll
        for (int m = 0; m < VR; ++m) {
            int j, r;
            row_piece(m, j, r);
            R.r[m] = *reinterpret_cast<const float4*>(rs + (tok0 + min(j, valid - 1)) * rd + r0 + r);
        }
    };
    // tile rows past `valid` zeroed; row slice weighted by zeta_{j,c-1} (zero past the end),
    // negated for S^H
    auto put = [&](const PassRegs& R, int valid) {
        if constexpr (SPLIT) {
#pragma unroll
            for (int m = 0; m < VT; m += 2) {
                int j, f;
                tile_piece(m, j, f);
                const float4 x0 = j < valid ? R.t[m] : float4{0.0f, 0.0f, 0.0f, 0.0f};
                const float4 x1 = j + 1 < valid ? R.t[m + 1] : float4{0.0f, 0.0f, 0.0f, 0.0f};
                const float a0[4] = {x0.x, x0.y, x0.z, x0.w}, a1[4] = {x1.x, x1.y, x1.z, x1.w};
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    uint32_t hi, lo;
                    split2(a0[i], a1[i], hi, lo);
                    pXh[(f + i) * kLdP + j / 2] = hi;
                    pXl[(f + i) * kLdP + j / 2] = lo;
                }
            }
#pragma unroll
            for (int m = 0; m < VR; m += 2) {
                int j, r;
                row_piece(m, j, r);
                const float w0 = j < valid ? (isG ? sW[j] : -sW[j]) : 0.0f;
                const float w1 = j + 1 < valid ? (isG ? sW[j + 1] : -sW[j + 1]) : 0.0f;
                const float a0[4] = {R.r[m].x, R.r[m].y, R.r[m].z, R.r[m].w};
                const float a1[4] = {R.r[m + 1].x, R.r[m + 1].y, R.r[m + 1].z, R.r[m + 1].w};
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    uint32_t hi, lo;
                    split2(w0 * a0[i], w1 * a1[i], hi, lo);
                    pYh[(r + i) * kLdP + j / 2] = hi;
                    pYl[(r + i) * kLdP + j / 2] = lo;
                }
            }
            return;
        }
#pragma unroll
        for (int m = 0; m < VT; ++m) {
            const int e = tid + kThreads * m, j = e / (DK / 4), f = 4 * (e % (DK / 4));
            const bool ok = j < valid;
            float* o = sX + j * kLdX + f;
            o[0] = ok ? R.t[m].x : 0.0f;
            o[1] = ok ? R.t[m].y : 0.0f;
            o[2] = ok ? R.t[m].z : 0.0f;
            o[3] = ok ? R.t[m].w : 0.0f;
        }
#pragma unroll
        for (int m = 0; m < VR; ++m) {
            const int e = tid + kThreads * m, j = e / (kAdjRows / 4), r = 4 * (e % (kAdjRows / 4));
            const float wy = isG ? sW[j] : -sW[j];
            float* o = sYr + j * kLdR + r;
            o[0] = wy * R.r[m].x;
            o[1] = wy * R.r[m].y;
            o[2] = wy * R.r[m].z;
            o[3] = wy * R.r[m].w;
        }
    };
    // X[r][c] += sum_j Yr[j][r] T[j][c]  (A(m, k) = sYr[k][m], B(k, n) = sX[k][n])
    // SPLIT: in step b lane (g, m) takes tokens 32 b + 4g .. + 3 and 32 b + 16 + 4g .. + 3
    // of plane row m (the bf16 product convention above), two 8-byte reads per plane
    auto frag = [&](const uint32_t* plane, int row, int b) {
        const uint32_t* q = plane + row * kLdP + 16 * b + 2 * g;
        const uint2 u0 = *reinterpret_cast<const uint2*>(q);
        const uint2 u1 = *reinterpret_cast<const uint2*>(q + 8);
        return __builtin_bit_cast(bf16x8, make_uint4(u0.x, u0.y, u1.x, u1.y));
    };
    auto multiply = [&](f32x4 (&acc)[NCT]) {
        if constexpr (SPLIT) {
#pragma unroll
            for (int b = 0; b < kC / 32; ++b) {
                const bf16x8 ah = frag(pYh, 16 * w + ln, b), al = frag(pYl, 16 * w + ln, b);
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct) {
                    const bf16x8 bh_ = frag(pXh, 16 * ct + ln, b), bl = frag(pXl, 16 * ct + ln, b);
                    acc[ct] = mfma16(ah, bh_, acc[ct]);
                    acc[ct] = mfma16(ah, bl, acc[ct]);
                    acc[ct] = mfma16(al, bh_, acc[ct]);
                }
            }
        } else {
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) acc[ct] = mma16<kC, 1, kLdR, kLdX, 1>(sYr + 16 * w, sX + 16 * ct, acc[ct]);
        }
    };
    float dprod = 1.0f;
    float* out = isG ? a.AG : a.SH;
    // the adjoint arriving at this chunk's end goes out; the chunk's gates into sLg, sZl, sW
    auto chunk_head = [&](int n, int valid, int64_t tok0) {
        if (!sg.totals) {
            float* dst = out + ((bh * nc + n) * nrow + r0 + 16 * w) * int64_t(DK);
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
                for (int r = 0; r < 4; ++r) dst[(4 * g + r) * DK + 16 * ct + ln] = st[ct][r];
        }
        if (tid < kWave) {
            chunk_log_decays(a.gamma + tok0, valid, sLg, sZl);
            sW[tid] = tid < valid ? decay_from_start(sLg, sZl, tid) : 0.0f;  // own lane's values
        }
    };
    if constexpr (SPLIT) {
        // A chunk's q* and e* tiles are fetched once for both passes of S^H: each is the token
        // tile of one pass and, where its features fall in this workgroup's row slice, the
        // weighted row operand of the other (the row slice r0 .. r0 + 63 is a column range of
        // the tile: its pieces 0 .. 3).  A^G takes the q* tile
        // and its own rows of dout.  The next chunk's data is fetched once this chunk's last
        // put has read the registers, and is in flight during its last product.
        float4 TA[VT], TB[VT];  // S^H: q*, e*; A^G: q*, dout rows (TB[0 .. VR - 1])
        auto fetch_chunk = [&](int n) {
            const int64_t t0 = int64_t(n) * kC;
            const int valid = int(min<int64_t>(kC, s.seq_len - t0));
            const int64_t tok0 = bh * s.seq_len + t0;
#pragma unroll
            for (int m = 0; m < VT; ++m) {
                int j, f;
                tile_piece(m, j, f);
                TA[m] = *reinterpret_cast<const float4*>(a.qstar + (tok0 + min(j, valid - 1)) * DK + f);
            }
            if (!isG) {
#pragma unroll
                for (int m = 0; m < VT; ++m) {
                    int j, f;
                    tile_piece(m, j, f);
                    TB[m] = *reinterpret_cast<const float4*>(a.estar + (tok0 + min(j, valid - 1)) * DK + f);
                }
            } else {
#pragma unroll
                for (int m = 0; m < VR; ++m) {
                    int j, r;
                    row_piece(m, j, r);
                    TB[m] = *reinterpret_cast<const float4*>(a.dout + (tok0 + min(j, valid - 1)) * DV + r0 + r);
                }
            }
        };
        // token tile planes from T (rows past `valid` zero)
        auto put_x = [&](const float4 (&T)[VT], int valid) {
#pragma unroll
            for (int m = 0; m < VT; m += 2) {
                int j, f;
                tile_piece(m, j, f);
                const float4 x0 = j < valid ? T[m] : float4{0.0f, 0.0f, 0.0f, 0.0f};
                const float4 x1 = j + 1 < valid ? T[m + 1] : float4{0.0f, 0.0f, 0.0f, 0.0f};
                const float a0[4] = {x0.x, x0.y, x0.z, x0.w}, a1[4] = {x1.x, x1.y, x1.z, x1.w};
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    uint32_t hi, lo;
                    split2(a0[i], a1[i], hi, lo);
                    pXh[(f + i) * kLdP + j / 2] = hi;
                    pXl[(f + i) * kLdP + j / 2] = lo;
                }
            }
        };
        // row planes: pieces (m, m + 1) of T hold rows r .. r + 3 of tokens j, j + 1, each
        // weighted by sgn zeta_{j,c-1} (zero past `valid`)
        auto put_y_pair = [&](const float4& y0, const float4& y1, int j, int r, int valid, float sgn) {
            const float w0 = j < valid ? sgn * sW[j] : 0.0f;
            const float w1 = j + 1 < valid ? sgn * sW[j + 1] : 0.0f;
            const float a0[4] = {y0.x, y0.y, y0.z, y0.w}, a1[4] = {y1.x, y1.y, y1.z, y1.w};
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                uint32_t hi, lo;
                split2(w0 * a0[i], w1 * a1[i], hi, lo);
                pYh[(r + i) * kLdP + j / 2] = hi;
                pYl[(r + i) * kLdP + j / 2] = lo;
            }
        };
        auto put_y_rows = [&](const float4 (&R)[VT], int valid) {  // A^G: dout rows, +zeta
#pragma unroll
            for (int m = 0; m < VR; m += 2) {
                int j, r;
                row_piece(m, j, r);
                put_y_pair(R[m], R[m + 1], j, r, valid, 1.0f);
            }
        };
        auto put_y_tile = [&](const float4 (&T)[VT], int valid) {  // S^H: the tile's slice, -zeta
#pragma unroll
            for (int m = 0; m < 4; m += 2) {
                int j, f;
                tile_piece(m, j, f);
                put_y_pair(T[m], T[m + 1], j, f - r0, valid, -1.0f);
            }
        };
        static_assert(kAdjRows == 64 && VR == 4 && VT % 4 == 0, "row slices of 64: two tile piece pairs each");
        if (nend > nbeg) fetch_chunk(nend - 1);
        for (int n = nend - 1; n >= nbeg; --n) {
            const int64_t t0 = int64_t(n) * kC;
            const int valid = int(min<int64_t>(kC, s.seq_len - t0));
            const int64_t tok0 = bh * s.seq_len + t0;
            chunk_head(n, valid, tok0);
            __syncthreads();  // the gates are published; the previous pass is done with the planes
            put_x(TA, valid);  // q*
            if (isG) {
                put_y_rows(TB, valid);  // zeta dout
                if (n > nbeg) fetch_chunk(n - 1);
            } else {
                put_y_tile(TB, valid);  // -zeta e*
            }
            __syncthreads();
            const float D = decay_from_start(sLg, sZl, kC - 1);
            dprod *= D;
            f32x4 acc[NCT];
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) acc[ct] = st[ct] * D;
            multiply(acc);
            if (!isG) {
                __syncthreads();
                put_x(TB, valid);       // e*
                put_y_tile(TA, valid);  // -zeta q*
                if (n > nbeg) fetch_chunk(n - 1);
                __syncthreads();
                multiply(acc);
            }
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) st[ct] = acc[ct];
            __syncthreads();  // every wave is done with this chunk's gates before they are rewritten
        }
    } else {
        PassRegs P0, P1;
        if (nend > nbeg) fetch(nend - 1, 0, P0);
        for (int n = nend - 1; n >= nbeg; --n) {
            const int64_t t0 = int64_t(n) * kC;
            const int valid = int(min<int64_t>(kC, s.seq_len - t0));
            const int64_t tok0 = bh * s.seq_len + t0;
            chunk_head(n, valid, tok0);
            __syncthreads();  // the gates are published; the previous pass is done with sX, sYr
            put(P0, valid);
            if (!isG)
                fetch(n, 1, P1);
            else if (n > nbeg)
                fetch(n - 1, 0, P1);
            __syncthreads();
            const float D = decay_from_start(sLg, sZl, kC - 1);
            dprod *= D;
            f32x4 acc[NCT];
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) acc[ct] = st[ct] * D;
            multiply(acc);
            if (!isG) {
                __syncthreads();
                put(P1, valid);
                if (n > nbeg) fetch(n - 1, 0, P0);
                __syncthreads();
                multiply(acc);
            } else {
                P0 = P1;
            }
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) st[ct] = acc[ct];
            __syncthreads();  // every wave is done with this chunk's gates before they are rewritten
        }
    }
    if (sg.totals) {
        float* tb = seg_tile(seg);
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
            for (int r = 0; r < 4; ++r) tb[r * DK + 16 * ct] = st[ct][r];
        if (tile == 0 && tid == 0) sg.dec[bh * sg.total + seg] = dprod;
    }
}

// ---------------------------------------------------------------- per-chunk gradients
// One workgroup of eight waves per chunk, two per SIMD, so one wave's LDS and memory
// waits overlap the other's products.  The C x C phases split the 4 x 4 result tiles
// over the waves (row tile w % 4, two column tiles); the token-by-feature phases give
// each wave one 16-column feature tile and the token tiles GradSplit assigns.
constexpr int kGradThreads = 512;
constexpr int kGW = kGradThreads / kWave;  // waves per workgroup

// Token-by-feature tiles of wave w for a feature dimension D: column tile col(w), token
// tiles st0(w) .. st0(w) + NST - 1.
template <int D>
struct GradSplit {
    static constexpr int NCOL = D / 16;          // feature column tiles
    static constexpr int WPC = kGW / NCOL;       // waves per column tile
    static constexpr int NST = (kC / 16) / WPC;  // token tiles per wave
    static_assert(WPC * NCOL == kGW && NST * WPC == kC / 16, "eight waves over the feature tiles");
    __device__ static int col(int w) { return w / WPC; }
    __device__ static int st0(int w) { return (w % WPC) * NST; }
    __device__ static bool own(int w, int st) { return st >= st0(w) && st < st0(w) + NST; }
};

template <typename Tin, int DK, int DV>
__global__ __launch_bounds__(kGradThreads) void bwd_grad_kernel(BwdArgs a)
{
    const ForwardShape s = a.s;
    const int nc = s.n_chunks;
    const int n = blockIdx.x % nc;
    const int64_t bh = blockIdx.x / nc;
    const int64_t t0 = int64_t(n) * kC;
    const int valid = int(min<int64_t>(kC, s.seq_len - t0));
    const int64_t tok0 = bh * s.seq_len + t0;
    const int tid = threadIdx.x;
    const int w = tid / kWave, lane = tid % kWave, g = lane / 16, ln = lane % 16;
    const Tin* kp = static_cast<const Tin*>(a.k);
    const Tin* vp = static_cast<const Tin*>(a.v);
    const int64_t mat = bh * nc + n;
    const float* AG = a.AG + mat * int64_t(DV) * DK;
    const float* SH = a.SH + mat * int64_t(DK) * DK;
    const float* Gc = a.Gs + mat * int64_t(DV) * DK;
    const float* Hc = a.Hs + mat * int64_t(DK) * DK;

    __shared__ __attribute__((aligned(16))) float sT0[kC * kLdT];
    __shared__ __attribute__((aligned(16))) float sT1[kC * kLdT];
    __shared__ __attribute__((aligned(16))) float sM0[kC * kLdC];  // KQ, then M1 = Z ⊙ KQ, then W
    __shared__ __attribute__((aligned(16))) float sM1[kC * kLdC];  // VE, then M2 = Z ⊙ (VE - KE)
    __shared__ __attribute__((aligned(16))) float sM2[kC * kLdC];  // KE, then Qm = beta_p (VE - KE) KQ
    __shared__ __attribute__((aligned(16))) float sZ[kC * kLdC];   // Z[s][t] = zeta_{t,s} (s <= t)
    __shared__ float sLg[kC];
    __shared__ int sZl[kC];
    __shared__ float sBeta[kC], sZe[kC], sPhi[kC];
    __shared__ float sTok[5][kC];     // per token: dbeta (intra), v^T A^G k, k^T A^H k, g, h
    __shared__ float sPart[kGW];
    __shared__ float sRed[kGW][kC];   // per-wave partial sums per token
    __shared__ float sRed2[kGW][kC];  // the same for a second quantity
    __shared__ float sF;
    // bf16 route: the chunk's keys stay in LDS as bf16 for the whole kernel (rows of
    // kLdKb elements: 2 mod 32 words, so the 16 rows of a fragment read fall in distinct
    // banks), read as matrix-core operands straight from there
    constexpr int kLdKb = DK + 4;
    __shared__ __attribute__((aligned(16))) uint16_t sKb[std::is_same<Tin, bf16_t>::value ? kC * kLdKb : 1];

    // The products with the d x d matrices (A^G, S^H, G_c, H_c) run on the bf16 matrix cores
    // with split operands on the bf16 route (keys and values exact in bf16), on the fp32
    // matrix cores otherwise.
    constexpr bool kSplit = std::is_same<Tin, bf16_t>::value;
    // Token tiles in registers: each phase's tiles are fetched while the phase before it
    // computes, then put into sT0 / sT1 once those are free.
    Tile<DK, Tin, kGradThreads> tk;
    Tile<DV, Tin, kGradThreads> tv;
    Tile<DK, float, kGradThreads> tq, te;
    Tile<DV, float, kGradThreads> td;
    tk.fetch(kp, tok0, valid);
    tq.fetch(a.qstar, tok0, valid);

    // ---- gates: Z, zeta_{E,s}, phi_s = zeta_{s-1,c-1}
    if (tid < kWave) chunk_log_decays(a.gamma + tok0, valid, sLg, sZl);
    __syncthreads();
    for (int e = tid; e < kC * kC; e += kGradThreads) {
        const int i = e / kC, j = e % kC;
        sZ[i * kLdC + j] = decay_between(sLg, sZl, i, j);
    }
    if (tid < kC) {
        sBeta[tid] = tid < valid ? a.beta[tok0 + tid] : 0.0f;
        sZe[tid] = decay_between(sLg, sZl, tid, kC - 1);
        sPhi[tid] = tid == 0 ? 1.0f : decay_from_start(sLg, sZl, tid - 1);
    }

    // ---- gram matrices [p][t] of the chunk's tokens: wave w forms row tile w % 4,
    // column tiles 2 (w / 4) and 2 (w / 4) + 1
    // (on the bf16 route sT0 holds keys or values, exact in bf16, and the other side
    // enters split)
    // (A_KEYS: on the bf16 route the A operand, the keys, comes from sKb)
    auto gram = [&](float* dst, auto d_tag, auto keys_tag) {
        constexpr int D = decltype(d_tag)::value;
        constexpr bool A_KEYS = decltype(keys_tag)::value;
        const int rt = w % 4;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int tt = 2 * (w / 4) + h;
            f32x4 gm;
            if constexpr (kSplit) {
                gm = kZero4;
#pragma unroll
                for (int b = 0; b < D / 32; ++b) {
                    f32x4 b0, b1;
                    row_step(sT1 + (16 * tt + ln) * kLdT, b, b0, b1);
                    bf16x8 bhi, blo;
                    split8(b0, b1, bhi, blo);
                    bf16x8 x;
                    if constexpr (A_KEYS) {
                        x = lds_frag(sKb + (16 * rt + ln) * kLdKb + 32 * b + 4 * g);
                    } else {
                        f32x4 a0, a1;
                        row_step(sT0 + (16 * rt + ln) * kLdT, b, a0, a1);
                        x = pack8(a0, a1);
                    }
                    gm = mfma16(x, bhi, gm);
                    gm = mfma16(x, blo, gm);
                }
            } else {
                gm = mma16<D, kLdT, 1, 1, kLdT>(sT0 + 16 * rt * kLdT, sT1 + 16 * tt * kLdT, kZero4);
            }
#pragma unroll
            for (int r = 0; r < 4; ++r) dst[(16 * rt + 4 * g + r) * kLdC + 16 * tt + ln] = gm[r];
        }
    };
    using KeysA = std::integral_constant<bool, kSplit>;
    using NoKeys = std::integral_constant<bool, false>;
    if constexpr (kSplit)
        tk.put_bf16(sKb, kLdKb, valid);
    else
        tk.put(sT0, valid);
    tq.put(sT1, valid);
    te.fetch(a.estar, tok0, valid);
    __syncthreads();
    gram(sM0, std::integral_constant<int, DK>{}, KeysA{});  // KQ[p][t] = k_p . q*_t
    __syncthreads();
    te.put(sT1, valid);
    tv.fetch(vp, tok0, valid);
    td.fetch(a.dout, tok0, valid);
    __syncthreads();
    gram(sM2, std::integral_constant<int, DK>{}, KeysA{});  // KE[p][t] = k_p . e*_t
    __syncthreads();
    tv.put(sT0, valid);
    td.put(sT1, valid);
    if constexpr (!kSplit) tk.fetch(kp, tok0, valid);
    __syncthreads();
    gram(sM1, std::integral_constant<int, DV>{}, NoKeys{});  // VE[p][t] = v_p . e_t
    __syncthreads();

    // ---- C x C combinations, one row p per wave pass (lane = t): DVK = VE - KE;
    // Qm = beta_p DVK KQ; the intra part of dbeta_p = sum_t Z[p][t] KQ[p][t] DVK[p][t]
    // (a wave sum); M1 = Z ⊙ KQ, M2 = Z ⊙ DVK
    for (int p = w; p < kC; p += kGW) {
        const int o = p * kLdC + lane;
        const float kq = sM0[o], z = sZ[o];
        const float dvk = sM1[o] - sM2[o];
        sM2[o] = sBeta[p] * dvk * kq;
        sM0[o] = z * kq;
        sM1[o] = z * dvk;
        const float db = wave_sum(z * kq * dvk);
        if (lane == 0) sTok[0][p] = db;
    }
    auto tok = [&](int st, int r) { return 16 * st + 4 * g + r; };
    // sum the partials p[st][r] and q[st][r] (token tok(st, r); zero on the token tiles the
    // wave does not own) over lanes and waves into out[token] and out2[token], each in a
    // fixed order (16-lane row sums, then waves 0 .. kGW - 1); wave 0 forms out, wave 1 out2
    auto reduce_tokens2 = [&](const float (&p)[4][4], const float (&q)[4][4], float* out, float* out2) {
#pragma unroll
        for (int st = 0; st < 4; ++st)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const float v = row16_sum(p[st][r]);
                const float u = row16_sum(q[st][r]);
                if (ln == 0) {
                    sRed[w][tok(st, r)] = v;
                    sRed2[w][tok(st, r)] = u;
                }
            }
        __syncthreads();
        if (tid < 2 * kC) {
            const int tk_ = tid % kC;
            float (*src)[kC] = tid < kC ? sRed : sRed2;
            float acc = 0.0f;
#pragma unroll
            for (int u = 0; u < kGW; ++u) acc += src[u][tk_];
            (tid < kC ? out : out2)[tk_] = acc;
        }
        __syncthreads();
    };

    // ---- dv_s = beta_s (sum_t M1[s][t] e_t + zeta_E[s] A^G k_s)   (sT1 holds e_t)
    {
        using S = GradSplit<DV>;
        const int at = S::col(w);
        float bv[DK / 4];                       // fp32 route: B(k, n) = A^G[16 at + n][k]
        float agr[DK / 32][8];                  // bf16 route: the same, split below
        bf16x8 arh[DK / 32], arl[DK / 32];
        if constexpr (kSplit)
            load_row8<DK>(AG, (16 * at + ln) * DK, agr);  // before the barriers
        else
            load_b<DK, 1, DK>(AG + 16 * at * DK, bv);
        __syncthreads();
        if constexpr (!kSplit) tk.put(sT0, valid);  // (the bf16 route reads the keys from sKb)
        tq.fetch(a.qstar, tok0, valid);
        te.fetch(a.estar, tok0, valid);
        __syncthreads();
        if constexpr (kSplit) split_steps<DK>(agr, arh, arl);
#pragma unroll
        for (int st = 0; st < 4; ++st) {
            if (!S::own(w, st)) continue;
            // M1[s][t] = 0 for t < s: the token sum of row tile st starts at 16 st
            const f32x4 in = mma16_from<kC, kLdC, 1, kLdT, 1>(sM0 + 16 * st * kLdC, sT1 + 16 * at, 16 * st, kZero4);
            f32x4 ex;  // (K A^G^T)[s][a]
            if constexpr (kSplit)
                ex = mma_bs<DK>(sKb + (16 * st + ln) * kLdKb, arh, arl, kZero4);
            else
                ex = mma16_b<DK, kLdT, 1>(sT0 + 16 * st * kLdT, bv, kZero4);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int t = tok(st, r);
                if (t < valid) a.dv[(tok0 + t) * DV + 16 * at + ln] = sBeta[t] * (in[r] + sZe[t] * ex[r]);
            }
        }
    }

    // ---- dk_s = beta_s (sum_t M2[s][t] q*_t - sum_t M1[s][t] e*_t + zeta_E[s] ((A^G)^T v_s + S^H k_s)),
    //      with v^T A^G k and k^T A^H k = (1/2) k^T S^H k per token
    // The inter part's operands: lane (sl, n) of the wave of column tile bt holds
    // A^G[k][16 bt + n] and S^H[16 bt + n][k] (S^H is symmetric; its rows are contiguous)
    // for the lane's contraction indices k.  The g and h products below load G_c and H_c in
    // the same patterns, so the Frobenius products of F are the lanes' own sums over their
    // registers (every element of the four matrices is read once).
    float bag[DV / 4], bsh[DK / 4];            // fp32 route, in flight during the intra part
    bf16x8 agh[DV / 32], agl[DV / 32], shh[DK / 32], shl[DK / 32];  // bf16 route, split
    {
        using S = GradSplit<DK>;
        const int bt = S::col(w);
        f32x4 in[4];
        float agc[DV / 32][8], shr[DK / 32][8];  // bf16 route, in flight during the intra part
        if constexpr (kSplit) {
            load_col8<DV>(AG, 16 * bt + ln, DK, agc);     // B(k, n) = A^G[k][16 bt + n]
            load_row8<DK>(SH, (16 * bt + ln) * DK, shr);  // B(k, n) = S^H[16 bt + n][k]
        } else {
            load_b<DV, DK, 1>(AG + 16 * bt, bag);       // B(k, n) = A^G[k][16 bt + n]
            load_b<DK, 1, DK>(SH + 16 * bt * DK, bsh);  // B(k, n) = S^H[16 bt + n][k] = S^H[k][16 bt + n]
        }
        __syncthreads();
        tq.put(sT0, valid);
        te.put(sT1, valid);
        if constexpr (!kSplit) tk.fetch(kp, tok0, valid);
        tv.fetch(vp, tok0, valid);
        __syncthreads();
#pragma unroll
        for (int st = 0; st < 4; ++st) {
            if (!S::own(w, st)) continue;
            const f32x4 pq = mma16_from<kC, kLdC, 1, kLdT, 1>(sM1 + 16 * st * kLdC, sT0 + 16 * bt, 16 * st, kZero4);
            const f32x4 pe = mma16_from<kC, kLdC, 1, kLdT, 1>(sM0 + 16 * st * kLdC, sT1 + 16 * bt, 16 * st, kZero4);
            in[st] = pq - pe;
        }
        __syncthreads();
        // the bf16 route keeps q* in sT0 for the g/h phase (its keys come from sKb)
        if constexpr (!kSplit) tk.put(sT0, valid);
        tv.put(sT1, valid);
        if constexpr (!kSplit) tq.fetch(a.qstar, tok0, valid);
        td.fetch(a.dout, tok0, valid);
        __syncthreads();
        if constexpr (kSplit) {
            split_steps<DV>(agc, agh, agl);
            split_steps<DK>(shr, shh, shl);
        }
        float pa[4][4] = {}, pk[4][4] = {};
#pragma unroll
        for (int st = 0; st < 4; ++st) {
            if (!S::own(w, st)) continue;
            f32x4 ag, sh;
            if constexpr (kSplit) {
                ag = mma_xs<DV>(sT1 + (16 * st + ln) * kLdT, agh, agl, kZero4);
                sh = mma_bs<DK>(sKb + (16 * st + ln) * kLdKb, shh, shl, kZero4);
            } else {
                ag = mma16_b<DV, kLdT, 1>(sT1 + 16 * st * kLdT, bag, kZero4);
                sh = mma16_b<DK, kLdT, 1>(sT0 + 16 * st * kLdT, bsh, kZero4);
            }
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int t = tok(st, r), b = 16 * bt + ln;
                const float kb = kSplit ? __uint_as_float(uint32_t(sKb[t * kLdKb + b]) << 16) : sT0[t * kLdT + b];
                if (t < valid) a.dk[(tok0 + t) * DK + b] = sBeta[t] * (in[st][r] + sZe[t] * (ag[r] + sh[r]));
                pa[st][r] += kb * ag[r];
                pk[st][r] += 0.5f * kb * sh[r];
            }
        }
        reduce_tokens2(pa, pk, sTok[1], sTok[2]);
    }

    // ---- g_t = e_t^T G_c q*_t, h_t = e*_t^T H_c q*_t, F = <A^G, G_c> + (1/2) <S^H, H_c>,
    //      and dLambda of the chunk
    {
        using S = GradSplit<DK>;
        const int bt = S::col(w);
        float bg[DV / 4], bh_[DK / 4];                             // fp32 route
        bf16x8 gch[DV / 32], gcl[DV / 32], hch[DK / 32], hcl[DK / 32];  // bf16 route, split
        float fr = 0.0f;
        float gcc[DV / 32][8];
        if constexpr (kSplit)
            load_col8<DV>(Gc, 16 * bt + ln, DK, gcc);  // B(k, n) = G_c[k][16 bt + n], before the barriers
        else
            load_b<DV, DK, 1>(Gc + 16 * bt, bg);
        __syncthreads();
        if constexpr (!kSplit) tq.put(sT0, valid);  // (on the bf16 route q* is still in sT0)
        td.put(sT1, valid);
        te.fetch(a.estar, tok0, valid);
        __syncthreads();
        // F = <A^G, G_c> + (1/2) <S^H, H_c>, this lane's elements (A^G and S^H held since dk;
        // on the bf16 route split, standing for the fp32 values to ~2^-16)
        if constexpr (kSplit) {
            fr = dot_split<DV>(agh, agl, gcc);
            split_steps<DV>(gcc, gch, gcl);
        } else {
#pragma unroll
            for (int i = 0; i < DV / 4; ++i) fr = fmaf(bag[i], bg[i], fr);
        }
        // B(k, n) = H_c[16 bt + n][k] = H_c[k][16 bt + n], in flight during g
        float hcr[DK / 32][8];
        if constexpr (kSplit)
            load_row8<DK>(Hc, (16 * bt + ln) * DK, hcr);
        else
            load_b<DK, 1, DK>(Hc + 16 * bt * DK, bh_);
        float pg[4][4] = {}, ph[4][4] = {};
#pragma unroll
        for (int st = 0; st < 4; ++st) {
            if (!S::own(w, st)) continue;
            f32x4 eg;
            if constexpr (kSplit)
                eg = mma_ss<DV>(sT1 + (16 * st + ln) * kLdT, gch, gcl, kZero4);
            else
                eg = mma16_b<DV, kLdT, 1>(sT1 + 16 * st * kLdT, bg, kZero4);
#pragma unroll
            for (int r = 0; r < 4; ++r) pg[st][r] += eg[r] * sT0[tok(st, r) * kLdT + 16 * bt + ln];
        }
        __syncthreads();  // every wave is done with d in sT1 (g's token sums wait for h's)
        te.put(sT1, valid);
        __syncthreads();
        {
            float fh = 0.0f;
            if constexpr (kSplit) {
                fh = dot_split<DK>(shh, shl, hcr);
                split_steps<DK>(hcr, hch, hcl);
            } else {
#pragma unroll
                for (int i = 0; i < DK / 4; ++i) fh = fmaf(bsh[i], bh_[i], fh);
            }
            fr = fmaf(0.5f, fh, fr);
        }
#pragma unroll
        for (int st = 0; st < 4; ++st) {
            if (!S::own(w, st)) continue;
            f32x4 eh;
            if constexpr (kSplit)
                eh = mma_ss<DK>(sT1 + (16 * st + ln) * kLdT, hch, hcl, kZero4);
            else
                eh = mma16_b<DK, kLdT, 1>(sT1 + 16 * st * kLdT, bh_, kZero4);
#pragma unroll
            for (int r = 0; r < 4; ++r) ph[st][r] += eh[r] * sT0[tok(st, r) * kLdT + 16 * bt + ln];
        }
        reduce_tokens2(pg, ph, sTok[3], sTok[4]);
        // (with d_k = 64 two waves share a column tile: the first of them counts it)
        fr = wave_sum(w % S::WPC == 0 ? fr : 0.0f);
        if (lane == 0) sPart[w] = fr;
        // dLambda of the chunk, -sum_t q*_t e*_t per feature: the tokens split into
        // kGradThreads / DK slices, one per thread of a feature, partial sums through sRed
        {
            constexpr int NP = kGradThreads / DK;
            const int f = tid % DK, sl = tid / DK;
            float acc = 0.0f;
#pragma unroll 8
            for (int t = sl * (kC / NP); t < (sl + 1) * (kC / NP); ++t) acc += sT0[t * kLdT + f] * sT1[t * kLdT + f];
            (&sRed[0][0])[tid] = acc;
        }
        __syncthreads();
        if (tid < DK) {
            constexpr int NP = kGradThreads / DK;
            float acc = 0.0f;
#pragma unroll
            for (int sl = 0; sl < NP; ++sl) acc += (&sRed[0][0])[sl * DK + tid];
            a.dlam_part[mat * DK + tid] = -acc;
        }
        if (tid == 0) {
            float t = 0.0f;
            for (int u = 0; u < kGW; ++u) t += sPart[u];
            sF = t;
        }
    }

    // ---- W[p][s] = sum_{t>=s} zeta_{t,s} Qm[p][t] (Qm Z^T), into sM0: wave w row tile
    // w % 4, column tiles w / 4 and 3 - w / 4 (the sum of column tile st starts at 16 st,
    // so every wave runs 20 of the 32 steps)
    {
        const int rt = w % 4;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int st = h ? 3 - w / 4 : w / 4;
            const f32x4 wq = mma16_from<kC, kLdC, 1, 1, kLdC>(sM2 + 16 * rt * kLdC, sZ + 16 * st * kLdC, 16 * st, kZero4);
#pragma unroll
            for (int r = 0; r < 4; ++r) sM0[(16 * rt + 4 * g + r) * kLdC + 16 * st + ln] = wq[r];
        }
        __syncthreads();
    }

    // ---- assemble dgamma_s and dbeta_s: wave w takes tokens s = (kC / kGW) w.., its lanes
    // the summation index q of the three sums (wave sums), the masks coming from Z:
    //   t2 = sum_{t >= s} zeta_{t,s} (g_t - h_t)                  (Z[s][q], 0 for q < s)
    //   t3 = sum_{p < s} zeta_{s-1,p} beta_p (v^T A^G k + k^T A^H k)_p,
    //   t4 = sum_{p < s} zeta_{s-1,p} W[p][s]                     (Z[q][s-1], 0 for q >= s)
    {
        const float gh = sTok[3][lane] - sTok[4][lane];
        const float bk = sBeta[lane] * (sTok[1][lane] + sTok[2][lane]);
#pragma unroll 4
        for (int i = 0; i < kC / kGW; ++i) {
            const int si = (kC / kGW) * w + i;
            const float v2 = sZ[si * kLdC + lane] * gh;
            float v3 = 0.0f, v4 = 0.0f;
            if (si > 0) {
                const float z = sZ[lane * kLdC + si - 1];  // zeta_{s-1,q}
                v3 = z * bk;
                v4 = z * sM0[lane * kLdC + si];
            }
            const float t2 = wave_sum(v2), t3 = wave_sum(v3), t4 = wave_sum(v4);
            if (lane == 0 && si < valid) {
                const float ze = sZe[si], phi = sPhi[si];
                a.dgamma[tok0 + si] = ze * phi * sF + phi * t2 + ze * t3 + t4;
                a.dbeta[tok0 + si] = sTok[0][si] + ze * (sTok[1][si] + sTok[2][si]);
            }
        }
    }
}

// ---------------------------------------------------------------- dLambda
// dLambda[h][b] = sum over the batch and the chunks of the per-chunk partial sums:
// one workgroup per head; thread (b, slot) sums every kThreads / d_k-th (batch, chunk)
// entry, eight loads in flight at a time into eight partial sums, then the partial
// sums and the slots are combined in a fixed order.
__global__ __launch_bounds__(kThreads) void bwd_dlam_kernel(BwdArgs a)
{
    const ForwardShape s = a.s;
    const int dk = s.d_k, slots = kThreads / dk;
    const int64_t h = blockIdx.x;
    const int b = threadIdx.x % dk, slot = threadIdx.x / dk;
    const int64_t per = s.batch * s.n_chunks;  // partial sums of this head
    __shared__ float sAcc[kThreads];
    auto part = [&](int64_t e) {
        const int64_t bb = e / s.n_chunks, n = e % s.n_chunks;
        return a.dlam_part[((bb * s.heads + h) * s.n_chunks + n) * dk + b];
    };
    float acc8[8] = {0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f};
    int64_t e = slot;
    for (; e + 7 * slots < per; e += 8 * slots) {
        float v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = part(e + u * slots);
#pragma unroll
        for (int u = 0; u < 8; ++u) acc8[u] += v[u];
    }
    for (; e < per; e += slots) acc8[0] += part(e);
    const float acc = ((acc8[0] + acc8[1]) + (acc8[2] + acc8[3])) + ((acc8[4] + acc8[5]) + (acc8[6] + acc8[7]));
    sAcc[threadIdx.x] = acc;
    __syncthreads();
    if (slot == 0) {
        float t = 0.0f;
        for (int u = 0; u < slots; ++u) t += sAcc[u * dk + b];
        a.dlam[h * dk + b] = t;
    }
}

template <typename Tin, int DK, int DV>
hipError_t launch_bwd_dims(const BwdArgs& a, hipStream_t stream, int stage)
{
    const int64_t bh = a.s.batch * a.s.heads;
    const unsigned chunks = unsigned(bh * a.s.n_chunks);
    constexpr bool kSplit = std::is_same<Tin, bf16_t>::value;  // the bf16 route's split products
    switch (stage) {
        case 0:
            hipLaunchKernelGGL((bwd_rhs_kernel<Tin, DK, DV>), dim3(chunks), dim3(kThreads), 0, stream, a);
            break;
        case 1: {
            // segments while the (sequence, slice, segment) workgroups fit the compute units
            // once (one per unit) and each keeps at least 8 chunks; the totals go to the
            // fp32 right-hand-side region, free once the solve has read it
            constexpr int NTILE = (DK + DV) / kAdjRows;
            const int nc = a.s.n_chunks;
            int S = 1;
            while (bh * NTILE * (2 * S) <= 256 && nc / (2 * S) >= 8) S *= 2;
            const int len = (nc + S - 1) / S;
            S = (nc + len - 1) / len;
            AdjSeg sg{len, S, 0, S, false, a.u, a.u + bh * S * int64_t(DK) * (DK + DV)};
            if (S > 1) {
                AdjSeg p1 = sg;
                p1.first = 1;
                p1.count = S - 1;
                p1.totals = true;
                hipLaunchKernelGGL((bwd_adjoint_kernel<DK, DV, kSplit>), dim3(unsigned(bh * NTILE * p1.count)), dim3(kThreads), 0,
                                   stream, a, p1);
                const hipError_t e = hipGetLastError();
                if (e != hipSuccess) return e;
            }
            hipLaunchKernelGGL((bwd_adjoint_kernel<DK, DV, kSplit>), dim3(unsigned(bh * NTILE * sg.count)), dim3(kThreads), 0,
                               stream, a, sg);
            break;
        }
        case 2:
            hipLaunchKernelGGL((bwd_grad_kernel<Tin, DK, DV>), dim3(chunks), dim3(kGradThreads), 0, stream, a);
            break;
        default:
            hipLaunchKernelGGL(bwd_dlam_kernel, dim3(unsigned(a.s.heads)), dim3(kThreads), 0, stream, a);
    }
    return hipGetLastError();
}

template <typename Tin>
hipError_t launch_bwd_tin(const BwdArgs& a, hipStream_t stream, int stage)
{
    if (a.s.d_k == 64)
        return a.s.d_v == 64 ? launch_bwd_dims<Tin, 64, 64>(a, stream, stage) : launch_bwd_dims<Tin, 64, 128>(a, stream, stage);
    return a.s.d_v == 64 ? launch_bwd_dims<Tin, 128, 64>(a, stream, stage) : launch_bwd_dims<Tin, 128, 128>(a, stream, stage);
}

}  // namespace

hipError_t launch_backward_stage(const BwdArgs& a, int stage, hipStream_t stream)
{
    if (a.s.chunk != kC) return hipErrorInvalidValue;
    return a.s.bf16 ? launch_bwd_tin<bf16_t>(a, stream, stage) : launch_bwd_tin<float>(a, stream, stage);
}

}  // namespace mesa
