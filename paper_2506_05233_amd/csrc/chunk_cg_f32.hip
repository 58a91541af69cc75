// Chunked conjugate gradients + read-out of the Mesa layer, fp32 products.
//
// One workgroup solves the C systems (H_t + Lambda) q*_t = q_t of one chunk
// together (App. C, Alg. 1, at most n_cg iterations and its relative tolerance;
// App. D, Eq. q_star_parallel) and
// then forms o_t = G_t q*_t (App. D, Eq. gla).  With c the chunk start, j the
// in-chunk token, Z[i][j] = zeta_{c+j,c+i} (Z upper triangular, unit diagonal)
// and zeta_j = zeta_{c+j,c}, every CG product over the chunk is
//
//   W = zeta ⊙_cols (H_c P) + K^T_cols (beta ⊙ Z ⊙ (K P)) + Lambda ⊙ P
//
// (the inter-chunk state term plus the intra-chunk, causally masked,
// gate-weighted K K^T term), and the read-out is
//
//   O = zeta ⊙_cols (G_c Q*) + V^T_cols (beta ⊙ Z ⊙ (K Q*)).
//
// The decay on the carried state (zeta_j) is the reading under which the
// chunkwise form equals the recurrence; App. D's compact equations omit it.
//
// This is the fp32 path: every product is exact fp32 (results agree with fp64 to
// about 1e-6).  Chunk 64 runs on the matrix cores (chunk_cg_f32_mma_kernel below);
// chunks 16 and 32 use fp32 FMAs with operands staged in LDS: matrices over the
// chunk are held as [feature a][token j]; thread t owns column j = t % C and rows
// a = t / C + (256 / C) m, so the per-column CG scalars reduce over 256 / C threads.
#include "mesa_device.hpp"
#include "mesa_kernels.hpp"

namespace mesa {
namespace {

constexpr int kThreads = 256;
constexpr int kLdW = 129;  // padded row stride of 128-wide LDS tiles

template <typename Tin, int DK, int C>
__global__ __launch_bounds__(kThreads) void chunk_cg_f32_kernel(CgArgs a)
{
    constexpr int NE = DK * C / kThreads;  // elements of a [DK][C] matrix per thread
    constexpr int GRP = kThreads / C;      // threads that share one column
    constexpr int LDH = DK + 1;
    constexpr int LDP = C + 1;

    const ForwardShape s = a.s;
    const int dv = s.d_v;
    const int n = blockIdx.x % s.n_chunks;
    const int64_t bh = blockIdx.x / s.n_chunks;
    const int h = int(bh % s.heads);
    const int64_t t0 = int64_t(n) * C;
    const int valid = int(min<int64_t>(C, s.seq_len - t0));
    const int64_t tok0 = bh * s.seq_len + t0;
    const int tid = threadIdx.x;
    const int j = tid % C;   // this thread's token (column)
    const int a0 = tid / C;  // this thread's first feature row

    __shared__ float sH[DK * kLdW];   // H_c [DK][DK+1]; later G_c^T as [DK][129]
    __shared__ float sKV[C * kLdW];   // K [C][DK] (row stride 129); later V [C][dv]
    __shared__ float sP[DK * LDP];    // P, q or x as [DK][C+1]
    __shared__ float sS[C * C];       // beta ⊙ Z ⊙ (K P) as [C][C]
    __shared__ float sRed[kThreads];
    __shared__ float sLg[64], sZeta[64], sBeta[64];
    __shared__ int sZl[64];

    const Tin* qp = static_cast<const Tin*>(a.q);
    const Tin* kp = static_cast<const Tin*>(a.k);
    const Tin* vp = static_cast<const Tin*>(a.v);

    for (int e = tid; e < C * DK; e += kThreads) {
        const int i = e / DK, c = e % DK;
        const bool ok = i < valid;
        sKV[i * kLdW + c] = ok ? to_f32(kp[(tok0 + i) * DK + c]) : 0.0f;
        sP[c * LDP + i] = ok ? (a.rhs ? a.rhs[(tok0 + i) * DK + c] : to_f32(qp[(tok0 + i) * DK + c])) : 0.0f;
    }
    const float* Hc = static_cast<const float*>(a.Hs) + (bh * s.n_chunks + n) * int64_t(DK) * DK;
    for (int e = tid; e < DK * DK; e += kThreads) sH[(e / DK) * LDH + e % DK] = Hc[e];
    if (tid < kWave) chunk_log_decays(a.gamma + tok0, valid, sLg, sZl);
    if (tid < C) sBeta[tid] = tid < valid ? a.beta[tok0 + tid] : 0.0f;
    __syncthreads();
    if (tid < C) sZeta[tid] = decay_from_start(sLg, sZl, tid);
    __syncthreads();

    const float* lam = a.lambda + int64_t(h) * DK;
    const float zeta_j = sZeta[j];

    // S = beta ⊙ Z ⊙ (K X) for X = the matrix currently in sP.
    auto masked_kx = [&]() {
        for (int e = tid; e < C * C; e += kThreads) {
            const int i = e / C, jj = e % C;
            float acc = 0.0f;
            if (i <= jj) {
#pragma unroll 8
                for (int c = 0; c < DK; ++c) acc += sKV[i * kLdW + c] * sP[c * LDP + jj];
                acc *= sBeta[i] * decay_between(sLg, sZl, i, jj);
            }
            sS[e] = acc;
        }
    };
    // w = (H_t + Lambda) p for this thread's elements; p is also written to sP.
    auto matvec = [&](const float (&pin)[NE], float (&wout)[NE]) {
        __syncthreads();
#pragma unroll
        for (int m = 0; m < NE; ++m) sP[(a0 + GRP * m) * LDP + j] = pin[m];
        __syncthreads();
        masked_kx();
        __syncthreads();
#pragma unroll
        for (int m = 0; m < NE; ++m) wout[m] = 0.0f;
#pragma unroll 2
        for (int b = 0; b < DK; ++b) {
            const float pb = sP[b * LDP + j];
#pragma unroll
            for (int m = 0; m < NE; ++m) wout[m] += sH[(a0 + GRP * m) * LDH + b] * pb;
        }
#pragma unroll
        for (int m = 0; m < NE; ++m) wout[m] = zeta_j * wout[m] + lam[a0 + GRP * m] * pin[m];
#pragma unroll 2
        for (int i = 0; i < C; ++i) {
            const float sij = sS[i * C + j];
#pragma unroll
            for (int m = 0; m < NE; ++m) wout[m] += sKV[i * kLdW + a0 + GRP * m] * sij;
        }
    };
    auto colsum = [&](float part) -> float {
        sRed[tid] = part;
        __syncthreads();
        float t = 0.0f;
#pragma unroll
        for (int g = 0; g < GRP; ++g) t += sRed[g * C + j];
        __syncthreads();
        return t;
    };

    float x[NE], r[NE], p[NE], w[NE];
    // Jacobi start: x0 = q / diag(H_t + Lambda), diag(H_t) = zeta_j diag(H_c) + sum_i beta_i Z_ij k_i^2.
    // r temporarily holds q and w the diagonal.
#pragma unroll
    for (int m = 0; m < NE; ++m) {
        const int rr = a0 + GRP * m;
        r[m] = sP[rr * LDP + j];
        w[m] = zeta_j * sH[rr * LDH + rr] + lam[rr];
    }
    // the column solves for q 2^-qsh (|q 2^-qsh|^2 in [1/2, 2)); x is scaled back at the end
    int qsh;
    {
        float part = 0.0f;
#pragma unroll
        for (int m = 0; m < NE; ++m) part += r[m] * r[m];
        qsh = cg_scale_shift(colsum(part));
        const float qs = __builtin_ldexpf(1.0f, -qsh);
#pragma unroll
        for (int m = 0; m < NE; ++m) r[m] *= qs;
    }
#pragma unroll 1
    for (int i = 0; i <= j; ++i) {
        const float wij = sBeta[i] * decay_between(sLg, sZl, i, j);
#pragma unroll
        for (int m = 0; m < NE; ++m) {
            const float kv = sKV[i * kLdW + a0 + GRP * m];
            w[m] += wij * kv * kv;
        }
    }
#pragma unroll
    for (int m = 0; m < NE; ++m) {
        x[m] = r[m] / w[m];
        p[m] = r[m];  // p keeps q until the first residual is formed
    }
    matvec(x, w);
    float part = 0.0f;
#pragma unroll
    for (int m = 0; m < NE; ++m) {
        r[m] = p[m] - w[m];
        p[m] = r[m];
        part += r[m] * r[m];
    }
    float delta = colsum(part);
    const float thr = a.eps2 * delta;  // Alg. 1: the column stops once |r|^2 <= eps^2 |r_0|^2
    bool active = delta >= kMinNormal;
    int steps = 0;  // iterations that updated x
    for (int it = 0; it < a.n_cg; ++it) {
        if (!__syncthreads_or(active)) break;
        matvec(p, w);
        part = 0.0f;
#pragma unroll
        for (int m = 0; m < NE; ++m) part += p[m] * w[m];
        const float pw = colsum(part);
        if (active && !(pw >= kMinNormal)) active = false;
        if (active) {
            const float alpha = delta / pw;
#pragma unroll
            for (int m = 0; m < NE; ++m) {
                x[m] += alpha * p[m];
                r[m] -= alpha * w[m];
            }
            ++steps;
        }
        part = 0.0f;
#pragma unroll
        for (int m = 0; m < NE; ++m) part += r[m] * r[m];
        const float dn = colsum(part);
        if (active) {
            if (dn <= thr || !(dn >= kMinNormal)) {
                active = false;
            } else {
                const float beta_cg = dn / delta;
#pragma unroll
                for (int m = 0; m < NE; ++m) p[m] = r[m] + beta_cg * p[m];
                delta = dn;
            }
        }
    }
    {
        const float us = __builtin_ldexpf(1.0f, qsh);
#pragma unroll
        for (int m = 0; m < NE; ++m) x[m] *= us;
    }

    if (a.steps && a0 == 0 && j < valid) a.steps[tok0 + j] = steps;

    // Read-out o_t = G_t q*_t, chunkwise.
    __syncthreads();
#pragma unroll
    for (int m = 0; m < NE; ++m) {
        const int rr = a0 + GRP * m;
        sP[rr * LDP + j] = x[m];
        if (a.qstar && j < valid) a.qstar[(tok0 + j) * DK + rr] = x[m];
    }
    if (!a.out) return;  // solve only (uniform across the workgroup)
    __syncthreads();
    masked_kx();
    __syncthreads();
    for (int e = tid; e < C * dv; e += kThreads) {
        const int i = e / dv, c = e % dv;
        sKV[i * kLdW + c] = i < valid ? to_f32(vp[(tok0 + i) * dv + c]) : 0.0f;
    }
    // G_c [dv][DK] staged transposed, sH[b][e] = G_c[e][b]
    const float* Gc = static_cast<const float*>(a.Gs) + (bh * s.n_chunks + n) * int64_t(DK) * dv;
    for (int e = tid; e < DK * dv; e += kThreads) sH[(e % DK) * kLdW + e / DK] = Gc[e];
    __syncthreads();
    for (int e = tid; e < C * dv; e += kThreads) {
        const int jj = e / dv, c = e % dv;
        float gq = 0.0f;
        for (int b = 0; b < DK; ++b) gq += sH[b * kLdW + c] * sP[b * LDP + jj];
        float vk = 0.0f;
        for (int i = 0; i <= jj; ++i) vk += sKV[i * kLdW + c] * sS[i * C + jj];
        if (jj < valid) a.out[(tok0 + jj) * dv + c] = sZeta[jj] * gq + vk;
    }
}

// ---------------------------------------------------------------- matrix-core variant
// Chunk 64: the same CG with every product on the matrix cores in fp32
// (v_mfma_f32_16x16x4f32: exact fp32 products and accumulation).  Wave w owns tokens
// 16w .. 16w+15 of the chunk (the columns j of its result tiles) and runs their CG
// without synchronising with the other waves: a CG product for its columns,
//   W = zeta ⊙ (H_c P) + K^T (beta Z ⊙ (K P)) + lambda ⊙ P,
// needs only its own columns of P and, causally, the keys of tokens up to 16w+15.
// Vectors live in the MFMA result layout (lane (g, l) holds rows 4g..4g+3 of each
// 16-row tile for token 16w + l), and every product over features takes them as its
// B operand straight from registers: in the four products of a 16-feature tile u,
// k-slot g stands for feature 16u + 4g + jj (jj = 0..3), which is where lane (g, l)
// already holds it; the A operand (H_c, K or K^T from LDS) is read with the same
// feature order as one 16-byte access.
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f32x4 mfma4(float a, float b, f32x4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ float4 load4(const float* p) { return *reinterpret_cast<const float4*>(p); }

template <int DK>
__device__ __forceinline__ f32x4 load_vec4(const float* p) { const float4 v = load4(p); return f32x4{v.x, v.y, v.z, v.w}; }
template <int DK>
__device__ __forceinline__ f32x4 load_vec4(const bf16_t* p)
{
    const uint2 u = *reinterpret_cast<const uint2*>(p);
    return f32x4{__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u), __uint_as_float(u.y << 16),
                 __uint_as_float(u.y & 0xffff0000u)};
}

template <typename Tin, int DK, int DV>
__global__ __launch_bounds__(kThreads) void chunk_cg_f32_mma_kernel(CgArgs a)
{
    constexpr int C = 64;
    constexpr int MT = DK / 16, MTV = DV / 16;
    constexpr int DM = DK > DV ? DK : DV;
    constexpr int LDH = DK + 4;   // [row][feature] fp32 rows, 16-byte aligned
    constexpr int LDT = C + 4;    // [feature][token] rows
    const ForwardShape s = a.s;
    const int n = blockIdx.x % s.n_chunks;
    const int64_t bh = blockIdx.x / s.n_chunks;
    const int h = int(bh % s.heads);
    const int64_t t0 = int64_t(n) * C;
    const int valid = int(min<int64_t>(C, s.seq_len - t0));
    const int64_t tok0 = bh * s.seq_len + t0;
    const int tid = threadIdx.x, w = tid / kWave, lane = tid % kWave, g = lane / 16, ln = lane % 16;
    const int j = 16 * w + ln;  // this lane's token

    __shared__ __attribute__((aligned(16))) float sH[DM * LDH];   // H_c [f][f'], then G_c [e][f]
    __shared__ __attribute__((aligned(16))) float sK[C * LDH];    // k_i [i][f]
    __shared__ __attribute__((aligned(16))) float sKT[DM * LDT];  // k_i as [f][i], then v_i as [e][i]
    __shared__ __attribute__((aligned(16))) float sLam[DK];
    __shared__ float sLg[C], sBeta[C];
    __shared__ int sZl[C];

    const Tin* kp = static_cast<const Tin*>(a.k);
    const Tin* vp = static_cast<const Tin*>(a.v);
    // ---- staging: H_c, keys (both orientations), lambda, gates
    {
        const float* Hc = static_cast<const float*>(a.Hs) + (bh * s.n_chunks + n) * int64_t(DK) * DK;
        constexpr int NV = DK * DK / 4 / kThreads;
        float4 hv[NV];
#pragma unroll
        for (int m = 0; m < NV; ++m) hv[m] = load4(Hc + 4 * (tid + kThreads * m));
        // keys: lane l stages token l, features 4 (w + 4m) .. + 3, so that consecutive lanes
        // write consecutive words of the transposed tile sKT (a lane per token of a feature
        // row; lanes along the features of one token put 16 lanes on each bank)
        constexpr int NKV = C * DK / 4 / kThreads;
        static_assert(C == kWave, "one token per lane");
        f32x4 kv[NKV];
#pragma unroll
        for (int m = 0; m < NKV; ++m) {
            const int f = 4 * (w + (kThreads / kWave) * m);
            kv[m] = load_vec4<DK>(kp + (tok0 + min(lane, valid - 1)) * DK + f);
        }
#pragma unroll
        for (int m = 0; m < NV; ++m) {
            const int e = 4 * (tid + kThreads * m);
            *reinterpret_cast<float4*>(sH + (e / DK) * LDH + e % DK) = hv[m];
        }
#pragma unroll
        for (int m = 0; m < NKV; ++m) {
            const int i = lane, f = 4 * (w + (kThreads / kWave) * m);
            const f32x4 kk = i < valid ? kv[m] : f32x4{0.0f, 0.0f, 0.0f, 0.0f};
            *reinterpret_cast<float4*>(sK + i * LDH + f) = float4{kk[0], kk[1], kk[2], kk[3]};
#pragma unroll
            for (int q = 0; q < 4; ++q) sKT[(f + q) * LDT + i] = kk[q];
        }
        for (int f = tid; f < DK; f += kThreads) sLam[f] = a.lambda[int64_t(h) * DK + f];
        if (tid < kWave) chunk_log_decays(a.gamma + tok0, valid, sLg, sZl);
        if (tid < C) sBeta[tid] = tid < valid ? a.beta[tok0 + tid] : 0.0f;
    }
    // right-hand side (this lane's token, features 16t + 4g ..), zero past the sequence
    f32x4 qv[MT];
#pragma unroll
    for (int t = 0; t < MT; ++t) {
        const int64_t off = (tok0 + min(j, valid - 1)) * DK + 16 * t + 4 * g;
        f32x4 v = a.rhs ? load_vec4<DK>(a.rhs + off) : load_vec4<DK>(static_cast<const Tin*>(a.q) + off);
        qv[t] = j < valid ? v : f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    }
    __syncthreads();
    const float zeta = decay_from_start(sLg, sZl, j);
    // beta_i zeta_{j,i} for i = 16 it + 4g + ii <= j (zero past the causal tiles)
    f32x4 wz[4];
#pragma unroll
    for (int it = 0; it < 4; ++it)
#pragma unroll
        for (int ii = 0; ii < 4; ++ii) {
            const int i = 16 * it + 4 * g + ii;
            wz[it][ii] = (i <= j && i < valid) ? sBeta[i] * decay_between(sLg, sZl, i, j) : 0.0f;
        }

    // S = wz ⊙ (K P) over the causal token tiles it <= w
    auto kp_product = [&](const f32x4 (&pv)[MT], f32x4 (&sv)[4]) {
#pragma unroll
        for (int it = 0; it < 4; ++it) {
            f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
            if (it <= w) {
#pragma unroll
                for (int u = 0; u < MT; ++u) {
                    const float4 a4 = load4(sK + (16 * it + ln) * LDH + 16 * u + 4 * g);
                    acc = mfma4(a4.x, pv[u][0], acc);
                    acc = mfma4(a4.y, pv[u][1], acc);
                    acc = mfma4(a4.z, pv[u][2], acc);
                    acc = mfma4(a4.w, pv[u][3], acc);
                }
            }
            sv[it] = acc * wz[it];
            __builtin_amdgcn_sched_barrier(0);
        }
    };
    // acc[t] += M^T-tile products: rows 16t.. of a [row][token] LDS matrix times S
    auto add_rows_times_s = [&](const float* Mt, const f32x4 (&sv)[4], f32x4& acc, int t) {
#pragma unroll
        for (int it = 0; it < 4; ++it) {
            if (it > w) continue;
            const float4 a4 = load4(Mt + (16 * t + ln) * LDT + 16 * it + 4 * g);
            acc = mfma4(a4.x, sv[it][0], acc);
            acc = mfma4(a4.y, sv[it][1], acc);
            acc = mfma4(a4.z, sv[it][2], acc);
            acc = mfma4(a4.w, sv[it][3], acc);
        }
    };
    // W = zeta ⊙ (H_c P) + K^T S + lambda ⊙ P
    auto matvec = [&](const f32x4 (&pv)[MT], f32x4 (&wv)[MT]) {
        f32x4 sv[4];
        kp_product(pv, sv);
#pragma unroll
        for (int t = 0; t < MT; ++t) {
            f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int u = 0; u < MT; ++u) {
                const float4 a4 = load4(sH + (16 * t + ln) * LDH + 16 * u + 4 * g);
                acc = mfma4(a4.x, pv[u][0], acc);
                acc = mfma4(a4.y, pv[u][1], acc);
                acc = mfma4(a4.z, pv[u][2], acc);
                acc = mfma4(a4.w, pv[u][3], acc);
            }
            acc *= zeta;
            add_rows_times_s(sKT, sv, acc, t);
            const float4 l4 = load4(sLam + 16 * t + 4 * g);
            wv[t] = acc + f32x4{l4.x, l4.y, l4.z, l4.w} * pv[t];
            // one output tile's operands at a time (not every tile's A values at once)
            __builtin_amdgcn_sched_barrier(0);
        }
    };
    auto colsum = [&](const f32x4 (&x)[MT], const f32x4 (&y)[MT]) -> float {
        f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int t = 0; t < MT; ++t) acc += x[t] * y[t];
        return row_pair_sums((acc[0] + acc[1]) + (acc[2] + acc[3]));
    };

    // the column solves for q 2^-qsh (|q 2^-qsh|^2 in [1/2, 2)); x is scaled back at the end
    const int qsh = cg_scale_shift(colsum(qv, qv));
    {
        const float qs = __builtin_ldexpf(1.0f, -qsh);
#pragma unroll
        for (int t = 0; t < MT; ++t) qv[t] *= qs;
    }
    // ---- Jacobi start: diag(H_t + Lambda) = zeta diag(H_c) + sum_i beta_i zeta_{j,i} k_i ⊙ k_i + lambda
    f32x4 x[MT], r[MT], p[MT], wv[MT];
#pragma unroll
    for (int t = 0; t < MT; ++t) {
        f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int it = 0; it < 4; ++it) {
            if (it > w) continue;
            const float4 a4 = load4(sKT + (16 * t + ln) * LDT + 16 * it + 4 * g);
            acc = mfma4(a4.x * a4.x, wz[it][0], acc);
            acc = mfma4(a4.y * a4.y, wz[it][1], acc);
            acc = mfma4(a4.z * a4.z, wz[it][2], acc);
            acc = mfma4(a4.w * a4.w, wz[it][3], acc);
        }
        // acc holds row 16t + 4g + i of column j for i = 0..3
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int f = 16 * t + 4 * g + i;
            const float dg = zeta * sH[f * LDH + f] + acc[i] + sLam[f];
            x[t][i] = qv[t][i] / dg;
        }
    }
    matvec(x, wv);
#pragma unroll
    for (int t = 0; t < MT; ++t) {
        r[t] = qv[t] - wv[t];
        p[t] = r[t];
    }
    float delta = colsum(r, r);
    const float thr = a.eps2 * delta;  // Alg. 1: the column stops once |r|^2 <= eps^2 |r_0|^2
    bool active = delta >= kMinNormal;
    int steps = 0;
    for (int it = 0; it < a.n_cg; ++it) {
        if (!__any(active)) break;
        matvec(p, wv);
        const float pw = colsum(p, wv);
        if (active && !(pw >= kMinNormal)) active = false;
        if (active) {
            const float alpha = delta / pw;
#pragma unroll
            for (int t = 0; t < MT; ++t) {
                x[t] += alpha * p[t];
                r[t] -= alpha * wv[t];
            }
            ++steps;
        }
        const float dn = colsum(r, r);
        if (active) {
            if (dn <= thr || !(dn >= kMinNormal)) {
                active = false;
            } else {
                const float bcg = dn / delta;
#pragma unroll
                for (int t = 0; t < MT; ++t) p[t] = r[t] + bcg * p[t];
                delta = dn;
            }
        }
    }
    {
        const float us = __builtin_ldexpf(1.0f, qsh);
#pragma unroll
        for (int t = 0; t < MT; ++t) x[t] *= us;
    }
    if (a.steps && g == 0 && j < valid) a.steps[tok0 + j] = steps;
    if (a.qstar && j < valid) {
#pragma unroll
        for (int t = 0; t < MT; ++t)
            *reinterpret_cast<float4*>(a.qstar + (tok0 + j) * DK + 16 * t + 4 * g) = float4{x[t][0], x[t][1], x[t][2], x[t][3]};
    }
    if (!a.out) return;  // solve only (uniform across the workgroup)

    // ---- read-out o_j = zeta_j G_c x_j + sum_{i<=j} beta_i zeta_{j,i} v_i (k_i . x_j)
    f32x4 sv[4];
    kp_product(x, sv);
    __syncthreads();  // every wave is done with sH and sKT
    {
        const float* Gc = static_cast<const float*>(a.Gs) + (bh * s.n_chunks + n) * int64_t(DV) * DK;
        constexpr int NG = DV * DK / 4 / kThreads;
        float4 gv[NG];
#pragma unroll
        for (int m = 0; m < NG; ++m) gv[m] = load4(Gc + 4 * (tid + kThreads * m));
        constexpr int NVV = C * DV / 4 / kThreads;  // values: token per lane, as the keys
        f32x4 vv[NVV];
#pragma unroll
        for (int m = 0; m < NVV; ++m)
            vv[m] = load_vec4<DV>(vp + (tok0 + min(lane, valid - 1)) * DV + 4 * (w + (kThreads / kWave) * m));
#pragma unroll
        for (int m = 0; m < NG; ++m) {
            const int e = 4 * (tid + kThreads * m);
            *reinterpret_cast<float4*>(sH + (e / DK) * LDH + e % DK) = gv[m];
        }
#pragma unroll
        for (int m = 0; m < NVV; ++m) {
            const int i = lane, c = 4 * (w + (kThreads / kWave) * m);
#pragma unroll
            for (int q = 0; q < 4; ++q) sKT[(c + q) * LDT + i] = i < valid ? vv[m][q] : 0.0f;
        }
    }
    __syncthreads();
#pragma unroll
    for (int t = 0; t < MTV; ++t) {
        f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int u = 0; u < MT; ++u) {
            const float4 a4 = load4(sH + (16 * t + ln) * LDH + 16 * u + 4 * g);
            acc = mfma4(a4.x, x[u][0], acc);
            acc = mfma4(a4.y, x[u][1], acc);
            acc = mfma4(a4.z, x[u][2], acc);
            acc = mfma4(a4.w, x[u][3], acc);
        }
        acc *= zeta;
        add_rows_times_s(sKT, sv, acc, t);
        if (j < valid)
            *reinterpret_cast<float4*>(a.out + (tok0 + j) * DV + 16 * t + 4 * g) = float4{acc[0], acc[1], acc[2], acc[3]};
        __builtin_amdgcn_sched_barrier(0);
    }
}

template <typename Tin, int DK>
hipError_t launch_mma(const CgArgs& a, hipStream_t stream)
{
    const unsigned blocks = unsigned(a.s.batch * a.s.heads * a.s.n_chunks);
    if (a.s.d_v == 64)
        hipLaunchKernelGGL((chunk_cg_f32_mma_kernel<Tin, DK, 64>), dim3(blocks), dim3(kThreads), 0, stream, a);
    else
        hipLaunchKernelGGL((chunk_cg_f32_mma_kernel<Tin, DK, 128>), dim3(blocks), dim3(kThreads), 0, stream, a);
    return hipGetLastError();
}

template <typename Tin, int DK>
hipError_t launch_dk(const CgArgs& a, hipStream_t stream)
{
    if (a.s.chunk == 64) return launch_mma<Tin, DK>(a, stream);
    const unsigned blocks = unsigned(a.s.batch * a.s.heads * a.s.n_chunks);
    switch (a.s.chunk) {
        case 16: hipLaunchKernelGGL((chunk_cg_f32_kernel<Tin, DK, 16>), dim3(blocks), dim3(kThreads), 0, stream, a); break;
        case 32: hipLaunchKernelGGL((chunk_cg_f32_kernel<Tin, DK, 32>), dim3(blocks), dim3(kThreads), 0, stream, a); break;
        default: hipLaunchKernelGGL((chunk_cg_f32_kernel<Tin, DK, 64>), dim3(blocks), dim3(kThreads), 0, stream, a); break;
    }
    return hipGetLastError();
}

template <typename Tin>
hipError_t launch_tin(const CgArgs& a, hipStream_t stream)
{
    return a.s.d_k == 64 ? launch_dk<Tin, 64>(a, stream) : launch_dk<Tin, 128>(a, stream);
}

}  // namespace

hipError_t launch_chunk_cg_f32(const CgArgs& a, hipStream_t stream)
{
    return a.s.bf16 ? launch_tin<bf16_t>(a, stream) : launch_tin<float>(a, stream);
}

}  // namespace mesa
