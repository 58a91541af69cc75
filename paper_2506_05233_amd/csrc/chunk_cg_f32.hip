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
// This is the fp32 path: every product is an fp32 FMA with operands staged in
// LDS, so results agree with fp64 to about 1e-6.  Matrices over the chunk are
// held as [feature a][token j]; thread t owns column j = t % C and rows
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
    bool active = delta > 0.0f;
    int steps = 0;  // iterations that updated x
    for (int it = 0; it < a.n_cg; ++it) {
        if (!__syncthreads_or(active)) break;
        matvec(p, w);
        part = 0.0f;
#pragma unroll
        for (int m = 0; m < NE; ++m) part += p[m] * w[m];
        const float pw = colsum(part);
        if (active && !(pw > 0.0f)) active = false;
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
            if (dn <= thr) {
                active = false;
            } else {
                const float beta_cg = dn / delta;
#pragma unroll
                for (int m = 0; m < NE; ++m) p[m] = r[m] + beta_cg * p[m];
                delta = dn;
            }
        }
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

template <typename Tin, int DK>
hipError_t launch_dk(const CgArgs& a, hipStream_t stream)
{
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
