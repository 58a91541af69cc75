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
// reverse adjoint scan, the per-chunk gradients, and the Lambda reduction.
#include "mesa_device.hpp"
#include "mesa_kernels.hpp"
#include "mesa_mfma.hpp"

namespace mesa {
namespace {

constexpr int kThreads = 256;
constexpr int kC = 64;       // tokens per chunk of the backward
constexpr int kLdT = 132;    // row stride of [token][feature] tiles (16-byte rows)
constexpr int kLdC = 68;     // row stride of [token][token] matrices (16-byte rows)

constexpr int kLdO = 129;    // odd row stride: tiles read one row per lane

template <typename T>
__device__ __forceinline__ void load_tile(float* dst, const T* src, int64_t tok0, int valid, int d, int ld = kLdT)
{
    for (int e = threadIdx.x; e < kC * d; e += kThreads) {
        const int i = e / d, f = e % d;
        dst[i * ld + f] = i < valid ? to_f32(src[(tok0 + i) * d + f]) : 0.0f;
    }
}

// Per-token sums over the D features of a token group (thread layout: feature
// tid % D, token group tid / D, tokens tg * NS + m): wave sums, then the waves of a
// group through LDS.  out[t] receives the sum for token t.
template <int D>
__device__ __forceinline__ void token_sums(const float (&part)[kC / (kThreads / D)], float* out, float (*sPart)[kC])
{
    constexpr int NTG = kThreads / D, NS = kC / NTG, WPG = D / kWave;
    const int tid = threadIdx.x, tg = tid / D, w = tid / kWave, lane = tid % kWave;
#pragma unroll
    for (int m = 0; m < NS; ++m) {
        const float v = wave_sum(part[m]);
        if (lane == 0) sPart[w][tg * NS + m] = v;
    }
    __syncthreads();
    if (tid < kC) {
        const int g = tid / NS;
        float acc = 0.0f;
#pragma unroll
        for (int u = 0; u < WPG; ++u) acc += sPart[g * WPG + u][tid];
        out[tid] = acc;
    }
    __syncthreads();
}

// ---------------------------------------------------------------- u = G^T e
// u_t = zeta_{t,c-1} G_c^T e_t + sum_{i<=t} zeta_{t,i} beta_i (v_i . e_t) k_i for
// the tokens of one chunk (the GLA form of App. D with the roles of k and v swapped).
template <typename Tin, int DK, int DV>
__global__ __launch_bounds__(kThreads) void bwd_rhs_kernel(BwdArgs a)
{
    constexpr int NTG = kThreads / DK, NS = kC / NTG;  // token groups; tokens per thread
    const ForwardShape s = a.s;
    const int nc = s.n_chunks;
    const int n = blockIdx.x % nc;
    const int64_t bh = blockIdx.x / nc;
    const int64_t t0 = int64_t(n) * kC;
    const int valid = int(min<int64_t>(kC, s.seq_len - t0));
    const int64_t tok0 = bh * s.seq_len + t0;
    const int tid = threadIdx.x;

    __shared__ float sE[kC * kLdO];   // e_t [t][a]
    __shared__ float sX[kC * kLdO];   // v_i, then k_i
    __shared__ float sS[kC * kLdC];   // beta_i zeta_{t,i} (v_i . e_t) as [t][i]
    __shared__ float sLg[kC];
    __shared__ int sZl[kC];

    load_tile(sE, a.dout, tok0, valid, DV, kLdO);
    load_tile(sX, static_cast<const Tin*>(a.v), tok0, valid, DV, kLdO);
    if (tid < kWave) chunk_log_decays(a.gamma + tok0, valid, sLg, sZl);
    __syncthreads();
    for (int e = tid; e < kC * kC; e += kThreads) {
        const int t = e / kC, i = e % kC;
        float acc = 0.0f;
        if (i <= t && i < valid) {
            for (int c = 0; c < DV; ++c) acc += sX[i * kLdO + c] * sE[t * kLdO + c];
            acc *= a.beta[tok0 + i] * decay_between(sLg, sZl, i, t);
        }
        sS[t * kLdC + i] = acc;
    }
    __syncthreads();
    load_tile(sX, static_cast<const Tin*>(a.k), tok0, valid, DK, kLdO);
    __syncthreads();

    const int b = tid % DK, tg = tid / DK;  // this thread's feature and token group
    float acc[NS];
#pragma unroll
    for (int m = 0; m < NS; ++m) acc[m] = 0.0f;
    const float* Gc = a.Gs + (bh * nc + n) * int64_t(DV) * DK;
    for (int c = 0; c < DV; ++c) {
        const float g = Gc[c * DK + b];  // G_c[c][b]: one row of G_c per step, coalesced
#pragma unroll
        for (int m = 0; m < NS; ++m) acc[m] += g * sE[(tg * NS + m) * kLdO + c];
    }
#pragma unroll
    for (int m = 0; m < NS; ++m) acc[m] *= decay_from_start(sLg, sZl, tg * NS + m);
    for (int i = 0; i < kC; ++i) {
        const float ki = sX[i * kLdO + b];
#pragma unroll
        for (int m = 0; m < NS; ++m) acc[m] += sS[(tg * NS + m) * kLdC + i] * ki;
    }
#pragma unroll
    for (int m = 0; m < NS; ++m) {
        const int t = tg * NS + m;
        if (t >= valid) continue;
        if (a.u16)
            a.u16[(tok0 + t) * DK + b] = uint16_t(pack_bf16x2(acc[m], 0.0f) & 0xffffu);  // round to nearest even
        else
            a.u[(tok0 + t) * DK + b] = acc[m];
    }
}

// ---------------------------------------------------------------- adjoint scan
// One workgroup owns 16 rows of S^H (d_k x d_k) or of A^G (d_v x d_k) of one
// sequence and walks the chunks from last to first; the tile stays in registers.
constexpr int kTileRows = 16;
constexpr int kPerThread = kTileRows * 128 / kThreads;  // 8

template <int DK, int DV>
__global__ __launch_bounds__(kThreads) void bwd_adjoint_kernel(BwdArgs a)
{
    constexpr int NTH = DK / kTileRows;          // row tiles of S^H
    constexpr int NTILE = NTH + DV / kTileRows;  // then row tiles of A^G
    constexpr int NEL = kTileRows * DK;
    const ForwardShape s = a.s;
    const int nc = s.n_chunks;
    const int blk = xcd_major_block(blockIdx.x, gridDim.x);
    const int tile = blk % NTILE;
    const int64_t bh = blk / NTILE;
    const bool isG = tile >= NTH;
    const int r0 = (isG ? tile - NTH : tile) * kTileRows;
    const int nrow = isG ? DV : DK;
    const int tid = threadIdx.x;

    __shared__ float sX[kC][DK + 1];             // q*_j, all columns
    __shared__ float sY[kC][DK + 1];             // -e*_j, all columns (S^H only)
    __shared__ float sYr[kC][kTileRows + 1];     // rows r0.. of e_j (A^G) or -e*_j (S^H)
    __shared__ float sXr[kC][kTileRows + 1];     // rows r0.. of q*_j (S^H only)
    __shared__ float sW[kC];                     // zeta_{j, c-1}: decay from the chunk's entry to j
    __shared__ float sLg[kC];
    __shared__ int sZl[kC];

    float st[kPerThread];
#pragma unroll
    for (int m = 0; m < kPerThread; ++m) st[m] = 0.0f;
    float* out = isG ? a.AG : a.SH;
    for (int n = nc - 1; n >= 0; --n) {
        const int64_t t0 = int64_t(n) * kC;
        const int valid = int(min<int64_t>(kC, s.seq_len - t0));
        const int64_t tok0 = bh * s.seq_len + t0;
        float* dst = out + ((bh * nc + n) * nrow + r0) * int64_t(DK);
#pragma unroll
        for (int m = 0; m < kPerThread; ++m) {
            const int e = tid + kThreads * m;
            if (e < NEL) dst[e] = st[m];
        }
        for (int e = tid; e < kC * DK; e += kThreads) {
            const int j = e / DK, c = e % DK;
            const bool ok = j < valid;
            sX[j][c] = ok ? a.qstar[(tok0 + j) * DK + c] : 0.0f;
            if (!isG) sY[j][c] = ok ? -a.estar[(tok0 + j) * DK + c] : 0.0f;
        }
        for (int e = tid; e < kC * kTileRows; e += kThreads) {
            const int j = e / kTileRows, r = e % kTileRows;
            const bool ok = j < valid;
            sYr[j][r] = ok ? (isG ? a.dout[(tok0 + j) * DV + r0 + r] : -a.estar[(tok0 + j) * DK + r0 + r]) : 0.0f;
            if (!isG) sXr[j][r] = ok ? a.qstar[(tok0 + j) * DK + r0 + r] : 0.0f;
        }
        if (tid < kWave) chunk_log_decays(a.gamma + tok0, valid, sLg, sZl);
        __syncthreads();
        if (tid < kC) sW[tid] = tid < valid ? decay_from_start(sLg, sZl, tid) : 0.0f;
        __syncthreads();
        const float D = decay_from_start(sLg, sZl, kC - 1);
#pragma unroll
        for (int m = 0; m < kPerThread; ++m) {
            const int e = tid + kThreads * m;
            if (e < NEL) {
                const int row = e / DK, col = e % DK;
                float acc = 0.0f;
                if (isG) {
                    for (int j = 0; j < kC; ++j) acc += sW[j] * sYr[j][row] * sX[j][col];
                } else {
                    for (int j = 0; j < kC; ++j) acc += sW[j] * (sYr[j][row] * sX[j][col] + sXr[j][row] * sY[j][col]);
                }
                st[m] = D * st[m] + acc;
            }
        }
        __syncthreads();
    }
}

// ---------------------------------------------------------------- per-chunk gradients
// Thread layout for per-feature outputs over D features: feature f = tid % D, token
// group tg = tid / D (uniform in a wave), tokens tg * (C / NTG) + m.
template <typename Tin, int DK, int DV>
__global__ __launch_bounds__(kThreads) void bwd_grad_kernel(BwdArgs a)
{
    const ForwardShape s = a.s;
    const int nc = s.n_chunks;
    const int n = blockIdx.x % nc;
    const int64_t bh = blockIdx.x / nc;
    const int64_t t0 = int64_t(n) * kC;
    const int valid = int(min<int64_t>(kC, s.seq_len - t0));
    const int64_t tok0 = bh * s.seq_len + t0;
    const int tid = threadIdx.x;
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
    __shared__ __attribute__((aligned(16))) float sM1[kC * kLdC];  // VE, then VE - KE, then M2 = Z ⊙ (VE - KE)
    __shared__ __attribute__((aligned(16))) float sM2[kC * kLdC];  // KE, then Qm = beta_p (VE - KE) KQ
    __shared__ __attribute__((aligned(16))) float sZ[kC * kLdC];   // Z[s][t] = zeta_{t,s} (s <= t)
    __shared__ float sLg[kC];
    __shared__ int sZl[kC];
    __shared__ float sBeta[kC], sZe[kC], sPhi[kC];
    __shared__ float sTok[5][kC];   // per-token: dbeta (intra), v^T A^G k, k^T A^H k, g, h
    __shared__ float sPart[kThreads / kWave][kC];
    __shared__ float sF;

    // ---- gates: Z, zeta_{E,s}, phi_s = zeta_{s-1,c-1}
    if (tid < kWave) chunk_log_decays(a.gamma + tok0, valid, sLg, sZl);
    __syncthreads();
    for (int e = tid; e < kC * kC; e += kThreads) {
        const int i = e / kC, j = e % kC;
        sZ[i * kLdC + j] = decay_between(sLg, sZl, i, j);
    }
    if (tid < kC) {
        sBeta[tid] = tid < valid ? a.beta[tok0 + tid] : 0.0f;
        sZe[tid] = decay_between(sLg, sZl, tid, kC - 1);
        sPhi[tid] = tid == 0 ? 1.0f : decay_from_start(sLg, sZl, tid - 1);
    }

    // ---- grams of the chunk's tokens, 4x4 register blocks: entry (p, t) with
    // p = pb + 16 i, t = tb + 16 j
    const int pb = tid / 16, tb = tid % 16;
    auto gram = [&](float* dst, int d) {
        float g[4][4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) g[i][j] = 0.0f;
        for (int f = 0; f < d; ++f) {
            float x[4], y[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) x[i] = sT0[(pb + 16 * i) * kLdT + f];
#pragma unroll
            for (int j = 0; j < 4; ++j) y[j] = sT1[(tb + 16 * j) * kLdT + f];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) g[i][j] += x[i] * y[j];
        }
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) dst[(pb + 16 * i) * kLdC + tb + 16 * j] = g[i][j];
    };
    load_tile(sT0, kp, tok0, valid, DK);
    load_tile(sT1, a.qstar, tok0, valid, DK);
    __syncthreads();
    gram(sM0, DK);  // KQ[p][t] = k_p . q*_t
    __syncthreads();
    load_tile(sT1, a.estar, tok0, valid, DK);
    __syncthreads();
    gram(sM2, DK);  // KE[p][t] = k_p . e*_t
    __syncthreads();
    load_tile(sT0, vp, tok0, valid, DV);
    load_tile(sT1, a.dout, tok0, valid, DV);
    __syncthreads();
    gram(sM1, DV);  // VE[p][t] = v_p . e_t
    __syncthreads();

    // ---- C x C combinations: DVK = VE - KE; Qm = beta_p DVK KQ; the intra part of
    // dbeta_s = sum_t Z[s][t] KQ[s][t] DVK[s][t]; then M1 = Z ⊙ KQ, M2 = Z ⊙ DVK
    for (int e = tid; e < kC * kC; e += kThreads) {
        const int p = e / kC, t = e % kC, o = p * kLdC + t;
        const float dvk = sM1[o] - sM2[o];
        sM1[o] = dvk;
        sM2[o] = sBeta[p] * dvk * sM0[o];
    }
    __syncthreads();
    if (tid < kC) {
        float acc = 0.0f;
        for (int t = 0; t < kC; ++t) acc += sZ[tid * kLdC + t] * sM0[tid * kLdC + t] * sM1[tid * kLdC + t];
        sTok[0][tid] = acc;
    }
    __syncthreads();
    for (int e = tid; e < kC * kC; e += kThreads) {
        const int p = e / kC, t = e % kC, o = p * kLdC + t;
        sM0[o] *= sZ[o];
        sM1[o] *= sZ[o];
    }
    __syncthreads();

    // ---- dv (features a over DV): beta_s (sum_t M1[s][t] e_t[a] + zeta_E[s] (A^G k_s)[a])
    {
        constexpr int NTG = kThreads / DV, NS = kC / NTG;
        const int f = tid % DV, tg = tid / DV;
        float acc[NS], inter[NS];
        // sT1 still holds e_t; sT0 gets k_s
        __syncthreads();
        load_tile(sT0, kp, tok0, valid, DK);
        __syncthreads();
#pragma unroll
        for (int m = 0; m < NS; ++m) acc[m] = inter[m] = 0.0f;
        for (int t = 0; t < kC; ++t) {
            const float et = sT1[t * kLdT + f];
#pragma unroll
            for (int m = 0; m < NS; ++m) acc[m] += sM0[(tg * NS + m) * kLdC + t] * et;
        }
        const float* row = AG + int64_t(f) * DK;  // A^G[f][.]
        for (int c = 0; c < DK; c += 4) {
            const float4 g4 = *reinterpret_cast<const float4*>(row + c);
#pragma unroll
            for (int m = 0; m < NS; ++m) {
                const float4 k4 = *reinterpret_cast<const float4*>(sT0 + (tg * NS + m) * kLdT + c);
                inter[m] += g4.x * k4.x + g4.y * k4.y + g4.z * k4.z + g4.w * k4.w;
            }
        }
#pragma unroll
        for (int m = 0; m < NS; ++m) {
            const int t = tg * NS + m;
            const float dgk = acc[m] + sZe[t] * inter[m];  // (DG_s k_s)[f]
            if (t < valid) a.dv[(tok0 + t) * DV + f] = sBeta[t] * dgk;
        }
    }

    // ---- dk (features b over DK): beta_s (sum_t M2[s][t] q*_t[b] - sum_t M1[s][t] e*_t[b]
    //      + zeta_E[s] ((A^G)^T v_s + S^H k_s)[b]);  also aG_s = v_s^T A^G k_s and
    //      kAHk_s = k_s^T A^H k_s = (1/2) k_s^T S^H k_s
    {
        constexpr int NTG = kThreads / DK, NS = kC / NTG;
        const int f = tid % DK, tg = tid / DK;
        float acc[NS], ag[NS], sh[NS];
        __syncthreads();
        load_tile(sT0, a.qstar, tok0, valid, DK);
        load_tile(sT1, a.estar, tok0, valid, DK);
        __syncthreads();
#pragma unroll
        for (int m = 0; m < NS; ++m) acc[m] = ag[m] = sh[m] = 0.0f;
        for (int t = 0; t < kC; ++t) {
            const float qt = sT0[t * kLdT + f], et = sT1[t * kLdT + f];
#pragma unroll
            for (int m = 0; m < NS; ++m) {
                const int o = (tg * NS + m) * kLdC + t;
                acc[m] += sM1[o] * qt - sM0[o] * et;
            }
        }
        __syncthreads();
        load_tile(sT0, kp, tok0, valid, DK);
        load_tile(sT1, vp, tok0, valid, DV);
        __syncthreads();
        for (int c = 0; c < DV; ++c) {
            const float g = AG[c * DK + f];  // A^G[c][f], coalesced over f
#pragma unroll
            for (int m = 0; m < NS; ++m) ag[m] += g * sT1[(tg * NS + m) * kLdT + c];
        }
        for (int c = 0; c < DK; ++c) {
            const float h = SH[c * DK + f];  // S^H[c][f] = S^H[f][c]
#pragma unroll
            for (int m = 0; m < NS; ++m) sh[m] += h * sT0[(tg * NS + m) * kLdT + c];
        }
        float pa[NS], pk[NS];
#pragma unroll
        for (int m = 0; m < NS; ++m) {
            const int t = tg * NS + m;
            const float kf = sT0[t * kLdT + f];
            if (t < valid) a.dk[(tok0 + t) * DK + f] = sBeta[t] * (acc[m] + sZe[t] * (ag[m] + sh[m]));
            pa[m] = kf * ag[m];          // k_s[f] ((A^G)^T v_s)[f]  -> v_s^T A^G k_s
            pk[m] = 0.5f * kf * sh[m];   // (1/2) k_s[f] (S^H k_s)[f] -> k_s^T A^H k_s
        }
        token_sums<DK>(pa, sTok[1], sPart);
        token_sums<DK>(pk, sTok[2], sPart);
    }

    // ---- g_t = e_t^T G_c q*_t and h_t = e*_t^T H_c q*_t (features b over DK), and
    //      F = <A^G, G_c> + (1/2) <S^H, H_c>
    {
        constexpr int NTG = kThreads / DK, NS = kC / NTG;
        const int f = tid % DK, tg = tid / DK;
        float w[NS];
        __syncthreads();
        load_tile(sT0, a.qstar, tok0, valid, DK);
        load_tile(sT1, a.dout, tok0, valid, DV);
        __syncthreads();
#pragma unroll
        for (int m = 0; m < NS; ++m) w[m] = 0.0f;
        for (int c = 0; c < DV; ++c) {
            const float g = Gc[c * DK + f];
#pragma unroll
            for (int m = 0; m < NS; ++m) w[m] += g * sT1[(tg * NS + m) * kLdT + c];
        }
        float pg[NS];
#pragma unroll
        for (int m = 0; m < NS; ++m) pg[m] = w[m] * sT0[(tg * NS + m) * kLdT + f];
        token_sums<DK>(pg, sTok[3], sPart);
        load_tile(sT1, a.estar, tok0, valid, DK);
        __syncthreads();
#pragma unroll
        for (int m = 0; m < NS; ++m) w[m] = 0.0f;
        for (int c = 0; c < DK; ++c) {
            const float h = Hc[c * DK + f];
#pragma unroll
            for (int m = 0; m < NS; ++m) w[m] += h * sT1[(tg * NS + m) * kLdT + c];
        }
#pragma unroll
        for (int m = 0; m < NS; ++m) pg[m] = w[m] * sT0[(tg * NS + m) * kLdT + f];
        token_sums<DK>(pg, sTok[4], sPart);
        // F: every thread a strided slice of the two Frobenius products
        float fr = 0.0f;
        for (int e = tid; e < DV * DK; e += kThreads) fr += AG[e] * Gc[e];
        for (int e = tid; e < DK * DK; e += kThreads) fr += 0.5f * SH[e] * Hc[e];
        fr = wave_sum(fr);
        if (tid % kWave == 0) sPart[tid / kWave][0] = fr;
        __syncthreads();
        if (tid == 0) {
            float t = 0.0f;
            for (int u = 0; u < kThreads / kWave; ++u) t += sPart[u][0];
            sF = t;
        }
        // dLambda of this chunk: -sum_t q*_t[b] e*_t[b]
        if (tid < DK) {
            float acc = 0.0f;
            for (int t = 0; t < kC; ++t) acc += sT0[t * kLdT + tid] * sT1[t * kLdT + tid];
            a.dlam_part[mat * DK + tid] = -acc;
        }
        __syncthreads();
    }

    // ---- W[p][s] = sum_{t>=s} zeta_{t,s} Qm[p][t] (4x4 blocks, into sM0)
    {
        float g[4][4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) g[i][j] = 0.0f;
        for (int t = 0; t < kC; ++t) {
            float x[4], y[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) x[i] = sM2[(pb + 16 * i) * kLdC + t];
#pragma unroll
            for (int j = 0; j < 4; ++j) y[j] = sZ[(tb + 16 * j) * kLdC + t];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) g[i][j] += x[i] * y[j];
        }
        __syncthreads();
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) sM0[(pb + 16 * i) * kLdC + tb + 16 * j] = g[i][j];
        __syncthreads();
    }

    // ---- assemble dgamma_s and dbeta_s (one thread per token)
    if (tid < kC) {
        const int si = tid;
        const float ze = sZe[si], phi = sPhi[si];
        float t2 = 0.0f, t3 = 0.0f, t4 = 0.0f;
        for (int t = si; t < kC; ++t) t2 += sZ[si * kLdC + t] * (sTok[3][t] - sTok[4][t]);
        for (int p = 0; p < si; ++p) {
            const float z = sZ[p * kLdC + si - 1];  // zeta_{s-1,p}
            t3 += z * sBeta[p] * (sTok[1][p] + sTok[2][p]);
            t4 += z * sM0[p * kLdC + si];
        }
        const float dg = ze * phi * sF + phi * t2 + ze * t3 + t4;
        const float db = sTok[0][si] + ze * (sTok[1][si] + sTok[2][si]);
        if (si < valid) {
            a.dgamma[tok0 + si] = dg;
            a.dbeta[tok0 + si] = db;
        }
    }
}

// ---------------------------------------------------------------- dLambda
// dLambda[h][b] = sum over the batch and the chunks of the per-chunk partial sums.
__global__ __launch_bounds__(kThreads) void bwd_dlam_kernel(BwdArgs a)
{
    const ForwardShape s = a.s;
    const int dk = s.d_k;
    const int64_t idx = int64_t(blockIdx.x) * kThreads + threadIdx.x;
    if (idx >= s.heads * dk) return;
    const int64_t h = idx / dk;
    const int b = int(idx % dk);
    float acc = 0.0f;
    for (int64_t bb = 0; bb < s.batch; ++bb) {
        const int64_t bh = bb * s.heads + h;
        for (int n = 0; n < s.n_chunks; ++n) acc += a.dlam_part[(bh * s.n_chunks + n) * dk + b];
    }
    a.dlam[idx] = acc;
}

template <typename Tin, int DK, int DV>
hipError_t launch_bwd_dims(const BwdArgs& a, hipStream_t stream, int stage)
{
    const int64_t bh = a.s.batch * a.s.heads;
    const unsigned chunks = unsigned(bh * a.s.n_chunks);
    switch (stage) {
        case 0:
            hipLaunchKernelGGL((bwd_rhs_kernel<Tin, DK, DV>), dim3(chunks), dim3(kThreads), 0, stream, a);
            break;
        case 1:
            hipLaunchKernelGGL((bwd_adjoint_kernel<DK, DV>), dim3(unsigned(bh * (DK + DV) / kTileRows)), dim3(kThreads), 0,
                               stream, a);
            break;
        case 2:
            hipLaunchKernelGGL((bwd_grad_kernel<Tin, DK, DV>), dim3(chunks), dim3(kThreads), 0, stream, a);
            break;
        default: {
            const int64_t n = a.s.heads * DK;
            hipLaunchKernelGGL(bwd_dlam_kernel, dim3(unsigned((n + kThreads - 1) / kThreads)), dim3(kThreads), 0, stream, a);
        }
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
