// Chunked conjugate gradients + read-out on the gfx950 matrix cores (bf16
// operands, fp32 accumulation), for bf16 q, k, v and chunk C = 64.
//
// Same mathematics as the fp32 path (App. C, Alg. 1 with tolerance 0; App. D,
// Eq. q_star_parallel and Eq. gla): for the chunk starting after token c,
// with zeta_j = zeta_{c+j,c} and Z[i][j] = zeta_{c+j,c+i},
//
//   (H_t + Lambda) p_j = H_c (zeta_j p_j) + sum_{i<=j} beta_i Z[i][j] k_i (k_i^T p_j) + Lambda p_j
//   o_j               = G_c (zeta_j x_j) + sum_{i<=j} beta_i Z[i][j] v_i (k_i^T x_j).
//
// Work split: a workgroup is one chunk; wave w owns the 16-token sub-chunk
// j = 16w .. 16w+15 and runs its own CG on it with no barrier.  Each wave
// first forms the state that enters its sub-chunk,
//
//   B_w = zeta_{16w-1} H_c + sum_{i < 16w} beta_i zeta_{16w-1,i} k_i k_i^T   (B_0 = H_c),
//
// on the matrix cores (a rank-16w update of H_c; H and B_w are symmetric, so
// the result tiles come out directly in the A-operand layout), and keeps it as
// bf16 A-fragments in registers.  Inside CG every product is then
//
//   (H_t + Lambda) p_j = B_w (zt_j p_j) + sum_{16w <= i <= j} beta_i Z[i][j] k_i (k_i^T p_j) + Lambda p_j,
//
// with zt_j = zeta_{c+j, c+16w-1}: d_k/16 x d_k/32 MFMAs for the state term
// (B_w read from the accumulation registers), a 16-token S = K_w p (d_k/32
// MFMAs), and one MFMA per 16-row tile that adds both K_w^T (beta Z ⊙ S) and
// Lambda p (half of its 32-long contraction each).  All four waves do the same
// work, and every operand of the CG loop stays in registers.
//
// Every per-token vector (x, r, p, w) lives in registers in the layout of a
// 16x16 MFMA result: lane (g = lane/16, n = lane%16) holds rows 16t + 4g + {0..3}
// of column n for each 16-row tile t.  The 32-long contraction of
// v_mfma_f32_16x16x32_bf16 takes, in lane group g, rows 32s + 4g + {0..3} and
// 32s + 16 + 4g + {0..3}: the lane's own values of two stacked tiles, so a CG
// vector feeds the next product straight from registers (A operands use the
// same index map).  CG scalars reduce over the 4 lanes of a column with two
// cross-lane shuffles.  Only the MFMA operands are bf16; x, r, p, w, alpha,
// beta and every reduction stay fp32.
//
// The read-out o_j = G_c (zeta_j x_j) + sum_{i <= j} beta_i Z[i][j] v_i (k_i^T x_j)
// runs once per chunk over the whole causal chunk.
#include "mesa_device.hpp"
#include "mesa_kernels.hpp"
#include "mesa_mfma.hpp"

namespace mesa {
namespace {

constexpr int kC = 64;         // chunk
constexpr int kThreads = 256;  // four waves, 16 tokens each

// Same, with every element squared (fp32 square, rounded back to bf16).
__device__ __forceinline__ bf16x8 lds_frag_sq(const uint16_t* base)
{
    bf16x8 f = lds_frag(base);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const float v = (float)f[e];
        f[e] = (__bf16)(v * v);
    }
    return f;
}

// Gate decays with the hardware exponential (relative error ~1e-7, far below
// the bf16 operand rounding of this path); same zero-gate rules as the
// shared helpers.
__device__ __forceinline__ float decay_between_hw(const float* lg, const int* zl, int i, int j)
{
    if (i > j || zl[j] > i) return 0.0f;
    return __expf(lg[j] - lg[i]);
}

__device__ __forceinline__ float decay_from_start_hw(const float* lg, const int* zl, int j)
{
    return zl[j] >= 0 ? 0.0f : __expf(lg[j]);
}

// Sum over the four lanes that hold one column (lanes n, n+16, n+32, n+48).
__device__ __forceinline__ float col_sum(float v) { return row_pair_sums(v); }

template <int DK, int DV>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
void chunk_cg_bf16_kernel(CgArgs a)
{
    constexpr int MT = DK / 16;    // 16-row tiles of a per-token vector
    constexpr int KS = DK / 32;    // 32-long contraction steps over features
    constexpr int MTV = DV / 16;   // 16-row tiles of an output column
    constexpr int LDK = DK + 8;    // row stride (elements) of token-major tiles
    constexpr int LDC = kC + 8;    // row stride of feature-major tiles

    const ForwardShape s = a.s;
    const int n = blockIdx.x % s.n_chunks;
    const int64_t bh = blockIdx.x / s.n_chunks;
    const int h = int(bh % s.heads);
    const int64_t t0 = int64_t(n) * kC;
    const int valid = int(min<int64_t>(kC, s.seq_len - t0));
    const int64_t tok0 = bh * s.seq_len + t0;
    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
    const int lane = tid % kWave;
    const int g = lane / 16;   // lane group: rows 4g..4g+3 of each tile
    const int ln = lane % 16;  // column (B / result layout) or row (A layout)
    const int j = wave * 16 + ln;  // this lane's token within the chunk

    __shared__ __attribute__((aligned(16))) uint16_t sK[kC * LDK];   // k_i[b], token-major
    __shared__ __attribute__((aligned(16))) uint16_t sKT[DK * LDC];  // k_i[b], feature-major
    __shared__ __attribute__((aligned(16))) uint16_t sVT[DV * LDC];  // v_i[e], feature-major
    __shared__ __attribute__((aligned(16))) uint16_t sQ[kC * LDK];   // q_j[b], token-major
    __shared__ float sLg[kWave], sBeta[kWave];
    __shared__ int sZl[kWave];
    __shared__ __attribute__((aligned(16))) float sLam[DK];
    __shared__ float sT[kC * (kC + 1)];  // beta_i Z[i][j] as [i][j] (row stride 65), 0 for i > j
    __shared__ float sZ0[kC];            // zeta_{c+j,c}: decay from the chunk's entering state

    // ---- stage the chunk's keys, values and queries (bf16 bits) in LDS
    const uint16_t* kp = static_cast<const uint16_t*>(a.k);
    const uint16_t* qp = static_cast<const uint16_t*>(a.q);
    const uint16_t* vp = static_cast<const uint16_t*>(a.v);
    // every global load of the chunk is issued before the first LDS write;
    // thread t stages tokens 2p, 2p+1 (p = t % 32) for 8 features per pass
    constexpr int NKQ = DK / 64;  // passes over the key features (8 groups of 8 per pass)
    constexpr int NV = DV / 64;
    const int p2 = tid % 32, fg = tid / 32;
    const int i0 = 2 * p2, i1 = 2 * p2 + 1;
    uint4 kv[NKQ][2], qv[NKQ][2], vv[NV][2];
#pragma unroll
    for (int m = 0; m < NKQ; ++m) {
        const int f0 = 64 * m + 8 * fg;
        kv[m][0] = kv[m][1] = qv[m][0] = qv[m][1] = make_uint4(0, 0, 0, 0);
        if (i0 < valid) {
            kv[m][0] = *reinterpret_cast<const uint4*>(kp + (tok0 + i0) * DK + f0);
            qv[m][0] = *reinterpret_cast<const uint4*>(qp + (tok0 + i0) * DK + f0);
        }
        if (i1 < valid) {
            kv[m][1] = *reinterpret_cast<const uint4*>(kp + (tok0 + i1) * DK + f0);
            qv[m][1] = *reinterpret_cast<const uint4*>(qp + (tok0 + i1) * DK + f0);
        }
    }
#pragma unroll
    for (int m = 0; m < NV; ++m) {
        const int f0 = 64 * m + 8 * fg;
        vv[m][0] = i0 < valid ? *reinterpret_cast<const uint4*>(vp + (tok0 + i0) * DV + f0) : make_uint4(0, 0, 0, 0);
        vv[m][1] = i1 < valid ? *reinterpret_cast<const uint4*>(vp + (tok0 + i1) * DV + f0) : make_uint4(0, 0, 0, 0);
    }
    // chunk states as bf16 A-fragments: fragment (t, s) of lane l at [(t * KS + s) * 64 + l] * 8
    const uint16_t* Hf = static_cast<const uint16_t*>(a.Hs) + (bh * s.n_chunks + n) * int64_t(DK) * DK;
    const uint16_t* Gf = static_cast<const uint16_t*>(a.Gs) + (bh * s.n_chunks + n) * int64_t(DV) * DK;
    bf16x8 hc[MT][KS];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
            hc[mt][ks] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(Hf + ((mt * KS + ks) * 64 + lane) * 8));
    // diag(H_c) for the rows r = 16mt + 4g + ii this lane holds: fragment (mt, mt/2),
    // lane 16g + 4g + ii, element 4 (mt % 2) + ii
    f32x4 hdiag[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int ii = 0; ii < 4; ++ii)
            hdiag[mt][ii] = bf16_bits_to_f32(Hf[((mt * KS + mt / 2) * 64 + 20 * g + ii) * 8 + 4 * (mt % 2) + ii]);
    const float* lam = a.lambda + int64_t(h) * DK;
    if (tid < DK) sLam[tid] = lam[tid];
#pragma unroll
    for (int m = 0; m < NKQ; ++m) {
        const int f0 = 64 * m + 8 * fg;
        *reinterpret_cast<uint4*>(sK + i0 * LDK + f0) = kv[m][0];
        *reinterpret_cast<uint4*>(sK + i1 * LDK + f0) = kv[m][1];
        *reinterpret_cast<uint4*>(sQ + i0 * LDK + f0) = qv[m][0];
        *reinterpret_cast<uint4*>(sQ + i1 * LDK + f0) = qv[m][1];
        stage_token_pair(reinterpret_cast<uint32_t*>(sKT), LDC / 2, f0, p2, kv[m][0], kv[m][1]);
    }
#pragma unroll
    for (int m = 0; m < NV; ++m)
        stage_token_pair(reinterpret_cast<uint32_t*>(sVT), LDC / 2, 64 * m + 8 * fg, p2, vv[m][0], vv[m][1]);
    if (tid < kWave) {
        chunk_log_decays(a.gamma + tok0, valid, sLg, sZl);
        sBeta[tid] = tid < valid ? a.beta[tok0 + tid] : 0.0f;
    }

    __syncthreads();
    for (int e = tid; e < kC * kC; e += kThreads) {
        const int i = e / kC, jj = e % kC;
        sT[i * (kC + 1) + jj] = sBeta[i] * decay_between_hw(sLg, sZl, i, jj);
    }
    if (tid < kC) sZ0[tid] = decay_from_start_hw(sLg, sZl, tid);
    __syncthreads();

    // ---- decays of this sub-chunk
    const int jb = 16 * wave - 1;  // token whose state enters the sub-chunk (-1: the chunk's H_c)
    const float Dw = wave == 0 ? 1.0f : sZ0[jb];
    // B_w = Dw H_c + sum_{i<16w} u_i k_i k_i^T with u_i = beta_i zeta_{16w-1,i}.  It is kept as
    // B'_w = B_w / Dw = H_c + sum (u_i / Dw) k_i k_i^T and the 1/Dw goes into the column scale:
    // zs_j = zt_j Dw = zeta_{c+j,c}.  When Dw is negligible (<= 1e-20, e.g. a zero gate) the
    // state term Dw H_c is dropped instead: B_w = sum u_i k_i k_i^T and zs_j = zt_j.
    const bool keepH = wave == 0 || Dw > 1e-20f;
    const float zs = keepH ? sZ0[j] : decay_between_hw(sLg, sZl, jb, j);
    const float ush = keepH && wave > 0 ? 1.0f / Dw : 1.0f;
    f32x4 zw;  // beta_i Z[i][j] for the sub-chunk rows i = 16w + 4g + ii met in S
#pragma unroll
    for (int ii = 0; ii < 4; ++ii) {
        const int i = 16 * wave + 4 * g + ii;
        zw[ii] = sT[i * (kC + 1) + j];
    }
    // rank-update weights (scaled) on this lane's k-indices
    bf16x8 uwb[2];
    float uw[2][8];
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int i = 32 * u + (e < 4 ? 4 * g + e : 16 + 4 * g + e - 4);
            uw[u][e] = i < 16 * wave ? sT[i * (kC + 1) + jb] * ush : 0.0f;
            uwb[u][e] = (__bf16)uw[u][e];
        }
    const int nu = (16 * wave + 31) / 32;  // 32-token steps holding tokens < 16w

    // ---- B'_w as bf16 A-fragments: hf[mt][s] covers rows 16mt.., columns 32s..
    // The A operand of the rank update for rows 32s + 16h.. does not depend on mt: load once.
    bf16x8 ka[KS][2][2];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
        for (int hh = 0; hh < 2; ++hh)
#pragma unroll
            for (int u = 0; u < 2; ++u)
                if (u < nu) ka[ks][hh][u] = lds_frag(sKT + (32 * ks + 16 * hh + ln) * LDC + 32 * u + 4 * g);
    // Identity operands that copy an A-fragment of H_c, read as a B operand, into the two
    // 16x16 result tiles (rows 32s + {0..15} and 32s + {16..31}) it belongs to.
    bf16x8 id_lo, id_hi;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        id_lo[e] = (__bf16)(4 * g + e == ln ? 1.0f : 0.0f);
        id_lo[4 + e] = (__bf16)0.0f;
        id_hi[e] = (__bf16)0.0f;
        id_hi[4 + e] = (__bf16)(4 * g + e == ln ? 1.0f : 0.0f);
    }
    bf16x8 hf[MT][KS];
    f32x4 dg1[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
        bf16x8 bw[2];
        dg1[mt] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            if (u < nu) {
                const bf16x8 raw = lds_frag(sKT + (16 * mt + ln) * LDC + 32 * u + 4 * g);
#pragma unroll
                for (int e = 0; e < 8; ++e) bw[u][e] = (__bf16)((float)raw[e] * uw[u][e]);
                dg1[mt] = mfma16(lds_frag_sq(sKT + (16 * mt + ln) * LDC + 32 * u + 4 * g), uwb[u], dg1[mt]);
            }
        }
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            if (nu == 0) {
                hf[mt][ks] = hc[mt][ks];  // B_0 = H_c
                continue;
            }
            f32x4 lo = f32x4{0.0f, 0.0f, 0.0f, 0.0f}, hi = lo;
            if (keepH) {
                lo = mfma16(id_lo, hc[mt][ks], lo);
                hi = mfma16(id_hi, hc[mt][ks], hi);
            }
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                if (u < nu) {
                    lo = mfma16(ka[ks][0][u], bw[u], lo);
                    hi = mfma16(ka[ks][1][u], bw[u], hi);
                }
            }
            hf[mt][ks] = pack8(lo, hi);
        }
    }
    // B'_w is read only as the A operand of the state products.  Those accept the
    // accumulation registers directly, so keep it there: the loop's fp32 vectors
    // then have the ordinary vector registers to themselves.
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) asm volatile("" : "=a"(hf[mt][ks]) : "0"(hf[mt][ks]));
    // ---- the sub-chunk's keys as A-fragments: rows of S (kf2), columns of W (kf3)
    bf16x8 kf2[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) kf2[ks] = lds_frag(sK + (16 * wave + ln) * LDK + 32 * ks + 4 * g);
    // kf3: one 32-long contraction per row tile adds both remaining terms of the
    // product: its lower half holds the 16 sub-chunk tokens (K_w^T, met by S'),
    // its upper half diag(lambda) of the tile's rows (met by the tile's own rows
    // of the vector), so W += K_w^T S' + Lambda vec is one v_mfma_f32_16x16x32_bf16.
    bf16x8 kf3[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
        const uint2 kk = *reinterpret_cast<const uint2*>(sKT + (16 * mt + ln) * LDC + 16 * wave + 4 * g);
        kf3[mt] = __builtin_bit_cast(bf16x8, make_uint4(kk.x, kk.y, 0u, 0u));
        const float lrow = sLam[16 * mt + ln];
#pragma unroll
        for (int e = 0; e < 4; ++e) kf3[mt][4 + e] = (__bf16)(4 * g + e == ln ? lrow : 0.0f);
    }
    const f32x4 zero4 = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    const bf16x8 zwb = pack8(zw, zero4);

    // W = A_j vec for this wave's 16 columns (A_j = H_t + Lambda of token j):
    // W = zs_j (B'_w vec) + K_w^T S' + Lambda vec, the column scale applied to the
    // state products' accumulators.
    auto matvec = [&](const f32x4 (&vec)[MT], f32x4 (&w)[MT]) {
        bf16x8 pb[KS];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) pb[ks] = pack8(vec[2 * ks], vec[2 * ks + 1]);
        f32x4 sacc = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) sacc = mfma16(kf2[ks], pb[ks], sacc);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            w[mt] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) w[mt] = mfma16(hf[mt][ks], pb[ks], w[mt]);
        }
        const f32x4 sz = sacc * zw;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) w[mt] = mfma16(kf3[mt], pack8(sz, vec[mt]), zs * w[mt]);
    };

    // ---- Jacobi start x0 = q / diag(H_t + Lambda),
    //      diag(H_t) = zs_j diag(B'_w) + sum_{16w <= i <= j} beta_i Z[i][j] k_i^2
    f32x4 x[MT], r[MT], p[MT], w[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
        bf16x8 ksq = kf3[mt];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float v = (float)ksq[e];
            ksq[e] = (__bf16)(v * v);
        }
        const f32x4 dg2 = mfma16(ksq, zwb, f32x4{0.0f, 0.0f, 0.0f, 0.0f});
        const uint2 qq = *reinterpret_cast<const uint2*>(sQ + j * LDK + 16 * mt + 4 * g);
        const f32x4 qf{bf16_bits_to_f32(qq.x & 0xffffu), bf16_bits_to_f32(qq.x >> 16),
                       bf16_bits_to_f32(qq.y & 0xffffu), bf16_bits_to_f32(qq.y >> 16)};
        const f32x4 d = zs * ((keepH ? 1.0f : 0.0f) * hdiag[mt] + dg1[mt]) + dg2 + *reinterpret_cast<const f32x4*>(sLam + 16 * mt + 4 * g);
        x[mt] = qf / d;
        p[mt] = qf;  // holds q until the first residual is formed
    }
    matvec(x, w);
    float part = 0.0f;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
        r[mt] = p[mt] - w[mt];
        p[mt] = r[mt];
        part += r[mt][0] * r[mt][0] + r[mt][1] * r[mt][1] + r[mt][2] * r[mt][2] + r[mt][3] * r[mt][3];
    }
    float delta = col_sum(part);
    bool active = delta > 0.0f;

    for (int it = 0; it < a.n_cg; ++it) {
        if (!__any(active)) break;
        matvec(p, w);
        part = 0.0f;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
            part += p[mt][0] * w[mt][0] + p[mt][1] * w[mt][1] + p[mt][2] * w[mt][2] + p[mt][3] * w[mt][3];
        const float pw = col_sum(part);
        if (!(pw > 0.0f)) active = false;
        if (active) {
            const float alpha = delta / pw;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                x[mt] += alpha * p[mt];
                r[mt] -= alpha * w[mt];
            }
        }
        part = 0.0f;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
            part += r[mt][0] * r[mt][0] + r[mt][1] * r[mt][1] + r[mt][2] * r[mt][2] + r[mt][3] * r[mt][3];
        const float dn = col_sum(part);
        if (active) {
            if (dn == 0.0f) {
                active = false;
            } else {
                const float beta_cg = dn / delta;
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) p[mt] = r[mt] + beta_cg * p[mt];
                delta = dn;
            }
        }
    }

    // ---- read-out o_j = G_c (zeta_j x_j) + sum_i beta_i Z[i][j] v_i (k_i^T x_j)
    if (a.qstar && j < valid) {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
            *reinterpret_cast<f32x4*>(a.qstar + (tok0 + j) * DK + 16 * mt + 4 * g) = x[mt];
    }
    const float zeta = sZ0[j];
    f32x4 zo[4];  // beta_i Z[i][j] over the causal tiles it <= wave
#pragma unroll
    for (int it = 0; it < 4; ++it)
#pragma unroll
        for (int ii = 0; ii < 4; ++ii) {
            const int i = 16 * it + 4 * g + ii;
            zo[it][ii] = (it <= wave) ? sT[i * (kC + 1) + j] : 0.0f;
        }
    bf16x8 xb[KS], xz[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
        xb[ks] = pack8(x[2 * ks], x[2 * ks + 1]);
        xz[ks] = pack8(zeta * x[2 * ks], zeta * x[2 * ks + 1]);
    }
    f32x4 sacc[4];
#pragma unroll
    for (int it = 0; it < 4; ++it) {
        sacc[it] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
        if (it <= wave) {
#pragma unroll
            for (int ks = 0; ks < KS; ++ks)
                sacc[it] = mfma16(lds_frag(sK + (16 * it + ln) * LDK + 32 * ks + 4 * g), xb[ks], sacc[it]);
        }
    }
    f32x4 o[MTV];
#pragma unroll
    for (int mt = 0; mt < MTV; ++mt) {
        o[mt] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
            o[mt] = mfma16(__builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(Gf + ((mt * KS + ks) * 64 + lane) * 8)),
                           xz[ks], o[mt]);
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        if (2 * u <= wave) {
            const bf16x8 sb = pack8(sacc[2 * u] * zo[2 * u], sacc[2 * u + 1] * zo[2 * u + 1]);
#pragma unroll
            for (int mt = 0; mt < MTV; ++mt)
                o[mt] = mfma16(lds_frag(sVT + (16 * mt + ln) * LDC + 32 * u + 4 * g), sb, o[mt]);
        }
    }
    if (j < valid) {
#pragma unroll
        for (int mt = 0; mt < MTV; ++mt)
            *reinterpret_cast<f32x4*>(a.out + (tok0 + j) * DV + 16 * mt + 4 * g) = o[mt];
    }
}

template <int DK, int DV>
hipError_t launch_shape(const CgArgs& a, hipStream_t stream)
{
    const unsigned blocks = unsigned(a.s.batch * a.s.heads * a.s.n_chunks);
    hipLaunchKernelGGL((chunk_cg_bf16_kernel<DK, DV>), dim3(blocks), dim3(kThreads), 0, stream, a);
    return hipGetLastError();
}

}  // namespace

bool chunk_cg_bf16_supported(const ForwardShape& s)
{
    return s.bf16 && s.chunk == kC && (s.d_k == 64 || s.d_k == 128) && (s.d_v == 64 || s.d_v == 128);
}

hipError_t launch_chunk_cg_bf16(const CgArgs& a, hipStream_t stream)
{
    if (!chunk_cg_bf16_supported(a.s)) return hipErrorInvalidValue;
    if (a.s.d_k == 64) return a.s.d_v == 64 ? launch_shape<64, 64>(a, stream) : launch_shape<64, 128>(a, stream);
    return a.s.d_v == 64 ? launch_shape<128, 64>(a, stream) : launch_shape<128, 128>(a, stream);
}

}  // namespace mesa
