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
// Work split: a workgroup is one chunk, each of its four waves owns 16 tokens
// (columns j = 16w .. 16w+15) over all d_k features and runs its own CG with
// no barrier.  Every per-token vector (x, r, p, w) lives in registers in the
// layout of a v_mfma_f32_16x16x32_bf16 result: lane (g = lane/16, n = lane%16)
// holds rows 16t + 4g + {0..3} of column n for each 16-row tile t.  The
// 32-long contraction of one MFMA consumes two such tiles: k-index
// e in 0..7 of lane group g stands for row 32s + 4g + e (e < 4) or
// 32s + 16 + 4g + (e - 4) (e >= 4).  The A operands (H_c, the keys) are laid
// out with the same index map, so a CG vector feeds the next product straight
// from its accumulator registers, with no LDS round trip.
//
// Per CG product and wave: H_c (zeta p) as d_k/16 x d_k/32 MFMAs with H_c held
// as bf16 A-fragments in registers for the whole solve; S = K_c p over the
// causal token tiles 0..w only; S' = beta Z ⊙ S in fp32; W += K_c^T S' over the
// same tiles.  CG scalars reduce over the 4 lanes of a column with two
// cross-lane shuffles.  Only the MFMA operands are bf16; x, r, p, w, alpha,
// beta and every reduction stay fp32.
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

// Sum over the four lanes that hold one column (lanes n, n+16, n+32, n+48).
__device__ __forceinline__ float col_sum(float v)
{
    v += __shfl_xor(v, 16, kWave);
    v += __shfl_xor(v, 32, kWave);
    return v;
}

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

    // ---- stage the chunk's keys, values and queries (bf16 bits) in LDS
    const uint16_t* kp = static_cast<const uint16_t*>(a.k);
    const uint16_t* qp = static_cast<const uint16_t*>(a.q);
    const uint16_t* vp = static_cast<const uint16_t*>(a.v);
    for (int e = tid; e < kC * DK / 8; e += kThreads) {
        const int i = e / (DK / 8), c8 = (e % (DK / 8)) * 8;
        uint4 kv = make_uint4(0, 0, 0, 0), qv = make_uint4(0, 0, 0, 0);
        if (i < valid) {
            kv = *reinterpret_cast<const uint4*>(kp + (tok0 + i) * DK + c8);
            qv = *reinterpret_cast<const uint4*>(qp + (tok0 + i) * DK + c8);
        }
        *reinterpret_cast<uint4*>(sK + i * LDK + c8) = kv;
        *reinterpret_cast<uint4*>(sQ + i * LDK + c8) = qv;
        const uint32_t w4[4] = {kv.x, kv.y, kv.z, kv.w};
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            sKT[(c8 + 2 * u) * LDC + i] = uint16_t(w4[u] & 0xffffu);
            sKT[(c8 + 2 * u + 1) * LDC + i] = uint16_t(w4[u] >> 16);
        }
    }
    for (int e = tid; e < kC * DV / 8; e += kThreads) {
        const int i = e / (DV / 8), c8 = (e % (DV / 8)) * 8;
        uint4 vv = make_uint4(0, 0, 0, 0);
        if (i < valid) vv = *reinterpret_cast<const uint4*>(vp + (tok0 + i) * DV + c8);
        const uint32_t w4[4] = {vv.x, vv.y, vv.z, vv.w};
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            sVT[(c8 + 2 * u) * LDC + i] = uint16_t(w4[u] & 0xffffu);
            sVT[(c8 + 2 * u + 1) * LDC + i] = uint16_t(w4[u] >> 16);
        }
    }
    if (tid < kWave) {
        chunk_log_decays(a.gamma + tok0, valid, sLg, sZl);
        sBeta[tid] = tid < valid ? a.beta[tok0 + tid] : 0.0f;
    }

    // ---- per-lane constants: H_c fragments, Lambda, decays
    const float* Hc = a.Hs + (bh * s.n_chunks + n) * int64_t(DK) * DK;
    bf16x8 hf[MT][KS];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) hf[mt][ks] = gmem_frag(Hc + (16 * mt + ln) * DK + 32 * ks + 4 * g);
    const float* lam = a.lambda + int64_t(h) * DK;
    f32x4 lamv[MT], hdiag[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
        lamv[mt] = *reinterpret_cast<const f32x4*>(lam + 16 * mt + 4 * g);
#pragma unroll
        for (int ii = 0; ii < 4; ++ii) {
            const int r = 16 * mt + 4 * g + ii;
            hdiag[mt][ii] = Hc[r * DK + r];
        }
    }
    __syncthreads();

    const float zeta = decay_from_start(sLg, sZl, j);
    // beta_i Z[i][j] for the rows i = 16 it + 4g + ii this lane meets in S (tiles it <= wave)
    f32x4 zw[4];
#pragma unroll
    for (int it = 0; it < 4; ++it)
#pragma unroll
        for (int ii = 0; ii < 4; ++ii) {
            const int i = 16 * it + 4 * g + ii;
            zw[it][ii] = (it <= wave) ? sBeta[i] * decay_between(sLg, sZl, i, j) : 0.0f;
        }
    bf16x8 zwb[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) zwb[u] = pack8(zw[2 * u], zw[2 * u + 1]);

    // W = A_j vec for this wave's 16 columns (A_j = H_t + Lambda of token j).
    auto matvec = [&](const f32x4 (&vec)[MT], f32x4 (&w)[MT]) {
        bf16x8 pb[KS], pz[KS];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            pb[ks] = pack8(vec[2 * ks], vec[2 * ks + 1]);
            pz[ks] = pack8(zeta * vec[2 * ks], zeta * vec[2 * ks + 1]);
        }
        f32x4 sacc[4];
#pragma unroll
        for (int it = 0; it < 4; ++it) {
            sacc[it] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
            if (it <= wave) {
#pragma unroll
                for (int ks = 0; ks < KS; ++ks)
                    sacc[it] = mfma16(lds_frag(sK + (16 * it + ln) * LDK + 32 * ks + 4 * g), pb[ks], sacc[it]);
            }
        }
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            w[mt] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) w[mt] = mfma16(hf[mt][ks], pz[ks], w[mt]);
        }
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            if (2 * u <= wave) {
                const bf16x8 sb = pack8(sacc[2 * u] * zw[2 * u], sacc[2 * u + 1] * zw[2 * u + 1]);
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
                    w[mt] = mfma16(lds_frag(sKT + (16 * mt + ln) * LDC + 32 * u + 4 * g), sb, w[mt]);
            }
        }
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) w[mt] += lamv[mt] * vec[mt];
    };

    // ---- Jacobi start x0 = q / diag(H_t + Lambda)
    f32x4 x[MT], r[MT], p[MT], w[MT];
    {
        f32x4 dg[MT];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) dg[mt] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            if (2 * u <= wave) {
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
                    dg[mt] = mfma16(lds_frag_sq(sKT + (16 * mt + ln) * LDC + 32 * u + 4 * g), zwb[u], dg[mt]);
            }
        }
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            const uint2 qq = *reinterpret_cast<const uint2*>(sQ + j * LDK + 16 * mt + 4 * g);
            const f32x4 qf{__uint_as_float(qq.x << 16), __uint_as_float(qq.x & 0xffff0000u),
                           __uint_as_float(qq.y << 16), __uint_as_float(qq.y & 0xffff0000u)};
            const f32x4 d = zeta * hdiag[mt] + dg[mt] + lamv[mt];
            x[mt] = qf / d;
            p[mt] = qf;  // holds q until the first residual is formed
        }
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
        const float alpha = active ? delta / pw : 0.0f;
        part = 0.0f;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            if (active) {
                x[mt] += alpha * p[mt];
                r[mt] -= alpha * w[mt];
            }
            part += r[mt][0] * r[mt][0] + r[mt][1] * r[mt][1] + r[mt][2] * r[mt][2] + r[mt][3] * r[mt][3];
        }
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
    const float* Gc = a.Gs + (bh * s.n_chunks + n) * int64_t(DV) * DK;
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
            o[mt] = mfma16(gmem_frag(Gc + (16 * mt + ln) * DK + 32 * ks + 4 * g), xz[ks], o[mt]);
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        if (2 * u <= wave) {
            const bf16x8 sb = pack8(sacc[2 * u] * zw[2 * u], sacc[2 * u + 1] * zw[2 * u + 1]);
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
