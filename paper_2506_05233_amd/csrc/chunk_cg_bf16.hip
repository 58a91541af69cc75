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

// Gate decay with the hardware exponential (relative error ~1e-7, far below
// the bf16 operand rounding of this path); same zero-gate rule as the shared
// helper.
__device__ __forceinline__ float decay_between_hw(const float* lg, const int* zl, int i, int j)
{
    if (i > j || zl[j] > i) return 0.0f;
    return __expf(lg[j] - lg[i]);
}


// v if c, else zero (per component, so the operands stay in registers)
__device__ __forceinline__ uint4 keep_if(bool c, const uint4& v)
{
    return make_uint4(c ? v.x : 0u, c ? v.y : 0u, c ? v.z : 0u, c ? v.w : 0u);
}

// Decays below this are treated as zero where a chunk-relative weight would need
// their reciprocal (see the sub-chunk states below).
constexpr float kMinDecay = 1e-20f;

// 8 bf16 (bits in v) times u, rounded back to bf16.
__device__ __forceinline__ uint4 scale_bf16x8(const uint4& v, float u)
{
    const bf16x8 x = __builtin_bit_cast(bf16x8, v);
    bf16x8 y;
#pragma unroll
    for (int e = 0; e < 8; ++e) y[e] = (__bf16)((float)x[e] * u);
    return __builtin_bit_cast(uint4, y);
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
    // the grid has fewer than 2^31 blocks (checked at launch): 32-bit index arithmetic
    const int n = int(blockIdx.x % unsigned(s.n_chunks));
    const int64_t bh = blockIdx.x / unsigned(s.n_chunks);
    const int h = int(unsigned(bh) % unsigned(s.heads));
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
    __shared__ __attribute__((aligned(16))) uint16_t sHf[DK * DK];   // H_c as A-fragments
    __shared__ __attribute__((aligned(16))) uint16_t sGf[DV * DK];   // G_c as A-fragments
    __shared__ __attribute__((aligned(16))) uint16_t sKU[DK * LDC];  // u_i k_i[b], feature-major
    __shared__ float sLg[kWave], sBeta[kWave];
    __shared__ int sZl[kWave];
    __shared__ __attribute__((aligned(16))) float sLam[DK];
    __shared__ float sZ0[kC];            // zeta_{c+j,c}: decay from the chunk's entering state
    __shared__ __attribute__((aligned(16))) float sDiag[kThreads / kWave][DK + kWave];  // diag(B'_w) per wave, spare slots

    // ---- stage the chunk's keys, values and queries (bf16 bits) in LDS
    const uint16_t* kp = static_cast<const uint16_t*>(a.k);
    const uint16_t* qp = static_cast<const uint16_t*>(a.q);
    const uint16_t* vp = static_cast<const uint16_t*>(a.v);
    // Every global load of the chunk is issued before the first use of any of them,
    // gates first (the first ones needed; vector memory returns in order).  Loads
    // never sit behind a branch: tokens past the end of the sequence read the last
    // valid token (valid >= 1) and are zeroed once the data is in registers.
    const int lt = min(lane, valid - 1);
    const float g_raw = a.gamma[tok0 + lt];
    const float b_raw = a.beta[tok0 + lt];
    // thread t stages tokens 2p, 2p+1 (p = t % 32) for 8 features per pass
    constexpr int NKQ = DK / 64;  // passes over the key features (8 groups of 8 per pass)
    constexpr int NV = DV / 64;
    const int p2 = tid % 32, fg = tid / 32;
    const int i0 = 2 * p2, i1 = 2 * p2 + 1;
    const int64_t r0 = tok0 + min(i0, valid - 1), r1 = tok0 + min(i1, valid - 1);
    uint4 kv[NKQ][2], qv[NKQ][2], vv[NV][2];
#pragma unroll
    for (int m = 0; m < NKQ; ++m) {
        const int f0 = 64 * m + 8 * fg;
        kv[m][0] = *reinterpret_cast<const uint4*>(kp + r0 * DK + f0);
        qv[m][0] = *reinterpret_cast<const uint4*>(qp + r0 * DK + f0);
        kv[m][1] = *reinterpret_cast<const uint4*>(kp + r1 * DK + f0);
        qv[m][1] = *reinterpret_cast<const uint4*>(qp + r1 * DK + f0);
    }
#pragma unroll
    for (int m = 0; m < NV; ++m) {
        const int f0 = 64 * m + 8 * fg;
        vv[m][0] = *reinterpret_cast<const uint4*>(vp + r0 * DV + f0);
        vv[m][1] = *reinterpret_cast<const uint4*>(vp + r1 * DV + f0);
    }
    // Chunk states as bf16 A-fragments, fragment f of lane l at [f * 64 + l] * 8: one
    // fragment is 1 KiB, so each is one direct global -> LDS load of the whole wave
    // (lane l's 16 bytes land at byte 16 l of the fragment).  Every wave needs all of
    // H_c and G_c; they cross the vector caches once per workgroup this way.  H_c is
    // needed first; G_c only by the read-out, so its loads go out after the barrier.
    const uint16_t* Hf = static_cast<const uint16_t*>(a.Hs) + (bh * s.n_chunks + n) * int64_t(DK) * DK;
    const uint16_t* Gf = static_cast<const uint16_t*>(a.Gs) + (bh * s.n_chunks + n) * int64_t(DV) * DK;
    constexpr int NHF = DK * DK / (8 * kWave) / 4;  // H_c fragments per wave
    constexpr int NGF = DV * DK / (8 * kWave) / 4;  // G_c fragments per wave
#pragma unroll
    for (int u = 0; u < NHF; ++u) {
        const int f = wave * NHF + u;
        load_lds16(Hf + (f * kWave + lane) * 8, sHf + f * kWave * 8);
    }
    // gates and write strengths of the chunk, one token per lane, in every wave;
    // absent tokens have gate 1 and strength 0
    const float gl = lane < valid ? g_raw : 1.0f;
    const float bl = lane < valid ? b_raw : 0.0f;
    if (valid < kC) {
        const bool k0 = i0 < valid, k1 = i1 < valid;
#pragma unroll
        for (int m = 0; m < NKQ; ++m) {
            kv[m][0] = keep_if(k0, kv[m][0]);
            qv[m][0] = keep_if(k0, qv[m][0]);
            kv[m][1] = keep_if(k1, kv[m][1]);
            qv[m][1] = keep_if(k1, qv[m][1]);
        }
#pragma unroll
        for (int m = 0; m < NV; ++m) {
            vv[m][0] = keep_if(k0, vv[m][0]);
            vv[m][1] = keep_if(k1, vv[m][1]);
        }
    }
    const float* lam = a.lambda + int64_t(h) * DK;
    if (tid < DK) sLam[tid] = lam[tid];
    // Gate log-cumsums of the chunk in registers (lane = token; the same rules as
    // chunk_log_decays: a zero gate resets memory through zl instead of log 0).
    const float lgl = wave_scan_add(gl > 0.0f ? logf(gl) : 0.0f);
    const int zll = wave_scan_max((lane < valid && !(gl > 0.0f)) ? lane : -1);
    const float zeta_l = zll >= 0 ? 0.0f : __expf(lgl);  // zeta_{c+l,c}
    if (wave == 0) {
        sLg[lane] = lgl;
        sZl[lane] = zll;
        sZ0[lane] = zeta_l;
        sBeta[lane] = bl;
    }
    // Rank-update weight of token i relative to the chunk's entering state,
    // u_i = beta_i / zeta_{c+i,c}; 0 where zeta_{c+i,c} <= kMinDecay (those tokens
    // only enter sub-chunk states built without H_c, below).
    const float u_l = zeta_l > kMinDecay ? bl * __expf(-lgl) : 0.0f;
    const float u0 = __shfl(u_l, i0), u1 = __shfl(u_l, i1);
#pragma unroll
    for (int m = 0; m < NKQ; ++m) {
        const int f0 = 64 * m + 8 * fg;
        *reinterpret_cast<uint4*>(sK + i0 * LDK + f0) = kv[m][0];
        *reinterpret_cast<uint4*>(sK + i1 * LDK + f0) = kv[m][1];
        *reinterpret_cast<uint4*>(sQ + i0 * LDK + f0) = qv[m][0];
        *reinterpret_cast<uint4*>(sQ + i1 * LDK + f0) = qv[m][1];
        stage_token_pair(reinterpret_cast<uint32_t*>(sKT), LDC / 2, f0, p2, kv[m][0], kv[m][1]);
        stage_token_pair(reinterpret_cast<uint32_t*>(sKU), LDC / 2, f0, p2, scale_bf16x8(kv[m][0], u0),
                         scale_bf16x8(kv[m][1], u1));
    }
#pragma unroll
    for (int m = 0; m < NV; ++m)
        stage_token_pair(reinterpret_cast<uint32_t*>(sVT), LDC / 2, 64 * m + 8 * fg, p2, vv[m][0], vv[m][1]);
    // this wave's H_c fragments have landed in LDS; the barrier publishes them
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
    __syncthreads();
#pragma unroll
    for (int u = 0; u < NGF; ++u) {
        const int f = wave * NGF + u;
        load_lds16(Gf + (f * kWave + lane) * 8, sGf + f * kWave * 8);
    }
    bf16x8 hc[MT][KS];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
            hc[mt][ks] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(sHf + ((mt * KS + ks) * kWave + lane) * 8));

    // ---- decays of this sub-chunk
    const int jb = 16 * wave - 1;  // token whose state enters the sub-chunk (-1: the chunk's H_c)
    const float Dw = wave == 0 ? 1.0f : sZ0[jb];
    // B_w = Dw H_c + sum_{i<16w} beta_i zeta_{16w-1,i} k_i k_i^T.  It is kept as
    // B'_w = B_w / Dw = H_c + sum_{i<16w} u_i k_i k_i^T (u_i = beta_i / zeta_{c+i,c}, the
    // staged sKU) and the 1/Dw goes into the column scale: zs_j = zt_j Dw = zeta_{c+j,c}.
    // When Dw is negligible (<= kMinDecay, e.g. after a zero gate) the state term Dw H_c
    // is dropped instead: B_w = sum_{i<16w} beta_i zeta_{16w-1,i} k_i k_i^T and zs_j = zt_j.
    const bool keepH = wave == 0 || Dw > kMinDecay;
    const float zs = keepH ? sZ0[j] : decay_between_hw(sLg, sZl, jb, j);
    f32x4 zw;  // beta_i Z[i][j] for the sub-chunk rows i = 16w + 4g + ii met in S
#pragma unroll
    for (int ii = 0; ii < 4; ++ii) {
        const int i = 16 * wave + 4 * g + ii;
        zw[ii] = sBeta[i] * decay_between_hw(sLg, sZl, i, j);
    }

    // ---- B'_w as bf16 A-fragments: hf[mt][s] covers rows 16mt.., columns 32s..
    // Every wave runs the same straight-line code: both 32-token steps of the rank update,
    // with the tokens i >= 16w zeroed in its A operand (rows 32s + 16h.., independent of mt,
    // loaded once).  Element e of step u is token 32u + 4g + e (e < 4) or 32u + 16 + 4g + e - 4,
    // so whole halves are in or out: the lower half of step u iff 32u + 16 <= 16w, the upper
    // half iff 32u + 32 <= 16w.
    bf16x8 ka[KS][2][2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        const bool in_lo = 32 * u + 16 <= 16 * wave, in_hi = 32 * u + 32 <= 16 * wave;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
#pragma unroll
            for (int hh = 0; hh < 2; ++hh) {
                const uint4 raw = __builtin_bit_cast(uint4, lds_frag(sKT + (32 * ks + 16 * hh + ln) * LDC + 32 * u + 4 * g));
                ka[ks][hh][u] = __builtin_bit_cast(bf16x8, make_uint4(in_lo ? raw.x : 0u, in_lo ? raw.y : 0u,
                                                                      in_hi ? raw.z : 0u, in_hi ? raw.w : 0u));
            }
    }
    // Without H_c the weights are per sub-chunk: beta_i zeta_{16w-1,i} on this lane's k-indices.
    float uw[2][8];
    if (!keepH) {
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int i = 32 * u + (e < 4 ? 4 * g + e : 16 + 4 * g + e - 4);
                uw[u][e] = i < 16 * wave ? sBeta[i] * decay_between_hw(sLg, sZl, i, jb) : 0.0f;
            }
    }
    // Identity operands that copy an A-fragment of H_c, read as a B operand, into the two
    // 16x16 result tiles (rows 32s + {0..15} and 32s + {16..31}) it belongs to; zero when
    // the state term is dropped.
    bf16x8 id_lo, id_hi;
    const float one = keepH ? 1.0f : 0.0f;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        id_lo[e] = (__bf16)(4 * g + e == ln ? one : 0.0f);
        id_lo[4 + e] = (__bf16)0.0f;
        id_hi[e] = (__bf16)0.0f;
        id_hi[4 + e] = (__bf16)(4 * g + e == ln ? one : 0.0f);
    }
    // diag(B'_w) goes to sDiag[wave][r]; lanes off the diagonal write a spare slot instead
    const int e_diag = ln - 4 * g;
    const bool on_diag = e_diag >= 0 && e_diag < 4;
    bf16x8 hf[MT][KS];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
        bf16x8 bw[2];
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            if (keepH) {
                bw[u] = lds_frag(sKU + (16 * mt + ln) * LDC + 32 * u + 4 * g);
            } else {
                const bf16x8 raw = lds_frag(sKT + (16 * mt + ln) * LDC + 32 * u + 4 * g);
#pragma unroll
                for (int e = 0; e < 8; ++e) bw[u][e] = (__bf16)((float)raw[e] * uw[u][e]);
            }
        }
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            f32x4 lo = mfma16(id_lo, hc[mt][ks], f32x4{0.0f, 0.0f, 0.0f, 0.0f});
            f32x4 hi = mfma16(id_hi, hc[mt][ks], f32x4{0.0f, 0.0f, 0.0f, 0.0f});
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                lo = mfma16(ka[ks][0][u], bw[u], lo);
                hi = mfma16(ka[ks][1][u], bw[u], hi);
            }
            hf[mt][ks] = pack8(lo, hi);
            // Tile rows 16mt.. of fragment (mt, mt/2) hold the diagonal block: lane (g, n)
            // has B'[16mt + 4g + e][16mt + n], on the diagonal for n = 4g + e.
            if (ks == mt / 2) {
                const f32x4 acc = (mt % 2) ? hi : lo;
                const float dv = e_diag == 0 ? acc[0] : e_diag == 1 ? acc[1] : e_diag == 2 ? acc[2] : acc[3];
                sDiag[wave][on_diag ? 16 * mt + ln : DK + lane] = dv;
            }
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
    //      diag(H_t) = zs_j diag(B'_w) + sum_{16w <= i <= j} beta_i Z[i][j] k_i^2, diag(B'_w)
    //      read back from this wave's sDiag rows (written by other lanes of the same wave;
    //      a wave's LDS accesses complete in order)
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
        const f32x4 d = zs * *reinterpret_cast<const f32x4*>(&sDiag[wave][16 * mt + 4 * g]) + dg2 +
                        *reinterpret_cast<const f32x4*>(sLam + 16 * mt + 4 * g);
#pragma unroll
        for (int e = 0; e < 4; ++e) x[mt][e] = qf[e] * __builtin_amdgcn_rcpf(d[e]);
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
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);  // this wave's G_c fragments have landed
    __syncthreads();
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
            zo[it][ii] = (it <= wave) ? sBeta[i] * decay_between_hw(sLg, sZl, i, j) : 0.0f;
        }
    bf16x8 xb[KS], xz[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
        xb[ks] = pack8(x[2 * ks], x[2 * ks + 1]);
        xz[ks] = pack8(zeta * x[2 * ks], zeta * x[2 * ks + 1]);
    }
    // every wave runs all four token tiles (zo is zero past the causal ones)
    f32x4 sacc[4];
#pragma unroll
    for (int it = 0; it < 4; ++it) {
        sacc[it] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
            sacc[it] = mfma16(lds_frag(sK + (16 * it + ln) * LDK + 32 * ks + 4 * g), xb[ks], sacc[it]);
    }
    f32x4 o[MTV];
#pragma unroll
    for (int mt = 0; mt < MTV; ++mt) {
        o[mt] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
            o[mt] = mfma16(__builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(sGf + ((mt * KS + ks) * kWave + lane) * 8)),
                           xz[ks], o[mt]);
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        const bf16x8 sb = pack8(sacc[2 * u] * zo[2 * u], sacc[2 * u + 1] * zo[2 * u + 1]);
#pragma unroll
        for (int mt = 0; mt < MTV; ++mt)
            o[mt] = mfma16(lds_frag(sVT + (16 * mt + ln) * LDC + 32 * u + 4 * g), sb, o[mt]);
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
