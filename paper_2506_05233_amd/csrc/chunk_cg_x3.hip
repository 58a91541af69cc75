// Chunked conjugate gradients + read-out on the gfx950 matrix cores with split
// operands (MESA_PREC_BF16X3), for bf16 q, k, v and chunk C = 64.
//
// The mathematics and the work split are those of the single-pass kernel
// (chunk_cg_bf16.hip; App. C, Alg. 1 with its relative tolerance; App. D,
// Eq. q_star_parallel and Eq. gla): wave w of a workgroup owns the 16-token
// sub-chunk j = 16w .. 16w+15 of the chunk, forms the state entering it,
//
//   B'_w = H_c + sum_{i < 16w} u_i k_i k_i^T,    u_i = beta_i / zeta_{c+i,c},
//
// and runs its own CG with every product
//
//   (H_t + Lambda) p_j = zeta_{c+j,c} (B'_w p_j) + sum_{16w <= i <= j} beta_i Z[i][j] k_i (k_i^T p_j) + Lambda p_j.
//
// What differs is the arithmetic of the products.  The paper keeps the solver's
// matrix products in fp32 (App. G.5) and warns that lower precision may keep CG
// from converging; on repeated keys with gates near one a single bf16 rounding of
// the state and of the direction costs ~1e-1 relative error.  Here every fp32
// operand x of a matrix-core product is carried as two bf16 numbers,
// x = hi + lo with hi = bf16(x) and lo = bf16(x - hi) (16 significant bits), and a
// product a b is formed as hi_a hi_b + hi_a lo_b + lo_a hi_b with fp32
// accumulation (three v_mfma_f32_16x16x32_bf16 passes): each product term then
// carries ~2^-16 relative error instead of ~2^-8.  The keys are exact in bf16,
// so their products need only the other operand's two parts; the k^2 and gate
// weights of the Jacobi diagonal are split the same way; Lambda p is an fp32
// multiply-add.  x, r, p, w, alpha, beta and every reduction are fp32.
//
// Data: the chunk states come from the scan as fp32 H_c in matrix-core fragment
// order (fragment f = 16-row tile mt x 32-column step ks; half e of lane l at
// [(2 f + e) 64 + l] x 4 floats) and G_c as bf16 high and low planes of the
// fragment layout.  The state build reads H_c straight from global memory into its
// accumulators, one row tile ahead (H and B'_w are symmetric, so a fragment's two
// halves are the two 16x16 result tiles it belongs to; the previous chunk's CG loop
// has requested H_c into the L2 cache), adds the rank update, and stores B'_w's
// high and low parts as matrix-core operands in the accumulation registers (256 of
// them at d_k = 128), where the state products read them.  G_c reaches LDS by
// direct global -> LDS loads issued under the chunk's own CG loop, for the
// read-out.  q is read from global memory at the Jacobi start.
#include "mesa_device.hpp"
#include "mesa_kernels.hpp"
#include "mesa_mfma.hpp"

namespace mesa {
namespace {

constexpr int kC = 64;         // chunk
constexpr int kThreads = 256;  // four waves, 16 tokens each

// Decays below this are treated as zero where a chunk-relative weight would need
// their reciprocal (the sub-chunk states are then built without H_c).
constexpr float kMinDecay = 1e-20f;

// Four values as one 8-wide operand: elements 0..3 their high parts, 4..7 their low
// parts.  Against an operand that repeats its four k-values in both halves, one
// product sums hi + lo.
__device__ __forceinline__ bf16x8 split4_stacked(const f32x4& a)
{
    uint32_t h0, l0, h1, l1;
    split2(a[0], a[1], h0, l0);
    split2(a[2], a[3], h1, l1);
    return __builtin_bit_cast(bf16x8, make_uint4(h0, h1, l0, l1));
}

// 8 bf16 (bits in v) times u, split into high and low bf16 parts.
__device__ __forceinline__ void scale_split8(const uint4& v, float u, uint4& hi, uint4& lo)
{
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
    uint32_t h[4], l[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) split2(__uint_as_float(w[q] << 16) * u, __uint_as_float(w[q] & 0xffff0000u) * u, h[q], l[q]);
    hi = make_uint4(h[0], h[1], h[2], h[3]);
    lo = make_uint4(l[0], l[1], l[2], l[3]);
}

// beta_i prod_{s=i+1..j} gamma_s for the four tokens i = i4 .. i4+3 (i4 a multiple of 4)
// and token j from the chunk's gate log-cumsums: 0 for i > j or when a zero gate lies
// in (i, j] (zl_j > i).  lgj = lg[j], zlj = zl[j].
__device__ __forceinline__ f32x4 decay_weights4(const float* lg, const float* beta, float lgj, int zlj, int i4, int j)
{
    const f32x4 lgi = *reinterpret_cast<const f32x4*>(lg + i4);
    const f32x4 bi = *reinterpret_cast<const f32x4*>(beta + i4);
    f32x4 r;
#pragma unroll
    for (int e = 0; e < 4; ++e) r[e] = (i4 + e <= j && zlj <= i4 + e) ? bi[e] * __expf(lgj - lgi[e]) : 0.0f;
    return r;
}

__device__ __forceinline__ float decay_between_hw(const float* lg, const int* zl, int i, int j)
{
    if (i > j || zl[j] > i) return 0.0f;
    return __expf(lg[j] - lg[i]);
}

__device__ __forceinline__ uint4 keep_if(bool c, const uint4& v)
{
    return make_uint4(c ? v.x : 0u, c ? v.y : 0u, c ? v.z : 0u, c ? v.w : 0u);
}

// Sum over the four lanes that hold one column (lanes n, n+16, n+32, n+48).
__device__ __forceinline__ float col_sum(float v) { return row_pair_sums(v); }

// LDS arena (byte offsets).  G_c lands in its own region under the chunk's CG loop;
// the next chunk's keys and values land on the key tiles (sKT, sKUh, sKUl), which
// only the state build and the operand set-up before CG read.
template <int DK, int DV>
struct CgX3Smem {
    // Row strides (bf16 elements) of the token-major and feature-major tiles.  A fragment
    // read (two 8-byte LDS reads per lane) is served 16 lanes at a time from 32 four-byte
    // banks; rows 2 banks apart (a stride of 2 mod 32 words) give its 16 rows distinct bank
    // pairs, where rows 4 apart (+8 elements) made every such read take twice its cycles.
    // The rows are then 8-byte aligned only, so 16-byte stores into them are split.
    static constexpr int LDK = DK + 4;
    static constexpr int LDC = kC + 4;
    static constexpr int NKQ = DK / 64;  // staging passes over the key features
    static constexpr int NV = DV / 64;
    static constexpr int kRawSlots = 2 * (NKQ + NV);
    static constexpr int oK = 0;                              // k_i[b], token-major bf16
    static constexpr int oVT = oK + kC * LDK * 2;             // v_i[e], feature-major bf16
    static constexpr int oLg = oVT + DV * LDC * 2;            // gate log-cumsums
    static constexpr int oBeta = oLg + kWave * 4;
    static constexpr int oZl = oBeta + kWave * 4;             // last zero gate
    static constexpr int oZ0 = oZl + kWave * 4;               // zeta_{c+j,c}
    static constexpr int oGc = oZ0 + kC * 4;                  // G_c, bf16 high then low fragments
    static constexpr int oKT = oGc + DV * DK * 4;             // k_i[b], feature-major
    static constexpr int oKUh = oKT + DK * LDC * 2;           // hi(u_i k_i[b]), feature-major
    static constexpr int oKUl = oKUh + DK * LDC * 2;          // lo(u_i k_i[b])
    static constexpr int oSink = oKUl + DK * LDC * 2;         // landing slot of the L2 requests for H_c
    static constexpr int oDiag = oSink + kWave * 16;          // diag(B'_w) per wave, spare slots
    static constexpr int oRaw = oKT;                          // next chunk's staging slots
    static constexpr int kEnd = oDiag + (kThreads / kWave) * (DK + kWave) * 4;
    static constexpr int kRawEnd = oRaw + kRawSlots * kThreads * 16;
    static constexpr int kBytes = kEnd;
    static_assert(kRawEnd <= oSink, "staging slots run past the key tiles");
    static_assert(oGc % 16 == 0 && oKT % 16 == 0 && oSink % 16 == 0, "misaligned LDS region");
    static_assert(kBytes <= 160 * 1024, "LDS use exceeds 160 KiB");
};

template <int DK, int DV, bool READOUT>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
void chunk_cg_x3_kernel(CgArgs a, int total)
{
    using L = CgX3Smem<DK, DV>;
    constexpr int MT = DK / 16;    // 16-row tiles of a per-token vector
    constexpr int KS = DK / 32;    // 32-long contraction steps over features
    constexpr int MTV = DV / 16;   // 16-row tiles of an output column
    constexpr int LDK = L::LDK, LDC = L::LDC, NKQ = L::NKQ, NV = L::NV;
    constexpr int kWaves = kThreads / kWave;
    constexpr int kHcReq = DK * DK * 4 / 1024 / kWaves;  // 1-KiB L2 requests for H_c per wave
    constexpr int kGLoads = DV * DK * 4 / 1024 / kWaves;  // 1-KiB G_c loads (high + low) per wave

    __shared__ __attribute__((aligned(16))) unsigned char smem[L::kBytes];
    // Lambda, read in every CG product, has an array of its own: the compiler can then
    // tell its reads apart from the direct loads into smem that run under the CG loop
    // and does not order them behind those loads.
    __shared__ __attribute__((aligned(16))) float sLam[DK];
    uint16_t* sK = reinterpret_cast<uint16_t*>(smem + L::oK);
    uint16_t* sVT = reinterpret_cast<uint16_t*>(smem + L::oVT);
    float* sLg = reinterpret_cast<float*>(smem + L::oLg);
    float* sBeta = reinterpret_cast<float*>(smem + L::oBeta);
    int* sZl = reinterpret_cast<int*>(smem + L::oZl);
    float* sZ0 = reinterpret_cast<float*>(smem + L::oZ0);
    uint16_t* sGc = reinterpret_cast<uint16_t*>(smem + L::oGc);
    uint16_t* sKT = reinterpret_cast<uint16_t*>(smem + L::oKT);
    uint16_t* sKUh = reinterpret_cast<uint16_t*>(smem + L::oKUh);
    uint16_t* sKUl = reinterpret_cast<uint16_t*>(smem + L::oKUl);
    unsigned char* sSink = smem + L::oSink;
    float* sDiag = reinterpret_cast<float*>(smem + L::oDiag);
    uint4* sRaw = reinterpret_cast<uint4*>(smem + L::oRaw);

    const ForwardShape s = a.s;
    const uint16_t* kp = static_cast<const uint16_t*>(a.k);
    const uint16_t* qp = static_cast<const uint16_t*>(a.q);
    const uint16_t* vp = static_cast<const uint16_t*>(a.v);
    const int n_chunks = s.n_chunks;
    const int heads = int(s.heads);
    const int64_t n_g = int64_t(total) * DV * DK;  // elements of one G_c plane

    // Loads for chunk c (fewer than 2^31, checked at launch; chunk c % n_chunks of
    // sequence c / n_chunks, and the index of its entering state).  They never sit
    // behind a branch: tokens past the end of the sequence read the last valid token
    // and are zeroed once in registers.  Pieces 0-3 request a quarter of H_c each into
    // the L2 cache (direct loads whose LDS copies land on a sink nobody reads; the
    // state build reads H_c from there), the rest bring the keys and values into the
    // thread's staging slots, four slots per piece.  One piece is issued per CG
    // iteration of the previous chunk.  The gates and lambda go to registers with
    // plain loads issued before that loop (load_gates), so that no register merge
    // after a conditional piece waits for the loads in flight.
    constexpr int kRawSlots = L::kRawSlots;
    constexpr int kHcPieces = 4, kRawPer = 4;
    constexpr int kPieces = kHcPieces + (kRawSlots + kRawPer - 1) / kRawPer;
    auto issue_piece = [&](int c, int piece, int tid_in) {
        int tid = tid_in;
        asm volatile("" : "+v"(tid));
        const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
        const int lane = tid % kWave, fg = tid / 32;
        const int i0 = 2 * (tid % 32), i1 = i0 + 1;
        const int nn = c % n_chunks;
        const int bh_ = c / n_chunks;
        const int64_t t0_ = int64_t(nn) * kC;
        const int valid_ = int(min<int64_t>(kC, s.seq_len - t0_));
        const int64_t tok0_ = int64_t(bh_) * s.seq_len + t0_;
        if (piece < kHcPieces) {
            const float* Hf = static_cast<const float*>(a.Hs) + int64_t(c) * DK * DK;
#pragma unroll
            for (int u = piece * (kHcReq / kHcPieces); u < (piece + 1) * (kHcReq / kHcPieces); ++u) {
                const int f = wave * kHcReq + u;  // 1-KiB block of the chunk's H_c
                load_lds16(Hf + (f * kWave + lane) * 4, sSink);
            }
            return;
        }
        // staging slots: per key pass m slots 2m, 2m+1 = k of tokens 2p, 2p+1; then per
        // value pass two slots
        const int64_t r0 = tok0_ + min(i0, valid_ - 1), r1 = tok0_ + min(i1, valid_ - 1);
        uint4* slot = sRaw + wave * kWave;
#pragma unroll
        for (int q = 0; q < kRawSlots; ++q) {
            if (q / kRawPer != piece - kHcPieces) continue;
            const bool kk = q < 2 * NKQ;
            const int m = kk ? q / 2 : (q - 2 * NKQ) / 2;
            const int f0 = 64 * m + 8 * fg;
            const int64_t row = (q % 2) ? r1 : r0;
            const uint16_t* src = kk ? kp + row * DK + f0 : vp + row * DV + f0;
            load_lds16(src, slot + q * kThreads);
        }
    };
    auto issue_all = [&](int c, int tid_in) {
#pragma unroll
        for (int piece = 0; piece < kPieces; ++piece) issue_piece(c, piece, tid_in);
    };
    // gate and input-gate value of token `lane` of chunk c, and lambda element tid of its head
    auto load_gates = [&](int c, int tid_in, float& g_out, float& b_out, float& lam_out) {
        const int lane = tid_in % kWave;
        const int nn = c % n_chunks;
        const int bh_ = c / n_chunks;
        const int64_t t0_ = int64_t(nn) * kC;
        const int valid_ = int(min<int64_t>(kC, s.seq_len - t0_));
        const int64_t tok = int64_t(bh_) * s.seq_len + t0_ + min(lane, valid_ - 1);
        g_out = a.gamma[tok];
        b_out = a.beta[tok];
        lam_out = a.lambda[(bh_ % heads) * DK + min(tid_in, DK - 1)];
    };
    // One quarter of this wave's share of chunk c's G_c (high and low planes) into sGc:
    // the high plane's blocks first, then the low plane's.
    auto load_g = [&](int c, int quarter, int lane_in) {
        int lane = lane_in;
        asm volatile("" : "+v"(lane));
        const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
        const uint16_t* G = static_cast<const uint16_t*>(a.Gs) + int64_t(c) * DV * DK;
        constexpr int kPlaneBlocks = DV * DK * 2 / 1024;
#pragma unroll
        for (int u = quarter * (kGLoads / 4); u < (quarter + 1) * (kGLoads / 4); ++u) {
            const int f = wave * kGLoads + u;
            const int plane = f / kPlaneBlocks, fb = f % kPlaneBlocks;
            load_lds16(G + plane * n_g + (fb * kWave + lane) * 8, sGc + f * kWave * 8);
        }
    };

    int cc = blockIdx.x;
    float g_cur = 1.0f, b_cur = 0.0f, lam_cur = 0.0f;
    load_gates(cc, threadIdx.x, g_cur, b_cur, lam_cur);
    issue_all(cc, threadIdx.x);
    // the first chunk's staging data has landed; later chunks' data is waited for before the
    // previous chunk's read-out (the staging then does not wait for the read-out's stores)
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
    for (;;) {
        int tid = threadIdx.x;
        asm volatile("" : "+v"(tid));
        int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
        asm volatile("" : "+s"(wave));
        const int lane = tid % kWave;
        const int g = lane / 16;   // lane group: rows 4g..4g+3 of each tile
        const int ln = lane % 16;  // column (B / result layout) or row (A layout)
        const int j = wave * 16 + ln;  // this lane's token within the chunk
        const int p2 = tid % 32, fg = tid / 32;
        const int i0 = 2 * p2, i1 = 2 * p2 + 1;
        const int cn = cc + int(gridDim.x);
        const bool more = cn < total;
        const int n = cc % n_chunks;
        const int bh = cc / n_chunks;
        const int64_t t0 = int64_t(n) * kC;
        const int valid = int(min<int64_t>(kC, s.seq_len - t0));
        const int64_t tok0 = int64_t(bh) * s.seq_len + t0;

        // the first row tile of H_c (requested into L2 under the previous chunk's CG) is
        // read now, so that its latency passes during the staging
        const float* Hc = static_cast<const float*>(a.Hs) + int64_t(cc) * DK * DK;
        f32x4 hc[2][KS][2];
        auto load_hc = [&](int mt, f32x4 (&dst)[KS][2]) {
#pragma unroll
            for (int ks = 0; ks < KS; ++ks)
#pragma unroll
                for (int e = 0; e < 2; ++e)
                    dst[ks][e] = *reinterpret_cast<const f32x4*>(Hc + ((2 * (mt * KS + ks) + e) * kWave + lane) * 4);
        };
        load_hc(0, hc[0]);
        // ---- this thread's staging data and gates have landed (and the previous chunk's
        // G_c); the barrier ends the previous chunk's read-out
        uint4 kv[NKQ][2], vv[NV][2];
#pragma unroll
        for (int m = 0; m < NKQ; ++m) {
            kv[m][0] = sRaw[(2 * m + 0) * kThreads + tid];
            kv[m][1] = sRaw[(2 * m + 1) * kThreads + tid];
        }
#pragma unroll
        for (int m = 0; m < NV; ++m) {
            vv[m][0] = sRaw[(2 * NKQ + 2 * m + 0) * kThreads + tid];
            vv[m][1] = sRaw[(2 * NKQ + 2 * m + 1) * kThreads + tid];
        }
        __syncthreads();
        const float gl = lane < valid ? g_cur : 1.0f;
        const float bl = lane < valid ? b_cur : 0.0f;
        if (valid < kC) {
            const bool k0 = i0 < valid, k1 = i1 < valid;
#pragma unroll
            for (int m = 0; m < NKQ; ++m) {
                kv[m][0] = keep_if(k0, kv[m][0]);
                kv[m][1] = keep_if(k1, kv[m][1]);
            }
#pragma unroll
            for (int m = 0; m < NV; ++m) {
                vv[m][0] = keep_if(k0, vv[m][0]);
                vv[m][1] = keep_if(k1, vv[m][1]);
            }
        }
        if (tid < DK) sLam[tid] = lam_cur;
        // gate log-cumsums of the chunk (lane = token); a zero gate resets memory through
        // zl instead of log 0
        const float lgl = wave_scan_add(gl > 0.0f ? logf(gl) : 0.0f);
        const int zll = wave_scan_max((lane < valid && !(gl > 0.0f)) ? lane : -1);
        const float zeta_l = zll >= 0 ? 0.0f : __expf(lgl);  // zeta_{c+l,c}
        if (wave == 0) {
            sLg[lane] = lgl;
            sZl[lane] = zll;
            sZ0[lane] = zeta_l;
            sBeta[lane] = bl;
        }
        // rank-update weight relative to the chunk's entering state, u_i = beta_i /
        // zeta_{c+i,c}; 0 where that decay is <= kMinDecay
        const float u_l = zeta_l > kMinDecay ? bl * __expf(-lgl) : 0.0f;
        const float u0 = shfl_lane(u_l, i0), u1 = shfl_lane(u_l, i1);
#pragma unroll
        for (int m = 0; m < NKQ; ++m) {
            const int f0 = 64 * m + 8 * fg;
            put8x2(sK + i0 * LDK + f0, kv[m][0]);
            put8x2(sK + i1 * LDK + f0, kv[m][1]);
            stage_token_pair(reinterpret_cast<uint32_t*>(sKT), LDC / 2, f0, p2, kv[m][0], kv[m][1]);
            uint4 h0, l0, h1, l1;
            scale_split8(kv[m][0], u0, h0, l0);
            scale_split8(kv[m][1], u1, h1, l1);
            stage_token_pair(reinterpret_cast<uint32_t*>(sKUh), LDC / 2, f0, p2, h0, h1);
            stage_token_pair(reinterpret_cast<uint32_t*>(sKUl), LDC / 2, f0, p2, l0, l1);
        }
#pragma unroll
        for (int m = 0; m < NV; ++m)
            stage_token_pair(reinterpret_cast<uint32_t*>(sVT), LDC / 2, 64 * m + 8 * fg, p2, vv[m][0], vv[m][1]);
        __syncthreads();

        // ---- decays of this sub-chunk (see chunk_cg_bf16.hip): B'_w = B_w / Dw, with the
        // column scale zs_j = zeta_{c+j,c}; when Dw <= kMinDecay the state term is dropped
        // and B_w = sum_{i<16w} beta_i zeta_{16w-1,i} k_i k_i^T with zs_j = zt_j.
        const int jb = 16 * wave - 1;
        const float Dw = wave == 0 ? 1.0f : sZ0[jb];
        const bool keepH = wave == 0 || Dw > kMinDecay;
        const float zs = keepH ? sZ0[j] : decay_between_hw(sLg, sZl, jb, j);
        const float lgj = sLg[j];
        const int zlj = sZl[j];
        const f32x4 zw = decay_weights4(sLg, sBeta, lgj, zlj, 16 * wave + 4 * g, j);

        // ---- B'_w in fp32, then its high and low parts as A-fragments in the accumulation
        // registers: hfh/hfl[mt][ks] cover rows 16mt.., columns 32ks..  The accumulators
        // start from H_c (read from global memory one row tile ahead), the rank update's A
        // operand is K^T with the tokens i >= 16w zeroed (element e of step u is token
        // 32u + 4g + e (e < 4) or 32u + 16 + 4g + e - 4), its B operand the scaled keys,
        // high and low parts.
        // q of this lane's token (rows 16mt + 4g .. +3), used at the Jacobi start; a token
        // past the end reads the last valid one and is zeroed there
        uint2 qraw[MT];
        {
            const int64_t qrow = tok0 + min(j, valid - 1);
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) qraw[mt] = *reinterpret_cast<const uint2*>(qp + qrow * DK + 16 * mt + 4 * g);
        }
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
        f32x4 uw[2][2];
        if (!keepH) {  // never for wave 0, so jb >= 0
            const float lgb = sLg[jb];
            const int zlb = sZl[jb];
#pragma unroll
            for (int u = 0; u < 2; ++u)
#pragma unroll
                for (int hh = 0; hh < 2; ++hh) uw[u][hh] = decay_weights4(sLg, sBeta, lgb, zlb, 32 * u + 16 * hh + 4 * g, jb);
        }
        const int e_diag = ln - 4 * g;
        const bool on_diag = e_diag >= 0 && e_diag < 4;
        bf16x8 hfh[MT][KS], hfl[MT][KS];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            if (mt + 1 < MT) load_hc(mt + 1, hc[(mt + 1) % 2]);
            // scaled keys of the tile's columns (features 16mt + ln), high and low parts
            bf16x8 bwh[2], bwl[2];
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                if (keepH) {
                    bwh[u] = lds_frag(sKUh + (16 * mt + ln) * LDC + 32 * u + 4 * g);
                    bwl[u] = lds_frag(sKUl + (16 * mt + ln) * LDC + 32 * u + 4 * g);
                } else {
                    const bf16x8 kt = lds_frag(sKT + (16 * mt + ln) * LDC + 32 * u + 4 * g);
                    f32x4 y0, y1;
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        y0[e] = (float)kt[e] * uw[u][0][e];
                        y1[e] = (float)kt[4 + e] * uw[u][1][e];
                    }
                    split8(y0, y1, bwh[u], bwl[u]);
                }
            }
            if (!keepH) {  // the state term is dropped (wave-uniform, rare)
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) hc[mt % 2][ks][0] = hc[mt % 2][ks][1] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
            }
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                f32x4 lo = hc[mt % 2][ks][0];
                f32x4 hi = hc[mt % 2][ks][1];
#pragma unroll
                for (int u = 0; u < 2; ++u) {
                    lo = mfma16(ka[ks][0][u], bwh[u], lo);
                    lo = mfma16(ka[ks][0][u], bwl[u], lo);
                    hi = mfma16(ka[ks][1][u], bwh[u], hi);
                    hi = mfma16(ka[ks][1][u], bwl[u], hi);
                }
                split8(lo, hi, hfh[mt][ks], hfl[mt][ks]);
                asm("" : "=a"(hfh[mt][ks]) : "0"(hfh[mt][ks]));
                asm("" : "=a"(hfl[mt][ks]) : "0"(hfl[mt][ks]));
                // tile rows 16mt.. of fragment (mt, mt/2) hold the diagonal block
                if (ks == mt / 2) {
                    const f32x4 acc = (mt % 2) ? hi : lo;
                    const float dv = e_diag == 0 ? acc[0] : e_diag == 1 ? acc[1] : e_diag == 2 ? acc[2] : acc[3];
                    sDiag[wave * (DK + kWave) + (on_diag ? 16 * mt + ln : DK + lane)] = dv;
                }
            }
        }
        // ---- the sub-chunk's keys as A-fragments: rows of S (kf2); columns of W (kf3),
        // its 16 tokens in both halves of the contraction, met by S's high and low parts
        bf16x8 kf2[KS];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) kf2[ks] = lds_frag(sK + (16 * wave + ln) * LDK + 32 * ks + 4 * g);
        bf16x8 kf3[MT];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            const uint2 kk = *reinterpret_cast<const uint2*>(sKT + (16 * mt + ln) * LDC + 16 * wave + 4 * g);
            kf3[mt] = __builtin_bit_cast(bf16x8, make_uint4(kk.x, kk.y, kk.x, kk.y));
        }
        const f32x4 zero4 = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
        f32x4 x[MT], r[MT], p[MT], w[MT];

        // W = A_j vec for this wave's 16 columns from vec (fp32):
        //   W = zs_j (B'_w vec) + K_w^T (beta Z ⊙ (K_w vec)) + Lambda vec,
        // each matrix-core product on split operands.
        auto matvec = [&](const f32x4 (&vec)[MT], f32x4 (&w)[MT]) {
            f32x4 sacc = zero4;
            bf16x8 vh[KS], vl[KS];
            split8(vec[0], vec[1], vh[0], vl[0]);
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                // the next step's split runs among this step's products
                if (ks + 1 < KS) split8(vec[2 * ks + 2], vec[2 * ks + 3], vh[ks + 1], vl[ks + 1]);
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) {
                    w[mt] = mfma16(hfh[mt][ks], vh[ks], ks == 0 ? zero4 : w[mt]);
                    w[mt] = mfma16(hfh[mt][ks], vl[ks], w[mt]);
                    w[mt] = mfma16(hfl[mt][ks], vh[ks], w[mt]);
                }
                sacc = mfma16(kf2[ks], vh[ks], sacc);
                sacc = mfma16(kf2[ks], vl[ks], sacc);
                // one matrix-core op, one vector op, ... (the split's vector ops under this
                // step's products; with one wave per SIMD the wave's own vector work is all
                // that can fill the matrix cores' latency)
                if (ks + 1 < KS) {
#pragma unroll
                    for (int i = 0; i < 3 * MT; ++i) {
                        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                        __builtin_amdgcn_sched_group_barrier(0x002, 1, 0);
                    }
                    __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
                }
                __builtin_amdgcn_sched_barrier(0);
            }
            const bf16x8 sb = split4_stacked(sacc * zw);
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                const f32x4 lam = *reinterpret_cast<const f32x4*>(sLam + 16 * mt + 4 * g);
                w[mt] = mfma16(kf3[mt], sb, zs * w[mt]);
                w[mt] += lam * vec[mt];
            }
        };

        // ---- Jacobi start x0 = q / diag(H_t + Lambda), diag(H_t) = zs_j diag(B'_w) +
        // sum_{16w <= i <= j} beta_i Z[i][j] k_i^2 (k_i^2 has 16 significant bits: its
        // bf16 high and low parts are exact; the gate weights are split), then r0 = q - A x0.
        // Each column solves for q scaled by a power of two that brings |q|^2 into [1/2, 2)
        // (exact; it keeps alpha and beta where the hardware reciprocal is exact).
        int qsh = 0;
        {
            f32x4 qf[MT];
            const bool jv = j < valid;
            float qq = 0.0f;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                const uint2 qv2 = jv ? qraw[mt] : make_uint2(0u, 0u);
                qf[mt] = f32x4{bf16_bits_to_f32(qv2.x & 0xffffu), bf16_bits_to_f32(qv2.x >> 16),
                               bf16_bits_to_f32(qv2.y & 0xffffu), bf16_bits_to_f32(qv2.y >> 16)};
                qq += qf[mt][0] * qf[mt][0] + qf[mt][1] * qf[mt][1] + qf[mt][2] * qf[mt][2] + qf[mt][3] * qf[mt][3];
            }
            qsh = cg_scale_shift(col_sum(qq));
            const float qs = __builtin_ldexpf(1.0f, -qsh);
            const bf16x8 zws = split4_stacked(zw);  // (hi, lo) of the weights of tokens 4g + e
            const uint4 zwu = __builtin_bit_cast(uint4, zws);
            const bf16x8 zwh = __builtin_bit_cast(bf16x8, make_uint4(zwu.x, zwu.y, zwu.x, zwu.y));  // (hi, hi)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                // k^2 of the sub-chunk tokens, exact as (hi, lo): (hi, hi) against (w_hi, w_lo),
                // then (lo, 0) against (w_hi, w_hi)
                const uint4 kk = __builtin_bit_cast(uint4, kf3[mt]);
                const float k0 = __uint_as_float(kk.x << 16), k1 = __uint_as_float(kk.x & 0xffff0000u);
                const float k2 = __uint_as_float(kk.y << 16), k3 = __uint_as_float(kk.y & 0xffff0000u);
                uint32_t h01, l01, h23, l23;
                split2(k0 * k0, k1 * k1, h01, l01);
                split2(k2 * k2, k3 * k3, h23, l23);
                const bf16x8 kh = __builtin_bit_cast(bf16x8, make_uint4(h01, h23, h01, h23));
                const bf16x8 kl = __builtin_bit_cast(bf16x8, make_uint4(l01, l23, 0u, 0u));
                f32x4 dg2 = mfma16(kh, zws, zero4);   // k2_hi (w_hi + w_lo)
                dg2 = mfma16(kl, zwh, dg2);          // + k2_lo w_hi
                const f32x4 d = zs * *reinterpret_cast<const f32x4*>(&sDiag[wave * (DK + kWave) + 16 * mt + 4 * g]) + dg2 +
                                *reinterpret_cast<const f32x4*>(sLam + 16 * mt + 4 * g);
                qf[mt] = qs * qf[mt];
#pragma unroll
                for (int e = 0; e < 4; ++e) x[mt][e] = qf[mt][e] * __builtin_amdgcn_rcpf(d[e]);
            }
            matvec(x, w);
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) r[mt] = qf[mt] - w[mt];
        }
        float part = 0.0f;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            p[mt] = r[mt];
            part += r[mt][0] * r[mt][0] + r[mt][1] * r[mt][1] + r[mt][2] * r[mt][2] + r[mt][3] * r[mt][3];
        }
        float delta = col_sum(part);
        const float thr = a.eps2 * delta;  // Alg. 1: stop once |r|^2 <= eps^2 |r_0|^2
        bool active = delta >= kMinNormal;
        int steps = 0;

        // ---- every wave is done with sKT, sKUh and sKUl: the next chunk's loads may land
        // there while this chunk's CG runs (and G_c's loads run under it: no access of this
        // chunk's build or Jacobi start is ordered behind them)
        if (more) __syncthreads();
        float g_nx, b_nx, lam_nx;
        load_gates(more ? cn : cc, tid, g_nx, b_nx, lam_nx);
        int pieces = 0;   // pieces of the next chunk's loads issued so far
        int gq = 0;       // quarters of this chunk's G_c loaded so far

        // One CG step (App. C, Alg. 1), branch-free: a stopped column takes alpha = 0 and
        // beta = 0 and keeps x.  A column stops, after its x update, when the new squared
        // residual meets Alg. 1's relative test or falls below the smallest normal number
        // (relative to |q|^2), and without an update when p^T A p is not a positive normal
        // number.  The vector updates are written as in-place fused multiply-adds.
        auto cg_step = [&]() {
            matvec(p, w);
            f32x4 acc = zero4;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) acc += p[mt] * w[mt];
            const float pw = col_sum((acc[0] + acc[1]) + (acc[2] + acc[3]));
            const bool act1 = active && pw >= kMinNormal;
            steps += act1 ? 1 : 0;
            const float alpha = act1 ? delta * __builtin_amdgcn_rcpf(pw) : 0.0f;
            const float nalpha = -alpha;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    asm("v_fmac_f32 %0, %1, %2" : "+v"(x[mt][e]) : "v"(alpha), "v"(p[mt][e]));
                    asm("v_fmac_f32 %0, %1, %2" : "+v"(r[mt][e]) : "v"(nalpha), "v"(w[mt][e]));
                }
            acc = zero4;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) acc += r[mt] * r[mt];
            const float dn = col_sum((acc[0] + acc[1]) + (acc[2] + acc[3]));
            const bool act2 = act1 && dn >= kMinNormal && dn > thr;
            const float bcg = act2 ? dn * __builtin_amdgcn_rcpf(delta) : 0.0f;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int e = 0; e < 4; ++e) asm("v_fma_f32 %0, %1, %0, %2" : "+v"(p[mt][e]) : "v"(bcg), "v"(r[mt][e]));
            delta = act2 ? dn : delta;
            active = act2;
        };
        // the next loads are issued between iterations
        auto issue_next = [&]() {
            if (READOUT && gq < 4) load_g(cc, gq++, lane);
            else if (more && pieces < kPieces) issue_piece(cn, pieces++, tid);
        };
        // two iterations per pass with no branch between them, so the compiler schedules
        // the end of the first (the direction update) together with the start of the second
        // (its first products); a stopped column takes alpha = 0, so a wave whose columns have
        // all stopped after the first loses nothing but time in the second
        int it = 0;
        for (; it + 2 <= a.n_cg; it += 2) {
            if (!__any(active)) break;
            issue_next();
            issue_next();
            cg_step();
            cg_step();
        }
        if (it + 2 > a.n_cg && it < a.n_cg && __any(active)) {
            issue_next();
            cg_step();
        }
        {
            const float us = __builtin_ldexpf(1.0f, qsh);  // undoes the power-of-two scale of q
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) x[mt] = us * x[mt];
        }
        if (READOUT)
            while (gq < 4) load_g(cc, gq++, lane);
        if (more)
            while (pieces < kPieces) issue_piece(cn, pieces++, tid);

        if (a.steps && g == 0 && j < valid) a.steps[tok0 + j] = steps;
        if (a.qstar && j < valid) {
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
                *reinterpret_cast<f32x4*>(a.qstar + (tok0 + j) * DK + 16 * mt + 4 * g) = x[mt];
        }
        // ---- read-out o_j = G_c (zeta_j x_j) + sum_i beta_i Z[i][j] v_i (k_i^T x_j), on
        // split operands.  This wave's G_c loads (and the next chunk's) have landed; the
        // barrier publishes G_c to every wave.
        __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
        __syncthreads();
        if constexpr (READOUT) {
            const float zeta = sZ0[j];
            f32x4 zo[4];
#pragma unroll
            for (int it = 0; it < 4; ++it) zo[it] = decay_weights4(sLg, sBeta, lgj, zlj, 16 * it + 4 * g, j);
            // S = K x over the chunk's four token tiles (every wave runs all four; zo is zero
            // past the causal ones)
            f32x4 sacc[4];
#pragma unroll
            for (int it = 0; it < 4; ++it) sacc[it] = zero4;
            bf16x8 xzh[KS], xzl[KS];
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                bf16x8 xh, xl;
                split8(x[2 * ks], x[2 * ks + 1], xh, xl);
#pragma unroll
                for (int it = 0; it < 4; ++it) {
                    const bf16x8 kfr = lds_frag(sK + (16 * it + ln) * LDK + 32 * ks + 4 * g);
                    sacc[it] = mfma16(kfr, xh, sacc[it]);
                    sacc[it] = mfma16(kfr, xl, sacc[it]);
                }
                split8(zeta * x[2 * ks], zeta * x[2 * ks + 1], xzh[ks], xzl[ks]);
            }
            const uint16_t* Gl = sGc + DV * DK;  // low plane
            f32x4 o[MTV];
#pragma unroll
            for (int mt = 0; mt < MTV; ++mt) {
                o[mt] = zero4;
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) {
                    const int off = ((mt * KS + ks) * kWave + lane) * 8;
                    const bf16x8 gh = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(sGc + off));
                    const bf16x8 gl = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(Gl + off));
                    o[mt] = mfma16(gh, xzh[ks], o[mt]);
                    o[mt] = mfma16(gh, xzl[ks], o[mt]);
                    o[mt] = mfma16(gl, xzh[ks], o[mt]);
                }
            }
            // + V (beta Z ⊙ S): the values as A operand (32 tokens per step), S' split into
            // high and low parts over two steps of the same tokens
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                bf16x8 sh, sl;
                split8(sacc[2 * u] * zo[2 * u], sacc[2 * u + 1] * zo[2 * u + 1], sh, sl);
#pragma unroll
                for (int mt = 0; mt < MTV; ++mt) {
                    const bf16x8 vfr = lds_frag(sVT + (16 * mt + ln) * LDC + 32 * u + 4 * g);
                    o[mt] = mfma16(vfr, sh, o[mt]);
                    o[mt] = mfma16(vfr, sl, o[mt]);
                }
            }
            if (j < valid) {
#pragma unroll
                for (int mt = 0; mt < MTV; ++mt)
                    *reinterpret_cast<f32x4*>(a.out + (tok0 + j) * DV + 16 * mt + 4 * g) = o[mt];
            }
        }  // READOUT

        if (!more) break;
        cc = cn;
        g_cur = g_nx;
        b_cur = b_nx;
        lam_cur = lam_nx;
    }
}

template <int DK, int DV>
hipError_t launch_shape(const CgArgs& a, hipStream_t stream)
{
    const int64_t total = a.s.batch * a.s.heads * a.s.n_chunks;
    if (total <= 0) return hipSuccess;
    if (total > INT32_MAX) return hipErrorInvalidValue;
    // one workgroup fills a compute unit's LDS
    const int64_t cus = device_compute_units();
    const unsigned blocks = unsigned(total < cus ? total : cus);
    if (a.out)
        hipLaunchKernelGGL((chunk_cg_x3_kernel<DK, DV, true>), dim3(blocks), dim3(kThreads), 0, stream, a, int(total));
    else
        hipLaunchKernelGGL((chunk_cg_x3_kernel<DK, DV, false>), dim3(blocks), dim3(kThreads), 0, stream, a, int(total));
    return hipGetLastError();
}

}  // namespace

bool chunk_cg_x3_supported(const ForwardShape& s)
{
    return s.bf16 && s.chunk == kC && (s.d_k == 64 || s.d_k == 128) && (s.d_v == 64 || s.d_v == 128);
}

hipError_t launch_chunk_cg_x3(const CgArgs& a, hipStream_t stream)
{
    if (!chunk_cg_x3_supported(a.s)) return hipErrorInvalidValue;
    if (a.s.d_k == 64) return a.s.d_v == 64 ? launch_shape<64, 64>(a, stream) : launch_shape<64, 128>(a, stream);
    return a.s.d_v == 64 ? launch_shape<128, 64>(a, stream) : launch_shape<128, 128>(a, stream);
}

}  // namespace mesa
