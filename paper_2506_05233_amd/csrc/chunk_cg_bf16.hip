// Chunked conjugate gradients + read-out on the gfx950 matrix cores (bf16
// operands, fp32 accumulation), for bf16 q, k, v and chunk C = 64.
//
// Same mathematics as the fp32 path (App. C, Alg. 1 with its relative tolerance; App. D,
// Eq. q_star_parallel and Eq. gla): for the chunk starting after token c,
// with zeta_j = zeta_{c+j,c} and Z[i][j] = zeta_{c+j,c+i},
//
//   (H_t + Lambda) p_j = H_c (zeta_j p_j) + sum_{i<=j} beta_i Z[i][j] k_i (k_i^T p_j) + Lambda p_j
//   o_j               = G_c (zeta_j x_j) + sum_{i<=j} beta_i Z[i][j] v_i (k_i^T x_j).
//
// Work split: a workgroup (one per CU, looping over chunks) takes one chunk at a
// time; wave w owns the 16-token sub-chunk j = 16w .. 16w+15 and runs its own
// CG on it with no barrier.  Each wave first forms the state that enters its
// sub-chunk,
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
//
// Memory: the chunk's keys, queries, values and H_c come in by direct global ->
// LDS loads issued while the previous chunk's CG runs, into LDS that only the
// state build and the Jacobi start use (so HBM traffic is spread over the whole
// kernel instead of arriving in bursts at every chunk start); G_c is loaded the
// same way during the chunk's own build and CG.
#include <atomic>

#include "mesa_device.hpp"
#include "mesa_kernels.hpp"
#include "mesa_mfma.hpp"

namespace mesa {
namespace {

constexpr int kC = 64;         // chunk
constexpr int kThreads = 256;  // four waves, 16 tokens each

// Gate decay with the hardware exponential (relative error ~1e-7, far below
// the bf16 operand rounding of this path); same zero-gate rule as the shared
// helper.
__device__ __forceinline__ float decay_between_hw(const float* lg, const int* zl, int i, int j)
{
    if (i > j || zl[j] > i) return 0.0f;
    return __expf(lg[j] - lg[i]);
}


// beta_i prod_{s=i+1..j} gamma_s for the four tokens i = i4 .. i4+3 (i4 a multiple
// of 4) and token j, from the chunk's gate log-cumsums and strengths: 0 for i > j or
// when a zero gate lies in (i, j] (zl_j > i).  lgj = lg[j], zlj = zl[j].
__device__ __forceinline__ f32x4 decay_weights4(const float* lg, const float* beta, float lgj, int zlj, int i4, int j)
{
    const f32x4 lgi = *reinterpret_cast<const f32x4*>(lg + i4);
    const f32x4 bi = *reinterpret_cast<const f32x4*>(beta + i4);
    f32x4 r;
#pragma unroll
    for (int e = 0; e < 4; ++e) r[e] = (i4 + e <= j && zlj <= i4 + e) ? bi[e] * __expf(lgj - lgi[e]) : 0.0f;
    return r;
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

// LDS arena of the kernel (byte offsets).  G_c and diag(B'_w) have arrays of their
// own: G_c's direct loads run under the state build and the Jacobi start, and
// accesses the compiler can tell apart from them are not ordered behind them.
// The next chunk's staging data lands on
// the key tiles, scaled keys and queries (sKT, sKU, sQ) while the CG loop runs:
// those are only read before it.  Thread t's 16-byte staging slot q is at raw
// slot q * kThreads + t, so one wave's direct load fills 64 consecutive slots and
// every thread reads back its own slots.
template <int DK, int DV>
struct CgSmem {
    // Row strides (bf16 elements) of the token-major and feature-major tiles.  A fragment
    // read (two 8-byte LDS reads per lane) is served 16 lanes at a time from 32 four-byte
    // banks; rows 2 banks apart (a stride of 2 mod 32 words) give its 16 rows distinct bank
    // pairs, where rows 4 apart (+8 elements) made every such read take twice its cycles.
    // The rows are then 8-byte aligned only, so 16-byte stores into them are split.
    static constexpr int LDK = DK + 4;
    static constexpr int LDC = kC + 4;
    static constexpr int NKQ = DK / 64;  // staging passes over the key features
    static constexpr int NV = DV / 64;
    static constexpr int kRawSlots = 2 * (2 * NKQ + NV);
    static constexpr int oK = 0;                              // k_i[b], token-major
    static constexpr int oVT = oK + kC * LDK * 2;             // v_i[e], feature-major
    static constexpr int oLam = oVT + DV * LDC * 2;           // lambda
    static constexpr int oLg = oLam + DK * 4;                 // gate log-cumsums
    static constexpr int oBeta = oLg + kWave * 4;
    static constexpr int oZl = oBeta + kWave * 4;             // last zero gate
    static constexpr int oZ0 = oZl + kWave * 4;               // zeta_{c+j,c}
    static constexpr int oHf = oZ0 + kC * 4;                  // H_c as A-fragments
    static constexpr int oKT = oHf + DK * DK * 2;             // k_i[b], feature-major
    static constexpr int oKU = oKT + DK * LDC * 2;            // u_i k_i[b], feature-major
    static constexpr int oQ = oKU + DK * LDC * 2;             // q_j[b], token-major
    static constexpr int oRaw = oKT;                          // next chunk's staging slots
    static constexpr int kEnd = oQ + kC * LDK * 2;
    static constexpr int kRawEnd = oRaw + kRawSlots * kThreads * 16;
    static constexpr int kBytes = kEnd > kRawEnd ? kEnd : kRawEnd;
    static_assert(kBytes + DV * DK * 2 + (kThreads / kWave) * (DK + kWave) * 4 <= 160 * 1024,
                  "LDS use exceeds 160 KiB");
};

template <int DK, int DV, bool READOUT>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
void chunk_cg_bf16_kernel(CgArgs a, int total)
{
    using L = CgSmem<DK, DV>;
    constexpr int MT = DK / 16;    // 16-row tiles of a per-token vector
    constexpr int KS = DK / 32;    // 32-long contraction steps over features
    constexpr int MTV = DV / 16;   // 16-row tiles of an output column
    constexpr int LDK = L::LDK, LDC = L::LDC, NKQ = L::NKQ, NV = L::NV;
    constexpr int NHF = DK * DK / (8 * kWave) / 4;  // H_c fragments per wave
    constexpr int NGF = DV * DK / (8 * kWave) / 4;  // G_c fragments per wave

    __shared__ __attribute__((aligned(16))) unsigned char smem[L::kBytes];
    uint16_t* sK = reinterpret_cast<uint16_t*>(smem + L::oK);
    uint16_t* sVT = reinterpret_cast<uint16_t*>(smem + L::oVT);
    __shared__ __attribute__((aligned(16))) uint16_t sGf[DV * DK];  // G_c as A-fragments
    float* sLam = reinterpret_cast<float*>(smem + L::oLam);
    float* sLg = reinterpret_cast<float*>(smem + L::oLg);
    float* sBeta = reinterpret_cast<float*>(smem + L::oBeta);
    int* sZl = reinterpret_cast<int*>(smem + L::oZl);
    float* sZ0 = reinterpret_cast<float*>(smem + L::oZ0);
    __shared__ __attribute__((aligned(16))) float sDiag[kThreads / kWave][DK + kWave];  // diag(B'_w), spare slots
    uint16_t* sHf = reinterpret_cast<uint16_t*>(smem + L::oHf);
    uint16_t* sKT = reinterpret_cast<uint16_t*>(smem + L::oKT);
    uint16_t* sKU = reinterpret_cast<uint16_t*>(smem + L::oKU);
    uint16_t* sQ = reinterpret_cast<uint16_t*>(smem + L::oQ);
    uint4* sRaw = reinterpret_cast<uint4*>(smem + L::oRaw);

    const ForwardShape s = a.s;
    const uint16_t* kp = static_cast<const uint16_t*>(a.k);
    const uint16_t* qp = static_cast<const uint16_t*>(a.q);
    const uint16_t* vp = static_cast<const uint16_t*>(a.v);
    const int n_chunks = s.n_chunks;
    const int heads = int(s.heads);

    // Chunk c (fewer than 2^31, checked at launch) is chunk c % n_chunks of the
    // sequence (b, h) = c / n_chunks; it is also the index of its entering state.
    // Its loads never sit behind a branch: tokens past the end of the sequence read
    // the last valid token (valid >= 1) and are zeroed once the data is in
    // registers.  The gates and lambda go to registers; keys, queries and values to
    // the thread's own staging slots; H_c, as bf16 A-fragments (fragment f of lane l
    // at [f * 64 + l] * 8, one 1-KiB direct load per fragment), to sHf.  They are
    // issued in kPieces pieces (H_c in pieces of two direct loads, the staging slots
    // in pieces of four): a wave that issues many more at once stalls until the
    // first ones return, so the next chunk's pieces are spread over the CG
    // iterations of the current one, one per iteration.
    constexpr int kRawSlots = L::kRawSlots;
    constexpr int kHcPieces = NHF < 4 ? NHF : 4, kRawPer = 4;
    constexpr int kPieces = kHcPieces + (kRawSlots + kRawPer - 1) / kRawPer;
    auto issue_piece = [&](int c, int piece, int tid_in, float& g_out, float& b_out, float& lam_out) {
        int tid = tid_in;
        asm volatile("" : "+v"(tid));  // recompute the addresses here, not hoisted
        const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
        const int lane = tid % kWave, fg = tid / 32;
        const int i0 = 2 * (tid % 32), i1 = i0 + 1;
        const int nn = c % n_chunks;
        const int bh_ = c / n_chunks;
        const int64_t t0_ = int64_t(nn) * kC;
        const int valid_ = int(min<int64_t>(kC, s.seq_len - t0_));
        const int64_t tok0_ = int64_t(bh_) * s.seq_len + t0_;
        if (piece < kHcPieces) {
            if (piece == 0) {
                const int lt = min(lane, valid_ - 1);
                g_out = a.gamma[tok0_ + lt];
                b_out = a.beta[tok0_ + lt];
                lam_out = a.lambda[(bh_ % heads) * DK + min(tid, DK - 1)];
            }
            const uint16_t* Hf = static_cast<const uint16_t*>(a.Hs) + int64_t(c) * DK * DK;
#pragma unroll
            for (int u = piece * (NHF / kHcPieces); u < (piece + 1) * (NHF / kHcPieces); ++u) {
                const int f = wave * NHF + u;
                load_lds16(Hf + (f * kWave + lane) * 8, sHf + f * kWave * 8);
            }
            return;
        }
        // staging slots 4 (piece - 2) .. +3: per key/query pass m slots 4m .. 4m+3 =
        // (k, token 2p), (k, 2p+1), (q, 2p), (q, 2p+1); then per value pass two slots
        const int64_t r0 = tok0_ + min(i0, valid_ - 1), r1 = tok0_ + min(i1, valid_ - 1);
        uint4* slot = sRaw + wave * kWave;  // this wave's threads' slots of staging slot 0
#pragma unroll
        for (int q = 0; q < kRawSlots; ++q) {
            if (q / kRawPer != piece - kHcPieces) continue;
            const bool kq = q < 4 * NKQ;
            const int m = kq ? q / 4 : (q - 4 * NKQ) / 2;
            const int f0 = 64 * m + 8 * fg;
            const int64_t row = (kq ? q % 2 : (q - 4 * NKQ) % 2) ? r1 : r0;
            const uint16_t* src = kq ? ((q % 4) < 2 ? kp + row * DK + f0 : qp + row * DK + f0) : vp + row * DV + f0;
            load_lds16(src, slot + q * kThreads);
        }
    };
    auto issue_all = [&](int c, int tid_in, float& g_out, float& b_out, float& lam_out) {
#pragma unroll
        for (int piece = 0; piece < kPieces; ++piece) issue_piece(c, piece, tid_in, g_out, b_out, lam_out);
    };

    int cc = blockIdx.x;
    float g_cur = 1.0f, b_cur = 0.0f, lam_cur = 0.0f;
    issue_all(cc, threadIdx.x, g_cur, b_cur, lam_cur);
    // the first chunk's staging data has landed; later chunks' data is waited for before the
    // previous chunk's read-out (the staging then does not wait for the read-out's stores)
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
    for (;;) {
        // The thread's index values are re-derived for every chunk from a copy the
        // compiler cannot see through, so the many per-lane LDS addresses below are
        // recomputed where they are used rather than hoisted out of the chunk loop
        // into registers held for the whole kernel.
        int tid = threadIdx.x;
        asm volatile("" : "+v"(tid));
        int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
        asm volatile("" : "+s"(wave));
        const int lane = tid % kWave;
        const int g = lane / 16;   // lane group: rows 4g..4g+3 of each tile
        const int ln = lane % 16;  // column (B / result layout) or row (A layout)
        const int j = wave * 16 + ln;  // this lane's token within the chunk
        // thread t stages tokens 2p, 2p+1 (p = t % 32) for 8 features per pass
        const int p2 = tid % 32, fg = tid / 32;
        const int i0 = 2 * p2, i1 = 2 * p2 + 1;
        const int cn = cc + int(gridDim.x);
        const bool more = cn < total;
        const int n = cc % n_chunks;
        const int bh = cc / n_chunks;
        const int64_t t0 = int64_t(n) * kC;
        const int valid = int(min<int64_t>(kC, s.seq_len - t0));
        const int64_t tok0 = int64_t(bh) * s.seq_len + t0;

        // ---- this thread's staging data, its gates and this wave's H_c fragments have
        // landed; the barrier publishes H_c and ends the previous chunk's read-out
        uint4 kv[NKQ][2], qv[NKQ][2], vv[NV][2];
#pragma unroll
        for (int m = 0; m < NKQ; ++m) {
            kv[m][0] = sRaw[(4 * m + 0) * kThreads + tid];
            kv[m][1] = sRaw[(4 * m + 1) * kThreads + tid];
            qv[m][0] = sRaw[(4 * m + 2) * kThreads + tid];
            qv[m][1] = sRaw[(4 * m + 3) * kThreads + tid];
        }
#pragma unroll
        for (int m = 0; m < NV; ++m) {
            vv[m][0] = sRaw[(4 * NKQ + 2 * m + 0) * kThreads + tid];
            vv[m][1] = sRaw[(4 * NKQ + 2 * m + 1) * kThreads + tid];
        }
        __syncthreads();
        // gates and write strengths of the chunk, one token per lane, in every wave;
        // absent tokens have gate 1 and strength 0
        const float gl = lane < valid ? g_cur : 1.0f;
        const float bl = lane < valid ? b_cur : 0.0f;
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
        if (tid < DK) sLam[tid] = lam_cur;
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
        const float u0 = shfl_lane(u_l, i0), u1 = shfl_lane(u_l, i1);
#pragma unroll
        for (int m = 0; m < NKQ; ++m) {
            const int f0 = 64 * m + 8 * fg;
            put8x2(sK + i0 * LDK + f0, kv[m][0]);
            put8x2(sK + i1 * LDK + f0, kv[m][1]);
            put8x2(sQ + i0 * LDK + f0, qv[m][0]);
            put8x2(sQ + i1 * LDK + f0, qv[m][1]);
            stage_token_pair(reinterpret_cast<uint32_t*>(sKT), LDC / 2, f0, p2, kv[m][0], kv[m][1]);
            stage_token_pair(reinterpret_cast<uint32_t*>(sKU), LDC / 2, f0, p2, scale_bf16x8(kv[m][0], u0),
                             scale_bf16x8(kv[m][1], u1));
        }
#pragma unroll
        for (int m = 0; m < NV; ++m)
            stage_token_pair(reinterpret_cast<uint32_t*>(sVT), LDC / 2, 64 * m + 8 * fg, p2, vv[m][0], vv[m][1]);
        __syncthreads();

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
        const float lgj = sLg[j];
        const int zlj = sZl[j];
        // beta_i Z[i][j] for the sub-chunk rows i = 16w + 4g + ii met in S
        const f32x4 zw = decay_weights4(sLg, sBeta, lgj, zlj, 16 * wave + 4 * g, j);

        // ---- B'_w as bf16 A-fragments: hf[mt][s] covers rows 16mt.., columns 32s..
        // Every wave runs the same straight-line code: both 32-token steps of the rank update
        // (of the second only its lower half: no sub-chunk state takes tokens 48..63), with the
        // tokens i >= 16w zeroed in its A operand (rows 32s + 16h.., independent of mt, loaded
        // once).  Element e of step u is token 32u + 4g + e (e < 4) or 32u + 16 + 4g + e - 4, so
        // whole halves are in or out: the lower half of step u iff 32u + 16 <= 16w, the upper
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
        // (tokens i > jb, i.e. i >= 16w, get 0)
        f32x4 uw[2][2];
        if (!keepH) {  // never for wave 0, so jb >= 0
            const float lgb = sLg[jb];
            const int zlb = sZl[jb];
#pragma unroll
            for (int u = 0; u < 2; ++u)
#pragma unroll
                for (int hh = 0; hh < 2; ++hh) uw[u][hh] = decay_weights4(sLg, sBeta, lgb, zlb, 32 * u + 16 * hh + 4 * g, jb);
        }
        // H_c enters through the contraction of the second rank step: no sub-chunk uses the
        // tokens 48..63 (its upper k-half), so that half carries an identity in the A operand
        // and an A-fragment half of H_c in the B operand, which adds H_c's rows 32s + {0..15}
        // or 32s + {16..31} to the 16x16 result tile they belong to (zero when the state term
        // is dropped).  Two products per result tile: step 0, then step 1's lower half with H_c.
        uint2 id_up;
        {
            bf16x8 t;
            const float one = keepH ? 1.0f : 0.0f;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                t[e] = (__bf16)0.0f;
                t[4 + e] = (__bf16)(4 * g + e == ln ? one : 0.0f);
            }
            const uint4 u = __builtin_bit_cast(uint4, t);
            id_up = make_uint2(u.z, u.w);
        }
        // diag(B'_w) goes to sDiag[wave][r]; lanes off the diagonal write a spare slot instead
        const int e_diag = ln - 4 * g;
        const bool on_diag = e_diag >= 0 && e_diag < 4;
        bf16x8 hf[MT][KS];
        // operands of row tile mt: H_c fragments (mt, 0..KS-1) and the scaled keys; the
        // next tile's are read from LDS while this tile's products run
        auto load_tile = [&](int mt, bf16x8 (&hcs)[KS], bf16x8 (&bw)[2]) {
#pragma unroll
            for (int ks = 0; ks < KS; ++ks)
                hcs[ks] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(sHf + ((mt * KS + ks) * kWave + lane) * 8));
#pragma unroll
            for (int u = 0; u < 2; ++u) bw[u] = lds_frag((keepH ? sKU : sKT) + (16 * mt + ln) * LDC + 32 * u + 4 * g);
        };
        bf16x8 hcA[KS], hcB[KS], bwA[2], bwB[2];
        load_tile(0, hcA, bwA);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            bf16x8 (&hcs)[KS] = (mt % 2) ? hcB : hcA;
            bf16x8 (&bw)[2] = (mt % 2) ? bwB : bwA;
            if (mt + 1 < MT) load_tile(mt + 1, (mt % 2) ? hcA : hcB, (mt % 2) ? bwA : bwB);
            if (!keepH) {
#pragma unroll
                for (int u = 0; u < 2; ++u)
#pragma unroll
                    for (int e = 0; e < 8; ++e) bw[u][e] = (__bf16)((float)bw[u][e] * uw[u][e / 4][e % 4]);
            }
            const uint4 b1 = __builtin_bit_cast(uint4, bw[1]);
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                const uint4 h = __builtin_bit_cast(uint4, hcs[ks]);
                const uint4 a0 = __builtin_bit_cast(uint4, ka[ks][0][1]), a1 = __builtin_bit_cast(uint4, ka[ks][1][1]);
                f32x4 lo = mfma16(ka[ks][0][0], bw[0], f32x4{0.0f, 0.0f, 0.0f, 0.0f});
                f32x4 hi = mfma16(ka[ks][1][0], bw[0], f32x4{0.0f, 0.0f, 0.0f, 0.0f});
                lo = mfma16(__builtin_bit_cast(bf16x8, make_uint4(a0.x, a0.y, id_up.x, id_up.y)),
                            __builtin_bit_cast(bf16x8, make_uint4(b1.x, b1.y, h.x, h.y)), lo);
                hi = mfma16(__builtin_bit_cast(bf16x8, make_uint4(a1.x, a1.y, id_up.x, id_up.y)),
                            __builtin_bit_cast(bf16x8, make_uint4(b1.x, b1.y, h.z, h.w)), hi);
                hf[mt][ks] = pack8(lo, hi);
                // B'_w is read only as the A operand of the state products.  Those accept the
                // accumulation registers directly, so it goes there as it is formed: the loop's
                // fp32 vectors then have the ordinary vector registers to themselves.  (Not
                // volatile: the move is not a scheduling barrier.)
                asm("" : "=a"(hf[mt][ks]) : "0"(hf[mt][ks]));
                // Tile rows 16mt.. of fragment (mt, mt/2) hold the diagonal block: lane (g, n)
                // has B'[16mt + 4g + e][16mt + n], on the diagonal for n = 4g + e.
                if (ks == mt / 2) {
                    const f32x4 acc = (mt % 2) ? hi : lo;
                    const float dv = e_diag == 0 ? acc[0] : e_diag == 1 ? acc[1] : e_diag == 2 ? acc[2] : acc[3];
                    sDiag[wave][on_diag ? 16 * mt + ln : DK + lane] = dv;
                }
            }
        }
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
        int qsh = 0;  // log2 of the power-of-two scale of q_j (below)
        // CG vectors; the search direction alternates between p and pa (below)
        f32x4 x[MT], r[MT], p[MT], pa[MT], w[MT];

        // W = A_j vec for this wave's 16 columns (A_j = H_t + Lambda of token j), from the
        // bf16 operand vb of vec: W = zs_j (B'_w vec) + K_w^T S' + Lambda vec, the column
        // scale applied to the state products' accumulators.  The state products run
        // feature-step-major, so the first ones need only vb[0].
        // Inside the CG loop the previous iteration's x update (x += alpha p, deferred: it is
        // off the loop's dependency chain) runs between the state products, two tiles of x
        // per feature step, where the matrix cores leave the vector unit idle.
        auto matvec_x = [&](const bf16x8 (&vb)[KS], f32x4 (&w)[MT], const f32x4 (&pd)[MT], float ad) {
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) w[mt] = zero4;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) w[mt] = mfma16(hf[mt][ks], vb[ks], w[mt]);
#pragma unroll
                for (int mt = ks * MT / KS; mt < (ks + 1) * MT / KS; ++mt) x[mt] += ad * pd[mt];
            }
            f32x4 sacc = zero4;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) sacc = mfma16(kf2[ks], vb[ks], sacc);
            const uint2 sb = pack4(sacc * zw);
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                const uint4 v = __builtin_bit_cast(uint4, vb[mt / 2]);
                const uint4 op = (mt % 2) ? make_uint4(sb.x, sb.y, v.z, v.w) : make_uint4(sb.x, sb.y, v.x, v.y);
                w[mt] *= zs;
                w[mt] = mfma16(kf3[mt], __builtin_bit_cast(bf16x8, op), w[mt]);
            }
        };

        // ---- Jacobi start x0 = q / diag(H_t + Lambda),
        //      diag(H_t) = zs_j diag(B'_w) + sum_{16w <= i <= j} beta_i Z[i][j] k_i^2, diag(B'_w)
        //      read back from this wave's sDiag rows (written by other lanes of the same wave;
        //      a wave's LDS accesses complete in order).
        // Each column's system is solved for q_j scaled by a power of two that brings |q_j|^2
        // into [1/4, 2): CG iterates are homogeneous in q and a power-of-two scale is exact, so
        // this changes no rounding, and it keeps the CG scalars in the range where the
        // hardware reciprocal is exact to an ulp.
        {
            const bf16x8 zwb = pack8(zw, zero4);
            // every LDS operand of the start in one batch: q_j, diag(B'_w) and lambda
            uint2 qv[MT];
            f32x4 dgl[MT], lml[MT];
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                qv[mt] = *reinterpret_cast<const uint2*>(sQ + j * LDK + 16 * mt + 4 * g);
                dgl[mt] = *reinterpret_cast<const f32x4*>(&sDiag[wave][16 * mt + 4 * g]);
                lml[mt] = *reinterpret_cast<const f32x4*>(sLam + 16 * mt + 4 * g);
            }
            __builtin_amdgcn_sched_barrier(0);
            f32x4 qf[MT];
            float qq = 0.0f;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                qf[mt] = f32x4{bf16_bits_to_f32(qv[mt].x & 0xffffu), bf16_bits_to_f32(qv[mt].x >> 16),
                               bf16_bits_to_f32(qv[mt].y & 0xffffu), bf16_bits_to_f32(qv[mt].y >> 16)};
                qq += qf[mt][0] * qf[mt][0] + qf[mt][1] * qf[mt][1] + qf[mt][2] * qf[mt][2] + qf[mt][3] * qf[mt][3];
            }
            qsh = __builtin_amdgcn_frexp_expf(col_sum(qq)) >> 1;  // |q|^2 = m 2^e, m in [1/2, 1)
            const float qs = __builtin_ldexpf(1.0f, -qsh);
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                bf16x8 ksq = kf3[mt];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float v = (float)ksq[e];
                    ksq[e] = (__bf16)(v * v);
                }
                const f32x4 dg2 = mfma16(ksq, zwb, zero4);
                const f32x4 d = zs * dgl[mt] + dg2 + lml[mt];
                qf[mt] = qs * qf[mt];
#pragma unroll
                for (int e = 0; e < 4; ++e) x[mt][e] = qf[mt][e] * __builtin_amdgcn_rcpf(d[e]);
            }
            // kf2 and kf3 are read only as A operands from here on: like B'_w they move to
            // the accumulation registers, leaving the ordinary ones to the CG vectors.
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) asm("" : "=a"(kf2[ks]) : "0"(kf2[ks]));
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) asm("" : "=a"(kf3[mt]) : "0"(kf3[mt]));
            bf16x8 xb[KS];
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) xb[ks] = pack8(x[2 * ks], x[2 * ks + 1]);
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) pa[mt] = zero4;
            matvec_x(xb, w, pa, 0.0f);
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
        const float thr = a.eps2 * delta;  // Alg. 1: the column stops once |r|^2 <= eps^2 |r_0|^2
        bool active = delta >= kMinNormal;
        int steps = 0;  // iterations that updated x

        // ---- every wave is done with sHf, sKT, sKU and sQ: the next chunk's loads may land
        // there while this chunk's CG runs (the barrier also waits for this wave's memory
        // operations, so nothing is issued before it)
        if (more) __syncthreads();
        // G_c is needed only by the read-out: its loads run under the CG loop (no LDS
        // access of this chunk's build or Jacobi start is ordered behind them)
        if constexpr (READOUT) {
            const uint16_t* Gf = static_cast<const uint16_t*>(a.Gs) + int64_t(cc) * DV * DK;
#pragma unroll
            for (int u = 0; u < NGF; ++u) {
                const int f = wave * NGF + u;
                load_lds16(Gf + (f * kWave + lane) * 8, sGf + f * kWave * 8);
            }
        }
        float g_nx = 1.0f, b_nx = 0.0f, lam_nx = 0.0f;
        int pieces = 0;  // pieces of the next chunk's loads issued so far

        // One CG step (App. C, Alg. 1), branch-free: a stopped column takes alpha = 0 and
        // keeps x.  A column stops, after its x update, when the new squared residual meets
        // Alg. 1's relative test (<= eps^2 |r_0|^2; with eps = 0 Alg. 1 stops at exactly zero)
        // or falls below the smallest normal number (relative to |q|^2, which the scaling
        // above keeps in [1/4, 2)); it stops without an update when p^T A p is not a
        // positive normal number (alpha would need the reciprocal of a subnormal).
        // Iteration k reads the direction from pc and writes the next one into pn, the
        // buffer holding the previous direction: its deferred x update has run by then
        // (inside the matrix-vector product).  Two iterations per pass swap the roles,
        // so no vector is copied.
        float alpha_d = 0.0f;  // the pending x update: x += alpha_d * (previous direction)
        auto cg_step = [&](f32x4 (&pc)[MT], f32x4 (&pn)[MT]) {
            {
                bf16x8 pb[KS];
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) pb[ks] = pack8(pc[2 * ks], pc[2 * ks + 1]);
                matvec_x(pb, w, pn, alpha_d);
            }
            // column dot products in four independent partial sums (one per element of a
            // tile), so consecutive fused multiply-adds do not wait on each other
            f32x4 acc = zero4;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) acc += pc[mt] * w[mt];
            const float pw = col_sum((acc[0] + acc[1]) + (acc[2] + acc[3]));
            const bool act1 = active && pw >= kMinNormal;
            steps += act1 ? 1 : 0;
            // Branch-free: a stopped column takes alpha = 0 and beta = 0.  Its r and x stay
            // as they are, and its direction becomes r (finite), which only ever meets
            // alpha = 0 again: a column never restarts.
            const float alpha = act1 ? delta * __builtin_amdgcn_rcpf(pw) : 0.0f;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) r[mt] -= alpha * w[mt];
            alpha_d = alpha;
            acc = zero4;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) acc += r[mt] * r[mt];
            const float dn = col_sum((acc[0] + acc[1]) + (acc[2] + acc[3]));
            const bool act2 = act1 && dn >= kMinNormal && dn > thr;
            const float bcg = act2 ? dn * __builtin_amdgcn_rcpf(delta) : 0.0f;
            // pn = r + bcg pc into pn's own registers: one three-address fma per element (the
            // compiler's two-address form would first copy r, which stays live)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int e = 0; e < 4; ++e) asm("v_fma_f32 %0, %1, %2, %3" : "=v"(pn[mt][e]) : "v"(bcg), "v"(pc[mt][e]), "v"(r[mt][e]));
            delta = act2 ? dn : delta;
            active = act2;
        };
        // Pairs of iterations (an odd count ends with one more), the pass's two pieces of the
        // next chunk's loads issued first: no branch between the two iterations, so the
        // compiler schedules the end of the first (the direction update) together with the
        // start of the second (its first products).  The wave leaves at a pass boundary once
        // every column has stopped (a stopped column takes alpha = 0, so a second iteration
        // after the last column stopped changes nothing).
        int it = 0;
        bool last_pa = false;  // the last iteration run read its direction from pa
        for (; it + 2 <= a.n_cg; it += 2) {
            if (!__any(active)) break;
            if (more && pieces < kPieces) issue_piece(cn, pieces++, tid, g_nx, b_nx, lam_nx);
            if (more && pieces < kPieces) issue_piece(cn, pieces++, tid, g_nx, b_nx, lam_nx);
            cg_step(p, pa);
            cg_step(pa, p);
            last_pa = true;
        }
        if (it + 2 > a.n_cg && it < a.n_cg && __any(active)) {
            if (more && pieces < kPieces) issue_piece(cn, pieces++, tid, g_nx, b_nx, lam_nx);
            cg_step(p, pa);
            last_pa = false;
        }
        // the last iteration's x update
        if (last_pa) {
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) x[mt] += alpha_d * pa[mt];
        } else {
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) x[mt] += alpha_d * p[mt];
        }
        {
            const float us = __builtin_ldexpf(1.0f, qsh);  // undoes the power-of-two scale of q
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) x[mt] = us * x[mt];
        }

        if (more)
            while (pieces < kPieces) issue_piece(cn, pieces++, tid, g_nx, b_nx, lam_nx);

        // ---- read-out o_j = G_c (zeta_j x_j) + sum_i beta_i Z[i][j] v_i (k_i^T x_j)
        // this wave's G_c fragments (and the next chunk's loads) have landed; the barrier
        // publishes G_c to every wave
        __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
        __syncthreads();
        if (a.steps && g == 0 && j < valid) a.steps[tok0 + j] = steps;
        if (a.qstar && j < valid) {
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
                *reinterpret_cast<f32x4*>(a.qstar + (tok0 + j) * DK + 16 * mt + 4 * g) = x[mt];
        }
        if constexpr (READOUT) {
            const float zeta = sZ0[j];
            // Operands come from LDS in batches issued ahead of their products (the CG
            // vectors and the state fragments are dead here, so registers are plentiful):
            // the keys of all four token tiles and the first half of G_c, then the rest of
            // G_c and the values while the first products run.
            constexpr int MTH = MTV / 2;
            bf16x8 kq[4][KS], g0[MTH][KS], g1[MTH][KS], vq[2][MTV];
#pragma unroll
            for (int it = 0; it < 4; ++it)
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) kq[it][ks] = lds_frag(sK + (16 * it + ln) * LDK + 32 * ks + 4 * g);
#pragma unroll
            for (int mt = 0; mt < MTH; ++mt)
#pragma unroll
                for (int ks = 0; ks < KS; ++ks)
                    g0[mt][ks] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(sGf + ((mt * KS + ks) * kWave + lane) * 8));
            f32x4 zo[4];  // beta_i Z[i][j] over the four token tiles (0 past the causal ones)
#pragma unroll
            for (int it = 0; it < 4; ++it) zo[it] = decay_weights4(sLg, sBeta, lgj, zlj, 16 * it + 4 * g, j);
            bf16x8 xb[KS], xz[KS];
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                xb[ks] = pack8(x[2 * ks], x[2 * ks + 1]);
                xz[ks] = pack8(zeta * x[2 * ks], zeta * x[2 * ks + 1]);
            }
#pragma unroll
            for (int mt = 0; mt < MTH; ++mt)
#pragma unroll
                for (int ks = 0; ks < KS; ++ks)
                    g1[mt][ks] = __builtin_bit_cast(
                        bf16x8, *reinterpret_cast<const uint4*>(sGf + (((MTH + mt) * KS + ks) * kWave + lane) * 8));
            // (the scheduler keeps these loads ahead of the products)
            __builtin_amdgcn_sched_barrier(0);
            // every wave runs all four token tiles (zo is zero past the causal ones)
            f32x4 sacc[4];
#pragma unroll
            for (int it = 0; it < 4; ++it) {
                sacc[it] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) sacc[it] = mfma16(kq[it][ks], xb[ks], sacc[it]);
            }
#pragma unroll
            for (int u = 0; u < 2; ++u)
#pragma unroll
                for (int mt = 0; mt < MTV; ++mt) vq[u][mt] = lds_frag(sVT + (16 * mt + ln) * LDC + 32 * u + 4 * g);
            __builtin_amdgcn_sched_barrier(0);
            f32x4 o[MTV];
#pragma unroll
            for (int mt = 0; mt < MTV; ++mt) {
                o[mt] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) o[mt] = mfma16(mt < MTH ? g0[mt][ks] : g1[mt - MTH][ks], xz[ks], o[mt]);
            }
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                const bf16x8 sb = pack8(sacc[2 * u] * zo[2 * u], sacc[2 * u + 1] * zo[2 * u + 1]);
#pragma unroll
                for (int mt = 0; mt < MTV; ++mt) o[mt] = mfma16(vq[u][mt], sb, o[mt]);
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
    // without an output the read-out (and the loads of G_c and v it needs) is skipped
    if (a.out)
        hipLaunchKernelGGL((chunk_cg_bf16_kernel<DK, DV, true>), dim3(blocks), dim3(kThreads), 0, stream, a, int(total));
    else
        hipLaunchKernelGGL((chunk_cg_bf16_kernel<DK, DV, false>), dim3(blocks), dim3(kThreads), 0, stream, a, int(total));
    return hipGetLastError();
}

}  // namespace

int device_compute_units()
{
    static std::atomic<int> cached[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0) return 1;
    if (dev < 64) {
        const int c = cached[dev].load(std::memory_order_relaxed);
        if (c > 0) return c;
    }
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 1;
    if (dev < 64) cached[dev].store(n, std::memory_order_relaxed);
    return n;
}

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
