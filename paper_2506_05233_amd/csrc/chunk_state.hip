// Chunk-state scan of the Mesa layer (App. D, chunkwise form): the states
// entering every chunk, H_c and G_c for c = 0, C, 2C, ...
//
//   H_{c+C} = zeta_{c+C,c} H_c + sum_{i in chunk} zeta_{c+C,i} beta_i k_i k_i^T
//   G_{c+C} = zeta_{c+C,c} G_c + sum_{i in chunk} zeta_{c+C,i} beta_i v_i k_i^T
//
// (the gated recurrences of Sec. 2 summed over one chunk, unrolled as in App. D).
// One workgroup owns a 16-row tile of H or of G for one (batch, head) and
// walks the chunks in order, so every state element is written exactly once per
// chunk with coalesced stores.  The tile stays in registers between chunks.
// HBM traffic per token-head: the states, 4 (d_k + d_v) d_k / C bytes, plus the
// chunk's k and v, read once per tile.
#include <type_traits>

#include "mesa_device.hpp"
#include "mesa_kernels.hpp"
#include "mesa_mfma.hpp"

namespace mesa {
namespace {

constexpr int kThreads = 256;
constexpr int kTileRows = 16;
constexpr int kMaxCols = 128;
constexpr int kPerThread = kTileRows * kMaxCols / kThreads;  // 8

template <typename Tin>
__global__ __launch_bounds__(kThreads) void chunk_state_kernel(StateArgs a)
{
    const ForwardShape s = a.s;
    const int dk = s.d_k, dv = s.d_v, C = s.chunk;
    const int ntile_h = dk / kTileRows;
    const int ntile = ntile_h + dv / kTileRows;
    const int blk = xcd_major_block(blockIdx.x, gridDim.x);
    const int tile = blk % ntile;
    const int64_t bh = blk / ntile;
    const bool isG = tile >= ntile_h;  // tiles [0, d_k/16): rows of H; then rows of G
    const int r0 = (isG ? tile - ntile_h : tile) * kTileRows;
    const int nrow = isG ? dv : dk;    // rows of the whole state
    const int nel = kTileRows * dk;    // a tile spans all d_k columns
    const int tid = threadIdx.x;
    const Tin* kp = static_cast<const Tin*>(a.k);
    const Tin* rp = static_cast<const Tin*>(isG ? a.v : a.k);

    __shared__ float sR[64][kTileRows + 1];  // rows r0.. of k_i (H) or v_i (G)
    __shared__ float sB[64][kMaxCols + 1];   // k_i, all d_k columns
    __shared__ float sW[64];                 // beta_i * zeta_{chunk end, i}
    __shared__ float sLg[64];
    __shared__ int sZl[64];
    __shared__ float sD;                     // zeta_{chunk end, chunk start}

    float st[kPerThread];
#pragma unroll
    for (int m = 0; m < kPerThread; ++m) st[m] = 0.0f;

    float* chunk_dst = static_cast<float*>(isG ? a.Gs : a.Hs);
    for (int n = 0; n < s.n_chunks; ++n) {
        const int64_t t0 = int64_t(n) * C;
        const int valid = int(min<int64_t>(C, s.seq_len - t0));
        const int64_t tok0 = bh * s.seq_len + t0;
        if (a.store_chunks) {
            float* dst = chunk_dst + ((bh * s.n_chunks + n) * nrow + r0) * int64_t(dk);
#pragma unroll
            for (int m = 0; m < kPerThread; ++m) {
                const int e = tid + kThreads * m;
                if (e < nel) dst[e] = st[m];
            }
        }
        for (int e = tid; e < C * dk; e += kThreads) {
            const int i = e / dk, c = e % dk;
            sB[i][c] = i < valid ? to_f32(kp[(tok0 + i) * dk + c]) : 0.0f;
        }
        for (int e = tid; e < C * kTileRows; e += kThreads) {
            const int i = e / kTileRows, r = e % kTileRows;
            sR[i][r] = i < valid ? to_f32(rp[(tok0 + i) * nrow + r0 + r]) : 0.0f;
        }
        if (tid < kWave) chunk_log_decays(a.gamma + tok0, valid, sLg, sZl);
        __syncthreads();
        if (tid < C) sW[tid] = tid < valid ? a.beta[tok0 + tid] * decay_between(sLg, sZl, tid, C - 1) : 0.0f;
        if (tid == 0) sD = decay_from_start(sLg, sZl, C - 1);
        __syncthreads();
        const float D = sD;
#pragma unroll
        for (int m = 0; m < kPerThread; ++m) {
            const int e = tid + kThreads * m;
            if (e < nel) {
                const int row = e / dk, col = e % dk;
                float acc = 0.0f;
                for (int i = 0; i < C; ++i) acc += sW[i] * sR[i][row] * sB[i][col];
                st[m] = D * st[m] + acc;
            }
        }
        __syncthreads();
    }
    float* fin = isG ? a.final_G : a.final_H;
    if (fin) {
        float* dst = fin + (bh * nrow + r0) * int64_t(dk);
#pragma unroll
        for (int m = 0; m < kPerThread; ++m) {
            const int e = tid + kThreads * m;
            if (e < nel) dst[e] = st[m];
        }
    }
}

// Matrix-core variant for bf16 k and v (chunk 64).  The stacked state
// [H; G] ((d_k + d_v) x d_k) is cut into 64-row x 32-column tiles, one per
// workgroup; wave w keeps rows 16w..16w+15 of the tile as two 16x16 MFMA
// result tiles and updates them in place, chunk after chunk:
//
//   M <- zeta_{end,start} M + X^T (w ⊙ K),   w_i = beta_i zeta_{end,i},
//
// with X = the chunk's keys (rows of H) or values (rows of G).  X is exact in
// bf16; w ⊙ K is split into a bf16 high part and a bf16 remainder and both are
// multiplied (two passes), so each term carries about 2^-17 relative error and
// the state stays fp32-accurate to ~1e-6.  The next chunk's inputs are
// prefetched into registers while the current one is multiplied, and each wave
// runs the gate scan itself, so a chunk costs two barriers.
__global__ __launch_bounds__(kThreads) void chunk_state_mfma_kernel(StateArgs a)
{
    constexpr int C = 64;
    constexpr int KST = C / 32;   // 32-token contraction steps per chunk
    // row stride (elements) of the token-minor LDS tiles: 34 words, so the 16 rows of a fragment
    // read (8 bytes per lane, 16 lanes at a time over 32 banks) fall in distinct bank pairs
    constexpr int LDT = C + 4;
    const ForwardShape s = a.s;
    const int dk = s.d_k, dv = s.d_v;
    const int nrt = (dk + dv) / 64, nct = dk / 32;
    const int blk = xcd_major_block(blockIdx.x, gridDim.x);
    const int ct = blk % nct;
    const int rt = (blk / nct) % nrt;
    const int64_t bh = blk / (nct * nrt);
    const bool isG = rt * 64 >= dk;
    const int xr0 = isG ? rt * 64 - dk : rt * 64;  // first row of the tile within H or G
    const int nX = isG ? dv : dk;                  // rows of that state = width of its source
    const int col0 = ct * 32;
    const uint16_t* xp = static_cast<const uint16_t*>(isG ? a.v : a.k);
    const uint16_t* kp = static_cast<const uint16_t*>(a.k);
    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
    const int lane = tid % kWave;
    const int g = lane / 16, ln = lane % 16;

    __shared__ __attribute__((aligned(16))) uint16_t sA[64 * LDT];   // X[i][row], as [row][i]
    __shared__ __attribute__((aligned(16))) uint16_t sBh[32 * LDT];  // hi(w_i K[i][c]), as [c][i]
    __shared__ __attribute__((aligned(16))) uint16_t sBl[32 * LDT];  // remainder
    __shared__ float sW[kWave];  // w_i = beta_i zeta_{chunk end, i} of the chunk being staged

    // register prefetch of one chunk: X rows, K columns, gates
    // inputs of one chunk, held in registers: prefetched two chunks ahead
    struct ChunkRegs {
        uint4 ra[2];  // A rows of tokens 2p, 2p+1
        uint4 rb[2];  // B columns of tokens 2p, 2p+1
        float gam, bet;
        int valid;
    };
    auto load_chunk = [&](int n, ChunkRegs& R) {
        const int64_t t0 = int64_t(n) * C;
        const int valid = int(min<int64_t>(C, s.seq_len - t0));
        const int64_t tok0 = bh * s.seq_len + t0;
        R.valid = valid;
        // thread t: tokens 2p, 2p+1 with p = t % 32; A rows f8 = 8 (t / 32), B columns f8 = 8 (t / 32 % 4)
        {
            const int p = tid % 32, f8 = 8 * (tid / 32);
#pragma unroll
            for (int h2 = 0; h2 < 2; ++h2) {
                const int i = 2 * p + h2;
                R.ra[h2] = i < valid ? *reinterpret_cast<const uint4*>(xp + (tok0 + i) * nX + xr0 + f8) : make_uint4(0, 0, 0, 0);
            }
        }
        {
            const int p = tid % 32, f8 = 8 * ((tid / 32) % 4);
#pragma unroll
            for (int h2 = 0; h2 < 2; ++h2) {
                const int i = 2 * p + h2;
                R.rb[h2] = i < valid ? *reinterpret_cast<const uint4*>(kp + (tok0 + i) * dk + col0 + f8) : make_uint4(0, 0, 0, 0);
            }
        }
        R.gam = lane < valid ? a.gamma[tok0 + lane] : 1.0f;
        R.bet = lane < valid ? a.beta[tok0 + lane] : 0.0f;
    };

    f32x4 acc[2] = {f32x4{0.0f, 0.0f, 0.0f, 0.0f}, f32x4{0.0f, 0.0f, 0.0f, 0.0f}};
    float* chunk_dst = static_cast<float*>(isG ? a.Gs : a.Hs);
    auto step = [&](int n, ChunkRegs& R) {
        // gate scan of this chunk, per wave (lane i = in-chunk token i)
        const float lg = wave_scan_add((lane < R.valid && R.gam > 0.0f) ? logf(R.gam) : 0.0f);
        const int zl = wave_scan_max((lane < R.valid && !(R.gam > 0.0f)) ? lane : -1);
        const float lgE = lane_value(lg, C - 1);
        const int zlE = lane_value(zl, C - 1);
        const float wl = lane < R.valid ? R.bet * (zlE > lane ? 0.0f : expf(lgE - lg)) : 0.0f;
        const float D = zlE >= 0 ? 0.0f : expf(lgE);

        if (wave == 0) sW[lane] = wl;  // all waves computed the same weights
        __syncthreads();  // the previous chunk's products are done with LDS
        stage_token_pair(reinterpret_cast<uint32_t*>(sA), LDT / 2, 8 * (tid / 32), tid % 32, R.ra[0], R.ra[1]);
        {
            // B = hi/lo split of w_i x_i[c] for tokens 2p, 2p+1 (threads t < 128)
            const int p = tid % 32, f8 = 8 * ((tid / 32) % 4);
            const float w0 = sW[2 * p], w1 = sW[2 * p + 1];
            if (tid < 128) {
                const uint32_t a4[4] = {R.rb[0].x, R.rb[0].y, R.rb[0].z, R.rb[0].w};
                const uint32_t b4[4] = {R.rb[1].x, R.rb[1].y, R.rb[1].z, R.rb[1].w};
                uint32_t* hi32 = reinterpret_cast<uint32_t*>(sBh);
                uint32_t* lo32 = reinterpret_cast<uint32_t*>(sBl);
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    const uint32_t ba = (q & 1) ? (a4[q / 2] >> 16) : (a4[q / 2] & 0xffffu);
                    const uint32_t bb = (q & 1) ? (b4[q / 2] >> 16) : (b4[q / 2] & 0xffffu);
                    const float va = w0 * bf16_bits_to_f32(ba), vb = w1 * bf16_bits_to_f32(bb);
                    const __bf16 ha = (__bf16)va, hb = (__bf16)vb;
                    const __bf16 la = (__bf16)(va - (float)ha), lb = (__bf16)(vb - (float)hb);
                    hi32[(f8 + q) * (LDT / 2) + p] = uint32_t(bf16_bits(ha)) | (uint32_t(bf16_bits(hb)) << 16);
                    lo32[(f8 + q) * (LDT / 2) + p] = uint32_t(bf16_bits(la)) | (uint32_t(bf16_bits(lb)) << 16);
                }
            }
        }
        __syncthreads();
        if (n + 2 < s.n_chunks) load_chunk(n + 2, R);

        if (a.store_chunks) {
            float* dst = chunk_dst + ((bh * s.n_chunks + n) * nX + xr0 + 16 * wave + 4 * g) * int64_t(dk) + col0 + ln;
#pragma unroll
            for (int nt = 0; nt < 2; ++nt)
#pragma unroll
                for (int ii = 0; ii < 4; ++ii) dst[ii * dk + 16 * nt] = acc[nt][ii];
        }
        acc[0] *= D;
        acc[1] *= D;
#pragma unroll
        for (int u = 0; u < KST; ++u) {
            const bf16x8 af = lds_frag(sA + (16 * wave + ln) * LDT + 32 * u + 4 * g);
#pragma unroll
            for (int nt = 0; nt < 2; ++nt) {
                acc[nt] = mfma16(af, lds_frag(sBh + (16 * nt + ln) * LDT + 32 * u + 4 * g), acc[nt]);
                acc[nt] = mfma16(af, lds_frag(sBl + (16 * nt + ln) * LDT + 32 * u + 4 * g), acc[nt]);
            }
        }
        };
    ChunkRegs R0, R1;
    load_chunk(0, R0);
    if (s.n_chunks > 1) load_chunk(1, R1);
    for (int n = 0; n < s.n_chunks; n += 2) {
        step(n, R0);
        if (n + 1 < s.n_chunks) step(n + 1, R1);
    }
    float* fin = isG ? a.final_G : a.final_H;
    if (fin) {
        float* dst = fin + (bh * nX + xr0 + 16 * wave + 4 * g) * int64_t(dk) + col0 + ln;
#pragma unroll
        for (int nt = 0; nt < 2; ++nt)
#pragma unroll
            for (int ii = 0; ii < 4; ++ii) dst[ii * dk + 16 * nt] = acc[nt][ii];
    }
}

// fp32 variant (fp32 k and v, chunk 64): the same update, M <- D M + X^T (w ⊙ K),
// on the matrix cores in fp32 (v_mfma_f32_16x16x4f32: exact fp32 products and
// fp32 sums, as the scalar kernel).  Each wave owns one 16x16 tile of the stacked
// state [H; G] -- a workgroup's four waves the four 16-column tiles of 64 columns
// of the same 16 rows -- and runs on its own: it scans the chunk's gates itself
// and passes its operands through a private LDS slice, so no barrier couples the
// waves.  A chunk is 16 dependent products (~512 cycles), shorter than a memory
// round trip, so a chunk's inputs are loaded kF32Depth chunks ahead; they travel
// as 16-byte row pieces (token-major), are scaled by w_i once, and each product
// reads k-slot g = tokens 4j + g of the staged slices.
constexpr int kF32Depth = 4;

template <int DK, bool STORE>
__global__ __launch_bounds__(kThreads) void chunk_state_f32_kernel(StateArgs a)
{
    constexpr int C = 64;
    constexpr int kGroups = DK / 64;  // 64-column groups per row tile
    const ForwardShape s = a.s;
    const int dv = s.d_v;
    const int nrt = (DK + dv) / 16;
    const int blk = xcd_major_block(blockIdx.x, gridDim.x);
    const int grp = blk % kGroups;
    const int rt = (blk / kGroups) % nrt;
    const int64_t bh = blk / (kGroups * nrt);
    const bool isG = rt * 16 >= DK;
    const int xr0 = isG ? rt * 16 - DK : rt * 16;  // first row of the tile within H or G
    const int nX = isG ? dv : DK;                  // rows of that state = width of its source
    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
    const int lane = tid % kWave;
    const int g = lane / 16, m = lane % 16;
    const int c0 = grp * 64 + 16 * wave;
    // staging: lane holds columns q4 .. q4 + 3 of in-chunk tokens tq + 16 r, r < 4
    const int q4 = 4 * (lane % 4), tq = lane / 4;
    const float* xp = static_cast<const float*>(isG ? a.v : a.k) + xr0 + q4;
    const float* yp = static_cast<const float*>(a.k) + c0 + q4;

    __shared__ __attribute__((aligned(16))) float sX[kThreads / kWave][C * 16];  // [token][row]
    __shared__ __attribute__((aligned(16))) float sY[kThreads / kWave][C * 16];  // [token][column], times w
    float* const wx = sX[wave];
    float* const wy = sY[wave];

    struct Regs {
        f32x4 x[4], y[4];
        float gam, bet;
        int valid;
    };
    // chunk n of a sequence with n_chunks >= 1.  Tokens past the end re-read the
    // chunk's last token (in bounds, branch-free); the step gives them beta = 0 and
    // gamma = 1, so they add exact zeros.  Nothing here waits for the loads.
    auto load = [&](int n, Regs& R) {
        const int64_t t0 = int64_t(n) * C;
        const int valid = int(min<int64_t>(C, s.seq_len - t0));
        const int64_t tok0 = bh * s.seq_len + t0;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int64_t tok = tok0 + min(tq + 16 * r, valid - 1);
            R.x[r] = *reinterpret_cast<const f32x4*>(xp + tok * nX);
            R.y[r] = *reinterpret_cast<const f32x4*>(yp + tok * DK);
        }
        R.gam = a.gamma[tok0 + min(lane, valid - 1)];
        R.bet = a.beta[tok0 + min(lane, valid - 1)];
        R.valid = valid;
    };

    f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
    const int64_t tile_off = (xr0 + 4 * g) * int64_t(DK) + c0 + m;  // element (4g, m) of the tile
    float* chunk_dst = STORE ? static_cast<float*>(isG ? a.Gs : a.Hs) + bh * s.n_chunks * nX * int64_t(DK) + tile_off
                                      : nullptr;
    auto step = [&](int n, const Regs& R) {
        // gate scan (lane i = in-chunk token i; absent tokens have gamma 1, beta 0)
        const bool in = lane < R.valid;
        const float gam = in ? R.gam : 1.0f;
        const float lg = wave_scan_add(gam > 0.0f ? logf(gam) : 0.0f);
        const int zl = wave_scan_max(gam > 0.0f ? -1 : lane);
        const float lgE = lane_value(lg, C - 1);
        const int zlE = lane_value(zl, C - 1);
        const float wl = in ? R.bet * (zlE > lane ? 0.0f : expf(lgE - lg)) : 0.0f;
        const float D = zlE >= 0 ? 0.0f : expf(lgE);

        if (STORE) {
            float* dst = chunk_dst + int64_t(n) * nX * DK;
#pragma unroll
            for (int ii = 0; ii < 4; ++ii) dst[ii * DK] = acc[ii];
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const float w = shfl_lane(wl, tq + 16 * r);
            *reinterpret_cast<f32x4*>(wx + (tq + 16 * r) * 16 + q4) = R.x[r];
            *reinterpret_cast<f32x4*>(wy + (tq + 16 * r) * 16 + q4) = w * R.y[r];
        }
        // the wave's own LDS traffic completes in order: its reads below see these writes
        __builtin_amdgcn_wave_barrier();
        acc *= D;
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            const int e = (4 * j + g) * 16 + m;
            acc = __builtin_amdgcn_mfma_f32_16x16x4f32(wx[e], wy[e], acc, 0, 0, 0);
        }
        __builtin_amdgcn_wave_barrier();
    };

    // A ring of kF32Depth (= 4) chunks in flight, in named registers.  Every pass of
    // the main loop issues the same loads (past the end: the last chunk again, in
    // bounds and unused), so the count of loads in flight is the same at every
    // point of every pass and each wait covers exactly the chunk it needs.
    static_assert(kF32Depth == 4, "the ring below holds four chunks");
    Regs R0, R1, R2, R3;
    const int nc = s.n_chunks;
    if (nc > 0) {
        load(0, R0);
        load(min(1, nc - 1), R1);
        load(min(2, nc - 1), R2);
        load(min(3, nc - 1), R3);
    }
    // The scheduling barriers keep each chunk's work in its slot: hoisted to the top
    // of the pass, the later chunks' gate scans would wait for their loads there.
    int n0 = 0;
    for (; n0 + kF32Depth <= nc; n0 += kF32Depth) {
        step(n0, R0);
        load(min(n0 + 4, nc - 1), R0);
        __builtin_amdgcn_sched_barrier(0);
        step(n0 + 1, R1);
        load(min(n0 + 5, nc - 1), R1);
        __builtin_amdgcn_sched_barrier(0);
        step(n0 + 2, R2);
        load(min(n0 + 6, nc - 1), R2);
        __builtin_amdgcn_sched_barrier(0);
        step(n0 + 3, R3);
        load(min(n0 + 7, nc - 1), R3);
        __builtin_amdgcn_sched_barrier(0);
    }
    if (n0 < nc) step(n0, R0);
    if (n0 + 1 < nc) step(n0 + 1, R1);
    if (n0 + 2 < nc) step(n0 + 2, R2);
    float* fin = isG ? a.final_G : a.final_H;
    if (fin) {
        float* dst = fin + bh * nX * int64_t(DK) + tile_off;
#pragma unroll
        for (int ii = 0; ii < 4; ++ii) dst[ii * DK] = acc[ii];
    }
}

// Wide variant (bf16 k and v, chunk 64, d_k and d_v in {64, 128}), used for the
// bf16 fragment chunk states and for the states-only call.  Two workgroups share the
// state of one (batch, head) sequence -- part 0 is H (d_k x d_k), part 1 is G^T
// (d_k x d_v), both as [key feature R][column c] -- in registers, and walk its chunks
// in order:
//
//   X_{next} = D X + K^T (w ⊙ Y),   Y = K (part 0) or V (part 1), w_i = beta_i zeta_{end,i}.
//
// With d_k = d_v and single products each workgroup owns half of the columns of both
// parts, so both read the same bytes (k and half of v) and write the same share of the
// states; otherwise one workgroup owns H and the other G^T.
//
// When fp32 states leave the kernel (the final states), w ⊙ Y is split into bf16
// high and low parts (two products, ~16-bit weights, states fp32-accurate); when
// only the bf16 chunk states are produced, the high part alone is used: its
// rounding (2^-9 per term, averaged over the chunk's 64 terms) stays well below the
// bf16 rounding of the stored states.
// Eight waves (two per SIMD, so one hides the other's latencies); wave w owns key
// rows 32 (w % NS) .. +31 (NS = d_k / 32) and a 1/CS share of the columns
// (CS = 8 / NS); its 16x16 result tiles pair up into complete bf16 A-fragments of
// the fragment layout (rows 32s.. of X^T are fragment row block s), so every chunk
// state is written with whole 1-KiB wave stores.  Staging is double-buffered in LDS
// (one barrier per chunk); the inputs of chunk n + 3 are loaded into registers while
// chunk n is consumed (a chunk's work is shorter than a memory round trip under
// load), and the staging of chunk n + 1 is interleaved with the products of chunk n.
//
// Few sequences (batch x heads below the compute units) leave most of the chip idle
// during this chained walk, so there the chunks are cut into segments and the scan
// runs in two launches.  The first computes each segment's total from a zero state,
// T_s = sum over its chunks of the decayed updates, and the decay across it, D_s
// (the product of its chunk decays).  The second starts every segment from the
// state entering it, E_0 = 0 and E_{s+1} = D_s E_s + T_s -- the same chunk recurrence
// applied to whole segments -- and walks the segment's chunks as above.
constexpr int kWideThreads = 512;  // eight waves: two per SIMD

// Segments of one launch of the wide scan.
struct SegPlan {
    int len;      // chunks per segment (the last may be shorter)
    int total;    // segments of a sequence
    int first;    // first segment this launch walks
    int count;    // segments this launch walks, per (sequence, part)
    bool totals;  // write T_s and D_s (first launch) instead of chunk and final states
    float* tot;   // [B*H, total - 1, d_k (d_k + d_v)]: T_s of H as [R][c], then of G as [c][R]
    float* dec;   // [B*H, total]: D_s
};

template <int DK, int DV, bool STORE, bool SPLIT, bool PLAIN = false, bool X3 = false>
__global__ __launch_bounds__(kWideThreads) void chunk_state_wide_kernel(StateArgs a, SegPlan sg)
{
    constexpr int C = 64;
    constexpr int LDT = C + 4;           // row stride of the [feature][token] tiles (34 words: see above)
    constexpr int NS = DK / 32;          // 32-row blocks of the key features
    constexpr int CS = kWideThreads / kWave / NS;  // column shares per row block
    constexpr int FPP = 8 * kWideThreads / 32;     // features staged per pass (8 per thread group)
    const ForwardShape s = a.s;
    const int blk = xcd_major_block(blockIdx.x, gridDim.x);  // the two halves of a segment share an L2
    // d_k = d_v, bf16 states only: workgroup `half` owns H's columns and G^T's columns
    // half * d/2 .. + d/2 - 1 (both halves then read k and half of v); otherwise half 0
    // owns H and half 1 owns G^T.  (The split-product variants ran 22-28% slower balanced.)
    constexpr bool BAL = DK == DV && !SPLIT;
    const int half = blk % 2;
    const int seg = sg.first + (blk / 2) % sg.count;
    const int64_t bh = blk / 2 / sg.count;
    const int nbeg = seg * sg.len, nend = min(nbeg + sg.len, s.n_chunks);  // this segment's chunks
    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
    const int lane = tid % kWave;
    const int g = lane / 16, ln = lane % 16;
    const int p = tid % 32, fg = tid / 32;  // staging: tokens 2p, 2p+1, features 8 fg + FPP m ..

    __shared__ __attribute__((aligned(16))) uint16_t sA[2][DK * LDT];                           // k_i[R], [R][i]
    __shared__ __attribute__((aligned(16))) uint16_t sBh[2][(DK > DV ? DK : DV) * LDT];         // hi(w_i y_i[c]), [c][i]
    __shared__ __attribute__((aligned(16))) uint16_t sBl[2][(DK > DV ? DK : DV) * LDT];         // lo(w_i y_i[c])

    auto run = [&](auto nc_tag) {
        constexpr int NC = decltype(nc_tag)::value;  // columns of this workgroup
        constexpr int NCT = NC / 16 / CS;            // 16-column tiles of this wave
        constexpr int NKQ = (DK + FPP - 1) / FPP, NY = (NC + FPP - 1) / FPP;  // staging passes
        const int sblk = wave % NS, cs = wave / NS;
        // Staged y column c: balanced, k feature c if c lies in this half's own region
        // (c / (NC/2) == half), else v feature half * NC/2 + c % (NC/2); otherwise k (half 0)
        // or v (half 1) feature c.  The wave's local column tiles lct0 .. are H's or G^T's
        // (`part`), its global column tiles ct0 .. of that part.
        auto y_from_k = [&](int c) { return BAL ? c / (NC / 2) == half : half == 0; };
        const int lct0 = cs * NCT;
        const int part = BAL ? int(!y_from_k(16 * lct0)) : half;
        const int ct0 = (BAL && part) ? half * (NC / 32) + lct0 % (NC / 32) : lct0;
        const uint16_t* kp = static_cast<const uint16_t*>(a.k);
        const uint16_t* vp = static_cast<const uint16_t*>(a.v);

        struct Regs {
            uint4 k[NKQ][2];  // k of tokens 2p, 2p+1, features 64m + 8fg ..
            uint4 y[NY][2];   // y of the same tokens (v; unused for H, whose y is k)
            float gam, bet;
            int valid;
        };
        auto load = [&](int n, Regs& R) {
            const int64_t t0 = int64_t(n) * C;
            const int valid = int(min<int64_t>(C, s.seq_len - t0));
            const int64_t tok0 = bh * s.seq_len + t0;
            R.valid = valid;
            const int lt = min(lane, valid - 1);
            R.gam = a.gamma[tok0 + lt];
            R.bet = a.beta[tok0 + lt];
            const int64_t r0 = tok0 + min(2 * p, valid - 1), r1 = tok0 + min(2 * p + 1, valid - 1);
            // feature offsets beyond the row wrap into it (those threads stage nothing)
#pragma unroll
            for (int m = 0; m < NKQ; ++m) {
                const int f0 = (FPP * m + 8 * fg) % DK;
                R.k[m][0] = *reinterpret_cast<const uint4*>(kp + r0 * DK + f0);
                R.k[m][1] = *reinterpret_cast<const uint4*>(kp + r1 * DK + f0);
            }
#pragma unroll
            for (int m = 0; m < NY; ++m) {
                const int f0 = (FPP * m + 8 * fg) % NC;
                if (y_from_k(f0)) continue;  // wave-uniform: k is already in R.k
                const int vf = BAL ? half * (NC / 2) + f0 % (NC / 2) : f0;
                R.y[m][0] = *reinterpret_cast<const uint4*>(vp + r0 * DV + vf);
                R.y[m][1] = *reinterpret_cast<const uint4*>(vp + r1 * DV + vf);
            }
        };
        // Staging of a chunk into buffer b, in three pieces that the chunk loop interleaves
        // with the previous chunk's products: the gate scan (write weights w_i = beta_i
        // zeta_{end,i} of this thread's two tokens, and the chunk decay D), the key tile, and
        // the weighted y tile split into bf16 high and low parts (features q0 .. q1-1 of this
        // thread's group).
        struct Gate {
            float w0, w1, D;
        };
        auto gates = [&](const Regs& R) -> Gate {
            const bool live = lane < R.valid;
            const float gl = live ? R.gam : 1.0f;
            const float lg = wave_scan_add(gl > 0.0f ? logf(gl) : 0.0f);
            const int zl = wave_scan_max((live && !(gl > 0.0f)) ? lane : -1);
            const float lgE = lane_value(lg, C - 1);
            const int zlE = lane_value(zl, C - 1);
            const float wl = live ? R.bet * (zlE > lane ? 0.0f : expf(lgE - lg)) : 0.0f;
            return Gate{shfl_lane(wl, 2 * p), shfl_lane(wl, 2 * p + 1), zlE >= 0 ? 0.0f : expf(lgE)};
        };
        auto stage_k = [&](const Regs& R, int b) {
            const bool k0 = 2 * p < R.valid, k1 = 2 * p + 1 < R.valid;
#pragma unroll
            for (int m = 0; m < NKQ; ++m) {
                if (FPP * m + 8 * fg >= DK) continue;
                const uint4 ka = k0 ? R.k[m][0] : make_uint4(0, 0, 0, 0);
                const uint4 kb = k1 ? R.k[m][1] : make_uint4(0, 0, 0, 0);
                stage_token_pair(reinterpret_cast<uint32_t*>(sA[b]), LDT / 2, FPP * m + 8 * fg, p, ka, kb);
            }
        };
        auto stage_y = [&](const Regs& R, int b, const Gate& gt, int q0, int q1) {
#pragma unroll
            for (int m = 0; m < NY; ++m) {
                if (FPP * m + 8 * fg >= NC) continue;
                const bool fk = m < NKQ && y_from_k(FPP * m + 8 * fg);
                const uint4 ya = fk ? R.k[m < NKQ ? m : 0][0] : R.y[m][0];
                const uint4 yb = fk ? R.k[m < NKQ ? m : 0][1] : R.y[m][1];
                const uint32_t a4[4] = {ya.x, ya.y, ya.z, ya.w};
                const uint32_t b4[4] = {yb.x, yb.y, yb.z, yb.w};
                uint32_t* hi32 = reinterpret_cast<uint32_t*>(sBh[b]);
                uint32_t* lo32 = reinterpret_cast<uint32_t*>(sBl[b]);
#pragma unroll
                for (int q = q0; q < q1; ++q) {
                    // feature q of tokens 2p and 2p+1: bf16 bits widened by a shift or a mask
                    const float va = gt.w0 * __uint_as_float((q & 1) ? (a4[q / 2] & 0xffff0000u) : (a4[q / 2] << 16));
                    const float vb = gt.w1 * __uint_as_float((q & 1) ? (b4[q / 2] & 0xffff0000u) : (b4[q / 2] << 16));
                    const uint32_t h2 = pack_bf16x2(va, vb);
                    const int c = FPP * m + 8 * fg + q;
                    hi32[c * (LDT / 2) + p] = h2;
                    if (SPLIT) lo32[c * (LDT / 2) + p] = pack_bf16x2(va - __uint_as_float(h2 << 16), vb - __uint_as_float(h2 & 0xffff0000u));
                }
            }
        };

        f32x4 acc[2][NCT];
#pragma unroll
        for (int rt = 0; rt < 2; ++rt)
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) acc[rt][ct] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
        constexpr bool frag_out = STORE;
        uint16_t* frag_base = static_cast<uint16_t*>(part ? a.Gs : a.Hs);
        constexpr int kStateElems = NC * DK;  // bf16 per chunk state of this part
        float* plain_base = part ? a.Gs32 : a.Hs32;  // fp32 plain chunk states (PLAIN)
        // element offset of this thread's tile value (rt, ct, ii) -- row R, column c of the
        // part -- in a [R][c] (H) or [c][R] (G) fp32 state
        auto tile_off = [&](int rt, int ct, int ii) -> int {
            const int R = 32 * sblk + 16 * rt + 4 * g + ii, c = 16 * (ct0 + ct) + ln;
            return part ? c * DK + R : R * DK + c;
        };

        // chunk n: its state is stored, then acc = D acc + K^T (w ⊙ Y) from buffer n % 2;
        // chunk n + 1 is staged (from Rn1) into the other buffer and chunk n + 3 loaded
        float dprod = 1.0f;  // decay across the chunks walked so far
        auto consume = [&](int n, float D, Regs& Rn1, Regs& Rfree, float& Dnext) {
            if (frag_out && X3 && part == 0) {
                // H_c as fp32 fragments: half e of fragment f, lane l at [(2 f + e) 64 + l] x 4
                float* base = static_cast<float*>(a.Hs) + (bh * s.n_chunks + n) * int64_t(kStateElems);
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct) {
                    const int f = (ct0 + ct) * NS + sblk;
                    *reinterpret_cast<f32x4*>(base + ((2 * f + 0) * kWave + lane) * 4) = acc[0][ct];
                    *reinterpret_cast<f32x4*>(base + ((2 * f + 1) * kWave + lane) * 4) = acc[1][ct];
                }
            } else if (frag_out) {
                // bf16 fragments; with X3 (G_c) the high parts, and the low parts
                // bf16(x - hi) in a second plane of the same layout after all chunks' states
                uint16_t* base = frag_base + (bh * s.n_chunks + n) * int64_t(kStateElems);
                const int64_t lo_plane = s.batch * s.heads * int64_t(s.n_chunks) * kStateElems;
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct) {
                    const uint4 pk = make_uint4(pack_bf16x2(acc[0][ct][0], acc[0][ct][1]), pack_bf16x2(acc[0][ct][2], acc[0][ct][3]),
                                                pack_bf16x2(acc[1][ct][0], acc[1][ct][1]), pack_bf16x2(acc[1][ct][2], acc[1][ct][3]));
                    const int64_t off = (((ct0 + ct) * NS + sblk) * kWave + lane) * 8;
                    *reinterpret_cast<uint4*>(base + off) = pk;
                    if constexpr (X3) {
                        auto lo2 = [](float x0, float x1, uint32_t h) {
                            return pack_bf16x2(x0 - __uint_as_float(h << 16), x1 - __uint_as_float(h & 0xffff0000u));
                        };
                        const uint4 pl = make_uint4(lo2(acc[0][ct][0], acc[0][ct][1], pk.x), lo2(acc[0][ct][2], acc[0][ct][3], pk.y),
                                                    lo2(acc[1][ct][0], acc[1][ct][1], pk.z), lo2(acc[1][ct][2], acc[1][ct][3], pk.w));
                        *reinterpret_cast<uint4*>(base + lo_plane + off) = pl;
                    }
                }
            }
            if constexpr (PLAIN) {
                float* dst = plain_base + (bh * s.n_chunks + n) * int64_t(kStateElems);
#pragma unroll
                for (int rt = 0; rt < 2; ++rt)
#pragma unroll
                    for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
                        for (int ii = 0; ii < 4; ++ii) dst[tile_off(rt, ct, ii)] = acc[rt][ct][ii];
            }
            const int b = (n - nbeg) % 2;
            dprod *= D;
#pragma unroll
            for (int rt = 0; rt < 2; ++rt)
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct) acc[rt][ct] *= D;
            // every operand of this chunk's products is read from LDS first; the products then
            // run in three batches with the staging pieces of the next chunk (into the other
            // buffer) between them, and scheduling barriers keep that order
            bf16x8 af[C / 32][2], bfh[C / 32][NCT], bfl[C / 32][NCT];
#pragma unroll
            for (int u = 0; u < C / 32; ++u) {
#pragma unroll
                for (int rt = 0; rt < 2; ++rt) af[u][rt] = lds_frag(sA[b] + (32 * sblk + 16 * rt + ln) * LDT + 32 * u + 4 * g);
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct) {
                    const int c = 16 * (lct0 + ct) + ln;
                    bfh[u][ct] = lds_frag(sBh[b] + c * LDT + 32 * u + 4 * g);
                    if (SPLIT) bfl[u][ct] = lds_frag(sBl[b] + c * LDT + 32 * u + 4 * g);
                }
            }
            auto products = [&](int u, int ct_lo, int ct_hi) {
#pragma unroll
                for (int ct = ct_lo; ct < ct_hi; ++ct)
#pragma unroll
                    for (int rt = 0; rt < 2; ++rt) {
                        acc[rt][ct] = mfma16(af[u][rt], bfh[u][ct], acc[rt][ct]);
                        if (SPLIT) acc[rt][ct] = mfma16(af[u][rt], bfl[u][ct], acc[rt][ct]);
                    }
            };
            const int bn = (n - nbeg + 1) % 2;  // a chunk past the end stages into a buffer nobody reads
            products(0, 0, NCT);
            const Gate gt = gates(Rn1);
            __builtin_amdgcn_sched_barrier(0);
            products(1, 0, NCT / 2);
            stage_k(Rn1, bn);
            stage_y(Rn1, bn, gt, 0, 4);
            __builtin_amdgcn_sched_barrier(0);
            products(1, NCT / 2, NCT);
            stage_y(Rn1, bn, gt, 4, 8);
            Dnext = gt.D;
            load(min(n + 3, nend - 1), Rfree);  // unconditional, so memory waits count statically
            __syncthreads();
        };

        constexpr int64_t kSegElems = int64_t(DK) * (DK + DV);  // one segment total, H then G
        // Segment totals are stored in this workgroup's own register order: value (rt, ct, ii)
        // of thread tid at [(rt NCT + ct) kWideThreads + tid] * 4 + ii of the half's region, so
        // the walk that adds them reads 16 contiguous bytes per value quadruple (the totals
        // launch has the walk's work split, so both see the same order)
        auto seg_total = [&](int t) -> float* { return sg.tot + (bh * (sg.total - 1) + t) * kSegElems + half * (DK * DK); };
        auto tot_at = [&](int rt, int ct) { return ((rt * NCT + ct) * kWideThreads + tid) * 4; };
        // inputs of the first three chunks (the walk keeps three chunks in flight)
        Regs R0, R1, R2;
        load(nbeg, R0);
        load(min(nbeg + 1, nend - 1), R1);
        load(min(nbeg + 2, nend - 1), R2);

        // the state entering this segment, E_seg = sum_{t < seg} c_t T_t with
        // c_t = D_{t+1} ... D_{seg-1} (the unrolled E_{t+1} = D_t E_t + T_t); the terms
        // are independent, so their loads are issued two segments at a time.  The
        // totals launch starts every segment from zero instead.
        if (!sg.totals) {
            float c[2];
            float cn = 1.0f;  // c_t for the highest t not yet added
            for (int t = seg - 1; t >= 0; t -= 2) {
                c[0] = cn;
                cn *= sg.dec[bh * sg.total + t];
                c[1] = t >= 1 ? cn : 0.0f;
                if (t >= 1) cn *= sg.dec[bh * sg.total + t - 1];
                const float* tb0 = seg_total(t);
                const float* tb1 = seg_total(t >= 1 ? t - 1 : t);
#pragma unroll
                for (int rt = 0; rt < 2; ++rt)
#pragma unroll
                    for (int ct = 0; ct < NCT; ++ct) {
                        const f32x4 v0 = *reinterpret_cast<const f32x4*>(tb0 + tot_at(rt, ct));
                        const f32x4 v1 = *reinterpret_cast<const f32x4*>(tb1 + tot_at(rt, ct));
#pragma unroll
                        for (int ii = 0; ii < 4; ++ii) acc[rt][ct][ii] += c[0] * v0[ii] + c[1] * v1[ii];
                    }
            }
        }
        float D0, D1 = 1.0f, D2 = 1.0f;
        {
            const Gate gt = gates(R0);
            stage_k(R0, 0);
            stage_y(R0, 0, gt, 0, 8);
            D0 = gt.D;
        }
        __syncthreads();
        for (int n = nbeg; n < nend; n += 3) {
            consume(n, D0, R1, R0, D1);  // stages chunk n+1 (R1), loads n+3 into R0
            if (n + 1 < nend) consume(n + 1, D1, R2, R1, D2);  // stages n+2 (R2), loads n+4 into R1
            if (n + 2 < nend) consume(n + 2, D2, R0, R2, D0);  // stages n+3 (R0), loads n+5 into R2
        }
        // fp32 output: the segment total and its decay, or, after the last segment, the
        // final states
        float* dst = nullptr;
        if (sg.totals) {
            float* tb = seg_total(seg);
#pragma unroll
            for (int rt = 0; rt < 2; ++rt)
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct) *reinterpret_cast<f32x4*>(tb + tot_at(rt, ct)) = acc[rt][ct];
            if (half == 0 && tid == 0) sg.dec[bh * sg.total + seg] = dprod;
        } else if (seg == sg.total - 1) {
            float* fin = part ? a.final_G : a.final_H;
            if (fin) dst = fin + bh * int64_t(NC) * DK;
        }
        if (dst) {
#pragma unroll
            for (int rt = 0; rt < 2; ++rt)
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
                    for (int ii = 0; ii < 4; ++ii) dst[tile_off(rt, ct, ii)] = acc[rt][ct][ii];
        }
    };
    if (BAL || half == 0)
        run(std::integral_constant<int, DK>{});
    else
        run(std::integral_constant<int, DV>{});
}

// Segments of the wide scan for bh sequences of n_chunks chunks: doubled while the
// (sequence, part, segment) workgroups still fit the compute units once (the kernel's
// LDS allows one workgroup per unit) and each segment keeps at least kMinSegChunks
// chunks, so the extra totals launch stays small next to the walk it shortens.
constexpr int kComputeUnits = 256;
constexpr int kMinSegChunks = 8;
int wide_segments(int64_t bh, int n_chunks)
{
    int S = 1;
    while (2 * bh * (2 * S) <= kComputeUnits && n_chunks / (2 * S) >= kMinSegChunks) S *= 2;
    return S;
}

template <int DK, int DV, bool STORE, bool SPLIT, bool PLAIN = false, bool X3 = false>
void launch_wide_kernel(const StateArgs& a, const SegPlan& sg, int64_t bh, hipStream_t stream)
{
    const unsigned blocks = unsigned(bh * 2 * sg.count);
    hipLaunchKernelGGL((chunk_state_wide_kernel<DK, DV, STORE, SPLIT, PLAIN, X3>), dim3(blocks), dim3(kWideThreads), 0, stream, a, sg);
}

template <int DK, int DV>
hipError_t launch_wide(const StateArgs& a, hipStream_t stream)
{
    const int64_t bh = a.s.batch * a.s.heads;
    const int nc = a.s.n_chunks;
    const bool fin = a.final_H != nullptr || a.final_G != nullptr;
    int S = wide_segments(bh, nc);
    int len = (nc + S - 1) / S;
    S = (nc + len - 1) / len;
    const int64_t tot_elems = bh * (S - 1) * int64_t(DK) * (DK + DV);
    const size_t need = size_t(tot_elems + bh * S) * sizeof(float);
    if (S > 1 && (a.seg_ws == nullptr || a.seg_bytes < need)) {
        S = 1;
        len = nc;
    }
    SegPlan sg{len, S, 0, S, false, a.seg_ws, S > 1 ? a.seg_ws + tot_elems : nullptr};
    if (S > 1) {
        // segment totals T_0 .. T_{S-2} (the last one is never needed); fp32-accurate
        // (split products) when fp32 final states come out
        // (the totals are kept in the walk's thread order, so they take the walk's product
        // form, which fixes its work split: single products only for the bf16 fragments
        // without fp32 outputs)
        SegPlan p1 = sg;
        p1.count = S - 1;
        p1.totals = true;
        const bool single = a.store_chunks && !a.x3 && a.frag && !a.Hs32 && !fin;
        if (single)
            launch_wide_kernel<DK, DV, false, false>(a, p1, bh, stream);
        else
            launch_wide_kernel<DK, DV, false, true>(a, p1, bh, stream);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (!a.store_chunks) {
        // final states only: the last segment's walk alone produces them
        sg.first = S - 1;
        sg.count = 1;
    }
    if (a.store_chunks && a.x3)  // fp32 H_c fragments, G_c high and low planes, fp32-accurate
        launch_wide_kernel<DK, DV, true, true, false, true>(a, sg, bh, stream);
    else if (a.store_chunks && a.frag && a.Hs32)  // fragments and fp32 plain states, fp32-accurate
        launch_wide_kernel<DK, DV, true, true, true>(a, sg, bh, stream);
    else if (a.store_chunks && a.frag && !fin)
        launch_wide_kernel<DK, DV, true, false>(a, sg, bh, stream);
    else if (a.store_chunks && a.frag)
        launch_wide_kernel<DK, DV, true, true>(a, sg, bh, stream);
    else
        launch_wide_kernel<DK, DV, false, true>(a, sg, bh, stream);
    return hipGetLastError();
}

__global__ __launch_bounds__(kThreads) void fill_zero_kernel(float* dst, int64_t n)
{
    const int64_t stride = int64_t(gridDim.x) * kThreads;
    for (int64_t i = int64_t(blockIdx.x) * kThreads + threadIdx.x; i < n; i += stride) dst[i] = 0.0f;
}

}  // namespace

hipError_t launch_fill_zero(float* dst, int64_t n, hipStream_t stream)
{
    if (n <= 0) return hipSuccess;
    const int64_t want = (n + kThreads - 1) / kThreads;
    const unsigned blocks = unsigned(want < 4096 ? want : 4096);
    hipLaunchKernelGGL(fill_zero_kernel, dim3(blocks), dim3(kThreads), 0, stream, dst, n);
    return hipGetLastError();
}

bool chunk_state_frag_supported(const ForwardShape& s)
{
    return s.bf16 && s.chunk == 64 && (s.d_k == 64 || s.d_k == 128) && (s.d_v == 64 || s.d_v == 128);
}

hipError_t launch_chunk_state(const StateArgs& a, hipStream_t stream)
{
    const int64_t bh = a.s.batch * a.s.heads;
    if ((a.frag || a.x3) && !chunk_state_frag_supported(a.s)) return hipErrorInvalidValue;
    if (chunk_state_frag_supported(a.s) && (a.frag || a.x3 || !a.store_chunks)) {
        if (a.s.d_k == 64) return a.s.d_v == 64 ? launch_wide<64, 64>(a, stream) : launch_wide<64, 128>(a, stream);
        return a.s.d_v == 64 ? launch_wide<128, 64>(a, stream) : launch_wide<128, 128>(a, stream);
    }
    if (!a.s.bf16 && a.s.chunk == 64) {
        const unsigned blocks = unsigned(bh * ((a.s.d_k + a.s.d_v) / 16) * (a.s.d_k / 64));
        auto kern = a.s.d_k == 64 ? (a.store_chunks ? chunk_state_f32_kernel<64, true> : chunk_state_f32_kernel<64, false>)
                                  : (a.store_chunks ? chunk_state_f32_kernel<128, true> : chunk_state_f32_kernel<128, false>);
        hipLaunchKernelGGL(kern, dim3(blocks), dim3(kThreads), 0, stream, a);
        return hipGetLastError();
    }
    if (a.s.bf16 && a.s.chunk == 64) {
        const unsigned blocks = unsigned(bh * ((a.s.d_k + a.s.d_v) / 64) * (a.s.d_k / 32));
        hipLaunchKernelGGL(chunk_state_mfma_kernel, dim3(blocks), dim3(kThreads), 0, stream, a);
        return hipGetLastError();
    }
    const int64_t blocks = bh * ((a.s.d_k + a.s.d_v) / kTileRows);
    if (a.s.bf16)
        hipLaunchKernelGGL(chunk_state_kernel<bf16_t>, dim3(unsigned(blocks)), dim3(kThreads), 0,
                           stream, a);
    else
        hipLaunchKernelGGL(chunk_state_kernel<float>, dim3(unsigned(blocks)), dim3(kThreads), 0,
                           stream, a);
    return hipGetLastError();
}

}  // namespace mesa
