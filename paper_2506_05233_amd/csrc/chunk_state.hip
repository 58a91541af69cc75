// Chunk-state scan of the Mesa layer (App. D, chunkwise form): the states
// entering every chunk, H_c and G_c for c = 0, C, 2C, ...
//
//   H_{c+C} = zeta_{c+C,c} H_c + sum_{i in chunk} zeta_{c+C,i} beta_i k_i k_i^T
//   G_{c+C} = zeta_{c+C,c} G_c + sum_{i in chunk} zeta_{c+C,i} beta_i v_i k_i^T
//
// (the gated recurrences of Sec. 3 summed over one chunk, unrolled as in App. D).
// One workgroup owns a 16-row tile of H or of G for one (batch, head) and
// walks the chunks in order, so every state element is written exactly once per
// chunk with coalesced stores.  The tile stays in registers between chunks.
// HBM traffic per token-head: the states, 4 (d_k + d_v) d_k / C bytes, plus the
// chunk's k and v, read once per tile.
#include "mesa_device.hpp"
#include "mesa_kernels.hpp"

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
    const int tile = blockIdx.x % ntile;
    const int64_t bh = blockIdx.x / ntile;
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

    float* chunk_dst = isG ? a.Gs : a.Hs;
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

hipError_t launch_chunk_state(const StateArgs& a, hipStream_t stream)
{
    const int64_t bh = a.s.batch * a.s.heads;
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
