// The Mesa layer's front and back end (App. E, "A Full Description of the Mesa
// Layer"; the gate cap and the Lambda floor of App. G.5), each one fused launch.
//
// Front end, per head, from the projections of a token (the heads side by side,
// [B, T, H, d], as a projection produces them):
//   q, k:  x_t <- sum_{i=0..3} w_{i+1} x_{t-i}  (window-4 causal convolution in time,
//          one filter per channel, zeros before the sequence start), SiLU(x) = x sigma(x),
//          then x / sqrt(|x|^2 + eps)                       -> [B, H, T, d_k]
//   v:     the same convolution and SiLU when a filter is given, else unchanged
//                                                           -> [B, H, T, d_v]
//   beta_t = sigma(a_t^beta),  gamma_t = sigma(a_t^gamma) (1 - (1 - b_gamma) beta_t^2)
//                                                           -> [B, H, T]
//   Lambda = 0.25 + softplus(theta)                         -> [H, d_k]
// Back end: y_t = o_t / sqrt(mean(o_t^2) + eps) w_h, the head's RMSNorm before the
// output projection, [B, H, T, d_v] -> [B, T, H, d_v].
//
// Both are HBM-bound elementwise passes.  A wave owns one (sequence, head) and a run of
// kRun consecutive tokens; lane l holds channels l, l + 64 (d = 128) or l (d = 64) of
// a token, so every token row is one coalesced wave access on both sides, and the
// per-token sums over the channels are wave reductions.  The convolution keeps the
// previous three tokens of its channels in registers, walking the run in order (the
// three tokens before the run are read once as its halo).  Tokens are read in groups
// of kGroup so that several loads are in flight per wave.
#include "mesa_device.hpp"
#include "mesa_kernels.hpp"

namespace mesa {
namespace {

constexpr int kThreads = 256;
constexpr int kRun = 64;    // tokens per wave
constexpr int kGroup = 8;   // tokens loaded together

template <typename T>
__device__ __forceinline__ T from_f32(float x);
template <>
__device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <>
__device__ __forceinline__ bf16_t from_f32<bf16_t>(float x)
{
    // round to nearest even (finite inputs)
    const uint32_t u = __float_as_uint(x);
    return bf16_t{uint16_t((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16)};
}

__device__ __forceinline__ float sigmoid_f(float x) { return 1.0f / (1.0f + __expf(-x)); }

// softplus(x) = max(x, 0) + log(1 + exp(-|x|))
__device__ __forceinline__ float softplus_f(float x) { return fmaxf(x, 0.0f) + log1pf(__expf(-fabsf(x))); }

// One tensor of the front end: kind 0 = q, 1 = k (convolution, SiLU, unit norm),
// 2 = v (convolution and SiLU if w != nullptr).  Wave `item` of the tensor's
// B * H * ceil(T / kRun) items.
template <typename Tin, int D>
__device__ void frontend_tensor(const FrontArgs& a, int kind, int64_t item)
{
    constexpr int NCH = D / kWave;  // channels per lane
    const int lane = threadIdx.x % kWave;
    const int64_t runs = (a.seq_len + kRun - 1) / kRun;
    const int64_t bh = item / runs;
    const int64_t t0 = (item % runs) * kRun;
    const int64_t b = bh / a.heads, h = bh % a.heads;
    const Tin* src = static_cast<const Tin*>(kind == 0 ? a.qp : kind == 1 ? a.kp : a.vp);
    Tin* dst = static_cast<Tin*>(kind == 0 ? a.q : kind == 1 ? a.k : a.v);
    const float* w = kind == 0 ? a.conv_q : kind == 1 ? a.conv_k : a.conv_v;
    const bool conv = w != nullptr;
    const bool norm = kind < 2;
    const int64_t row_stride = a.heads * D;  // elements between consecutive tokens of a head
    const Tin* in = src + b * a.seq_len * row_stride + h * D;
    Tin* out = dst + (bh * a.seq_len) * D;
    float wt[NCH][4];
    float prev[NCH][3];  // x_{t-1}, x_{t-2}, x_{t-3}
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        const int ch = c * kWave + lane;
#pragma unroll
        for (int i = 0; i < 4; ++i) wt[c][i] = conv ? w[(h * D + ch) * 4 + i] : 0.0f;
#pragma unroll
        for (int i = 0; i < 3; ++i) {
            const int64_t t = t0 - 1 - i;
            prev[c][i] = (conv && t >= 0) ? to_f32(in[t * row_stride + ch]) : 0.0f;
        }
    }
    const int64_t t_end = min<int64_t>(t0 + kRun, a.seq_len);
    for (int64_t tg = t0; tg < t_end; tg += kGroup) {
        float xg[kGroup][NCH];
#pragma unroll
        for (int u = 0; u < kGroup; ++u) {
            const int64_t t = min<int64_t>(tg + u, t_end - 1);  // past the end: re-read, not stored
#pragma unroll
            for (int c = 0; c < NCH; ++c) xg[u][c] = to_f32(in[t * row_stride + c * kWave + lane]);
        }
#pragma unroll
        for (int u = 0; u < kGroup; ++u) {
            if (tg + u >= t_end) break;  // wave-uniform
            float y[NCH];
            float ss = 0.0f;
#pragma unroll
            for (int c = 0; c < NCH; ++c) {
                const float x = xg[u][c];
                if (conv) {
                    float s = wt[c][0] * x;
                    s = fmaf(wt[c][1], prev[c][0], s);
                    s = fmaf(wt[c][2], prev[c][1], s);
                    s = fmaf(wt[c][3], prev[c][2], s);
                    prev[c][2] = prev[c][1];
                    prev[c][1] = prev[c][0];
                    prev[c][0] = x;
                    y[c] = s * sigmoid_f(s);
                } else {
                    y[c] = x;
                }
                ss = fmaf(y[c], y[c], ss);
            }
            if (norm) {
                const float inv = rsqrtf(wave_sum(ss) + a.l2_eps);
#pragma unroll
                for (int c = 0; c < NCH; ++c) y[c] *= inv;
            }
            const int64_t t = tg + u;
#pragma unroll
            for (int c = 0; c < NCH; ++c) out[t * D + c * kWave + lane] = from_f32<Tin>(y[c]);
        }
    }
}

template <typename Tin, int DK, int DV>
__global__ __launch_bounds__(kThreads) void frontend_kernel(FrontArgs a, int64_t n_tensor_blocks,
                                                            int64_t n_gate_blocks)
{
    const int64_t blk = blockIdx.x;
    const int wave = threadIdx.x / kWave;
    const int64_t runs = (a.seq_len + kRun - 1) / kRun;
    const int64_t items = a.batch * a.heads * runs;
    if (blk < 3 * n_tensor_blocks) {
        const int kind = int(blk / n_tensor_blocks);
        const int64_t item = (blk % n_tensor_blocks) * (kThreads / kWave) + wave;
        if (item >= items) return;
        if (kind < 2)
            frontend_tensor<Tin, DK>(a, kind, item);
        else
            frontend_tensor<Tin, DV>(a, kind, item);
        return;
    }
    const int64_t gb = blk - 3 * n_tensor_blocks;
    if (gb < n_gate_blocks) {
        // gates, one thread per (b, h, t) of the output (consecutive threads: consecutive t)
        const int64_t i = gb * kThreads + threadIdx.x;
        const int64_t n = a.batch * a.heads * a.seq_len;
        if (i >= n) return;
        const int64_t t = i % a.seq_len, bh = i / a.seq_len;
        const int64_t b = bh / a.heads, h = bh % a.heads;
        const int64_t src = (b * a.seq_len + t) * a.heads + h;
        const float beta = sigmoid_f(a.a_beta[src]);
        a.beta[i] = beta;
        a.gamma[i] = sigmoid_f(a.a_gamma[src]) * (1.0f - (1.0f - a.gamma_cap) * beta * beta);
        return;
    }
    // Lambda = 0.25 + softplus(theta)
    const int64_t i = (gb - n_gate_blocks) * kThreads + threadIdx.x;
    if (i < a.heads * DK) a.lambda[i] = 0.25f + softplus_f(a.theta[i]);
}

template <typename Tout, int DV>
__global__ __launch_bounds__(kThreads) void output_norm_kernel(NormArgs a)
{
    constexpr int NCH = DV / kWave;
    const int lane = threadIdx.x % kWave;
    const int64_t runs = (a.seq_len + kRun - 1) / kRun;
    const int64_t item = int64_t(blockIdx.x) * (kThreads / kWave) + threadIdx.x / kWave;
    if (item >= a.batch * a.heads * runs) return;
    const int64_t bh = item / runs;
    const int64_t t0 = (item % runs) * kRun;
    const int64_t b = bh / a.heads, h = bh % a.heads;
    float wt[NCH];
#pragma unroll
    for (int c = 0; c < NCH; ++c) wt[c] = a.weight[h * DV + c * kWave + lane];
    const float* in = a.o + bh * a.seq_len * DV;
    Tout* out = static_cast<Tout*>(a.y) + (b * a.seq_len * a.heads + h) * DV;
    const int64_t t_end = min<int64_t>(t0 + kRun, a.seq_len);
    for (int64_t tg = t0; tg < t_end; tg += kGroup) {
        float xg[kGroup][NCH];
#pragma unroll
        for (int u = 0; u < kGroup; ++u) {
            const int64_t t = min<int64_t>(tg + u, t_end - 1);
#pragma unroll
            for (int c = 0; c < NCH; ++c) xg[u][c] = in[t * DV + c * kWave + lane];
        }
#pragma unroll
        for (int u = 0; u < kGroup; ++u) {
            if (tg + u >= t_end) break;  // wave-uniform
            float ss = 0.0f;
#pragma unroll
            for (int c = 0; c < NCH; ++c) ss = fmaf(xg[u][c], xg[u][c], ss);
            const float inv = rsqrtf(wave_sum(ss) * (1.0f / DV) + a.eps);
            const int64_t t = tg + u;
#pragma unroll
            for (int c = 0; c < NCH; ++c)
                out[t * a.heads * DV + c * kWave + lane] = from_f32<Tout>(xg[u][c] * inv * wt[c]);
        }
    }
}

template <typename Tin, int DK, int DV>
hipError_t launch_front(const FrontArgs& a, hipStream_t stream)
{
    const int64_t runs = (a.seq_len + kRun - 1) / kRun;
    const int64_t items = a.batch * a.heads * runs;
    const int64_t per = kThreads / kWave;
    const int64_t tb = (items + per - 1) / per;
    const int64_t gbk = (a.batch * a.heads * a.seq_len + kThreads - 1) / kThreads;
    const int64_t lbk = (a.heads * DK + kThreads - 1) / kThreads;
    const int64_t blocks = 3 * tb + gbk + lbk;
    if (blocks > INT32_MAX) return hipErrorInvalidValue;
    hipLaunchKernelGGL((frontend_kernel<Tin, DK, DV>), dim3(unsigned(blocks)), dim3(kThreads), 0, stream, a, tb, gbk);
    return hipGetLastError();
}

template <typename Tin>
hipError_t launch_front_dims(const FrontArgs& a, hipStream_t stream)
{
    if (a.d_k == 64) return a.d_v == 64 ? launch_front<Tin, 64, 64>(a, stream) : launch_front<Tin, 64, 128>(a, stream);
    return a.d_v == 64 ? launch_front<Tin, 128, 64>(a, stream) : launch_front<Tin, 128, 128>(a, stream);
}

template <typename Tout, int DV>
hipError_t launch_norm(const NormArgs& a, hipStream_t stream)
{
    const int64_t runs = (a.seq_len + kRun - 1) / kRun;
    const int64_t items = a.batch * a.heads * runs;
    const int64_t per = kThreads / kWave;
    const int64_t blocks = (items + per - 1) / per;
    if (blocks > INT32_MAX) return hipErrorInvalidValue;
    hipLaunchKernelGGL((output_norm_kernel<Tout, DV>), dim3(unsigned(blocks)), dim3(kThreads), 0, stream, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_frontend(const FrontArgs& a, hipStream_t stream)
{
    if (a.heads == 0) return hipSuccess;  // otherwise Lambda is written even without tokens
    return a.bf16 ? launch_front_dims<bf16_t>(a, stream) : launch_front_dims<float>(a, stream);
}

hipError_t launch_output_norm(const NormArgs& a, hipStream_t stream)
{
    if (a.batch * a.heads * a.seq_len == 0) return hipSuccess;
    if (a.d_v == 64) return a.bf16_out ? launch_norm<bf16_t, 64>(a, stream) : launch_norm<float, 64>(a, stream);
    return a.bf16_out ? launch_norm<bf16_t, 128>(a, stream) : launch_norm<float, 128>(a, stream);
}

}  // namespace mesa
