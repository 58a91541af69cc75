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
// Both are HBM-bound elementwise passes, written so that every lane moves 16 bytes
// per access: a token row of d channels is d / c lanes (c = 8 bf16 or 4 fp32 channels
// per lane), so a wave holds 64 c / d tokens side by side, and each such group of
// lanes walks its own run of kSub consecutive tokens of one (sequence, head).  The
// per-token sums over the channels are reductions within a group.  The convolution
// keeps the previous three tokens of the lane's channels in registers while walking
// the run (the three tokens before the run are read once as its halo).  Tokens are
// loaded kBatch at a time so that several loads are in flight per lane.
#include <type_traits>

#include "mesa_device.hpp"
#include "mesa_kernels.hpp"

namespace mesa {
namespace {

constexpr int kThreads = 256;
constexpr int kSub = 16;    // tokens per group of lanes
constexpr int kBatch = 8;   // tokens loaded together

__device__ __forceinline__ float sigmoid_f(float x) { return 1.0f / (1.0f + __expf(-x)); }

// softplus(x) = max(x, 0) + log(1 + exp(-|x|))
__device__ __forceinline__ float softplus_f(float x) { return fmaxf(x, 0.0f) + log1pf(__expf(-fabsf(x))); }

// round to nearest even (finite inputs), bf16 bits
__device__ __forceinline__ uint32_t bf16_rne(float x)
{
    const uint32_t u = __float_as_uint(x);
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

// 16 bytes of channels <-> fp32: 8 bf16 or 4 fp32 per lane
template <typename T>
struct Vec;
template <>
struct Vec<bf16_t> {
    static constexpr int N = 8;
    __device__ static void unpack(const uint4& v, float (&x)[8])
    {
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            x[2 * q] = __uint_as_float(w[q] << 16);
            x[2 * q + 1] = __uint_as_float(w[q] & 0xffff0000u);
        }
    }
    __device__ static uint4 pack(const float (&y)[8])
    {
        uint32_t w[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) w[q] = bf16_rne(y[2 * q]) | (bf16_rne(y[2 * q + 1]) << 16);
        return make_uint4(w[0], w[1], w[2], w[3]);
    }
};
template <>
struct Vec<float> {
    static constexpr int N = 4;
    __device__ static void unpack(const uint4& v, float (&x)[4])
    {
        x[0] = __uint_as_float(v.x);
        x[1] = __uint_as_float(v.y);
        x[2] = __uint_as_float(v.z);
        x[3] = __uint_as_float(v.w);
    }
    __device__ static uint4 pack(const float (&y)[4])
    {
        return make_uint4(__float_as_uint(y[0]), __float_as_uint(y[1]), __float_as_uint(y[2]), __float_as_uint(y[3]));
    }
};

// Sum over the L consecutive lanes of a group (L a power of two up to 64); every lane
// of the group receives it.
template <int L>
__device__ __forceinline__ float group_sum(float v)
{
#pragma unroll
    for (int m = L / 2; m >= 1; m /= 2) v += __shfl_xor(v, m);
    return v;
}

// Tokens one wave covers for a tensor of D channels of type T.
template <typename T, int D>
constexpr int wave_tokens()
{
    return (kWave / (D / Vec<T>::N)) * kSub;
}

// One tensor of the front end: kind 0 = q, 1 = k (convolution, SiLU, unit norm),
// 2 = v (convolution and SiLU if a filter is given).  Wave `item` of the tensor's
// B * H * ceil(T / wave_tokens) items.
template <typename Tin, int D>
__device__ void frontend_tensor(const FrontArgs& a, int kind, int64_t item)
{
    constexpr int C = Vec<Tin>::N;  // channels per lane
    constexpr int LPT = D / C;      // lanes per token
    constexpr int WT = wave_tokens<Tin, D>();
    const int lane = threadIdx.x % kWave;
    const int grp = lane / LPT, cl = lane % LPT;
    const int64_t runs = (a.seq_len + WT - 1) / WT;
    const int64_t bh = item / runs;
    const int64_t t0 = (item % runs) * WT + int64_t(grp) * kSub;  // this group's first token
    const int64_t t_end = min<int64_t>(t0 + kSub, a.seq_len);     // may be <= t0: idle group
    const int64_t b = bh / a.heads, h = bh % a.heads;
    const Tin* src = static_cast<const Tin*>(kind == 0 ? a.qp : kind == 1 ? a.kp : a.vp);
    Tin* dst = static_cast<Tin*>(kind == 0 ? a.q : kind == 1 ? a.k : a.v);
    const float* w = kind == 0 ? a.conv_q : kind == 1 ? a.conv_k : a.conv_v;
    const bool conv = w != nullptr;
    const bool norm = kind < 2;
    const int64_t row_stride = a.heads * D;  // elements between consecutive tokens of a head
    const Tin* in = src + b * a.seq_len * row_stride + h * D + cl * C;
    Tin* out = dst + bh * a.seq_len * D + cl * C;
    float wt[C][4];
    float prev[C][3];  // x_{t-1}, x_{t-2}, x_{t-3}
#pragma unroll
    for (int c = 0; c < C; ++c) {
        if (conv) {
            const float4 f = *reinterpret_cast<const float4*>(w + (h * D + cl * C + c) * 4);
            wt[c][0] = f.x;
            wt[c][1] = f.y;
            wt[c][2] = f.z;
            wt[c][3] = f.w;
        } else {
            wt[c][0] = wt[c][1] = wt[c][2] = wt[c][3] = 0.0f;
        }
        prev[c][0] = prev[c][1] = prev[c][2] = 0.0f;
    }
    if (conv) {
#pragma unroll
        for (int i = 0; i < 3; ++i) {
            const int64_t t = t0 - 1 - i;
            if (t >= 0 && t < a.seq_len) {
                float x[C];
                Vec<Tin>::unpack(*reinterpret_cast<const uint4*>(in + t * row_stride), x);
#pragma unroll
                for (int c = 0; c < C; ++c) prev[c][i] = x[c];
            }
        }
    }
    // Every group runs all kSub steps (the group sums need every lane); a step past the
    // group's last token re-reads that token (or the sequence's first) and stores nothing.
    const int64_t t_last = max<int64_t>(min<int64_t>(t_end, a.seq_len) - 1, 0);
#pragma unroll 1
    for (int s0 = 0; s0 < kSub; s0 += kBatch) {
        uint4 xv[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            const int64_t t = min<int64_t>(t0 + s0 + u, t_last);
            xv[u] = *reinterpret_cast<const uint4*>(in + t * row_stride);
        }
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            const int64_t t = t0 + s0 + u;
            float x[C], y[C];
            Vec<Tin>::unpack(xv[u], x);
            float ss = 0.0f;
#pragma unroll
            for (int c = 0; c < C; ++c) {
                if (conv) {
                    float sc = wt[c][0] * x[c];
                    sc = fmaf(wt[c][1], prev[c][0], sc);
                    sc = fmaf(wt[c][2], prev[c][1], sc);
                    sc = fmaf(wt[c][3], prev[c][2], sc);
                    prev[c][2] = prev[c][1];
                    prev[c][1] = prev[c][0];
                    prev[c][0] = x[c];
                    y[c] = sc * sigmoid_f(sc);
                } else {
                    y[c] = x[c];
                }
                ss = fmaf(y[c], y[c], ss);
            }
            if (norm) {
                const float inv = rsqrtf(group_sum<LPT>(ss) + a.l2_eps);
#pragma unroll
                for (int c = 0; c < C; ++c) y[c] *= inv;
            }
            if (t < t_end) *reinterpret_cast<uint4*>(out + t * D) = Vec<Tin>::pack(y);
        }
    }
}

template <typename Tin, int DK, int DV>
__global__ __launch_bounds__(kThreads) void frontend_kernel(FrontArgs a, int64_t nqk, int64_t nv, int64_t n_gate_blocks)
{
    const int64_t blk = blockIdx.x;
    const int wave = threadIdx.x / kWave;
    constexpr int kWavesPerBlock = kThreads / kWave;
    const int64_t bh_all = a.batch * a.heads;
    if (blk < 2 * nqk + nv) {
        const int kind = blk < nqk ? 0 : blk < 2 * nqk ? 1 : 2;
        const int64_t item = (blk - (kind < 2 ? kind * nqk : 2 * nqk)) * kWavesPerBlock + wave;
        if (kind < 2) {
            constexpr int WT = wave_tokens<Tin, DK>();
            if (item < bh_all * ((a.seq_len + WT - 1) / WT)) frontend_tensor<Tin, DK>(a, kind, item);
        } else {
            constexpr int WT = wave_tokens<Tin, DV>();
            if (item < bh_all * ((a.seq_len + WT - 1) / WT)) frontend_tensor<Tin, DV>(a, kind, item);
        }
        return;
    }
    const int64_t gb = blk - 2 * nqk - nv;
    if (gb < n_gate_blocks) {
        // gates, one thread per (b, h, t) of the output (consecutive threads: consecutive t)
        const int64_t i = gb * kThreads + threadIdx.x;
        const int64_t n = bh_all * a.seq_len;
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

// Per-head RMSNorm: o [B, H, T, d_v] fp32 (4 channels per lane) -> y [B, T, H, d_v].
template <typename Tout, int DV>
__global__ __launch_bounds__(kThreads) void output_norm_kernel(NormArgs a)
{
    constexpr int C = 4;
    constexpr int LPT = DV / C;
    constexpr int WT = wave_tokens<float, DV>();
    const int lane = threadIdx.x % kWave;
    const int grp = lane / LPT, cl = lane % LPT;
    const int64_t runs = (a.seq_len + WT - 1) / WT;
    const int64_t item = int64_t(blockIdx.x) * (kThreads / kWave) + threadIdx.x / kWave;
    if (item >= a.batch * a.heads * runs) return;
    const int64_t bh = item / runs;
    const int64_t t0 = (item % runs) * WT + int64_t(grp) * kSub;
    const int64_t t_end = min<int64_t>(t0 + kSub, a.seq_len);
    const int64_t t_last = max<int64_t>(t_end - 1, 0);
    const int64_t b = bh / a.heads, h = bh % a.heads;
    const float4 wt = *reinterpret_cast<const float4*>(a.weight + h * DV + cl * C);
    const float* in = a.o + bh * a.seq_len * DV + cl * C;
    Tout* out = static_cast<Tout*>(a.y) + (b * a.seq_len * a.heads + h) * DV + cl * C;
    const float inv_d = 1.0f / DV;
#pragma unroll 1
    for (int s0 = 0; s0 < kSub; s0 += kBatch) {
        float4 xv[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u)
            xv[u] = *reinterpret_cast<const float4*>(in + min<int64_t>(t0 + s0 + u, t_last) * DV);
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            const int64_t t = t0 + s0 + u;
            const float4 x = xv[u];
            const float ss = x.x * x.x + x.y * x.y + x.z * x.z + x.w * x.w;
            const float inv = rsqrtf(group_sum<LPT>(ss) * inv_d + a.eps);
            const float y0 = x.x * inv * wt.x, y1 = x.y * inv * wt.y, y2 = x.z * inv * wt.z, y3 = x.w * inv * wt.w;
            if (t < t_end) {
                Tout* o = out + t * a.heads * DV;
                if constexpr (std::is_same<Tout, float>::value)
                    *reinterpret_cast<float4*>(o) = make_float4(y0, y1, y2, y3);
                else
                    *reinterpret_cast<uint2*>(o) = make_uint2(bf16_rne(y0) | (bf16_rne(y1) << 16), bf16_rne(y2) | (bf16_rne(y3) << 16));
            }
        }
    }
}

template <typename Tin, int DK, int DV>
hipError_t launch_front(const FrontArgs& a, hipStream_t stream)
{
    constexpr int per = kThreads / kWave;
    constexpr int WK = wave_tokens<Tin, DK>(), WV = wave_tokens<Tin, DV>();
    const int64_t bh = a.batch * a.heads;
    const int64_t nqk = (bh * ((a.seq_len + WK - 1) / WK) + per - 1) / per;
    const int64_t nv = (bh * ((a.seq_len + WV - 1) / WV) + per - 1) / per;
    const int64_t gbk = (bh * a.seq_len + kThreads - 1) / kThreads;
    const int64_t lbk = (a.heads * DK + kThreads - 1) / kThreads;
    const int64_t blocks = 2 * nqk + nv + gbk + lbk;
    if (blocks > INT32_MAX) return hipErrorInvalidValue;
    hipLaunchKernelGGL((frontend_kernel<Tin, DK, DV>), dim3(unsigned(blocks)), dim3(kThreads), 0, stream, a, nqk, nv, gbk);
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
    constexpr int WT = wave_tokens<float, DV>();
    const int64_t items = a.batch * a.heads * ((a.seq_len + WT - 1) / WT);
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
