// Recurrent decode step of the Mesa layer (Sec. 3, recurrent inference mode;
// App. C, last paragraph: at inference CG runs on H_t + Lambda directly).
// One workgroup per (sequence, head):
//   1. H <- gamma H + beta k k^T, written back in place; H + Lambda kept in LDS.
//   2. n_cg iterations of Alg. 1 (tolerance 0) on (H + Lambda) x = q, each
//      product a GEMV from LDS.
//   3. G <- gamma G + beta v k^T streamed through registers and written back,
//      with o = G x formed on the way.
// All arithmetic is fp32.  The step is bound by HBM: each (sequence, head)
// reads and writes its two fp32 states, 8 (d_k + d_v) d_k bytes.
#include "mesa_device.hpp"
#include "mesa_kernels.hpp"

namespace mesa {
namespace {

constexpr int kThreads = 256;

template <typename Tin, int DK>
__global__ __launch_bounds__(kThreads) void decode_step_kernel(DecodeArgs a)
{
    constexpr int TPR = kThreads / DK;  // threads per row of H in a GEMV
    constexpr int LDA = DK + 1;
    const int64_t pair = blockIdx.x;
    const int h = int(pair % a.heads);
    const int dv = a.d_v;
    const int tid = threadIdx.x;

    __shared__ float sA[DK * LDA];
    __shared__ float sk[DK], sq[DK], sv[128], sx[DK], sp[DK];
    __shared__ float sRed[kThreads / kWave];
    __shared__ float sO[128 * (DK / kWave)];

    const Tin* qp = static_cast<const Tin*>(a.q) + pair * DK;
    const Tin* kp = static_cast<const Tin*>(a.k) + pair * DK;
    const Tin* vp = static_cast<const Tin*>(a.v) + pair * dv;
    const float* lam = a.lambda + int64_t(h) * DK;
    if (tid < DK) {
        sk[tid] = to_f32(kp[tid]);
        sq[tid] = to_f32(qp[tid]);
    }
    if (tid < dv) sv[tid] = to_f32(vp[tid]);
    const float g = a.gamma[pair], bt = a.beta[pair];
    __syncthreads();

    float* H = a.H + pair * DK * DK;
    for (int e = tid; e < DK * DK; e += kThreads) {
        const int rr = e / DK, c = e % DK;
        const float hn = g * H[e] + bt * sk[rr] * sk[c];
        H[e] = hn;
        sA[rr * LDA + c] = hn + (rr == c ? lam[rr] : 0.0f);
    }
    __syncthreads();

    const int row = tid / TPR, part = tid % TPR;
    auto gemv = [&](const float* vec) -> float {
        float acc = 0.0f;
        for (int b = part; b < DK; b += TPR) acc += sA[row * LDA + b] * vec[b];
#pragma unroll
        for (int off = TPR / 2; off >= 1; off >>= 1) acc += __shfl_xor(acc, off, kWave);
        return acc;
    };
    // Sum of one value per row (the TPR copies of a row count once).
    auto rowsum = [&](float v) -> float {
        v = wave_sum(part == 0 ? v : 0.0f);
        if ((tid & (kWave - 1)) == 0) sRed[tid / kWave] = v;
        __syncthreads();
        float t = 0.0f;
#pragma unroll
        for (int w = 0; w < kThreads / kWave; ++w) t += sRed[w];
        __syncthreads();
        return t;
    };

    const float qv = sq[row];
    float x = qv / sA[row * LDA + row];
    if (part == 0) sx[row] = x;
    __syncthreads();
    float r = qv - gemv(sx);
    float p = r;
    float delta = rowsum(r * r);
    if (delta > 0.0f) {
        for (int it = 0; it < a.n_cg; ++it) {
            if (part == 0) sp[row] = p;
            __syncthreads();
            const float w = gemv(sp);
            const float pw = rowsum(p * w);
            if (!(pw > 0.0f)) break;
            const float alpha = delta / pw;
            x += alpha * p;
            r -= alpha * w;
            const float dn = rowsum(r * r);
            if (dn == 0.0f) break;
            p = r + (dn / delta) * p;
            delta = dn;
        }
    }
    if (part == 0) sx[row] = x;
    __syncthreads();

    float* G = a.G + pair * int64_t(dv) * DK;
    for (int e = tid; e < dv * DK; e += kThreads) {
        const int rr = e / DK, c = e % DK;
        const float gn = g * G[e] + bt * sv[rr] * sk[c];
        G[e] = gn;
        const float s = wave_sum(gn * sx[c]);
        if ((tid & (kWave - 1)) == 0) sO[rr * (DK / kWave) + c / kWave] = s;
    }
    __syncthreads();
    if (tid < dv) {
        float o = 0.0f;
#pragma unroll
        for (int u = 0; u < DK / kWave; ++u) o += sO[tid * (DK / kWave) + u];
        a.out[pair * dv + tid] = o;
    }
}

template <typename Tin>
hipError_t launch_tin(const DecodeArgs& a, hipStream_t stream)
{
    const unsigned blocks = unsigned(a.batch * a.heads);
    if (a.d_k == 64)
        hipLaunchKernelGGL((decode_step_kernel<Tin, 64>), dim3(blocks), dim3(kThreads), 0, stream, a);
    else
        hipLaunchKernelGGL((decode_step_kernel<Tin, 128>), dim3(blocks), dim3(kThreads), 0, stream, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_decode_step(const DecodeArgs& a, hipStream_t stream)
{
    return a.bf16 ? launch_tin<bf16_t>(a, stream) : launch_tin<float>(a, stream);
}

}  // namespace mesa
