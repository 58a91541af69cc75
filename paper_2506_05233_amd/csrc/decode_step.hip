// Recurrent decode step of the Mesa layer (Sec. 3, recurrent inference mode;
// App. C, last paragraph: at inference CG runs on H_t + Lambda directly).
//
// One 64-lane wave per (sequence, head); the step is bound by HBM, since each
// pair reads and writes its two fp32 states (8 (d_k + d_v) d_k bytes).
//   1. H <- gamma H + beta k k^T.  Lane l keeps rows R(l) = {l, l + 64, ...}
//      of H in registers.  H is symmetric, so row r is read as column r,
//      H[c][r] for c = 0..d_k-1, which makes every load and store one
//      contiguous 256-byte wave access; the updated column is written back
//      in place.
//   2. Alg. 1 with tolerance 0 on (H + Lambda) x = q: each product is a
//      register-resident GEMV against p broadcast through LDS; the CG scalars
//      are wave reductions, so no barrier beyond the wave is needed.
//   3. Lane l streams rows R(l) of G through registers: G <- gamma G +
//      beta v k^T, written back, and o_e = sum_b G[e][b] x_b formed per row.
// All arithmetic is fp32.
#include "mesa_device.hpp"
#include "mesa_kernels.hpp"

namespace mesa {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

template <typename Tin, int DK, int DV>
__global__ __launch_bounds__(kWave) void decode_step_kernel(DecodeArgs a)
{
    constexpr int RH = DK / kWave;  // rows of H per lane
    constexpr int RG = DV / kWave;  // rows of G per lane
    const int64_t pair = blockIdx.x;
    const int h = int(pair % a.heads);
    const int lane = threadIdx.x;

    __shared__ __attribute__((aligned(16))) float sk[DK];
    __shared__ __attribute__((aligned(16))) float sp[DK];

    const Tin* qp = static_cast<const Tin*>(a.q) + pair * DK;
    const Tin* kp = static_cast<const Tin*>(a.k) + pair * DK;
    const Tin* vp = static_cast<const Tin*>(a.v) + pair * DV;
    const float* lam = a.lambda + int64_t(h) * DK;
    const float gam = a.gamma[pair], bet = a.beta[pair];

    float kr[RH], qr[RH], lr[RH], vr[RG];
#pragma unroll
    for (int u = 0; u < RH; ++u) {
        const int r = lane + kWave * u;
        kr[u] = to_f32(kp[r]);
        qr[u] = to_f32(qp[r]);
        lr[u] = lam[r];
        sk[r] = kr[u];
    }
#pragma unroll
    for (int u = 0; u < RG; ++u) vr[u] = to_f32(vp[lane + kWave * u]);
    __syncthreads();

    // ---- 1. state update of H, rows R(lane) held as hrow[u][c]
    float* Hp = a.H + pair * DK * DK;
    float hrow[RH][DK];
    float hdiag[RH];
#pragma unroll
    for (int c = 0; c < DK; ++c)
#pragma unroll
        for (int u = 0; u < RH; ++u) hrow[u][c] = Hp[c * DK + lane + kWave * u];
#pragma unroll
    for (int u = 0; u < RH; ++u) {
        const int r = lane + kWave * u;
        hdiag[u] = gam * Hp[r * DK + r] + bet * kr[u] * kr[u] + lr[u];
    }
#pragma unroll
    for (int c4 = 0; c4 < DK; c4 += 4) {
        const f32x4 kc = *reinterpret_cast<const f32x4*>(sk + c4);
#pragma unroll
        for (int e = 0; e < 4; ++e)
#pragma unroll
            for (int u = 0; u < RH; ++u) {
                const float hn = gam * hrow[u][c4 + e] + bet * kr[u] * kc[e];
                hrow[u][c4 + e] = hn;
                Hp[(c4 + e) * DK + lane + kWave * u] = hn;
            }
    }

    // ---- 2. CG on (H + Lambda) x = q
    auto gemv = [&](const float (&pin)[RH], float (&wout)[RH]) {
        __syncthreads();  // previous readers of sp are done
#pragma unroll
        for (int u = 0; u < RH; ++u) sp[lane + kWave * u] = pin[u];
        __syncthreads();
#pragma unroll
        for (int u = 0; u < RH; ++u) wout[u] = lr[u] * pin[u];
#pragma unroll
        for (int c4 = 0; c4 < DK; c4 += 4) {
            const f32x4 pc = *reinterpret_cast<const f32x4*>(sp + c4);
#pragma unroll
            for (int e = 0; e < 4; ++e)
#pragma unroll
                for (int u = 0; u < RH; ++u) wout[u] += hrow[u][c4 + e] * pc[e];
        }
    };
    auto dot = [&](const float (&x)[RH], const float (&y)[RH]) -> float {
        float s = 0.0f;
#pragma unroll
        for (int u = 0; u < RH; ++u) s += x[u] * y[u];
        return wave_sum(s);
    };

    float x[RH], r[RH], p[RH], w[RH];
#pragma unroll
    for (int u = 0; u < RH; ++u) x[u] = qr[u] / hdiag[u];
    gemv(x, w);
#pragma unroll
    for (int u = 0; u < RH; ++u) {
        r[u] = qr[u] - w[u];
        p[u] = r[u];
    }
    float delta = dot(r, r);
    if (delta > 0.0f) {
        for (int it = 0; it < a.n_cg; ++it) {
            gemv(p, w);
            const float pw = dot(p, w);
            if (!(pw > 0.0f)) break;
            const float alpha = delta / pw;
#pragma unroll
            for (int u = 0; u < RH; ++u) {
                x[u] += alpha * p[u];
                r[u] -= alpha * w[u];
            }
            const float dn = dot(r, r);
            if (dn == 0.0f) break;
            const float beta_cg = dn / delta;
#pragma unroll
            for (int u = 0; u < RH; ++u) p[u] = r[u] + beta_cg * p[u];
            delta = dn;
        }
    }

    // ---- 3. G update and read-out, rows R(lane) of G
    __syncthreads();
#pragma unroll
    for (int u = 0; u < RH; ++u) sp[lane + kWave * u] = x[u];
    __syncthreads();
    float* Gp = a.G + pair * int64_t(DV) * DK;
#pragma unroll
    for (int u = 0; u < RG; ++u) {
        const int e = lane + kWave * u;
        float* grow = Gp + int64_t(e) * DK;
        float o = 0.0f;
#pragma unroll
        for (int c4 = 0; c4 < DK; c4 += 4) {
            const f32x4 gv = *reinterpret_cast<const f32x4*>(grow + c4);
            const f32x4 kc = *reinterpret_cast<const f32x4*>(sk + c4);
            const f32x4 xc = *reinterpret_cast<const f32x4*>(sp + c4);
            f32x4 gn;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                gn[q] = gam * gv[q] + bet * vr[u] * kc[q];
                o += gn[q] * xc[q];
            }
            *reinterpret_cast<f32x4*>(grow + c4) = gn;
        }
        a.out[pair * DV + e] = o;
    }
}

template <typename Tin, int DK>
hipError_t launch_dk(const DecodeArgs& a, hipStream_t stream)
{
    const unsigned blocks = unsigned(a.batch * a.heads);
    if (a.d_v == 64)
        hipLaunchKernelGGL((decode_step_kernel<Tin, DK, 64>), dim3(blocks), dim3(kWave), 0, stream, a);
    else
        hipLaunchKernelGGL((decode_step_kernel<Tin, DK, 128>), dim3(blocks), dim3(kWave), 0, stream, a);
    return hipGetLastError();
}

template <typename Tin>
hipError_t launch_tin(const DecodeArgs& a, hipStream_t stream)
{
    return a.d_k == 64 ? launch_dk<Tin, 64>(a, stream) : launch_dk<Tin, 128>(a, stream);
}

}  // namespace

hipError_t launch_decode_step(const DecodeArgs& a, hipStream_t stream)
{
    return a.bf16 ? launch_tin<bf16_t>(a, stream) : launch_tin<float>(a, stream);
}

}  // namespace mesa
