// Recurrent decode step of the Mesa layer (Sec. 3, recurrent inference mode;
// App. C, last paragraph: at inference CG runs on H_t + Lambda directly).
//
// One workgroup of d_k threads (d_k / 64 waves) per (sequence, head); the step
// is bound by HBM, since each pair reads and writes its two fp32 states
// (8 (d_k + d_v) d_k bytes), so the kernel is built for many pairs in flight
// per compute unit: about 160 registers per thread let three workgroups share
// a SIMD, and pairs in different phases (state traffic, CG) overlap.
//   1. H <- gamma H + beta k k^T.  Thread R keeps row R of H in registers.  H is
//      symmetric, so row R is read as column R, H[c][R] for c = 0..d_k-1: the
//      threads of a wave read and write 64 consecutive floats of one row of H
//      per access (256 contiguous bytes); the updated values are written back in
//      place.
//   2. Alg. 1 with tolerance 0 on (H + Lambda) x = q: thread R owns element R of
//      x, r, p, w; each product is a register-resident row times p, with p
//      broadcast through LDS; the CG scalars are wave reductions combined across
//      the waves through LDS (every wave adds the partial sums in the same order,
//      so all waves take the same branches).
//   3. G <- gamma G + beta v k^T and o = G x: thread e streams row e of G through
//      registers (rows e, e + d_k, ... when d_v > d_k), writes it back and forms
//      o_e on the way.
// All arithmetic is fp32.
#include "mesa_device.hpp"
#include "mesa_kernels.hpp"

namespace mesa {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

// Word 3 of a raw buffer resource on gfx9 (32-bit data format, no swizzle).
constexpr int kBufferRsrcWord3 = 0x00020000;

template <typename Tin, int DK, int DV>
__global__ __launch_bounds__(DK) __attribute__((amdgpu_waves_per_eu(3)))
void decode_step_kernel(DecodeArgs a)
{
    constexpr int NW = DK / kWave;  // waves per pair
    const int64_t pair = blockIdx.x;
    const int h = int(pair % a.heads);
    const int tid = threadIdx.x;    // this thread's row of H and element of the CG vectors
    const int lane = tid % kWave, wv = tid / kWave;

    __shared__ __attribute__((aligned(16))) float sk[DK];
    __shared__ __attribute__((aligned(16))) float sp[DK];
    __shared__ float sred[2][NW];

    const Tin* qp = static_cast<const Tin*>(a.q) + pair * DK;
    const Tin* kp = static_cast<const Tin*>(a.k) + pair * DK;
    const Tin* vp = static_cast<const Tin*>(a.v) + pair * DV;
    const float gam = a.gamma[pair], bet = a.beta[pair];
    const float kR = to_f32(kp[tid]), qR = to_f32(qp[tid]), lR = a.lambda[int64_t(h) * DK + tid];
    sk[tid] = kR;

    // ---- 1. state update of H, row tid held as hc[c] = H[c][tid].  The pair's H is
    // addressed through a buffer resource: the column offset c d_k is a scalar, so the
    // 2 d_k accesses need no per-access address registers (the buffer builtins move raw
    // 32-bit words, hence the bit casts).
    float* Hp = a.H + pair * DK * DK;
    const __amdgpu_buffer_rsrc_t hr = __builtin_amdgcn_make_buffer_rsrc(Hp, 0, DK * DK * 4, kBufferRsrcWord3);
    float hc[DK];
#pragma unroll
    for (int c = 0; c < DK; ++c) hc[c] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(hr, tid * 4, c * DK * 4, 0));
    const float hdiag = gam * __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(hr, tid * (DK + 1) * 4, 0, 0)) + bet * kR * kR + lR;
    __syncthreads();
#pragma unroll
    for (int c4 = 0; c4 < DK; c4 += 4) {
        const f32x4 kc = *reinterpret_cast<const f32x4*>(sk + c4);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            hc[c4 + e] = gam * hc[c4 + e] + bet * kR * kc[e];
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(hc[c4 + e]), hr, tid * 4, (c4 + e) * DK * 4, 0);
        }
    }

    // ---- 2. CG on (H + Lambda) x = q
    // w = (H + Lambda) p for this thread's row; p goes through sp (its previous readers
    // passed at least one barrier of a dot product since)
    auto gemv = [&](float pin) -> float {
        sp[tid] = pin;
        __syncthreads();
        f32x4 acc = {lR * pin, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int c4 = 0; c4 < DK; c4 += 4) {
            const f32x4 pc = *reinterpret_cast<const f32x4*>(sp + c4);
#pragma unroll
            for (int e = 0; e < 4; ++e) acc[e] += hc[c4 + e] * pc[e];
        }
        return (acc[0] + acc[1]) + (acc[2] + acc[3]);
    };
    // sum over the d_k rows of x*y: wave sums, then the waves' partial sums from LDS in
    // wave order (slots alternate, so a slot is rewritten only after every wave has
    // passed the barrier of the dot product in between)
    int slot = 0;
    auto dot = [&](float x, float y) -> float {
        const float s = wave_sum(x * y);
        if (lane == 0) sred[slot][wv] = s;
        __syncthreads();
        float t = sred[slot][0];
#pragma unroll
        for (int u = 1; u < NW; ++u) t += sred[slot][u];
        slot ^= 1;
        return t;
    };

    float x = qR / hdiag;
    float r = qR - gemv(x);
    float p = r;
    float delta = dot(r, r);
    if (delta > 0.0f) {
        for (int it = 0; it < a.n_cg; ++it) {
            const float w = gemv(p);
            const float pw = dot(p, w);
            if (!(pw > 0.0f)) break;
            const float alpha = delta / pw;
            x += alpha * p;
            r -= alpha * w;
            const float dn = dot(r, r);
            if (dn == 0.0f) break;
            p = r + (dn / delta) * p;
            delta = dn;
        }
    }

    // ---- 3. G update and read-out, rows e = tid, tid + d_k, ... of G
    sp[tid] = x;  // sp's last readers (the last product) passed a dot product's barrier
    __syncthreads();
    float* Gp = a.G + pair * int64_t(DV) * DK;
#pragma unroll
    for (int e = tid; e < DV; e += DK) {
        float* grow = Gp + int64_t(e) * DK;
        const float bv = bet * to_f32(vp[e]);
        f32x4 o4 = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int c4 = 0; c4 < DK; c4 += 4) {
            const f32x4 gv = *reinterpret_cast<const f32x4*>(grow + c4);
            const f32x4 kc = *reinterpret_cast<const f32x4*>(sk + c4);
            const f32x4 xc = *reinterpret_cast<const f32x4*>(sp + c4);
            f32x4 gn;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                gn[q] = gam * gv[q] + bv * kc[q];
                o4[q] += gn[q] * xc[q];
            }
            *reinterpret_cast<f32x4*>(grow + c4) = gn;
        }
        a.out[pair * DV + e] = (o4[0] + o4[1]) + (o4[2] + o4[3]);
    }
}

template <typename Tin, int DK>
hipError_t launch_dk(const DecodeArgs& a, hipStream_t stream)
{
    const unsigned blocks = unsigned(a.batch * a.heads);
    if (a.d_v == 64)
        hipLaunchKernelGGL((decode_step_kernel<Tin, DK, 64>), dim3(blocks), dim3(DK), 0, stream, a);
    else
        hipLaunchKernelGGL((decode_step_kernel<Tin, DK, 128>), dim3(blocks), dim3(DK), 0, stream, a);
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
