// Recurrent decode step of the Mesa layer (Sec. 2, recurrent inference mode;
// App. C, last paragraph: at inference CG runs on H_t + Lambda directly).
//
// One workgroup of d_k threads (d_k / 64 waves) per (sequence, head); the step
// is bound by HBM, since each pair reads and writes its two fp32 states
// (8 (d_k + d_v) d_k bytes), so the kernel is built for many pairs in flight
// per compute unit: about 160 registers per thread let three workgroups share
// a SIMD, and pairs in different phases (state traffic, CG) overlap.  Every
// state access of a wave is one row segment of 256 contiguous bytes.
//   1. H <- gamma H + beta k k^T.  Thread R keeps row R of H in registers.  H is
//      symmetric, so row R is read as column R, H[c][R] for c = 0..d_k-1; the
//      updated values are written back in place.
//   2. Alg. 1 (at most n_cg iterations, relative tolerance eps) on (H + Lambda) x = q:
//      thread R owns element R of x, r, p, w; each product is a register-resident
//      row times p, with p broadcast through LDS; the CG scalars are wave
//      reductions combined across the waves through LDS (every wave adds the
//      partial sums in the same order, so all waves take the same branches).
//   3. G <- gamma G + beta v k^T and o = G x: thread c keeps column c of G,
//      writes it back, and the row sums of G diag(x) are reduced across lanes
//      and waves.
// All arithmetic is fp32.
#include "mesa_device.hpp"
#include "mesa_kernels.hpp"

namespace mesa {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

// Word 3 of a raw buffer resource on gfx9 (32-bit data format, no swizzle).
constexpr int kBufferRsrcWord3 = 0x00020000;
constexpr int kXB = 8;  // diagonals per LDS exchange of the packed layout

template <typename Tin, int DK, int DV, bool PACKED>
__global__ __launch_bounds__(DK) __attribute__((amdgpu_waves_per_eu(3)))
void decode_step_kernel(DecodeArgs a)
{
    constexpr int NW = DK / kWave;  // waves per pair
    const int64_t pair = blockIdx.x;
    const int h = int(pair % a.heads);
    const int tid = threadIdx.x;    // this thread's row of H and element of the CG vectors
    const int lane = tid % kWave, wv = tid / kWave;

    // k and p are kept twice over (entries i and i + d_k) in the packed layout, so the
    // rotated reads of its diagonals are a base register plus immediate offsets
    __shared__ __attribute__((aligned(16))) float sk[PACKED ? 2 * DK : DK];
    __shared__ __attribute__((aligned(16))) float sp[PACKED ? 2 * DK : DK];
    __shared__ float sred[2][NW];
    __shared__ __attribute__((aligned(16))) float sv[DV];
    __shared__ float so[NW][DV];
    __shared__ float sx[PACKED ? kXB : 1][2 * DK];  // packed layout: diagonal exchange

    const Tin* qp = static_cast<const Tin*>(a.q) + pair * DK;
    const Tin* kp = static_cast<const Tin*>(a.k) + pair * DK;
    const Tin* vp = static_cast<const Tin*>(a.v) + pair * DV;
    const float gam = a.gamma[pair], bet = a.beta[pair];
    const float kR = to_f32(kp[tid]), qR = to_f32(qp[tid]), lR = a.lambda[int64_t(h) * DK + tid];
    sk[tid] = kR;
    if constexpr (PACKED) sk[tid + DK] = kR;
    for (int e = tid; e < DV; e += DK) sv[e] = to_f32(vp[e]);

    // ---- 1. state update of H.  The pair's H is addressed through a buffer resource:
    // the row offsets are scalars, so the accesses need no per-access address registers
    // (the buffer builtins move raw 32-bit words, hence the bit casts).
    // Full layout: thread R holds hc[c] = H[c][R] (row R, read as column R).
    // Packed layout (HP[k][i] = H[i][(i + k) mod d_k]): thread R holds ho[k] = H[R][R + k]
    // = HP[k][R] for k = 0 .. d_k/2 (its own entries, which it updates and writes back)
    // and hx[k] = H[R][R - k] = HP[k][R - k] for k = 1 .. d_k/2 - 1 (owned by thread
    // R - k; thread R applies the same update, with the owner's operation order, to its
    // copy).  On the last diagonal the copy at i < d_k/2 is the stored one.
    constexpr int NH = PACKED ? DK / 2 + 1 : DK;   // rows of the stored state
    float* Hp = a.H + pair * NH * DK;
    const __amdgpu_buffer_rsrc_t hr = __builtin_amdgcn_make_buffer_rsrc(Hp, 0, NH * DK * 4, kBufferRsrcWord3);
    float hc[PACKED ? 1 : DK];
    float ho[PACKED ? DK / 2 + 1 : 1], hx[PACKED ? DK / 2 : 1];
    float hdiag;
    if constexpr (!PACKED) {
#pragma unroll
        for (int c = 0; c < DK; ++c) hc[c] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(hr, tid * 4, c * DK * 4, 0));
        hdiag = gam * __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(hr, tid * (DK + 1) * 4, 0, 0)) + bet * kR * kR + lR;
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
    } else {
        constexpr int HALF = DK / 2;
        const int rl = tid % HALF;  // the owner of this thread's last-diagonal entry
#pragma unroll
        for (int k = 0; k < HALF; ++k) ho[k] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(hr, tid * 4, k * DK * 4, 0));
        ho[HALF] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(hr, rl * 4, HALF * DK * 4, 0));
        __syncthreads();
        const float bkR = bet * kR;
#pragma unroll
        for (int k = 0; k < HALF; ++k) {
            ho[k] = gam * ho[k] + bkR * sk[tid + k];
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(ho[k]), hr, tid * 4, k * DK * 4, 0);
        }
        ho[HALF] = gam * ho[HALF] + (bet * sk[rl]) * sk[rl + HALF];
        if (tid < HALF) __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(ho[HALF]), hr, tid * 4, HALF * DK * 4, 0);
        // H[R][R - k] is thread (R - k)'s updated entry of diagonal k: exchanged through
        // LDS, kXB diagonals at a time
#pragma unroll
        for (int k0 = 1; k0 < HALF; k0 += kXB) {
#pragma unroll
            for (int j = 0; j < kXB; ++j)
                if (k0 + j < HALF) {
                    sx[j][tid] = ho[k0 + j];
                    sx[j][tid + DK] = ho[k0 + j];
                }
            __syncthreads();
#pragma unroll
            for (int j = 0; j < kXB; ++j)
                if (k0 + j < HALF) hx[k0 + j] = sx[j][tid + DK - k0 - j];
            __syncthreads();
        }
        hdiag = ho[0] + lR;
    }

    // ---- 2. CG on (H + Lambda) x = q
    // w = (H + Lambda) p for this thread's row; p goes through sp (its previous readers
    // passed at least one barrier of a dot product since)
    auto gemv = [&](float pin) -> float {
        sp[tid] = pin;
        if constexpr (PACKED) sp[tid + DK] = pin;
        __syncthreads();
        f32x4 acc = {lR * pin, 0.0f, 0.0f, 0.0f};
        if constexpr (!PACKED) {
#pragma unroll
            for (int c4 = 0; c4 < DK; c4 += 4) {
                const f32x4 pc = *reinterpret_cast<const f32x4*>(sp + c4);
#pragma unroll
                for (int e = 0; e < 4; ++e) acc[e] += hc[c4 + e] * pc[e];
            }
        } else {
            // H[R][R + k] p_{R+k} for k = 0 .. d_k/2 and H[R][R - k] p_{R-k} for k = 1 .. d_k/2 - 1
            // (rotated LDS reads: consecutive lanes, consecutive words)
            const float* pr = sp + tid;
#pragma unroll
            for (int k = 0; k <= DK / 2; ++k) acc[k & 3] += ho[k] * pr[k];
#pragma unroll
            for (int k = 1; k < DK / 2; ++k) acc[(k + 2) & 3] += hx[k] * pr[DK - k];
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

    // solve for q 2^-qsh (|q 2^-qsh|^2 in [1/2, 2)); x is scaled back after the loop
    const int qsh = cg_scale_shift(dot(qR, qR));
    const float qRs = qR * __builtin_ldexpf(1.0f, -qsh);
    float x = qRs / hdiag;
    float r = qRs - gemv(x);
    float p = r;
    float delta = dot(r, r);
    const float thr = a.eps2 * delta;  // Alg. 1: stop once |r|^2 <= eps^2 |r_0|^2
    int steps = 0;                     // iterations that updated x
    if (delta >= kMinNormal) {
        for (int it = 0; it < a.n_cg; ++it) {
            const float w = gemv(p);
            const float pw = dot(p, w);
            if (!(pw >= kMinNormal)) break;
            const float alpha = delta / pw;
            x += alpha * p;
            r -= alpha * w;
            ++steps;
            const float dn = dot(r, r);
            if (dn <= thr || !(dn >= kMinNormal)) break;
            p = r + (dn / delta) * p;
            delta = dn;
        }
    }
    x *= __builtin_ldexpf(1.0f, qsh);

    if (a.steps && tid == 0) a.steps[pair] = steps;

    // ---- 3. G update and read-out.  Thread c owns column c of G: G[e][c] for every row e
    // is read and written as one 256-byte wave access per row (like H), and the row sums
    // o_e = sum_c G[e][c] x_c are formed by a transposing reduction across the lanes
    // (blocks of 32 rows: two lane-half swaps leave 8 rows per lane summed over 4 lanes,
    // a 16-lane reduction completes each), then across the waves through LDS.
    float* Gp = a.G + pair * int64_t(DV) * DK;
    const __amdgpu_buffer_rsrc_t gr = __builtin_amdgcn_make_buffer_rsrc(Gp, 0, DV * DK * 4, kBufferRsrcWord3);
    float gc[DV];
#pragma unroll
    for (int e = 0; e < DV; ++e) gc[e] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(gr, tid * 4, e * DK * 4, 0));
    const float bk = bet * kR;
#pragma unroll
    for (int e4 = 0; e4 < DV; e4 += 4) {
        const f32x4 ve = *reinterpret_cast<const f32x4*>(sv + e4);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            gc[e4 + q] = gam * gc[e4 + q] + bk * ve[q];
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(gc[e4 + q]), gr, tid * 4, (e4 + q) * DK * 4, 0);
            gc[e4 + q] *= x;
        }
    }
#pragma unroll
    for (int b = 0; b < DV; b += 32) {
        float s16[16], s8[8];
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const auto t = __builtin_amdgcn_permlane32_swap(__float_as_uint(gc[b + i]), __float_as_uint(gc[b + 16 + i]), false, false);
            s16[i] = __uint_as_float(t[0]) + __uint_as_float(t[1]);
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const auto t = __builtin_amdgcn_permlane16_swap(__float_as_uint(s16[i]), __float_as_uint(s16[8 + i]), false, false);
            s8[i] = __uint_as_float(t[0]) + __uint_as_float(t[1]);
        }
        // lanes of 16-lane row rr hold rows b + 8 rr + i; sum over the row's 16 lanes
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            float v = s8[i];
            v += dpp_f32<kDppQuadSwap1>(v, v);
            v += dpp_f32<kDppQuadSwap2>(v, v);
            v += dpp_f32<kDppRowRor4>(v, v);
            v += dpp_f32<kDppRowRor8>(v, v);
            s8[i] = v;
        }
        if (lane % 16 == 0) {
#pragma unroll
            for (int i = 0; i < 8; ++i) so[wv][b + 8 * (lane / 16) + i] = s8[i];
        }
    }
    __syncthreads();
    for (int e = tid; e < DV; e += DK) {
        float o = so[0][e];
#pragma unroll
        for (int u = 1; u < NW; ++u) o += so[u][e];
        a.out[pair * DV + e] = o;
    }
}

template <typename Tin, int DK, bool PACKED>
hipError_t launch_dk(const DecodeArgs& a, hipStream_t stream)
{
    const unsigned blocks = unsigned(a.batch * a.heads);
    if (a.d_v == 64)
        hipLaunchKernelGGL((decode_step_kernel<Tin, DK, 64, PACKED>), dim3(blocks), dim3(DK), 0, stream, a);
    else
        hipLaunchKernelGGL((decode_step_kernel<Tin, DK, 128, PACKED>), dim3(blocks), dim3(DK), 0, stream, a);
    return hipGetLastError();
}

// full <-> packed symmetric state (one thread per stored element; the packed
// element HP[k][i] is H[i][(i + k) mod d_k], so unpacking writes it to (i, i + k)
// and (i + k, i))
__global__ __launch_bounds__(256) void pack_state_kernel(const float* H, float* HP, int64_t pairs, int dk)
{
    const int64_t per = int64_t(dk / 2 + 1) * dk;
    const int64_t idx = int64_t(blockIdx.x) * 256 + threadIdx.x;
    if (idx >= pairs * per) return;
    const int64_t pr = idx / per;
    const int e = int(idx % per), k = e / dk, i = e % dk;
    HP[idx] = H[pr * dk * dk + int64_t(i) * dk + ((i + k) & (dk - 1))];
}

__global__ __launch_bounds__(256) void unpack_state_kernel(const float* HP, float* H, int64_t pairs, int dk)
{
    const int64_t idx = int64_t(blockIdx.x) * 256 + threadIdx.x;
    if (idx >= pairs * dk * dk) return;
    const int64_t pr = idx / (int64_t(dk) * dk);
    const int e = int(idx % (int64_t(dk) * dk)), i = e / dk, j = e % dk;
    // H[i][j] is stored as HP[k][i] with k = (j - i) mod d_k when k <= d_k/2, else as
    // HP[(i - j) mod d_k][j]; on the last diagonal the copy at the smaller index of
    // {i, j} mod d_k/2 is the stored one
    int k = (j - i) & (dk - 1), at = i;
    if (k > dk / 2) {
        k = (i - j) & (dk - 1);
        at = j;
    }
    if (k == dk / 2) at = i % (dk / 2);
    H[idx] = HP[pr * (dk / 2 + 1) * dk + int64_t(k) * dk + at];
}

template <typename Tin>
hipError_t launch_tin(const DecodeArgs& a, hipStream_t stream)
{
    if (a.packed) return a.d_k == 64 ? launch_dk<Tin, 64, true>(a, stream) : launch_dk<Tin, 128, true>(a, stream);
    return a.d_k == 64 ? launch_dk<Tin, 64, false>(a, stream) : launch_dk<Tin, 128, false>(a, stream);
}

}  // namespace

hipError_t launch_decode_step(const DecodeArgs& a, hipStream_t stream)
{
    return a.bf16 ? launch_tin<bf16_t>(a, stream) : launch_tin<float>(a, stream);
}

hipError_t launch_pack_state(const float* H, float* HP, int64_t pairs, int d_k, hipStream_t stream)
{
    const int64_t n = pairs * (d_k / 2 + 1) * d_k;
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(pack_state_kernel, dim3(unsigned((n + 255) / 256)), dim3(256), 0, stream, H, HP, pairs, d_k);
    return hipGetLastError();
}

hipError_t launch_unpack_state(const float* HP, float* H, int64_t pairs, int d_k, hipStream_t stream)
{
    const int64_t n = pairs * int64_t(d_k) * d_k;
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(unpack_state_kernel, dim3(unsigned((n + 255) / 256)), dim3(256), 0, stream, HP, H, pairs, d_k);
    return hipGetLastError();
}

}  // namespace mesa
