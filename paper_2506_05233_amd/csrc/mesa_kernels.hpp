// Host-side launchers of the libmesa kernels.  Each kernel source file defines
// its kernels and the launcher declared here; the C ABI (libmesa.hip) validates
// arguments and calls the launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mesa {

// Shapes of one forward call.  Token (b, h, t) lives at row (b*heads + h)*seq_len + t.
struct ForwardShape {
    int64_t batch, heads, seq_len;
    int d_k, d_v, chunk;
    int n_chunks;  // ceil(seq_len / chunk)
    bool bf16;     // q, k, v element type
};

// Chunk-state scan: writes the states entering every chunk when store_chunks,
// and the fp32 states after the last token (final_H [B*H, d_k, d_k], final_G
// [B*H, d_v, d_k]) when those pointers are non-null.  Two layouts of the
// chunk states:
//   plain (frag == false): fp32 Hs [B*H, n_chunks, d_k, d_k], Gs [B*H, n_chunks, d_v, d_k];
//   fragment (frag == true, bf16 inputs, chunk 64): bf16 MFMA A-operand
//     fragments, Hs as [B*H, n_chunks, d_k/16, d_k/32, 64 lanes, 8] and Gs as
//     [B*H, n_chunks, d_v/16, d_k/32, 64 lanes, 8]; fragment (t, s) lane
//     (g, m) element e holds X[16t + m][32s + (e < 4 ? 4g + e : 16 + 4g + e - 4)].
struct StateArgs {
    ForwardShape s;
    const void* k;
    const void* v;
    const float* gamma;
    const float* beta;
    void* Hs;
    void* Gs;
    float* final_H;
    float* final_G;
    bool store_chunks;
    bool frag;
    // Scratch for the segmented scan (may be null: then one segment): fp32
    // segment totals and decays, seg_bytes bytes.  Used by the bf16 scan only.
    float* seg_ws = nullptr;
    size_t seg_bytes = 0;
    // With frag: also the same chunk states as plain fp32 (layout of frag == false), from
    // the same fp32-accurate pass (may be null).
    float* Hs32 = nullptr;
    float* Gs32 = nullptr;
    // Split-operand layout (bf16 inputs, chunk 64; instead of frag), fp32-accurate:
    // Hs fp32 H_c fragments, half e of fragment f = (t, s), lane l at
    // [B*H, n_chunks][(2 f + e) * 64 + l][4]; Gs the bf16 G_c fragments (high parts)
    // followed by a second plane of the same shape with the low parts bf16(x - hi).
    bool x3 = false;
};
bool chunk_state_frag_supported(const ForwardShape& s);
hipError_t launch_chunk_state(const StateArgs& a, hipStream_t stream);

// dst[0 .. n) = 0 with a fill kernel (no memset node, so the call can be graph-captured).
hipError_t launch_fill_zero(float* dst, int64_t n, hipStream_t stream);

// Chunked CG + read-out: q*_t for every token and o_t = G_t q*_t.
struct CgArgs {
    ForwardShape s;
    const void* q;
    const void* k;
    const void* v;
    const float* gamma;
    const float* beta;
    const float* lambda;
    const void* Hs;   // chunk states, plain fp32 (fp32 path) or bf16 fragments (bf16 path)
    const void* Gs;
    int n_cg;        // at most n_cg CG iterations per token
    float* out;
    float* qstar;    // may be null
    float eps2;      // Alg. 1 relative tolerance, squared: stop once |r|^2 <= eps2 |r_0|^2
    int32_t* steps;  // may be null: [B, H, T] iterations each token used
    // fp32 right-hand sides [B, H, T, d_k] solved for instead of q (fp32 path only),
    // may be null; with out null the read-out is skipped and only qstar is written
    const float* rhs = nullptr;
};
hipError_t launch_chunk_cg_f32(const CgArgs& a, hipStream_t stream);

// Backward pass (fp32, chunk 64), in stages on one stream: 0 the right-hand sides
// u_t = G_t^T e_t, 1 the reverse adjoint scan, 2 the per-chunk gradients, 3 the
// Lambda reduction (the chunk-state scan and the solve for e* run between, through
// launch_chunk_state and launch_chunk_cg_f32).
struct BwdArgs {
    ForwardShape s;        // chunk 64
    const void* k;
    const void* v;
    const float* gamma;
    const float* beta;
    const float* qstar;    // [B, H, T, d_k]
    const float* dout;     // [B, H, T, d_v]: e_t
    const float* estar;    // [B, H, T, d_k]: e*_t
    const float* Hs;       // forward chunk states, plain fp32 [B*H, n_chunks, d_k, d_k]
    const float* Gs;       // [B*H, n_chunks, d_v, d_k]
    float* SH;             // symmetric H adjoint arriving at each chunk's end [B*H, n_chunks, d_k, d_k]
    float* AG;             // G adjoint [B*H, n_chunks, d_v, d_k]
    float* u;              // [B, H, T, d_k]
    uint16_t* u16;         // if non-null, u is written here instead, rounded to bf16
    float* dk;
    float* dv;
    float* dgamma;
    float* dbeta;
    float* dlam_part;      // [B*H, n_chunks, d_k]
    float* dlam;           // [H, d_k]
};
hipError_t launch_backward_stage(const BwdArgs& a, int stage, hipStream_t stream);
hipError_t launch_chunk_cg_bf16(const CgArgs& a, hipStream_t stream);
bool chunk_cg_bf16_supported(const ForwardShape& s);
// The same solve and read-out with split operands (hi + lo bf16 pairs, three matrix-core
// passes per product) from the split-operand chunk-state layout.
hipError_t launch_chunk_cg_x3(const CgArgs& a, hipStream_t stream);
bool chunk_cg_x3_supported(const ForwardShape& s);

// One recurrent decode step for batch*heads pairs.
struct DecodeArgs {
    int64_t batch, heads;
    int d_k, d_v;
    bool bf16;
    float* H;
    float* G;
    const void* q;
    const void* k;
    const void* v;
    const float* gamma;
    const float* beta;
    const float* lambda;
    int n_cg;
    float* out;
    float eps2;      // Alg. 1 relative tolerance, squared (0: fixed steps)
    int32_t* steps;  // may be null: [batch, heads] iterations each pair used
    bool packed = false;  // H in the packed symmetric layout (see launch_pack_state)
};
hipError_t launch_decode_step(const DecodeArgs& a, hipStream_t stream);

// Packed symmetric decode state: HP [pairs, d_k/2 + 1, d_k] with
// HP[k][i] = H[i][(i + k) mod d_k] (row k = the k-th cyclic diagonal).  Every
// unordered pair {i, j} is stored once, except on the last diagonal (k = d_k/2),
// where the copy at i < d_k/2 is the one read and written.
hipError_t launch_pack_state(const float* H, float* HP, int64_t pairs, int d_k, hipStream_t stream);
hipError_t launch_unpack_state(const float* HP, float* H, int64_t pairs, int d_k, hipStream_t stream);

// The layer's front end (App. E; gate cap and Lambda floor of App. G.5), one launch:
// q, k [B, H, T, d_k] and v [B, H, T, d_v] (element type of the projections) from the
// projections qp, kp [B, T, H, d_k], vp [B, T, H, d_v]; gamma, beta [B, H, T] from the
// gate projections a_gamma, a_beta [B, T, H]; lambda [H, d_k] from theta [H, d_k].
// conv_q, conv_k [H * d_k, 4], conv_v [H * d_v, 4] or null (values unchanged).
struct FrontArgs {
    int64_t batch, heads, seq_len;
    int d_k, d_v;
    bool bf16;
    const void* qp;
    const void* kp;
    const void* vp;
    const float* conv_q;
    const float* conv_k;
    const float* conv_v;
    const float* a_gamma;
    const float* a_beta;
    const float* theta;
    float gamma_cap, l2_eps;
    void* q;
    void* k;
    void* v;
    float* gamma;
    float* beta;
    float* lambda;
};
hipError_t launch_frontend(const FrontArgs& a, hipStream_t stream);

// The back end: per-head RMSNorm, o [B, H, T, d_v] fp32 -> y [B, T, H, d_v] (fp32 or
// bf16), weight [H, d_v].
struct NormArgs {
    int64_t batch, heads, seq_len;
    int d_v;
    bool bf16_out;
    const float* o;
    const float* weight;
    float eps;
    void* y;
};
hipError_t launch_output_norm(const NormArgs& a, hipStream_t stream);

// Compute units of the current device (queried once per device), for the persistent
// kernels that launch one workgroup per unit.
int device_compute_units();

}  // namespace mesa
