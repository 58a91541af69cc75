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
};
hipError_t launch_chunk_cg_f32(const CgArgs& a, hipStream_t stream);
hipError_t launch_chunk_cg_bf16(const CgArgs& a, hipStream_t stream);
bool chunk_cg_bf16_supported(const ForwardShape& s);

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
};
hipError_t launch_decode_step(const DecodeArgs& a, hipStream_t stream);

}  // namespace mesa
