// libmesa C ABI: argument validation, workspace sizing and kernel launches.
// The contract of every entry point is documented in include/libmesa.h.
#include "libmesa.h"

#include <float.h>
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <initializer_list>
#include <mutex>

#include "mesa_kernels.hpp"

namespace {

using mesa::ForwardShape;

bool dim_ok(int64_t d) { return d == 64 || d == 128; }
bool chunk_ok(int c) { return c == 16 || c == 32 || c == 64; }

int64_t n_chunks_of(int64_t seq_len, int chunk) { return (seq_len + chunk - 1) / chunk; }

// Byte range [p, p + n) of a device array, for overlap checks.
struct Range {
    uintptr_t lo, hi;
};
Range range_of(const void* p, int64_t bytes) { return {uintptr_t(p), uintptr_t(p) + uintptr_t(bytes)}; }
bool overlaps(Range a, Range b) { return a.lo < b.hi && b.lo < a.hi; }

// MESA_SYNC_AFTER_LAUNCH (read once, at the first call): when set to anything but
// "" or "0", every entry point synchronises its stream after its launches and turns
// an execution error into MESA_ERR_HIP.
bool sync_after_launch()
{
    static const bool on = [] {
        const char* e = getenv("MESA_SYNC_AFTER_LAUNCH");
        return e != nullptr && e[0] != '\0' && strcmp(e, "0") != 0;
    }();
    return on;
}

// The status an entry point returns once its launches are enqueued on `stream`.
int finish(int status, void* stream)
{
    if (status != MESA_OK || !sync_after_launch()) return status;
    if (hipStreamSynchronize(static_cast<hipStream_t>(stream)) != hipSuccess) return MESA_ERR_HIP;
    return hipGetLastError() == hipSuccess ? MESA_OK : MESA_ERR_HIP;
}

// MESA_CHECK_FINITE (read once, at the first call): when set to anything but "" or
// "0", the forward and decode calls check the values of their inputs before their
// launches and of their outputs after them (a debugging aid that reads device memory
// and synchronises the stream).
bool check_values_on()
{
    static const bool on = [] {
        const char* e = getenv("MESA_CHECK_FINITE");
        return e != nullptr && e[0] != '\0' && strcmp(e, "0") != 0;
    }();
    return on;
}

// A device array to check: n values (fp32, or bf16 bits), each to lie in [lo, hi] (a NaN
// lies in no range).
struct ValueRange {
    const void* p;
    int64_t n;
    bool bf16;
    float lo, hi;
};
constexpr float kFinite = FLT_MAX;

// Set by value_range_kernel when a value lies outside its range; one per device, in the
// library's code object (host code takes its address from hipGetSymbolAddress).
__device__ int value_flag;

__global__ __launch_bounds__(64) void value_flag_clear_kernel(int* flag)
{
    if (threadIdx.x == 0) flag[0] = 0;
}

__global__ __launch_bounds__(256) void value_range_kernel(const void* p, int64_t n, int bf16, float lo, float hi,
                                                          int* flag)
{
    bool bad = false;
    const int64_t stride = int64_t(gridDim.x) * blockDim.x;
    for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += stride) {
        const float x = bf16 ? __uint_as_float(uint32_t(static_cast<const uint16_t*>(p)[i]) << 16)
                             : static_cast<const float*>(p)[i];
        bad = bad || !(x >= lo && x <= hi);
    }
    if (bad) flag[0] = 1;
}

constexpr int kMaxFlagDevices = 64;
std::mutex g_flag_mutex;
int* g_flag_ptr[kMaxFlagDevices] = {};

// Checks `vals` on `stream` (when MESA_CHECK_FINITE is on): returns `bad` if a value lies
// outside its range, MESA_OK if none does or the checks are off.  Synchronises the stream.
int check_values(std::initializer_list<ValueRange> vals, void* stream, int bad)
{
    if (!check_values_on()) return MESA_OK;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxFlagDevices) return MESA_ERR_HIP;
    int* flag = nullptr;
    {
        std::lock_guard<std::mutex> lock(g_flag_mutex);
        if (g_flag_ptr[dev] == nullptr) {
            void* ptr = nullptr;
            if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(value_flag)) != hipSuccess || ptr == nullptr) return MESA_ERR_HIP;
            g_flag_ptr[dev] = static_cast<int*>(ptr);
        }
        flag = g_flag_ptr[dev];
    }
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipLaunchKernelGGL(value_flag_clear_kernel, dim3(1), dim3(64), 0, s, flag);
    for (const ValueRange& v : vals) {
        if (v.p == nullptr || v.n <= 0) continue;
        const int64_t blocks = std::min<int64_t>((v.n + 255) / 256, 1024);
        hipLaunchKernelGGL(value_range_kernel, dim3(unsigned(blocks)), dim3(256), 0, s, v.p, v.n, int(v.bf16), v.lo,
                           v.hi, flag);
    }
    if (hipGetLastError() != hipSuccess) return MESA_ERR_HIP;
    int h = 0;
    if (hipMemcpyAsync(&h, flag, sizeof(int), hipMemcpyDeviceToHost, s) != hipSuccess) return MESA_ERR_HIP;
    if (hipStreamSynchronize(s) != hipSuccess) return MESA_ERR_HIP;
    return h ? bad : MESA_OK;
}

int check_sizes(int64_t batch, int64_t heads, int64_t seq_len, int64_t d_k, int64_t d_v,
                int dtype, int n_cg)
{
    if (batch < 0 || heads < 0 || seq_len < 0 || d_k < 0 || d_v < 0) return MESA_ERR_SHAPE;
    if (!dim_ok(d_k) || !dim_ok(d_v)) return MESA_ERR_UNSUPPORTED;
    if (dtype != MESA_DTYPE_F32 && dtype != MESA_DTYPE_BF16) return MESA_ERR_UNSUPPORTED;
    if (n_cg < 0 || n_cg > MESA_MAX_NCG) return MESA_ERR_ARG;
    // Grid sizes are 32-bit: batch * heads * chunks (and tiles) must stay well inside.
    if (batch > 0 && heads > (int64_t(1) << 30) / batch) return MESA_ERR_SHAPE;
    return MESA_OK;
}

}  // namespace

namespace {

// fp32 bytes of the states entering every chunk (H_c then G_c), 0 for unsupported or
// empty sizes.
size_t states_bytes(int64_t batch, int64_t heads, int64_t seq_len, int64_t d_k, int64_t d_v, int chunk)
{
    if (batch <= 0 || heads <= 0 || seq_len <= 0) return 0;
    if (!dim_ok(d_k) || !dim_ok(d_v) || !chunk_ok(chunk)) return 0;
    const int64_t nc = n_chunks_of(seq_len, chunk);
    return size_t(batch) * size_t(heads) * size_t(nc) * size_t(d_k) * size_t(d_k + d_v) * sizeof(float);
}

// Checks shared by the forward entry points.  `need_ws` is the workspace the
// call reads or writes (0 when it uses none).  Returns a status code.
struct FwdCall {
    const void *q, *k, *v;
    const float *gamma, *beta, *lambda;
    int64_t batch, heads, seq_len, d_k, d_v;
    int dtype, n_cg, chunk, precision;
    float *out, *qstar, *final_H, *final_G;
    const void* workspace;
    size_t workspace_bytes;
    bool needs_q;       // the solve reads q and lambda
    bool needs_ws;      // the call uses the chunk-state workspace
    float eps = 0.0f;            // CG relative tolerance (0: fixed steps)
    int32_t* steps = nullptr;    // per-token CG iterations, may be NULL
};

bool eps_ok(float eps) { return isfinite(eps) && eps >= 0.0f; }

int validate_forward(const FwdCall& c)
{
    int st = check_sizes(c.batch, c.heads, c.seq_len, c.d_k, c.d_v, c.dtype, c.n_cg);
    if (st != MESA_OK) return st;
    if (!eps_ok(c.eps)) return MESA_ERR_ARG;
    if (!chunk_ok(c.chunk)) return MESA_ERR_UNSUPPORTED;
    if (c.precision != MESA_PREC_AUTO && c.precision != MESA_PREC_F32 && c.precision != MESA_PREC_BF16 &&
        c.precision != MESA_PREC_BF16X3)
        return MESA_ERR_UNSUPPORTED;
    const ForwardShape probe{c.batch, c.heads, c.seq_len, int(c.d_k), int(c.d_v), c.chunk, 0,
                             c.dtype == MESA_DTYPE_BF16};
    if (c.precision == MESA_PREC_BF16 && !mesa::chunk_cg_bf16_supported(probe)) return MESA_ERR_UNSUPPORTED;
    if (c.precision == MESA_PREC_BF16X3 && !mesa::chunk_cg_x3_supported(probe)) return MESA_ERR_UNSUPPORTED;
    if (c.batch == 0 || c.heads == 0) return MESA_OK;
    // Arrays with no elements (seq_len == 0) may be NULL; lambda never is empty.
    if (c.seq_len > 0 && (!c.k || !c.v || !c.gamma || !c.beta)) return MESA_ERR_NULL;
    if (c.needs_q && (!c.lambda || (c.seq_len > 0 && (!c.q || !c.out)))) return MESA_ERR_NULL;
    const int64_t nc = n_chunks_of(c.seq_len, c.chunk);
    if (nc * c.batch * c.heads > (int64_t(1) << 31) / 16) return MESA_ERR_SHAPE;
    // The kernels move q, k, v, Lambda, states and outputs with 16-byte accesses.
    for (const void* ptr : {c.q, c.k, c.v, static_cast<const void*>(c.lambda), static_cast<const void*>(c.out),
                            static_cast<const void*>(c.qstar), static_cast<const void*>(c.final_H),
                            static_cast<const void*>(c.final_G), c.workspace})
        if (uintptr_t(ptr) % 16 != 0) return MESA_ERR_ARG;
    if (uintptr_t(c.steps) % 4 != 0) return MESA_ERR_ARG;
    const size_t need = c.needs_ws ? mesa_forward_workspace_bytes(c.batch, c.heads, c.seq_len, c.d_k,
                                                                  c.d_v, c.chunk)
                                   : 0;
    if (need > 0) {
        if (!c.workspace) return MESA_ERR_NULL;
        if (c.workspace_bytes < need) return MESA_ERR_WORKSPACE;
    }
    const int64_t tokens = c.batch * c.heads * c.seq_len;
    const int64_t in_sz = c.dtype == MESA_DTYPE_BF16 ? 2 : 4;
    // Outputs must overlap neither an input nor each other.  The workspace is an
    // output of the state scan and an input of the solve; either way no other
    // output may touch it.
    const Range ins[] = {range_of(c.q, c.q ? tokens * c.d_k * in_sz : 0),
                         range_of(c.k, tokens * c.d_k * in_sz),
                         range_of(c.v, tokens * c.d_v * in_sz),
                         range_of(c.gamma, tokens * 4),
                         range_of(c.beta, tokens * 4),
                         range_of(c.lambda, c.lambda ? c.heads * c.d_k * 4 : 0),
                         range_of(c.workspace, int64_t(need))};
    const Range outs[] = {range_of(c.out, c.out ? tokens * c.d_v * 4 : 0),
                          range_of(c.qstar, c.qstar ? tokens * c.d_k * 4 : 0),
                          range_of(c.final_H, c.final_H ? c.batch * c.heads * c.d_k * c.d_k * 4 : 0),
                          range_of(c.final_G, c.final_G ? c.batch * c.heads * c.d_v * c.d_k * 4 : 0),
                          range_of(c.steps, c.steps ? tokens * 4 : 0)};
    for (const Range& o : outs) {
        if (o.lo == o.hi) continue;
        for (const Range& i : ins)
            if (i.lo != i.hi && overlaps(o, i)) return MESA_ERR_ARG;
    }
    for (int x = 0; x < 5; ++x)
        for (int y = x + 1; y < 5; ++y)
            if (outs[x].lo != outs[x].hi && outs[y].lo != outs[y].hi && overlaps(outs[x], outs[y]))
                return MESA_ERR_ARG;
    return MESA_OK;
}

// MESA_CHECK_FINITE: the forward's inputs (before its launches) and outputs (after them)
int check_forward_inputs(const FwdCall& c, void* stream)
{
    const int64_t nt = c.batch * c.heads * c.seq_len;
    const bool b16 = c.dtype == MESA_DTYPE_BF16;
    return check_values({{c.needs_q ? c.q : nullptr, nt * c.d_k, b16, -kFinite, kFinite},
                         {c.k, nt * c.d_k, b16, -kFinite, kFinite}, {c.v, nt * c.d_v, b16, -kFinite, kFinite},
                         {c.gamma, nt, false, 0.0f, 1.0f}, {c.beta, nt, false, 0.0f, 1.0f},
                         {c.needs_q ? c.lambda : nullptr, c.heads * c.d_k, false, FLT_MIN, kFinite}},
                        stream, MESA_ERR_ARG);
}
int check_forward_outputs(const FwdCall& c, void* stream)
{
    const int64_t nt = c.batch * c.heads * c.seq_len, bh = c.batch * c.heads;
    return check_values({{c.out, nt * c.d_v, false, -kFinite, kFinite}, {c.qstar, nt * c.d_k, false, -kFinite, kFinite},
                         {c.final_H, bh * c.d_k * c.d_k, false, -kFinite, kFinite},
                         {c.final_G, bh * c.d_v * c.d_k, false, -kFinite, kFinite}},
                        stream, MESA_ERR_NONFINITE);
}

ForwardShape shape_of(const FwdCall& c)
{
    return ForwardShape{c.batch, c.heads, c.seq_len, int(c.d_k), int(c.d_v), c.chunk,
                        int(n_chunks_of(c.seq_len, c.chunk)), c.dtype == MESA_DTYPE_BF16};
}

// The solve path a call resolves to.  The state scan and the solve of one
// forward must resolve to the same path: it fixes the workspace layout.
int resolve_precision(const FwdCall& c)
{
    const ForwardShape s = shape_of(c);
    if (c.precision == MESA_PREC_AUTO)
        return s.bf16 && mesa::chunk_cg_x3_supported(s) ? MESA_PREC_BF16X3 : MESA_PREC_F32;
    return c.precision;
}

// Workspace: H states then G states, fp32 plain (MESA_PREC_F32), bf16 fragments
// (MESA_PREC_BF16, half the bytes) or the split-operand layout (MESA_PREC_BF16X3: fp32
// H_c fragments, then G_c's bf16 high and low planes).
void* ws_H(const FwdCall& c) { return const_cast<void*>(c.workspace); }
void* ws_G(const FwdCall& c)
{
    const ForwardShape s = shape_of(c);
    const size_t elem = resolve_precision(c) == MESA_PREC_BF16 ? 2 : 4;
    return static_cast<char*>(ws_H(c)) + size_t(s.batch * s.heads * s.n_chunks) * size_t(s.d_k) * size_t(s.d_k) * elem;
}

int launch_states(const FwdCall& c, bool store_chunks, hipStream_t s)
{
    if (c.seq_len == 0) {
        // No tokens: the final states are the initial ones, H_0 = G_0 = 0.
        if (c.final_H && mesa::launch_fill_zero(c.final_H, c.batch * c.heads * c.d_k * c.d_k, s) != hipSuccess)
            return MESA_ERR_HIP;
        if (c.final_G && mesa::launch_fill_zero(c.final_G, c.batch * c.heads * c.d_v * c.d_k, s) != hipSuccess)
            return MESA_ERR_HIP;
        return MESA_OK;
    }
    const bool frag = store_chunks && resolve_precision(c) == MESA_PREC_BF16;
    mesa::StateArgs sa{shape_of(c), c.k, c.v, c.gamma, c.beta,
                       store_chunks ? ws_H(c) : nullptr, store_chunks ? ws_G(c) : nullptr,
                       c.final_H, c.final_G, store_chunks, frag};
    sa.x3 = store_chunks && resolve_precision(c) == MESA_PREC_BF16X3;
    // The bf16 chunk states fill half of the workspace (and a states-only call none
    // of it): the other half is scratch for the segmented scan of few sequences.
    if (c.workspace && (frag || !store_chunks)) {
        const size_t full = mesa_forward_workspace_bytes(c.batch, c.heads, c.seq_len, c.d_k, c.d_v, c.chunk);
        sa.seg_ws = reinterpret_cast<float*>(static_cast<char*>(const_cast<void*>(c.workspace)) + full / 2);
        sa.seg_bytes = full - full / 2;
    } else if (sa.x3 && c.workspace) {
        // the split-operand states fill the fp32-sized part: the segment totals go after it
        const size_t states = states_bytes(c.batch, c.heads, c.seq_len, c.d_k, c.d_v, c.chunk);
        const size_t full = mesa_forward_workspace_bytes(c.batch, c.heads, c.seq_len, c.d_k, c.d_v, c.chunk);
        if (full > states) {
            sa.seg_ws = reinterpret_cast<float*>(static_cast<char*>(const_cast<void*>(c.workspace)) + states);
            sa.seg_bytes = full - states;
        }
    }
    return mesa::launch_chunk_state(sa, s) == hipSuccess ? MESA_OK : MESA_ERR_HIP;
}

int launch_solve(const FwdCall& c, hipStream_t s)
{
    if (c.seq_len == 0) return MESA_OK;
    const ForwardShape shape = shape_of(c);
    const int prec = resolve_precision(c);
    mesa::CgArgs ca{shape, c.q, c.k, c.v, c.gamma, c.beta, c.lambda, ws_H(c), ws_G(c), c.n_cg, c.out, c.qstar,
                    c.eps * c.eps, c.steps};
    const hipError_t e = prec == MESA_PREC_BF16     ? mesa::launch_chunk_cg_bf16(ca, s)
                         : prec == MESA_PREC_BF16X3 ? mesa::launch_chunk_cg_x3(ca, s)
                                                    : mesa::launch_chunk_cg_f32(ca, s);
    return e == hipSuccess ? MESA_OK : MESA_ERR_HIP;
}

}  // namespace

extern "C" {

int mesa_version(void) { return 101; }

const char* mesa_status_string(int status)
{
    switch (status) {
        case MESA_OK: return "ok";
        case MESA_ERR_NULL: return "a required pointer is NULL";
        case MESA_ERR_SHAPE: return "a size is negative or the sizes are inconsistent";
        case MESA_ERR_UNSUPPORTED: return "d_k, d_v, chunk, dtype or precision not supported";
        case MESA_ERR_ARG: return "n_cg or eps out of range, a misaligned pointer, or an output overlapping an input";
        case MESA_ERR_WORKSPACE: return "workspace too small";
        case MESA_ERR_HIP: return "the HIP runtime refused a launch";
        case MESA_ERR_NONFINITE: return "an output holds a NaN or an infinity (MESA_CHECK_FINITE)";
        default: return "unknown status";
    }
}

size_t mesa_forward_workspace_bytes(int64_t batch, int64_t heads, int64_t seq_len, int64_t d_k,
                                    int64_t d_v, int chunk)
{
    const size_t states = states_bytes(batch, heads, seq_len, d_k, d_v, chunk);
    if (states == 0) return 0;
    // Few long sequences (at most 64, at least 16 chunks each) are scanned in segments
    // (at most 128 segment totals in all, none for a sequence's last segment, and at most
    // one per 8 chunks): room for the totals and the segment decays after the states.
    const int64_t bh = batch * heads, nc = n_chunks_of(seq_len, chunk);
    if (bh > 64 || nc < 16) return states;
    const int64_t totals = std::min<int64_t>(bh * (nc / 8), 128);
    return states + size_t(totals) * size_t(d_k) * size_t(d_k + d_v) * sizeof(float) + 128 * sizeof(float);
}

int mesa_forward_ex(const void* q, const void* k, const void* v, const float* gamma,
                    const float* beta, const float* lambda, int64_t batch, int64_t heads,
                    int64_t seq_len, int64_t d_k, int64_t d_v, int dtype, int n_cg, int chunk,
                    int precision, float* out, float* qstar_out, float* final_H, float* final_G,
                    void* workspace, size_t workspace_bytes, void* stream)
{
    const bool states_only = out == nullptr;
    if (states_only && (qstar_out || !final_H || !final_G)) return MESA_ERR_NULL;
    // a states-only call uses the workspace (as scratch) only when one is given
    FwdCall c{q, k, v, gamma, beta, lambda, batch, heads, seq_len, d_k, d_v, dtype, n_cg, chunk,
              precision, out, qstar_out, final_H, final_G, workspace, workspace_bytes,
              !states_only, !states_only || workspace != nullptr};
    int st = validate_forward(c);
    if (st != MESA_OK || batch == 0 || heads == 0) return st;
    st = check_forward_inputs(c, stream);
    if (st != MESA_OK) return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    st = launch_states(c, !states_only, s);
    if (st == MESA_OK && !states_only) st = launch_solve(c, s);
    st = finish(st, stream);
    return st == MESA_OK ? check_forward_outputs(c, stream) : st;
}

int mesa_forward(const void* q, const void* k, const void* v, const float* gamma,
                 const float* beta, const float* lambda, int64_t batch, int64_t heads,
                 int64_t seq_len, int64_t d_k, int64_t d_v, int dtype, int n_cg, int chunk,
                 float* out, void* workspace, size_t workspace_bytes, void* stream)
{
    if (!out) return MESA_ERR_NULL;
    return mesa_forward_ex(q, k, v, gamma, beta, lambda, batch, heads, seq_len, d_k, d_v, dtype,
                           n_cg, chunk, MESA_PREC_AUTO, out, nullptr, nullptr, nullptr, workspace,
                           workspace_bytes, stream);
}

int mesa_forward_states(const void* k, const void* v, const float* gamma, const float* beta,
                        int64_t batch, int64_t heads, int64_t seq_len, int64_t d_k, int64_t d_v,
                        int dtype, int chunk, int precision, float* final_H, float* final_G,
                        void* workspace, size_t workspace_bytes, void* stream)
{
    FwdCall c{nullptr, k, v, gamma, beta, nullptr, batch, heads, seq_len, d_k, d_v, dtype, 0, chunk,
              precision, nullptr, nullptr, final_H, final_G, workspace, workspace_bytes, false,
              true};
    int st = validate_forward(c);
    if (st != MESA_OK || batch == 0 || heads == 0) return st;
    return finish(launch_states(c, true, static_cast<hipStream_t>(stream)), stream);
}

int mesa_forward_solve(const void* q, const void* k, const void* v, const float* gamma,
                       const float* beta, const float* lambda, int64_t batch, int64_t heads,
                       int64_t seq_len, int64_t d_k, int64_t d_v, int dtype, int n_cg, int chunk,
                       int precision, float* out, float* qstar_out, const void* workspace,
                       size_t workspace_bytes, void* stream)
{
    FwdCall c{q, k, v, gamma, beta, lambda, batch, heads, seq_len, d_k, d_v, dtype, n_cg, chunk,
              precision, out, qstar_out, nullptr, nullptr, workspace, workspace_bytes, true, true};
    int st = validate_forward(c);
    if (st != MESA_OK || batch == 0 || heads == 0) return st;
    return finish(launch_solve(c, static_cast<hipStream_t>(stream)), stream);
}

int mesa_decode_step(float* state_H, float* state_G, const void* q, const void* k, const void* v,
                     const float* gamma, const float* beta, const float* lambda, int64_t batch,
                     int64_t heads, int64_t d_k, int64_t d_v, int dtype, int n_cg, float* out,
                     void* stream)
{
    return mesa_decode_step_tol(state_H, state_G, q, k, v, gamma, beta, lambda, batch, heads, d_k, d_v,
                                dtype, n_cg, 0.0f, out, nullptr, stream);
}

}  // extern "C"

namespace {

int decode_step(float* state_H, float* state_G, const void* q, const void* k, const void* v,
                const float* gamma, const float* beta, const float* lambda, int64_t batch, int64_t heads,
                int64_t d_k, int64_t d_v, int dtype, int max_cg, float eps, float* out, int32_t* steps_out,
                bool packed, void* stream)
{
    int st = check_sizes(batch, heads, 1, d_k, d_v, dtype, max_cg);
    if (st != MESA_OK) return st;
    if (!eps_ok(eps)) return MESA_ERR_ARG;
    if (batch == 0 || heads == 0) return MESA_OK;
    if (!state_H || !state_G || !q || !k || !v || !gamma || !beta || !lambda || !out)
        return MESA_ERR_NULL;
    if (uintptr_t(steps_out) % 4 != 0) return MESA_ERR_ARG;
    const int64_t pairs = batch * heads;
    if (pairs > (int64_t(1) << 31) - 1) return MESA_ERR_SHAPE;
    const int64_t in_sz = dtype == MESA_DTYPE_BF16 ? 2 : 4;
    {
        const Range ins[] = {range_of(q, pairs * d_k * in_sz), range_of(k, pairs * d_k * in_sz),
                             range_of(v, pairs * d_v * in_sz), range_of(gamma, pairs * 4),
                             range_of(beta, pairs * 4), range_of(lambda, heads * d_k * 4)};
        const int64_t h_rows = packed ? d_k / 2 + 1 : d_k;
        const Range outs[] = {range_of(state_H, pairs * h_rows * d_k * 4),
                              range_of(state_G, pairs * d_v * d_k * 4), range_of(out, pairs * d_v * 4),
                              range_of(steps_out, steps_out ? pairs * 4 : 0)};
        for (const Range& o : outs) {
            if (o.lo == o.hi) continue;
            for (const Range& i : ins)
                if (overlaps(o, i)) return MESA_ERR_ARG;
        }
        for (int x = 0; x < 4; ++x)
            for (int y = x + 1; y < 4; ++y)
                if (outs[x].lo != outs[x].hi && outs[y].lo != outs[y].hi && overlaps(outs[x], outs[y]))
                    return MESA_ERR_ARG;
    }
    const bool b16 = dtype == MESA_DTYPE_BF16;
    const int64_t h_elems = pairs * (packed ? d_k / 2 + 1 : d_k) * d_k, g_elems = pairs * d_v * d_k;
    st = check_values({{q, pairs * d_k, b16, -kFinite, kFinite}, {k, pairs * d_k, b16, -kFinite, kFinite},
                       {v, pairs * d_v, b16, -kFinite, kFinite}, {gamma, pairs, false, 0.0f, 1.0f},
                       {beta, pairs, false, 0.0f, 1.0f}, {lambda, heads * d_k, false, FLT_MIN, kFinite},
                       {state_H, h_elems, false, -kFinite, kFinite}, {state_G, g_elems, false, -kFinite, kFinite}},
                      stream, MESA_ERR_ARG);
    if (st != MESA_OK) return st;
    mesa::DecodeArgs da{batch, heads, int(d_k), int(d_v), b16, state_H, state_G,
                        q, k, v, gamma, beta, lambda, max_cg, out, eps * eps, steps_out, packed};
    st = finish(mesa::launch_decode_step(da, static_cast<hipStream_t>(stream)) == hipSuccess ? MESA_OK : MESA_ERR_HIP,
                stream);
    if (st != MESA_OK) return st;
    return check_values({{out, pairs * d_v, false, -kFinite, kFinite}, {state_H, h_elems, false, -kFinite, kFinite},
                         {state_G, g_elems, false, -kFinite, kFinite}},
                        stream, MESA_ERR_NONFINITE);
}

// pack (to_packed) or unpack the symmetric decode state H of batch x heads pairs
int convert_state(const float* src, float* dst, int64_t batch, int64_t heads, int64_t d_k, bool to_packed,
                  void* stream)
{
    if (batch < 0 || heads < 0 || d_k < 0) return MESA_ERR_SHAPE;
    if (!dim_ok(d_k)) return MESA_ERR_UNSUPPORTED;
    if (batch > 0 && heads > (int64_t(1) << 30) / batch) return MESA_ERR_SHAPE;
    const int64_t pairs = batch * heads;
    if (pairs == 0) return MESA_OK;
    if (!src || !dst) return MESA_ERR_NULL;
    const int64_t full = pairs * d_k * d_k * 4, pk = pairs * (d_k / 2 + 1) * d_k * 4;
    if (overlaps(range_of(src, to_packed ? full : pk), range_of(dst, to_packed ? pk : full))) return MESA_ERR_ARG;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const hipError_t e = to_packed ? mesa::launch_pack_state(src, dst, pairs, int(d_k), s)
                                   : mesa::launch_unpack_state(src, dst, pairs, int(d_k), s);
    return finish(e == hipSuccess ? MESA_OK : MESA_ERR_HIP, stream);
}

}  // namespace

extern "C" {

int mesa_decode_step_tol(float* state_H, float* state_G, const void* q, const void* k, const void* v,
                         const float* gamma, const float* beta, const float* lambda, int64_t batch,
                         int64_t heads, int64_t d_k, int64_t d_v, int dtype, int max_cg, float eps,
                         float* out, int32_t* steps_out, void* stream)
{
    return decode_step(state_H, state_G, q, k, v, gamma, beta, lambda, batch, heads, d_k, d_v, dtype, max_cg, eps,
                       out, steps_out, false, stream);
}

int mesa_decode_step_packed(float* state_HP, float* state_G, const void* q, const void* k, const void* v,
                            const float* gamma, const float* beta, const float* lambda, int64_t batch,
                            int64_t heads, int64_t d_k, int64_t d_v, int dtype, int max_cg, float eps,
                            float* out, int32_t* steps_out, void* stream)
{
    return decode_step(state_HP, state_G, q, k, v, gamma, beta, lambda, batch, heads, d_k, d_v, dtype, max_cg, eps,
                       out, steps_out, true, stream);
}

int mesa_pack_state(const float* state_H, float* state_HP, int64_t batch, int64_t heads, int64_t d_k, void* stream)
{
    return convert_state(state_H, state_HP, batch, heads, d_k, true, stream);
}

int mesa_unpack_state(const float* state_HP, float* state_H, int64_t batch, int64_t heads, int64_t d_k, void* stream)
{
    return convert_state(state_HP, state_H, batch, heads, d_k, false, stream);
}

int mesa_forward_tol(const void* q, const void* k, const void* v, const float* gamma,
                     const float* beta, const float* lambda, int64_t batch, int64_t heads,
                     int64_t seq_len, int64_t d_k, int64_t d_v, int dtype, int max_cg, float eps,
                     int chunk, int precision, float* out, float* qstar_out, int32_t* steps_out,
                     void* workspace, size_t workspace_bytes, void* stream)
{
    if (!out) return MESA_ERR_NULL;
    FwdCall c{q, k, v, gamma, beta, lambda, batch, heads, seq_len, d_k, d_v, dtype, max_cg, chunk,
              precision, out, qstar_out, nullptr, nullptr, workspace, workspace_bytes, true, true,
              eps, steps_out};
    int st = validate_forward(c);
    if (st != MESA_OK || batch == 0 || heads == 0) return st;
    st = check_forward_inputs(c, stream);
    if (st != MESA_OK) return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    st = launch_states(c, true, s);
    if (st == MESA_OK) st = launch_solve(c, s);
    st = finish(st, stream);
    return st == MESA_OK ? check_forward_outputs(c, stream) : st;
}

}  // extern "C"

namespace {

constexpr int kBwdChunk = 64;  // the backward's own chunking (independent of the forward's)

// Backward workspace: fp32 forward chunk states H_c, G_c; the fp32 adjoints S^H,
// A^G arriving at every chunk's end; the fp32 right-hand sides u; per-chunk dLambda
// sums; then, for the matrix-core solve, the bf16 chunk states (fragment layout) and
// u rounded to bf16.
struct BwdLayout {
    int64_t nc, hs, gs, sh, ag, u, dl, fh, fg, u16, total;  // byte offsets and total
};
BwdLayout bwd_layout(int64_t batch, int64_t heads, int64_t seq_len, int64_t d_k, int64_t d_v)
{
    BwdLayout L;
    const int64_t bh = batch * heads;
    L.nc = n_chunks_of(seq_len, kBwdChunk);
    const int64_t nH = bh * L.nc * d_k * d_k, nG = bh * L.nc * d_v * d_k;
    L.hs = 0;
    L.gs = L.hs + 4 * nH;
    L.sh = L.gs + 4 * nG;
    L.ag = L.sh + 4 * nH;
    L.u = L.ag + 4 * nG;
    L.dl = L.u + 4 * bh * seq_len * d_k;
    L.fh = L.dl + 4 * bh * L.nc * d_k;
    L.fg = L.fh + 2 * nH;
    L.u16 = L.fg + 2 * nG;
    L.total = L.u16 + 2 * bh * seq_len * d_k;
    L.total = (L.total + 15) / 16 * 16;
    return L;
}

}  // namespace

extern "C" {

size_t mesa_backward_workspace_bytes(int64_t batch, int64_t heads, int64_t seq_len, int64_t d_k, int64_t d_v)
{
    if (batch <= 0 || heads <= 0 || seq_len <= 0) return 0;
    if (!dim_ok(d_k) || !dim_ok(d_v)) return 0;
    return size_t(bwd_layout(batch, heads, seq_len, d_k, d_v).total);
}

}  // extern "C"

namespace {

int backward_launch(const void* k, const void* v, const float* gamma, const float* beta, const float* lambda,
                    int64_t batch, int64_t heads, int64_t seq_len, int64_t d_k, int64_t d_v, int dtype, int n_cg,
                    int precision, const float* qstar, const float* dout, float* dq, float* dk, float* dv,
                    float* dgamma, float* dbeta, float* dlambda, void* workspace, size_t workspace_bytes,
                    void* stream, bool& launched)
{
    launched = false;
    int st = check_sizes(batch, heads, seq_len, d_k, d_v, dtype, n_cg);
    if (st != MESA_OK) return st;
    if (precision != MESA_PREC_AUTO && precision != MESA_PREC_F32 && precision != MESA_PREC_BF16)
        return MESA_ERR_UNSUPPORTED;
    const mesa::ForwardShape probe{batch, heads, seq_len, int(d_k), int(d_v), kBwdChunk, 0, dtype == MESA_DTYPE_BF16};
    const bool cg_bf16 = mesa::chunk_cg_bf16_supported(probe);
    if (precision == MESA_PREC_BF16 && !cg_bf16) return MESA_ERR_UNSUPPORTED;
    const bool use_bf16 = precision == MESA_PREC_BF16 || (precision == MESA_PREC_AUTO && cg_bf16);
    if (batch == 0 || heads == 0) return MESA_OK;
    if (!lambda || !dlambda) return MESA_ERR_NULL;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int64_t bh = batch * heads, tokens = bh * seq_len;
    if (seq_len > 0) {
        if (!k || !v || !gamma || !beta || !qstar || !dout || !dq || !dk || !dv || !dgamma || !dbeta)
            return MESA_ERR_NULL;
        if (n_chunks_of(seq_len, kBwdChunk) * bh > (int64_t(1) << 31) / 16) return MESA_ERR_SHAPE;
        const size_t need = mesa_backward_workspace_bytes(batch, heads, seq_len, d_k, d_v);
        if (!workspace) return MESA_ERR_NULL;
        if (workspace_bytes < need) return MESA_ERR_WORKSPACE;
        for (const void* ptr : {k, v, static_cast<const void*>(qstar), static_cast<const void*>(dout),
                                static_cast<const void*>(dq), static_cast<const void*>(workspace)})
            if (uintptr_t(ptr) % 16 != 0) return MESA_ERR_ARG;
        const int64_t in_sz = dtype == MESA_DTYPE_BF16 ? 2 : 4;
        const Range ins[] = {range_of(k, tokens * d_k * in_sz), range_of(v, tokens * d_v * in_sz),
                             range_of(gamma, tokens * 4), range_of(beta, tokens * 4),
                             range_of(lambda, heads * d_k * 4), range_of(qstar, tokens * d_k * 4),
                             range_of(dout, tokens * d_v * 4), range_of(workspace, int64_t(need))};
        const Range outs[] = {range_of(dq, tokens * d_k * 4), range_of(dk, tokens * d_k * 4),
                              range_of(dv, tokens * d_v * 4), range_of(dgamma, tokens * 4),
                              range_of(dbeta, tokens * 4), range_of(dlambda, heads * d_k * 4)};
        for (const Range& o : outs)
            for (const Range& i : ins)
                if (overlaps(o, i)) return MESA_ERR_ARG;
        for (int x = 0; x < 6; ++x)
            for (int y = x + 1; y < 6; ++y)
                if (overlaps(outs[x], outs[y])) return MESA_ERR_ARG;
    } else if (overlaps(range_of(dlambda, heads * d_k * 4), range_of(lambda, heads * d_k * 4))) {
        return MESA_ERR_ARG;
    }
    launched = true;
    if (seq_len == 0)  // no tokens: dLambda is an empty sum
        return mesa::launch_fill_zero(dlambda, heads * d_k, s) == hipSuccess ? MESA_OK : MESA_ERR_HIP;

    const BwdLayout L = bwd_layout(batch, heads, seq_len, d_k, d_v);
    char* base = static_cast<char*>(workspace);
    auto f32_at = [&](int64_t off) { return reinterpret_cast<float*>(base + off); };
    auto u16_at = [&](int64_t off) { return reinterpret_cast<uint16_t*>(base + off); };
    const mesa::ForwardShape shape{batch, heads, seq_len, int(d_k), int(d_v), kBwdChunk, int(L.nc),
                                   dtype == MESA_DTYPE_BF16};
    // forward chunk states (fp32, plain layout), and for the matrix-core solve the bf16
    // fragment states as the forward's solve reads them
    if (use_bf16) {
        // one pass: bf16 fragments for the solve and fp32 plain states for the gradients;
        // the adjoint region, written only later, is the scratch of a segmented walk
        mesa::StateArgs fa{shape, k, v, gamma, beta, u16_at(L.fh), u16_at(L.fg), nullptr, nullptr, true, true};
        fa.Hs32 = f32_at(L.hs);
        fa.Gs32 = f32_at(L.gs);
        fa.seg_ws = f32_at(L.sh);
        fa.seg_bytes = size_t(L.u - L.sh);
        if (mesa::launch_chunk_state(fa, s) != hipSuccess) return MESA_ERR_HIP;
    } else {
        mesa::StateArgs sa{shape, k, v, gamma, beta, f32_at(L.hs), f32_at(L.gs), nullptr, nullptr, true, false};
        if (mesa::launch_chunk_state(sa, s) != hipSuccess) return MESA_ERR_HIP;
    }
    mesa::BwdArgs ba{shape, k, v, gamma, beta, qstar, dout, dq, f32_at(L.hs), f32_at(L.gs), f32_at(L.sh),
                     f32_at(L.ag), f32_at(L.u), use_bf16 ? u16_at(L.u16) : nullptr, dk, dv, dgamma, dbeta,
                     f32_at(L.dl), dlambda};
    // u_t = G_t^T e_t, then e*_t = (H_t + Lambda)^{-1} u_t into dq: on the matrix cores
    // (bf16 operands, u rounded to bf16, no read-out) or with fp32 products
    if (mesa::launch_backward_stage(ba, 0, s) != hipSuccess) return MESA_ERR_HIP;
    if (use_bf16) {
        mesa::CgArgs ca{shape, u16_at(L.u16), k, v, gamma, beta, lambda, u16_at(L.fh), u16_at(L.fg), n_cg,
                        nullptr, dq, 0.0f, nullptr};
        if (mesa::launch_chunk_cg_bf16(ca, s) != hipSuccess) return MESA_ERR_HIP;
    } else {
        mesa::CgArgs ca{shape, nullptr, k, v, gamma, beta, lambda, f32_at(L.hs), f32_at(L.gs), n_cg, nullptr, dq,
                        0.0f, nullptr, f32_at(L.u)};
        if (mesa::launch_chunk_cg_f32(ca, s) != hipSuccess) return MESA_ERR_HIP;
    }
    for (int stage = 1; stage <= 3; ++stage)
        if (mesa::launch_backward_stage(ba, stage, s) != hipSuccess) return MESA_ERR_HIP;
    return MESA_OK;
}

}  // namespace

extern "C" {

int mesa_backward(const void* k, const void* v, const float* gamma, const float* beta, const float* lambda,
                  int64_t batch, int64_t heads, int64_t seq_len, int64_t d_k, int64_t d_v, int dtype, int n_cg,
                  int precision, const float* qstar, const float* dout, float* dq, float* dk, float* dv,
                  float* dgamma, float* dbeta, float* dlambda, void* workspace, size_t workspace_bytes,
                  void* stream)
{
    bool launched = false;
    const int st = backward_launch(k, v, gamma, beta, lambda, batch, heads, seq_len, d_k, d_v, dtype, n_cg,
                                   precision, qstar, dout, dq, dk, dv, dgamma, dbeta, dlambda, workspace,
                                   workspace_bytes, stream, launched);
    return launched ? finish(st, stream) : st;
}

}  // extern "C"

namespace {

// Chunk-state workspace of mesa_forward_noalloc: a fixed buffer in device memory
// that comes with the library's code object, so each GPU the library runs on holds
// one copy until the process ends.  In host code its name is only a stand-in for
// the symbol: kernels get the device address that hipGetSymbolAddress returns on
// the current device (each device's copy has its own address), never the name.
// Nothing in it has to start at zero: the chunk-state scan writes every state (and
// every segment total of the segmented scan) before anything reads it.
__device__ __align__(256) unsigned char scratch[MESA_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of `scratch` on the current device, looked up on the first call
// per device (with that device current) and kept.
int scratch_address(void** ptr)
{
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return MESA_ERR_HIP;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (g_scratch_ptr[dev] == nullptr) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return MESA_ERR_HIP;
        g_scratch_ptr[dev] = p;
    }
    *ptr = g_scratch_ptr[dev];
    return MESA_OK;
}

}  // namespace

extern "C" {

int mesa_forward_noalloc(const void* q, const void* k, const void* v, const float* gamma,
                         const float* beta, const float* lambda, int64_t batch, int64_t heads,
                         int64_t seq_len, int64_t d_k, int64_t d_v, int dtype, int n_cg, int chunk,
                         float* out, void* stream)
{
    if (!out) return MESA_ERR_NULL;
    // every argument check except the workspace's, before the device is touched
    FwdCall c{q, k, v, gamma, beta, lambda, batch, heads, seq_len, d_k, d_v, dtype, n_cg, chunk,
              MESA_PREC_AUTO, out, nullptr, nullptr, nullptr, nullptr, 0, true, false};
    int st = validate_forward(c);
    if (st != MESA_OK || batch == 0 || heads == 0) return st;
    const size_t need = mesa_forward_workspace_bytes(batch, heads, seq_len, d_k, d_v, chunk);
    if (need > size_t(MESA_NOALLOC_SCRATCH_BYTES)) return MESA_ERR_WORKSPACE;
    if (need > 0) {
        st = scratch_address(const_cast<void**>(&c.workspace));
        if (st != MESA_OK) return st;
        c.workspace_bytes = MESA_NOALLOC_SCRATCH_BYTES;
        c.needs_ws = true;
        st = validate_forward(c);
        if (st != MESA_OK) return st;
    }
    hipStream_t s = static_cast<hipStream_t>(stream);
    st = launch_states(c, true, s);
    if (st == MESA_OK) st = launch_solve(c, s);
    return finish(st, stream);
}

}  // extern "C"

extern "C" {

int mesa_frontend(const void* qp, const void* kp, const void* vp, const float* conv_q, const float* conv_k,
                  const float* conv_v, const float* a_gamma, const float* a_beta, const float* theta,
                  float gamma_cap, float l2_eps, int64_t batch, int64_t heads, int64_t seq_len, int64_t d_k,
                  int64_t d_v, int dtype, void* q, void* k, void* v, float* gamma, float* beta, float* lambda,
                  void* stream)
{
    int st = check_sizes(batch, heads, seq_len, d_k, d_v, dtype, 0);
    if (st != MESA_OK) return st;
    if (!(isfinite(gamma_cap) && gamma_cap >= 0.0f && gamma_cap <= 1.0f)) return MESA_ERR_ARG;
    if (!(isfinite(l2_eps) && l2_eps >= 0.0f)) return MESA_ERR_ARG;
    if (heads == 0) return MESA_OK;
    if (!theta || !lambda) return MESA_ERR_NULL;
    const int64_t tokens = batch * heads * seq_len;
    if (tokens > 0 && (!qp || !kp || !vp || !conv_q || !conv_k || !a_gamma || !a_beta || !q || !k || !v ||
                       !gamma || !beta))
        return MESA_ERR_NULL;
    if (tokens > (int64_t(1) << 40)) return MESA_ERR_SHAPE;
    const int64_t es = dtype == MESA_DTYPE_BF16 ? 2 : 4;
    // the kernel moves projections, outputs and filter rows in 16-byte pieces
    for (const void* ptr : {qp, kp, vp, static_cast<const void*>(q), static_cast<const void*>(k),
                            static_cast<const void*>(v), static_cast<const void*>(conv_q),
                            static_cast<const void*>(conv_k), static_cast<const void*>(conv_v)})
        if (uintptr_t(ptr) % 16 != 0) return MESA_ERR_ARG;
    for (const void* ptr : {static_cast<const void*>(a_gamma), static_cast<const void*>(a_beta),
                            static_cast<const void*>(theta), static_cast<const void*>(gamma),
                            static_cast<const void*>(beta), static_cast<const void*>(lambda)})
        if (uintptr_t(ptr) % 4 != 0) return MESA_ERR_ARG;
    const Range ins[] = {range_of(qp, tokens * d_k * es), range_of(kp, tokens * d_k * es),
                         range_of(vp, tokens * d_v * es), range_of(conv_q, heads * d_k * 16),
                         range_of(conv_k, heads * d_k * 16), range_of(conv_v, conv_v ? heads * d_v * 16 : 0),
                         range_of(a_gamma, tokens * 4), range_of(a_beta, tokens * 4),
                         range_of(theta, heads * d_k * 4)};
    const Range outs[] = {range_of(q, tokens * d_k * es), range_of(k, tokens * d_k * es),
                          range_of(v, tokens * d_v * es), range_of(gamma, tokens * 4),
                          range_of(beta, tokens * 4), range_of(lambda, heads * d_k * 4)};
    for (const Range& o : outs) {
        if (o.lo == o.hi) continue;
        for (const Range& i : ins)
            if (i.lo != i.hi && overlaps(o, i)) return MESA_ERR_ARG;
    }
    for (int x = 0; x < 6; ++x)
        for (int y = x + 1; y < 6; ++y)
            if (outs[x].lo != outs[x].hi && outs[y].lo != outs[y].hi && overlaps(outs[x], outs[y]))
                return MESA_ERR_ARG;
    mesa::FrontArgs fa{batch, heads, seq_len, int(d_k), int(d_v), dtype == MESA_DTYPE_BF16, qp, kp, vp,
                       conv_q, conv_k, conv_v, a_gamma, a_beta, theta, gamma_cap, l2_eps, q, k, v, gamma,
                       beta, lambda};
    const hipError_t e = mesa::launch_frontend(fa, static_cast<hipStream_t>(stream));
    return finish(e == hipSuccess ? MESA_OK : MESA_ERR_HIP, stream);
}

int mesa_output_norm(const float* o, const float* weight, float eps, int64_t batch, int64_t heads,
                     int64_t seq_len, int64_t d_v, int out_dtype, void* y, void* stream)
{
    int st = check_sizes(batch, heads, seq_len, 64, d_v, out_dtype, 0);
    if (st != MESA_OK) return st;
    if (!(isfinite(eps) && eps >= 0.0f)) return MESA_ERR_ARG;
    const int64_t tokens = batch * heads * seq_len;
    if (tokens == 0) return MESA_OK;
    if (!o || !weight || !y) return MESA_ERR_NULL;
    if (tokens > (int64_t(1) << 40)) return MESA_ERR_SHAPE;
    const int64_t es = out_dtype == MESA_DTYPE_BF16 ? 2 : 4;
    if (uintptr_t(o) % 16 != 0 || uintptr_t(weight) % 16 != 0 || uintptr_t(y) % 16 != 0) return MESA_ERR_ARG;
    const Range out = range_of(y, tokens * d_v * es);
    if (overlaps(out, range_of(o, tokens * d_v * 4)) || overlaps(out, range_of(weight, heads * d_v * 4)))
        return MESA_ERR_ARG;
    mesa::NormArgs na{batch, heads, seq_len, int(d_v), out_dtype == MESA_DTYPE_BF16, o, weight, eps, y};
    const hipError_t e = mesa::launch_output_norm(na, static_cast<hipStream_t>(stream));
    return finish(e == hipSuccess ? MESA_OK : MESA_ERR_HIP, stream);
}

}  // extern "C"
