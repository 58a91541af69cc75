// Chunked CG with bf16 matrix-core products (placeholder until the MFMA kernel lands).
#include "mesa_kernels.hpp"

namespace mesa {

bool chunk_cg_bf16_supported(const ForwardShape&) { return false; }

hipError_t launch_chunk_cg_bf16(const CgArgs&, hipStream_t) { return hipErrorInvalidValue; }

}  // namespace mesa
