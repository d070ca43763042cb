// Launcher stubs for the sanitizer build of the host runtime (test only).
// The host runtime is compiled as plain C++ without its kernels; every
// launcher reports an error, so a run that reaches device work fails cleanly.
// The driver only exercises host validation, metadata and error paths.
#include "tss_internal.h"

namespace tss {
hipError_t launch_gemm(bool, int, int, int, const GemmArgs&, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_attn(bool, int, int, int, const AttnArgs&, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_embed(bool, const EmbedArgs&, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_accept(const AcceptArgs&, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_compact(bool, int, const CompactArgs&, hipStream_t) { return hipErrorInvalidValue; }
const void* embed_kernel(bool) { return nullptr; }
hipError_t init_kernel_attributes() { return hipErrorInvalidValue; }
hipError_t init_gemm_attributes() { return hipErrorInvalidValue; }
hipError_t launch_rope_table(float2*, int, int, float, hipStream_t) { return hipErrorInvalidValue; }
}  // namespace tss
