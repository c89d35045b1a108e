// MFMA grouped GEMM instantiations for the forward Dyad-OT pass of a layer
// whose input is GELU(in), the activation applied as the input is staged.
#include "gemm_mfma_dispatch.h"

namespace dyad {
hipError_t launch_mfma_fwd_gin_ot(const GemmPass &p, hipStream_t s) { return dispatch_d_gelu_in<false, true>(p, s); }
}  // namespace dyad
