// MFMA grouped GEMM instantiations for the forward Dyad-IT pass of a layer
// whose input is GELU(in), the activation applied as the input is staged.
#include "gemm_mfma_dispatch.h"

namespace dyad {
hipError_t launch_mfma_fwd_gin_it(const GemmPass &p, hipStream_t s) { return dispatch_d_gelu_in<true, false>(p, s); }
}  // namespace dyad
