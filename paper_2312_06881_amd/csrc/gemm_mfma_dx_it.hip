// MFMA grouped GEMM instantiations for the input-gradient Dyad-IT pass.
#include "gemm_mfma_dispatch.h"

namespace dyad {
hipError_t launch_mfma_dx_it(const GemmPass &p, hipStream_t s) { return dispatch_d<false, true, true>(p, s); }
}  // namespace dyad
