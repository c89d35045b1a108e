// MFMA grouped GEMM instantiations for the input-gradient Dyad-OT pass.
#include "gemm_mfma_dispatch.h"

namespace dyad {
hipError_t launch_mfma_dx_ot(const GemmPass &p, hipStream_t s) { return dispatch_d<true, false, true>(p, s); }
}  // namespace dyad
