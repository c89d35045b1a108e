// MFMA grouped GEMM instantiations for the input-gradient Dyad-DT pass.
#include "gemm_mfma_dispatch.h"

namespace dyad {
hipError_t launch_mfma_dx_dt(const GemmPass &p, hipStream_t s) { return dispatch_d<true, true, true>(p, s); }
}  // namespace dyad
