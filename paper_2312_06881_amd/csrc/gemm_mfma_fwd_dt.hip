// MFMA grouped GEMM instantiations for the forward Dyad-DT pass.
#include "gemm_mfma_dispatch.h"

namespace dyad {
hipError_t launch_mfma_fwd_dt(const GemmPass &p, hipStream_t s) { return dispatch_d<true, true, false>(p, s); }
}  // namespace dyad
