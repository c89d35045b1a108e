// MFMA grouped GEMM instantiations for the forward Dyad-OT pass.
#include "gemm_mfma_dispatch.h"

namespace dyad {
hipError_t launch_mfma_fwd_ot(const GemmPass &p, hipStream_t s) { return dispatch_d<false, true, false>(p, s); }
}  // namespace dyad
