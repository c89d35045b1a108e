// MFMA grouped GEMM instantiations for the forward Dyad-IT pass.
#include "gemm_mfma_dispatch.h"

namespace dyad {
hipError_t launch_mfma_fwd_it(const GemmPass &p, hipStream_t s) { return dispatch_d<true, false, false>(p, s); }
}  // namespace dyad
