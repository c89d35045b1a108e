// Entry to the MFMA grouped GEMM: routes a pass to the instantiation of its
// (pass, variant); returns hipErrorNotSupported, launching nothing, for
// shapes or dtypes the MFMA kernels do not cover.
#include "gemm_mfma_dispatch.h"

namespace dyad {

hipError_t launch_mfma_gemm(const GemmPass &p, hipStream_t s) {
    if (p.dtype != kBF16) return hipErrorNotSupported;
    // zero-padded widths (Kin or Nout not D times the block size) stay on the SIMT path
    if (p.Kin != p.D * p.bk || p.Nout != p.D * p.bn) return hipErrorNotSupported;
    if (p.gelu_in) {
        if (p.w_t) return hipErrorNotSupported;
        if (p.in_t && !p.out_t) return launch_mfma_fwd_gin_it(p, s);
        if (!p.in_t && p.out_t) return launch_mfma_fwd_gin_ot(p, s);
        if (p.in_t && p.out_t) return launch_mfma_fwd_gin_dt(p, s);
        return hipErrorNotSupported;
    }
    if (!p.w_t) {
        if (p.in_t && !p.out_t) return launch_mfma_fwd_it(p, s);
        if (!p.in_t && p.out_t) return launch_mfma_fwd_ot(p, s);
        if (p.in_t && p.out_t) return launch_mfma_fwd_dt(p, s);
    } else {
        if (!p.in_t && p.out_t) return launch_mfma_dx_it(p, s);
        if (p.in_t && !p.out_t) return launch_mfma_dx_ot(p, s);
        if (p.in_t && p.out_t) return launch_mfma_dx_dt(p, s);
    }
    return hipErrorNotSupported;
}

}  // namespace dyad
