// Weight-gradient kernels of Dyad-IT for a layer whose input is GELU(X), the
// activation applied to X as it is staged; every tile configuration and n_dyad.
#include "dw_mfma.h"

namespace dyad {

hipError_t launch_dw_xg_it(const DwPass &p, const DwPlan &pl, hipStream_t s) {
    return launch_dw_variant<true, false, true>(p, pl, s);
}

}  // namespace dyad
