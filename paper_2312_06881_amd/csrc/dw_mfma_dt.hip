// Weight-gradient kernels of Dyad-DT, every tile configuration and n_dyad.
#include "dw_mfma.h"

namespace dyad {

hipError_t launch_dw_dt(const DwPass &p, const DwPlan &pl, hipStream_t s) {
    return launch_dw_variant<true, true>(p, pl, s);
}

}  // namespace dyad
