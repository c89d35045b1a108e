// Weight-gradient kernels of Dyad-IT, every tile configuration and n_dyad.
#include "dw_mfma.h"

namespace dyad {

hipError_t launch_dw_it(const DwPass &p, const DwPlan &pl, hipStream_t s) {
    return launch_dw_variant<true, false>(p, pl, s);
}

}  // namespace dyad
