// Weight-gradient kernels with both components on block-ordered operands
// (component 2 reading de-interleaved copies of dZ / X), n_dyad 3, 6, 8 and 16.
#include "dw_mfma.h"

namespace dyad {

hipError_t launch_dw_plain(const DwPass &p, const DwPlan &pl, hipStream_t s) {
#define DYAD_DW_PLAIN(J_, K_, WJ_, WK_)                                                  \
    if (pl.BJ == J_ && pl.BK == K_ && pl.WJN == WJ_ && pl.WKN == WK_) switch (p.D) {     \
        case 3: return launch_dw_cfg<3, J_, K_, WJ_, WK_, false, false>(p, pl, s);       \
        case 6: return launch_dw_cfg<6, J_, K_, WJ_, WK_, false, false>(p, pl, s);       \
        case 8: return launch_dw_cfg<8, J_, K_, WJ_, WK_, false, false>(p, pl, s);       \
        case 16: return launch_dw_cfg<16, J_, K_, WJ_, WK_, false, false>(p, pl, s);     \
        default: return hipErrorNotSupported;                                            \
    }
    DYAD_DW_CONFIGS(DYAD_DW_PLAIN)
#undef DYAD_DW_PLAIN
    return hipErrorNotSupported;
}

}  // namespace dyad
