// Weight-gradient kernels with both components on block-ordered operands
// (component 2 reading de-interleaved or zero-padded copies of dZ / X).  On
// such operands the kernel does not depend on n_dyad, which it takes at run
// time (DwArgs::groups): one instance serves every n_dyad.
#include "dw_mfma.h"

namespace dyad {

hipError_t launch_dw_plain(const DwPass &p, const DwPlan &pl, hipStream_t s) {
#define DYAD_DW_PLAIN(J_, K_, WJ_, WK_)                                              \
    if (pl.BJ == J_ && pl.BK == K_ && pl.WJN == WJ_ && pl.WKN == WK_)                \
        return launch_dw_cfg<1, J_, K_, WJ_, WK_, false, false>(p, pl, s);
    DYAD_DW_CONFIGS(DYAD_DW_PLAIN)
#undef DYAD_DW_PLAIN
    return hipErrorNotSupported;
}

}  // namespace dyad
