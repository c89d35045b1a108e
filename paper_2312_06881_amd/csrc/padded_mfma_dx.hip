// Zero-padded forms of the input gradient (weights read transposed).
#include "padded_mfma.h"

namespace dyad {

hipError_t launch_padded_dx(const GemmPass &p, hipStream_t s) { return launch_padded_as<true>(p, s); }

}  // namespace dyad
