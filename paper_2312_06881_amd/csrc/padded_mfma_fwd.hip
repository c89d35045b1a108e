// Zero-padded forms of the forward pass (weights read as stored).
#include "padded_mfma.h"

namespace dyad {

hipError_t launch_padded_fwd(const GemmPass &p, hipStream_t s) { return launch_padded_as<false>(p, s); }

}  // namespace dyad
