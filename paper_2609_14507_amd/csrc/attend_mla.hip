// Split-KV decode attention over an MLA latent partition (pass 1), gfx950.
#include "wsk_internal.h"

namespace wsk {

hipError_t launch_mla_attend(const AttendParams &, int, hipStream_t) { return hipErrorNotSupported; }

}  // namespace wsk
