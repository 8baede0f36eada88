// Host-only helpers shared by the C-ABI sources that are not HIP code.
#pragma once

#include "rp.h"

namespace rp {
// Records the detail text returned by rp_last_error() on this thread.
rp_status set_error(rp_status st, const char* msg);
void clear_error();
}  // namespace rp
