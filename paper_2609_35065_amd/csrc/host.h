// host.h -- declarations shared by the host-only code (host.cpp) and the
// GPU entry points; no HIP header.
#pragma once

#include <stdint.h>

#include "tempokv.h"

namespace tkv {

// Layout checks shared by the copy directions and staging.  Returns KV_OK or
// a negative kv_status.
int check_layout(const kv_layout *lo);

}  // namespace tkv
