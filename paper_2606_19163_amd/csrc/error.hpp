// Thread-local last-error text behind pulse_last_error(), shared by the
// library's translation units.
#pragma once

#include "pulse_stage.h"

namespace pulse {
// Record `msg` as the calling thread's last error and return `s`.
pulse_status set_last_error(pulse_status s, const char* msg);
}  // namespace pulse
