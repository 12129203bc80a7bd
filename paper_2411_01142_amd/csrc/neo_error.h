// Thread-local error message of the C ABI, shared by the device (HIP) and
// host (CPU) halves of the library.
#pragma once

#include "libneoattn.h"

namespace neo {

// Records the formatted message for neo_last_error() and returns `st`.
neo_status set_error(neo_status st, const char* fmt, ...) __attribute__((format(printf, 2, 3)));

// Clears the message and returns NEO_OK.
neo_status clear_error();

}  // namespace neo
