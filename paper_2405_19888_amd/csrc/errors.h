// Thread-local error message of libparrot_attn (parrot_last_error), shared by
// the decode entry points and the host-side context store.
#pragma once

#include "parrot_attn.h"

namespace parrot {

// Set the calling thread's message (cleared for PARROT_OK) and return `s`.
parrot_status set_error(parrot_status s, const char* fmt, ...);

}  // namespace parrot
