// Host-side helpers of the C ABI layer (error reporting).
#pragma once

#include "../../include/ism_attn.h"

namespace ism {

// Record a formatted detail for ism_last_error() and return `s`.
ism_status fail(ism_status s, const char *fmt, ...)
    __attribute__((format(printf, 2, 3)));
void clear_error();
const char *last_error();

}  // namespace ism
