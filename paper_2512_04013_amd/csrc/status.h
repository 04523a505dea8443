// Status helpers shared by the library's translation units.
#pragma once

#include "aug.h"

namespace aug {

// Record a printf-style message for aug_last_error() and return `s`.
aug_status fail(aug_status s, const char* fmt, ...) __attribute__((format(printf, 2, 3)));

}  // namespace aug
