// Argument checks shared by the library's translation units (host code).
#pragma once

#include "aug.h"

namespace aug {

// A supported layer shape (heads, group size, head_dim, block size, dtype
// set, softmax scale); otherwise the status, with the reason recorded.
aug_status check_shape(const aug_attn_shape* s, const char* who);

// `info` is a plan's (non-negative counts, plan_bytes matching its layout)
// and was planned for `s` (heads, head_dim, dtypes).
aug_status check_plan_info(const aug_attn_plan_info* info, const aug_attn_shape* s, const char* who);

}  // namespace aug
