// Internal host-side helpers of the C ABI: error reporting and shared constants.
#pragma once

#include <string>

#pragma GCC visibility push(default)
#include "../../include/pkv.h"
#pragma GCC visibility pop

namespace pkv {

constexpr int kSupportedBlockSize = 16;

// Record a failure message for pkv_last_error() and return the status.
pkv_status fail(pkv_status status, const std::string& message);
// Clear the message and return PKV_OK.
pkv_status ok();

}  // namespace pkv
