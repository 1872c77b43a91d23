// Shared between the C-ABI translation units: the opaque handle types and
// the per-thread error string.
#pragma once

#include <string>

#include "../../include/ar_plan.h"
#include "plan.hpp"

struct ar_plan : arp::Plan {};

namespace arp {

void set_error(const std::string& msg);
void clear_error();
ar_status fail(ar_status s, const std::string& msg);

// Release the device-side state of a plan (executor translation unit).
void exec_release(Plan& p);

}  // namespace arp

#define AR_EXPORT extern "C" __attribute__((visibility("default")))
