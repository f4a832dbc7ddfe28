// Controls of the host-only HIP stand-ins (see runtime_stub.cpp).
#pragma once
#include <string>
#include <vector>

#include "kernels.hpp"

namespace stub {
extern std::vector<std::string> launches;  // kernel kinds "launched", in order
extern hipError_t launch_result;           // what every stub launcher returns
extern bool validate_reports_bad;          // the validate stub reports a bad page
extern int cus;                            // compute units reported by the device query
extern bool symbol_lookup_fails;           // the first device-symbol lookup fails
extern int symbol_lookups;                 // device-symbol lookups so far
extern const float* last_part_o;           // split-partial buffer of the last decode launch
}  // namespace stub
