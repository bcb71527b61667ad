// int8.hip -- low-bit (INT8) path.  Placeholder launchers: not built yet.
#include "launch.hpp"

namespace gdn {

hipError_t launch_quantize_i8(const float*, int8_t*, int32_t*, int64_t, int, hipStream_t) {
  return hipErrorNotSupported;
}

hipError_t launch_neumann_i8(const int8_t*, const int32_t*, int8_t*, int32_t*, float*, int64_t,
                             int, int, int, hipStream_t) {
  return hipErrorNotSupported;
}

}  // namespace gdn
