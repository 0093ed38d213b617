// Range tile kernel instantiations for the bf16 filter (see rtile.h).
#include "rtile.h"

namespace tod {

hipError_t launch_range_tile_bf16(const Plan& p, const Args& a, int64_t q_begin, int64_t q_rows,
                                 bool fill, hipStream_t s) {
  return rt::launch_range_any<__bf16>(p, a, q_begin, q_rows, fill, s);
}

}  // namespace tod
