// Register-list MFMA tile kernel instantiations for the f16 filter (see mtile.h).
#include "mtile.h"

namespace tod {

hipError_t launch_mtile_f16(const Plan& p, const Args& a, int64_t q_begin, int64_t q_rows,
                          hipStream_t s, TileTail* tail) {
  return mt::launch_mtile_any<_Float16>(p, a, q_begin, q_rows, s, tail);
}

}  // namespace tod
