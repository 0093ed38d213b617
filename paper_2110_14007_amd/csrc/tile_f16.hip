// Tile kernel instantiations for the f16 filter (see tile.h).
#include "tile.h"

namespace tod {

hipError_t launch_tile_f16(const Plan& p, const Args& a, int64_t q_begin, int64_t q_rows,
                          hipStream_t s) {
  return tile::launch_prec<TOD_PREC_FP16>(p, a, q_begin, q_rows, s);
}

}  // namespace tod
