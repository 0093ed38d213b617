// Tile kernel instantiations for the f32 filter (see tile.h).
#include "tile.h"

namespace tod {

hipError_t launch_tile_f32(const Plan& p, const Args& a, int64_t q_begin, int64_t q_rows,
                          hipStream_t s) {
  return tile::launch_prec<TOD_PREC_FP32>(p, a, q_begin, q_rows, s);
}

}  // namespace tod
