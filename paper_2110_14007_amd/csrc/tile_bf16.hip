// Tile kernel instantiations for the bf16 filter (see tile.h).
#include "tile.h"

namespace tod {

hipError_t launch_tile_bf16(const Plan& p, const Args& a, int64_t q_begin, int64_t q_rows,
                          hipStream_t s) {
  return tile::launch_prec<TOD_PREC_BF16>(p, a, q_begin, q_rows, s);
}

}  // namespace tod
