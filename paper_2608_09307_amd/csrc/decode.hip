// LinSimp autoregressive decode step on gfx950.
#include "common.h"
#include "linsimp_internal.h"

namespace linsimp {

int launch_decode(int64_t, int, int D, int, int m, int, int dtype, float, const void*, const void*,
                  const void*, const void*, const void*, const float*, float*, float*, float*,
                  void*, void*, int64_t*, void*, hipStream_t) {
  set_error("decode not built for dtype=%d D=%d m=%d", dtype, D, m);
  return -2;
}

}  // namespace linsimp
