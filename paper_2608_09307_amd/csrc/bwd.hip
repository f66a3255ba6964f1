// LinSimp backward on gfx950 (query sweep, state sweep, key side).
#include "common.h"
#include "linsimp_internal.h"

namespace linsimp {

int launch_backward(const Shape& s, const void*, const void*, const void*, const void*,
                    const void*, const float*, const void*, const float*, const void*, void*,
                    void*, void*, void*, void*, const Workspace&, hipStream_t) {
  set_error("backward not built for dtype=%d D=%d m=%d", s.dtype, s.D, s.m);
  return -2;
}

}  // namespace linsimp
