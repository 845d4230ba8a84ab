// Tile attention backward for gfx950 (MI355X): placeholder until the
// backward kernels land.
#include <hip/hip_runtime.h>

#include "internal.h"

namespace mesh_attn {

hipError_t launch_tile_bwd(const BwdParams&, int, int, int, hipStream_t) {
  return hipErrorNotSupported;
}

}  // namespace mesh_attn
