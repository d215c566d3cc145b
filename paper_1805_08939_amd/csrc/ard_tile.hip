// Tile-based dropout pattern layer (Sec. III-B). Placeholder entry points.
#include <hip/hip_runtime.h>

#include "ard_internal.hpp"

using namespace ard;

extern "C" {

size_t ard_tile_plan_workspace_bytes(int32_t, int32_t) { return 0; }
int ard_plan_tiles(int32_t, int32_t, int32_t, const uint32_t*, int32_t, void*, size_t, ard_tile_plan*,
                   void*) {
  return fail(ARD_ERR_UNSUPPORTED, "tile plans are not built yet");
}
int ard_tile_fwd(const ard_tile_desc*, const ard_tile_plan*, const void*, const void*, void*, void*) {
  return fail(ARD_ERR_UNSUPPORTED, "tile layer is not built yet");
}
int ard_tile_bwd_data(const ard_tile_desc*, const ard_tile_plan*, const void*, const void*, void*,
                      void*) {
  return fail(ARD_ERR_UNSUPPORTED, "tile layer is not built yet");
}
int ard_tile_bwd_weight(const ard_tile_desc*, const ard_tile_plan*, const void*, const void*, float*,
                        void*) {
  return fail(ARD_ERR_UNSUPPORTED, "tile layer is not built yet");
}
}
