// Internal helpers shared by the library's translation units: error state,
// argument checks and HIP error propagation. Not part of the public ABI.
#pragma once

#include <cstdarg>
#include <cstdint>
#include <cstdio>

#include "../../include/ard.h"

namespace ard {

// Records a formatted message as the calling thread's last error and returns
// `status`, so that a check reads `return fail(ARD_ERR_INVALID_ARG, ...)`.
int fail(int status, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
void clear_error();

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Validates a row plan against the neuron count it is applied to. A NULL plan
// is "everything kept". needs_list: the caller reads the device kept-index
// list, so a plan that drops neurons must carry one. Returns ARD_OK or an
// error with a message.
int check_row_plan(const ard_row_plan* plan, int32_t n, const char* what, bool needs_list);

// The fp32 tile layer's forward (fwd) or transposed product with the kept-tile
// lists split over several workgroups for small grids, partial sums in the
// caller's buffer (ard_tile.hip). Falls back to ard_tile_fwd / ard_tile_bwd_data.
int tdp_product_f32_split(bool fwd, const ard_tile_desc* d, const ard_tile_plan* p, const void* act, const void* W,
                          void* out, float* partial, size_t partial_floats, void* stream,
                          int* splits_left = nullptr);

// Kept count of a row pattern (see ard_row_kept).
inline int32_t kept_count(int32_t n, int32_t period, int32_t offset) {
  if (offset >= n) return 0;
  return (n - offset + period - 1) / period;
}

}  // namespace ard

// Propagates a HIP error from a launch or runtime call as ARD_ERR_HIP.
#define ARD_HIP_CHECK(expr)                                                           \
  do {                                                                                \
    hipError_t _e = (expr);                                                           \
    if (_e != hipSuccess)                                                             \
      return ::ard::fail(ARD_ERR_HIP, "%s failed: %s", #expr, hipGetErrorString(_e)); \
  } while (0)

#define ARD_LAUNCH_CHECK()                                                            \
  do {                                                                                \
    hipError_t _e = hipGetLastError();                                                \
    if (_e != hipSuccess)                                                             \
      return ::ard::fail(ARD_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(_e)); \
  } while (0)
