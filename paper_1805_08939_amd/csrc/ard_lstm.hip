// LSTM layer with hidden-unit row pattern (Sec. IV-C). Placeholder entry points.
#include <hip/hip_runtime.h>

#include "ard_internal.hpp"

using namespace ard;

extern "C" {

size_t ard_lstm_workspace_bytes(const ard_lstm_desc*) { return 0; }
int ard_lstm_fwd(const ard_lstm_desc*, const void*, const void*, const float*, const void*,
                 const void*, void*, void*, void*, void*, size_t, void*) {
  return fail(ARD_ERR_UNSUPPORTED, "LSTM layer is not built yet");
}
int ard_lstm_bwd(const ard_lstm_desc*, const void*, const void*, const void*, const void*, void*,
                 size_t, void*, float*, float*, void*, void*, void*) {
  return fail(ARD_ERR_UNSUPPORTED, "LSTM layer is not built yet");
}
}
