// Conventional (Bernoulli) dropout on a feature-major activation: the baseline
// the method replaces (Sec. II-C). Every element draws its own keep decision,
// so the layer GEMMs stay dense and a separate kernel multiplies the output by
// the mask in the forward pass and the output derivative by the same mask in
// the backward pass. Reading of the paper's baseline: one independent
// Bernoulli(1 - p) draw per element and sample, the counter-based generator of
// the pattern sampler (element e = neuron * batch + sample takes draw e of the
// (seed, stream, iteration) sequence, kept iff its 53-bit uniform is >= p).

#include <hip/hip_runtime.h>

#include <cstdint>

#include "ard_gemm.hpp"
#include "ard_internal.hpp"

namespace ard {
namespace {

// Draw t (0-based) of the SplitMix64 sequence started at s0 (Steele, Lea &
// Flood, OOPSLA 2014): the Weyl state after t + 1 golden-ratio steps through
// the 64-bit finaliser.
__device__ __forceinline__ uint64_t mix_draw(uint64_t s0, uint64_t t) {
  uint64_t z = s0 + (t + 1) * 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// One thread per element: draw, keep bit, scaled (or zeroed) value; each
// 32-lane half of a wave writes its 32 bits of the mask as one word.
template <typename T>
__global__ void __launch_bounds__(256) dropout_fwd_kernel(T* __restrict__ y, uint32_t* __restrict__ mask,
                                                          int64_t total, uint64_t s0, double p, float scale) {
  const int64_t e = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  bool keep = false;
  if (e < total) {
    keep = static_cast<double>(mix_draw(s0, static_cast<uint64_t>(e)) >> 11) * 0x1.0p-53 >= p;
    y[e] = from_f32<T>(keep ? scale * to_f32(y[e]) : 0.0f);
  }
  const uint64_t bits = __ballot(keep);
  const int lane = threadIdx.x & 63;
  const int64_t w = e >> 5;  // word of this lane's element
  if ((lane & 31) == 0 && (w << 5) < total) mask[w] = static_cast<uint32_t>(bits >> lane);
}

// dY *= scale * mask, one thread per element.
template <typename T>
__global__ void __launch_bounds__(256) dropout_bwd_kernel(T* __restrict__ dy, const uint32_t* __restrict__ mask,
                                                          int64_t total, float scale) {
  const int64_t e = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (e >= total) return;
  const bool keep = (mask[e >> 5] >> (e & 31)) & 1u;
  dy[e] = from_f32<T>(keep ? scale * to_f32(dy[e]) : 0.0f);
}

int check_dropout(int32_t dtype, int32_t n, int32_t batch, const void* y, const uint32_t* mask) {
  if (dtype != ARD_F32 && dtype != ARD_BF16) return fail(ARD_ERR_UNSUPPORTED, "dtype %d not supported", dtype);
  if (n < 1 || batch < 1) return fail(ARD_ERR_INVALID_ARG, "sizes must be >= 1 (n %d, batch %d)", n, batch);
  if (!y || !mask) return fail(ARD_ERR_INVALID_ARG, "activation or mask is NULL");
  if (reinterpret_cast<uintptr_t>(mask) % 4 != 0) return fail(ARD_ERR_INVALID_ARG, "mask is not 4-byte aligned");
  if (reinterpret_cast<uintptr_t>(y) % (dtype == ARD_BF16 ? 2 : 4) != 0)
    return fail(ARD_ERR_INVALID_ARG, "activation is not aligned to its element size");
  return ARD_OK;
}

}  // namespace
}  // namespace ard

using namespace ard;

extern "C" {

int ard_dropout_fwd(int32_t dtype, int32_t n, int32_t batch, double p, float scale, uint64_t seed,
                    uint32_t stream_id, uint64_t iter, void* Yt, uint32_t* mask, void* stream) {
  clear_error();
  int st = check_dropout(dtype, n, batch, Yt, mask);
  if (st != ARD_OK) return st;
  if (!(p >= 0.0 && p < 1.0)) return fail(ARD_ERR_INVALID_ARG, "p must be in [0, 1)");
  if (stream_id >= (1u << 24)) return fail(ARD_ERR_INVALID_ARG, "stream %u must be < 2^24", stream_id);
  if (iter >= (1ull << 40)) return fail(ARD_ERR_INVALID_ARG, "iter must be < 2^40");
  const uint64_t s0 = seed ^ ((static_cast<uint64_t>(stream_id) << 40) | iter);
  const int64_t total = static_cast<int64_t>(n) * batch;
  const dim3 grid(static_cast<unsigned>((total + 255) / 256));
  hipStream_t sm = static_cast<hipStream_t>(stream);
  if (dtype == ARD_BF16)
    hipLaunchKernelGGL(dropout_fwd_kernel<bf16>, grid, dim3(256), 0, sm, static_cast<bf16*>(Yt), mask, total, s0, p,
                       scale);
  else
    hipLaunchKernelGGL(dropout_fwd_kernel<float>, grid, dim3(256), 0, sm, static_cast<float*>(Yt), mask, total, s0,
                       p, scale);
  ARD_LAUNCH_CHECK();
  return ARD_OK;
}

int ard_dropout_bwd(int32_t dtype, int32_t n, int32_t batch, float scale, const uint32_t* mask, void* dYt,
                    void* stream) {
  clear_error();
  int st = check_dropout(dtype, n, batch, dYt, mask);
  if (st != ARD_OK) return st;
  const int64_t total = static_cast<int64_t>(n) * batch;
  const dim3 grid(static_cast<unsigned>((total + 255) / 256));
  hipStream_t sm = static_cast<hipStream_t>(stream);
  if (dtype == ARD_BF16)
    hipLaunchKernelGGL(dropout_bwd_kernel<bf16>, grid, dim3(256), 0, sm, static_cast<bf16*>(dYt), mask, total, scale);
  else
    hipLaunchKernelGGL(dropout_bwd_kernel<float>, grid, dim3(256), 0, sm, static_cast<float*>(dYt), mask, total,
                       scale);
  ARD_LAUNCH_CHECK();
  return ARD_OK;
}

}  // extern "C"
