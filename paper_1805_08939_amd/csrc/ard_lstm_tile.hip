// LSTM layer whose weight matrix W = [W_ih | W_hh] (4H x (I + H)) takes a
// tile-based pattern (Sec. III-B applied to the LSTM's matrix products,
// Sec. IV-C): only the kept tiles of W are read by the gate products and only
// they receive a weight gradient. Every hidden unit is kept.
//
// Per step t the gate product runs on the tile layer's kernels with the
// stacked input xh_t = [x_t; h_{t-1}] ((I + H) x B, contiguous):
//   z_t = (W * M) xh_t,  then a pointwise kernel adds the bias, applies the
// gate nonlinearities and the cell update, and writes h_t both into the next
// step's xh and into the time-batched copy XH[(I + H)][T B] that the weight
// gradient contracts over. The backward pass walks the steps in reverse: a
// pointwise kernel forms dz_t (into dZ[4H][T B] and a contiguous step copy),
// the tile layer's transposed product gives d xh_t = (W * M)^T dz_t, whose
// lower rows are the recurrent gradient of the next (earlier) step; one tile
// weight-gradient call over all T B columns gives dW = M * (dZ XH^T).

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "ard_internal.hpp"

namespace ard {
namespace {

__device__ __forceinline__ float sgm(float x) { return 1.0f / (1.0f + expf(-x)); }

struct TileLstm {
  int32_t T, B, I, H;
  int64_t TB;           // T * B: columns of XH and dZ
  float* xh;            // [(I + H)][B] step input
  float* XH;            // [(I + H)][T B]
  float* z;             // [4H][B] step gate product
  float* G;             // [T][4H][B] activated gates i, f, g, o
  float* C;             // [T + 1][H][B] cell states, C[0] = c0
  float* dz;            // [4H][B] step gate derivative
  float* dZ;            // [4H][T B]
  float* dxh;           // [(I + H)][B] step input derivative
  float* dc;            // [H][B] cell derivative carry
  float* part;          // split partial sums of the step products
  size_t part_floats;
  int32_t zsplits;      // partial sums of z (1: z itself holds the product)
  int32_t dsplits;      // partial sums of dxh (1: dxh itself holds the product)
};

size_t al256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

struct TileLayout {
  size_t xh, XH, z, G, C, dz, dZ, dxh, dc, part, part_floats, total;
};

TileLayout tile_layout(int64_t T, int64_t B, int64_t I, int64_t H) {
  TileLayout L;
  size_t off = 0;
  const int64_t K = I + H;
  L.xh = off;  off += al256(4 * K * B);
  L.XH = off;  off += al256(4 * K * T * B);
  L.z = off;   off += al256(4 * 4 * H * B);
  L.G = off;   off += al256(4 * T * 4 * H * B);
  L.C = off;   off += al256(4 * (T + 1) * H * B);
  L.dz = off;  off += al256(4 * 4 * H * B);
  L.dZ = off;  off += al256(4 * 4 * H * T * B);
  L.dxh = off; off += al256(4 * K * B);
  L.dc = off;  off += al256(4 * H * B);
  // up to 8 splits of the larger step product (4H or I + H rows, rounded to whole 64-row tiles)
  const int64_t rows = ((4 * H > K ? 4 * H : K) + 63) / 64 * 64;
  L.part_floats = static_cast<size_t>(8 * rows * B);
  L.part = off; off += al256(4 * L.part_floats);
  L.total = off;
  return L;
}

TileLstm tile_args(const TileLayout& L, char* w, int32_t T, int32_t B, int32_t I, int32_t H) {
  TileLstm s;
  s.T = T;
  s.B = B;
  s.I = I;
  s.H = H;
  s.TB = static_cast<int64_t>(T) * B;
  s.xh = reinterpret_cast<float*>(w + L.xh);
  s.XH = reinterpret_cast<float*>(w + L.XH);
  s.z = reinterpret_cast<float*>(w + L.z);
  s.G = reinterpret_cast<float*>(w + L.G);
  s.C = reinterpret_cast<float*>(w + L.C);
  s.dz = reinterpret_cast<float*>(w + L.dz);
  s.dZ = reinterpret_cast<float*>(w + L.dZ);
  s.dxh = reinterpret_cast<float*>(w + L.dxh);
  s.dc = reinterpret_cast<float*>(w + L.dc);
  s.part = reinterpret_cast<float*>(w + L.part);
  s.part_floats = L.part_floats;
  s.zsplits = s.dsplits = 1;
  return s;
}

// Element e of a step product: the product buffer itself, or the sum of its
// split partial sums (n elements each) in split order, the loads of up to
// eight splits issued together.
__device__ __forceinline__ float step_val(const float* direct, const float* part, int splits, int64_t n, int64_t e) {
  if (splits <= 1) return direct[e];
  float v = 0.0f;
  for (int q0 = 0; q0 < splits; q0 += 8) {
    float t[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) t[u] = q0 + u < splits ? part[(q0 + u) * n + e] : 0.0f;
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (q0 + u < splits) v += t[u];
  }
  return v;
}

// Before the first step: x_t into the input rows of XH for every t, h0 (or 0)
// into the recurrent rows of XH's first column block and of xh, x_0 into xh,
// c0 (or 0) into C[0].
__global__ void tile_lstm_init_kernel(TileLstm s, const float* __restrict__ X, const float* __restrict__ h0,
                                      const float* __restrict__ c0) {
  const int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t nx = static_cast<int64_t>(s.T) * s.I * s.B;
  if (e < nx) {  // X[t][k][b] -> XH[k][t B + b]
    const int64_t t = e / (static_cast<int64_t>(s.I) * s.B), r = e % (static_cast<int64_t>(s.I) * s.B);
    const int64_t k = r / s.B, b = r % s.B;
    s.XH[k * s.TB + t * s.B + b] = X[e];
    if (t == 0) s.xh[r] = X[e];
  }
  const int64_t nh = static_cast<int64_t>(s.H) * s.B;
  if (e < nh) {
    const int64_t j = e / s.B, b = e % s.B;
    const float h = h0 ? h0[e] : 0.0f;
    s.XH[(s.I + j) * s.TB + b] = h;
    s.xh[(s.I + j) * s.B + b] = h;
    s.C[e] = c0 ? c0[e] : 0.0f;
  }
}

// Step t: gates from z + bias, cell and hidden state; h_t into Hs, into the
// next step's xh and XH block; x_{t+1} into xh.
__global__ void tile_lstm_point_fwd_kernel(TileLstm s, int32_t t, const float* __restrict__ bias,
                                           const float* __restrict__ X, float* __restrict__ Hs) {
  const int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t HB = static_cast<int64_t>(s.H) * s.B;
  if (e < HB) {
    const int64_t j = e / s.B, b = e % s.B;
    float zv[4];
#pragma unroll
    for (int q = 0; q < 4; ++q)
      zv[q] = step_val(s.z, s.part, s.zsplits, 4 * HB, (q * s.H + j) * s.B + b) + (bias ? bias[q * s.H + j] : 0.0f);
    const float ig = sgm(zv[0]), fg = sgm(zv[1]), gg = tanhf(zv[2]), og = sgm(zv[3]);
    const float cp = s.C[static_cast<int64_t>(t) * HB + e];
    const float c = fg * cp + ig * gg;
    const float h = og * tanhf(c);
    float* Gt = s.G + static_cast<int64_t>(t) * 4 * HB;
    Gt[(0 * s.H + j) * s.B + b] = ig;
    Gt[(1 * s.H + j) * s.B + b] = fg;
    Gt[(2 * s.H + j) * s.B + b] = gg;
    Gt[(3 * s.H + j) * s.B + b] = og;
    s.C[static_cast<int64_t>(t + 1) * HB + e] = c;
    Hs[static_cast<int64_t>(t) * HB + e] = h;
    if (t + 1 < s.T) {
      s.xh[(s.I + j) * s.B + b] = h;
      s.XH[(s.I + j) * s.TB + static_cast<int64_t>(t + 1) * s.B + b] = h;
    }
  }
  const int64_t IB = static_cast<int64_t>(s.I) * s.B;
  if (t + 1 < s.T && e < IB) s.xh[e] = X[static_cast<int64_t>(t + 1) * IB + e];
}

// Step t backward: dh = dHs[t] + (recurrent rows of dxh from step t + 1, or
// dhT at the last step); dz_t into dz and dZ's block t; dc carry. At steps
// below the last, the input rows of dxh (d x_{t+1}) go to dX[t + 1].
__global__ void tile_lstm_point_bwd_kernel(TileLstm s, int32_t t, const float* __restrict__ dHs,
                                           const float* __restrict__ dhT, const float* __restrict__ dcT,
                                           float* __restrict__ dX) {
  const int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t HB = static_cast<int64_t>(s.H) * s.B;
  const bool last = t == s.T - 1;
  const int64_t IB = static_cast<int64_t>(s.I) * s.B;
  const int64_t KB = static_cast<int64_t>(s.I + s.H) * s.B;
  if (!last && dX && e < IB) dX[static_cast<int64_t>(t + 1) * IB + e] = step_val(s.dxh, s.part, s.dsplits, KB, e);
  if (e >= HB) return;
  const int64_t j = e / s.B, b = e % s.B;
  float dh = dHs[static_cast<int64_t>(t) * HB + e];
  float dcin;
  if (last) {
    if (dhT) dh += dhT[e];
    dcin = dcT ? dcT[e] : 0.0f;
  } else {
    dh += step_val(s.dxh, s.part, s.dsplits, KB, (s.I + j) * s.B + b);
    dcin = s.dc[e];
  }
  const float* Gt = s.G + static_cast<int64_t>(t) * 4 * HB;
  const float ig = Gt[(0 * s.H + j) * s.B + b], fg = Gt[(1 * s.H + j) * s.B + b];
  const float gg = Gt[(2 * s.H + j) * s.B + b], og = Gt[(3 * s.H + j) * s.B + b];
  const float c = s.C[static_cast<int64_t>(t + 1) * HB + e];
  const float cp = s.C[static_cast<int64_t>(t) * HB + e];
  const float tc = tanhf(c);
  const float d_o = dh * tc;
  const float dcv = dcin + dh * og * (1.0f - tc * tc);
  s.dc[e] = dcv * fg;
  const float dzq[4] = {dcv * gg * ig * (1.0f - ig), dcv * cp * fg * (1.0f - fg), dcv * ig * (1.0f - gg * gg),
                        d_o * og * (1.0f - og)};
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    s.dz[(q * s.H + j) * s.B + b] = dzq[q];
    s.dZ[(q * s.H + j) * s.TB + static_cast<int64_t>(t) * s.B + b] = dzq[q];
  }
}

// After the last backward step: d x_0 into dX[0], dh0 and dc0.
__global__ void tile_lstm_bwd_final_kernel(TileLstm s, float* __restrict__ dX, float* __restrict__ dh0,
                                           float* __restrict__ dc0) {
  const int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t IB = static_cast<int64_t>(s.I) * s.B, HB = static_cast<int64_t>(s.H) * s.B;
  const int64_t KB = static_cast<int64_t>(s.I + s.H) * s.B;
  if (dX && e < IB) dX[e] = step_val(s.dxh, s.part, s.dsplits, KB, e);
  if (e < HB) {
    const int64_t j = e / s.B, b = e % s.B;
    if (dh0) dh0[e] = step_val(s.dxh, s.part, s.dsplits, KB, (s.I + j) * s.B + b);
    if (dc0) dc0[e] = s.dc[e];
  }
}

// dbias[r] = sum over the T B columns of dZ row r, one block per row in a
// fixed order (each thread strides the row, then a tree in LDS).
__global__ void __launch_bounds__(256) tile_lstm_dbias_kernel(const float* __restrict__ dZ, int64_t cols,
                                                              float* __restrict__ dbias) {
  __shared__ float part[256];
  const float* row = dZ + static_cast<int64_t>(blockIdx.x) * cols;
  float v = 0.0f;
  for (int64_t c = threadIdx.x; c < cols; c += 256) v += row[c];
  part[threadIdx.x] = v;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (static_cast<int>(threadIdx.x) < w) part[threadIdx.x] += part[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) dbias[blockIdx.x] = part[0];
}

inline dim3 grid_of(int64_t n) { return dim3(static_cast<unsigned>((n + 255) / 256)); }

int check_tile_lstm(const ard_lstm_tile_desc* d) {
  if (!d) return fail(ARD_ERR_INVALID_ARG, "desc is NULL");
  if (d->dtype != ARD_F32) return fail(ARD_ERR_UNSUPPORTED, "the tile-pattern LSTM supports ARD_F32 only");
  if (d->seq_len < 1 || d->batch < 1 || d->input_size < 1 || d->hidden_size < 1)
    return fail(ARD_ERR_INVALID_ARG, "sizes must be >= 1");
  const ard_tile_plan* p = d->weight_plan;
  if (!p) return fail(ARD_ERR_INVALID_ARG, "weight_plan is NULL");
  if (p->n != 4 * d->hidden_size || p->k != d->input_size + d->hidden_size)
    return fail(ARD_ERR_INVALID_ARG, "weight_plan covers %d x %d, W is %d x %d", p->n, p->k, 4 * d->hidden_size,
                d->input_size + d->hidden_size);
  if (static_cast<int64_t>(d->seq_len) * d->batch >= (int64_t{1} << 31))
    return fail(ARD_ERR_INVALID_ARG, "seq_len * batch must be < 2^31");
  return ARD_OK;
}

ard_tile_desc step_desc(const ard_lstm_tile_desc* d, int32_t batch) {
  ard_tile_desc td;
  td.dtype = ARD_F32;
  td.batch = batch;
  td.in_features = d->input_size + d->hidden_size;
  td.out_features = 4 * d->hidden_size;
  td.scale = 1.0f;
  td.dropped = ARD_DROPPED_ZERO;
  return td;
}

}  // namespace
}  // namespace ard

using namespace ard;

extern "C" {

size_t ard_lstm_tile_workspace_bytes(const ard_lstm_tile_desc* desc) {
  if (check_tile_lstm(desc) != ARD_OK) return 0;
  return tile_layout(desc->seq_len, desc->batch, desc->input_size, desc->hidden_size).total;
}

int ard_lstm_tile_fwd(const ard_lstm_tile_desc* desc, const void* X, const void* W, const float* bias,
                      const void* h0, const void* c0, void* Hs, void* hT, void* cT, void* ws, size_t ws_bytes,
                      void* stream) {
  clear_error();
  int st = check_tile_lstm(desc);
  if (st != ARD_OK) return st;
  if (!X || !W || !Hs) return fail(ARD_ERR_INVALID_ARG, "X, W and Hs must not be NULL");
  const TileLayout L = tile_layout(desc->seq_len, desc->batch, desc->input_size, desc->hidden_size);
  if (!ws || ws_bytes < L.total)
    return fail(ARD_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", L.total, ws_bytes);
  if (!aligned16(ws)) return fail(ARD_ERR_INVALID_ARG, "workspace is not 16-byte aligned");
  hipStream_t sm = static_cast<hipStream_t>(stream);
  TileLstm s = tile_args(L, static_cast<char*>(ws), desc->seq_len, desc->batch, desc->input_size,
                         desc->hidden_size);
  const int64_t IB = static_cast<int64_t>(s.I) * s.B, HB = static_cast<int64_t>(s.H) * s.B;
  hipLaunchKernelGGL(tile_lstm_init_kernel, grid_of(static_cast<int64_t>(s.T) * IB > HB ? s.T * IB : HB), dim3(256),
                     0, sm, s, static_cast<const float*>(X), static_cast<const float*>(h0),
                     static_cast<const float*>(c0));
  ARD_LAUNCH_CHECK();
  const ard_tile_desc td = step_desc(desc, s.B);
  for (int32_t t = 0; t < s.T; ++t) {
    if ((st = tdp_product_f32_split(true, &td, desc->weight_plan, s.xh, W, s.z, s.part, s.part_floats, stream,
                                    &s.zsplits)) != ARD_OK)
      return st;
    hipLaunchKernelGGL(tile_lstm_point_fwd_kernel, grid_of(IB > HB ? IB : HB), dim3(256), 0, sm, s, t, bias,
                       static_cast<const float*>(X), static_cast<float*>(Hs));
    ARD_LAUNCH_CHECK();
  }
  if (hT) ARD_HIP_CHECK(hipMemcpyAsync(hT, static_cast<float*>(Hs) + (s.T - 1) * HB, 4 * HB,
                                       hipMemcpyDeviceToDevice, sm));
  if (cT) ARD_HIP_CHECK(hipMemcpyAsync(cT, s.C + s.T * HB, 4 * HB, hipMemcpyDeviceToDevice, sm));
  return ARD_OK;
}

int ard_lstm_tile_bwd(const ard_lstm_tile_desc* desc, const void* W, const void* dHs, const void* dhT,
                      const void* dcT, void* ws, size_t ws_bytes, void* dX, float* dW, float* dbias, void* dh0,
                      void* dc0, void* stream) {
  clear_error();
  int st = check_tile_lstm(desc);
  if (st != ARD_OK) return st;
  if (!W || !dHs) return fail(ARD_ERR_INVALID_ARG, "W and dHs must not be NULL");
  const TileLayout L = tile_layout(desc->seq_len, desc->batch, desc->input_size, desc->hidden_size);
  if (!ws || ws_bytes < L.total)
    return fail(ARD_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", L.total, ws_bytes);
  if (!aligned16(ws)) return fail(ARD_ERR_INVALID_ARG, "workspace is not 16-byte aligned");
  hipStream_t sm = static_cast<hipStream_t>(stream);
  TileLstm s = tile_args(L, static_cast<char*>(ws), desc->seq_len, desc->batch, desc->input_size,
                         desc->hidden_size);
  const int64_t IB = static_cast<int64_t>(s.I) * s.B, HB = static_cast<int64_t>(s.H) * s.B;
  const ard_tile_desc td = step_desc(desc, s.B);
  for (int32_t t = s.T - 1; t >= 0; --t) {
    hipLaunchKernelGGL(tile_lstm_point_bwd_kernel, grid_of(IB > HB ? IB : HB), dim3(256), 0, sm, s, t,
                       static_cast<const float*>(dHs), static_cast<const float*>(dhT),
                       static_cast<const float*>(dcT), static_cast<float*>(dX));
    ARD_LAUNCH_CHECK();
    if ((st = tdp_product_f32_split(false, &td, desc->weight_plan, s.dz, W, s.dxh, s.part, s.part_floats,
                                    stream, &s.dsplits)) != ARD_OK)
      return st;
  }
  hipLaunchKernelGGL(tile_lstm_bwd_final_kernel, grid_of(IB > HB ? IB : HB), dim3(256), 0, sm, s,
                     static_cast<float*>(dX), static_cast<float*>(dh0), static_cast<float*>(dc0));
  ARD_LAUNCH_CHECK();
  if (dW) {
    const ard_tile_desc tw = step_desc(desc, static_cast<int32_t>(s.TB));
    if ((st = ard_tile_bwd_weight(&tw, desc->weight_plan, s.XH, s.dZ, dW, stream)) != ARD_OK) return st;
  }
  if (dbias) {
    hipLaunchKernelGGL(tile_lstm_dbias_kernel, dim3(static_cast<unsigned>(4 * s.H)), dim3(256), 0, sm, s.dZ, s.TB,
                       dbias);
    ARD_LAUNCH_CHECK();
  }
  return ARD_OK;
}

}  // extern "C"
