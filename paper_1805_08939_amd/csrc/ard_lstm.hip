// LSTM layer with a row-based dropout pattern on its hidden units, fixed for
// the whole sequence (Sec. IV-C applies the method to LSTM's matrix products).
//
// Dropped units are removed from the layer: their h and c stay 0, so every
// gate GEMM runs on the compact set S of kept units. The layer compacts its
// weights once per sequence into the workspace:
//   Wc[4u + g][c] = W[g*H + S(u)][c]          for input columns c < I
//   Wc[4u + g][I + v] = W[g*H + S(u)][I + S(v)]  for recurrent columns
// with rows padded with zeros to a multiple of 4 entries (16-byte rows for
// the direct-load GEMMs whatever |S| is)
// Rows are unit-major (4u + g, g = i, f, g, o), so in the 32x32 MFMA
// accumulator layout each lane holds the four gates of one unit in four
// consecutive registers, and the cell update runs in registers.
//
// fwd: one batched GEMM for the input projection of all steps (bias folded
// in), then per step a kernel computing Wc_h h_{t-1} for a 32-row x 32-column
// tile (four waves split the contraction and reduce through LDS; 16 x 16
// tiles for small kept sets) fused with the gate nonlinearities and the state
// update.
// bwd: per step a split-K kernel for dh = Wc_h^T dA_{t+1} (the contraction
// over the 4 |S| gate rows cut into slices, one partial sum each, so that the
// small product still fills the chip), then the pointwise backward of step t,
// which adds the partial sums in a fixed order; for small kept sets instead
// one kernel per step that runs the whole contraction on 16 x 16 output tiles
// and the pointwise backward on its outputs. Then K-batched GEMMs over all
// steps for the weight gradients and one batched GEMM for dX.

#include <hip/hip_runtime.h>

#include <cmath>

#include "ard_gemm.hpp"
#include "ard_gemm_fast.hpp"
#include "ard_internal.hpp"

namespace ard {

namespace {

// 32 x 64 output tiles on eight waves (two columns of 32, four k shares of a
// 128-deep slab), three stages: the backward recurrence at a batch of 64.
using RecWideCfg = FastCfg<float, 32, 64, 128, 3, 1, 2, 4>;

struct Layout {
  int64_t T, B, I, H, ns, G4, KW, S;
  int64_t Ic, ip, io;  // kept inputs (compact input width) and their pattern
  int64_t R;           // first recurrent column of a compact row: Ic rounded up to 16 bytes
  size_t wc, bc, rowmap, z, cc, hc, da, dc, part, total;
};

// Splits of the backward recurrent contraction (length 4 ns): enough
// workgroups of 32 x 32 outputs to fill the chip twice, each split at least
// one 64-wide slab.
int64_t bwd_splits(int64_t ns, int64_t B) {
  const int64_t tiles = ((ns + 31) / 32) * ((B + 31) / 32);
  const int64_t slabs = (4 * ns + 63) / 64;
  int64_t sp = 512 / (tiles > 0 ? tiles : 1);
  if (sp > slabs) sp = slabs;
  return sp < 1 ? 1 : sp;
}

size_t al256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

Layout make_layout(const ard_lstm_desc* d, int32_t ns) {
  Layout L;
  L.T = d->seq_len;
  L.B = d->batch;
  L.I = d->input_size;
  L.H = d->hidden_size;
  L.ns = ns;
  L.G4 = 4 * static_cast<int64_t>(ns);
  const bool in_all = !d->input_plan || d->input_plan->period == 1;
  L.Ic = in_all ? L.I : d->input_plan->kept;
  L.ip = in_all ? 1 : d->input_plan->period;
  L.io = in_all ? 0 : d->input_plan->offset;
  // compact rows [Ic inputs][zeros to R][|S| recurrent][zeros to KW]: the
  // recurrent part starts on a 16-byte boundary whatever the input pattern
  // keeps, so the step kernels' direct loads can read it
  L.R = (L.Ic + 3) / 4 * 4;
  L.KW = (L.R + ns + 3) / 4 * 4;
  L.S = bwd_splits(ns, L.B);
  size_t off = 0;
  L.wc = off;     off += al256(4 * L.G4 * L.KW);
  L.bc = off;     off += al256(4 * L.G4 + 4);
  L.rowmap = off; off += al256(4 * L.G4 + 4);
  L.z = off;      off += al256(4 * L.T * L.G4 * L.B);
  L.cc = off;     off += al256(4 * (L.T + 1) * ns * L.B);
  L.hc = off;     off += al256(4 * (L.T + 1) * ns * L.B);
  L.da = off;     off += al256(4 * L.T * L.G4 * L.B);
  L.dc = off;     off += al256(4 * static_cast<int64_t>(ns) * L.B + 4);
  L.part = off;   off += al256(4 * L.S * ns * L.B + 4);
  L.total = off;
  return L;
}

}  // namespace

__device__ __forceinline__ int64_t unit_row(const int32_t* idx, int64_t u) { return idx ? idx[u] : u; }
__device__ __forceinline__ float sigm(float x) { return 1.0f / (1.0f + expf(-x)); }

// Compact weights (rows of KW entries: the Ic kept inputs, zeros up to R,
// the |S| kept recurrent columns from R on, zeros after), bias and row map;
// one block per compact row 4u + g.
__global__ void lstm_prepare_kernel(const float* __restrict__ W, const float* __restrict__ bias,
                                    const int32_t* __restrict__ idx, int32_t I, int32_t Ic, int32_t R, int32_t ip,
                                    int32_t io, int32_t H, int32_t ns, int32_t KW, float* __restrict__ Wc,
                                    float* __restrict__ bc, int32_t* __restrict__ rowmap) {
  const int r = blockIdx.x;
  const int u = r >> 2, g = r & 3;
  const int64_t src = static_cast<int64_t>(g) * H + unit_row(idx, u);
  const float* wrow = W + src * (I + H);
  float* crow = Wc + static_cast<int64_t>(r) * KW;
  for (int c = threadIdx.x; c < KW; c += blockDim.x)
    crow[c] = c < Ic                  ? wrow[io + static_cast<int64_t>(ip) * c]
              : c >= R && c < R + ns ? wrow[I + unit_row(idx, c - R)]
                                     : 0.0f;
  if (threadIdx.x == 0) {
    bc[r] = bias ? bias[src] : 0.0f;
    rowmap[r] = static_cast<int32_t>(src);
  }
}

// Compact initial state: dst[u][b] = src ? src[S(u)][b] : 0.
__global__ void lstm_gather_state_kernel(const float* __restrict__ src, const int32_t* __restrict__ idx,
                                         int32_t ns, int32_t B, float* __restrict__ dst) {
  const int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (e >= static_cast<int64_t>(ns) * B) return;
  const int64_t u = e / B, b = e % B;
  dst[e] = src ? src[unit_row(idx, u) * B + b] : 0.0f;
}

// Full state from compact: dst[j][b] = kept(j) ? src[u(j)][b] : 0 over H rows.
__global__ void lstm_scatter_state_kernel(const float* __restrict__ src, int32_t H, int32_t B,
                                          int32_t period, int32_t offset, float* __restrict__ dst) {
  const int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (e >= static_cast<int64_t>(H) * B) return;
  const int64_t j = e / B, b = e % B;
  dst[e] = (j % period == offset) ? src[((j - offset) / period) * B + b] : 0.0f;
}

// Zeroes rows r of out[rows][cols] whose unit (r % H) is dropped.
__global__ void lstm_zero_dropped_rows_kernel(float* __restrict__ out, int64_t rows, int32_t cols,
                                              int32_t H, int32_t period, int32_t offset) {
  const int64_t r = blockIdx.x;
  if (r >= rows || ((r % H) % period) == offset) return;
  for (int c = threadIdx.x; c < cols; c += blockDim.x) out[r * cols + c] = 0.0f;
}

// dW[4H][I+H]: zero the rows of dropped units, the recurrent columns of
// dropped units and the input columns of dropped inputs (pattern ip, io);
// dbias entries of dropped units.
__global__ void lstm_zero_dropped_dw_kernel(float* __restrict__ dW, float* __restrict__ dbias, int32_t I,
                                            int32_t H, int32_t period, int32_t offset, int32_t ip, int32_t io) {
  const int r = blockIdx.x;
  const bool row_kept = ((r % H) % period) == offset;
  float* row = dW + static_cast<int64_t>(r) * (I + H);
  for (int c = threadIdx.x; c < I + H; c += blockDim.x)
    if (!row_kept || (c >= I ? ((c - I) % period) != offset : (c % ip) != io)) row[c] = 0.0f;
  if (threadIdx.x == 0 && dbias && !row_kept) dbias[r] = 0.0f;
}

__global__ void fill_kernel(float* __restrict__ p, int64_t n, float v) {
  const int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (e < n) p[e] = v;
}

// rowmap[4u + g] = g H + idx[u]: the W row of compact gate row r, from the
// plan (the backward rebuilds it rather than trust the forward's workspace).
__global__ void lstm_rowmap_kernel(const int32_t* __restrict__ idx, int32_t H, int32_t rows,
                                   int32_t* __restrict__ rowmap) {
  const int r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r < rows) rowmap[r] = static_cast<int32_t>(static_cast<int64_t>(r & 3) * H + unit_row(idx, r >> 2));
}

// dbias[rowmap[r]] = sum over t, b of dA[t][r][b]; one block per row r.
__global__ void __launch_bounds__(256) lstm_dbias_kernel(const float* __restrict__ dA,
                                                         const int32_t* __restrict__ rowmap, int32_t T,
                                                         int32_t G4, int32_t B, float* __restrict__ dbias) {
  __shared__ float part[256];
  const int r = blockIdx.x;
  float s = 0.0f;
  for (int64_t e = threadIdx.x; e < static_cast<int64_t>(T) * B; e += 256) {
    const int64_t t = e / B, b = e % B;
    s += dA[(t * G4 + r) * B + b];
  }
  part[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (threadIdx.x < w) part[threadIdx.x] += part[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) dbias[rowmap[r]] = part[0];
}

struct LstmStep {
  const float* Wc;      // compact weights [G4][KW]
  const int32_t* idx;   // S list or NULL
  float* Z;             // [T][G4][B]: input projection + bias, then activated gates
  float* Cc;            // [T+1][ns][B]
  float* Hc;            // [T+1][ns][B]
  float* Hs;            // [T][H][B] output
  float* dA;            // [T][G4][B]
  float* dc;            // [ns][B] carry
  const float* dHs;     // [T][H][B]
  float* dh0;           // [H][B] or NULL (final backward step)
  int32_t t, B, I, H, ns, G4, KW;
  int32_t R;            // first recurrent column of a Wc row (16-byte aligned)
};

constexpr int kStepBK = 64;
constexpr int kStepLDK = kStepBK + 4;

// 32 x 32 output block over a contraction of length K held in two operand
// views; the four waves of the block take disjoint quarters of each 64-wide
// slab, then reduce through LDS. On return wave w holds, for its lane, the
// full sums of accumulator registers 4w..4w+3 (rows 8w + 4*(lane/32) + q,
// column lane % 32 of the block).
template <int AMODE, int BMODE>
__device__ __forceinline__ void splitk_32x32(const GemmOperand& a, const float* abase, const GemmOperand& b,
                                             const float* bbase, int m0, int n0, int M, int N, int K,
                                             float (&out)[4]) {
  __shared__ __attribute__((aligned(16))) float As[32 * kStepLDK];
  __shared__ __attribute__((aligned(16))) float Bs[32 * kStepLDK];
  __shared__ float red[4 * 16 * 64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int lr = lane & 31, lh = lane >> 5;
  f32x16 acc;
#pragma unroll
  for (int r = 0; r < 16; ++r) acc[r] = 0.0f;
  for (int k0 = 0; k0 < K; k0 += kStepBK) {
    load_tile<float, AMODE, false, 32, kStepBK, kStepLDK, 256>(a, abase, nullptr, As, m0, k0, M, K);
    load_tile<float, BMODE, false, 32, kStepBK, kStepLDK, 256>(b, bbase, nullptr, Bs, n0, k0, N, K);
    __syncthreads();
#pragma unroll
    for (int kk = 16 * w; kk < 16 * w + 16; kk += 8) {
      const f32x4 av = *reinterpret_cast<const f32x4*>(As + lr * kStepLDK + kk + 4 * lh);
      const f32x4 bv = *reinterpret_cast<const f32x4*>(Bs + lr * kStepLDK + kk + 4 * lh);
#pragma unroll
      for (int e = 0; e < 4; ++e) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(av[e], bv[e], acc, 0, 0, 0);
    }
    __syncthreads();
  }
#pragma unroll
  for (int r = 0; r < 16; ++r) red[(w * 16 + r) * 64 + lane] = acc[r];
  __syncthreads();
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    float s = 0.0f;
#pragma unroll
    for (int v = 0; v < 4; ++v) s += red[(v * 16 + 4 * w + q) * 64 + lane];
    out[q] = s;
  }
}

// Forward step t: gates of 8 units x 32 samples.
template <bool AVEC, bool BVEC>
__global__ void __launch_bounds__(256) lstm_fwd_step_kernel(LstmStep s) {
  const int r0 = blockIdx.y * 32, n0 = blockIdx.x * 32;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  GemmOperand a = {}, b = {};
  a.ld = s.KW;
  b.ld = s.B;
  const float* hprev = s.Hc + static_cast<int64_t>(s.t) * s.ns * s.B;
  float z[4];
  splitk_32x32<AVEC ? KC_VEC : KC_ELEM, BVEC ? MC_VEC : MC_ELEM>(a, s.Wc + s.R, b, hprev, r0, n0, s.G4, s.B,
                                                                  s.ns, z);
  const int64_t u = r0 / 4 + 2 * w + (lane >> 5);
  const int64_t col = n0 + (lane & 31);
  if (u >= s.ns || col >= s.B) return;
  float* Zt = s.Z + static_cast<int64_t>(s.t) * s.G4 * s.B;
  float gate[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) gate[q] = z[q] + Zt[(4 * u + q) * s.B + col];
  const float ig = sigm(gate[0]), fg = sigm(gate[1]), gg = tanhf(gate[2]), og = sigm(gate[3]);
  const float cp = s.Cc[(static_cast<int64_t>(s.t) * s.ns + u) * s.B + col];
  const float c = fg * cp + ig * gg;
  const float h = og * tanhf(c);
  Zt[(4 * u + 0) * s.B + col] = ig;
  Zt[(4 * u + 1) * s.B + col] = fg;
  Zt[(4 * u + 2) * s.B + col] = gg;
  Zt[(4 * u + 3) * s.B + col] = og;
  s.Cc[(static_cast<int64_t>(s.t + 1) * s.ns + u) * s.B + col] = c;
  s.Hc[(static_cast<int64_t>(s.t + 1) * s.ns + u) * s.B + col] = h;
  s.Hs[(static_cast<int64_t>(s.t) * s.H + unit_row(s.idx, u)) * s.B + col] = h;
}

// The same forward step on the direct-load pipeline: 32 gate rows x 32
// samples, the four waves splitting each slab's k; after the LDS reduction
// wave w holds the four gates of units r0 / 4 + 2 w + lane / 32. Needs
// 16-byte aligned rows (I, KW and B multiples of 4).
using StepCfg = FastCfg<float, 32, 32, 64, 4, 1, 1, 4>;  // 64 KB LDS

__global__ void __launch_bounds__(StepCfg::NT) lstm_fwd_step_fast_kernel(LstmStep s) {
  using Cfg = StepCfg;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int r0 = blockIdx.y * 32, n0 = blockIdx.x * 32;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  f32x16 acc[1][1];
#pragma unroll
  for (int r = 0; r < 16; ++r) acc[0][0][r] = 0.0f;
  const int nslab = (s.ns + Cfg::BK - 1) / Cfg::BK;
  SlabLoader<Cfg, false, true> ld;
  ld.wv = __builtin_amdgcn_readfirstlane(w);
  ld.lds0 = __builtin_amdgcn_readfirstlane(lds_addr(smem));
  ld.da.init(s.KW, r0, s.G4, ld.wv);
  ld.db.init(s.B, n0, s.B, ld.wv);
  ld.K = s.ns;
  ld.ik = 0;
  ld.is = 0;
  ld.left = nslab - 1;
  ld.a_step = Cfg::BK * 4;
  ld.b_step = static_cast<int64_t>(s.B) * Cfg::BK * 4;
  ld.a_wrap = 0;
  ld.b_wrap = 0;
  ld.na = uniform_ptr(reinterpret_cast<const char*>(s.Wc + s.R));
  ld.nb = uniform_ptr(reinterpret_cast<const char*>(s.Hc + static_cast<int64_t>(s.t) * s.ns * s.B));
  run_slabs<Cfg, false, true, true>(ld, nslab, s.ns, 0, acc, 0, 0, w * Cfg::KW, smem);
  // wave v's registers 4 w' .. 4 w' + 3 (rows 8 w' + 4 (lane / 32) + q) go to wave w'
  float* red = reinterpret_cast<float*>(smem);
  lds_barrier();
#pragma unroll
  for (int r = 0; r < 16; ++r) red[(w * 16 + r) * 64 + lane] = acc[0][0][r];
  lds_barrier();
  float z[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    float v = 0.0f;
#pragma unroll
    for (int u = 0; u < Cfg::KSPLIT; ++u) v += red[(u * 16 + 4 * w + q) * 64 + lane];
    z[q] = v;
  }
  const int64_t u = r0 / 4 + 2 * w + (lane >> 5);
  const int64_t col = n0 + (lane & 31);
  if (u >= s.ns || col >= s.B) return;
  float* Zt = s.Z + static_cast<int64_t>(s.t) * s.G4 * s.B;
  float gate[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) gate[q] = z[q] + Zt[(4 * u + q) * s.B + col];
  const float ig = sigm(gate[0]), fg = sigm(gate[1]), gg = tanhf(gate[2]), og = sigm(gate[3]);
  const float cp = s.Cc[(static_cast<int64_t>(s.t) * s.ns + u) * s.B + col];
  const float c = fg * cp + ig * gg;
  const float h = og * tanhf(c);
  Zt[(4 * u + 0) * s.B + col] = ig;
  Zt[(4 * u + 1) * s.B + col] = fg;
  Zt[(4 * u + 2) * s.B + col] = gg;
  Zt[(4 * u + 3) * s.B + col] = og;
  s.Cc[(static_cast<int64_t>(s.t + 1) * s.ns + u) * s.B + col] = c;
  s.Hc[(static_cast<int64_t>(s.t + 1) * s.ns + u) * s.B + col] = h;
  s.Hs[(static_cast<int64_t>(s.t) * s.H + unit_row(s.idx, u)) * s.B + col] = h;
}

// The same step on 16 x 16 tiles (four units x 16 samples), for kept sets
// whose 32 x 32 tiles leave most of the chip idle: four times the
// workgroups, each operand read twice as often. In the 16x16x4 MFMA
// accumulator layout lane l holds rows 4 (l / 16) .. + 3 of column l % 16,
// the four gates of one unit, so after the reduction wave 0 updates the
// cell of (unit l / 16, sample l % 16) in registers. A (k-contiguous): the
// recurrent columns of Wc; B (n-contiguous): h_{t-1}.
using StepCfg16 = FastCfg<float, 16, 16, 128, 4, 1, 1, 4>;  // 64 KB LDS

__global__ void __launch_bounds__(StepCfg16::NT) lstm_fwd_step16_kernel(LstmStep s) {
  using Cfg = StepCfg16;
  constexpr int ACPR = Cfg::BK * 4 / 16, BCPR = Cfg::BN * 4 / 16;
  static_assert(Cfg::BM == 16 && Cfg::BN == 16 && Cfg::NW == 4 && Cfg::KW % 8 == 0, "16 x 16 tile, 4 waves");
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int r0 = blockIdx.y * 16, n0 = blockIdx.x * 16;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int nslab = (s.ns + Cfg::BK - 1) / Cfg::BK;
  SlabLoader<Cfg, false, true> ld;
  ld.wv = __builtin_amdgcn_readfirstlane(w);
  ld.lds0 = __builtin_amdgcn_readfirstlane(lds_addr(smem));
  ld.da.init(s.KW, r0, s.G4, ld.wv);
  ld.db.init(s.B, n0, s.B, ld.wv);
  ld.K = s.ns;
  ld.ik = 0;
  ld.is = 0;
  ld.left = nslab - 1;
  ld.a_step = Cfg::BK * 4;
  ld.b_step = static_cast<int64_t>(s.B) * Cfg::BK * 4;
  ld.a_wrap = 0;
  ld.b_wrap = 0;
  ld.na = uniform_ptr(reinterpret_cast<const char*>(s.Wc + s.R));
  ld.nb = uniform_ptr(reinterpret_cast<const char*>(s.Hc + static_cast<int64_t>(s.t) * s.ns * s.B));
  f32x4 acc0 = {0.0f, 0.0f, 0.0f, 0.0f}, acc1 = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
  for (int q = 0; q < Cfg::STAGES - 1; ++q) ld.issue();
  const int mn = lane & 15, kl = lane >> 4;
  int cs = 0, ck = 0;
  for (int q = 0; q < nslab; ++q) {
    wait_vm<(Cfg::STAGES - 2) * Cfg::LPW>();
    lds_barrier();  // slab q is in LDS; no wave reads slab q - 1 any more
    const char* st = smem + cs * Cfg::STAGE;
    if (s.ns - ck < Cfg::BK) {
      fast_zero_tail<Cfg, Cfg::BM, false>(smem + cs * Cfg::STAGE, s.ns - ck);
      fast_zero_tail<Cfg, Cfg::BN, true>(smem + cs * Cfg::STAGE + Cfg::ABYTES, s.ns - ck);
      lds_barrier();
    }
    ld.issue();  // slab q + STAGES - 1, into the stage slab q - 1 held
#pragma unroll
    for (int j = 0; j < Cfg::KW / 4; j += 2) {
      const int k0 = w * Cfg::KW + 4 * j + kl;
      const float a0 = *reinterpret_cast<const float*>(st + kc_off<ACPR>(mn, k0 >> 2) + (k0 & 3) * 4);
      const float a1 = *reinterpret_cast<const float*>(st + kc_off<ACPR>(mn, (k0 + 4) >> 2) + (k0 & 3) * 4);
      const float b0v =
          *reinterpret_cast<const float*>(st + Cfg::ABYTES + mc_off<BCPR, 4>(k0, mn >> 2) + (mn & 3) * 4);
      const float b1v =
          *reinterpret_cast<const float*>(st + Cfg::ABYTES + mc_off<BCPR, 4>(k0 + 4, mn >> 2) + (mn & 3) * 4);
      acc0 = __builtin_amdgcn_mfma_f32_16x16x4f32(a0, b0v, acc0, 0, 0, 0);
      acc1 = __builtin_amdgcn_mfma_f32_16x16x4f32(a1, b1v, acc1, 0, 0, 0);
    }
    cs = cs + 1 == Cfg::STAGES ? 0 : cs + 1;
    ck += Cfg::BK;
  }
  wait_vm<0>();  // no direct load may still write LDS past this point
  float* red = reinterpret_cast<float*>(smem);
  lds_barrier();  // every wave is done with the stages
#pragma unroll
  for (int i = 0; i < 4; ++i) red[(w * 4 + i) * 64 + lane] = acc0[i] + acc1[i];
  lds_barrier();
  if (w != 0) return;
  float z[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    float v = 0.0f;
#pragma unroll
    for (int ww = 0; ww < 4; ++ww) v += red[(ww * 4 + q) * 64 + lane];
    z[q] = v;
  }
  const int64_t u = r0 / 4 + (lane >> 4);
  const int64_t col = n0 + (lane & 15);
  if (u >= s.ns || col >= s.B) return;
  float* Zt = s.Z + static_cast<int64_t>(s.t) * s.G4 * s.B;
  float gate[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) gate[q] = z[q] + Zt[(4 * u + q) * s.B + col];
  const float ig = sigm(gate[0]), fg = sigm(gate[1]), gg = tanhf(gate[2]), og = sigm(gate[3]);
  const float cp = s.Cc[(static_cast<int64_t>(s.t) * s.ns + u) * s.B + col];
  const float c = fg * cp + ig * gg;
  const float h = og * tanhf(c);
  Zt[(4 * u + 0) * s.B + col] = ig;
  Zt[(4 * u + 1) * s.B + col] = fg;
  Zt[(4 * u + 2) * s.B + col] = gg;
  Zt[(4 * u + 3) * s.B + col] = og;
  s.Cc[(static_cast<int64_t>(s.t + 1) * s.ns + u) * s.B + col] = c;
  s.Hc[(static_cast<int64_t>(s.t + 1) * s.ns + u) * s.B + col] = h;
  s.Hs[(static_cast<int64_t>(s.t) * s.H + unit_row(s.idx, u)) * s.B + col] = h;
}

// Pointwise backward of step t for unit u, sample b, given dL/dh_t.
__device__ __forceinline__ void lstm_point_bwd(const LstmStep& s, int t, int64_t u, int64_t b, float dh) {
  const float* Zt = s.Z + static_cast<int64_t>(t) * s.G4 * s.B;
  const float ig = Zt[(4 * u + 0) * s.B + b], fg = Zt[(4 * u + 1) * s.B + b];
  const float gg = Zt[(4 * u + 2) * s.B + b], og = Zt[(4 * u + 3) * s.B + b];
  const float c = s.Cc[(static_cast<int64_t>(t + 1) * s.ns + u) * s.B + b];
  const float cp = s.Cc[(static_cast<int64_t>(t) * s.ns + u) * s.B + b];
  const float tc = tanhf(c);
  const float d_o = dh * tc;
  const float dcv = s.dc[u * s.B + b] + dh * og * (1.0f - tc * tc);
  s.dc[u * s.B + b] = dcv * fg;
  float* dAt = s.dA + static_cast<int64_t>(t) * s.G4 * s.B;
  dAt[(4 * u + 0) * s.B + b] = dcv * gg * ig * (1.0f - ig);
  dAt[(4 * u + 1) * s.B + b] = dcv * cp * fg * (1.0f - fg);
  dAt[(4 * u + 2) * s.B + b] = dcv * ig * (1.0f - gg * gg);
  dAt[(4 * u + 3) * s.B + b] = d_o * og * (1.0f - og);
}

// Last step: dh = dHs[T-1] + dhT, dc carry starts at dcT.
__global__ void lstm_bwd_last_kernel(LstmStep s, const float* __restrict__ dhT, const float* __restrict__ dcT) {
  const int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (e >= static_cast<int64_t>(s.ns) * s.B) return;
  const int64_t u = e / s.B, b = e % s.B;
  const int64_t j = unit_row(s.idx, u);
  s.dc[e] = dcT ? dcT[j * s.B + b] : 0.0f;
  float dh = s.dHs[(static_cast<int64_t>(s.t) * s.H + j) * s.B + b];
  if (dhT) dh += dhT[j * s.B + b];
  lstm_point_bwd(s, s.t, u, b, dh);
}

// Partial sums of dh_rec = Wc_h^T dA[t]: workgroup (x, y, z) computes 32
// units x 32 samples over gate rows [z * ks, (z + 1) * ks) into part[z].
template <bool AVEC, bool BVEC>
__global__ void __launch_bounds__(256) lstm_bwd_rec_kernel(LstmStep s, float* __restrict__ part, int32_t ks) {
  const int m0 = blockIdx.y * 32, n0 = blockIdx.x * 32;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t k0 = static_cast<int64_t>(blockIdx.z) * ks;
  const int klen = static_cast<int>(s.G4 - k0 < ks ? s.G4 - k0 : ks);
  GemmOperand a = {}, b = {};
  a.ld = s.KW;
  b.ld = s.B;
  const float* dAt = s.dA + static_cast<int64_t>(s.t) * s.G4 * s.B;
  float z[4];
  splitk_32x32<AVEC ? MC_VEC : MC_ELEM, BVEC ? MC_VEC : MC_ELEM>(a, s.Wc + s.R + k0 * s.KW, b, dAt + k0 * s.B, m0,
                                                                  n0, s.ns, s.B, klen, z);
  const int64_t col = n0 + (lane & 31);
  if (col >= s.B) return;
  float* out = part + static_cast<int64_t>(blockIdx.z) * s.ns * s.B;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int64_t u = m0 + 8 * w + 4 * (lane >> 5) + q;
    if (u < s.ns) out[u * s.B + col] = z[q];
  }
}

// dh_rec of unit u, sample b: the splits' partial sums added in split order.
// The loads of up to eight splits are issued together, then added in order.
__device__ __forceinline__ float rec_sum(const float* __restrict__ part, int32_t splits, int64_t nsB, int64_t e) {
  float v = 0.0f;
  for (int z0 = 0; z0 < splits; z0 += 8) {
    float t[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) t[u] = z0 + u < splits ? part[(z0 + u) * nsB + e] : 0.0f;
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (z0 + u < splits) v += t[u];
  }
  return v;
}

// Pointwise backward of step t - 1 with dh = dHs[t - 1] + dh_rec (FINAL:
// dh0 = dh_rec instead), one thread per unit and sample.
template <bool FINAL>
__global__ void __launch_bounds__(256) lstm_bwd_point_kernel(LstmStep s, const float* __restrict__ part,
                                                             int32_t splits) {
  const int64_t nsB = static_cast<int64_t>(s.ns) * s.B;
  const int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (e >= nsB) return;
  const int64_t u = e / s.B, b = e % s.B;
  const int64_t j = unit_row(s.idx, u);
  const float r = rec_sum(part, splits, nsB, e);
  if (FINAL) {
    if (s.dh0) s.dh0[j * s.B + b] = r;
  } else {
    lstm_point_bwd(s, s.t - 1, u, b, s.dHs[(static_cast<int64_t>(s.t - 1) * s.H + j) * s.B + b] + r);
  }
}

// The backward recurrence in one launch per step. A workgroup owns 16 units x
// 16 samples of dh_rec = Wc_h^T dA[t] and runs the whole contraction over the
// 4 |S| gate rows itself (on the direct-load pipeline, the four waves on
// disjoint quarters of each slab, 16x16x4 fp32 MFMAs),
// adds the waves' sums through LDS in wave order, and the same threads then
// run the pointwise backward of step t - 1 on their outputs (after step 0:
// dh0 = dh_rec). Small output tiles give the grid its width in place of a
// split contraction, so no partial sums leave the workgroup and no second
// kernel is needed per step. A (m-contiguous): column I + u of Wc's gate rows;
// B (n-contiguous): dA[t]. Needs 16-byte aligned rows (I, KW and B multiples
// of 4). 128 gate rows per slab, 4 stages: the deeper 256-row slabs and 3 to
// 8 stages measured the same or slower.
using RecStepCfg = FastCfg<float, 16, 16, 128, 4, 1, 1, 4>;  // 64 KB LDS

template <bool FINAL>
__global__ void __launch_bounds__(RecStepCfg::NT) lstm_bwd_step_fused_kernel(LstmStep s) {
  using Cfg = RecStepCfg;
  constexpr int CPR = Cfg::BM * 4 / 16;  // 16-byte chunks per k-row of either operand
  static_assert(Cfg::BM == 16 && Cfg::BN == 16 && Cfg::NW == 4 && Cfg::KW % 8 == 0, "16 x 16 tile, 4 waves");
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int u0 = blockIdx.y * 16, b0 = blockIdx.x * 16;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int nslab = (s.G4 + Cfg::BK - 1) / Cfg::BK;
  SlabLoader<Cfg, true, true> ld;
  ld.wv = __builtin_amdgcn_readfirstlane(w);
  ld.lds0 = __builtin_amdgcn_readfirstlane(lds_addr(smem));
  ld.da.init(s.KW, u0, s.ns, ld.wv);
  ld.db.init(s.B, b0, s.B, ld.wv);
  ld.K = s.G4;
  ld.ik = 0;
  ld.is = 0;
  ld.left = nslab - 1;
  ld.a_step = static_cast<int64_t>(Cfg::BK) * s.KW * 4;
  ld.b_step = static_cast<int64_t>(Cfg::BK) * s.B * 4;
  ld.a_wrap = 0;
  ld.b_wrap = 0;
  ld.na = uniform_ptr(reinterpret_cast<const char*>(s.Wc + s.R));
  ld.nb = uniform_ptr(reinterpret_cast<const char*>(s.dA + static_cast<int64_t>(s.t) * s.G4 * s.B));
  // two accumulators on alternate k steps, so that consecutive MFMAs do not
  // wait for each other's result
  f32x4 acc0 = {0.0f, 0.0f, 0.0f, 0.0f}, acc1 = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
  for (int q = 0; q < Cfg::STAGES - 1; ++q) ld.issue();
  // MFMA operands: lane l holds A[m][k] and B[k][n] for m = n = l % 16 and
  // k = l / 16 of each 4-deep step
  const int mn = lane & 15, kl = lane >> 4;
  int cs = 0, ck = 0;
  for (int q = 0; q < nslab; ++q) {
    wait_vm<(Cfg::STAGES - 2) * Cfg::LPW>();
    lds_barrier();  // slab q is in LDS; no wave reads slab q - 1 any more
    const char* st = smem + cs * Cfg::STAGE;
    if (s.G4 - ck < Cfg::BK) {
      fast_zero_tail<Cfg, Cfg::BM, true>(smem + cs * Cfg::STAGE, s.G4 - ck);
      fast_zero_tail<Cfg, Cfg::BN, true>(smem + cs * Cfg::STAGE + Cfg::ABYTES, s.G4 - ck);
      lds_barrier();
    }
    ld.issue();  // slab q + STAGES - 1, into the stage slab q - 1 held
#pragma unroll
    for (int j = 0; j < Cfg::KW / 4; j += 2) {
      const int k0 = w * Cfg::KW + 4 * j + kl;
      const int o0 = mc_off<CPR, 4>(k0, mn >> 2) + (mn & 3) * 4;
      const int o1 = mc_off<CPR, 4>(k0 + 4, mn >> 2) + (mn & 3) * 4;
      const float a0 = *reinterpret_cast<const float*>(st + o0);
      const float b0v = *reinterpret_cast<const float*>(st + Cfg::ABYTES + o0);
      const float a1 = *reinterpret_cast<const float*>(st + o1);
      const float b1v = *reinterpret_cast<const float*>(st + Cfg::ABYTES + o1);
      acc0 = __builtin_amdgcn_mfma_f32_16x16x4f32(a0, b0v, acc0, 0, 0, 0);
      acc1 = __builtin_amdgcn_mfma_f32_16x16x4f32(a1, b1v, acc1, 0, 0, 0);
    }
    cs = cs + 1 == Cfg::STAGES ? 0 : cs + 1;
    ck += Cfg::BK;
  }
  wait_vm<0>();  // no direct load may still write LDS past this point
  // output (row r, column c) of the 16 x 16 MFMA tile: register r % 4 of lane
  // 16 (r / 4) + c
  float* red = reinterpret_cast<float*>(smem);
  lds_barrier();  // every wave is done with the stages
#pragma unroll
  for (int i = 0; i < 4; ++i) red[(w * 4 + i) * 64 + lane] = acc0[i] + acc1[i];
  lds_barrier();
  const int tm = threadIdx.x >> 4, tn = threadIdx.x & 15;
  const int src = (tm >> 2) * 16 + tn, reg = tm & 3;
  float v = 0.0f;
#pragma unroll
  for (int ww = 0; ww < 4; ++ww) v += red[(ww * 4 + reg) * 64 + src];
  const int64_t u = u0 + tm, b = b0 + tn;
  if (u >= s.ns || b >= s.B) return;
  const int64_t j = unit_row(s.idx, u);
  if (FINAL) {
    if (s.dh0) s.dh0[j * s.B + b] = v;
  } else {
    lstm_point_bwd(s, s.t - 1, u, b, s.dHs[(static_cast<int64_t>(s.t - 1) * s.H + j) * s.B + b] + v);
  }
}

namespace {

int check_lstm(const ard_lstm_desc* d, int32_t* ns, int32_t* period, int32_t* offset, const int32_t** idx) {
  if (!d) return fail(ARD_ERR_INVALID_ARG, "desc is NULL");
  if (d->dtype != ARD_F32) return fail(ARD_ERR_UNSUPPORTED, "LSTM supports ARD_F32 only");
  if (d->seq_len < 1 || d->batch < 1 || d->input_size < 1 || d->hidden_size < 1)
    return fail(ARD_ERR_INVALID_ARG, "sizes must be >= 1");
  int st = check_row_plan(d->hidden_plan, d->hidden_size, "hidden_plan", true);
  if (st != ARD_OK) return st;
  if ((st = check_row_plan(d->input_plan, d->input_size, "input_plan", false)) != ARD_OK) return st;
  if (d->input_plan && d->input_plan->kept == 0) return fail(ARD_ERR_INVALID_ARG, "input_plan keeps no input");
  const bool all = !d->hidden_plan || d->hidden_plan->period == 1;
  *ns = all ? d->hidden_size : d->hidden_plan->kept;
  *period = all ? 1 : d->hidden_plan->period;
  *offset = all ? 0 : d->hidden_plan->offset;
  *idx = all ? nullptr : d->hidden_plan->d_idx;
  return ARD_OK;
}

int check_ws(const Layout& L, void* ws, size_t ws_bytes) {
  if (!ws || ws_bytes < L.total)
    return fail(ARD_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", L.total, ws_bytes);
  if (!aligned16(ws)) return fail(ARD_ERR_INVALID_ARG, "workspace is not 16-byte aligned");
  return ARD_OK;
}

int check_opt(const void* p, const char* name) {
  if (p && !aligned16(p)) return fail(ARD_ERR_INVALID_ARG, "%s is not 16-byte aligned", name);
  return ARD_OK;
}

inline dim3 grid1d(int64_t n, int threads) { return dim3(static_cast<unsigned>((n + threads - 1) / threads)); }

LstmStep step_args(const Layout& L, char* w, const int32_t* idx) {
  LstmStep s = {};
  s.Wc = reinterpret_cast<const float*>(w + L.wc);
  s.idx = idx;
  s.Z = reinterpret_cast<float*>(w + L.z);
  s.Cc = reinterpret_cast<float*>(w + L.cc);
  s.Hc = reinterpret_cast<float*>(w + L.hc);
  s.dA = reinterpret_cast<float*>(w + L.da);
  s.dc = reinterpret_cast<float*>(w + L.dc);
  s.B = static_cast<int32_t>(L.B);
  s.I = static_cast<int32_t>(L.Ic);  // compact input width
  s.R = static_cast<int32_t>(L.R);   // the recurrent columns of Wc start here
  s.H = static_cast<int32_t>(L.H);
  s.ns = static_cast<int32_t>(L.ns);
  s.G4 = static_cast<int32_t>(L.G4);
  s.KW = static_cast<int32_t>(L.KW);
  return s;
}

}  // namespace
}  // namespace ard

using namespace ard;

extern "C" {

size_t ard_lstm_workspace_bytes(const ard_lstm_desc* desc) {
  int32_t ns, period, offset;
  const int32_t* idx;
  if (check_lstm(desc, &ns, &period, &offset, &idx) != ARD_OK) return 0;
  return make_layout(desc, ns).total;
}

int ard_lstm_fwd(const ard_lstm_desc* desc, const void* X, const void* W, const float* bias, const void* h0,
                 const void* c0, void* Hs, void* hT, void* cT, void* ws, size_t ws_bytes, void* stream) {
  clear_error();
  int32_t ns, period, offset;
  const int32_t* idx;
  int st = check_lstm(desc, &ns, &period, &offset, &idx);
  if (st != ARD_OK) return st;
  if (!X || !W || !Hs) return fail(ARD_ERR_INVALID_ARG, "X, W and Hs must not be NULL");
  if ((st = check_opt(X, "X")) || (st = check_opt(W, "W")) || (st = check_opt(Hs, "Hs")) ||
      (st = check_opt(bias, "bias")) || (st = check_opt(h0, "h0")) || (st = check_opt(c0, "c0")) ||
      (st = check_opt(hT, "hT")) || (st = check_opt(cT, "cT")))
    return st;
  const Layout L = make_layout(desc, ns);
  if ((st = check_ws(L, ws, ws_bytes))) return st;
  hipStream_t sm = static_cast<hipStream_t>(stream);
  char* w = static_cast<char*>(ws);
  LstmStep s = step_args(L, w, idx);
  float* Hsf = static_cast<float*>(Hs);
  s.Hs = Hsf;
  const int64_t HB = L.H * L.B;

  if (ns == 0) {  // every unit dropped: the layer outputs zeros
    hipLaunchKernelGGL(fill_kernel, grid1d(L.T * HB, 256), dim3(256), 0, sm, Hsf, L.T * HB, 0.0f);
    if (hT) hipLaunchKernelGGL(fill_kernel, grid1d(HB, 256), dim3(256), 0, sm, static_cast<float*>(hT), HB, 0.0f);
    if (cT) hipLaunchKernelGGL(fill_kernel, grid1d(HB, 256), dim3(256), 0, sm, static_cast<float*>(cT), HB, 0.0f);
    ARD_LAUNCH_CHECK();
    return ARD_OK;
  }

  hipLaunchKernelGGL(lstm_prepare_kernel, dim3(static_cast<unsigned>(L.G4)), dim3(256), 0, sm,
                     static_cast<const float*>(W), bias, idx, static_cast<int32_t>(L.I), s.I, s.R,
                     static_cast<int32_t>(L.ip), static_cast<int32_t>(L.io), s.H, ns, s.KW, const_cast<float*>(s.Wc),
                     reinterpret_cast<float*>(w + L.bc), reinterpret_cast<int32_t*>(w + L.rowmap));
  ARD_LAUNCH_CHECK();
  const int64_t nsB = static_cast<int64_t>(ns) * L.B;
  hipLaunchKernelGGL(lstm_gather_state_kernel, grid1d(nsB, 256), dim3(256), 0, sm,
                     static_cast<const float*>(h0), idx, ns, s.B, s.Hc);
  hipLaunchKernelGGL(lstm_gather_state_kernel, grid1d(nsB, 256), dim3(256), 0, sm,
                     static_cast<const float*>(c0), idx, ns, s.B, s.Cc);
  ARD_LAUNCH_CHECK();

  // input projection of every step, bias folded in: Z[t] = Wc_x X[t] + bc
  GemmArgs g = {};
  g.M = static_cast<int32_t>(L.G4);
  g.N = s.B;
  g.K = s.I;
  g.a = {s.Wc, nullptr, L.KW, nullptr, nullptr, 0, 0, 1.0f, 0};
  // the kept input rows io + ip * k of X[t]: a strided view
  g.b = {static_cast<const float*>(X) + L.io * L.B, nullptr, L.ip * L.B, nullptr, nullptr, L.I * L.B, 0, 1.0f, 0};
  g.c = {s.Z, L.B, nullptr, nullptr, L.G4 * L.B, reinterpret_cast<const float*>(w + L.bc), 0, 1.0f};
  const bool kw_vec = L.KW % 4 == 0;
  const bool b_vec = L.B % 4 == 0 && L.I % 4 == 0;
  if (fast_ok<false, true>(g, sizeof(float))) {
    ARD_HIP_CHECK((run_fast_gemm<float, false, true, float, EPI_FWD>(g, static_cast<int>(L.T), sm, nullptr)));
  } else {
    ARD_HIP_CHECK((run_gemm<float, float, KC_VEC, KC_ELEM, MC_VEC, MC_ELEM, false, false, EPI_FWD>(
        g, static_cast<int>(L.T), kw_vec, b_vec, sm)));
  }

  const dim3 sgrid(static_cast<unsigned>((L.B + 31) / 32), static_cast<unsigned>((L.G4 + 31) / 32));
  const bool avec = kw_vec, bvec = L.B % 4 == 0;  // the recurrent columns start aligned (R)
  // direct loads: aligned rows, and every chunk offset of a slab below 2^31 bytes
  const bool step_fast = avec && bvec && aligned16(s.Wc) &&
                         (L.G4 + 1) * L.KW * 4 < (int64_t{1} << 31) && (L.ns + 64) * L.B * 4 < (int64_t{1} << 31);
  // 16 x 16 tiles where the 32 x 32 grid holds fewer than 128 workgroups
  // (measured on MI355X, T 35, batch 64, H 1024: 255-269 against 288-290 us per
  // forward at |S| = 256, 210-218 against 237-244 us at 128, equal at 342 and
  // 64, slower at 512 and 1024)
  const bool step16 = step_fast && ((L.G4 + 31) / 32) * ((L.B + 31) / 32) < 128;
  if (step_fast) {
    static const hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void*>(lstm_fwd_step_fast_kernel),
                                                       hipFuncAttributeMaxDynamicSharedMemorySize, StepCfg::LDS);
    static const hipError_t attr16 = hipFuncSetAttribute(reinterpret_cast<const void*>(lstm_fwd_step16_kernel),
                                                         hipFuncAttributeMaxDynamicSharedMemorySize, StepCfg16::LDS);
    ARD_HIP_CHECK(attr);
    ARD_HIP_CHECK(attr16);
  }
  const dim3 sgrid16(static_cast<unsigned>((L.B + 15) / 16), static_cast<unsigned>((L.G4 + 15) / 16));
  for (int t = 0; t < L.T; ++t) {
    s.t = t;
    if (step16)
      hipLaunchKernelGGL(lstm_fwd_step16_kernel, sgrid16, dim3(StepCfg16::NT), StepCfg16::LDS, sm, s);
    else if (step_fast)
      hipLaunchKernelGGL(lstm_fwd_step_fast_kernel, sgrid, dim3(StepCfg::NT), StepCfg::LDS, sm, s);
    else if (avec && bvec)
      hipLaunchKernelGGL((lstm_fwd_step_kernel<true, true>), sgrid, dim3(256), 0, sm, s);
    else
      hipLaunchKernelGGL((lstm_fwd_step_kernel<false, false>), sgrid, dim3(256), 0, sm, s);
    ARD_LAUNCH_CHECK();
  }
  if (period > 1) {
    hipLaunchKernelGGL(lstm_zero_dropped_rows_kernel, dim3(static_cast<unsigned>(L.T * L.H)), dim3(256), 0, sm,
                       Hsf, L.T * L.H, s.B, s.H, period, offset);
    ARD_LAUNCH_CHECK();
  }
  if (hT)
    hipLaunchKernelGGL(lstm_scatter_state_kernel, grid1d(HB, 256), dim3(256), 0, sm,
                       s.Hc + L.T * nsB, s.H, s.B, period, offset, static_cast<float*>(hT));
  if (cT)
    hipLaunchKernelGGL(lstm_scatter_state_kernel, grid1d(HB, 256), dim3(256), 0, sm,
                       s.Cc + L.T * nsB, s.H, s.B, period, offset, static_cast<float*>(cT));
  ARD_LAUNCH_CHECK();
  return ARD_OK;
}

int ard_lstm_bwd(const ard_lstm_desc* desc, const void* X, const void* dHs, const void* dhT, const void* dcT,
                 void* ws, size_t ws_bytes, void* dX, float* dW, float* dbias, void* dh0, void* dc0,
                 void* stream) {
  clear_error();
  int32_t ns, period, offset;
  const int32_t* idx;
  int st = check_lstm(desc, &ns, &period, &offset, &idx);
  if (st != ARD_OK) return st;
  if (!X || !dHs) return fail(ARD_ERR_INVALID_ARG, "X and dHs must not be NULL");
  if ((st = check_opt(X, "X")) || (st = check_opt(dHs, "dHs")) || (st = check_opt(dhT, "dhT")) ||
      (st = check_opt(dcT, "dcT")) || (st = check_opt(dX, "dX")) || (st = check_opt(dW, "dW")) ||
      (st = check_opt(dbias, "dbias")) || (st = check_opt(dh0, "dh0")) || (st = check_opt(dc0, "dc0")))
    return st;
  const Layout L = make_layout(desc, ns);
  if ((st = check_ws(L, ws, ws_bytes))) return st;
  hipStream_t sm = static_cast<hipStream_t>(stream);
  char* w = static_cast<char*>(ws);
  LstmStep s = step_args(L, w, idx);
  s.dHs = static_cast<const float*>(dHs);
  const int64_t HB = L.H * L.B;
  const int64_t rowsW = 4 * L.H, colsW = L.I + L.H;

  if (ns == 0) {
    if (dX) hipLaunchKernelGGL(fill_kernel, grid1d(L.T * L.I * L.B, 256), dim3(256), 0, sm, static_cast<float*>(dX), L.T * L.I * L.B, 0.0f);
    if (dW) hipLaunchKernelGGL(fill_kernel, grid1d(rowsW * colsW, 256), dim3(256), 0, sm, dW, rowsW * colsW, 0.0f);
    if (dbias) hipLaunchKernelGGL(fill_kernel, grid1d(rowsW, 256), dim3(256), 0, sm, dbias, rowsW, 0.0f);
    if (dh0) hipLaunchKernelGGL(fill_kernel, grid1d(HB, 256), dim3(256), 0, sm, static_cast<float*>(dh0), HB, 0.0f);
    if (dc0) hipLaunchKernelGGL(fill_kernel, grid1d(HB, 256), dim3(256), 0, sm, static_cast<float*>(dc0), HB, 0.0f);
    ARD_LAUNCH_CHECK();
    return ARD_OK;
  }

  const int64_t nsB = static_cast<int64_t>(ns) * L.B;
  s.t = static_cast<int32_t>(L.T - 1);
  hipLaunchKernelGGL(lstm_bwd_last_kernel, grid1d(nsB, 256), dim3(256), 0, sm, s,
                     static_cast<const float*>(dhT), static_cast<const float*>(dcT));
  ARD_LAUNCH_CHECK();
  // dh_rec(t) by split-K partial sums, then the pointwise backward of step t - 1.
  // With a split count that divides the 4 |S| gate rows, the splits are the
  // batch of one strided direct-load GEMM (slice z: Wc_h^T rows z ks .. and
  // dA rows z ks .., output part[z]); otherwise the 32 x 32 split kernel.
  int32_t ks = static_cast<int32_t>(((L.G4 + L.S - 1) / L.S + 63) / 64 * 64);  // whole slabs per split
  int32_t splits = static_cast<int32_t>((L.G4 + ks - 1) / ks);
  float* part = reinterpret_cast<float*>(w + L.part);
  // exact split count for the direct-load GEMM (0 = none): its 32 x 32 tiles
  // run one workgroup per compute unit, so the splits stop at one round of
  // 256 workgroups (a second, partial round costs more than longer splits)
  const int64_t rtiles = ((ns + 31) / 32) * ((L.B + 31) / 32);
  int32_t fs = 0;
  for (int32_t d = static_cast<int32_t>(L.S); d >= 1; --d)
    if (L.G4 % d == 0 && L.G4 / d >= 256 && (d == 1 || rtiles * d <= 256)) {
      fs = d;
      break;
    }
  // A batch of 64 is one column of 32 x 64 tiles: each block of the recurrent
  // weights is then read by one workgroup per step instead of two. Taken when
  // those tiles alone fill one round of 256 workgroups.
  const int64_t wtiles = ((ns + 31) / 32) * ((L.B + 63) / 64);
  bool rec_wide = false;
  if (L.B > 32 && L.B <= 64) {
    for (int32_t d = static_cast<int32_t>(L.S); d >= 1; --d)
      if (L.G4 % d == 0 && L.G4 / d >= 256 && wtiles * d == 256) {
        fs = d;
        rec_wide = true;
        break;
      }
  }
  GemmArgs gr = {};
  bool rec_fast = false;
  if (fs > 0) {
    gr.M = ns;
    gr.N = s.B;
    gr.K = static_cast<int32_t>(L.G4 / fs);
    gr.a = {s.Wc + L.R, nullptr, L.KW, nullptr, nullptr, gr.K * L.KW, 0, 1.0f, 0};
    gr.b = {s.dA, nullptr, L.B, nullptr, nullptr, gr.K * L.B, 0, 1.0f, 0};
    gr.c = {part, L.B, nullptr, nullptr, nsB, nullptr, 0, 1.0f};
    rec_fast = fast_ok<true, true>(gr, sizeof(float));
    if (rec_fast) {
      ks = gr.K;
      splits = fs;
    }
  }
  const dim3 rgrid(static_cast<unsigned>((L.B + 31) / 32), static_cast<unsigned>((ns + 31) / 32),
                   static_cast<unsigned>(splits));
  const bool vec = L.KW % 4 == 0 && L.B % 4 == 0;
  // One fused launch per step where the direct loads can take the operands
  // (aligned rows; chunk offsets of a slab below 2^31 bytes) and the operand
  // stream stays small: 16-wide tiles read each operand twice as often as the
  // 32-wide tiles of the split path, ns * 4 ns * B / 2 bytes per step. Measured
  // on MI355X (T 35, batch 64, H 1024, backward per sequence): fused 262 / 329
  // / 373 / 514 us at |S| = 64 / 128 / 256 / 342 against 408 / 460 / 463 / 600
  // us split; 650 against 586 us at |S| = 512, where the stream is 32 MB.
  const bool rec_fused = vec && aligned16(s.Wc) && aligned16(s.dA) &&
                         int64_t{RecStepCfg::BK} * L.KW * 4 < (int64_t{1} << 31) &&
                         int64_t{RecStepCfg::BK} * L.B * 4 < (int64_t{1} << 31) &&
                         static_cast<int64_t>(ns) * L.G4 * L.B / 2 <= (int64_t{16} << 20);
  if (rec_fused) {
    static const hipError_t a0 = hipFuncSetAttribute(
        reinterpret_cast<const void*>(lstm_bwd_step_fused_kernel<false>), hipFuncAttributeMaxDynamicSharedMemorySize,
        RecStepCfg::LDS);
    static const hipError_t a1 = hipFuncSetAttribute(
        reinterpret_cast<const void*>(lstm_bwd_step_fused_kernel<true>), hipFuncAttributeMaxDynamicSharedMemorySize,
        RecStepCfg::LDS);
    ARD_HIP_CHECK(a0);
    ARD_HIP_CHECK(a1);
  }
  const dim3 fgrid(static_cast<unsigned>((L.B + 15) / 16), static_cast<unsigned>((ns + 15) / 16));
  for (int t = static_cast<int>(L.T) - 1; t >= 0; --t) {
    if (t == 0 && !dh0) break;
    s.t = t;
    if (rec_fused) {
      if (t > 0) {
        hipLaunchKernelGGL(lstm_bwd_step_fused_kernel<false>, fgrid, dim3(RecStepCfg::NT), RecStepCfg::LDS, sm, s);
      } else {
        s.dh0 = static_cast<float*>(dh0);
        hipLaunchKernelGGL(lstm_bwd_step_fused_kernel<true>, fgrid, dim3(RecStepCfg::NT), RecStepCfg::LDS, sm, s);
      }
      ARD_LAUNCH_CHECK();
      continue;
    }
    if (rec_fast) {
      gr.b.p = s.dA + static_cast<int64_t>(t) * L.G4 * L.B;
      if (rec_wide)
        ARD_HIP_CHECK((launch_fast<RecWideCfg, true, true, float, EPI_FWD>(gr, splits, sm)));
      else
        ARD_HIP_CHECK((run_fast_gemm<float, true, true, float, EPI_FWD>(gr, splits, sm, nullptr)));
    } else if (vec) {
      hipLaunchKernelGGL((lstm_bwd_rec_kernel<true, true>), rgrid, dim3(256), 0, sm, s, part, ks);
    } else {
      hipLaunchKernelGGL((lstm_bwd_rec_kernel<false, false>), rgrid, dim3(256), 0, sm, s, part, ks);
    }
    ARD_LAUNCH_CHECK();
    if (t > 0) {
      hipLaunchKernelGGL((lstm_bwd_point_kernel<false>), grid1d(nsB, 256), dim3(256), 0, sm, s, part, splits);
    } else {
      s.dh0 = static_cast<float*>(dh0);
      hipLaunchKernelGGL((lstm_bwd_point_kernel<true>), grid1d(nsB, 256), dim3(256), 0, sm, s, part, splits);
    }
    ARD_LAUNCH_CHECK();
  }
  if (dh0 && period > 1) {
    hipLaunchKernelGGL(lstm_zero_dropped_rows_kernel, dim3(static_cast<unsigned>(L.H)), dim3(256), 0, sm,
                       static_cast<float*>(dh0), L.H, s.B, s.H, period, offset);
    ARD_LAUNCH_CHECK();
  }
  if (dc0) {
    hipLaunchKernelGGL(lstm_scatter_state_kernel, grid1d(HB, 256), dim3(256), 0, sm, s.dc, s.H, s.B, period,
                       offset, static_cast<float*>(dc0));
    ARD_LAUNCH_CHECK();
  }

  // rowmap: built when a product below scatters through it
  int32_t* rowmap = reinterpret_cast<int32_t*>(w + L.rowmap);
  auto build_rowmap = [&]() -> hipError_t {
    if (L.G4 <= 0) return hipSuccess;
    hipLaunchKernelGGL(lstm_rowmap_kernel, grid1d(L.G4, 256), dim3(256), 0, sm, idx, static_cast<int32_t>(L.H),
                       static_cast<int32_t>(L.G4), rowmap);
    return hipGetLastError();
  };
  bool rowmap_built = false;
  const bool bv = L.B % 4 == 0;
  // Per gate q the compact rows 4u + q of dA are every fourth row, and the
  // output rows q H + S(u) and recurrent columns I + S(v) of a row pattern are
  // strided views of dW: the weight gradient runs as four plain strided
  // GEMMs (one launch, batched over the gates) when the operands allow.
  bool dw_done = false, dbias_done = false;
  if (dW) {
    GemmArgs g = {};
    g.M = ns;
    g.N = s.I;
    g.K = s.B;
    g.kbatch = static_cast<int32_t>(L.T);
    g.a = {s.dA, nullptr, 4 * L.B, nullptr, nullptr, L.B, 0, 1.0f, L.G4 * L.B};
    g.b = {static_cast<const float*>(X) + L.io * L.B, nullptr, L.ip * L.B, nullptr, nullptr, 0, 0, 1.0f, L.I * L.B};
    g.c = {dW + static_cast<int64_t>(offset) * colsW + L.io, period * colsW, nullptr, nullptr, L.H * colsW, nullptr,
           0, 1.0f};
    g.c.col_stride = L.ip;
    GemmArgs gr = g;  // recurrent columns
    gr.N = ns;
    gr.b = {s.Hc, nullptr, L.B, nullptr, nullptr, 0, 0, 1.0f, nsB};
    gr.c.p = dW + static_cast<int64_t>(offset) * colsW + L.I + offset;
    gr.c.col_stride = period;
    if (fast_ok<false, false>(g, sizeof(float)) && fast_ok<false, false>(gr, sizeof(float))) {
      // dbias[q H + S(u)] = sum over t, b of dA: the row sums of the first product's A
      if (dbias) {
        g.rsum = dbias + offset;
        g.rsum_ld = period;
        g.rsum_bstride = L.H;
      }
      ARD_HIP_CHECK((run_fast_gemm<float, false, false, float, EPI_FWD, true>(g, 4, sm, nullptr, &dbias_done)));
      ARD_HIP_CHECK((run_fast_gemm<float, false, false, float, EPI_FWD>(gr, 4, sm, nullptr)));
      dw_done = true;
    }
  }
  if (dW && !dw_done) {
    // dW[rowmap][:I] = sum_t dA[t] X[t]^T ; dW[rowmap][I + S] = sum_t dA[t] Hc[t]^T
    ARD_HIP_CHECK(build_rowmap());
    rowmap_built = true;
    GemmArgs g = {};
    g.M = static_cast<int32_t>(L.G4);
    g.N = s.I;
    g.K = s.B;
    g.kbatch = static_cast<int32_t>(L.T);
    g.a = {s.dA, nullptr, L.B, nullptr, nullptr, 0, 0, 1.0f, L.G4 * L.B};
    g.b = {static_cast<const float*>(X) + L.io * L.B, nullptr, L.ip * L.B, nullptr, nullptr, 0, 0, 1.0f, L.I * L.B};
    g.c = {dW + L.io, colsW, rowmap, nullptr, 0, nullptr, 0, 1.0f};
    g.c.col_stride = L.ip;
    ARD_HIP_CHECK((run_gemm<float, float, KC_VEC, KC_ELEM, KC_VEC, KC_ELEM, false, false, EPI_FWD>(
        g, 1, bv, bv && L.I % 4 == 0, sm)));
    g.N = ns;
    g.b = {s.Hc, nullptr, L.B, nullptr, nullptr, 0, 0, 1.0f, nsB};
    g.c = {dW + L.I, colsW, rowmap, idx, 0, nullptr, 0, 1.0f};
    ARD_HIP_CHECK((run_gemm<float, float, KC_VEC, KC_ELEM, KC_VEC, KC_ELEM, false, false, EPI_FWD>(
        g, 1, bv, bv, sm)));
  }
  if (dbias && !dbias_done) {
    if (!rowmap_built) ARD_HIP_CHECK(build_rowmap());
    hipLaunchKernelGGL(lstm_dbias_kernel, dim3(static_cast<unsigned>(L.G4)), dim3(256), 0, sm, s.dA, rowmap,
                       static_cast<int32_t>(L.T), static_cast<int32_t>(L.G4), s.B, dbias);
    ARD_LAUNCH_CHECK();
  }
  if ((period > 1 && (dW || dbias)) || (L.ip > 1 && dW)) {
    if (dW) {
      hipLaunchKernelGGL(lstm_zero_dropped_dw_kernel, dim3(static_cast<unsigned>(rowsW)), dim3(256), 0, sm, dW,
                         dbias, static_cast<int32_t>(L.I), s.H, period, offset, static_cast<int32_t>(L.ip),
                         static_cast<int32_t>(L.io));
    } else {
      hipLaunchKernelGGL(lstm_zero_dropped_rows_kernel, dim3(static_cast<unsigned>(rowsW)), dim3(64), 0, sm,
                         dbias, rowsW, 1, s.H, period, offset);
    }
    ARD_LAUNCH_CHECK();
  }
  if (dX) {
    // dX[t] = Wc_x^T dA[t] for every step
    GemmArgs g = {};
    g.M = s.I;
    g.N = s.B;
    g.K = static_cast<int32_t>(L.G4);
    g.a = {s.Wc, nullptr, L.KW, nullptr, nullptr, 0, 0, 1.0f, 0};
    g.b = {s.dA, nullptr, L.B, nullptr, nullptr, L.G4 * L.B, 0, 1.0f, 0};
    // rows io + ip * k of dX[t]; the rows of dropped inputs are written 0
    g.c = {static_cast<float*>(dX) + L.io * L.B, L.ip * L.B, nullptr, nullptr, L.I * L.B, nullptr, 0, 1.0f};
    if (fast_ok<true, true>(g, sizeof(float))) {
      ARD_HIP_CHECK((run_fast_gemm<float, true, true, float, EPI_FWD>(g, static_cast<int>(L.T), sm, nullptr)));
    } else {
      ARD_HIP_CHECK((run_gemm<float, float, MC_VEC, MC_ELEM, MC_VEC, MC_ELEM, false, false, EPI_FWD>(
          g, static_cast<int>(L.T), L.KW % 4 == 0 && L.Ic % 4 == 0, bv, sm)));
    }
    if (L.ip > 1) {
      hipLaunchKernelGGL(lstm_zero_dropped_rows_kernel, dim3(static_cast<unsigned>(L.T * L.I)), dim3(256), 0, sm,
                         static_cast<float*>(dX), L.T * L.I, s.B, static_cast<int32_t>(L.I),
                         static_cast<int32_t>(L.ip), static_cast<int32_t>(L.io));
      ARD_LAUNCH_CHECK();
    }
  }
  return ARD_OK;
}

}  // extern "C"
