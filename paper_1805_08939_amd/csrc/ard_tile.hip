// Tile-based dropout pattern (Sec. III-B): compaction of the kept-tile bitmap
// into gather lists, and the layer's fwd / bwd_data / bwd_weight on kept tiles.
//
// Sec. III-B fetches only non-dropped tiles and lets each processing element
// multiply one tile pair. Here a workgroup owns one tile row (fwd) or one tile
// column (bwd_data) of W and walks that row's (column's) list of kept tiles,
// each a dense tile x tile MFMA slab; bwd_weight runs one workgroup per kept
// tile. Dropped tiles are never read or computed.

#include <hip/hip_runtime.h>

#include "ard_gemm.hpp"
#include "ard_internal.hpp"

namespace ard {

constexpr int kScanThreads = 1024;
constexpr int kMaxTileDim = 8192;  // tiles per side handled by the scan kernel

// Exclusive scan of cnt[0..n) (LDS, n >= 1): writes the n+1 prefix sums to out
// and leaves the exclusive prefix in cnt.
__device__ void block_exclusive_scan(int32_t* cnt, int n, int32_t* out, int32_t* part) {
  const int tid = threadIdx.x;
  const int per = (n + kScanThreads - 1) / kScanThreads;
  const int lo = min(n, tid * per), hi = min(n, lo + per);
  int32_t s = 0;
  for (int i = lo; i < hi; ++i) s += cnt[i];
  part[tid] = s;
  __syncthreads();
  if (tid == 0) {  // kScanThreads partial sums
    int32_t run = 0;
    for (int i = 0; i < kScanThreads; ++i) {
      const int32_t v = part[i];
      part[i] = run;
      run += v;
    }
  }
  __syncthreads();
  int32_t run = part[tid];
  for (int i = lo; i < hi; ++i) {
    const int32_t c = cnt[i];
    out[i] = run;
    cnt[i] = run;  // the prefix stays in LDS for the list-writing pass
    run += c;
  }
  if (hi == n && lo < hi) out[n] = run;
  __syncthreads();
}

__device__ __forceinline__ bool tile_bit(const uint32_t* bits, int64_t t) {
  return (bits[t >> 5] >> (t & 31)) & 1u;
}

// One workgroup: bitmap -> row_ptr/row_cols (CSR), col_ptr/col_rows (CSC), flat.
__global__ void __launch_bounds__(kScanThreads)
    plan_tiles_kernel(const uint32_t* __restrict__ bits, int32_t tiles_n, int32_t tiles_k,
                      int32_t* __restrict__ row_ptr, int32_t* __restrict__ row_cols,
                      int32_t* __restrict__ col_ptr, int32_t* __restrict__ col_rows,
                      int32_t* __restrict__ flat) {
  __shared__ int32_t cnt[kMaxTileDim];
  __shared__ int32_t part[kScanThreads];
  const int tid = threadIdx.x;
  // rows
  for (int r = tid; r < tiles_n; r += kScanThreads) {
    int32_t c = 0;
    for (int k = 0; k < tiles_k; ++k) c += tile_bit(bits, static_cast<int64_t>(r) * tiles_k + k);
    cnt[r] = c;
  }
  __syncthreads();
  block_exclusive_scan(cnt, tiles_n, row_ptr, part);
  for (int r = tid; r < tiles_n; r += kScanThreads) {
    int32_t w = cnt[r];
    for (int k = 0; k < tiles_k; ++k) {
      const int64_t t = static_cast<int64_t>(r) * tiles_k + k;
      if (tile_bit(bits, t)) {
        row_cols[w] = k;
        flat[w] = static_cast<int32_t>(t);
        ++w;
      }
    }
  }
  __syncthreads();
  // columns
  for (int k = tid; k < tiles_k; k += kScanThreads) {
    int32_t c = 0;
    for (int r = 0; r < tiles_n; ++r) c += tile_bit(bits, static_cast<int64_t>(r) * tiles_k + k);
    cnt[k] = c;
  }
  __syncthreads();
  block_exclusive_scan(cnt, tiles_k, col_ptr, part);
  for (int k = tid; k < tiles_k; k += kScanThreads) {
    int32_t w = cnt[k];
    for (int r = 0; r < tiles_n; ++r)
      if (tile_bit(bits, static_cast<int64_t>(r) * tiles_k + k)) col_rows[w++] = r;
  }
}

enum TdpPass { TDP_FWD = 0, TDP_BWD_DATA = 1, TDP_BWD_WEIGHT = 2 };

struct TdpArgs {
  const void* act;      // Xt (fwd, bwd_weight) or dYt (bwd_data)
  const void* act2;     // dYt (bwd_weight)
  const void* W;
  void* out;            // Yt, dXt or dW
  int32_t B, N, K, tile, tiles_k;
  const int32_t* ptr;   // row_ptr (fwd) or col_ptr (bwd_data)
  const int32_t* list;  // row_cols (fwd), col_rows (bwd_data) or flat (bwd_weight)
  float scale;
};

template <typename T, typename OutT, class Cfg, int PASS, bool VEC>
__global__ void __launch_bounds__(Cfg::NT) tdp_kernel(TdpArgs a) {
  constexpr int LDK = Cfg::BK + 16 / sizeof(T);
  __shared__ __attribute__((aligned(16))) T As[Cfg::BM * LDK];
  __shared__ __attribute__((aligned(16))) T Bs[Cfg::BN * LDK];
  constexpr int KCM = VEC ? KC_VEC : KC_ELEM;
  constexpr int MCM = VEC ? MC_VEC : MC_ELEM;
  const int wave = threadIdx.x >> 6;
  const int wm = wave / Cfg::WGN, wn = wave % Cfg::WGN;
  const int T_ = a.tile;

  f32x16 acc[Cfg::FM][Cfg::FN];
#pragma unroll
  for (int i = 0; i < Cfg::FM; ++i)
#pragma unroll
    for (int j = 0; j < Cfg::FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  GemmOperand opa = {}, opb = {};
  GemmArgs st = {};
  st.c.relu = 0;
  st.c.scale = a.scale;
  int n0 = 0;
  const T* W = static_cast<const T*>(a.W);

  if constexpr (PASS == TDP_FWD || PASS == TDP_BWD_DATA) {
    // fwd: Yt[tn-block][:] += W(tn, tk) Xt[tk-block][:] over kept tk of tile row tn
    // bwd_data: dXt[tk-block][:] += W(tn, tk)^T dYt[tn-block][:] over kept tn of column tk
    const int own = blockIdx.y;  // tn (fwd) or tk (bwd_data)
    n0 = blockIdx.x * Cfg::BN;
    const T* act = static_cast<const T*>(a.act);
    opa.ld = a.K;
    opb.ld = a.B;
    const int s0 = a.ptr[own], s1 = a.ptr[own + 1];
    for (int s = s0; s < s1; ++s) {
      const int other = a.list[s];
      const int tn = PASS == TDP_FWD ? own : other;
      const int tk = PASS == TDP_FWD ? other : own;
      const T* Ab = W + static_cast<int64_t>(tn) * T_ * a.K + static_cast<int64_t>(tk) * T_;
      const T* Bb = act + static_cast<int64_t>(PASS == TDP_FWD ? tk : tn) * T_ * a.B;
      for (int kk = 0; kk < T_; kk += Cfg::BK) {
        if constexpr (PASS == TDP_FWD)
          load_tile<T, KC_VEC, false, Cfg::BM, Cfg::BK, LDK, Cfg::NT>(opa, Ab, nullptr, As, 0, kk, T_, T_);
        else
          load_tile<T, MC_VEC, false, Cfg::BM, Cfg::BK, LDK, Cfg::NT>(opa, Ab, nullptr, As, 0, kk, T_, T_);
        load_tile<T, MCM, false, Cfg::BN, Cfg::BK, LDK, Cfg::NT>(opb, Bb, nullptr, Bs, n0, kk, a.B, T_);
        __syncthreads();
        mma_slab<T, Cfg, LDK>(As, Bs, acc, wm, wn);
        __syncthreads();
      }
    }
    st.M = T_;
    st.N = a.B;
    st.c.p = static_cast<OutT*>(a.out) + static_cast<int64_t>(own) * T_ * a.B;
    st.c.ld = a.B;
  } else {
    // bwd_weight: dW(tn, tk) = dYt[tn-block][:] Xt[tk-block][:]^T for one kept tile
    const int t = a.list[blockIdx.x];
    const int tn = t / a.tiles_k, tk = t % a.tiles_k;
    const T* Ab = static_cast<const T*>(a.act2) + static_cast<int64_t>(tn) * T_ * a.B;
    const T* Bb = static_cast<const T*>(a.act) + static_cast<int64_t>(tk) * T_ * a.B;
    opa.ld = a.B;
    opb.ld = a.B;
    for (int kb = 0; kb < a.B; kb += Cfg::BK) {
      load_tile<T, KCM, false, Cfg::BM, Cfg::BK, LDK, Cfg::NT>(opa, Ab, nullptr, As, 0, kb, T_, a.B);
      load_tile<T, KCM, false, Cfg::BN, Cfg::BK, LDK, Cfg::NT>(opb, Bb, nullptr, Bs, 0, kb, T_, a.B);
      __syncthreads();
      mma_slab<T, Cfg, LDK>(As, Bs, acc, wm, wn);
      __syncthreads();
    }
    st.M = T_;
    st.N = T_;
    st.c.p = static_cast<OutT*>(a.out) + static_cast<int64_t>(tn) * T_ * a.K + static_cast<int64_t>(tk) * T_;
    st.c.ld = a.K;
  }
  store_tile<OutT, Cfg, EPI_FWD>(st, acc, 0, n0, wm, wn, 0, 0);
}

// ZERO mode: clears every dropped tile of dW.
__global__ void zero_dropped_tiles_kernel(const uint32_t* __restrict__ bits, float* __restrict__ dW,
                                          int32_t K, int32_t tile, int32_t tiles_k) {
  const int tk = blockIdx.x, tn = blockIdx.y;
  if (tile_bit(bits, static_cast<int64_t>(tn) * tiles_k + tk)) return;
  float* base = dW + static_cast<int64_t>(tn) * tile * K + static_cast<int64_t>(tk) * tile;
  for (int e = threadIdx.x; e < tile * tile; e += blockDim.x) base[(e / tile) * static_cast<int64_t>(K) + e % tile] = 0.0f;
}

namespace {

template <typename T>
struct TdpCfgs;
template <>
struct TdpCfgs<bf16> {
  using Rows64 = TileCfg<64, 128, 32, 2, 2>;
  using Rows32 = TileCfg<32, 128, 32, 1, 4>;
  using Tile64 = TileCfg<64, 64, 32, 2, 2>;
  using Tile32 = TileCfg<32, 32, 32, 1, 1>;
};
template <>
struct TdpCfgs<float> {
  using Rows64 = TileCfg<64, 128, 16, 2, 2>;
  using Rows32 = TileCfg<32, 128, 16, 1, 4>;
  using Tile64 = TileCfg<64, 64, 16, 2, 2>;
  using Tile32 = TileCfg<32, 32, 16, 1, 1>;
};

template <typename T, typename OutT, class Cfg, int PASS>
hipError_t launch_tdp(const TdpArgs& a, dim3 grid, bool vec, hipStream_t s) {
  if (vec)
    hipLaunchKernelGGL((tdp_kernel<T, OutT, Cfg, PASS, true>), grid, dim3(Cfg::NT), 0, s, a);
  else
    hipLaunchKernelGGL((tdp_kernel<T, OutT, Cfg, PASS, false>), grid, dim3(Cfg::NT), 0, s, a);
  return hipGetLastError();
}

template <typename T>
hipError_t run_tdp(int pass, const TdpArgs& a, int owners, int nnz, hipStream_t s) {
  const bool vec = (static_cast<int64_t>(a.B) * sizeof(T)) % 16 == 0;
  using C = TdpCfgs<T>;
  if (pass == TDP_BWD_WEIGHT) {
    if (nnz == 0) return hipSuccess;
    if (a.tile == 64) return launch_tdp<T, float, typename C::Tile64, TDP_BWD_WEIGHT>(a, dim3(nnz), vec, s);
    return launch_tdp<T, float, typename C::Tile32, TDP_BWD_WEIGHT>(a, dim3(nnz), vec, s);
  }
  const dim3 grid((a.B + 127) / 128, owners);
  if (pass == TDP_FWD) {
    if (a.tile == 64) return launch_tdp<T, T, typename C::Rows64, TDP_FWD>(a, grid, vec, s);
    return launch_tdp<T, T, typename C::Rows32, TDP_FWD>(a, grid, vec, s);
  }
  if (a.tile == 64) return launch_tdp<T, T, typename C::Rows64, TDP_BWD_DATA>(a, grid, vec, s);
  return launch_tdp<T, T, typename C::Rows32, TDP_BWD_DATA>(a, grid, vec, s);
}

size_t align256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

int check_tile_call(const ard_tile_desc* d, const ard_tile_plan* p) {
  if (!d || !p) return fail(ARD_ERR_INVALID_ARG, "desc or plan is NULL");
  if (d->dtype != ARD_F32 && d->dtype != ARD_BF16)
    return fail(ARD_ERR_UNSUPPORTED, "dtype %d not supported", d->dtype);
  if (d->batch < 1) return fail(ARD_ERR_INVALID_ARG, "batch must be >= 1");
  if (d->dropped != ARD_DROPPED_ZERO && d->dropped != ARD_DROPPED_SKIP)
    return fail(ARD_ERR_INVALID_ARG, "unknown dropped-output mode %d", d->dropped);
  if (!(d->scale == d->scale) || d->scale == __builtin_inff() || d->scale == -__builtin_inff())
    return fail(ARD_ERR_INVALID_ARG, "scale must be finite");
  if (p->tile != 32 && p->tile != 64) return fail(ARD_ERR_INVALID_ARG, "plan tile must be 32 or 64");
  if (d->in_features != p->k || d->out_features != p->n)
    return fail(ARD_ERR_INVALID_ARG, "desc (%d -> %d) does not match the plan (%d x %d)",
                d->in_features, d->out_features, p->n, p->k);
  if (p->tiles_n != p->n / p->tile || p->tiles_k != p->k / p->tile || p->n % p->tile || p->k % p->tile)
    return fail(ARD_ERR_INVALID_ARG, "plan tile grid is inconsistent");
  if (p->nnz < 0 || p->nnz > p->tiles_n * p->tiles_k) return fail(ARD_ERR_INVALID_ARG, "plan nnz out of range");
  if (!p->d_bits || !p->d_row_ptr || !p->d_row_cols || !p->d_col_ptr || !p->d_col_rows || !p->d_flat)
    return fail(ARD_ERR_INVALID_ARG, "plan has NULL lists");
  return ARD_OK;
}

int check_dev_ptr(const void* p, const char* name) {
  if (!p) return fail(ARD_ERR_INVALID_ARG, "%s is NULL", name);
  if (!aligned16(p)) return fail(ARD_ERR_INVALID_ARG, "%s is not 16-byte aligned", name);
  return ARD_OK;
}

}  // namespace
}  // namespace ard

using namespace ard;

extern "C" {

size_t ard_tile_plan_workspace_bytes(int32_t tiles_n, int32_t tiles_k) {
  if (tiles_n < 1 || tiles_k < 1) return 0;
  const size_t nnz = static_cast<size_t>(tiles_n) * tiles_k;
  return align256(4 * (tiles_n + 1)) + align256(4 * (tiles_k + 1)) + 3 * align256(4 * nnz);
}

int ard_plan_tiles(int32_t n, int32_t k, int32_t tile, const uint32_t* d_bits, int32_t nnz, void* d_ws,
                   size_t ws_bytes, ard_tile_plan* plan, void* stream) {
  clear_error();
  if (!plan) return fail(ARD_ERR_INVALID_ARG, "plan is NULL");
  if (tile != 32 && tile != 64) return fail(ARD_ERR_INVALID_ARG, "tile must be 32 or 64, got %d", tile);
  if (n < tile || k < tile || n % tile || k % tile)
    return fail(ARD_ERR_INVALID_ARG, "n (%d) and k (%d) must be positive multiples of the tile %d", n, k, tile);
  const int32_t tn = n / tile, tk = k / tile;
  if (tn > kMaxTileDim || tk > kMaxTileDim)
    return fail(ARD_ERR_UNSUPPORTED, "tile grid %d x %d exceeds %d per side", tn, tk, kMaxTileDim);
  if (nnz < 0 || static_cast<int64_t>(nnz) > static_cast<int64_t>(tn) * tk)
    return fail(ARD_ERR_INVALID_ARG, "nnz %d out of range", nnz);
  if (!d_bits) return fail(ARD_ERR_INVALID_ARG, "d_bits is NULL");
  const size_t need = ard_tile_plan_workspace_bytes(tn, tk);
  if (!d_ws || ws_bytes < need)
    return fail(ARD_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need, ws_bytes);
  if (!aligned16(d_ws)) return fail(ARD_ERR_INVALID_ARG, "workspace is not 16-byte aligned");
  char* w = static_cast<char*>(d_ws);
  const size_t full = static_cast<size_t>(tn) * tk;
  plan->n = n;
  plan->k = k;
  plan->tile = tile;
  plan->tiles_n = tn;
  plan->tiles_k = tk;
  plan->nnz = nnz;
  plan->d_bits = d_bits;
  plan->d_row_ptr = reinterpret_cast<int32_t*>(w);
  w += align256(4 * (tn + 1));
  plan->d_col_ptr = reinterpret_cast<int32_t*>(w);
  w += align256(4 * (tk + 1));
  plan->d_row_cols = reinterpret_cast<int32_t*>(w);
  w += align256(4 * full);
  plan->d_col_rows = reinterpret_cast<int32_t*>(w);
  w += align256(4 * full);
  plan->d_flat = reinterpret_cast<int32_t*>(w);
  hipLaunchKernelGGL(plan_tiles_kernel, dim3(1), dim3(kScanThreads), 0, static_cast<hipStream_t>(stream),
                     d_bits, tn, tk, plan->d_row_ptr, plan->d_row_cols, plan->d_col_ptr,
                     plan->d_col_rows, plan->d_flat);
  ARD_LAUNCH_CHECK();
  return ARD_OK;
}

int ard_tile_fwd(const ard_tile_desc* desc, const ard_tile_plan* plan, const void* Xt, const void* W,
                 void* Yt, void* stream) {
  clear_error();
  int st = check_tile_call(desc, plan);
  if (st != ARD_OK) return st;
  if ((st = check_dev_ptr(Xt, "Xt")) || (st = check_dev_ptr(W, "W")) || (st = check_dev_ptr(Yt, "Yt")))
    return st;
  TdpArgs a = {Xt, nullptr, W, Yt, desc->batch, plan->n, plan->k, plan->tile, plan->tiles_k,
               plan->d_row_ptr, plan->d_row_cols, desc->scale};
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (desc->dtype == ARD_BF16) {
    ARD_HIP_CHECK(run_tdp<bf16>(TDP_FWD, a, plan->tiles_n, plan->nnz, s));
  } else {
    ARD_HIP_CHECK(run_tdp<float>(TDP_FWD, a, plan->tiles_n, plan->nnz, s));
  }
  return ARD_OK;
}

int ard_tile_bwd_data(const ard_tile_desc* desc, const ard_tile_plan* plan, const void* dYt,
                      const void* W, void* dXt, void* stream) {
  clear_error();
  int st = check_tile_call(desc, plan);
  if (st != ARD_OK) return st;
  if ((st = check_dev_ptr(dYt, "dYt")) || (st = check_dev_ptr(W, "W")) || (st = check_dev_ptr(dXt, "dXt")))
    return st;
  TdpArgs a = {dYt, nullptr, W, dXt, desc->batch, plan->n, plan->k, plan->tile, plan->tiles_k,
               plan->d_col_ptr, plan->d_col_rows, desc->scale};
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (desc->dtype == ARD_BF16) {
    ARD_HIP_CHECK(run_tdp<bf16>(TDP_BWD_DATA, a, plan->tiles_k, plan->nnz, s));
  } else {
    ARD_HIP_CHECK(run_tdp<float>(TDP_BWD_DATA, a, plan->tiles_k, plan->nnz, s));
  }
  return ARD_OK;
}

int ard_tile_bwd_weight(const ard_tile_desc* desc, const ard_tile_plan* plan, const void* Xt,
                        const void* dYt, float* dW, void* stream) {
  clear_error();
  int st = check_tile_call(desc, plan);
  if (st != ARD_OK) return st;
  if ((st = check_dev_ptr(Xt, "Xt")) || (st = check_dev_ptr(dYt, "dYt")) || (st = check_dev_ptr(dW, "dW")))
    return st;
  TdpArgs a = {Xt, dYt, nullptr, dW, desc->batch, plan->n, plan->k, plan->tile, plan->tiles_k,
               nullptr, plan->d_flat, desc->scale};
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (desc->dtype == ARD_BF16) {
    ARD_HIP_CHECK(run_tdp<bf16>(TDP_BWD_WEIGHT, a, 0, plan->nnz, s));
  } else {
    ARD_HIP_CHECK(run_tdp<float>(TDP_BWD_WEIGHT, a, 0, plan->nnz, s));
  }
  if (desc->dropped == ARD_DROPPED_ZERO && plan->nnz < plan->tiles_n * plan->tiles_k) {
    hipLaunchKernelGGL(zero_dropped_tiles_kernel, dim3(plan->tiles_k, plan->tiles_n), dim3(256), 0, s,
                       plan->d_bits, dW, plan->k, plan->tile, plan->tiles_k);
    ARD_LAUNCH_CHECK();
  }
  return ARD_OK;
}

}  // extern "C"
