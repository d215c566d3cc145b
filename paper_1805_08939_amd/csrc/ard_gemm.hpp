// Gathered GEMM on CDNA4 matrix cores (gfx950).
//
// Every GEMM of the hot path multiplies COMPACT matrices whose rows (and, for
// a weight matrix under two patterns, columns) are picked from a larger matrix
// by an ascending index list. Sec. III-A builds these compact matrices from the
// kept rows only; here they are never materialised in HBM: the loaders fetch
// kept rows straight from the full matrices into LDS, and the epilogue scatters
// the compact result back. Dropped rows are never read.
//
// C(m, n) = sum_k A(m, k) B(k, n) over compact extents M, N, K.
//
// An operand is a gathered view V(r, c) = base[ridx(r) * ld + cidx(c)]
// (ridx/cidx NULL = identity) read in one of four ways:
//   KC_VEC  : A(m,k) = V(m,k) / B(k,n) = V(n,k), contiguous in k, 16-byte loads
//   KC_ELEM : the same with a gathered or unaligned contiguous dimension
//   MC_VEC  : A(m,k) = V(k,m) / B(k,n) = V(k,n), contiguous in m (or n):
//             16-byte loads, transposed in registers on the way into LDS
//   MC_ELEM : the same with element loads
// LDS always holds [rows of the tile][k] so that each MFMA operand fragment is
// one 16-byte LDS read. A "gated" operand computes scale * dY * [Y > 0] (or
// scale * dY) on load, fusing the dropout/activation derivative of the
// backward pass (Sec. II-C: the derivative is masked by the forward mask).
//
// Matrix cores: bf16 uses v_mfma_f32_32x32x16_bf16 (8 k per lane); fp32 uses
// v_mfma_f32_32x32x2_f32 with each lane reading 4 consecutive k from LDS and
// issuing four MFMAs, so that both operands stay k-contiguous.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace ard {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

enum LoadMode { KC_VEC = 0, KC_ELEM = 1, MC_VEC = 2, MC_ELEM = 3 };
enum Epilogue { EPI_STORE = 0, EPI_FWD = 1 };

struct GemmOperand {
  const void* p;         // view base
  const void* y;         // gate source (forward output) for a gated operand, else NULL
  int64_t ld;            // row stride of the view, elements
  const int32_t* ridx;   // gather list of view rows, NULL = identity
  const int32_t* cidx;   // gather list of view columns, NULL = identity
  int64_t bstride;       // elements between batch entries (blockIdx.z)
  int32_t relu;          // gated operand: multiply by [Y > 0]
  float scale;           // gated operand: scale factor
  int64_t kbstride;      // elements between K batches (see GemmArgs::kbatch)
};

struct GemmOutput {
  void* p;
  int64_t ld;
  const int32_t* ridx;
  const int32_t* cidx;
  int64_t bstride;
  const float* bias;     // EPI_FWD: bias[ridx(m)], may be NULL
  int32_t relu;          // EPI_FWD: apply ReLU
  float scale;           // EPI_FWD: multiply after the activation (also the
                         // dropout scale of the backward passes)
};

// The contraction runs over kbatch x K: K batch kb reads both operands at
// base + kb * kbstride (a sum over time steps of an LSTM, say). kbatch 0 or 1
// is a plain GEMM.
struct GemmArgs {
  int32_t M, N, K;
  GemmOperand a, b;
  GemmOutput c;
  int32_t kbatch;
};

template <typename T>
struct TypeTraits;
template <>
struct TypeTraits<float> {
  static constexpr int VE = 4;   // elements per 16 bytes
  static constexpr int KP = 1;   // k values per 32-bit LDS word
};
template <>
struct TypeTraits<bf16> {
  static constexpr int VE = 8;
  static constexpr int KP = 2;
};

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16 x) { return static_cast<float>(x); }
template <typename T>
__device__ __forceinline__ T from_f32(float x);
template <>
__device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <>
__device__ __forceinline__ bf16 from_f32<bf16>(float x) { return static_cast<bf16>(x); }

__device__ __forceinline__ int64_t gather(const int32_t* idx, int64_t i) {
  return idx ? static_cast<int64_t>(idx[i]) : i;
}

// One element of an operand view, with the optional fused gate.
template <typename T, bool GATED>
__device__ __forceinline__ T load_elem(const GemmOperand& op, const T* base, const T* ybase,
                                       int64_t off) {
  if constexpr (!GATED) {
    return base[off];
  } else {
    float g = op.scale * to_f32(base[off]);
    if (op.relu && !(to_f32(ybase[off]) > 0.0f)) g = 0.0f;
    return from_f32<T>(g);
  }
}

// Sixteen bytes (VE elements) of an operand view, with the optional gate.
template <typename T, bool GATED>
__device__ __forceinline__ u32x4 load_vec(const GemmOperand& op, const T* base, const T* ybase,
                                          int64_t off) {
  u32x4 raw = *reinterpret_cast<const u32x4*>(base + off);
  if constexpr (!GATED) {
    return raw;
  } else {
    constexpr int VE = TypeTraits<T>::VE;
    u32x4 yr = raw;
    if (op.relu) yr = *reinterpret_cast<const u32x4*>(ybase + off);
    const T* xv = reinterpret_cast<const T*>(&raw);
    const T* yv = reinterpret_cast<const T*>(&yr);
    u32x4 out;
    T* ov = reinterpret_cast<T*>(&out);
#pragma unroll
    for (int e = 0; e < VE; ++e) {
      float g = op.scale * to_f32(xv[e]);
      if (op.relu && !(to_f32(yv[e]) > 0.0f)) g = 0.0f;
      ov[e] = from_f32<T>(g);
    }
    return out;
  }
}

// Loads the R x BK tile (tile rows r0.., compact k k0..) of an operand into LDS
// laid out [R][LDK] (k contiguous). rext / kext are the compact extents.
template <typename T, int MODE, bool GATED, int R, int BK, int LDK, int NT>
__device__ __forceinline__ void load_tile(const GemmOperand& op, const T* base, const T* ybase,
                                          T* lds, int r0, int k0, int rext, int kext) {
  constexpr int VE = TypeTraits<T>::VE;
  constexpr int KP = TypeTraits<T>::KP;
  const int tid = threadIdx.x;
  if constexpr (MODE == KC_VEC || MODE == KC_ELEM) {
    // view row = tile row, view column = k
    constexpr int CPR = BK / VE;  // 16-byte chunks per tile row
    constexpr int CHUNKS = R * CPR;
#pragma unroll
    for (int c = tid; c < CHUNKS; c += NT) {
      const int r = c / CPR;
      const int kc = (c % CPR) * VE;
      const int gr = r0 + r, gk = k0 + kc;
      u32x4 v = {0u, 0u, 0u, 0u};
      if (gr < rext) {
        const int64_t rowoff = gather(op.ridx, gr) * op.ld;
        if (MODE == KC_VEC && gk + VE <= kext) {
          v = load_vec<T, GATED>(op, base, ybase, rowoff + gk);
        } else {
          T* vv = reinterpret_cast<T*>(&v);
#pragma unroll
          for (int e = 0; e < VE; ++e)
            if (gk + e < kext) vv[e] = load_elem<T, GATED>(op, base, ybase, rowoff + gather(op.cidx, gk + e));
        }
      }
      *reinterpret_cast<u32x4*>(lds + r * LDK + kc) = v;
    }
  } else if constexpr (MODE == MC_VEC) {
    // view row = k, view column = tile row; KP k-rows x VE columns per unit,
    // transposed into VE 32-bit LDS words. k runs fastest across threads so
    // that one wave's LDS writes of a column land in distinct banks.
    constexpr int KU = BK / KP;     // k units per column chunk
    constexpr int CC = R / VE;      // column chunks
    constexpr int UNITS = KU * CC;
#pragma unroll
    for (int u = tid; u < UNITS; u += NT) {
      const int kp = (u % KU) * KP;
      const int rc = (u / KU) * VE;
      const int gk = k0 + kp, gr = r0 + rc;
      u32x4 rows[KP];
#pragma unroll
      for (int q = 0; q < KP; ++q) {
        rows[q] = u32x4{0u, 0u, 0u, 0u};
        if (gk + q < kext) {
          const int64_t rowoff = gather(op.ridx, gk + q) * op.ld;
          if (gr + VE <= rext) {
            rows[q] = load_vec<T, GATED>(op, base, ybase, rowoff + gr);
          } else {
            T* vv = reinterpret_cast<T*>(&rows[q]);
#pragma unroll
            for (int e = 0; e < VE; ++e)
              if (gr + e < rext) vv[e] = load_elem<T, GATED>(op, base, ybase, rowoff + gr + e);
          }
        }
      }
#pragma unroll
      for (int e = 0; e < VE; ++e) {
        uint32_t word;
        if constexpr (KP == 1) {
          word = rows[0][e];
        } else {
          const uint16_t* r0p = reinterpret_cast<const uint16_t*>(&rows[0]);
          const uint16_t* r1p = reinterpret_cast<const uint16_t*>(&rows[1]);
          word = static_cast<uint32_t>(r0p[e]) | (static_cast<uint32_t>(r1p[e]) << 16);
        }
        *reinterpret_cast<uint32_t*>(lds + (rc + e) * LDK + kp) = word;
      }
    }
  } else {  // MC_ELEM: each thread gathers VE consecutive k of one tile row
    constexpr int CPR = BK / VE;
    constexpr int CHUNKS = R * CPR;
#pragma unroll
    for (int c = tid; c < CHUNKS; c += NT) {
      const int r = c % R;
      const int kc = (c / R) * VE;
      const int gr = r0 + r, gk = k0 + kc;
      u32x4 v = {0u, 0u, 0u, 0u};
      if (gr < rext) {
        const int64_t coloff = gather(op.cidx, gr);
        T* vv = reinterpret_cast<T*>(&v);
#pragma unroll
        for (int e = 0; e < VE; ++e)
          if (gk + e < kext)
            vv[e] = load_elem<T, GATED>(op, base, ybase, gather(op.ridx, gk + e) * op.ld + coloff);
      }
      *reinterpret_cast<u32x4*>(lds + r * LDK + kc) = v;
    }
  }
}

template <int BM_, int BN_, int BK_, int WGM_, int WGN_>
struct TileCfg {
  static constexpr int BM = BM_, BN = BN_, BK = BK_, WGM = WGM_, WGN = WGN_;
  static constexpr int NT = 64 * WGM * WGN;
  static constexpr int TM = BM / WGM, TN = BN / WGN;  // wave tile
  static constexpr int FM = TM / 32, FN = TN / 32;    // 32x32 MFMA blocks per wave
};

// MFMA over one BK slab held in LDS.
template <typename T, class Cfg, int LDK>
__device__ __forceinline__ void mma_slab(const T* As, const T* Bs, f32x16 (&acc)[Cfg::FM][Cfg::FN],
                                         int wm, int wn) {
  const int lane = threadIdx.x & 63;
  const int lr = lane & 31, lh = lane >> 5;
  if constexpr (sizeof(T) == 2) {
#pragma unroll
    for (int kk = 0; kk < Cfg::BK; kk += 16) {
      bf16x8 a[Cfg::FM], b[Cfg::FN];
#pragma unroll
      for (int i = 0; i < Cfg::FM; ++i)
        a[i] = *reinterpret_cast<const bf16x8*>(As + (wm * Cfg::TM + 32 * i + lr) * LDK + kk + 8 * lh);
#pragma unroll
      for (int j = 0; j < Cfg::FN; ++j)
        b[j] = *reinterpret_cast<const bf16x8*>(Bs + (wn * Cfg::TN + 32 * j + lr) * LDK + kk + 8 * lh);
#pragma unroll
      for (int i = 0; i < Cfg::FM; ++i)
#pragma unroll
        for (int j = 0; j < Cfg::FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
  } else {
#pragma unroll
    for (int kk = 0; kk < Cfg::BK; kk += 8) {
      f32x4 a[Cfg::FM], b[Cfg::FN];
#pragma unroll
      for (int i = 0; i < Cfg::FM; ++i)
        a[i] = *reinterpret_cast<const f32x4*>(As + (wm * Cfg::TM + 32 * i + lr) * LDK + kk + 4 * lh);
#pragma unroll
      for (int j = 0; j < Cfg::FN; ++j)
        b[j] = *reinterpret_cast<const f32x4*>(Bs + (wn * Cfg::TN + 32 * j + lr) * LDK + kk + 4 * lh);
#pragma unroll
      for (int e = 0; e < 4; ++e)
#pragma unroll
        for (int i = 0; i < Cfg::FM; ++i)
#pragma unroll
          for (int j = 0; j < Cfg::FN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[i][e], b[j][e], acc[i][j], 0, 0, 0);
    }
  }
}

// Writes the accumulators through the epilogue. Output element (m, n) goes to
// c.p[ridx(m) * ld + cidx(n)] of the batch entry.
template <typename OutT, class Cfg, int EPI>
__device__ __forceinline__ void store_tile(const GemmArgs& g, f32x16 (&acc)[Cfg::FM][Cfg::FN],
                                           int m0, int n0, int wm, int wn, int64_t bz) {
  const int lane = threadIdx.x & 63;
  const int lr = lane & 31, lh = lane >> 5;
  OutT* out = static_cast<OutT*>(g.c.p) + bz * g.c.bstride;
#pragma unroll
  for (int i = 0; i < Cfg::FM; ++i) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int m = m0 + wm * Cfg::TM + 32 * i + 8 * (r >> 2) + 4 * lh + (r & 3);
      if (m >= g.M) continue;
      const int64_t orow = gather(g.c.ridx, m);
      float bias = 0.0f;
      if constexpr (EPI == EPI_FWD) {
        if (g.c.bias) bias = g.c.bias[orow];
      }
#pragma unroll
      for (int j = 0; j < Cfg::FN; ++j) {
        const int n = n0 + wn * Cfg::TN + 32 * j + lr;
        if (n >= g.N) continue;
        float v = acc[i][j][r];
        if constexpr (EPI == EPI_FWD) {
          v += bias;
          if (g.c.relu) v = v > 0.0f ? v : 0.0f;
          v *= g.c.scale;
        }
        out[orow * g.c.ld + gather(g.c.cidx, n)] = from_f32<OutT>(v);
      }
    }
  }
}

template <typename T, typename OutT, class Cfg, int AMODE, int BMODE, bool AGATE, bool BGATE, int EPI>
__global__ void __launch_bounds__(Cfg::NT) gemm_kernel(GemmArgs g) {
  constexpr int LDK = Cfg::BK + 16 / sizeof(T);
  __shared__ __attribute__((aligned(16))) T As[Cfg::BM * LDK];
  __shared__ __attribute__((aligned(16))) T Bs[Cfg::BN * LDK];

  const int n0 = blockIdx.x * Cfg::BN;
  const int m0 = blockIdx.y * Cfg::BM;
  const int64_t bz = blockIdx.z;
  const int wave = threadIdx.x >> 6;
  const int wm = wave / Cfg::WGN, wn = wave % Cfg::WGN;

  const T* abase = static_cast<const T*>(g.a.p) + bz * g.a.bstride;
  const T* aybase = AGATE ? static_cast<const T*>(g.a.y) + bz * g.a.bstride : nullptr;
  const T* bbase = static_cast<const T*>(g.b.p) + bz * g.b.bstride;
  const T* bybase = BGATE ? static_cast<const T*>(g.b.y) + bz * g.b.bstride : nullptr;

  f32x16 acc[Cfg::FM][Cfg::FN];
#pragma unroll
  for (int i = 0; i < Cfg::FM; ++i)
#pragma unroll
    for (int j = 0; j < Cfg::FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  const int kbatch = g.kbatch > 0 ? g.kbatch : 1;
  for (int kb = 0; kb < kbatch; ++kb) {
    const T* ab = abase + kb * g.a.kbstride;
    const T* aby = AGATE ? aybase + kb * g.a.kbstride : nullptr;
    const T* bb = bbase + kb * g.b.kbstride;
    const T* bby = BGATE ? bybase + kb * g.b.kbstride : nullptr;
    for (int k0 = 0; k0 < g.K; k0 += Cfg::BK) {
      load_tile<T, AMODE, AGATE, Cfg::BM, Cfg::BK, LDK, Cfg::NT>(g.a, ab, aby, As, m0, k0, g.M, g.K);
      load_tile<T, BMODE, BGATE, Cfg::BN, Cfg::BK, LDK, Cfg::NT>(g.b, bb, bby, Bs, n0, k0, g.N, g.K);
      __syncthreads();
      mma_slab<T, Cfg, LDK>(As, Bs, acc, wm, wn);
      __syncthreads();
    }
  }
  store_tile<OutT, Cfg, EPI>(g, acc, m0, n0, wm, wn, bz);
}

// Host-side launch of one instantiation over an (N/BN, M/BM, batch) grid.
template <typename T, typename OutT, class Cfg, int AMODE, int BMODE, bool AGATE, bool BGATE, int EPI>
inline hipError_t launch_gemm(const GemmArgs& g, int batch, hipStream_t stream) {
  dim3 grid((g.N + Cfg::BN - 1) / Cfg::BN, (g.M + Cfg::BM - 1) / Cfg::BM, batch);
  hipLaunchKernelGGL((gemm_kernel<T, OutT, Cfg, AMODE, BMODE, AGATE, BGATE, EPI>), grid,
                     dim3(Cfg::NT), 0, stream, g);
  return hipGetLastError();
}

// Launches the instantiation matching whether each operand can use 16-byte
// vector loads (A0/B0) or needs element loads (A1/B1).
template <typename T, typename OutT, class Cfg, int A0, int A1, int B0, int B1, bool AGATE,
          bool BGATE, int EPI>
inline hipError_t dispatch_gemm(const GemmArgs& g, int batch, bool a_vec, bool b_vec,
                                hipStream_t stream) {
  if (a_vec) {
    if (b_vec) return launch_gemm<T, OutT, Cfg, A0, B0, AGATE, BGATE, EPI>(g, batch, stream);
    return launch_gemm<T, OutT, Cfg, A0, B1, AGATE, BGATE, EPI>(g, batch, stream);
  }
  if (b_vec) return launch_gemm<T, OutT, Cfg, A1, B0, AGATE, BGATE, EPI>(g, batch, stream);
  return launch_gemm<T, OutT, Cfg, A1, B1, AGATE, BGATE, EPI>(g, batch, stream);
}

// Tile shapes: 128x128 output tiles for large problems, 64x64 when the large
// tiles would leave most of the 256 compute units idle.
template <typename T>
struct GemmCfgs;
template <>
struct GemmCfgs<bf16> {
  using Big = TileCfg<128, 128, 32, 2, 2>;
  using Small = TileCfg<64, 64, 32, 2, 2>;
};
template <>
struct GemmCfgs<float> {
  using Big = TileCfg<128, 128, 16, 2, 2>;
  using Small = TileCfg<64, 64, 16, 2, 2>;
};

inline bool use_big_tiles(int M, int N, int batch) {
  const int64_t big = static_cast<int64_t>((M + 127) / 128) * ((N + 127) / 128) * batch;
  return big >= 160;
}

template <typename T, typename OutT, int A0, int A1, int B0, int B1, bool AGATE, bool BGATE, int EPI>
inline hipError_t run_gemm(const GemmArgs& g, int batch, bool a_vec, bool b_vec,
                           hipStream_t stream) {
  if (g.M <= 0 || g.N <= 0 || batch <= 0) return hipSuccess;
  if (use_big_tiles(g.M, g.N, batch))
    return dispatch_gemm<T, OutT, typename GemmCfgs<T>::Big, A0, A1, B0, B1, AGATE, BGATE, EPI>(
        g, batch, a_vec, b_vec, stream);
  return dispatch_gemm<T, OutT, typename GemmCfgs<T>::Small, A0, A1, B0, B1, AGATE, BGATE, EPI>(
      g, batch, a_vec, b_vec, stream);
}

}  // namespace ard
