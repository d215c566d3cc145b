// Gathered GEMM on CDNA4 matrix cores (gfx950).
//
// Every GEMM of the hot path multiplies COMPACT matrices whose rows are picked
// from a larger matrix by an ascending index list. Sec. III-A builds these
// compact matrices from the kept rows only; here the row gathers happen in the
// loaders, which fetch kept rows straight from the full matrices into LDS, and
// in the epilogue, which scatters the compact result back. Dropped rows are
// never read or written.
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
// one 16-byte LDS read. A "gated" operand multiplies by [Y > 0] on load: the
// activation derivative of the backward pass (Sec. II-C: the derivative is
// masked by the forward mask), exact in any dtype because the gate is 0/1.
//
// Main loop: each thread loads its share of the next K slab into registers
// while the waves run MFMA on the current slab from LDS; LDS is double
// buffered, so one barrier per slab suffices. Small output grids split the
// contraction over workgroups (grid z); each split writes fp32 partial tiles
// to a workspace and a second kernel sums them in fixed order (deterministic)
// and applies the epilogue.
//
// Matrix cores: bf16 uses v_mfma_f32_32x32x16_bf16 (8 k per lane); fp32 uses
// v_mfma_f32_32x32x2_f32 with each lane reading 4 consecutive k from LDS and
// issuing four MFMAs, so that both operands stay k-contiguous in LDS.
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
  float scale;           // unused by the loaders (kept for layout stability)
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
  const void* gate;      // EPI_FWD: if set, multiply by [gate > 0] at the output
                         // position (the ReLU derivative of the layer below)
  int64_t col_stride;    // elements between consecutive output columns when cidx is NULL (0 = 1)
  int64_t bias_stride;   // elements between the bias entries of consecutive rows when ridx is NULL (0 = 1)
};

// Output column offset of compact column n, and bias index of compact row m.
__device__ __forceinline__ int64_t out_col(const GemmOutput& c, int64_t n) {
  return c.cidx ? static_cast<int64_t>(c.cidx[n]) : n * (c.col_stride > 1 ? c.col_stride : 1);
}
__device__ __forceinline__ int64_t bias_row(const GemmOutput& c, int64_t m) {
  return c.ridx ? static_cast<int64_t>(c.ridx[m]) : m * (c.bias_stride > 1 ? c.bias_stride : 1);
}

// The contraction runs over kbatch x K: K batch kb reads both operands at
// base + kb * kbstride (a sum over time steps of an LSTM, say). kbatch 0 or 1
// is a plain GEMM. splits > 1 divides the kbatch x ceil(K / BK) slabs over
// that many workgroups per output tile; `partial` then receives
// [batch][splits][M][N] fp32 sums for the reduction kernel.
// rsum, when set (fast kernel with a k-contiguous A and no split only), also
// receives c.scale times the sum of row m of A over the whole contraction at
// rsum[bz * rsum_bstride + m * rsum_ld]: a bias gradient taken from the A
// operand of the weight-gradient product that reads it anyway.
struct GemmArgs {
  int32_t M, N, K;
  GemmOperand a, b;
  GemmOutput c;
  int32_t kbatch;
  int32_t splits;
  float* partial;
  float* rsum;
  int64_t rsum_ld, rsum_bstride;
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
    T v = base[off];
    if (op.relu && !(to_f32(ybase[off]) > 0.0f)) v = from_f32<T>(0.0f);
    return v;
  }
}

// Sixteen bytes (VE elements) of an operand view, with the optional gate.
template <typename T, bool GATED>
__device__ __forceinline__ u32x4 load_vec(const GemmOperand& op, const T* base, const T* ybase,
                                          int64_t off) {
  u32x4 raw = *reinterpret_cast<const u32x4*>(base + off);
  if constexpr (GATED) {
    if (op.relu) {
      constexpr int VE = TypeTraits<T>::VE;
      const u32x4 yr = *reinterpret_cast<const u32x4*>(ybase + off);
      T* xv = reinterpret_cast<T*>(&raw);
      const T* yv = reinterpret_cast<const T*>(&yr);
#pragma unroll
      for (int e = 0; e < VE; ++e)
        if (!(to_f32(yv[e]) > 0.0f)) xv[e] = from_f32<T>(0.0f);
    }
  }
  return raw;
}

// Per-thread share of one R x BK operand tile: global -> registers (load)
// and registers -> LDS [R][LDK] (store). rext / kext are the compact extents;
// out-of-range elements are zero.
template <typename T, int MODE, bool GATED, int R, int BK, int LDK, int NT>
struct TileLoader {
  static constexpr int VE = TypeTraits<T>::VE;
  static constexpr int KP = TypeTraits<T>::KP;
  static constexpr bool MCV = MODE == MC_VEC;
  // KC_* and MC_ELEM: one 16-byte vector per unit; MC_VEC: KP vectors per unit
  static constexpr int UNITS = MCV ? (BK / KP) * (R / VE) : R * (BK / VE);
  static constexpr int PER = (UNITS + NT - 1) / NT;
  static constexpr int RPU = MCV ? KP : 1;
  u32x4 v[PER * RPU];

  __device__ __forceinline__ void load(const GemmOperand& op, const T* base, const T* ybase, int r0,
                                       int k0, int rext, int kext) {
    const int tid = threadIdx.x;
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int u = tid + p * NT;
#pragma unroll
      for (int q = 0; q < RPU; ++q) v[p * RPU + q] = u32x4{0u, 0u, 0u, 0u};
      if (UNITS % NT != 0 && u >= UNITS) continue;
      if constexpr (MODE == KC_VEC || MODE == KC_ELEM) {
        constexpr int CPR = BK / VE;
        const int r = u / CPR, kc = (u % CPR) * VE;
        const int gr = r0 + r, gk = k0 + kc;
        if (gr < rext) {
          const int64_t rowoff = gather(op.ridx, gr) * op.ld;
          if (MODE == KC_VEC && gk + VE <= kext) {
            v[p] = load_vec<T, GATED>(op, base, ybase, rowoff + gk);
          } else {
            T* vv = reinterpret_cast<T*>(&v[p]);
#pragma unroll
            for (int e = 0; e < VE; ++e)
              if (gk + e < kext) vv[e] = load_elem<T, GATED>(op, base, ybase, rowoff + gather(op.cidx, gk + e));
          }
        }
      } else if constexpr (MODE == MC_VEC) {
        // k runs fastest across threads so that the transposed 32-bit LDS
        // writes of one wave land in distinct banks
        constexpr int KU = BK / KP;
        const int kp = (u % KU) * KP, rc = (u / KU) * VE;
        const int gk = k0 + kp, gr = r0 + rc;
#pragma unroll
        for (int q = 0; q < KP; ++q) {
          if (gk + q < kext) {
            const int64_t rowoff = gather(op.ridx, gk + q) * op.ld;
            if (gr + VE <= rext) {
              v[p * KP + q] = load_vec<T, GATED>(op, base, ybase, rowoff + gr);
            } else {
              T* vv = reinterpret_cast<T*>(&v[p * KP + q]);
#pragma unroll
              for (int e = 0; e < VE; ++e)
                if (gr + e < rext) vv[e] = load_elem<T, GATED>(op, base, ybase, rowoff + gr + e);
            }
          }
        }
      } else {  // MC_ELEM: VE consecutive k of one tile row
        const int r = u % R, kc = (u / R) * VE;
        const int gr = r0 + r, gk = k0 + kc;
        if (gr < rext) {
          const int64_t coloff = gather(op.cidx, gr);
          T* vv = reinterpret_cast<T*>(&v[p]);
#pragma unroll
          for (int e = 0; e < VE; ++e)
            if (gk + e < kext) vv[e] = load_elem<T, GATED>(op, base, ybase, gather(op.ridx, gk + e) * op.ld + coloff);
        }
      }
    }
  }

  __device__ __forceinline__ void store(T* lds) const {
    const int tid = threadIdx.x;
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int u = tid + p * NT;
      if (UNITS % NT != 0 && u >= UNITS) continue;
      if constexpr (MODE == KC_VEC || MODE == KC_ELEM) {
        constexpr int CPR = BK / VE;
        *reinterpret_cast<u32x4*>(lds + (u / CPR) * LDK + (u % CPR) * VE) = v[p];
      } else if constexpr (MODE == MC_VEC) {
        constexpr int KU = BK / KP;
        const int kp = (u % KU) * KP, rc = (u / KU) * VE;
#pragma unroll
        for (int e = 0; e < VE; ++e) {
          uint32_t word;
          if constexpr (KP == 1) {
            word = v[p][e];
          } else {
            const uint16_t* a = reinterpret_cast<const uint16_t*>(&v[p * KP]);
            const uint16_t* b = reinterpret_cast<const uint16_t*>(&v[p * KP + 1]);
            word = static_cast<uint32_t>(a[e]) | (static_cast<uint32_t>(b[e]) << 16);
          }
          *reinterpret_cast<uint32_t*>(lds + (rc + e) * LDK + kp) = word;
        }
      } else {
        *reinterpret_cast<u32x4*>(lds + (u % R) * LDK + (u / R) * VE) = v[p];
      }
    }
  }
};

// One-shot load of a tile into LDS (load then store).
template <typename T, int MODE, bool GATED, int R, int BK, int LDK, int NT>
__device__ __forceinline__ void load_tile(const GemmOperand& op, const T* base, const T* ybase, T* lds,
                                          int r0, int k0, int rext, int kext) {
  TileLoader<T, MODE, GATED, R, BK, LDK, NT> t;
  t.load(op, base, ybase, r0, k0, rext, kext);
  t.store(lds);
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

// Applies the epilogue to one accumulator value of compact element (m, n).
template <int EPI>
__device__ __forceinline__ float epilogue(const GemmOutput& c, float v, float bias) {
  if constexpr (EPI == EPI_FWD) {
    v += bias;
    if (c.relu) v = v > 0.0f ? v : 0.0f;
    v *= c.scale;
  }
  return v;
}

// Writes the accumulators through the epilogue (splits == 1) or as raw fp32
// partial sums (splits > 1). Output element (m, n) goes to
// c.p[ridx(m) * ld + cidx(n)] of the batch entry.
template <typename OutT, class Cfg, int EPI>
__device__ __forceinline__ void store_tile(const GemmArgs& g, f32x16 (&acc)[Cfg::FM][Cfg::FN],
                                           int m0, int n0, int wm, int wn, int64_t bz, int split) {
  const int lane = threadIdx.x & 63;
  const int lr = lane & 31, lh = lane >> 5;
  if (g.splits > 1) {
    float* part = g.partial + (bz * g.splits + split) * static_cast<int64_t>(g.M) * g.N;
#pragma unroll
    for (int i = 0; i < Cfg::FM; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int m = m0 + wm * Cfg::TM + 32 * i + 8 * (r >> 2) + 4 * lh + (r & 3);
        if (m >= g.M) continue;
#pragma unroll
        for (int j = 0; j < Cfg::FN; ++j) {
          const int n = n0 + wn * Cfg::TN + 32 * j + lr;
          if (n < g.N) part[static_cast<int64_t>(m) * g.N + n] = acc[i][j][r];
        }
      }
    return;
  }
  OutT* out = static_cast<OutT*>(g.c.p) + bz * g.c.bstride;
#pragma unroll
  for (int i = 0; i < Cfg::FM; ++i) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int m = m0 + wm * Cfg::TM + 32 * i + 8 * (r >> 2) + 4 * lh + (r & 3);
      if (m >= g.M) continue;
      const int64_t orow = gather(g.c.ridx, m);
      const float bias = (EPI == EPI_FWD && g.c.bias) ? g.c.bias[bias_row(g.c, m)] : 0.0f;
#pragma unroll
      for (int j = 0; j < Cfg::FN; ++j) {
        const int n = n0 + wn * Cfg::TN + 32 * j + lr;
        if (n >= g.N) continue;
        const int64_t o = orow * g.c.ld + out_col(g.c, n);
        float v = epilogue<EPI>(g.c, acc[i][j][r], bias);
        if (EPI == EPI_FWD && g.c.gate && !(to_f32(static_cast<const OutT*>(g.c.gate)[bz * g.c.bstride + o]) > 0.0f))
          v = 0.0f;
        out[o] = from_f32<OutT>(v);
      }
    }
  }
}

template <typename T, typename OutT, class Cfg, int AMODE, int BMODE, bool AGATE, bool BGATE, int EPI>
__global__ void __launch_bounds__(Cfg::NT) gemm_kernel(GemmArgs g) {
  constexpr int LDK = Cfg::BK + 16 / sizeof(T);
  __shared__ __attribute__((aligned(16))) T As[2][Cfg::BM * LDK];
  __shared__ __attribute__((aligned(16))) T Bs[2][Cfg::BN * LDK];

  const int n0 = blockIdx.x * Cfg::BN;
  const int m0 = blockIdx.y * Cfg::BM;
  const int splits = g.splits > 1 ? g.splits : 1;
  const int64_t bz = blockIdx.z / splits;
  const int split = blockIdx.z % splits;
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

  // slabs q = kb * nks + ks over the kbatch x ceil(K / BK) contraction
  const int nks = (g.K + Cfg::BK - 1) / Cfg::BK;
  const int kbatch = g.kbatch > 0 ? g.kbatch : 1;
  const int nslab = kbatch * nks;
  const int q0 = static_cast<int>((static_cast<int64_t>(nslab) * split) / splits);
  const int q1 = static_cast<int>((static_cast<int64_t>(nslab) * (split + 1)) / splits);

  TileLoader<T, AMODE, AGATE, Cfg::BM, Cfg::BK, LDK, Cfg::NT> la;
  TileLoader<T, BMODE, BGATE, Cfg::BN, Cfg::BK, LDK, Cfg::NT> lb;
  auto load = [&](int q) {
    const int kb = q / nks, k0 = (q % nks) * Cfg::BK;
    la.load(g.a, abase + kb * g.a.kbstride, AGATE ? aybase + kb * g.a.kbstride : nullptr, m0, k0, g.M, g.K);
    lb.load(g.b, bbase + kb * g.b.kbstride, BGATE ? bybase + kb * g.b.kbstride : nullptr, n0, k0, g.N, g.K);
  };

  if (q0 < q1) {
    load(q0);
    la.store(As[0]);
    lb.store(Bs[0]);
  }
  __syncthreads();
  for (int q = q0; q < q1; ++q) {
    const int cur = (q - q0) & 1;
    const bool more = q + 1 < q1;
    if (more) load(q + 1);
    mma_slab<T, Cfg, LDK>(As[cur], Bs[cur], acc, wm, wn);
    if (more) {
      la.store(As[cur ^ 1]);
      lb.store(Bs[cur ^ 1]);
    }
    __syncthreads();
  }
  store_tile<OutT, Cfg, EPI>(g, acc, m0, n0, wm, wn, bz, split);
}

// The same for 4 consecutive elements of one output row per thread (N a
// multiple of 4, output columns contiguous, output, gate and partial rows 4-
// element aligned): 16-byte partial loads, 32-bit index arithmetic (M N <
// 2^31), one vector store.
template <typename OutT, int EPI>
__global__ void __launch_bounds__(256) splitk_reduce4_kernel(GemmArgs g) {
  const int32_t mn = g.M * g.N;
  const int32_t e = (static_cast<int32_t>(blockIdx.x) * 256 + static_cast<int32_t>(threadIdx.x)) * 4;
  if (e >= mn) return;
  const int64_t bz = blockIdx.y;
  const float* part = g.partial + bz * g.splits * static_cast<int64_t>(mn) + e;
  // partials loaded eight at a time, then added in split order: the loads of a
  // group are in flight together instead of one round trip per split
  f32x4 v = {0.0f, 0.0f, 0.0f, 0.0f};
  int s = 0;
  for (; s + 8 <= g.splits; s += 8) {
    f32x4 t[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) t[u] = *reinterpret_cast<const f32x4*>(part + static_cast<int64_t>(s + u) * mn);
#pragma unroll
    for (int u = 0; u < 8; ++u) v += t[u];
  }
  for (; s < g.splits; ++s) v += *reinterpret_cast<const f32x4*>(part + static_cast<int64_t>(s) * mn);
  const int32_t m = e / g.N, n = e - m * g.N;
  const float bias = (EPI == EPI_FWD && g.c.bias) ? g.c.bias[bias_row(g.c, m)] : 0.0f;
  const int64_t o = bz * g.c.bstride + static_cast<int64_t>(m) * g.c.ld + n;
  OutT w[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float x = epilogue<EPI>(g.c, v[i], bias);
    if (EPI == EPI_FWD && g.c.gate && !(to_f32(static_cast<const OutT*>(g.c.gate)[o + i]) > 0.0f)) x = 0.0f;
    w[i] = from_f32<OutT>(x);
  }
  OutT* out = static_cast<OutT*>(g.c.p) + o;
  if constexpr (sizeof(OutT) == 2)
    *reinterpret_cast<uint2*>(out) = *reinterpret_cast<const uint2*>(w);
  else
    *reinterpret_cast<f32x4*>(out) = *reinterpret_cast<const f32x4*>(w);
}

// Whether splitk_reduce4_kernel can finish a problem.
template <typename OutT>
inline bool reduce4_ok(const GemmArgs& g) {
  const int64_t mn = static_cast<int64_t>(g.M) * g.N;
  return mn < (int64_t{1} << 31) && g.N % 4 == 0 && g.c.ridx == nullptr && g.c.cidx == nullptr &&
         g.c.col_stride <= 1 && g.c.ld % 4 == 0 && g.c.bstride % 4 == 0 &&
         (reinterpret_cast<uintptr_t>(g.c.p) % (4 * sizeof(OutT))) == 0 &&
         (reinterpret_cast<uintptr_t>(g.c.gate) % (4 * sizeof(OutT))) == 0 &&
         (reinterpret_cast<uintptr_t>(g.partial) % 16) == 0;
}

// Sums the split partials of every compact element in fixed split order and
// applies the epilogue.
template <typename OutT, int EPI>
__global__ void __launch_bounds__(256) splitk_reduce_kernel(GemmArgs g) {
  const int64_t mn = static_cast<int64_t>(g.M) * g.N;
  const int64_t e = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (e >= mn) return;
  const int64_t bz = blockIdx.y;
  const float* part = g.partial + bz * g.splits * mn + e;
  float v = 0.0f;
  int s = 0;
  for (; s + 8 <= g.splits; s += 8) {  // eight loads in flight, added in split order
    float t[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) t[u] = part[(s + u) * mn];
#pragma unroll
    for (int u = 0; u < 8; ++u) v += t[u];
  }
  for (; s < g.splits; ++s) v += part[s * mn];
  const int64_t m = e / g.N, n = e % g.N;
  const int64_t orow = gather(g.c.ridx, m);
  const float bias = (EPI == EPI_FWD && g.c.bias) ? g.c.bias[bias_row(g.c, m)] : 0.0f;
  OutT* out = static_cast<OutT*>(g.c.p) + bz * g.c.bstride;
  const int64_t o = orow * g.c.ld + out_col(g.c, n);
  v = epilogue<EPI>(g.c, v, bias);
  if (EPI == EPI_FWD && g.c.gate && !(to_f32(static_cast<const OutT*>(g.c.gate)[bz * g.c.bstride + o]) > 0.0f))
    v = 0.0f;
  out[o] = from_f32<OutT>(v);
}

// Small output grids: one 32 x 32 output block per workgroup; the four waves
// take disjoint quarters of every K slab and reduce through LDS, which fills
// the chip without a second (reduction) launch when M x N is small.
template <typename T>
struct SmallCfg {
  static constexpr int BK = sizeof(T) == 2 ? 128 : 64;
  static constexpr int LDK = BK + 16 / sizeof(T);
  static constexpr int QK = BK / 4;  // k per wave per slab
};

template <typename T, typename OutT, int AMODE, int BMODE, bool AGATE, bool BGATE, int EPI>
__global__ void __launch_bounds__(256) gemm_small_kernel(GemmArgs g) {
  using C = SmallCfg<T>;
  __shared__ __attribute__((aligned(16))) T As[2][32 * C::LDK];
  __shared__ __attribute__((aligned(16))) T Bs[2][32 * C::LDK];
  __shared__ float red[4 * 16 * 64];
  const int n0 = blockIdx.x * 32, m0 = blockIdx.y * 32;
  const int splits = g.splits > 1 ? g.splits : 1;
  const int64_t bz = blockIdx.z / splits;
  const int split = blockIdx.z % splits;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int lr = lane & 31, lh = lane >> 5;

  const T* abase = static_cast<const T*>(g.a.p) + bz * g.a.bstride;
  const T* aybase = AGATE ? static_cast<const T*>(g.a.y) + bz * g.a.bstride : nullptr;
  const T* bbase = static_cast<const T*>(g.b.p) + bz * g.b.bstride;
  const T* bybase = BGATE ? static_cast<const T*>(g.b.y) + bz * g.b.bstride : nullptr;

  f32x16 acc;
#pragma unroll
  for (int r = 0; r < 16; ++r) acc[r] = 0.0f;

  const int nks = (g.K + C::BK - 1) / C::BK;
  const int kbatch = g.kbatch > 0 ? g.kbatch : 1;
  const int nslab = kbatch * nks;
  const int q0 = static_cast<int>((static_cast<int64_t>(nslab) * split) / splits);
  const int q1 = static_cast<int>((static_cast<int64_t>(nslab) * (split + 1)) / splits);

  TileLoader<T, AMODE, AGATE, 32, C::BK, C::LDK, 256> la;
  TileLoader<T, BMODE, BGATE, 32, C::BK, C::LDK, 256> lb;
  auto load = [&](int q) {
    const int kb = q / nks, k0 = (q % nks) * C::BK;
    la.load(g.a, abase + kb * g.a.kbstride, AGATE ? aybase + kb * g.a.kbstride : nullptr, m0, k0, g.M, g.K);
    lb.load(g.b, bbase + kb * g.b.kbstride, BGATE ? bybase + kb * g.b.kbstride : nullptr, n0, k0, g.N, g.K);
  };
  if (q0 < q1) {
    load(q0);
    la.store(As[0]);
    lb.store(Bs[0]);
  }
  __syncthreads();
  for (int q = q0; q < q1; ++q) {
    const int cur = (q - q0) & 1;
    const bool more = q + 1 < q1;
    if (more) load(q + 1);
    const T* as = As[cur] + lr * C::LDK + w * C::QK;
    const T* bs = Bs[cur] + lr * C::LDK + w * C::QK;
    if constexpr (sizeof(T) == 2) {
#pragma unroll
      for (int kk = 0; kk < C::QK; kk += 16) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(as + kk + 8 * lh);
        const bf16x8 b = *reinterpret_cast<const bf16x8*>(bs + kk + 8 * lh);
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc, 0, 0, 0);
      }
    } else {
#pragma unroll
      for (int kk = 0; kk < C::QK; kk += 8) {
        const f32x4 a = *reinterpret_cast<const f32x4*>(as + kk + 4 * lh);
        const f32x4 b = *reinterpret_cast<const f32x4*>(bs + kk + 4 * lh);
#pragma unroll
        for (int e = 0; e < 4; ++e) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a[e], b[e], acc, 0, 0, 0);
      }
    }
    if (more) {
      la.store(As[cur ^ 1]);
      lb.store(Bs[cur ^ 1]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int r = 0; r < 16; ++r) red[(w * 16 + r) * 64 + lane] = acc[r];
  __syncthreads();
  // wave w finishes accumulator registers 4w..4w+3: rows 8w + 4*lh + q, column lr
  const int n = n0 + lr;
  if (n >= g.N) return;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int m = m0 + 8 * w + 4 * lh + q;
    if (m >= g.M) continue;
    float v = 0.0f;
#pragma unroll
    for (int u = 0; u < 4; ++u) v += red[(u * 16 + 4 * w + q) * 64 + lane];
    if (splits > 1) {
      g.partial[(bz * splits + split) * static_cast<int64_t>(g.M) * g.N + static_cast<int64_t>(m) * g.N + n] = v;
      continue;
    }
    const int64_t orow = gather(g.c.ridx, m);
    const float bias = (EPI == EPI_FWD && g.c.bias) ? g.c.bias[bias_row(g.c, m)] : 0.0f;
    const int64_t o = orow * g.c.ld + out_col(g.c, n);
    v = epilogue<EPI>(g.c, v, bias);
    if (EPI == EPI_FWD && g.c.gate && !(to_f32(static_cast<const OutT*>(g.c.gate)[bz * g.c.bstride + o]) > 0.0f))
      v = 0.0f;
    (static_cast<OutT*>(g.c.p) + bz * g.c.bstride)[o] = from_f32<OutT>(v);
  }
}

// Host-side launch of one instantiation over an (N/BN, M/BM, batch x splits)
// grid, followed by the reduction when the contraction is split.
template <typename T, typename OutT, class Cfg, int AMODE, int BMODE, bool AGATE, bool BGATE, int EPI>
inline hipError_t launch_gemm(const GemmArgs& g, int batch, hipStream_t stream) {
  const int splits = g.splits > 1 ? g.splits : 1;
  dim3 grid((g.N + Cfg::BN - 1) / Cfg::BN, (g.M + Cfg::BM - 1) / Cfg::BM, batch * splits);
  hipLaunchKernelGGL((gemm_kernel<T, OutT, Cfg, AMODE, BMODE, AGATE, BGATE, EPI>), grid, dim3(Cfg::NT), 0,
                     stream, g);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || splits == 1) return e;
  const int64_t mn = static_cast<int64_t>(g.M) * g.N;
  hipLaunchKernelGGL((splitk_reduce_kernel<OutT, EPI>), dim3(static_cast<unsigned>((mn + 255) / 256), batch),
                     dim3(256), 0, stream, g);
  return hipGetLastError();
}

template <typename T, typename OutT, int AMODE, int BMODE, bool AGATE, bool BGATE, int EPI>
inline hipError_t launch_small(const GemmArgs& g, int batch, hipStream_t stream) {
  const int splits = g.splits > 1 ? g.splits : 1;
  dim3 grid((g.N + 31) / 32, (g.M + 31) / 32, batch * splits);
  hipLaunchKernelGGL((gemm_small_kernel<T, OutT, AMODE, BMODE, AGATE, BGATE, EPI>), grid, dim3(256), 0, stream, g);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || splits == 1) return e;
  const int64_t mn = static_cast<int64_t>(g.M) * g.N;
  hipLaunchKernelGGL((splitk_reduce_kernel<OutT, EPI>), dim3(static_cast<unsigned>((mn + 255) / 256), batch),
                     dim3(256), 0, stream, g);
  return hipGetLastError();
}

template <typename T, typename OutT, int A0, int A1, int B0, int B1, bool AGATE, bool BGATE, int EPI>
inline hipError_t dispatch_small(const GemmArgs& g, int batch, bool a_vec, bool b_vec, hipStream_t stream) {
  if (a_vec) {
    if (b_vec) return launch_small<T, OutT, A0, B0, AGATE, BGATE, EPI>(g, batch, stream);
    return launch_small<T, OutT, A0, B1, AGATE, BGATE, EPI>(g, batch, stream);
  }
  if (b_vec) return launch_small<T, OutT, A1, B0, AGATE, BGATE, EPI>(g, batch, stream);
  return launch_small<T, OutT, A1, B1, AGATE, BGATE, EPI>(g, batch, stream);
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

// Tile shapes of the general kernel: 128x128 and 64x64 output tiles.
template <typename T>
struct GemmCfgs;
template <>
struct GemmCfgs<bf16> {
  using Big = TileCfg<128, 128, 64, 2, 2>;
  using Small = TileCfg<64, 64, 64, 2, 2>;
};
template <>
struct GemmCfgs<float> {
  using Big = TileCfg<128, 128, 32, 2, 2>;
  using Small = TileCfg<64, 64, 32, 2, 2>;
};

constexpr int kTargetBlocks = 256;   // one workgroup per compute unit
constexpr int kMaxSplits = 16;
constexpr int kMinSlabsPerSplit = 4;

enum TileKind { TILE_BIG = 0, TILE_MEDIUM = 1, TILE_SMALL = 2 };

struct GemmPlan {
  int kind;
  int splits;
};

// Picks the tile shape and the split of the contraction for a problem:
// 128x128 tiles when they fill half the chip, 64x64 when those fill it,
// otherwise 32x32 blocks with the contraction split inside the workgroup
// (and over workgroups while the grid stays below one workgroup per CU).
template <typename T>
inline GemmPlan plan_gemm(int M, int N, int K, int kbatch, int batch) {
  using C = GemmCfgs<T>;
  auto tiles_of = [&](int bm, int bn) {
    return static_cast<int64_t>((M + bm - 1) / bm) * ((N + bn - 1) / bn) * batch;
  };
  GemmPlan p;
  int bk;
  int64_t tiles;
  if (tiles_of(C::Big::BM, C::Big::BN) >= kTargetBlocks / 2) {
    p.kind = TILE_BIG;
    bk = C::Big::BK;
    tiles = tiles_of(C::Big::BM, C::Big::BN);
  } else if (tiles_of(C::Small::BM, C::Small::BN) >= kTargetBlocks) {
    p.kind = TILE_MEDIUM;
    bk = C::Small::BK;
    tiles = tiles_of(C::Small::BM, C::Small::BN);
  } else {
    p.kind = TILE_SMALL;
    bk = SmallCfg<T>::BK;
    tiles = tiles_of(32, 32);
  }
  const int64_t slabs = static_cast<int64_t>(kbatch > 0 ? kbatch : 1) * ((K + bk - 1) / bk);
  int s = 1;
  while (tiles * s * 2 <= kTargetBlocks && slabs / (s * 2) >= kMinSlabsPerSplit && s * 2 <= kMaxSplits) s *= 2;
  p.splits = s;
  return p;
}

// fp32 elements of split-K partials a problem needs (0 when it is not split).
template <typename T>
inline size_t gemm_partial_floats(int M, int N, int K, int kbatch, int batch) {
  const GemmPlan p = plan_gemm<T>(M, N, K, kbatch, batch);
  return p.splits > 1 ? static_cast<size_t>(p.splits) * batch * M * N : 0;
}

// Runs a gathered GEMM. `partial` must hold gemm_partial_floats() floats when
// that is nonzero; with partial == NULL the contraction is never split.
template <typename T, typename OutT, int A0, int A1, int B0, int B1, bool AGATE, bool BGATE, int EPI>
inline hipError_t run_gemm(GemmArgs g, int batch, bool a_vec, bool b_vec, hipStream_t stream,
                           float* partial = nullptr) {
  if (g.M <= 0 || g.N <= 0 || batch <= 0) return hipSuccess;
  GemmPlan p = plan_gemm<T>(g.M, g.N, g.K, g.kbatch, batch);
  if (!partial) p.splits = 1;
  g.splits = p.splits;
  g.partial = partial;
  if (p.kind == TILE_BIG)
    return dispatch_gemm<T, OutT, typename GemmCfgs<T>::Big, A0, A1, B0, B1, AGATE, BGATE, EPI>(
        g, batch, a_vec, b_vec, stream);
  if (p.kind == TILE_MEDIUM)
    return dispatch_gemm<T, OutT, typename GemmCfgs<T>::Small, A0, A1, B0, B1, AGATE, BGATE, EPI>(
        g, batch, a_vec, b_vec, stream);
  return dispatch_small<T, OutT, A0, A1, B0, B1, AGATE, BGATE, EPI>(g, batch, a_vec, b_vec, stream);
}

}  // namespace ard
