// bf16 gathered GEMM for large compact problems on gfx950.
//
// The same contraction as gemm_kernel (ard_gemm.hpp) with operands that allow
// 16-byte chunks (rows of a multiple of 8 elements, no column gathers, no
// load-time gates), shaped for MFMA throughput:
//
//  * global -> LDS without register staging: each lane issues
//    global_load_lds_dwordx4 for one 16-byte chunk of a (row-gathered) tile;
//    a wave writes 64 consecutive LDS chunks, and the lane picks the global
//    chunk that belongs at its LDS position under an XOR swizzle, which keeps
//    the MFMA fragment reads free of bank conflicts;
//  * k-contiguous operands live in LDS as [rows][64 k] and are read with
//    ds_read_b128; m/n-contiguous operands (feature-major activations,
//    transposed weights) live as [64 k][rows] exactly as in HBM and are read
//    with ds_read_b64_tr_b16, whose 16-lane transpose delivers 4 consecutive
//    k of one column per lane — no transpose pass anywhere;
//  * two LDS stages of a 64-deep K slab: the loads of slab q+1 are in flight
//    while the waves run v_mfma_f32_32x32x16_bf16 on slab q;
//  * the last, partial K slab is cleaned in LDS (entries past the contraction
//    length set to 0) before use; rows past the output extents load a clamped
//    valid row and their results are discarded.
#pragma once

#include "ard_gemm.hpp"

namespace ard {

typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;

template <int BM_, int BN_, int WGM_, int WGN_>
struct FastCfg {
  static constexpr int BM = BM_, BN = BN_, BK = 64, WGM = WGM_, WGN = WGN_;
  static constexpr int NT = 64 * WGM * WGN, NW = WGM * WGN;
  static constexpr int TM = BM / WGM, TN = BN / WGN;
  static constexpr int FM = TM / 32, FN = TN / 32;
};

// Byte offsets of 16-byte chunk c of row r. k-contiguous tiles have 8 chunks
// (64 k) per row, swizzled by row / 2; m/n-contiguous tiles have CPR chunks per
// k-row, the low three chunk bits swizzled by k. Loads and fragment reads use
// the same maps.
__device__ __forceinline__ int kc_chunk(int r, int c) { return (r * 8 + (c ^ ((r >> 1) & 7))) * 16; }
template <int CPR>
__device__ __forceinline__ int mc_chunk(int k, int c) { return (k * CPR + (c ^ (k & 7))) * 16; }

// Issues this wave's direct loads of one operand tile for the slab at k0.
//   KC: tile rows r0.. (R of them, gathered by ridx), 64 k per row, LDS [R][64]
//   MC: tile k-rows k0.. (64, gathered by ridx), R columns, LDS [64][R]
template <class Cfg, int R, bool MC>
__device__ __forceinline__ void fast_issue(const bf16* base, int64_t ld, const int32_t* ridx, int r0,
                                           int rext, int k0, int kext, char* region) {
  constexpr int CHUNKS = R * 8;                      // R * 64 bf16 / 8 per chunk
  constexpr int PER_WAVE = CHUNKS / 64 / Cfg::NW;     // load instructions per wave
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
#pragma unroll
  for (int i = 0; i < PER_WAVE; ++i) {
    const int blk = wave * PER_WAVE + i;
    const int pos = blk * 64 + lane;  // chunk position in the LDS region
    int64_t off;
    if constexpr (!MC) {
      const int r = pos >> 3;
      const int c = (pos & 7) ^ ((r >> 1) & 7);
      int row = r0 + r;
      row = row < rext ? row : rext - 1;
      int k = k0 + c * 8;
      k = k < kext ? k : 0;
      off = gather(ridx, row) * ld + k;
    } else {
      constexpr int CPR = R / 8;
      const int kk = pos / CPR;
      const int c = (pos % CPR) ^ (kk & 7);
      int krow = k0 + kk;
      krow = krow < kext ? krow : kext - 1;
      int col = r0 + c * 8;
      col = col < rext ? col : 0;
      off = gather(ridx, krow) * ld + col;
    }
    __builtin_amdgcn_global_load_lds(base + off, (lds_void*)(region + blk * 1024), 16, 0, 0);
  }
}

// Zeroes the entries of a loaded slab whose k is >= kvalid (k counted from the
// slab start).
template <class Cfg, int R, bool MC>
__device__ __forceinline__ void fast_zero_tail(char* region, int kvalid) {
  if constexpr (!MC) {
    // rows of 64 k: element (r, k) lives in chunk k / 8 of row r
    for (int e = threadIdx.x; e < R * 64; e += Cfg::NT) {
      const int r = e >> 6, k = e & 63;
      if (k >= kvalid)
        *reinterpret_cast<uint16_t*>(region + kc_chunk(r, k >> 3) + (k & 7) * 2) = 0;
    }
  } else {
    // k-rows of R columns: clear whole rows kk >= kvalid
    constexpr int CPR = R / 8;
    for (int e = threadIdx.x; e < 64 * CPR; e += Cfg::NT) {
      const int kk = e / CPR;
      if (kk >= kvalid) *reinterpret_cast<u32x4*>(region + kk * CPR * 16 + (e % CPR) * 16) = u32x4{0u, 0u, 0u, 0u};
    }
  }
}

// MFMA operand fragment (8 k of one row/column for this lane) at k offset kk
// of the slab, for the 32-row block starting at tile row rb.
template <int R, bool MC>
__device__ __forceinline__ bf16x8 fast_frag(const char* region, int rb, int kk) {
  const int lane = threadIdx.x & 63;
  if constexpr (!MC) {
    const int row = rb + (lane & 31);
    const int c = (kk >> 3) + (lane >> 5);
    return *reinterpret_cast<const bf16x8*>(region + kc_chunk(row, c));
  } else {
    // 16-lane groups: group g covers columns rb + 16 (g % 2) .. +15 and k
    // kk + 8 (g / 2) .. +7, read as two 4-k transposed halves
    constexpr int CPR = R / 8;
    const int g = lane >> 4, s = lane & 15;
    const int col = rb + 16 * (g & 1) + 4 * (s & 3);
    const int kbase = kk + 8 * (g >> 1) + (s >> 2);
    i16x4 lo, hi;
    {
      const int kr = kbase;
      const char* p = region + mc_chunk<CPR>(kr, col >> 3) + (col & 7) * 2;
      lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)(p));
    }
    {
      const int kr = kbase + 4;
      const char* p = region + mc_chunk<CPR>(kr, col >> 3) + (col & 7) * 2;
      hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)(p));
    }
    bf16x8 out;
    const bf16* l4 = reinterpret_cast<const bf16*>(&lo);
    const bf16* h4 = reinterpret_cast<const bf16*>(&hi);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      out[e] = l4[e];
      out[e + 4] = h4[e];
    }
    return out;
  }
}

template <class Cfg, bool AMC, bool BMC, typename OutT, int EPI>
__global__ void __launch_bounds__(Cfg::NT) fast_gemm_kernel(GemmArgs g) {
  constexpr int ABYTES = Cfg::BM * 64 * 2, BBYTES = Cfg::BN * 64 * 2;
  constexpr int STAGE = ABYTES + BBYTES;
  extern __shared__ __attribute__((aligned(16))) char smem[];

  // XCD-aware order: consecutive workgroups land on different XCDs, so give
  // each XCD a contiguous run of output tiles (shared operand rows in its L2).
  const int nx = gridDim.x, ny = gridDim.y;
  const int nxy = nx * ny;
  int bid = blockIdx.y * nx + blockIdx.x;
  if (nxy % 8 == 0) bid = (bid % 8) * (nxy / 8) + bid / 8;
  const int n0 = (bid % nx) * Cfg::BN;
  const int m0 = (bid / nx) * Cfg::BM;
  const int splits = g.splits > 1 ? g.splits : 1;
  const int64_t bz = blockIdx.z / splits;
  const int split = blockIdx.z % splits;
  const int wave = threadIdx.x >> 6;
  const int wm = wave / Cfg::WGN, wn = wave % Cfg::WGN;

  const bf16* abase = static_cast<const bf16*>(g.a.p) + bz * g.a.bstride;
  const bf16* bbase = static_cast<const bf16*>(g.b.p) + bz * g.b.bstride;

  f32x16 acc[Cfg::FM][Cfg::FN];
#pragma unroll
  for (int i = 0; i < Cfg::FM; ++i)
#pragma unroll
    for (int j = 0; j < Cfg::FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  const int nks = (g.K + 63) / 64;
  const int kbatch = g.kbatch > 0 ? g.kbatch : 1;
  const int nslab = kbatch * nks;
  const int q0 = static_cast<int>((static_cast<int64_t>(nslab) * split) / splits);
  const int q1 = static_cast<int>((static_cast<int64_t>(nslab) * (split + 1)) / splits);

  auto issue = [&](int q, int stage) {
    const int kb = q / nks, k0 = (q % nks) * 64;
    char* st = smem + stage * STAGE;
    fast_issue<Cfg, Cfg::BM, AMC>(abase + kb * g.a.kbstride, g.a.ld, g.a.ridx, m0, g.M, k0, g.K, st);
    fast_issue<Cfg, Cfg::BN, BMC>(bbase + kb * g.b.kbstride, g.b.ld, g.b.ridx, n0, g.N, k0, g.K, st + ABYTES);
  };

  if (q0 < q1) issue(q0, 0);
  for (int q = q0; q < q1; ++q) {
    const int cur = (q - q0) & 1;
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (q + 1 < q1) issue(q + 1, cur ^ 1);
    char* st = smem + cur * STAGE;
    const int kvalid = g.K - (q % nks) * 64;
    if (kvalid < 64) {
      fast_zero_tail<Cfg, Cfg::BM, AMC>(st, kvalid);
      fast_zero_tail<Cfg, Cfg::BN, BMC>(st + ABYTES, kvalid);
      __syncthreads();
    }
#pragma unroll
    for (int kk = 0; kk < 64; kk += 16) {
      bf16x8 a[Cfg::FM], b[Cfg::FN];
#pragma unroll
      for (int i = 0; i < Cfg::FM; ++i) a[i] = fast_frag<Cfg::BM, AMC>(st, wm * Cfg::TM + 32 * i, kk);
#pragma unroll
      for (int j = 0; j < Cfg::FN; ++j) b[j] = fast_frag<Cfg::BN, BMC>(st + ABYTES, wn * Cfg::TN + 32 * j, kk);
#pragma unroll
      for (int i = 0; i < Cfg::FM; ++i)
#pragma unroll
        for (int j = 0; j < Cfg::FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
  }
  store_tile<OutT, Cfg, EPI>(g, acc, m0, n0, wm, wn, bz, split);
}

using FastHuge = FastCfg<256, 256, 2, 2>;
using FastBig = FastCfg<128, 128, 2, 2>;

template <class Cfg>
constexpr int fast_lds_bytes() { return 2 * (Cfg::BM + Cfg::BN) * 64 * 2; }

// Whether a bf16 problem can run on fast_gemm_kernel: every operand view is
// read in whole 16-byte chunks (row stride a multiple of 8 elements, aligned
// base, no column gather, no load-time gate).
inline bool fast_ok(const GemmOperand& a, const GemmOperand& b) {
  auto ok = [](const GemmOperand& o) {
    return o.cidx == nullptr && o.y == nullptr && o.ld % 8 == 0 && o.bstride % 8 == 0 && o.kbstride % 8 == 0 &&
           (reinterpret_cast<uintptr_t>(o.p) & 15u) == 0;
  };
  return ok(a) && ok(b);
}

struct FastPlan {
  int cfg;     // 0: 256x256, 1: 128x128
  int splits;
};

inline FastPlan plan_fast(int M, int N, int K, int kbatch, int batch) {
  FastPlan p;
  const int64_t huge = static_cast<int64_t>((M + 255) / 256) * ((N + 255) / 256) * batch;
  p.cfg = huge >= 160 ? 0 : 1;
  const int bm = p.cfg == 0 ? 256 : 128;
  const int64_t tiles = static_cast<int64_t>((M + bm - 1) / bm) * ((N + bm - 1) / bm) * batch;
  const int64_t slabs = static_cast<int64_t>(kbatch > 0 ? kbatch : 1) * ((K + 63) / 64);
  int s = 1;
  while (tiles * s * 2 <= kTargetBlocks && slabs / (s * 2) >= kMinSlabsPerSplit && s * 2 <= kMaxSplits) s *= 2;
  p.splits = s;
  return p;
}

inline size_t fast_partial_floats(int M, int N, int K, int kbatch, int batch) {
  const FastPlan p = plan_fast(M, N, K, kbatch, batch);
  return p.splits > 1 ? static_cast<size_t>(p.splits) * batch * M * N : 0;
}

template <class Cfg, bool AMC, bool BMC, typename OutT, int EPI>
inline hipError_t launch_fast(const GemmArgs& g, int batch, hipStream_t stream) {
  const int splits = g.splits > 1 ? g.splits : 1;
  auto kern = fast_gemm_kernel<Cfg, AMC, BMC, OutT, EPI>;
  static bool attr_set = false;  // per instantiation: allow > 64 KB of dynamic LDS
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, fast_lds_bytes<Cfg>());
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  dim3 grid((g.N + Cfg::BN - 1) / Cfg::BN, (g.M + Cfg::BM - 1) / Cfg::BM, batch * splits);
  hipLaunchKernelGGL(kern, grid, dim3(Cfg::NT), fast_lds_bytes<Cfg>(), stream, g);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || splits == 1) return e;
  const int64_t mn = static_cast<int64_t>(g.M) * g.N;
  hipLaunchKernelGGL((splitk_reduce_kernel<OutT, EPI>), dim3(static_cast<unsigned>((mn + 255) / 256), batch),
                     dim3(256), 0, stream, g);
  return hipGetLastError();
}

// Runs a bf16 GEMM on the fast kernel; the caller has checked fast_ok().
template <bool AMC, bool BMC, typename OutT, int EPI>
inline hipError_t run_fast_gemm(GemmArgs g, int batch, hipStream_t stream, float* partial) {
  if (g.M <= 0 || g.N <= 0 || batch <= 0) return hipSuccess;
  FastPlan p = plan_fast(g.M, g.N, g.K, g.kbatch, batch);
  if (!partial) p.splits = 1;
  g.splits = p.splits;
  g.partial = partial;
  if (p.cfg == 0) return launch_fast<FastHuge, AMC, BMC, OutT, EPI>(g, batch, stream);
  return launch_fast<FastBig, AMC, BMC, OutT, EPI>(g, batch, stream);
}

}  // namespace ard
