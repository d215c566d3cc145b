// GEMM with direct global -> LDS loads and a deep K pipeline (gfx950).
//
// The same contraction as gemm_kernel (ard_gemm.hpp) for operand views that
// can be read in whole 16-byte chunks (row stride a multiple of 16 bytes,
// aligned base, no row or column gather, no load-time gate):
//
//  * global -> LDS without register staging: each lane issues
//    global_load_lds_dwordx4 for one 16-byte chunk of a tile;
//    a wave writes 64 consecutive LDS chunks, and the lane picks the global
//    chunk that belongs at its LDS position under an XOR swizzle that keeps the
//    MFMA fragment reads free of bank conflicts;
//  * k-contiguous operands live in LDS as [rows][BK] and are read as whole
//    fragments (ds_read_b128); m/n-contiguous operands (feature-major
//    activations, transposed weights) stay [BK][rows] exactly as in HBM: bf16
//    fragments come from ds_read_b64_tr_b16, whose 16-lane transpose delivers
//    4 consecutive k of one column per lane, fp32 fragments from one
//    ds_read_b32 per k (consecutive lanes read consecutive columns);
//  * STAGES LDS stages: the loads of the next STAGES - 1 slabs are in flight
//    while the waves run MFMA on the current one; a wave waits only for the
//    slab it is about to use (vmcnt counts the later slabs it has issued);
//  * optionally the waves of a workgroup split each slab's k between them and
//    reduce through LDS at the end (small output tiles that still fill the
//    chip);
//  * the last, partial K slab is cleaned in LDS (entries past the contraction
//    length set to 0) before use; rows past the output extents load a clamped
//    valid row and their results are discarded;
//  * operands are plain strided views (a row-based pattern's gather is folded
//    into base and row stride by the caller), so the main loop reads no index
//    lists: an index load would make the wave wait for every earlier direct load.
//
// The direct loads are issued as inline assembly and ordered only by the
// explicit vmcnt waits and LDS barriers of the main loop: the compiler, which
// cannot tell that an LDS read targets another stage than the loads in
// flight, would otherwise wait for all of them before such reads, and
// __syncthreads() waits for all outstanding vector memory operations.
#pragma once

#include <type_traits>

#include "ard_gemm.hpp"

namespace ard {

typedef short i16x4 __attribute__((ext_vector_type(4)));

template <typename T_, int BM_, int BN_, int BK_, int STAGES_, int WGM_, int WGN_, int KSPLIT_>
struct FastCfg {
  using T = T_;
  static constexpr int BM = BM_, BN = BN_, BK = BK_, STAGES = STAGES_;
  static constexpr int WGM = WGM_, WGN = WGN_, KSPLIT = KSPLIT_;
  static constexpr int NW = WGM * WGN * KSPLIT, NT = 64 * NW;
  static constexpr int TM = BM / WGM, TN = BN / WGN;  // wave tile
  static constexpr int FM = TM / 32, FN = TN / 32;    // 32x32 MFMA blocks per wave
  static constexpr int KW = BK / KSPLIT;              // k per wave per slab
  static constexpr int ES = sizeof(T);
  static constexpr int ABYTES = BM * BK * ES, BBYTES = BN * BK * ES;
  static constexpr int STAGE = ABYTES + BBYTES;
  static constexpr int LDS = STAGES * STAGE;
  // 16-byte load instructions per wave per slab
  static constexpr int LPW = (ABYTES + BBYTES) / 16 / 64 / NW;
  static_assert(ABYTES % (1024 * NW) == 0 && BBYTES % (1024 * NW) == 0, "tile must split into wave loads");
  static_assert(KW % (ES == 2 ? 16 : 8) == 0, "per-wave k must hold whole MFMA steps");
};

// LDS layout. gfx950 LDS has 64 banks of 4 bytes: a wave's 16-byte reads are
// served 16 lanes per pass, its 8-byte reads 32 lanes per pass, and a pass is
// free of bank conflicts when its lanes touch 16 different 16-byte bank groups
// (byte address / 16 mod 16). Chunk c of row r goes to position
// r * CPR + (c ^ swizzle(r)); the swizzles make the fragment reads below
// conflict-free.
//
// k-contiguous tiles [R][BK] (CPR = BK*ES/16 chunks per row), read as 16 bytes
// per lane from 16 consecutive rows at one chunk: rows r and r + 16/CPR share
// bank groups unless the swizzle tells them apart.
template <int CPR>
__device__ __forceinline__ int kc_swz(int r) {
  constexpr int SH = CPR >= 16 ? 0 : CPR == 8 ? 1 : CPR == 4 ? 2 : 3;
  return (r >> SH) & (CPR - 1);
}
// m/n-contiguous tiles [BK][R] (CPR = R*ES/16 chunks per k-row). 16-bit data
// is read transposed: per 32 lanes, 4 consecutive k-rows x 4 consecutive
// chunks; 32-bit data per lane from k-rows k and k + 4, 8 chunks each.
template <int CPR, int ES>
__device__ __forceinline__ int mc_swz(int k) {
  if constexpr (ES == 2) {
    if constexpr (CPR >= 16)
      return (k & 3) << 2;
    else if constexpr (CPR == 8)
      return ((k >> 1) & 1) << 2;
    else
      return 0;
  } else {
    if constexpr (CPR >= 16)
      return ((k >> 2) & 1) << 3;
    else
      return 0;
  }
}

template <int CPR>
__device__ __forceinline__ int kc_off(int r, int c) {
  return (r * CPR + (c ^ kc_swz<CPR>(r))) * 16;
}
template <int CPR, int ES>
__device__ __forceinline__ int mc_off(int k, int c) {
  return (k * CPR + (c ^ mc_swz<CPR, ES>(k))) * 16;
}

// One direct load of 16 bytes per lane from sbase + voff into LDS at
// lds_base + 16 * lane. sbase (an SGPR pair) and lds_base are wave-uniform;
// lds_base travels in M0, which the compiler writes before the statement and
// which the load reads one wait state later at the earliest. The compiler's
// hazard tracking does not look into the statement: the first load of a group
// (FIRST) also waits the 5 states a vector memory instruction needs after a
// VALU write (v_readfirstlane) of an SGPR it reads; later loads of the group
// use the same base. No memory clobber: the load writes a stage that no LDS
// access between two loop barriers touches, and volatile statements keep
// their order relative to the barriers and waits.
template <bool FIRST>
__device__ __forceinline__ void dma16(const void* sbase, uint32_t voff, uint32_t lds_base) {
  if constexpr (FIRST)
    asm volatile(
        "s_nop 4\n\t"
        "global_load_lds_dwordx4 %0, %1"
        :
        : "v"(voff), "s"(sbase), "{m0}"(lds_base));
  else
    asm volatile(
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %0, %1"
        :
        : "v"(voff), "s"(sbase), "{m0}"(lds_base));
}

// A wave-uniform pointer as such (SGPR pair): integer division and other VALU
// lowerings leave uniform values in VGPRs.
__device__ __forceinline__ const char* uniform_ptr(const char* p) {
  const uint64_t v = reinterpret_cast<uint64_t>(p);
  const uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(v));
  const uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(v >> 32));
  return reinterpret_cast<const char*>((static_cast<uint64_t>(hi) << 32) | lo);
}

// LDS address (byte offset in the workgroup's LDS) of a pointer into shared memory.
__device__ __forceinline__ uint32_t lds_addr(const char* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((const __attribute__((address_space(3))) char*)p));
}

// Workgroup barrier for the LDS hand-off: waits for this wave's own LDS
// operations only, not for its direct loads in flight.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// Per-lane sources of one operand's direct loads. Per slab a wave loads
// PER_WAVE blocks of 64 16-byte chunks; LDS chunk pos = blk * 64 + lane of the
// operand's region holds, for a k-contiguous tile [R][BK], row pos / CPR and
// the swizzled k chunk; for an m/n-contiguous tile [BK][R], k-row pos / CPR
// and the swizzled column chunk. A chunk is addressed as a 32-bit byte offset
// from the slab's first element (uniform, in SGPRs). Rows and columns past the
// extents are clamped once to a valid one (their results are discarded); a
// chunk past the contraction length of a partial slab loads the same row's
// (or column's) chunk at k 0 of the slab instead, and the slab's tail is
// zeroed in LDS before use.
template <class Cfg, int R, bool MC>
struct DmaSrc {
  static constexpr int ES = Cfg::ES, EPC = 16 / ES;  // EPC: elements per chunk
  static constexpr int CPR = MC ? R * ES / 16 : Cfg::BK * ES / 16;
  static constexpr int PER_WAVE = R * Cfg::BK * ES / 1024 / Cfg::NW;
  uint32_t off[PER_WAVE];   // byte offset of the lane's chunk from the slab base
  uint32_t off0[PER_WAVE];  // the same chunk at k (KC) or k-row (MC) 0 of the slab
  int k[PER_WAVE];          // the chunk's k (KC) or k-row (MC) within the slab

  __device__ __forceinline__ void init(int64_t ld, int r0, int rext, int wave) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int i = 0; i < PER_WAVE; ++i) {
      const int pos = (wave * PER_WAVE + i) * 64 + lane;
      if constexpr (!MC) {
        const int r = pos / CPR;
        const int c = (pos % CPR) ^ kc_swz<CPR>(r);
        const int row = r0 + r < rext ? r0 + r : rext - 1;
        off0[i] = static_cast<uint32_t>(row * ld * ES);
        off[i] = off0[i] + static_cast<uint32_t>(c * 16);
        k[i] = c * EPC;
      } else {
        const int kk = pos / CPR;
        const int c = (pos % CPR) ^ mc_swz<CPR, ES>(kk);
        const int col = r0 + c * EPC < rext ? r0 + c * EPC : 0;
        off0[i] = static_cast<uint32_t>(col * ES);
        off[i] = off0[i] + static_cast<uint32_t>(kk * ld * ES);
        k[i] = kk;
      }
    }
  }

  // A k-contiguous operand whose tile row r is row rowof(r) of the view: a
  // row gather folded into the lane offsets once, so the main loop reads no
  // index. Every rowof(r) must be a valid row.
  template <class F>
  __device__ __forceinline__ void init_rows(int64_t ld, F rowof, int wave) {
    static_assert(!MC, "row gather of a k-contiguous operand");
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int i = 0; i < PER_WAVE; ++i) {
      const int pos = (wave * PER_WAVE + i) * 64 + lane;
      const int r = pos / CPR;
      const int c = (pos % CPR) ^ kc_swz<CPR>(r);
      off0[i] = static_cast<uint32_t>(static_cast<int64_t>(rowof(r)) * ld * ES);
      off[i] = off0[i] + static_cast<uint32_t>(c * 16);
      k[i] = c * EPC;
    }
  }

  // Loads the slab whose first element is at sbase (uniform), of which the
  // first kv k (k-rows) are valid, into the LDS region at byte address region.
  __device__ __forceinline__ void issue(const char* sbase, int kv, uint32_t region, int wave) const {
    const char* b = uniform_ptr(sbase);
    const uint32_t r0 = region + static_cast<uint32_t>(wave * PER_WAVE * 1024);
    dma16<true>(b, k[0] < kv ? off[0] : off0[0], r0);
#pragma unroll
    for (int i = 1; i < PER_WAVE; ++i) dma16<false>(b, k[i] < kv ? off[i] : off0[i], r0 + static_cast<uint32_t>(i * 1024));
  }
};

// Zeroes the entries of a loaded slab whose k is >= kvalid (k from the slab start).
template <class Cfg, int R, bool MC>
__device__ __forceinline__ void fast_zero_tail(char* region, int kvalid) {
  constexpr int ES = Cfg::ES, EPC = 16 / ES;
  if constexpr (!MC) {
    constexpr int CPR = Cfg::BK * ES / 16;
    for (int e = threadIdx.x; e < R * Cfg::BK; e += Cfg::NT) {
      const int r = e / Cfg::BK, k = e % Cfg::BK;
      if (k >= kvalid) {
        char* p = region + kc_off<CPR>(r, k / EPC) + (k % EPC) * ES;
        if constexpr (ES == 2)
          *reinterpret_cast<uint16_t*>(p) = 0;
        else
          *reinterpret_cast<uint32_t*>(p) = 0;
      }
    }
  } else {
    constexpr int CPR = R * ES / 16;
    for (int e = threadIdx.x; e < Cfg::BK * CPR; e += Cfg::NT) {
      const int kk = e / CPR;
      if (kk >= kvalid) *reinterpret_cast<u32x4*>(region + e * 16) = u32x4{0u, 0u, 0u, 0u};
    }
  }
}

// bf16 MFMA operand fragment: 8 k (kk .. kk+15 split over the two lane halves)
// of the row/column rb + lane % 32.
template <class Cfg, int R, bool MC>
__device__ __forceinline__ bf16x8 frag_bf16(const char* region, int rb, int kk) {
  const int lane = threadIdx.x & 63;
  if constexpr (!MC) {
    constexpr int CPR = Cfg::BK * 2 / 16;
    return *reinterpret_cast<const bf16x8*>(region + kc_off<CPR>(rb + (lane & 31), (kk >> 3) + (lane >> 5)));
  } else {
    // 16-lane group g covers columns rb + 16 (g % 2) .. +15 and k kk + 8 (g / 2) .. +7,
    // read as two transposed 4-k halves
    constexpr int CPR = R * 2 / 16;
    const int g = lane >> 4, s = lane & 15;
    const int col = rb + 16 * (g & 1) + 4 * (s & 3);
    const int kr = kk + 8 * (g >> 1) + (s >> 2);
    const char* p0 = region + mc_off<CPR, 2>(kr, col >> 3) + (col & 7) * 2;
    const char* p1 = region + mc_off<CPR, 2>(kr + 4, col >> 3) + (col & 7) * 2;
    const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)(p0));
    const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)(p1));
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

// fp32 MFMA operands: 4 k (kk + 4 * (lane / 32) + 0..3) of row/column rb + lane % 32.
template <class Cfg, int R, bool MC>
__device__ __forceinline__ f32x4 frag_f32(const char* region, int rb, int kk) {
  const int lane = threadIdx.x & 63;
  const int rc = rb + (lane & 31), k = kk + 4 * (lane >> 5);
  if constexpr (!MC) {
    constexpr int CPR = Cfg::BK * 4 / 16;
    return *reinterpret_cast<const f32x4*>(region + kc_off<CPR>(rc, k >> 2));
  } else {
    constexpr int CPR = R * 4 / 16;
    f32x4 v;
#pragma unroll
    for (int e = 0; e < 4; ++e)
      v[e] = *reinterpret_cast<const float*>(region + mc_off<CPR, 4>(k + e, rc >> 2) + (rc & 3) * 4);
    return v;
  }
}

template <int N>
__device__ __forceinline__ void wait_vm() {
  if constexpr (N == 0)
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  else
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Fragments of one k step (16 bf16 or 8 fp32 k) of a wave's output tile, and
// the MFMAs that consume them.
template <class Cfg, bool AMC, bool BMC>
struct StepFrags {
  static constexpr int KSTEP = Cfg::ES == 2 ? 16 : 8;
  using FT = typename std::conditional<Cfg::ES == 2, bf16x8, f32x4>::type;
  FT a[Cfg::FM], b[Cfg::FN];

  __device__ __forceinline__ void load(const char* st, int wm, int wn, int kk) {
#pragma unroll
    for (int i = 0; i < Cfg::FM; ++i) {
      if constexpr (Cfg::ES == 2)
        a[i] = frag_bf16<Cfg, Cfg::BM, AMC>(st, wm * Cfg::TM + 32 * i, kk);
      else
        a[i] = frag_f32<Cfg, Cfg::BM, AMC>(st, wm * Cfg::TM + 32 * i, kk);
    }
#pragma unroll
    for (int j = 0; j < Cfg::FN; ++j) {
      if constexpr (Cfg::ES == 2)
        b[j] = frag_bf16<Cfg, Cfg::BN, BMC>(st + Cfg::ABYTES, wn * Cfg::TN + 32 * j, kk);
      else
        b[j] = frag_f32<Cfg, Cfg::BN, BMC>(st + Cfg::ABYTES, wn * Cfg::TN + 32 * j, kk);
    }
  }

  // Adds the A values of this k step to per-lane row sums: with a
  // k-contiguous A, lane l holds k values of row rb + l % 32 only. bf16 pairs
  // go through v_dot2 against (1, 1), which needs no unpacked temporaries
  // (the 256x256 tile has no registers to spare).
  __device__ __forceinline__ void rowsum(float (&rs)[Cfg::FM]) const {
    static_assert(!AMC, "row sums need a k-contiguous A");
#pragma unroll
    for (int i = 0; i < Cfg::FM; ++i) {
      if constexpr (Cfg::ES == 2) {
        typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
        const bf16x2 one = {static_cast<bf16>(1.0f), static_cast<bf16>(1.0f)};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const bf16x2 pr = {a[i][2 * e], a[i][2 * e + 1]};
          rs[i] = __builtin_amdgcn_fdot2_f32_bf16(pr, one, rs[i], false);
        }
      } else {
        rs[i] += (a[i][0] + a[i][1]) + (a[i][2] + a[i][3]);
      }
    }
  }

  __device__ __forceinline__ void mma(f32x16 (&acc)[Cfg::FM][Cfg::FN]) const {
    if constexpr (Cfg::ES == 2) {
#pragma unroll
      for (int i = 0; i < Cfg::FM; ++i)
#pragma unroll
        for (int j = 0; j < Cfg::FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e)
#pragma unroll
        for (int i = 0; i < Cfg::FM; ++i)
#pragma unroll
          for (int j = 0; j < Cfg::FN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[i][e], b[j][e], acc[i][j], 0, 0, 0);
    }
  }
};

// The direct loads of one operand pair, slab after slab: wave-uniform
// pointers to the next slab's first element, its first k, its stage, and how
// many slabs of the split are still to come after it. Past the last slab the
// last one is loaded again (into a stage no longer read), so every wave issues
// the same number of loads per slab.
template <class Cfg, bool AMC, bool BMC>
struct SlabLoader {
  DmaSrc<Cfg, Cfg::BM, AMC> da;
  DmaSrc<Cfg, Cfg::BN, BMC> db;
  const char* na;
  const char* nb;
  int64_t a_step, b_step, a_wrap, b_wrap;
  int K, ik, is, left, wv;
  uint32_t lds0;

  // One slab's loads in two halves: A (issue_a), then B and the advance to
  // the next slab (issue_b); issue() does both.
  __device__ __forceinline__ void issue_a() {
    da.issue(na, K - ik, lds0 + static_cast<uint32_t>(is * Cfg::STAGE), wv);
  }
  __device__ __forceinline__ void issue_b() {
    db.issue(nb, K - ik, lds0 + static_cast<uint32_t>(is * Cfg::STAGE) + Cfg::ABYTES, wv);
    is = is + 1 == Cfg::STAGES ? 0 : is + 1;
    if (left > 0) {
      --left;
      na += a_step;
      nb += b_step;
      ik += Cfg::BK;
      if (ik >= K) ik = 0, na += a_wrap, nb += b_wrap;
    }
  }
  __device__ __forceinline__ void issue() {
    issue_a();
    issue_b();
  }
};

// Tile order. Workgroup i runs on XCD i % 8, each XCD with its own L2, so
// XCD x takes a contiguous run of positions t (xcd_position) in a grouped
// order: kGroupRows tile rows at a time, column by column within the group.
// The workgroups running together on one XCD then share a few A row panels
// and a few B column panels instead of each bringing its own. grouped_tile
// returns the tile row and column of workgroup bid in a grid of nx columns and
// ny rows.
__device__ __forceinline__ int xcd_position(int bid, int total) {
  const int xcd = bid % 8, per = total / 8, extra = total % 8;
  return xcd * per + (xcd < extra ? xcd : extra) + bid / 8;
}
// Tile row and column of position t of an nx x ny grid in the grouped order.
__device__ __forceinline__ void grouped_order(int t, int nx, int ny, int& row, int& col) {
  constexpr int kGroupRows = 8;
  const int first_row = (t / (kGroupRows * nx)) * kGroupRows;
  const int rows = ny - first_row < kGroupRows ? ny - first_row : kGroupRows;
  const int local = t % (kGroupRows * nx);
  col = local / rows;
  row = first_row + local % rows;
}
__device__ __forceinline__ void grouped_tile(int bid, int nx, int ny, int& row, int& col) {
  grouped_order(xcd_position(bid, nx * ny), nx, ny, row, col);
}

// The slab pipeline of one workgroup: nslab slabs that the loader issues one
// after the other into STAGES LDS stages. Each wave waits only for its own
// loads of the slab it is about to read (vmcnt: exactly (STAGES - 2) * LPW
// younger loads are allowed), then a barrier makes every wave's loads of that
// slab visible and certifies that all waves have finished reading the
// previous slab, whose stage takes the next load. Fragments are
// double-buffered in registers: the reads of the next k step (the first step
// of the next slab, behind the barrier) are issued before the MFMAs of the
// current one, so LDS latency and the barrier overlap MFMA execution. The
// loads issued at a barrier are split: the A half right behind it, the B half
// after the MFMAs of the slab's first k step, so that the waves do not all
// queue at the load unit at once while the matrix cores wait (measured on
// MI355X: 13% fewer cycles per slab for the 256x256 tile).
// With TAIL, ck is the first k of the first slab within a contraction of
// length K (slabs wrap to k 0 past K), and a slab with fewer than BK valid k
// is zeroed past them in LDS before use. With RSUM, rs[i] also sums the A
// values the lane reads (StepFrags::rowsum). Returns with no direct load in
// flight.
template <class Cfg, bool AMC, bool BMC, bool TAIL, bool RSUM = false, class Loader>
__device__ __forceinline__ void run_slabs(Loader& ld, int nslab, int K, int ck, f32x16 (&acc)[Cfg::FM][Cfg::FN],
                                          int wm, int wn, int kw0, char* smem, float* rs = nullptr) {
  using Frags = StepFrags<Cfg, AMC, BMC>;
  constexpr int STEPS = Cfg::KW / Frags::KSTEP;
  static_assert(STEPS % 2 == 0, "a slab holds an even number of k steps");
  int cs = 0;  // stage of the slab being computed
  Frags fr[2];
  char* st = smem;
  if (nslab > 0) {
#pragma unroll
    for (int s = 0; s < Cfg::STAGES - 1; ++s) ld.issue();
    wait_vm<(Cfg::STAGES - 2) * Cfg::LPW>();
    lds_barrier();
    if (TAIL && K - ck < Cfg::BK) {
      fast_zero_tail<Cfg, Cfg::BM, AMC>(st, K - ck);
      fast_zero_tail<Cfg, Cfg::BN, BMC>(st + Cfg::ABYTES, K - ck);
      lds_barrier();
    }
    ld.issue_a();  // B half after the first k step below
    fr[0].load(st, wm, wn, kw0);
  }
  // all slabs but the last one: the last k step crosses into the next slab
  for (int q = 0; q < nslab - 1; ++q) {
#pragma unroll
    for (int s = 0; s < STEPS; ++s) {
      if (s + 1 < STEPS) {
        fr[(s + 1) & 1].load(st, wm, wn, kw0 + (s + 1) * Frags::KSTEP);
      } else {
        cs = cs + 1 == Cfg::STAGES ? 0 : cs + 1;
        if (TAIL) {
          ck += Cfg::BK;
          if (ck >= K) ck = 0;
        }
        st = smem + cs * Cfg::STAGE;
        wait_vm<(Cfg::STAGES - 2) * Cfg::LPW>();
        lds_barrier();  // slab q + 1 visible; slab q read by no wave any more
        if (TAIL && K - ck < Cfg::BK) {
          fast_zero_tail<Cfg, Cfg::BM, AMC>(st, K - ck);
          fast_zero_tail<Cfg, Cfg::BN, BMC>(st + Cfg::ABYTES, K - ck);
          lds_barrier();
        }
        ld.issue_a();  // into the stage of slab q; B half after the next slab's first k step
        fr[(s + 1) & 1].load(st, wm, wn, kw0);
      }
      fr[s & 1].mma(acc);
      if constexpr (RSUM) fr[s & 1].rowsum(*reinterpret_cast<float(*)[Cfg::FM]>(rs));
      if (s == 0) ld.issue_b();
    }
  }
  if (nslab > 0) {  // the last slab (a separate copy keeps the loop body's LDS waits exact)
#pragma unroll
    for (int s = 0; s < STEPS; ++s) {
      if (s + 1 < STEPS) fr[(s + 1) & 1].load(st, wm, wn, kw0 + (s + 1) * Frags::KSTEP);
      fr[s & 1].mma(acc);
      if constexpr (RSUM) fr[s & 1].rowsum(*reinterpret_cast<float(*)[Cfg::FM]>(rs));
      if (s == 0) ld.issue_b();
    }
  }
  wait_vm<0>();  // no direct load may still write LDS past this point
}

// Output of one wave's accumulator tile. Each block row of 32 rows passes
// through the wave's own LDS region in fp32 (epilogue applied on the way in),
// and every lane then writes 4 consecutive values of one output row (16 bytes
// fp32, 8 bytes bf16): a store instruction covers whole 128-byte lines instead
// of one element per lane. The ReLU gate of the layer below is read the same
// way. Falls back to element stores when the output rows are not contiguous
// or not aligned for those pieces. Called by all waves (it holds a barrier).
template <typename OutT, class Cfg, int EPI>
__device__ __forceinline__ void fast_store(const GemmArgs& g, f32x16 (&acc)[Cfg::FM][Cfg::FN], int m0, int n0,
                                           int wm, int wn, int64_t bz, int split, char* smem) {
  const bool part = g.splits > 1;
  const int64_t es = part ? 4 : static_cast<int64_t>(sizeof(OutT));
  const int64_t ld = part ? g.N : g.c.ld;
  char* base = part ? reinterpret_cast<char*>(g.partial + (bz * g.splits + split) * static_cast<int64_t>(g.M) * g.N)
                    : reinterpret_cast<char*>(static_cast<OutT*>(g.c.p) + bz * g.c.bstride);
  const char* gate = (!part && EPI == EPI_FWD && g.c.gate)
                         ? reinterpret_cast<const char*>(static_cast<const OutT*>(g.c.gate) + bz * g.c.bstride)
                         : nullptr;
  const int64_t piece = 4 * es;
  const bool vec = (part || (g.c.cidx == nullptr && g.c.col_stride <= 1 && g.c.ridx == nullptr)) &&
                   (ld * es) % piece == 0 && reinterpret_cast<uintptr_t>(base) % piece == 0 &&
                   reinterpret_cast<uintptr_t>(gate) % piece == 0;
  if (!vec) {
    store_tile<OutT, Cfg, EPI>(g, acc, m0, n0, wm, wn, bz, split);
    return;
  }
  // fp32 rows of TN values plus 32 bytes: the two half-waves' writes (rows r
  // and r + 4) then fall on disjoint banks
  constexpr int ROW = Cfg::TN * 4 + 32;
  constexpr int CPRW = Cfg::TN / 4;  // 16-byte pieces per row
  constexpr int RPI = 64 / CPRW;     // rows per read instruction
  // the bias of the wave's TM rows sits behind the staging regions
  static_assert(Cfg::NW * (32 * ROW + Cfg::TM * 4) <= Cfg::LDS, "epilogue staging exceeds LDS");
  lds_barrier();  // every wave is done with the stages
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int lr = lane & 31, lh = lane >> 5;
  char* region = smem + wave * 32 * ROW;
  const int m0w = m0 + wm * Cfg::TM, n0w = n0 + wn * Cfg::TN;
  // The bias entries of the wave's rows, loaded once with every load in
  // flight together (a load per accumulator row, each waited for before its
  // row's values are staged, cost ~4 us per call of a small product), then
  // read from LDS: the wave reads only what it wrote itself.
  const bool has_bias = !part && EPI == EPI_FWD && g.c.bias;
  float* bias_lds = reinterpret_cast<float*>(smem + Cfg::NW * 32 * ROW) + wave * Cfg::TM;
  if (has_bias) {
    float bv[(Cfg::TM + 63) / 64];
#pragma unroll
    for (int e = 0; e * 64 < Cfg::TM; ++e) {
      const int m = m0w + e * 64 + lane;
      bv[e] = (e * 64 + lane < Cfg::TM && m < g.M) ? g.c.bias[bias_row(g.c, m)] : 0.0f;
    }
#pragma unroll
    for (int e = 0; e * 64 < Cfg::TM; ++e)
      if (e * 64 + lane < Cfg::TM) bias_lds[e * 64 + lane] = bv[e];
  }
#pragma unroll
  for (int i = 0; i < Cfg::FM; ++i) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int rl = 8 * (r >> 2) + 4 * lh + (r & 3);
      const float bias = has_bias ? bias_lds[32 * i + rl] : 0.0f;
#pragma unroll
      for (int j = 0; j < Cfg::FN; ++j) {
        float v = acc[i][j][r];
        if (!part) v = epilogue<EPI>(g.c, v, bias);
        *reinterpret_cast<float*>(region + rl * ROW + (32 * j + lr) * 4) = v;
      }
    }
    // the ReLU gate of the rows this lane writes, every load issued before
    // the first store (the stores may alias the gate as far as the compiler
    // knows, so loads between them would each wait for the one before)
    typedef typename std::conditional<sizeof(OutT) == 2, uint2, f32x4>::type GateT;
    GateT gpre[32 / RPI];
    if (gate) {
#pragma unroll
      for (int t = 0; t < 32 / RPI; ++t) {
        const int rl = lane / CPRW + RPI * t, ch = lane % CPRW;
        const int m = m0w + 32 * i + rl, n = n0w + 4 * ch;
        if (m < g.M && n + 3 < g.N)
          gpre[t] = *reinterpret_cast<const GateT*>(reinterpret_cast<const OutT*>(gate) +
                                                    static_cast<int64_t>(m) * ld + n);
      }
    }
#pragma unroll
    for (int t = 0; t < 32 / RPI; ++t) {
      const int rl = lane / CPRW + RPI * t, ch = lane % CPRW;
      const f32x4 v = *reinterpret_cast<const f32x4*>(region + rl * ROW + ch * 16);
      const int m = m0w + 32 * i + rl, n = n0w + 4 * ch;
      if (m >= g.M) continue;
      const int64_t o = static_cast<int64_t>(m) * ld + n;
      if (part) {
        float* out = reinterpret_cast<float*>(base) + o;
        if (n + 3 < g.N) {
          *reinterpret_cast<f32x4*>(out) = v;
        } else {
          for (int e = 0; e < 4; ++e)
            if (n + e < g.N) out[e] = v[e];
        }
        continue;
      }
      OutT* out = reinterpret_cast<OutT*>(base) + o;
      const OutT* gt = gate ? reinterpret_cast<const OutT*>(gate) + o : nullptr;
      if (n + 3 < g.N) {
        OutT w[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) w[e] = from_f32<OutT>(v[e]);
        if (gt) {
          OutT gv[4];
          *reinterpret_cast<GateT*>(gv) = gpre[t];
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (!(to_f32(gv[e]) > 0.0f)) w[e] = from_f32<OutT>(0.0f);
        }
        if constexpr (sizeof(OutT) == 2)
          *reinterpret_cast<uint2*>(out) = *reinterpret_cast<const uint2*>(w);
        else
          *reinterpret_cast<f32x4*>(out) = *reinterpret_cast<const f32x4*>(w);
      } else {
        for (int e = 0; e < 4; ++e) {
          if (n + e >= g.N) break;
          float x = v[e];
          if (gt && !(to_f32(gt[e]) > 0.0f)) x = 0.0f;
          out[e] = from_f32<OutT>(x);
        }
      }
    }
  }
}

// Row sums of A (RSUM, see GemmArgs::rsum) for the tile row of a workgroup
// in tile column 0: lanes l and l + 32 of a wave hold the two k halves of
// row 32 i + l % 32, the waves of a k split are added in LDS in split order.
// One workgroup's output tile: position bid of an nx x ny tile grid in the
// grouped order, batch-and-split index bzs.
template <class Cfg, bool AMC, bool BMC, typename OutT, int EPI, bool RSUM = false>
__device__ __forceinline__ void fast_gemm_tile(const GemmArgs& g, int tile_row, int tile_col, int bzs, char* smem) {
  using T = typename Cfg::T;
  const int n0 = tile_col * Cfg::BN;
  const int m0 = tile_row * Cfg::BM;
  const int splits = g.splits > 1 ? g.splits : 1;
  const int64_t bz = splits > 1 ? bzs / splits : bzs;
  const int split = splits > 1 ? bzs % splits : 0;
  const int wave = threadIdx.x >> 6;
  const int ks = wave / (Cfg::WGM * Cfg::WGN);
  const int wmn = wave % (Cfg::WGM * Cfg::WGN);
  const int wm = wmn / Cfg::WGN, wn = wmn % Cfg::WGN;

  const T* abase = static_cast<const T*>(g.a.p) + bz * g.a.bstride;
  const T* bbase = static_cast<const T*>(g.b.p) + bz * g.b.bstride;

  f32x16 acc[Cfg::FM][Cfg::FN];
#pragma unroll
  for (int i = 0; i < Cfg::FM; ++i)
#pragma unroll
    for (int j = 0; j < Cfg::FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  const int nks = (g.K + Cfg::BK - 1) / Cfg::BK;
  const int kbatch = g.kbatch > 0 ? g.kbatch : 1;
  const int nslab = kbatch * nks;
  // slabs of this split (32-bit divisions: nslab * splits < 2^31; none without a split)
  int q0 = 0, q1 = nslab;
  if (splits > 1) {
    q0 = __builtin_amdgcn_readfirstlane(static_cast<int>(static_cast<uint32_t>(nslab * split) / splits));
    q1 = __builtin_amdgcn_readfirstlane(static_cast<int>(static_cast<uint32_t>(nslab * (split + 1)) / splits));
  }

  // slabs q0 .. q1 - 1 of this split
  SlabLoader<Cfg, AMC, BMC> ld;
  ld.wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  ld.lds0 = __builtin_amdgcn_readfirstlane(lds_addr(smem));
  static_assert(DmaSrc<Cfg, Cfg::BM, AMC>::PER_WAVE + DmaSrc<Cfg, Cfg::BN, BMC>::PER_WAVE == Cfg::LPW, "load count");
  if (q0 < q1) {
    ld.da.init(g.a.ld, m0, g.M, ld.wv);
    ld.db.init(g.b.ld, n0, g.N, ld.wv);
  }
  constexpr int ES = Cfg::ES;
  ld.K = g.K;
  ld.a_step = (AMC ? g.a.ld : 1) * Cfg::BK * ES;
  ld.b_step = (BMC ? g.b.ld : 1) * Cfg::BK * ES;
  ld.a_wrap = g.a.kbstride * ES - nks * ld.a_step;
  ld.b_wrap = g.b.kbstride * ES - nks * ld.b_step;
  const int ib = q0 == 0 ? 0 : q0 / (nks > 0 ? nks : 1);
  ld.ik = (q0 - ib * nks) * Cfg::BK;
  ld.is = 0;
  ld.left = q1 - q0 - 1;
  ld.na = uniform_ptr(reinterpret_cast<const char*>(abase) + (ib * g.a.kbstride) * ES + ld.ik / Cfg::BK * ld.a_step);
  ld.nb = uniform_ptr(reinterpret_cast<const char*>(bbase) + (ib * g.b.kbstride) * ES + ld.ik / Cfg::BK * ld.b_step);
  float rs[Cfg::FM];
#pragma unroll
  for (int i = 0; i < Cfg::FM; ++i) rs[i] = 0.0f;
  run_slabs<Cfg, AMC, BMC, true, RSUM>(ld, q1 - q0, g.K, ld.ik, acc, wm, wn, ks * Cfg::KW, smem, rs);
  const int rlane = threadIdx.x & 63;
  if constexpr (RSUM) {
#pragma unroll
    for (int i = 0; i < Cfg::FM; ++i) rs[i] += __shfl_xor(rs[i], 32);
  }
  const bool rs_out = RSUM && splits == 1 && tile_col == 0 && wn == 0 && rlane < 32;
  auto put_rsum = [&](int i, float v) {
    const int m = m0 + wm * Cfg::TM + 32 * i + rlane;
    if (m < g.M) g.rsum[bz * g.rsum_bstride + static_cast<int64_t>(m) * g.rsum_ld] = g.c.scale * v;
  };
  if constexpr (Cfg::KSPLIT == 1) {
    if (rs_out) {
#pragma unroll
      for (int i = 0; i < Cfg::FM; ++i) put_rsum(i, rs[i]);
    }
    fast_store<OutT, Cfg, EPI>(g, acc, m0, n0, wm, wn, bz, split, smem);
  } else {
    // the KSPLIT waves of one output tile reduce through LDS; wave ks finishes
    // the accumulator registers t (flattened over i, j, r) with t % KSPLIT == ks
    constexpr int NREG = Cfg::FM * Cfg::FN * 16;
    static_assert(Cfg::KSPLIT * Cfg::WGM * Cfg::WGN * NREG * 64 * 4 <= Cfg::LDS, "reduction buffer exceeds LDS");
    float* red = reinterpret_cast<float*>(smem);
    const int lane = threadIdx.x & 63;
    __syncthreads();
#pragma unroll
    for (int i = 0; i < Cfg::FM; ++i)
#pragma unroll
      for (int j = 0; j < Cfg::FN; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          red[((ks * Cfg::WGM * Cfg::WGN + wmn) * NREG + (i * Cfg::FN + j) * 16 + r) * 64 + lane] = acc[i][j][r];
    // row sums of the k splits after the accumulators: [KSPLIT][WGM][FM][32]
    float* rred = red + Cfg::KSPLIT * Cfg::WGM * Cfg::WGN * NREG * 64;
    if constexpr (RSUM) {
      static_assert((Cfg::KSPLIT * Cfg::WGM * Cfg::WGN * NREG * 64 + Cfg::KSPLIT * Cfg::WGM * Cfg::FM * 32) * 4 <=
                        Cfg::LDS,
                    "row-sum buffer exceeds LDS");
      if (wn == 0 && lane < 32) {
#pragma unroll
        for (int i = 0; i < Cfg::FM; ++i) rred[((ks * Cfg::WGM + wm) * Cfg::FM + i) * 32 + lane] = rs[i];
      }
    }
    __syncthreads();
    if (rs_out && ks == 0) {
#pragma unroll
      for (int i = 0; i < Cfg::FM; ++i) {
        float v = 0.0f;
#pragma unroll
        for (int u = 0; u < Cfg::KSPLIT; ++u) v += rred[((u * Cfg::WGM + wm) * Cfg::FM + i) * 32 + lane];
        put_rsum(i, v);
      }
    }
    const int lr = lane & 31, lh = lane >> 5;
#pragma unroll
    for (int t = ks; t < NREG; t += Cfg::KSPLIT) {
      const int i = t / (Cfg::FN * 16), j = (t / 16) % Cfg::FN, r = t % 16;
      float v = 0.0f;
#pragma unroll
      for (int u = 0; u < Cfg::KSPLIT; ++u) v += red[((u * Cfg::WGM * Cfg::WGN + wmn) * NREG + t) * 64 + lane];
      const int m = m0 + wm * Cfg::TM + 32 * i + 8 * (r >> 2) + 4 * lh + (r & 3);
      const int n = n0 + wn * Cfg::TN + 32 * j + lr;
      if (m >= g.M || n >= g.N) continue;
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
}

// The grid is nx x ny output tiles times nz (batch entries times k splits).
// When every z-slice reads its own operands (a split contraction, or a batch
// with no operand shared between entries), XCD positions run over the whole
// grid, z-major: a z-slice goes to as few XCDs as possible, so that the
// workgroups on one XCD share the A and B panels of one slice (split z on
// XCD z when the tiles of a slice are a multiple of 8) instead of each XCD
// holding a few tiles of every slice. When an operand is shared by the batch
// entries (batch stride 0), positions run within each slice: XCD x then holds
// the same tiles of every entry and the shared panels stay in its L2.
template <class Cfg, bool AMC, bool BMC, typename OutT, int EPI, bool RSUM = false>
__global__ void __launch_bounds__(Cfg::NT) fast_gemm_kernel(GemmArgs g) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int nx = gridDim.x, ny = gridDim.y, nxy = nx * ny;
  int tile_row, tile_col, z;
  if (gridDim.z > 1 && g.splits <= 1 && (g.a.bstride == 0 || g.b.bstride == 0)) {
    grouped_tile(blockIdx.y * nx + blockIdx.x, nx, ny, tile_row, tile_col);
    z = blockIdx.z;
  } else {
    const int bid = (blockIdx.z * ny + blockIdx.y) * nx + blockIdx.x;
    const int t = xcd_position(bid, nxy * gridDim.z);
    grouped_order(t % nxy, nx, ny, tile_row, tile_col);
    z = t / nxy;
  }
  fast_gemm_tile<Cfg, AMC, BMC, OutT, EPI, RSUM>(g, tile_row, tile_col, z, smem);
}

// Two independent GEMMs of one configuration in one launch (no batch, no k
// split): the first workgroups take the tiles of g1, the rest those of g2.
// One launch instead of two saves a kernel's fixed start and drain time, and
// two problems too small to fill the chip alone run side by side.
template <class Cfg, bool AMC1, bool BMC1, typename OutT1, int EPI1, bool RSUM1, bool AMC2, bool BMC2,
          typename OutT2, int EPI2, bool RSUM2>
__global__ void __launch_bounds__(Cfg::NT) fast_gemm_pair_kernel(GemmArgs g1, GemmArgs g2) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int nx1 = (g1.N + Cfg::BN - 1) / Cfg::BN, ny1 = (g1.M + Cfg::BM - 1) / Cfg::BM;
  const int b = static_cast<int>(blockIdx.x);
  int row, col;
  if (b < nx1 * ny1) {
    grouped_tile(b, nx1, ny1, row, col);
    fast_gemm_tile<Cfg, AMC1, BMC1, OutT1, EPI1, RSUM1>(g1, row, col, 0, smem);
  } else {
    const int nx2 = (g2.N + Cfg::BN - 1) / Cfg::BN, ny2 = (g2.M + Cfg::BM - 1) / Cfg::BM;
    grouped_tile(b - nx1 * ny1, nx2, ny2, row, col);
    fast_gemm_tile<Cfg, AMC2, BMC2, OutT2, EPI2, RSUM2>(g2, row, col, 0, smem);
  }
}

// Whether a problem can run on fast_gemm_kernel with operand A m-contiguous
// (AMC) or not, B n-contiguous (BMC) or not: every operand is a plain strided
// view read in whole 16-byte chunks, and every chunk of a slab lies less than
// 2^31 bytes past the slab's first element (the lanes' 32-bit load offsets;
// the slab base itself is a 64-bit pointer). A slab of a k-contiguous operand
// spans rows 0 .. ext - 1 of ld elements, BK <= 256 k each; one of an
// m/n-contiguous operand spans at most 256 k-rows of ld elements and columns
// 0 .. ext - 1.
template <bool AMC, bool BMC>
inline bool fast_ok(const GemmArgs& g, size_t esize) {
  const int64_t epc = static_cast<int64_t>(16 / esize);
  auto ok = [epc, esize](const GemmOperand& o, int ext, bool mc) {
    const int64_t e = ext > 0 ? ext : 1;
    const int64_t span = mc ? e + 256 * o.ld : (e - 1) * o.ld + 256;
    return o.ridx == nullptr && o.cidx == nullptr && o.y == nullptr && o.ld % epc == 0 && o.bstride % epc == 0 &&
           o.kbstride % epc == 0 && (reinterpret_cast<uintptr_t>(o.p) & 15u) == 0 && o.ld >= 0 &&
           span * static_cast<int64_t>(esize) < (int64_t{1} << 31);
  };
  return ok(g.a, g.M, AMC) && ok(g.b, g.N, BMC);
}

// Configurations: large tiles for large grids, 32x32 tiles with the k of each
// slab split over the waves (4 for bf16, 8 for fp32) for small grids.
template <typename T>
struct FastCfgs;
template <>
struct FastCfgs<bf16> {
  using Huge = FastCfg<bf16, 256, 256, 64, 2, 2, 4, 1>;   // 128 KB LDS, 8 waves (2 per SIMD)
  using Wide = FastCfg<bf16, 128, 256, 32, 4, 2, 4, 1>;   // 96 KB, 8 waves
  using Tall = FastCfg<bf16, 256, 128, 32, 4, 4, 2, 1>;   // 96 KB, 8 waves
  using Big = FastCfg<bf16, 128, 128, 64, 3, 2, 2, 1>;    // 96 KB
  using Small = FastCfg<bf16, 32, 32, 128, 4, 1, 1, 4>;   // 64 KB
};
template <>
struct FastCfgs<float> {
  using Huge = FastCfg<float, 128, 128, 32, 4, 2, 4, 1>;  // 128 KB, 8 waves
  using Wide = Huge;
  using Tall = Huge;
  using Big = FastCfg<float, 64, 64, 64, 3, 2, 2, 2>;     // 96 KB, 8 waves on 32-deep k shares
  using Narrow = FastCfg<float, 128, 32, 32, 4, 2, 1, 2>; // 80 KB, 4 waves on 16-deep k shares
  using Small = FastCfg<float, 32, 32, 128, 4, 1, 1, 8>;  // 128 KB, 8 waves on 16-deep k shares
};

enum FastKind { FAST_HUGE, FAST_WIDE, FAST_TALL, FAST_BIG, FAST_SMALL, FAST_NARROW };

struct FastPlan {
  int kind;    // FastKind
  int splits;  // workgroups per output tile along K (partials reduced by a second kernel)
};

// Split count s for a tile count: the largest power of two that keeps the grid
// within one round of the chip and every split at least kMinSlabsPerSplit slabs.
inline int fast_splits(int64_t tiles, int64_t slabs) {
  int s = 1;
  while (tiles * s * 2 <= kTargetBlocks && slabs / (s * 2) >= kMinSlabsPerSplit && s * 2 <= kMaxSplits) s *= 2;
  return s;
}

// fp32: the largest tile that the output fills along both sides and whose
// grid still covers 5/8 of the chip, then split-K.
inline FastPlan plan_fast_f32(int M, int N, int K, int kbatch, int batch) {
  using C = FastCfgs<float>;
  auto tiles_of = [&](int bm, int bn) {
    return static_cast<int64_t>((M + bm - 1) / bm) * ((N + bn - 1) / bn) * batch;
  };
  FastPlan p;
  int bk;
  int64_t tiles;
  const int64_t kb = kbatch > 0 ? kbatch : 1;
  // at most 32 columns (an LSTM's per-step products at a small batch): 128 x
  // 32 tiles, so that most of each tile is not zero padding of the columns
  if (N <= C::Narrow::BN && tiles_of(C::Narrow::BM, C::Narrow::BN) >= kTargetBlocks * 5 / 8) {
    p.kind = FAST_NARROW;
    tiles = tiles_of(C::Narrow::BM, C::Narrow::BN);
    p.splits = kb * K >= 8192 ? fast_splits(tiles, kb * ((K + C::Narrow::BK - 1) / C::Narrow::BK)) : 1;
    return p;
  }
  if (M > C::Big::BM && N > C::Big::BN && tiles_of(C::Huge::BM, C::Huge::BN) >= kTargetBlocks * 5 / 8) {
    p.kind = FAST_HUGE;
    bk = C::Huge::BK;
    tiles = tiles_of(C::Huge::BM, C::Huge::BN);
  } else if (tiles_of(C::Big::BM, C::Big::BN) >= kTargetBlocks * 5 / 8) {
    p.kind = FAST_BIG;
    bk = C::Big::BK;
    tiles = tiles_of(C::Big::BM, C::Big::BN);
  } else {
    p.kind = FAST_SMALL;
    bk = C::Small::BK;
    tiles = tiles_of(C::Small::BM, C::Small::BN);
  }
  const int64_t slabs = kb * ((K + bk - 1) / bk);
  if (p.kind == FAST_SMALL) {
    // A 32x32 workgroup takes about 0.9 us per 128-deep slab however many run
    // beside it (measured on MI355X), so a long contraction over few tiles is
    // a serial chain: split it over more workgroups (up to one round of the
    // chip) when that saves more than the partial-sum round trip and the
    // reduction launch cost (about 3 us).
    double best_t = 0.9 * static_cast<double>(slabs);
    p.splits = 1;
    for (int s = 2; s <= kMaxSplits && tiles * s <= kTargetBlocks && slabs >= s; s *= 2) {
      const double t = 0.9 * static_cast<double>((slabs + s - 1) / s) + 3.0;
      if (t < best_t) {
        best_t = t;
        p.splits = s;
      }
    }
    return p;
  }
  // larger tiles: split-K pays for its partial-sum round trip and reduction
  // launch only on long contractions (measured on MI355X: never below K = 2048)
  p.splits = kb * K >= 8192 ? fast_splits(tiles, slabs) : 1;
  return p;
}

// bf16: the (configuration, split) pair with the smallest modelled time. A
// workgroup's time is its MFMA work (whole tiles and slabs) over the rate one
// workgroup of that configuration reaches with the chip full (measured on
// MI355X), somewhat faster when fewer workgroups than compute units share the
// chip; workgroups beyond the first 256 run in further rounds; a split adds
// the partial-sum round trip and its reduction launch.
inline FastPlan plan_fast_bf16(int M, int N, int K, int kbatch, int batch) {
  using C = FastCfgs<bf16>;
  struct Cand {
    int kind, bm, bn, bk;
    double rate;  // flop/s per workgroup with 256 workgroups resident
  };
  static const Cand cands[] = {
      {FAST_HUGE, C::Huge::BM, C::Huge::BN, C::Huge::BK, 4.2e12},
      {FAST_WIDE, C::Wide::BM, C::Wide::BN, C::Wide::BK, 3.5e12},
      {FAST_TALL, C::Tall::BM, C::Tall::BN, C::Tall::BK, 3.4e12},
      {FAST_BIG, C::Big::BM, C::Big::BN, C::Big::BK, 2.7e12},
      {FAST_SMALL, C::Small::BM, C::Small::BN, C::Small::BK, 0.5e12},
  };
  const int64_t kb = kbatch > 0 ? kbatch : 1;
  FastPlan best = {FAST_SMALL, 1};
  double best_t = 1e300;
  for (const Cand& c : cands) {
    const int64_t tiles = static_cast<int64_t>((M + c.bm - 1) / c.bm) * ((N + c.bn - 1) / c.bn) * batch;
    const int64_t slabs = kb * ((K + c.bk - 1) / c.bk);
    for (int s = 1; s <= kMaxSplits; s *= 2) {
      if (s > 1 && (slabs / s < kMinSlabsPerSplit || tiles * s > 2 * kTargetBlocks)) break;
      const int64_t wgs = tiles * s;
      const int64_t rounds = (wgs + kTargetBlocks - 1) / kTargetBlocks;
      const double occ = wgs < kTargetBlocks ? static_cast<double>(wgs) / kTargetBlocks : 1.0;
      const double rate = c.rate * (1.0 + 0.3 * (1.0 - occ));
      const double work = 2.0 * c.bm * c.bn * c.bk * ((slabs + s - 1) / s);
      double t = rounds * work / rate;
      if (s > 1) t += 4.0 * M * N * batch * (s + 1) / 5e12 + 3e-6;
      if (t < best_t) {
        best_t = t;
        best = {c.kind, s};
      }
    }
  }
  return best;
}

template <typename T>
inline FastPlan plan_fast(int M, int N, int K, int kbatch, int batch) {
  if constexpr (sizeof(T) == 2)
    return plan_fast_bf16(M, N, K, kbatch, batch);
  else
    return plan_fast_f32(M, N, K, kbatch, batch);
}

template <typename T>
inline size_t fast_partial_floats(int M, int N, int K, int kbatch, int batch) {
  const FastPlan p = plan_fast<T>(M, N, K, kbatch, batch);
  return p.splits > 1 ? static_cast<size_t>(p.splits) * batch * M * N : 0;
}

template <class Cfg, bool AMC, bool BMC, typename OutT, int EPI, bool RSUM = false>
inline hipError_t launch_fast(const GemmArgs& g, int batch, hipStream_t stream) {
  const int splits = g.splits > 1 ? g.splits : 1;
  auto kern = fast_gemm_kernel<Cfg, AMC, BMC, OutT, EPI, RSUM>;
  // per instantiation, once (thread-safe static initialisation): allow more than 64 KB of dynamic LDS
  static const hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                                     hipFuncAttributeMaxDynamicSharedMemorySize, Cfg::LDS);
  if (attr != hipSuccess) return attr;
  dim3 grid((g.N + Cfg::BN - 1) / Cfg::BN, (g.M + Cfg::BM - 1) / Cfg::BM, batch * splits);
  hipLaunchKernelGGL(kern, grid, dim3(Cfg::NT), Cfg::LDS, stream, g);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || splits == 1) return e;
  const int64_t mn = static_cast<int64_t>(g.M) * g.N;
  if (reduce4_ok<OutT>(g)) {
    hipLaunchKernelGGL((splitk_reduce4_kernel<OutT, EPI>), dim3(static_cast<unsigned>((mn / 4 + 255) / 256), batch),
                       dim3(256), 0, stream, g);
  } else {
    hipLaunchKernelGGL((splitk_reduce_kernel<OutT, EPI>), dim3(static_cast<unsigned>((mn + 255) / 256), batch),
                       dim3(256), 0, stream, g);
  }
  return hipGetLastError();
}

// Launches g1 and g2 (both fast_ok, splits 1, no batch) as one grid of
// fast_gemm_pair_kernel on the 32x32 configuration of T.
template <typename T, bool AMC1, bool BMC1, typename OutT1, int EPI1, bool RSUM1, bool AMC2, bool BMC2,
          typename OutT2, int EPI2, bool RSUM2>
inline hipError_t launch_fast_pair(GemmArgs g1, GemmArgs g2, hipStream_t stream) {
  using Cfg = typename FastCfgs<T>::Small;
  auto kern = fast_gemm_pair_kernel<Cfg, AMC1, BMC1, OutT1, EPI1, RSUM1, AMC2, BMC2, OutT2, EPI2, RSUM2>;
  static const hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                                     hipFuncAttributeMaxDynamicSharedMemorySize, Cfg::LDS);
  if (attr != hipSuccess) return attr;
  g1.splits = g2.splits = 1;
  if (!RSUM1) g1.rsum = nullptr;
  if (!RSUM2) g2.rsum = nullptr;
  const int64_t n1 = static_cast<int64_t>((g1.N + Cfg::BN - 1) / Cfg::BN) * ((g1.M + Cfg::BM - 1) / Cfg::BM);
  const int64_t n2 = static_cast<int64_t>((g2.N + Cfg::BN - 1) / Cfg::BN) * ((g2.M + Cfg::BM - 1) / Cfg::BM);
  if (n1 + n2 == 0) return hipSuccess;
  hipLaunchKernelGGL(kern, dim3(static_cast<unsigned>(n1 + n2)), dim3(Cfg::NT), Cfg::LDS, stream, g1, g2);
  return hipGetLastError();
}

// Whether two problems run as one fast_gemm_pair_kernel launch: both take the
// 32x32 configuration without a k split on their own, and each has a tile.
template <typename T>
inline bool fast_pair_ok(const GemmArgs& g1, const GemmArgs& g2) {
  if (g1.M <= 0 || g1.N <= 0 || g2.M <= 0 || g2.N <= 0) return false;
  const FastPlan p1 = plan_fast<T>(g1.M, g1.N, g1.K, 1, 1), p2 = plan_fast<T>(g2.M, g2.N, g2.K, 1, 1);
  return p1.kind == FAST_SMALL && p2.kind == FAST_SMALL && p1.splits == 1 && p2.splits == 1;
}

template <typename T, bool AMC, bool BMC, typename OutT, int EPI, bool RSUM>
inline hipError_t launch_planned(const GemmArgs& g, int kind, int batch, hipStream_t stream) {
  using C = FastCfgs<T>;
  switch (kind) {
    case FAST_HUGE:
      // the bf16 256x256 tile has no registers left for row sums (it spills)
      if constexpr (RSUM && sizeof(T) == 2) return hipErrorNotSupported;
      else return launch_fast<typename C::Huge, AMC, BMC, OutT, EPI, RSUM>(g, batch, stream);
    case FAST_WIDE:
      return launch_fast<typename C::Wide, AMC, BMC, OutT, EPI, RSUM>(g, batch, stream);
    case FAST_TALL:
      return launch_fast<typename C::Tall, AMC, BMC, OutT, EPI, RSUM>(g, batch, stream);
    case FAST_BIG:
      return launch_fast<typename C::Big, AMC, BMC, OutT, EPI, RSUM>(g, batch, stream);
    case FAST_NARROW:  // fp32 only
      if constexpr (sizeof(T) == 4) return launch_fast<typename C::Narrow, AMC, BMC, OutT, EPI, RSUM>(g, batch, stream);
      else return hipErrorNotSupported;
    default:
      return launch_fast<typename C::Small, AMC, BMC, OutT, EPI, RSUM>(g, batch, stream);
  }
}

// Runs a GEMM on the fast kernel; the caller has checked fast_ok(). With
// RSUM, g.rsum receives the row sums of A when the plan has no k split and is
// not the bf16 256x256 tile, and *rsum_done says whether it did (else the
// caller computes them itself).
template <typename T, bool AMC, bool BMC, typename OutT, int EPI, bool RSUM = false>
inline hipError_t run_fast_gemm(GemmArgs g, int batch, hipStream_t stream, float* partial,
                                bool* rsum_done = nullptr) {
  if (rsum_done) *rsum_done = false;
  if (g.M <= 0 || g.N <= 0 || batch <= 0) return hipSuccess;
  FastPlan p = plan_fast<T>(g.M, g.N, g.K, g.kbatch, batch);
  // the kernel splits the slabs with 32-bit arithmetic
  const int64_t kb = g.kbatch > 0 ? g.kbatch : 1;
  if (!partial || kb * (g.K / 32 + 1) * p.splits >= int64_t{1} << 31) p.splits = 1;
  g.splits = p.splits;
  g.partial = partial;
  if (RSUM && g.rsum && p.splits == 1 && !(sizeof(T) == 2 && p.kind == FAST_HUGE)) {
    if (rsum_done) *rsum_done = true;
    return launch_planned<T, AMC, BMC, OutT, EPI, RSUM>(g, p.kind, batch, stream);
  }
  g.rsum = nullptr;
  return launch_planned<T, AMC, BMC, OutT, EPI, false>(g, p.kind, batch, stream);
}

}  // namespace ard
