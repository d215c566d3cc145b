// Tile-based dropout pattern (Sec. III-B): compaction of the kept-tile bitmap
// into gather lists, and the layer's fwd / bwd_data / bwd_weight on kept tiles.
//
// Sec. III-B fetches only non-dropped tiles and lets each processing element
// multiply one tile pair. Here a workgroup owns one tile row (fwd) or one tile
// column (bwd_data) of W and one block of the batch, and walks that row's
// (column's) list of kept tiles: each kept tile is one slab of the direct-load
// pipeline of the fast GEMM, its base taken from the list. bwd_weight runs one
// workgroup per group of up to kTdpChunk kept tiles of one tile row, which
// share their dY rows; the X rows of the group's tiles are gathered through
// the lanes' load offsets. Dropped tiles are never read or computed.

#include <hip/hip_runtime.h>

#include "ard_gemm.hpp"
#include "ard_gemm_fast.hpp"
#include "ard_internal.hpp"

namespace ard {

constexpr int kScanThreads = 1024;
constexpr int kMaxTileDim = 4096;    // tiles per side handled by the scan kernel
constexpr int kLdsBitWords = 2048;   // bitmaps of up to 65536 tiles are scanned from LDS
constexpr int kTdpChunk = 4;         // kept tiles of one tile row per bwd_weight workgroup
constexpr int kTdpRec = 4 + kTdpChunk;  // ints per bwd_weight group record

// Exclusive prefix sum of one value per thread over the workgroup (wave scans
// by shuffles, then the 16 wave totals). Returns the prefix; total receives
// the sum of all values. wsum: kScanThreads / 64 + 1 entries of LDS.
__device__ int32_t block_prefix(int32_t v, int32_t* wsum, int32_t& total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  constexpr int kWaves = kScanThreads / 64;
  int32_t inc = v;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int32_t t = __shfl_up(inc, d, 64);
    if (lane >= d) inc += t;
  }
  if (lane == 63) wsum[wave] = inc;
  __syncthreads();
  if (wave == 0) {  // the wave totals, scanned by the first kWaves lanes
    const int32_t x = lane < kWaves ? wsum[lane] : 0;
    int32_t y = x;
#pragma unroll
    for (int d = 1; d < kWaves; d <<= 1) {
      const int32_t t = __shfl_up(y, d, 64);
      if (lane >= d) y += t;
    }
    if (lane < kWaves) wsum[lane] = y - x;
    if (lane == kWaves - 1) wsum[kWaves] = y;
  }
  __syncthreads();
  const int32_t out = wsum[wave] + inc - v;
  total = wsum[kWaves];
  __syncthreads();  // wsum may be reused right away
  return out;
}

// Exclusive scan of cnt[0..n) (LDS, n >= 1), each thread summing a contiguous
// run of entries: writes the n + 1 prefix sums to out (if not NULL), leaves
// the exclusive prefix in cnt and returns the total. Up to 1024 entries the
// first wave scans alone (16 entries per lane at most, shuffles, one barrier):
// the block-wide version costs four barriers of all 16 waves.
__device__ int32_t block_exclusive_scan(int32_t* cnt, int n, int32_t* out, int32_t* wsum) {
  const int tid = threadIdx.x;
  if (n <= 1024) {
    if (tid < 64) {
      const int per = (n + 63) / 64;
      const int lo = min(n, tid * per), hi = min(n, lo + per);
      int32_t v = 0;
      for (int i = lo; i < hi; ++i) v += cnt[i];
      int32_t inc = v;
#pragma unroll
      for (int d = 1; d < 64; d <<= 1) {
        const int32_t t = __shfl_up(inc, d, 64);
        if (tid >= d) inc += t;
      }
      int32_t run = inc - v;
      for (int i = lo; i < hi; ++i) {
        const int32_t c = cnt[i];
        if (out) out[i] = run;
        cnt[i] = run;
        run += c;
      }
      if (tid == 63) {
        wsum[0] = inc;
        if (out) out[n] = inc;
      }
    }
    __syncthreads();
    const int32_t total = wsum[0];
    __syncthreads();  // wsum may be reused right away
    return total;
  }
  const int per = (n + kScanThreads - 1) / kScanThreads;
  const int lo = min(n, tid * per), hi = min(n, lo + per);
  int32_t s = 0;
  for (int i = lo; i < hi; ++i) s += cnt[i];
  int32_t total;
  int32_t run = block_prefix(s, wsum, total);
  for (int i = lo; i < hi; ++i) {
    const int32_t c = cnt[i];
    if (out) out[i] = run;
    cnt[i] = run;  // the prefix stays in LDS for the list-writing pass
    run += c;
  }
  if (out && tid == 0) out[n] = total;
  __syncthreads();
  return total;
}

// Bitmap words, from LDS when the bitmap was staged there.
struct BitSrc {
  const uint32_t* g;
  const uint32_t* s;
  __device__ __forceinline__ uint32_t word(int64_t w) const { return s ? s[w] : g[w]; }
  __device__ __forceinline__ bool bit(int64_t t) const { return (word(t >> 5) >> (t & 31)) & 1u; }
  // the bits of word w that lie in [lo, hi)
  __device__ __forceinline__ uint32_t masked(int64_t w, int64_t lo, int64_t hi) const {
    uint32_t x = word(w);
    const int64_t b0 = w * 32;
    if (lo > b0) x &= ~0u << (lo - b0);
    if (hi < b0 + 32) x &= (hi - b0 <= 0) ? 0u : (~0u >> (32 - (hi - b0)));
    return x;
  }
  __device__ __forceinline__ int32_t count(int64_t lo, int64_t hi) const {
    int32_t c = 0;
    if (hi <= lo) return 0;
    for (int64_t w = lo >> 5; w <= (hi - 1) >> 5; ++w) c += __popc(masked(w, lo, hi));
    return c;
  }
};

__device__ __forceinline__ bool tile_bit(const uint32_t* bits, int64_t t) {
  return (bits[t >> 5] >> (t & 31)) & 1u;
}

// Draw t (0-based) of the SplitMix64 stream with start state s0 (Steele, Lea
// & Flood, OOPSLA 2014): the Weyl state after t + 1 golden-ratio steps, put
// through the 64-bit finaliser. The host sampler walks the same sequence one
// draw after the other; here every tile computes its own draw.
__device__ __forceinline__ uint64_t splitmix_draw(uint64_t s0, uint64_t t) {
  uint64_t z = s0 + (t + 1) * 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// Keep-bitmap sampling of the plan kernel: tile t is kept iff its draw as a
// 53-bit uniform in [0, 1) is >= p.
struct TileSampler {
  int enabled;
  double p;
  uint64_t s0;
};

// One workgroup: bitmap -> row_ptr/row_cols (CSR), col_ptr/col_rows (CSC),
// flat, and the bwd_weight groups: the groups of a row take its kept tiles
// kTdpChunk at a time, in row order. chunks[0] = their number (chunks[1..3]
// = 0); group c is the record at chunks + 4 + c * kTdpRec: tile row, first
// position in row_cols, tile count n, 0, then the n tile columns followed by
// the last one repeated up to kTdpChunk entries.
// Small bitmaps are staged in LDS together with their transpose (built with
// LDS atomics while the rows are listed), so both list passes walk whole words
// (popcount, find-first-set); larger ones are read bit by bit from memory.
__global__ void __launch_bounds__(kScanThreads)
    plan_tiles_kernel(uint32_t* bits, TileSampler smp, int32_t tiles_n, int32_t tiles_k,
                      int32_t* __restrict__ row_ptr, int32_t* __restrict__ row_cols,
                      int32_t* __restrict__ col_ptr, int32_t* __restrict__ col_rows,
                      int32_t* __restrict__ flat, int32_t* __restrict__ chunks) {
  __shared__ int32_t cnt[kMaxTileDim];   // per row, then per column: count, then exclusive prefix
  __shared__ int32_t gpre[kMaxTileDim];  // per row: groups, then their exclusive prefix
  __shared__ int32_t wsum[kScanThreads / 64 + 1];
  __shared__ uint32_t sbits[kLdsBitWords];
  __shared__ uint32_t tbits[kLdsBitWords];  // column c, rows 32w .. 32w + 31 at word c * wpc + w
  __shared__ int32_t wpre[kLdsBitWords];    // set bits before each word of sbits, then of tbits
  const int tid = threadIdx.x;
  const int64_t nbits = static_cast<int64_t>(tiles_n) * tiles_k;
  const int64_t nwords = (nbits + 31) / 32;
  const int wpc = (tiles_n + 31) / 32;
  const bool in_lds = nwords <= kLdsBitWords && static_cast<int64_t>(tiles_k) * wpc <= kLdsBitWords;
  if (smp.enabled) {  // sample the bitmap first (written out, and kept in LDS when it fits)
    const int lane = tid & 63, wave = tid >> 6;
    for (int64_t base = 0; base < nbits; base += kScanThreads) {
      const int64_t t = base + tid;
      bool keep = false;
      if (t < nbits)
        keep = static_cast<double>(splitmix_draw(smp.s0, static_cast<uint64_t>(t)) >> 11) * 0x1.0p-53 >= smp.p;
      const uint64_t m = __ballot(keep);  // the wave's 64 consecutive tiles, two words
      const int64_t w0 = (base + 64 * wave) / 32;
      if (lane < 2 && w0 + lane < nwords) {
        const uint32_t x = static_cast<uint32_t>(m >> (32 * lane));
        bits[w0 + lane] = x;
        if (in_lds) sbits[w0 + lane] = x;
      }
    }
    __syncthreads();
  }
  BitSrc src = {bits, nullptr};
  if (in_lds) {
    if (!smp.enabled)
      for (int w = tid; w < nwords; w += kScanThreads) sbits[w] = bits[w];
    for (int w = tid; w < tiles_k * wpc; w += kScanThreads) tbits[w] = 0u;
    src.s = sbits;
    __syncthreads();
  }
  // rows: counts, groups, prefixes
  for (int r = tid; r < tiles_n; r += kScanThreads) {
    const int32_t kept = src.count(static_cast<int64_t>(r) * tiles_k, static_cast<int64_t>(r + 1) * tiles_k);
    cnt[r] = kept;
    gpre[r] = (kept + kTdpChunk - 1) / kTdpChunk;
  }
  __syncthreads();
  const int32_t total = block_exclusive_scan(cnt, tiles_n, row_ptr, wsum);
  const int32_t groups = block_exclusive_scan(gpre, tiles_n, nullptr, wsum);
  if (tid < 4) chunks[tid] = tid == 0 ? groups : 0;
  if (in_lds) {
    // rows, one thread per tile: kept tile t of word w lands at position
    // (set bits before word w) + (set bits of word w below t)
    for (int w = tid; w < nwords; w += kScanThreads) wpre[w] = __popc(sbits[w]);
    __syncthreads();
    block_exclusive_scan(wpre, static_cast<int>(nwords), nullptr, wsum);
    for (int t = tid; t < nbits; t += kScanThreads) {
      const int w = t >> 5, b = t & 31;
      const uint32_t x = sbits[w];
      if (!((x >> b) & 1u)) continue;
      const int32_t pos = wpre[w] + __popc(x & ((1u << b) - 1u));
      const int r = t / tiles_k;
      const int32_t col = t - r * tiles_k;
      row_cols[pos] = col;
      flat[pos] = t;
      atomicOr(&tbits[col * wpc + (r >> 5)], 1u << (r & 31));
      const int32_t rank = pos - cnt[r];
      const int32_t kept = (r + 1 < tiles_n ? cnt[r + 1] : total) - cnt[r];
      int32_t* rec = chunks + 4 + static_cast<int64_t>(gpre[r] + rank / kTdpChunk) * kTdpRec;
      const int slot = rank % kTdpChunk;
      if (slot == 0) {
        rec[0] = r;
        rec[1] = pos;
        rec[2] = kept - rank < kTdpChunk ? kept - rank : kTdpChunk;
        rec[3] = 0;
      }
      rec[4 + slot] = col;
      if (rank == kept - 1)  // the row's last tile pads its group
        for (int i = slot + 1; i < kTdpChunk; ++i) rec[4 + i] = col;
    }
    __syncthreads();
    // columns, one thread per bit of the transpose (column-major words, so the
    // positions run in column order)
    const int ntw = tiles_k * wpc;
    for (int w = tid; w < ntw; w += kScanThreads) wpre[w] = __popc(tbits[w]);
    __syncthreads();
    block_exclusive_scan(wpre, ntw, nullptr, wsum);
    for (int k = tid; k < tiles_k; k += kScanThreads) col_ptr[k] = wpre[k * wpc];
    if (tid == 0) col_ptr[tiles_k] = total;
    for (int u = tid; u < ntw * 32; u += kScanThreads) {
      const int w = u >> 5, b = u & 31;
      const uint32_t x = tbits[w];
      if ((x >> b) & 1u) col_rows[wpre[w] + __popc(x & ((1u << b) - 1u))] = 32 * (w % wpc) + b;
    }
    return;
  }
  // rows: lists and group records (bitmap in memory)
  for (int r = tid; r < tiles_n; r += kScanThreads) {
    const int32_t first = cnt[r];
    int32_t pos = first, last = 0;
    const int64_t lo = static_cast<int64_t>(r) * tiles_k, hi = lo + tiles_k;
    for (int64_t w = lo >> 5; w <= (hi - 1) >> 5; ++w) {
      uint32_t x = src.masked(w, lo, hi);
      while (x) {
        const int64_t t = w * 32 + (__ffs(x) - 1);
        const int32_t col = static_cast<int32_t>(t - lo);
        row_cols[pos] = col;
        flat[pos] = static_cast<int32_t>(t);
        const int32_t rank = pos - first;
        int32_t* rec = chunks + 4 + static_cast<int64_t>(gpre[r] + rank / kTdpChunk) * kTdpRec;
        if (rank % kTdpChunk == 0) {
          rec[0] = r;
          rec[1] = pos;
          rec[3] = 0;
        }
        rec[4 + rank % kTdpChunk] = col;
        last = col;
        ++pos;
        x &= x - 1;
      }
    }
    const int32_t kept = pos - first;
    for (int32_t g = 0; g * kTdpChunk < kept; ++g) {
      int32_t* rec = chunks + 4 + static_cast<int64_t>(gpre[r] + g) * kTdpRec;
      const int32_t n = kept - g * kTdpChunk < kTdpChunk ? kept - g * kTdpChunk : kTdpChunk;
      rec[2] = n;
      for (int i = n; i < kTdpChunk; ++i) rec[4 + i] = last;  // only the row's last group is short
    }
  }
  __syncthreads();
  // columns
  for (int k = tid; k < tiles_k; k += kScanThreads) {
    int32_t c = 0;
    for (int r = 0; r < tiles_n; ++r) c += src.bit(static_cast<int64_t>(r) * tiles_k + k);
    cnt[k] = c;
  }
  __syncthreads();
  block_exclusive_scan(cnt, tiles_k, col_ptr, wsum);
  for (int k = tid; k < tiles_k; k += kScanThreads) {
    int32_t pos = cnt[k];
    for (int r = 0; r < tiles_n; ++r)
      if (src.bit(static_cast<int64_t>(r) * tiles_k + k)) col_rows[pos++] = r;
  }
}

// The same plan for grids of at most kWideDim tiles per side, spread over
// tiles_n + tiles_k workgroups of kWideThreads: workgroup r < tiles_n lists
// tile row r (CSR, flat, its bwd_weight groups), workgroup tiles_n + c lists
// tile column c (CSC). Every workgroup stages the whole bitmap in LDS
// (drawing it itself when sampling; workgroup 0 writes it out) and derives
// its row's (column's) start from the counts of the rows (columns) before
// it, so no workgroup waits for another. The outputs are those of
// plan_tiles_kernel, entry for entry.
constexpr int kWideThreads = 256;
constexpr int kWideDim = 256;
constexpr int kWideWords = kWideDim * kWideDim / 32;

__global__ void __launch_bounds__(kWideThreads)
    plan_tiles_wide_kernel(uint32_t* bits, TileSampler smp, int32_t tiles_n, int32_t tiles_k,
                           int32_t* __restrict__ row_ptr, int32_t* __restrict__ row_cols,
                           int32_t* __restrict__ col_ptr, int32_t* __restrict__ col_rows,
                           int32_t* __restrict__ flat, int32_t* __restrict__ chunks) {
  __shared__ uint32_t sbits[kWideWords];
  __shared__ int32_t red[2][kWideThreads / 64];
  __shared__ int32_t wpre[kWideThreads / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t nbits = static_cast<int64_t>(tiles_n) * tiles_k;
  const int nwords = static_cast<int>((nbits + 31) / 32);
  if (smp.enabled) {
    for (int64_t base = 0; base < nbits; base += kWideThreads) {
      const int64_t t = base + tid;
      bool keep = false;
      if (t < nbits)
        keep = static_cast<double>(splitmix_draw(smp.s0, static_cast<uint64_t>(t)) >> 11) * 0x1.0p-53 >= smp.p;
      const uint64_t m = __ballot(keep);
      const int64_t w0 = (base + 64 * wave) / 32;
      if (lane < 2 && w0 + lane < nwords) {
        const uint32_t x = static_cast<uint32_t>(m >> (32 * lane));
        sbits[w0 + lane] = x;
        if (blockIdx.x == 0) bits[w0 + lane] = x;
      }
    }
  } else {
    for (int w = tid; w < nwords; w += kWideThreads) sbits[w] = bits[w];
  }
  __syncthreads();
  BitSrc src = {nullptr, sbits};
  const bool is_row = static_cast<int>(blockIdx.x) < tiles_n;
  const int own = is_row ? static_cast<int>(blockIdx.x) : static_cast<int>(blockIdx.x) - tiles_n;
  const int len = is_row ? tiles_k : tiles_n;     // entries of the own row (column)
  const int nown = is_row ? tiles_n : tiles_k;    // rows (columns) in all
  // counts of the rows (columns) before this one (and groups, for rows):
  // thread i counts row (column) i
  int32_t c_before = 0, g_before = 0, c_total = 0, g_total = 0;
  {
    int32_t c = 0;
    if (tid < nown) {
      if (is_row) {
        c = src.count(static_cast<int64_t>(tid) * tiles_k, static_cast<int64_t>(tid + 1) * tiles_k);
      } else {
        for (int r = 0; r < tiles_n; ++r) c += src.bit(static_cast<int64_t>(r) * tiles_k + tid);
      }
    }
    const int32_t g = (c + kTdpChunk - 1) / kTdpChunk;
    int32_t cb = tid < own ? c : 0, gb = tid < own ? g : 0;
    int32_t ct = c, gt = g;
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) {
      cb += __shfl_xor(cb, d, 64);
      gb += __shfl_xor(gb, d, 64);
      ct += __shfl_xor(ct, d, 64);
      gt += __shfl_xor(gt, d, 64);
    }
    __shared__ int32_t tot[2][kWideThreads / 64];
    if (lane == 0) {
      red[0][wave] = cb;
      red[1][wave] = gb;
      tot[0][wave] = ct;
      tot[1][wave] = gt;
    }
    __syncthreads();
#pragma unroll
    for (int v = 0; v < kWideThreads / 64; ++v) {
      c_before += red[0][v];
      g_before += red[1][v];
      c_total += tot[0][v];
      g_total += tot[1][v];
    }
  }
  // the own row's (column's) entries: thread i takes entry i, its rank among
  // the kept ones from a ballot per wave and the kept counts of the waves before
  const bool kept = tid < len && (is_row ? src.bit(static_cast<int64_t>(own) * tiles_k + tid)
                                         : src.bit(static_cast<int64_t>(tid) * tiles_k + own));
  const uint64_t m = __ballot(kept);
  if (lane == 0) wpre[wave] = __popcll(m);
  __syncthreads();
  int32_t rank = __popcll(m & ((uint64_t{1} << lane) - 1));
  int32_t nkept = 0;
#pragma unroll
  for (int v = 0; v < kWideThreads / 64; ++v) {
    if (v < wave) rank += wpre[v];
    nkept += wpre[v];
  }
  if (is_row) {
    if (tid == 0) row_ptr[own] = c_before;
    if (own == tiles_n - 1 && tid == 0) {
      row_ptr[tiles_n] = c_total;
      chunks[0] = g_total;
      chunks[1] = chunks[2] = chunks[3] = 0;
    }
    if (kept) {
      const int32_t pos = c_before + rank;
      row_cols[pos] = tid;
      flat[pos] = own * tiles_k + tid;
      int32_t* rec = chunks + 4 + static_cast<int64_t>(g_before + rank / kTdpChunk) * kTdpRec;
      const int slot = rank % kTdpChunk;
      if (slot == 0) {
        rec[0] = own;
        rec[1] = pos;
        rec[2] = nkept - rank < kTdpChunk ? nkept - rank : kTdpChunk;
        rec[3] = 0;
      }
      rec[4 + slot] = tid;
      if (rank == nkept - 1)  // the row's last tile pads its group
        for (int i = slot + 1; i < kTdpChunk; ++i) rec[4 + i] = tid;
    }
  } else {
    if (tid == 0) col_ptr[own] = c_before;
    if (own == tiles_k - 1 && tid == 0) col_ptr[tiles_k] = c_total;
    if (kept) col_rows[c_before + rank] = tid;
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
  const int32_t* count;  // kept tiles (device), the length of flat
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
    if (static_cast<int>(blockIdx.x) >= *a.count) return;  // the grid may be an upper bound
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

// Direct loads of one operand pair whose slabs follow a list of kept tiles:
// slab q is part q % SPT (BK wide in k) of the tile named by entry q / SPT of
// the workgroup's list, at a0 + entry * a_tile + part * a_part (B alike).
// Entry e sits in lane e - wbase of the per-lane window win and is read with
// readlane, so the main loop makes no memory access for the list but one
// window refill per 64 entries. Past the last slab the last one is loaded
// again, so every wave issues the same number of loads per slab.
template <class Cfg, bool AMC, bool BMC, int SPT>
struct ListLoader {
  DmaSrc<Cfg, Cfg::BM, AMC> da;
  DmaSrc<Cfg, Cfg::BN, BMC> db;
  const char* a0;
  const char* b0;
  int64_t a_tile, b_tile, a_part, b_part;
  const int32_t* list;
  int n, q, nq, wbase, win, is, wv;
  uint32_t lds0;

  // The load waits for itself inside the statement: a compiler-visible load
  // here would make every later readlane wait for all direct loads in flight.
  // Lanes past the list read its last entry.
  __device__ __forceinline__ void refill() {
    const int lane = threadIdx.x & 63;
    const int32_t* p = list + (wbase + lane < n ? wbase + lane : n - 1);
    int32_t v;
    asm volatile("global_load_dword %0, %1, off\n\ts_waitcnt vmcnt(0)" : "=v"(v) : "v"(p) : "memory");
    win = v;
  }

  // One slab's loads in two halves (see run_slabs): A, then B and the advance.
  int64_t tcur;
  __device__ __forceinline__ void issue_a() {
    const int e = q / SPT, part = q % SPT;
    if (e - wbase >= 64) {
      wbase += 64;
      refill();
    }
    tcur = __builtin_amdgcn_readlane(win, e - wbase);
    da.issue(a0 + tcur * a_tile + part * a_part, Cfg::BK, lds0 + static_cast<uint32_t>(is * Cfg::STAGE), wv);
  }
  __device__ __forceinline__ void issue_b() {
    const int part = q % SPT;
    db.issue(b0 + tcur * b_tile + part * b_part, Cfg::BK,
             lds0 + static_cast<uint32_t>(is * Cfg::STAGE) + Cfg::ABYTES, wv);
    is = is + 1 == Cfg::STAGES ? 0 : is + 1;
    if (q + 1 < nq) ++q;
  }
  __device__ __forceinline__ void issue() {
    issue_a();
    issue_b();
  }
};

struct TdpFastArgs {
  const void* act;      // Xt (fwd, bwd_weight) or dYt (bwd_data)
  const void* act2;     // dYt (bwd_weight)
  const void* W;
  void* out;            // Yt, dXt or dW
  int32_t B, K;         // batch; in_features (row stride of W and dW)
  int32_t nx, ny;       // fwd / bwd_data grid: batch blocks x tile rows (columns)
  const int32_t* ptr;   // row_ptr (fwd, bwd_weight) or col_ptr (bwd_data)
  const int32_t* list;  // row_cols (fwd, bwd_weight) or col_rows (bwd_data)
  const int32_t* chunks;
  float scale;
  // split lists (fp32 output only): workgroup (tile, split) sums its share of
  // the row's (column's) kept tiles into partial[split][rows][B]
  int32_t splits, rows;
  float* partial;
};

constexpr int kFastTile = 64;

// fwd:       Yt[tn block][n0 ..] = scale * sum over kept tk of row tn: W(tn, tk) Xt[tk block][n0 ..]
// bwd_data:  dXt[tk block][n0 ..] = scale * sum over kept tn of column tk: W(tn, tk)^T dYt[tn block][n0 ..]
// A tile row (column) without kept tiles gets zeros.
// One workgroup of the fwd / bwd_data product: position bid of the grid of
// nx x ny (batch block, tile row or column), split sp.
template <class Cfg, int PASS, typename OutT>
__device__ __forceinline__ void tdp_rows_tile(const TdpFastArgs& a, int bid, int sp, char* smem) {
  constexpr int TT = kFastTile, ES = Cfg::ES, SPT = TT / Cfg::BK;
  constexpr bool AMC = PASS == TDP_BWD_DATA;
  static_assert(Cfg::BM == TT && TT % Cfg::BK == 0, "one tile row per workgroup");
  const int wave = threadIdx.x >> 6;
  const int ks = wave / (Cfg::WGM * Cfg::WGN), wmn = wave % (Cfg::WGM * Cfg::WGN);
  const int wm = wmn / Cfg::WGN, wn = wmn % Cfg::WGN;
  int own, col;
  grouped_tile(bid, a.nx, a.ny, own, col);
  const int n0 = col * Cfg::BN;
  const int splits = a.splits > 1 ? a.splits : 1;
  const int pa = __builtin_amdgcn_readfirstlane(a.ptr[own]);
  const int nall = __builtin_amdgcn_readfirstlane(a.ptr[own + 1]) - pa;
  const int p0 = pa + nall * sp / splits;  // this split's share of the list
  const int p1 = pa + nall * (sp + 1) / splits;

  f32x16 acc[Cfg::FM][Cfg::FN];
#pragma unroll
  for (int i = 0; i < Cfg::FM; ++i)
#pragma unroll
    for (int j = 0; j < Cfg::FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  ListLoader<Cfg, AMC, true, SPT> ld;
  ld.wv = __builtin_amdgcn_readfirstlane(wave);
  ld.lds0 = __builtin_amdgcn_readfirstlane(lds_addr(smem));
  ld.list = a.list + p0;
  ld.n = p1 - p0;
  ld.q = 0;
  ld.nq = ld.n * SPT;
  ld.wbase = 0;
  ld.is = 0;
  const char* W = static_cast<const char*>(a.W);
  const int64_t K = a.K, B = a.B;
  if constexpr (PASS == TDP_FWD) {
    ld.a0 = W + own * TT * K * ES;  // W(tn, tk) at column tk * TT of the tile row
    ld.a_tile = TT * ES;
    ld.a_part = Cfg::BK * ES;
  } else {
    ld.a0 = W + own * TT * ES;      // W(tn, tk)^T: k-rows tn * TT .. of the tile column
    ld.a_tile = TT * K * ES;
    ld.a_part = Cfg::BK * K * ES;
  }
  ld.b0 = static_cast<const char*>(a.act);
  ld.b_tile = TT * B * ES;
  ld.b_part = Cfg::BK * B * ES;
  if (ld.nq > 0) {
    ld.refill();
    ld.da.init(K, 0, TT, ld.wv);
    ld.db.init(B, n0, a.B, ld.wv);
  }
  run_slabs<Cfg, AMC, true, false>(ld, ld.nq, 0, 0, acc, wm, wn, ks * Cfg::KW, smem);
  if constexpr (Cfg::KSPLIT > 1) {
    // the waves of k slices 1.. hand their sums to slice 0 through LDS
    constexpr int NREG = Cfg::FM * Cfg::FN * 16;
    static_assert((Cfg::KSPLIT - 1) * Cfg::WGM * Cfg::WGN * NREG * 64 * 4 <= Cfg::LDS, "reduction buffer exceeds LDS");
    float* red = reinterpret_cast<float*>(smem);
    const int lane = threadIdx.x & 63;
    lds_barrier();  // every wave is done with the stages
    if (ks > 0) {
#pragma unroll
      for (int i = 0; i < Cfg::FM; ++i)
#pragma unroll
        for (int j = 0; j < Cfg::FN; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            red[(((ks - 1) * Cfg::WGM * Cfg::WGN + wmn) * NREG + (i * Cfg::FN + j) * 16 + r) * 64 + lane] =
                acc[i][j][r];
    }
    lds_barrier();
    if (ks == 0) {
#pragma unroll
      for (int u = 1; u < Cfg::KSPLIT; ++u)
#pragma unroll
        for (int i = 0; i < Cfg::FM; ++i)
#pragma unroll
          for (int j = 0; j < Cfg::FN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r)
              acc[i][j][r] += red[(((u - 1) * Cfg::WGM * Cfg::WGN + wmn) * NREG + (i * Cfg::FN + j) * 16 + r) * 64 + lane];
    }
  }

  GemmArgs g = {};
  g.M = ks == 0 ? TT : 0;  // only k slice 0 writes
  g.N = a.B;
  g.c.p = static_cast<OutT*>(a.out) + static_cast<int64_t>(own) * TT * B;
  g.c.ld = B;
  g.c.scale = a.scale;
  if constexpr (sizeof(OutT) == 4) {
    if (splits > 1) {  // unscaled partial sums; the reduction applies the scale
      g.c.p = a.partial + (static_cast<int64_t>(sp) * a.rows + static_cast<int64_t>(own) * TT) * B;
      g.c.scale = 1.0f;
    }
  }
  fast_store<OutT, Cfg, EPI_FWD>(g, acc, 0, n0, wm, wn, 0, 0, smem);
}

template <class Cfg, int PASS, typename OutT>
__global__ void __launch_bounds__(Cfg::NT) tdp_fast_kernel(TdpFastArgs a) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  tdp_rows_tile<Cfg, PASS, OutT>(a, static_cast<int>(blockIdx.x), a.splits > 1 ? static_cast<int>(blockIdx.y) : 0,
                                 smem);
}

// out[e] = scale * sum over the splits of partial[split][e], in split order
// (the loads of up to eight splits issued together).
__global__ void __launch_bounds__(256) tdp_split_reduce_kernel(const float* __restrict__ partial, int32_t splits,
                                                               int64_t n, float scale, float* __restrict__ out) {
  const int64_t e = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (e >= n) return;
  float v = 0.0f;
  for (int s0 = 0; s0 < splits; s0 += 8) {
    float t[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) t[u] = s0 + u < splits ? partial[(s0 + u) * n + e] : 0.0f;
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (s0 + u < splits) v += t[u];
  }
  out[e] = scale * v;
}

// bwd_weight: dW(tn, tk) = scale * dYt[tn block] Xt[tk block]^T (contraction
// over the batch) for a group of up to kTdpChunk kept tiles of tile row tn;
// wave column wn computes the group's tile wn. Each workgroup takes the groups
// t, t + gridDim.x, ... of the list (t its position in the XCD-aware order),
// so the grid can stay at what the chip holds at once.
// Workgroup bid of nw walking the weight-gradient groups bid', bid' + nw, ...
// (bid' its position in the XCD-aware order).
template <class Cfg, typename OutT>
__device__ __forceinline__ void tdp_dw_walk(const TdpFastArgs& a, int bid, int nw, char* smem) {
  constexpr int TT = kFastTile, ES = Cfg::ES;
  static_assert(Cfg::BM == TT && Cfg::TN == TT && Cfg::BN == TT * kTdpChunk && Cfg::KSPLIT == 1,
                "one kept tile per wave column");
  int unused, c0;
  grouped_tile(bid, nw, 1, unused, c0);
  const int count = __builtin_amdgcn_readfirstlane(a.chunks[0]);
  const int wave = threadIdx.x >> 6;
  const int wm = wave / Cfg::WGN, wn = wave % Cfg::WGN;
  const int64_t B = a.B, K = a.K;
  const int nslab = (a.B + Cfg::BK - 1) / Cfg::BK;

  for (int c = c0; c < count; c += nw) {
    const int32_t* rec = a.chunks + 4 + static_cast<int64_t>(c) * kTdpRec;
    const int tn = __builtin_amdgcn_readfirstlane(rec[0]);
    const int cnt = __builtin_amdgcn_readfirstlane(rec[2]);
    const int32_t* cols = rec + 4;  // padded with the last column up to kTdpChunk

    f32x16 acc[Cfg::FM][Cfg::FN];
#pragma unroll
    for (int i = 0; i < Cfg::FM; ++i)
#pragma unroll
      for (int j = 0; j < Cfg::FN; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

    SlabLoader<Cfg, false, false> ld;
    ld.wv = __builtin_amdgcn_readfirstlane(wave);
    ld.lds0 = __builtin_amdgcn_readfirstlane(lds_addr(smem));
    ld.da.init(B, 0, TT, ld.wv);
    // row r of the B tile: row r % TT of X block cols[r / TT]
    ld.db.init_rows(B, [&](int r) { return cols[r / TT] * TT + r % TT; }, ld.wv);
    ld.K = a.B;
    ld.ik = 0;
    ld.is = 0;
    ld.left = nslab - 1;
    ld.a_step = Cfg::BK * ES;
    ld.b_step = Cfg::BK * ES;
    ld.a_wrap = 0;
    ld.b_wrap = 0;
    ld.na = uniform_ptr(static_cast<const char*>(a.act2) + static_cast<int64_t>(tn) * TT * B * ES);
    ld.nb = uniform_ptr(static_cast<const char*>(a.act));
    run_slabs<Cfg, false, false, true>(ld, nslab, a.B, 0, acc, wm, wn, 0, smem);

    // wave column wn writes tile cols[wn]: its columns wn * TT .. land at
    // column cols[wn] * TT of dW (cols ascend, so cols[wn] >= wn)
    const int j = wn < cnt ? wn : 0;  // wave columns past the group write nothing
    GemmArgs g = {};
    g.M = TT;
    g.N = cnt * TT;
    g.c.p = static_cast<OutT*>(a.out) + static_cast<int64_t>(tn) * TT * K + static_cast<int64_t>(cols[j]) * TT -
            static_cast<int64_t>(j) * TT;
    g.c.ld = K;
    g.c.scale = a.scale;
    fast_store<OutT, Cfg, EPI_FWD>(g, acc, 0, 0, wm, wn, 0, 0, smem);
    lds_barrier();  // the next group's loads overwrite the epilogue's staging
  }
}

template <class Cfg, typename OutT>
__global__ void __launch_bounds__(Cfg::NT) tdp_fast_dw_kernel(TdpFastArgs a) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  tdp_dw_walk<Cfg, OutT>(a, static_cast<int>(blockIdx.x), static_cast<int>(gridDim.x), smem);
}

// The layer's backward in one launch: workgroups 0 .. nd - 1 run bwd_data
// (one per tile column and batch block), the nw after them walk the
// weight-gradient groups. A compute unit that finishes its bwd_data tile
// takes up weight-gradient work at once, with no kernel boundary between the
// two products; every output is computed by the same code as in the separate
// kernels, so the results are theirs bit for bit.
template <class CfgD, class CfgW, typename T>
__global__ void __launch_bounds__(CfgD::NT) tdp_fast_bwd_kernel(TdpFastArgs d, TdpFastArgs w, int32_t nd,
                                                                int32_t nw) {
  static_assert(CfgD::NT == CfgW::NT, "one block size");
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int b = static_cast<int>(blockIdx.x);
  if (b < nd)
    tdp_rows_tile<CfgD, TDP_BWD_DATA, T>(d, b, 0, smem);
  else
    tdp_dw_walk<CfgW, float>(w, b - nd, nw, smem);
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
hipError_t run_tdp(int pass, const TdpArgs& a, int owners, int nnz, int tiles, hipStream_t s) {
  const bool vec = (static_cast<int64_t>(a.B) * sizeof(T)) % 16 == 0;
  using C = TdpCfgs<T>;
  if (pass == TDP_BWD_WEIGHT) {
    if (nnz == 0) return hipSuccess;
    const dim3 grid(static_cast<unsigned>(nnz > 0 ? nnz : tiles));  // nnz < 0: known on the device only
    if (a.tile == 64) return launch_tdp<T, float, typename C::Tile64, TDP_BWD_WEIGHT>(a, grid, vec, s);
    return launch_tdp<T, float, typename C::Tile32, TDP_BWD_WEIGHT>(a, grid, vec, s);
  }
  const dim3 grid((a.B + 127) / 128, owners);
  if (pass == TDP_FWD) {
    if (a.tile == 64) return launch_tdp<T, T, typename C::Rows64, TDP_FWD>(a, grid, vec, s);
    return launch_tdp<T, T, typename C::Rows32, TDP_FWD>(a, grid, vec, s);
  }
  if (a.tile == 64) return launch_tdp<T, T, typename C::Rows64, TDP_BWD_DATA>(a, grid, vec, s);
  return launch_tdp<T, T, typename C::Rows32, TDP_BWD_DATA>(a, grid, vec, s);
}

// Direct-load configurations of the fast path (64 x 64 tiles): one tile row
// (column) by 128 batch columns for fwd / bwd_data, one tile row by a group of
// kTdpChunk kept tiles for bwd_weight.
template <typename T>
struct TdpFastCfgs;
// Rows: four waves of 64 x 64 outputs, two of them per k half of each slab
// (fewer LDS bytes per MFMA than 32 x 64 wave tiles over the whole slab).
// Group: one workgroup per compute unit walking the groups.
template <>
struct TdpFastCfgs<bf16> {
  using Rows = FastCfg<bf16, 64, 128, 64, 4, 1, 2, 2>;   // 96 KB LDS
  using Group = FastCfg<bf16, 64, 256, 64, 3, 1, 4, 1>;  // 120 KB
};
// Narrow: 64 batch columns for batches of at most 64 (the tile-pattern
// LSTM's steps), so that no half-empty batch tile is loaded and multiplied.
template <>
struct TdpFastCfgs<float> {
  using Rows = FastCfg<float, 64, 128, 32, 4, 1, 2, 2>;  // 96 KB
  using Narrow = FastCfg<float, 64, 64, 32, 4, 1, 2, 2>; // 64 KB
  using Group = FastCfg<float, 64, 256, 32, 3, 1, 4, 1>; // 120 KB
};

// One instantiation per kernel, so each kernel's attribute is set once
// (thread-safe static initialisation) to allow more than 64 KB of dynamic LDS.
template <class Cfg, void (*KERN)(TdpFastArgs)>
hipError_t launch_with_lds(dim3 grid, const TdpFastArgs& a, hipStream_t s) {
  static const hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void*>(KERN),
                                                     hipFuncAttributeMaxDynamicSharedMemorySize, Cfg::LDS);
  if (attr != hipSuccess) return attr;
  auto kern = KERN;
  hipLaunchKernelGGL(kern, grid, dim3(Cfg::NT), Cfg::LDS, s, a);
  return hipGetLastError();
}

// The fast path takes 64 x 64 tiles, batch rows of whole 16-byte chunks, and
// operands whose chunk offsets from a slab's first element stay below 2^31.
template <typename T>
bool tdp_fast_ok(const TdpArgs& a) {
  const int64_t es = sizeof(T);
  return a.tile == kFastTile && (static_cast<int64_t>(a.B) * es) % 16 == 0 &&
         static_cast<int64_t>(a.K) * a.B * es < (int64_t{1} << 31) &&
         static_cast<int64_t>(a.N) * a.B * es < (int64_t{1} << 31) &&
         static_cast<int64_t>(kFastTile + 1) * a.K * es < (int64_t{1} << 31);
}

// fwd or bwd_data on tile configuration Cfg: batch blocks of Cfg::BN, one
// workgroup per (tile row or column, batch block, split).
template <class Cfg, typename T>
hipError_t launch_rows(int pass, TdpFastArgs& f, int owners, int splits, hipStream_t s) {
  f.nx = (f.B + Cfg::BN - 1) / Cfg::BN;
  f.ny = owners;
  const dim3 grid(static_cast<unsigned>(f.nx * f.ny), static_cast<unsigned>(splits));
  if (pass == TDP_FWD) return launch_with_lds<Cfg, tdp_fast_kernel<Cfg, TDP_FWD, T>>(grid, f, s);
  return launch_with_lds<Cfg, tdp_fast_kernel<Cfg, TDP_BWD_DATA, T>>(grid, f, s);
}

template <typename T>
hipError_t run_tdp_fast(int pass, const TdpArgs& a, const int32_t* chunks, int owners, int nnz, hipStream_t s) {
  using C = TdpFastCfgs<T>;
  TdpFastArgs f = {a.act, a.act2, a.W, a.out, a.B, a.K, 0, 0, a.ptr, a.list, chunks, a.scale};
  if (pass == TDP_BWD_WEIGHT) {
    if (nnz == 0) return hipSuccess;
    // groups: sum over rows of ceil(kept / kTdpChunk) <= (nnz + (kTdpChunk - 1) * rows with a kept tile) / kTdpChunk;
    // with the count known on the device only (nnz < 0), every row full
    const int64_t rows = owners < nnz ? owners : nnz;
    int64_t bound = nnz > 0 ? (nnz + (kTdpChunk - 1) * rows) / kTdpChunk
                            : static_cast<int64_t>(owners) * ((a.tiles_k + kTdpChunk - 1) / kTdpChunk);
    // one workgroup per compute unit, each walking several groups
    if (bound > kTargetBlocks) bound = kTargetBlocks;
    return launch_with_lds<typename C::Group, tdp_fast_dw_kernel<typename C::Group, float>>(
        dim3(static_cast<unsigned>(bound)), f, s);
  }
  if constexpr (sizeof(T) == 4) {
    if (a.B <= C::Narrow::BN) return launch_rows<typename C::Narrow, T>(pass, f, owners, 1, s);
  }
  return launch_rows<typename C::Rows, T>(pass, f, owners, 1, s);
}

// bwd_data and bwd_weight as one launch of tdp_fast_bwd_kernel (both on the
// fast path): the bwd_data workgroups first, then the weight-gradient walkers.
template <class CfgD, typename T>
hipError_t launch_tdp_fast_bwd(const TdpArgs& ad, const TdpArgs& aw, const int32_t* chunks, int tiles_n,
                               int tiles_k, int nnz, hipStream_t s) {
  using CfgW = typename TdpFastCfgs<T>::Group;
  constexpr int LDS = CfgD::LDS > CfgW::LDS ? CfgD::LDS : CfgW::LDS;
  auto kern = tdp_fast_bwd_kernel<CfgD, CfgW, T>;
  static const hipError_t attr =
      hipFuncSetAttribute(reinterpret_cast<const void*>(kern), hipFuncAttributeMaxDynamicSharedMemorySize, LDS);
  if (attr != hipSuccess) return attr;
  TdpFastArgs d = {ad.act, nullptr, ad.W, ad.out, ad.B, ad.K, 0, 0, ad.ptr, ad.list, chunks, ad.scale};
  d.nx = (d.B + CfgD::BN - 1) / CfgD::BN;
  d.ny = tiles_k;
  TdpFastArgs w = {aw.act, aw.act2, aw.W, aw.out, aw.B, aw.K, 0, 0, aw.ptr, aw.list, chunks, aw.scale};
  const int64_t rows = tiles_n < nnz ? tiles_n : nnz;
  int64_t nw = nnz > 0 ? (nnz + (kTdpChunk - 1) * rows) / kTdpChunk
                       : nnz == 0 ? 0 : static_cast<int64_t>(tiles_n) * ((tiles_k + kTdpChunk - 1) / kTdpChunk);
  if (nw > kTargetBlocks) nw = kTargetBlocks;
  const int64_t nd = static_cast<int64_t>(d.nx) * d.ny;
  hipLaunchKernelGGL(kern, dim3(static_cast<unsigned>(nd + nw)), dim3(CfgD::NT), LDS, s, d, w,
                     static_cast<int32_t>(nd), static_cast<int32_t>(nw));
  return hipGetLastError();
}

template <typename T>
hipError_t run_tdp_fast_bwd(const TdpArgs& ad, const TdpArgs& aw, const int32_t* chunks, int tiles_n, int tiles_k,
                            int nnz, hipStream_t s) {
  using C = TdpFastCfgs<T>;
  if constexpr (sizeof(T) == 4) {
    if (ad.B <= C::Narrow::BN) return launch_tdp_fast_bwd<typename C::Narrow, T>(ad, aw, chunks, tiles_n, tiles_k, nnz, s);
  }
  return launch_tdp_fast_bwd<typename C::Rows, T>(ad, aw, chunks, tiles_n, tiles_k, nnz, s);
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
  if (p->nnz < -1 || p->nnz > p->tiles_n * p->tiles_k) return fail(ARD_ERR_INVALID_ARG, "plan nnz out of range");
  if (!p->d_bits || !p->d_row_ptr || !p->d_row_cols || !p->d_col_ptr || !p->d_col_rows || !p->d_flat ||
      !p->d_chunks)
    return fail(ARD_ERR_INVALID_ARG, "plan has NULL lists");
  return ARD_OK;
}

int check_dev_ptr(const void* p, const char* name) {
  if (!p) return fail(ARD_ERR_INVALID_ARG, "%s is NULL", name);
  if (!aligned16(p)) return fail(ARD_ERR_INVALID_ARG, "%s is not 16-byte aligned", name);
  return ARD_OK;
}

// Shared by both plan entry points: validates, lays the lists out in the
// workspace and launches the plan kernel (sampling the bitmap first if asked).
int plan_tiles(int32_t n, int32_t k, int32_t tile, uint32_t* d_bits, int32_t nnz, TileSampler smp, void* d_ws,
               size_t ws_bytes, ard_tile_plan* plan, void* stream) {
  if (!plan) return fail(ARD_ERR_INVALID_ARG, "plan is NULL");
  if (tile != 32 && tile != 64) return fail(ARD_ERR_INVALID_ARG, "tile must be 32 or 64, got %d", tile);
  if (n < tile || k < tile || n % tile || k % tile)
    return fail(ARD_ERR_INVALID_ARG, "n (%d) and k (%d) must be positive multiples of the tile %d", n, k, tile);
  const int32_t tn = n / tile, tk = k / tile;
  if (tn > kMaxTileDim || tk > kMaxTileDim)
    return fail(ARD_ERR_UNSUPPORTED, "tile grid %d x %d exceeds %d per side", tn, tk, kMaxTileDim);
  if (static_cast<int64_t>(nnz) > static_cast<int64_t>(tn) * tk)
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
  w += align256(4 * full);
  plan->d_chunks = reinterpret_cast<int32_t*>(w);
  if (tn <= kWideDim && tk <= kWideDim)
    hipLaunchKernelGGL(plan_tiles_wide_kernel, dim3(static_cast<unsigned>(tn + tk)), dim3(kWideThreads), 0,
                       static_cast<hipStream_t>(stream), d_bits, smp, tn, tk, plan->d_row_ptr, plan->d_row_cols,
                       plan->d_col_ptr, plan->d_col_rows, plan->d_flat, plan->d_chunks);
  else
    hipLaunchKernelGGL(plan_tiles_kernel, dim3(1), dim3(kScanThreads), 0, static_cast<hipStream_t>(stream),
                       d_bits, smp, tn, tk, plan->d_row_ptr, plan->d_row_cols, plan->d_col_ptr,
                       plan->d_col_rows, plan->d_flat, plan->d_chunks);
  ARD_LAUNCH_CHECK();
  return ARD_OK;
}

}  // namespace

// The fp32 tile layer's forward (fwd) or transposed product with each tile
// row's (column's) kept-tile list split over up to 8 workgroups when the tile
// rows (columns) alone would leave most of the chip idle, as for a recurrent
// step at a small batch: partial sums in `partial` (partial_floats floats),
// then a fixed-order reduction that applies the scale. Runs the single-pass
// call when no split applies (another dtype, the register-staged path, too
// many workgroups already, or too small a partial buffer).
int tdp_product_f32_split(bool fwd, const ard_tile_desc* d, const ard_tile_plan* p, const void* act, const void* W,
                          void* out, float* partial, size_t partial_floats, void* stream, int* splits_left) {
  if (splits_left) *splits_left = 1;
  int st = check_tile_call(d, p);
  if (st != ARD_OK) return st;
  auto single = [&]() {
    return fwd ? ard_tile_fwd(d, p, act, W, out, stream) : ard_tile_bwd_data(d, p, act, W, out, stream);
  };
  if (d->dtype != ARD_F32 || !partial || !aligned16(partial)) return single();
  if ((st = check_dev_ptr(act, "act")) || (st = check_dev_ptr(W, "W")) || (st = check_dev_ptr(out, "out")))
    return st;
  TdpArgs a = {act, nullptr, W, out, d->batch, p->n, p->k, p->tile, p->tiles_k,
               fwd ? p->d_row_ptr : p->d_col_ptr, fwd ? p->d_row_cols : p->d_col_rows, d->scale,
               p->d_row_ptr + p->tiles_n};
  if (!tdp_fast_ok<float>(a)) return single();
  using C = TdpFastCfgs<float>;
  const int owners = fwd ? p->tiles_n : p->tiles_k;
  const bool narrow = a.B <= C::Narrow::BN;
  const int bn = narrow ? C::Narrow::BN : C::Rows::BN;
  const int nx = (a.B + bn - 1) / bn;
  int splits = 1;
  while (splits < 8 && static_cast<int64_t>(nx) * owners * splits * 2 <= kTargetBlocks) splits *= 2;
  const int64_t rows = static_cast<int64_t>(owners) * kFastTile;
  if (splits == 1 || static_cast<size_t>(splits) * rows * a.B > partial_floats) return single();
  TdpFastArgs f = {a.act, nullptr, a.W, a.out, a.B, a.K, nx, owners, a.ptr, a.list, p->d_chunks, a.scale,
                   splits, static_cast<int32_t>(rows), partial};
  hipStream_t sm = static_cast<hipStream_t>(stream);
  const int pass = fwd ? TDP_FWD : TDP_BWD_DATA;
  if (narrow)
    ARD_HIP_CHECK((launch_rows<C::Narrow, float>(pass, f, owners, splits, sm)));
  else
    ARD_HIP_CHECK((launch_rows<C::Rows, float>(pass, f, owners, splits, sm)));
  if (splits_left) {  // the caller adds the partial sums itself (scale 1 only)
    *splits_left = splits;
    return ARD_OK;
  }
  const int64_t n = rows * a.B;
  hipLaunchKernelGGL(tdp_split_reduce_kernel, dim3(static_cast<unsigned>((n + 255) / 256)), dim3(256), 0, sm,
                     partial, splits, n, a.scale, static_cast<float*>(out));
  ARD_LAUNCH_CHECK();
  return ARD_OK;
}

}  // namespace ard

using namespace ard;

extern "C" {

size_t ard_tile_plan_workspace_bytes(int32_t tiles_n, int32_t tiles_k) {
  if (tiles_n < 1 || tiles_k < 1) return 0;
  const size_t nnz = static_cast<size_t>(tiles_n) * tiles_k;
  return align256(4 * (tiles_n + 1)) + align256(4 * (tiles_k + 1)) + 3 * align256(4 * nnz) +
         align256(4 * (4 + kTdpRec * nnz));
}

int ard_plan_tiles(int32_t n, int32_t k, int32_t tile, const uint32_t* d_bits, int32_t nnz, void* d_ws,
                   size_t ws_bytes, ard_tile_plan* plan, void* stream) {
  clear_error();
  if (nnz < 0) return fail(ARD_ERR_INVALID_ARG, "nnz %d out of range", nnz);
  return plan_tiles(n, k, tile, const_cast<uint32_t*>(d_bits), nnz, TileSampler{0, 0.0, 0}, d_ws, ws_bytes, plan,
                    stream);
}

int ard_plan_tiles_bernoulli(int32_t n, int32_t k, int32_t tile, double p, uint64_t seed, uint32_t stream_id,
                             uint64_t iter, uint32_t* d_bits, void* d_ws, size_t ws_bytes, ard_tile_plan* plan,
                             void* stream) {
  clear_error();
  if (!(p >= 0.0 && p <= 1.0)) return fail(ARD_ERR_INVALID_ARG, "p must lie in [0, 1]");
  if (stream_id >= (1u << 24)) return fail(ARD_ERR_INVALID_ARG, "stream %u must be < 2^24", stream_id);
  if (iter >= (uint64_t{1} << 40)) return fail(ARD_ERR_INVALID_ARG, "iter must be < 2^40");
  const TileSampler smp = {1, p, seed ^ ((static_cast<uint64_t>(stream_id) << 40) | iter)};
  return plan_tiles(n, k, tile, d_bits, -1, smp, d_ws, ws_bytes, plan, stream);
}

int ard_tile_fwd(const ard_tile_desc* desc, const ard_tile_plan* plan, const void* Xt, const void* W,
                 void* Yt, void* stream) {
  clear_error();
  int st = check_tile_call(desc, plan);
  if (st != ARD_OK) return st;
  if ((st = check_dev_ptr(Xt, "Xt")) || (st = check_dev_ptr(W, "W")) || (st = check_dev_ptr(Yt, "Yt")))
    return st;
  TdpArgs a = {Xt, nullptr, W, Yt, desc->batch, plan->n, plan->k, plan->tile, plan->tiles_k,
               plan->d_row_ptr, plan->d_row_cols, desc->scale, plan->d_row_ptr + plan->tiles_n};
  const int full = plan->tiles_n * plan->tiles_k;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (desc->dtype == ARD_BF16) {
    if (tdp_fast_ok<bf16>(a))
      ARD_HIP_CHECK(run_tdp_fast<bf16>(TDP_FWD, a, plan->d_chunks, plan->tiles_n, plan->nnz, s));
    else
      ARD_HIP_CHECK(run_tdp<bf16>(TDP_FWD, a, plan->tiles_n, plan->nnz, full, s));
  } else {
    if (tdp_fast_ok<float>(a))
      ARD_HIP_CHECK(run_tdp_fast<float>(TDP_FWD, a, plan->d_chunks, plan->tiles_n, plan->nnz, s));
    else
      ARD_HIP_CHECK(run_tdp<float>(TDP_FWD, a, plan->tiles_n, plan->nnz, full, s));
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
               plan->d_col_ptr, plan->d_col_rows, desc->scale, plan->d_row_ptr + plan->tiles_n};
  const int full = plan->tiles_n * plan->tiles_k;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (desc->dtype == ARD_BF16) {
    if (tdp_fast_ok<bf16>(a))
      ARD_HIP_CHECK(run_tdp_fast<bf16>(TDP_BWD_DATA, a, plan->d_chunks, plan->tiles_k, plan->nnz, s));
    else
      ARD_HIP_CHECK(run_tdp<bf16>(TDP_BWD_DATA, a, plan->tiles_k, plan->nnz, full, s));
  } else {
    if (tdp_fast_ok<float>(a))
      ARD_HIP_CHECK(run_tdp_fast<float>(TDP_BWD_DATA, a, plan->d_chunks, plan->tiles_k, plan->nnz, s));
    else
      ARD_HIP_CHECK(run_tdp<float>(TDP_BWD_DATA, a, plan->tiles_k, plan->nnz, full, s));
  }
  return ARD_OK;
}

int ard_tile_bwd(const ard_tile_desc* desc, const ard_tile_plan* plan, const void* Xt, const void* dYt,
                 const void* W, void* dXt, float* dW, void* stream) {
  clear_error();
  int st = check_tile_call(desc, plan);
  if (st != ARD_OK) return st;
  if ((st = check_dev_ptr(Xt, "Xt")) || (st = check_dev_ptr(dYt, "dYt")) || (st = check_dev_ptr(W, "W")) ||
      (st = check_dev_ptr(dXt, "dXt")) || (st = check_dev_ptr(dW, "dW")))
    return st;
  const TdpArgs ad = {dYt, nullptr, W, dXt, desc->batch, plan->n, plan->k, plan->tile, plan->tiles_k,
                      plan->d_col_ptr, plan->d_col_rows, desc->scale, plan->d_row_ptr + plan->tiles_n};
  const TdpArgs aw = {Xt, dYt, nullptr, dW, desc->batch, plan->n, plan->k, plan->tile, plan->tiles_k,
                      plan->d_row_ptr, plan->d_row_cols, desc->scale, plan->d_row_ptr + plan->tiles_n};
  const bool bf = desc->dtype == ARD_BF16;
  if (!(bf ? tdp_fast_ok<bf16>(ad) : tdp_fast_ok<float>(ad))) {  // the two calls one after the other
    if ((st = ard_tile_bwd_data(desc, plan, dYt, W, dXt, stream)) != ARD_OK) return st;
    return ard_tile_bwd_weight(desc, plan, Xt, dYt, dW, stream);
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (bf)
    ARD_HIP_CHECK(run_tdp_fast_bwd<bf16>(ad, aw, plan->d_chunks, plan->tiles_n, plan->tiles_k, plan->nnz, s));
  else
    ARD_HIP_CHECK(run_tdp_fast_bwd<float>(ad, aw, plan->d_chunks, plan->tiles_n, plan->tiles_k, plan->nnz, s));
  const int full = plan->tiles_n * plan->tiles_k;
  if (desc->dropped == ARD_DROPPED_ZERO && plan->nnz != full) {
    hipLaunchKernelGGL(zero_dropped_tiles_kernel, dim3(plan->tiles_k, plan->tiles_n), dim3(256), 0, s,
                       plan->d_bits, dW, plan->k, plan->tile, plan->tiles_k);
    ARD_LAUNCH_CHECK();
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
               nullptr, plan->d_flat, desc->scale, plan->d_row_ptr + plan->tiles_n};
  const int full = plan->tiles_n * plan->tiles_k;
  TdpArgs f = a;  // the fast path walks the groups of row_cols
  f.ptr = plan->d_row_ptr;
  f.list = plan->d_row_cols;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (desc->dtype == ARD_BF16) {
    if (tdp_fast_ok<bf16>(a))
      ARD_HIP_CHECK(run_tdp_fast<bf16>(TDP_BWD_WEIGHT, f, plan->d_chunks, plan->tiles_n, plan->nnz, s));
    else
      ARD_HIP_CHECK(run_tdp<bf16>(TDP_BWD_WEIGHT, a, 0, plan->nnz, full, s));
  } else {
    if (tdp_fast_ok<float>(a))
      ARD_HIP_CHECK(run_tdp_fast<float>(TDP_BWD_WEIGHT, f, plan->d_chunks, plan->tiles_n, plan->nnz, s));
    else
      ARD_HIP_CHECK(run_tdp<float>(TDP_BWD_WEIGHT, a, 0, plan->nnz, full, s));
  }
  if (desc->dropped == ARD_DROPPED_ZERO && plan->nnz != full) {
    hipLaunchKernelGGL(zero_dropped_tiles_kernel, dim3(plan->tiles_k, plan->tiles_n), dim3(256), 0, s,
                       plan->d_bits, dW, plan->k, plan->tile, plan->tiles_k);
    ARD_LAUNCH_CHECK();
  }
  return ARD_OK;
}

}  // extern "C"
