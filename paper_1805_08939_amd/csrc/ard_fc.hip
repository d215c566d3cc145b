// Row-pattern compaction and the fully connected layer under row-based
// dropout patterns (Sec. III-A), fwd / bwd_data / bwd_weight.
//
// The compact problem of each pass is handed to the gathered GEMM: kept output
// neurons select rows of W and of the output, kept input neurons select rows
// of the activations and columns of W. With feature-major activations every
// neuron gather is a whole contiguous row.

#include <hip/hip_runtime.h>

#include <mutex>

#include "ard_gemm.hpp"
#include "ard_gemm_fast.hpp"
#include "ard_internal.hpp"

namespace ard {

// d_idx[i] = offset + period * i for i < kept: the ascending kept list.
__global__ void plan_rows_kernel(int32_t* __restrict__ idx, int32_t kept, int32_t period,
                                 int32_t offset) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < kept) idx[i] = offset + period * i;
}

// ZERO mode: writes 0 to every row r of out[rows][cols] with r % period != offset.
template <typename T>
__global__ void zero_dropped_rows_kernel(T* __restrict__ out, int64_t ld, int32_t cols,
                                         int32_t period, int32_t offset) {
  const int r = blockIdx.x;
  if (r % period == offset) return;
  T* row = out + r * ld;
  for (int c = threadIdx.x; c < cols; c += blockDim.x) row[c] = static_cast<T>(0.0f);
}

// ZERO mode for the weight gradient dW[N][K]: 0 wherever the output row or
// the input column is dropped.
__global__ void zero_dropped_weights_kernel(float* __restrict__ dW, int32_t K, int32_t out_period,
                                            int32_t out_offset, int32_t in_period,
                                            int32_t in_offset) {
  const int r = blockIdx.x;
  float* row = dW + static_cast<int64_t>(r) * K;
  const bool row_kept = (r % out_period) == out_offset;
  for (int c = threadIdx.x; c < K; c += blockDim.x)
    if (!row_kept || (c % in_period) != in_offset) row[c] = 0.0f;
}

// SGD with momentum restricted to the kept weights of a row pattern: for kept
// rows n = out_offset + out_period i and kept columns k = in_offset +
// in_period j, V = mu V + dW and W -= lr V; the same for the bias entries of
// kept rows. Dropped weights, their momentum and their bias entries keep their
// values (frozen for the step). One block per kept row. ldg > 0: the gradient
// is the compact dWc[i][j] with rows of ldg; else dW[n][k], rows of K.
template <typename T>
__global__ void __launch_bounds__(256) sgd_momentum_kernel(T* __restrict__ W, float* __restrict__ V,
                                                           const float* __restrict__ dW, int32_t K, int64_t ldg,
                                                           int32_t out_period, int32_t out_offset, int32_t in_period,
                                                           int32_t in_offset, int32_t kin, float* __restrict__ bias,
                                                           float* __restrict__ Vb, const float* __restrict__ db,
                                                           float lr, float mu) {
  const int64_t n = out_offset + static_cast<int64_t>(out_period) * blockIdx.x;
  T* w = W + n * K;
  float* v = V + n * K;
  const float* g = ldg > 0 ? dW + static_cast<int64_t>(blockIdx.x) * ldg : dW + n * K;
  for (int64_t j = threadIdx.x; j < kin; j += 256) {
    const int64_t k = in_offset + static_cast<int64_t>(in_period) * j;
    const float vn = mu * v[k] + g[ldg > 0 ? j : k];
    v[k] = vn;
    w[k] = from_f32<T>(to_f32(w[k]) - lr * vn);
  }
  if (threadIdx.x == 0 && bias) {
    const float vb = mu * Vb[n] + db[n];
    Vb[n] = vb;
    bias[n] -= lr * vb;
  }
}

// dbias[r] = scale * sum_b G[r][b] for the kept rows r = offset + period * i,
// with G = dY * [Y > 0] when Y is given, else dY. One wave per kept row: each
// lane sums its 16-byte chunks of the row in order, then the lanes are summed
// in a fixed tree, so the result does not depend on timing. vec: rows start
// 16-byte aligned and B is a whole number of chunks.
template <typename T>
__global__ void __launch_bounds__(256) dbias_kernel(const T* __restrict__ dYt, const T* __restrict__ Yt, int32_t B,
                                                    int32_t kept, int32_t period, int32_t offset, float scale,
                                                    int32_t relu, int32_t vec, float* __restrict__ dbias) {
  const int i = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (i >= kept) return;  // whole waves leave together
  const int lane = threadIdx.x & 63;
  const int64_t row = offset + static_cast<int64_t>(period) * i;
  const T* dy = dYt + row * B;
  const T* y = Yt ? Yt + row * B : nullptr;
  constexpr int EPC = 16 / static_cast<int>(sizeof(T));
  float sum = 0.0f;
  if (vec) {
    for (int b0 = lane * EPC; b0 < B; b0 += 64 * EPC) {
      const u32x4 gv = *reinterpret_cast<const u32x4*>(dy + b0);
      u32x4 yv = u32x4{0u, 0u, 0u, 0u};
      if (relu) yv = *reinterpret_cast<const u32x4*>(y + b0);
      const T* ge = reinterpret_cast<const T*>(&gv);
      const T* ye = reinterpret_cast<const T*>(&yv);
#pragma unroll
      for (int e = 0; e < EPC; ++e) sum += (relu && !(to_f32(ye[e]) > 0.0f)) ? 0.0f : to_f32(ge[e]);
    }
  } else {
    for (int b = lane; b < B; b += 64) sum += (relu && !(to_f32(y[b]) > 0.0f)) ? 0.0f : to_f32(dy[b]);
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) sum += __shfl_down(sum, off, 64);
  if (lane == 0) dbias[row] = scale * sum;
}

namespace {

// Gathers W[S_out][S_in] into Wc[kout][ldc]; padding columns are 0. Kept rows
// and columns are arithmetic progressions (source row out_offset +
// out_period * i, source column in_offset + in_period * j). One block per
// compact row: the source row passes through LDS in segments read with
// coalesced 16-byte loads (vec: rows start 16-byte aligned and hold whole
// chunks; else element loads), then consecutive threads write consecutive
// kept columns.
template <typename T>
struct CompactJob {
  const T* W;
  int64_t K;
  int32_t out_period, out_offset, in_period, in_offset, kin;
  int64_t ldc;
  int32_t vec;
  T* Wc;
  int32_t rows;  // kept output rows: one block each
};

constexpr int kMaxCompactJobs = 4;

template <typename T>
struct CompactJobs {
  CompactJob<T> job[kMaxCompactJobs];
  int32_t count;
};

template <typename T>
__device__ __forceinline__ void compact_row(const CompactJob<T>& jb, int64_t i, T* seg) {
  constexpr int SEG = 16384 / static_cast<int>(sizeof(T));  // source columns per segment: 16 KB of LDS
  constexpr int EPC = 16 / static_cast<int>(sizeof(T));
  const int64_t K = jb.K;
  const int32_t in_period = jb.in_period, kin = jb.kin;
  const T* row = jb.W + (jb.out_offset + static_cast<int64_t>(jb.out_period) * i) * K;
  T* crow = jb.Wc + i * jb.ldc;
  const int t = threadIdx.x;
  if (kin > 0) {
    const int64_t first = jb.in_offset, last = jb.in_offset + static_cast<int64_t>(in_period) * (kin - 1);
    for (int64_t s0 = first / SEG * SEG; s0 <= last; s0 += SEG) {
      const int64_t n = K - s0 < SEG ? K - s0 : SEG;  // columns of this segment
      __syncthreads();  // the previous segment is no longer read
      if (jb.vec) {
        // every load of the segment in flight before the first LDS store (a
        // loop of load-then-store waits out one memory latency per chunk)
        constexpr int PER = SEG / EPC / 256;  // 16-byte chunks per thread per segment
        u32x4 v[PER];
#pragma unroll
        for (int u = 0; u < PER; ++u) {
          const int64_t c = static_cast<int64_t>(t + u * 256) * EPC;
          if (c < n) v[u] = *reinterpret_cast<const u32x4*>(row + s0 + c);
        }
#pragma unroll
        for (int u = 0; u < PER; ++u) {
          const int64_t c = static_cast<int64_t>(t + u * 256) * EPC;
          if (c < n) *reinterpret_cast<u32x4*>(seg + c) = v[u];
        }
      } else {
        for (int64_t c = t; c < n; c += 256) seg[c] = row[s0 + c];
      }
      __syncthreads();
      // kept columns j with source in [s0, s0 + n)
      int64_t jlo = s0 <= first ? 0 : (s0 - first + in_period - 1) / in_period;
      int64_t jhi = (s0 + n - 1 - first) / in_period + 1;
      if (jhi > kin) jhi = kin;
      for (int64_t j = jlo + t; j < jhi; j += 256) crow[j] = seg[first + in_period * j - s0];
    }
  }
  for (int64_t j = kin + t; j < jb.ldc; j += 256) crow[j] = from_f32<T>(0.0f);
}

// Gathers W[S_out][S_in] into Wc[kout][ldc] for up to kMaxCompactJobs layers
// in one launch; padding columns are 0. Kept rows and columns are arithmetic
// progressions (source row out_offset + out_period * i, source column
// in_offset + in_period * j). One block per compact row (the blocks of job 0
// first): the source row passes through LDS in segments read with coalesced
// 16-byte loads (vec: rows start 16-byte aligned and hold whole chunks; else
// element loads), then consecutive threads write consecutive kept columns.
template <typename T>
__global__ void __launch_bounds__(256) compact_weights_kernel(CompactJobs<T> jobs) {
  __shared__ __attribute__((aligned(16))) T seg[16384 / sizeof(T)];
  int64_t i = blockIdx.x;
  for (int q = 0; q < jobs.count; ++q) {
    if (i < jobs.job[q].rows) {
      compact_row(jobs.job[q], i, seg);
      return;
    }
    i -= jobs.job[q].rows;
  }
}

struct FcShape {
  int32_t B, K, N;
  int32_t kin, kout;                 // kept counts
  int32_t in_period, in_offset, out_period, out_offset;
  size_t esize;
  int64_t ldc;                       // compact weight row length
  bool compact_given;                // W argument is the compact matrix
  bool grad_compact;                 // dW is written as the compact dWc[kout][ldc]
  bool needs_compact;                // fwd / bwd_data gather W through a compact copy
  bool input_major;                  // W is stored W^T[K][N] (every output kept), dW as dW^T[K][N]
};

int check_desc(const ard_fc_desc* d, FcShape* s) {
  if (!d) return fail(ARD_ERR_INVALID_ARG, "desc is NULL");
  if (d->dtype != ARD_F32 && d->dtype != ARD_BF16)
    return fail(ARD_ERR_UNSUPPORTED, "dtype %d not supported", d->dtype);
  if (d->batch < 1 || d->in_features < 1 || d->out_features < 1)
    return fail(ARD_ERR_INVALID_ARG, "sizes must be >= 1 (batch %d, in %d, out %d)", d->batch,
                d->in_features, d->out_features);
  if (d->act != ARD_ACT_NONE && d->act != ARD_ACT_RELU)
    return fail(ARD_ERR_INVALID_ARG, "unknown activation %d", d->act);
  if (d->dropped != ARD_DROPPED_ZERO && d->dropped != ARD_DROPPED_SKIP)
    return fail(ARD_ERR_INVALID_ARG, "unknown dropped-output mode %d", d->dropped);
  if (d->weight_layout != ARD_WEIGHTS_FULL && d->weight_layout != ARD_WEIGHTS_COMPACT &&
      d->weight_layout != ARD_WEIGHTS_COMPACT_GRAD && d->weight_layout != ARD_WEIGHTS_INPUT_MAJOR)
    return fail(ARD_ERR_INVALID_ARG, "unknown weight layout %d", d->weight_layout);
  if (!(d->scale == d->scale) || d->scale == __builtin_inff() || d->scale == -__builtin_inff())
    return fail(ARD_ERR_INVALID_ARG, "scale must be finite");
  int st = check_row_plan(d->in_plan, d->in_features, "in_plan", false);
  if (st != ARD_OK) return st;
  st = check_row_plan(d->out_plan, d->out_features, "out_plan", false);
  if (st != ARD_OK) return st;
  s->B = d->batch;
  s->K = d->in_features;
  s->N = d->out_features;
  const bool in_all = !d->in_plan || d->in_plan->period == 1;
  const bool out_all = !d->out_plan || d->out_plan->period == 1;
  s->kin = in_all ? s->K : d->in_plan->kept;
  s->kout = out_all ? s->N : d->out_plan->kept;
  s->in_period = in_all ? 1 : d->in_plan->period;
  s->in_offset = in_all ? 0 : d->in_plan->offset;
  s->out_period = out_all ? 1 : d->out_plan->period;
  s->out_offset = out_all ? 0 : d->out_plan->offset;
  s->esize = d->dtype == ARD_BF16 ? 2 : 4;
  s->ldc = (static_cast<int64_t>(s->kin) + 7) / 8 * 8;
  s->compact_given = d->weight_layout == ARD_WEIGHTS_COMPACT || d->weight_layout == ARD_WEIGHTS_COMPACT_GRAD;
  s->grad_compact = d->weight_layout == ARD_WEIGHTS_COMPACT_GRAD;
  s->input_major = d->weight_layout == ARD_WEIGHTS_INPUT_MAJOR;
  // input-major rows are the inputs: the kept ones are whole rows, read in place
  s->needs_compact = !s->compact_given && !s->input_major && s->in_period > 1;
  if (s->input_major && !out_all)
    return fail(ARD_ERR_UNSUPPORTED, "input-major weights need every output kept (out_plan NULL or period 1)");
  return ARD_OK;
}

size_t al256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

size_t compact_bytes(const FcShape& s) { return static_cast<size_t>(s.kout) * s.ldc * s.esize; }

// Split-K partial floats of one problem under whichever kernel may run it.
template <typename T>
size_t problem_partials(int M, int N, int K) {
  size_t f = gemm_partial_floats<T>(M, N, K, 1, 1);
  const size_t h = fast_partial_floats<T>(M, N, K, 1, 1);
  return f > h ? f : h;
}

template <typename T>
size_t partial_bytes(const FcShape& s) {
  size_t f = problem_partials<T>(s.kout, s.B, s.kin);                 // fwd
  const size_t d = problem_partials<T>(s.kin, s.B, s.kout);           // bwd_data
  const size_t w = problem_partials<T>(s.kout, s.kin, s.B);           // bwd_weight
  f = f > d ? f : d;
  f = f > w ? f : w;
  return 4 * f;
}

size_t workspace_bytes(const FcShape& s, int dtype) {
  const size_t part = dtype == ARD_BF16 ? partial_bytes<bf16>(s) : partial_bytes<float>(s);
  return (s.needs_compact ? al256(compact_bytes(s)) : 0) + al256(part);
}

int check_ptr(const void* p, const char* name) {
  if (!p) return fail(ARD_ERR_INVALID_ARG, "%s is NULL", name);
  if (!aligned16(p)) return fail(ARD_ERR_INVALID_ARG, "%s is not 16-byte aligned", name);
  return ARD_OK;
}

int check_ws(const FcShape& s, int dtype, void* ws, size_t ws_bytes) {
  const size_t need = workspace_bytes(s, dtype);
  if (need == 0) return ARD_OK;
  if (!ws || ws_bytes < need)
    return fail(ARD_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need, ws_bytes);
  if (!aligned16(ws)) return fail(ARD_ERR_INVALID_ARG, "workspace is not 16-byte aligned");
  return ARD_OK;
}

// Rows of `ld` elements start 16-byte aligned.
inline bool vec_rows(int64_t ld, size_t esize) { return (ld * static_cast<int64_t>(esize)) % 16 == 0; }

template <typename T>
CompactJob<T> compact_job(const FcShape& s, const void* W, void* Wc) {
  CompactJob<T> j;
  j.W = static_cast<const T*>(W);
  j.K = s.K;
  j.out_period = s.out_period;
  j.out_offset = s.out_offset;
  j.in_period = s.in_period;
  j.in_offset = s.in_offset;
  j.kin = s.kin;
  j.ldc = s.ldc;
  j.vec = aligned16(W) && (static_cast<int64_t>(s.K) * static_cast<int64_t>(sizeof(T))) % 16 == 0;
  j.Wc = static_cast<T*>(Wc);
  j.rows = s.kout;
  return j;
}

template <typename T>
hipError_t launch_compact_jobs(const CompactJobs<T>& jobs, hipStream_t stream) {
  int64_t rows = 0;
  for (int q = 0; q < jobs.count; ++q) rows += jobs.job[q].rows;
  if (rows == 0) return hipSuccess;
  hipLaunchKernelGGL(compact_weights_kernel<T>, dim3(static_cast<unsigned>(rows)), dim3(256), 0, stream, jobs);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_compact(const FcShape& s, const void* W, void* Wc, hipStream_t stream) {
  CompactJobs<T> jobs = {};
  jobs.job[0] = compact_job<T>(s, W, Wc);
  jobs.count = 1;
  return launch_compact_jobs<T>(jobs, stream);
}

// The kept rows offset + period * i of a row-major matrix (row stride ld): a
// row-based pattern keeps an arithmetic progression of neurons (Sec. III-A,
// Eq. 1), so the gather folds into the view's base and row stride and the
// GEMM reads no index list. y, when set, is the gate source of the same shape.
GemmOperand kept_rows(const void* p, const void* y, int64_t ld, int32_t period, int32_t offset, size_t esize,
                      int32_t relu) {
  const int64_t skip = static_cast<int64_t>(offset) * ld * static_cast<int64_t>(esize);
  GemmOperand o = {};
  o.p = static_cast<const char*>(p) + skip;
  o.y = y ? static_cast<const char*>(y) + skip : nullptr;
  o.ld = ld * period;
  o.relu = relu;
  o.scale = 1.0f;
  return o;
}

// The output view of the fast GEMM: rows offset + period * i of a row-major
// matrix (row stride ld, elements of esize bytes) and columns col_offset +
// col_period * j, folded into base and strides like the operands; the bias
// and the output gate (same layout as the output) follow the rows.
GemmOutput strided_out(void* p, int64_t ld, size_t esize, int32_t period, int32_t offset, int32_t col_period,
                       int32_t col_offset, const float* bias, int32_t relu, float scale, const void* gate) {
  const int64_t skip = static_cast<int64_t>(offset) * ld + col_offset;
  GemmOutput c = {};
  c.p = static_cast<char*>(p) + skip * static_cast<int64_t>(esize);
  c.ld = ld * period;
  c.bias = bias ? bias + offset : nullptr;
  c.bias_stride = period;
  c.relu = relu;
  c.scale = scale;
  c.gate = gate ? static_cast<const char*>(gate) + skip * static_cast<int64_t>(esize) : nullptr;
  c.col_stride = col_period;
  return c;
}

// The view of W used by fwd / bwd_data: the full matrix's kept output rows (no
// input gather), a compact copy (given, or built into ws), or the kept input
// rows of an input-major W^T.
struct WeightView {
  GemmOperand op;
  float* partial;  // split-K partial sums in ws, or NULL
};

template <typename T>
int weight_view(const FcShape& s, const void* W, void* ws, hipStream_t stream, WeightView* v) {
  char* w = static_cast<char*>(ws);
  if (s.compact_given) {
    v->op = kept_rows(W, nullptr, s.ldc, 1, 0, sizeof(T), 0);
  } else if (s.input_major) {  // the kept input rows of W^T[K][N]
    v->op = kept_rows(W, nullptr, s.N, s.in_period, s.in_offset, sizeof(T), 0);
  } else if (s.needs_compact) {
    ARD_HIP_CHECK(launch_compact<T>(s, W, w, stream));
    v->op = kept_rows(w, nullptr, s.ldc, 1, 0, sizeof(T), 0);
    w += al256(compact_bytes(s));
  } else {
    v->op = kept_rows(W, nullptr, s.K, s.out_period, s.out_offset, sizeof(T), 0);
  }
  v->partial = ws ? reinterpret_cast<float*>(w) : nullptr;
  return ARD_OK;
}

template <typename T>
int fc_fwd_impl(const ard_fc_desc* d, const FcShape& s, const void* Xt, const void* W,
                const float* bias, void* Yt, void* ws, hipStream_t stream) {
  WeightView wv;
  int st = weight_view<T>(s, W, ws, stream, &wv);
  if (st != ARD_OK) return st;
  GemmArgs g = {};
  g.M = s.kout;
  g.N = s.B;
  g.K = s.kin;
  g.a = wv.op;
  g.b = kept_rows(Xt, nullptr, s.B, s.in_period, s.in_offset, sizeof(T), 0);
  g.c = strided_out(Yt, s.B, sizeof(T), s.out_period, s.out_offset, 1, 0, bias, d->act == ARD_ACT_RELU, d->scale,
                    nullptr);
  const bool a_vec = vec_rows(g.a.ld, sizeof(T));
  const bool b_vec = vec_rows(s.B, sizeof(T));
  if (s.input_major) {  // A(m, k) = W^T[in(k)][m]: m-contiguous
    if (fast_ok<true, true>(g, sizeof(T))) {
      ARD_HIP_CHECK((run_fast_gemm<T, true, true, T, EPI_FWD>(g, 1, stream, wv.partial)));
    } else {
      ARD_HIP_CHECK((run_gemm<T, T, MC_VEC, MC_ELEM, MC_VEC, MC_ELEM, false, false, EPI_FWD>(
          g, 1, a_vec, b_vec, stream, wv.partial)));
    }
  } else if (fast_ok<false, true>(g, sizeof(T))) {
    ARD_HIP_CHECK((run_fast_gemm<T, false, true, T, EPI_FWD>(g, 1, stream, wv.partial)));
  } else {
    ARD_HIP_CHECK((run_gemm<T, T, KC_VEC, KC_ELEM, MC_VEC, MC_ELEM, false, false, EPI_FWD>(
        g, 1, a_vec, b_vec, stream, wv.partial)));
  }
  if (d->dropped == ARD_DROPPED_ZERO && s.out_period > 1) {
    hipLaunchKernelGGL(zero_dropped_rows_kernel<T>, dim3(s.N), dim3(256), 0, stream,
                       static_cast<T*>(Yt), static_cast<int64_t>(s.B), s.B, s.out_period,
                       s.out_offset);
    ARD_LAUNCH_CHECK();
  }
  return ARD_OK;
}

// bwd_data as a GEMM: dXt[S_in] = W[S_out][S_in]^T G over the kept outputs.
template <typename T>
GemmArgs bwd_data_args(const ard_fc_desc* d, const FcShape& s, const void* dYt, const void* Yt,
                       const GemmOperand& wop, void* dXt, const void* Xgate) {
  GemmArgs g = {};
  g.M = s.kin;
  g.N = s.B;
  g.K = s.kout;
  // A(m, t) = W[out(t)][in(m)]: the view's rows are the contraction index.
  g.a = wop;
  // B(t, n) = dY[out(t)][n] * [Y > 0] (no gate when Yt is NULL: dY is already
  // the gated gradient); the 0/1 gate keeps bf16 operands exact, and scale is
  // applied to the fp32 accumulators in the epilogue, as is the optional gate
  // [Xgate > 0] of the layer below.
  const bool gated = d->act == ARD_ACT_RELU && Yt != nullptr;
  g.b = kept_rows(dYt, gated ? Yt : nullptr, s.B, s.out_period, s.out_offset, sizeof(T), gated);
  g.c = strided_out(dXt, s.B, sizeof(T), s.in_period, s.in_offset, 1, 0, nullptr, 0, d->scale, Xgate);
  return g;
}

// bwd_weight as a GEMM: dW[S_out][S_in] = G X^T over the batch (input-major:
// dW^T[S_in][:] = X G^T).
template <typename T>
GemmArgs bwd_weight_args(const ard_fc_desc* d, const FcShape& s, const void* Xt, const void* dYt,
                         const void* Yt, float* dW) {
  GemmArgs g = {};
  const bool gated = d->act == ARD_ACT_RELU && Yt != nullptr;
  if (s.input_major) {
    // dW^T[S_in][n] = X G^T over the batch: whole rows of N outputs
    g.M = s.kin;
    g.N = s.N;
    g.K = s.B;
    g.a = kept_rows(Xt, nullptr, s.B, s.in_period, s.in_offset, sizeof(T), 0);
    g.b = kept_rows(dYt, gated ? Yt : nullptr, s.B, 1, 0, sizeof(T), gated);
    g.c = strided_out(dW, s.N, sizeof(float), s.in_period, s.in_offset, 1, 0, nullptr, 0, d->scale, nullptr);
    return g;
  }
  g.M = s.kout;
  g.N = s.kin;
  g.K = s.B;
  g.a = kept_rows(dYt, gated ? Yt : nullptr, s.B, s.out_period, s.out_offset, sizeof(T), gated);
  g.b = kept_rows(Xt, nullptr, s.B, s.in_period, s.in_offset, sizeof(T), 0);
  if (s.grad_compact)  // dWc[i][j]: contiguous rows of ldc
    g.c = strided_out(dW, s.ldc, sizeof(float), 1, 0, 1, 0, nullptr, 0, d->scale, nullptr);
  else
    g.c = strided_out(dW, s.K, sizeof(float), s.out_period, s.out_offset, s.in_period, s.in_offset, nullptr, 0,
                      d->scale, nullptr);
  return g;
}

template <typename T>
int zero_dropped_inputs(const ard_fc_desc* d, const FcShape& s, void* dXt, hipStream_t stream) {
  if (d->dropped == ARD_DROPPED_ZERO && s.in_period > 1) {
    hipLaunchKernelGGL(zero_dropped_rows_kernel<T>, dim3(s.K), dim3(256), 0, stream,
                       static_cast<T*>(dXt), static_cast<int64_t>(s.B), s.B, s.in_period,
                       s.in_offset);
    ARD_LAUNCH_CHECK();
  }
  return ARD_OK;
}

// The bias gradient where the weight-gradient GEMM did not take it, and the
// ZERO-mode fills of dropped weight-gradient entries.
template <typename T>
int finish_bwd_weight(const ard_fc_desc* d, const FcShape& s, const void* dYt, const void* Yt, float* dW,
                      float* dbias, bool dbias_done, hipStream_t stream) {
  const bool gated = d->act == ARD_ACT_RELU && Yt != nullptr;
  if (dbias && s.kout > 0 && !dbias_done) {
    const int vec = aligned16(dYt) && (!gated || aligned16(Yt)) &&
                    (static_cast<int64_t>(s.B) * static_cast<int64_t>(sizeof(T))) % 16 == 0;
    hipLaunchKernelGGL(dbias_kernel<T>, dim3((s.kout + 3) / 4), dim3(256), 0, stream,
                       static_cast<const T*>(dYt), static_cast<const T*>(Yt), s.B, s.kout, s.out_period,
                       s.out_offset, d->scale, gated ? 1 : 0, vec, dbias);
    ARD_LAUNCH_CHECK();
  }
  if (d->dropped == ARD_DROPPED_ZERO && s.input_major && s.in_period > 1) {  // the dropped input rows of dW^T
    hipLaunchKernelGGL(zero_dropped_rows_kernel<float>, dim3(s.K), dim3(256), 0, stream, dW,
                       static_cast<int64_t>(s.N), s.N, s.in_period, s.in_offset);
    ARD_LAUNCH_CHECK();
    return ARD_OK;
  }
  if (d->dropped == ARD_DROPPED_ZERO && (s.out_period > 1 || s.in_period > 1)) {
    if (!s.grad_compact) {  // a compact gradient has no dropped entries
      hipLaunchKernelGGL(zero_dropped_weights_kernel, dim3(s.N), dim3(256), 0, stream, dW, s.K,
                         s.out_period, s.out_offset, s.in_period, s.in_offset);
      ARD_LAUNCH_CHECK();
    }
    if (dbias && s.out_period > 1) {
      hipLaunchKernelGGL(zero_dropped_rows_kernel<float>, dim3(s.N), dim3(64), 0, stream, dbias,
                         static_cast<int64_t>(1), 1, s.out_period, s.out_offset);
      ARD_LAUNCH_CHECK();
    }
  }
  return ARD_OK;
}

template <typename T>
int run_bwd_data(const ard_fc_desc* d, const FcShape& s, const GemmArgs& g, const void* Yt, void* dXt,
                 float* partial, hipStream_t stream) {
  const bool gated = d->act == ARD_ACT_RELU && Yt != nullptr;
  const bool a_vec = vec_rows(g.a.ld, sizeof(T));
  const bool b_vec = vec_rows(s.B, sizeof(T));
  if (s.input_major) {  // A(m, t) = W^T[in(m)][t]: k-contiguous rows
    if (fast_ok<false, true>(g, sizeof(T))) {
      ARD_HIP_CHECK((run_fast_gemm<T, false, true, T, EPI_FWD>(g, 1, stream, partial)));
    } else if (gated) {
      ARD_HIP_CHECK((run_gemm<T, T, KC_VEC, KC_ELEM, MC_VEC, MC_ELEM, false, true, EPI_FWD>(
          g, 1, a_vec, b_vec, stream, partial)));
    } else {
      ARD_HIP_CHECK((run_gemm<T, T, KC_VEC, KC_ELEM, MC_VEC, MC_ELEM, false, false, EPI_FWD>(
          g, 1, a_vec, b_vec, stream, partial)));
    }
  } else if (fast_ok<true, true>(g, sizeof(T))) {
    ARD_HIP_CHECK((run_fast_gemm<T, true, true, T, EPI_FWD>(g, 1, stream, partial)));
  } else if (gated) {
    ARD_HIP_CHECK((run_gemm<T, T, MC_VEC, MC_ELEM, MC_VEC, MC_ELEM, false, true, EPI_FWD>(
        g, 1, a_vec, b_vec, stream, partial)));
  } else {
    ARD_HIP_CHECK((run_gemm<T, T, MC_VEC, MC_ELEM, MC_VEC, MC_ELEM, false, false, EPI_FWD>(
        g, 1, a_vec, b_vec, stream, partial)));
  }
  return zero_dropped_inputs<T>(d, s, dXt, stream);
}

template <typename T>
int fc_bwd_data_impl(const ard_fc_desc* d, const FcShape& s, const void* dYt, const void* Yt,
                     const void* W, void* dXt, const void* Xgate, void* ws, hipStream_t stream) {
  WeightView wv;
  int st = weight_view<T>(s, W, ws, stream, &wv);
  if (st != ARD_OK) return st;
  return run_bwd_data<T>(d, s, bwd_data_args<T>(d, s, dYt, Yt, wv.op, dXt, Xgate), Yt, dXt, wv.partial, stream);
}

template <typename T>
int fc_bwd_weight_impl(const ard_fc_desc* d, const FcShape& s, const void* Xt, const void* dYt,
                       const void* Yt, float* dW, float* dbias, void* ws, hipStream_t stream) {
  GemmArgs g = bwd_weight_args<T>(d, s, Xt, dYt, Yt, dW);
  const bool gated = d->act == ARD_ACT_RELU && Yt != nullptr;
  const bool v = vec_rows(s.B, sizeof(T));
  float* partial = ws ? reinterpret_cast<float*>(static_cast<char*>(ws) +
                                                 (s.needs_compact ? al256(compact_bytes(s)) : 0))
                      : nullptr;
  bool dbias_done = false;
  if (s.input_major) {  // the bias gradient from dbias_kernel (G is the B operand here)
    if (fast_ok<false, false>(g, sizeof(T))) {
      ARD_HIP_CHECK((run_fast_gemm<T, false, false, float, EPI_FWD>(g, 1, stream, partial)));
    } else if (gated) {
      ARD_HIP_CHECK((run_gemm<T, float, KC_VEC, KC_ELEM, KC_VEC, KC_ELEM, false, true, EPI_FWD>(
          g, 1, v, v, stream, partial)));
    } else {
      ARD_HIP_CHECK((run_gemm<T, float, KC_VEC, KC_ELEM, KC_VEC, KC_ELEM, false, false, EPI_FWD>(
          g, 1, v, v, stream, partial)));
    }
  } else if (fast_ok<false, false>(g, sizeof(T))) {
    // dbias = scale * G 1: the row sums of A, taken by the same kernel
    if (dbias) {
      g.rsum = dbias + s.out_offset;
      g.rsum_ld = s.out_period;
    }
    ARD_HIP_CHECK((run_fast_gemm<T, false, false, float, EPI_FWD, true>(g, 1, stream, partial, &dbias_done)));
  } else if (gated) {
    ARD_HIP_CHECK((run_gemm<T, float, KC_VEC, KC_ELEM, KC_VEC, KC_ELEM, true, false, EPI_FWD>(
        g, 1, v, v, stream, partial)));
  } else {
    ARD_HIP_CHECK((run_gemm<T, float, KC_VEC, KC_ELEM, KC_VEC, KC_ELEM, false, false, EPI_FWD>(
        g, 1, v, v, stream, partial)));
  }
  return finish_bwd_weight<T>(d, s, dYt, Yt, dW, dbias, dbias_done, stream);
}

// bwd_data and bwd_weight of one layer. When both GEMMs take the fast 32x32
// configuration without a k split they run as one launch (the bias gradient
// from the weight-gradient GEMM's row sums); otherwise the two calls one
// after the other. The results are bitwise those of the separate calls: each
// output tile is computed by the same code on the same operands.
template <typename T>
int fc_bwd_impl(const ard_fc_desc* d, const FcShape& s, const void* Xt, const void* dYt, const void* Yt,
                const void* W, void* dXt, const void* Xgate, float* dW, float* dbias, void* ws,
                hipStream_t stream) {
  WeightView wv;
  int st = weight_view<T>(s, W, ws, stream, &wv);
  if (st != ARD_OK) return st;
  const GemmArgs gd = bwd_data_args<T>(d, s, dYt, Yt, wv.op, dXt, Xgate);
  GemmArgs gw = bwd_weight_args<T>(d, s, Xt, dYt, Yt, dW);
  if (!s.input_major && fast_ok<true, true>(gd, sizeof(T)) && fast_ok<false, false>(gw, sizeof(T)) &&
      fast_pair_ok<T>(gd, gw)) {
    if (dbias) {
      gw.rsum = dbias + s.out_offset;
      gw.rsum_ld = s.out_period;
      ARD_HIP_CHECK((launch_fast_pair<T, true, true, T, EPI_FWD, false, false, false, float, EPI_FWD, true>(
          gd, gw, stream)));
    } else {
      ARD_HIP_CHECK((launch_fast_pair<T, true, true, T, EPI_FWD, false, false, false, float, EPI_FWD, false>(
          gd, gw, stream)));
    }
    if ((st = zero_dropped_inputs<T>(d, s, dXt, stream)) != ARD_OK) return st;
    return finish_bwd_weight<T>(d, s, dYt, Yt, dW, dbias, dbias != nullptr, stream);
  }
  // the compact weights (if built into ws) are not needed past bwd_data,
  // whose partial sums lie behind them: bwd_weight's own call layout
  if ((st = run_bwd_data<T>(d, s, gd, Yt, dXt, wv.partial, stream)) != ARD_OK) return st;
  return fc_bwd_weight_impl<T>(d, s, Xt, dYt, Yt, dW, dbias, ws, stream);
}

}  // namespace
}  // namespace ard

// The scratch of ard_fc_fwd_noalloc: a file-scope device array, one copy per
// GPU the library runs on, held until the process ends. Its host-side name is
// only a stand-in for the symbol: host code uses the per-device address that
// hipGetSymbolAddress returns, never the name.
constexpr size_t kNoAllocScratchBytes = size_t{32} << 20;
static __device__ __align__(256) char scratch[kNoAllocScratchBytes];

namespace ard {
namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The current device's copy of scratch, looked up on the first call on that
// device (with it current) and kept.
int device_scratch(void** out) {
  int dev = -1;
  ARD_HIP_CHECK(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) return fail(ARD_ERR_UNSUPPORTED, "device %d: at most %d devices", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    ARD_HIP_CHECK(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return ARD_OK;
}

}  // namespace
}  // namespace ard

using namespace ard;

extern "C" {

int ard_fc_fwd_noalloc(const ard_fc_desc* desc, const void* Xt, const void* W, const float* bias, void* Yt,
                       void* stream) {
  clear_error();
  FcShape s;
  int st = check_desc(desc, &s);
  if (st != ARD_OK) return st;
  if ((st = check_ptr(Xt, "Xt")) || (st = check_ptr(W, "W")) || (st = check_ptr(Yt, "Yt")))
    return st;
  if (bias && !aligned16(bias)) return fail(ARD_ERR_INVALID_ARG, "bias is not 16-byte aligned");
  const size_t need = workspace_bytes(s, desc->dtype);
  if (need > kNoAllocScratchBytes)
    return fail(ARD_ERR_WORKSPACE,
                "the layer needs %zu bytes of scratch, the static scratch holds %zu (use ard_fc_fwd with a workspace)",
                need, kNoAllocScratchBytes);
  void* ws = nullptr;
  if (need > 0 && (st = device_scratch(&ws)) != ARD_OK) return st;
  hipStream_t sm = static_cast<hipStream_t>(stream);
  if (desc->dtype == ARD_BF16) return fc_fwd_impl<bf16>(desc, s, Xt, W, bias, Yt, ws, sm);
  return fc_fwd_impl<float>(desc, s, Xt, W, bias, Yt, ws, sm);
}

int ard_plan_rows(int32_t n, int32_t period, int32_t offset, int32_t* d_idx, ard_row_plan* plan,
                  void* stream) {
  clear_error();
  if (!plan) return fail(ARD_ERR_INVALID_ARG, "plan is NULL");
  if (n < 1) return fail(ARD_ERR_INVALID_ARG, "n must be >= 1");
  if (period < 1 || offset < 0 || offset >= period)
    return fail(ARD_ERR_INVALID_ARG, "invalid pattern (period %d, offset %d)", period, offset);
  const int32_t kept = kept_count(n, period, offset);
  plan->n = n;
  plan->period = period;
  plan->offset = offset;
  plan->kept = kept;
  plan->d_idx = d_idx;
  if (kept > 0 && d_idx) {
    hipLaunchKernelGGL(plan_rows_kernel, dim3((kept + 255) / 256), dim3(256), 0,
                       static_cast<hipStream_t>(stream), d_idx, kept, period, offset);
    ARD_LAUNCH_CHECK();
  }
  return ARD_OK;
}

int32_t ard_fc_compact_ld(const ard_fc_desc* desc) {
  FcShape s;
  if (check_desc(desc, &s) != ARD_OK) return -1;
  return static_cast<int32_t>(s.ldc);
}

size_t ard_fc_compact_bytes(const ard_fc_desc* desc) {
  FcShape s;
  if (check_desc(desc, &s) != ARD_OK) return 0;
  return compact_bytes(s);
}

int ard_fc_compact_weights(const ard_fc_desc* desc, const void* W, void* Wc, void* stream) {
  clear_error();
  FcShape s;
  int st = check_desc(desc, &s);
  if (st != ARD_OK) return st;
  if (s.input_major) return fail(ARD_ERR_INVALID_ARG, "input-major weights have no compact copy");
  if ((st = check_ptr(W, "W")) || (st = check_ptr(Wc, "Wc"))) return st;
  hipStream_t sm = static_cast<hipStream_t>(stream);
  if (desc->dtype == ARD_BF16) {
    ARD_HIP_CHECK(launch_compact<bf16>(s, W, Wc, sm));
  } else {
    ARD_HIP_CHECK(launch_compact<float>(s, W, Wc, sm));
  }
  return ARD_OK;
}

int ard_fc_compact_weights_batch(int32_t count, const ard_fc_desc* const* descs, const void* const* W,
                                 void* const* Wc, void* stream) {
  clear_error();
  if (count < 1 || count > kMaxCompactJobs)
    return fail(ARD_ERR_INVALID_ARG, "count %d outside 1..%d", count, kMaxCompactJobs);
  if (!descs || !W || !Wc) return fail(ARD_ERR_INVALID_ARG, "descs, W or Wc is NULL");
  CompactJobs<float> jf = {};
  CompactJobs<bf16> jb = {};
  const int dtype = descs[0] ? descs[0]->dtype : -1;
  for (int q = 0; q < count; ++q) {
    FcShape s;
    int st = check_desc(descs[q], &s);
    if (st != ARD_OK) return st;
    if (descs[q]->dtype != dtype) return fail(ARD_ERR_INVALID_ARG, "descs[%d]: dtypes differ", q);
    if (s.input_major) return fail(ARD_ERR_INVALID_ARG, "descs[%d]: input-major weights have no compact copy", q);
    if ((st = check_ptr(W[q], "W")) || (st = check_ptr(Wc[q], "Wc"))) return st;
    jf.job[q] = compact_job<float>(s, W[q], Wc[q]);
    jb.job[q] = compact_job<bf16>(s, W[q], Wc[q]);
  }
  jf.count = jb.count = count;
  hipStream_t sm = static_cast<hipStream_t>(stream);
  if (dtype == ARD_BF16) {
    ARD_HIP_CHECK(launch_compact_jobs<bf16>(jb, sm));
  } else {
    ARD_HIP_CHECK(launch_compact_jobs<float>(jf, sm));
  }
  return ARD_OK;
}

int ard_fc_sgd_momentum(const ard_fc_desc* desc, void* W, float* V, const float* dW, float* bias, float* Vb,
                        const float* dbias, float lr, float momentum, void* stream) {
  clear_error();
  FcShape s;
  int st = check_desc(desc, &s);
  if (st != ARD_OK) return st;
  if (!W || !V || !dW) return fail(ARD_ERR_INVALID_ARG, "W, V or dW is NULL");
  if ((bias == nullptr) != (Vb == nullptr) || (bias == nullptr) != (dbias == nullptr))
    return fail(ARD_ERR_INVALID_ARG, "bias, Vb and dbias must be all given or all NULL");
  if (reinterpret_cast<uintptr_t>(W) % s.esize || reinterpret_cast<uintptr_t>(V) % 4 ||
      reinterpret_cast<uintptr_t>(dW) % 4)
    return fail(ARD_ERR_INVALID_ARG, "W, V or dW is not aligned to its element size");
  if (!(lr == lr) || !(momentum == momentum)) return fail(ARD_ERR_INVALID_ARG, "lr and momentum must be numbers");
  if (s.kout == 0) return ARD_OK;
  hipStream_t sm = static_cast<hipStream_t>(stream);
  if (s.input_major) {
    // the kept input rows of W^T, V^T and dW^T, whole (every output kept);
    // the bias of every output as one more row
    if (s.kin > 0) {
      if (desc->dtype == ARD_BF16)
        hipLaunchKernelGGL(sgd_momentum_kernel<bf16>, dim3(s.kin), dim3(256), 0, sm, static_cast<bf16*>(W), V, dW,
                           s.N, int64_t{0}, s.in_period, s.in_offset, 1, 0, s.N, nullptr, nullptr, nullptr, lr,
                           momentum);
      else
        hipLaunchKernelGGL(sgd_momentum_kernel<float>, dim3(s.kin), dim3(256), 0, sm, static_cast<float*>(W), V,
                           dW, s.N, int64_t{0}, s.in_period, s.in_offset, 1, 0, s.N, nullptr, nullptr, nullptr, lr,
                           momentum);
      ARD_LAUNCH_CHECK();
    }
    if (bias) {
      hipLaunchKernelGGL(sgd_momentum_kernel<float>, dim3(1), dim3(256), 0, sm, bias, Vb, dbias, s.N, int64_t{0}, 1,
                         0, 1, 0, s.N, nullptr, nullptr, nullptr, lr, momentum);
      ARD_LAUNCH_CHECK();
    }
    return ARD_OK;
  }
  const int64_t ldg = s.grad_compact ? s.ldc : 0;
  if (desc->dtype == ARD_BF16)
    hipLaunchKernelGGL(sgd_momentum_kernel<bf16>, dim3(s.kout), dim3(256), 0, sm, static_cast<bf16*>(W), V, dW, s.K,
                       ldg, s.out_period, s.out_offset, s.in_period, s.in_offset, s.kin, bias, Vb, dbias, lr,
                       momentum);
  else
    hipLaunchKernelGGL(sgd_momentum_kernel<float>, dim3(s.kout), dim3(256), 0, sm, static_cast<float*>(W), V, dW,
                       s.K, ldg, s.out_period, s.out_offset, s.in_period, s.in_offset, s.kin, bias, Vb, dbias, lr,
                       momentum);
  ARD_LAUNCH_CHECK();
  return ARD_OK;
}

size_t ard_fc_workspace_bytes(const ard_fc_desc* desc) {
  FcShape s;
  if (check_desc(desc, &s) != ARD_OK) return 0;
  return workspace_bytes(s, desc->dtype);
}

int ard_fc_fwd(const ard_fc_desc* desc, const void* Xt, const void* W, const float* bias, void* Yt,
               void* ws, size_t ws_bytes, void* stream) {
  clear_error();
  FcShape s;
  int st = check_desc(desc, &s);
  if (st != ARD_OK) return st;
  if ((st = check_ptr(Xt, "Xt")) || (st = check_ptr(W, "W")) || (st = check_ptr(Yt, "Yt")))
    return st;
  if (bias && !aligned16(bias)) return fail(ARD_ERR_INVALID_ARG, "bias is not 16-byte aligned");
  if ((st = check_ws(s, desc->dtype, ws, ws_bytes))) return st;
  hipStream_t sm = static_cast<hipStream_t>(stream);
  if (desc->dtype == ARD_BF16) return fc_fwd_impl<bf16>(desc, s, Xt, W, bias, Yt, ws, sm);
  return fc_fwd_impl<float>(desc, s, Xt, W, bias, Yt, ws, sm);
}

int ard_fc_bwd_data(const ard_fc_desc* desc, const void* dYt, const void* Yt, const void* W,
                    void* dXt, const void* Xgate, void* ws, size_t ws_bytes, void* stream) {
  clear_error();
  FcShape s;
  int st = check_desc(desc, &s);
  if (st != ARD_OK) return st;
  if ((st = check_ptr(dYt, "dYt")) || (st = check_ptr(W, "W")) || (st = check_ptr(dXt, "dXt")))
    return st;
  if (Yt && !aligned16(Yt)) return fail(ARD_ERR_INVALID_ARG, "Yt is not 16-byte aligned");
  if (Xgate && !aligned16(Xgate)) return fail(ARD_ERR_INVALID_ARG, "Xgate is not 16-byte aligned");
  if ((st = check_ws(s, desc->dtype, ws, ws_bytes))) return st;
  hipStream_t sm = static_cast<hipStream_t>(stream);
  if (desc->dtype == ARD_BF16) return fc_bwd_data_impl<bf16>(desc, s, dYt, Yt, W, dXt, Xgate, ws, sm);
  return fc_bwd_data_impl<float>(desc, s, dYt, Yt, W, dXt, Xgate, ws, sm);
}

int ard_fc_bwd(const ard_fc_desc* desc, const void* Xt, const void* dYt, const void* Yt, const void* W,
               void* dXt, const void* Xgate, float* dW, float* dbias, void* ws, size_t ws_bytes, void* stream) {
  clear_error();
  FcShape s;
  int st = check_desc(desc, &s);
  if (st != ARD_OK) return st;
  if ((st = check_ptr(Xt, "Xt")) || (st = check_ptr(dYt, "dYt")) || (st = check_ptr(W, "W")) ||
      (st = check_ptr(dXt, "dXt")) || (st = check_ptr(dW, "dW")))
    return st;
  if (Yt && !aligned16(Yt)) return fail(ARD_ERR_INVALID_ARG, "Yt is not 16-byte aligned");
  if (Xgate && !aligned16(Xgate)) return fail(ARD_ERR_INVALID_ARG, "Xgate is not 16-byte aligned");
  if (dbias && !aligned16(dbias)) return fail(ARD_ERR_INVALID_ARG, "dbias is not 16-byte aligned");
  if ((st = check_ws(s, desc->dtype, ws, ws_bytes))) return st;
  hipStream_t sm = static_cast<hipStream_t>(stream);
  if (desc->dtype == ARD_BF16) return fc_bwd_impl<bf16>(desc, s, Xt, dYt, Yt, W, dXt, Xgate, dW, dbias, ws, sm);
  return fc_bwd_impl<float>(desc, s, Xt, dYt, Yt, W, dXt, Xgate, dW, dbias, ws, sm);
}

int ard_fc_bwd_weight(const ard_fc_desc* desc, const void* Xt, const void* dYt, const void* Yt,
                      float* dW, float* dbias, void* ws, size_t ws_bytes, void* stream) {
  clear_error();
  FcShape s;
  int st = check_desc(desc, &s);
  if (st != ARD_OK) return st;
  if ((st = check_ptr(Xt, "Xt")) || (st = check_ptr(dYt, "dYt")) || (st = check_ptr(dW, "dW")))
    return st;
  if (Yt && !aligned16(Yt)) return fail(ARD_ERR_INVALID_ARG, "Yt is not 16-byte aligned");
  if (dbias && !aligned16(dbias)) return fail(ARD_ERR_INVALID_ARG, "dbias is not 16-byte aligned");
  if ((st = check_ws(s, desc->dtype, ws, ws_bytes))) return st;
  hipStream_t sm = static_cast<hipStream_t>(stream);
  if (desc->dtype == ARD_BF16)
    return fc_bwd_weight_impl<bf16>(desc, s, Xt, dYt, Yt, dW, dbias, ws, sm);
  return fc_bwd_weight_impl<float>(desc, s, Xt, dYt, Yt, dW, dbias, ws, sm);
}

}  // extern "C"
