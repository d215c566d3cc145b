/*
 * ard.h - Approximate Random Dropout hot path for AMD Instinct MI355X (gfx950).
 *
 * Method: Song et al., "Approximate Random Dropout for DNN training
 * acceleration in GPGPU" (arXiv 1805.08939). Random dropout is replaced by
 * regular patterns so that dropped neurons (row-based pattern, Sec. III-A) and
 * dropped weight tiles (tile-based pattern, Sec. III-B) are skipped outright:
 * the GEMMs below never load, multiply or store them. Each iteration a pattern
 * is sampled from a distribution K (Sec. III-D) that the SGD-based search of
 * Sec. III-C (Alg. 1) produces.
 *
 * Conventions shared by every call:
 *  - Every function returns an ard_status (0 = ARD_OK). On failure a
 *    thread-local message is available from ard_last_error(), and no device
 *    work has been enqueued. Nothing aborts or throws across this boundary.
 *  - Buffers are caller-owned. The library never allocates or frees device
 *    memory; where a call needs scratch space its size is queried first and the
 *    caller passes it in (ws, ws_bytes).
 *  - "stream" is a hipStream_t passed as void* (NULL = the null stream). Device
 *    calls are asynchronous and stream-ordered; the library never synchronises.
 *  - Device pointers must be 16-byte aligned. Matrices are dense row-major
 *    with the row lengths stated at each argument.
 *  - Activations are stored feature-major: Xt[K][B] holds input feature k of
 *    every sample in one contiguous row (the transpose of the math layout
 *    X[B][K]), so that a dropped neuron is a skipped row. Weights are stored
 *    output-major, W[N][K]: one row per output neuron.
 *  - dtype ARD_BF16 means bf16 activations, weights and activation gradients
 *    with fp32 accumulation; bias, weight and bias gradients are always fp32.
 */
#ifndef ARD_H
#define ARD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ARD_VERSION 3

typedef enum {
  ARD_OK = 0,
  ARD_ERR_INVALID_ARG = 1,   /* a size, pointer, pattern or option is invalid */
  ARD_ERR_UNSUPPORTED = 2,   /* valid but not implemented (e.g. a dtype) */
  ARD_ERR_HIP = 3,           /* the HIP runtime reported an error */
  ARD_ERR_NOT_CONVERGED = 4, /* the search hit max_iters; its output is the last iterate */
  ARD_ERR_WORKSPACE = 5      /* ws is NULL or smaller than the queried size */
} ard_status;

typedef enum { ARD_F32 = 0, ARD_BF16 = 1 } ard_dtype;

/* Human-readable name of a status code (static string). */
const char* ard_status_string(int status);
/* Detail of the last failure on the calling thread ("" if none). */
const char* ard_last_error(void);
/* ARD_VERSION of the built library. */
int ard_version(void);

/* ------------------------------------------------------------------------ */
/* Pattern distribution search (host).                                      */
/* ------------------------------------------------------------------------ */
/*
 * Alg. 1 (Sec. III-C): find K = softmax(v) over periods 1..n_max minimising
 *     lambda1 * (K . p_u - p)^2 + (1 - lambda1) * (1/n_max) * sum_i K_i log K_i,
 * p_u[i] = (i - 1) / i, by gradient descent on v from v = 0 until the change of
 * the loss is below `threshold`.
 *   mode ARD_SEARCH_PLAIN : v -= lr * dL/dv  (the paper's iteration)
 *   mode ARD_SEARCH_MIRROR: v -= lr * dL/dK  (entropic mirror descent; same
 *                           minimiser, far fewer iterations for large n_max)
 */
enum { ARD_SEARCH_PLAIN = 0, ARD_SEARCH_MIRROR = 1 };

typedef struct {
  int32_t n_max;      /* number of candidate periods, >= 1 */
  int32_t mode;       /* ARD_SEARCH_PLAIN or ARD_SEARCH_MIRROR */
  double lambda1;     /* weight of the rate term, in (0, 1); lambda2 = 1 - lambda1 */
  double lr;          /* step size, > 0 */
  double threshold;   /* stop when |loss_t - loss_{t-1}| < threshold, >= 0 */
  int64_t max_iters;  /* >= 1 */
} ard_search_opts;

typedef struct {
  int64_t iters;        /* iterations run */
  double loss;          /* final loss */
  double p_global;      /* Eq. 3: sum_i K_i (i - 1) / i */
  double kkt_residual;  /* max_i dL/dK_i - min_i dL/dK_i (0 at the optimum) */
  int32_t converged;    /* 1 if the stop rule fired */
  int32_t reserved;
} ard_search_info;

/* Defaults: n_max 16, PLAIN, lambda1 0.99, lr 10, threshold 1e-15, max_iters 1e6. */
void ard_search_opts_default(ard_search_opts* opts);

/*
 * Search K for target rate p. K_out: host array of opts->n_max doubles
 * (caller-owned). info may be NULL. opts NULL = defaults.
 * p = 0 returns K = e_1 exactly without iterating. p must satisfy
 * 0 <= p < (n_max - 1) / n_max, else ARD_ERR_INVALID_ARG. If max_iters is
 * reached K_out holds the last iterate and ARD_ERR_NOT_CONVERGED is returned.
 */
int ard_search_distribution(double p, const ard_search_opts* opts, double* K_out,
                            ard_search_info* info);

/* ------------------------------------------------------------------------ */
/* Pattern sampling (host).                                                 */
/* ------------------------------------------------------------------------ */
/*
 * A row pattern (Sec. III-A, Eq. 1): neuron j (0-based) is KEPT iff
 * j % period == offset. The paper's (dp, b) is (period, offset + 1).
 */
typedef struct {
  int32_t period;  /* >= 1; 1 = no dropout */
  int32_t offset;  /* 0 <= offset < period */
} ard_row_pattern;

/*
 * Sec. III-D: draw period ~ K (inverse CDF over sequential fp64 partial sums)
 * and offset uniform in [0, period) from the counter-based SplitMix64 stream of
 * (seed, stream, iter): initial state seed ^ ((stream << 40) | iter),
 * stream < 2^24, iter < 2^40. Reproducible from any iteration; one stream per
 * dropout layer. K: host, n_max entries, non-negative with a positive entry.
 */
int ard_sample_row_pattern(const double* K, int32_t n_max, uint64_t seed, uint32_t stream,
                           uint64_t iter, ard_row_pattern* out);

/* Kept count of n neurons under (period, offset): 0 if offset >= n, else
 * ceil((n - offset) / period). Returns -1 on invalid arguments. */
int32_t ard_row_kept(int32_t n, int32_t period, int32_t offset);

/*
 * Tile bitmaps over the tiles_n x tiles_k tile grid of W[N][K] (Sec. III-B).
 * Tile t = tn * tiles_k + tk (row-major) is KEPT iff bit t is set, stored in
 * word t / 32 at bit t % 32. bits: host, ceil(tiles_n * tiles_k / 32) words.
 *   _tdp      : kept iff t % period == offset (the paper's tile pattern)
 *   _bernoulli: tile t takes the t-th uniform of the (seed, stream, iter)
 *               stream and is kept iff it is >= p (DropConnect-style tiles)
 */
int ard_tile_bitmap_tdp(int32_t tiles_n, int32_t tiles_k, int32_t period, int32_t offset,
                        uint32_t* bits);
int ard_tile_bitmap_bernoulli(int32_t tiles_n, int32_t tiles_k, double p, uint64_t seed,
                              uint32_t stream, uint64_t iter, uint32_t* bits);
/* Number of set bits among the first `total` bits (host). -1 on invalid args. */
int32_t ard_bitmap_popcount(const uint32_t* bits, int32_t total);

/* ------------------------------------------------------------------------ */
/* Compaction: patterns -> gather lists (device kernels).                   */
/* ------------------------------------------------------------------------ */
/*
 * The compact index list of a row pattern (Sec. III-A: the compact matrices are
 * built from the kept rows only). Fills the plan struct (host) with n, the
 * pattern and the host-known kept count, so that later launches need no device
 * readback, and d_idx[0..kept) with the kept neuron indices in ascending order.
 * d_idx: device, capacity >= ard_row_kept(n, period, offset), caller-owned; or
 * NULL for a list-free plan (nothing is launched). The kept set of a row pattern
 * is the arithmetic progression offset + period * i, so the FC calls fold it
 * into strided operand and output views and never read the list: they accept
 * list-free plans. The LSTM calls read the list and reject a list-free plan
 * that drops units (ARD_ERR_INVALID_ARG).
 */
typedef struct {
  int32_t n;
  int32_t period;
  int32_t offset;
  int32_t kept;
  int32_t* d_idx;
} ard_row_plan;

int ard_plan_rows(int32_t n, int32_t period, int32_t offset, int32_t* d_idx, ard_row_plan* plan,
                  void* stream);

/*
 * Tile plan (Sec. III-B: only non-dropped tiles are fetched). From the device
 * bitmap d_bits of an N x K weight matrix in tile x tile tiles, a scan kernel
 * writes into the workspace:
 *   row_ptr[tiles_n + 1], row_cols[nnz]  kept tile columns per tile row (CSR)
 *   col_ptr[tiles_k + 1], col_rows[nnz]  kept tile rows per tile column (CSC)
 *   flat[nnz]                            kept linear tile indices
 *   chunks[4 + 8 * groups]               groups of up to 4 kept tiles of one
 *                                        tile row, in row order: chunks[0] =
 *                                        groups, chunks[1..3] = 0, then per
 *                                        group 8 ints: tile row, first position
 *                                        in row_cols, tile count n, 0, the n
 *                                        tile columns and the last of them
 *                                        repeated up to 4 entries
 * all ascending. nnz must equal the popcount of the bitmap (host-known, see
 * ard_bitmap_popcount). tile must be 32 or 64, n and k multiples of it, and
 * the tile grid at most 4096 tiles per side.
 */
typedef struct {
  int32_t n, k, tile, tiles_n, tiles_k;
  int32_t nnz;  /* kept tiles, or -1 when known on the device only */
  const uint32_t* d_bits;
  int32_t* d_row_ptr;
  int32_t* d_row_cols;
  int32_t* d_col_ptr;
  int32_t* d_col_rows;
  int32_t* d_flat;
  int32_t* d_chunks;
} ard_tile_plan;

size_t ard_tile_plan_workspace_bytes(int32_t tiles_n, int32_t tiles_k);
int ard_plan_tiles(int32_t n, int32_t k, int32_t tile, const uint32_t* d_bits, int32_t nnz,
                   void* d_ws, size_t ws_bytes, ard_tile_plan* plan, void* stream);

/*
 * The same plan with the bitmap sampled on the device, in the plan kernel:
 * the bits of ard_tile_bitmap_bernoulli(tiles_n, tiles_k, p, seed, stream_id,
 * iter) exactly (each tile's draw of the counter-based stream computed on its
 * own), written to d_bits (device, ceil(tiles_n * tiles_k / 32) words,
 * caller-owned, read by the layer calls in ZERO mode). For patterns drawn
 * every step with no host sampling or upload. The kept count then exists on
 * the device only: plan->nnz = -1, row_ptr[tiles_n] holds it, and the layer
 * calls launch for the largest possible count (surplus workgroups exit at
 * once). Errors as for ard_plan_tiles, and for p outside [0, 1], stream_id
 * >= 2^24 or iter >= 2^40.
 */
int ard_plan_tiles_bernoulli(int32_t n, int32_t k, int32_t tile, double p, uint64_t seed,
                             uint32_t stream_id, uint64_t iter, uint32_t* d_bits, void* d_ws,
                             size_t ws_bytes, ard_tile_plan* plan, void* stream);

/* ------------------------------------------------------------------------ */
/* Fully connected layer under row patterns (device).                       */
/* ------------------------------------------------------------------------ */
/*
 * Sec. III-A with the dropout layer folded in (Sec. III-B, last paragraph):
 * in_plan is the pattern of the layer's input neurons (the previous layer's
 * output pattern), out_plan that of its outputs; NULL or period 1 = all kept.
 * With S_in, S_out the kept sets and G = scale * act'(.) * dY on kept rows:
 *   fwd       Yt[S_out,:] = scale * act(W[S_out,S_in] Xt[S_in,:] + bias[S_out])
 *   bwd_data  dXt[S_in,:] = W[S_out,S_in]^T G[S_out,:]
 *   bwd_weight dW[S_out,S_in] = G[S_out,:] Xt[S_in,:]^T,  dbias[S_out] = G 1
 * Only kept rows/columns are read or computed. Entries outside the kept sets
 * are written 0 (ARD_DROPPED_ZERO) or left untouched (ARD_DROPPED_SKIP).
 * The ReLU derivative is taken from the stored forward output: [Yt > 0].
 * Layouts: Xt[K][B], W[N][K], bias[N] fp32, Yt and dYt[N][B], dXt[K][B],
 * dW[N][K] fp32, dbias[N] fp32 (K = in_features, N = out_features, B = batch).
 */
typedef enum { ARD_ACT_NONE = 0, ARD_ACT_RELU = 1 } ard_act;
typedef enum { ARD_DROPPED_ZERO = 0, ARD_DROPPED_SKIP = 1 } ard_dropped;
/*
 * How the W argument of fwd / bwd_data (and the dW of bwd_weight) is stored:
 *   ARD_WEIGHTS_FULL        : the full W[N][K]; dW[N][K].
 *   ARD_WEIGHTS_COMPACT     : the compact Wc[kept_out][ldc] written by
 *                             ard_fc_compact_weights for this descriptor's
 *                             patterns, Wc[i][j] = W[S_out(i)][S_in(j)]
 *                             (Sec. III-A's compact weight matrix),
 *                             ldc = ard_fc_compact_ld(desc); dW[N][K].
 *   ARD_WEIGHTS_COMPACT_GRAD: W as for COMPACT, and bwd_weight writes the
 *                             gradient of the compact matrix,
 *                             dWc[i][j] = dW[S_out(i)][S_in(j)], as fp32
 *                             [kept_out][ldc] (columns kept_in..ldc-1 are not
 *                             written; the dropped/ZERO rule does not apply to
 *                             it). Every store of dW is then a whole row run:
 *                             with a strided input side, a full-layout dW
 *                             leaves every 32-byte sector partly written.
 *                             ard_fc_sgd_momentum takes dW in this layout too.
 *   ARD_WEIGHTS_INPUT_MAJOR : W stored input-major, W^T[K][N] (row k holds
 *                             the weights of input k to every output), dW
 *                             likewise dW^T[K][N], V of ard_fc_sgd_momentum
 *                             too. Every output must be kept (out_plan NULL
 *                             or of period 1, else ARD_ERR_UNSUPPORTED); a
 *                             dropped input is then a skipped row, so no
 *                             compact copy is built or accepted (the compact
 *                             calls return ARD_ERR_INVALID_ARG). For a last
 *                             layer, whose outputs carry no pattern.
 * With FULL weights and a gathered input side, fwd and bwd_data build the
 * compact copy in their workspace themselves; a training step that compacts
 * once and passes COMPACT to both saves one pass over W. With an ungathered
 * input side FULL reads the kept rows of W in place, and where those rows do
 * not start on a 16-byte boundary the products run on the general kernel:
 * Y and dX of FULL and COMPACT then agree up to the order of rounding, not
 * bit for bit.
 */
typedef enum {
  ARD_WEIGHTS_FULL = 0,
  ARD_WEIGHTS_COMPACT = 1,
  ARD_WEIGHTS_COMPACT_GRAD = 2,
  ARD_WEIGHTS_INPUT_MAJOR = 3
} ard_weight_layout;

typedef struct {
  int32_t dtype;        /* ard_dtype */
  int32_t batch;        /* B >= 1 */
  int32_t in_features;  /* K >= 1 */
  int32_t out_features; /* N >= 1 */
  const ard_row_plan* in_plan;   /* n == K, or NULL */
  const ard_row_plan* out_plan;  /* n == N, or NULL */
  float scale;          /* multiplies kept outputs (1 = pure mask) */
  int32_t act;          /* ard_act */
  int32_t dropped;      /* ard_dropped */
  int32_t weight_layout;/* ard_weight_layout of the W argument */
} ard_fc_desc;

/* Row length (elements) of the compact weight matrix: kept inputs rounded up
 * to a multiple of 8. -1 on an invalid descriptor. */
int32_t ard_fc_compact_ld(const ard_fc_desc* desc);
/* Bytes of the compact weight matrix (kept_out * ldc * element size). */
size_t ard_fc_compact_bytes(const ard_fc_desc* desc);
/* Gathers W[S_out][S_in] (W full, [N][K]) into Wc (device, compact bytes,
 * caller-owned); padding columns are written 0. */
int ard_fc_compact_weights(const ard_fc_desc* desc, const void* W, void* Wc, void* stream);
/* The same for count (1..4) layers of one dtype in one kernel launch: layer q
 * gathers W[q] (full) into Wc[q] under descs[q]. A network's compact weights
 * for one step's patterns come from one launch instead of one per layer.
 * descs, W and Wc are host arrays of count entries. */
int ard_fc_compact_weights_batch(int32_t count, const ard_fc_desc* const* descs, const void* const* W,
                                 void* const* Wc, void* stream);

/* Workspace (bytes) that fwd, bwd_data and bwd_weight of this descriptor need:
 * split-contraction partial sums for small output grids and, for FULL weights
 * with a gathered input side, the compact weight copy. Depends on the kept
 * counts, so query it per pattern (or once for the dense pattern, which bounds
 * every other one of the same layer). ws may be NULL when this is 0. */
size_t ard_fc_workspace_bytes(const ard_fc_desc* desc);

int ard_fc_fwd(const ard_fc_desc* desc, const void* Xt, const void* W, const float* bias,
               void* Yt, void* ws, size_t ws_bytes, void* stream);
/*
 * Backward gating. With act == ARD_ACT_RELU the output derivative is gated by
 * [Yt > 0], Yt being the stored forward output. Yt == NULL means dYt is
 * already gated (for instance written by the layer above through Xgate) and is
 * used as is. Xgate (optional, [K][B], dtype) is this layer's input as
 * produced by a ReLU: when given, dXt is multiplied by [Xgate > 0], so that it
 * is directly the gated gradient of the layer below. Both gates are 0/1.
 */
int ard_fc_bwd_data(const ard_fc_desc* desc, const void* dYt, const void* Yt, const void* W,
                    void* dXt, const void* Xgate, void* ws, size_t ws_bytes, void* stream);
/*
 * ard_fc_fwd for callers that cannot allocate device memory or pass a
 * workspace: code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc. The same computation, kernels and results, bit for bit,
 * as ard_fc_fwd with a workspace; the scratch the layer needs (the compact
 * weight copy of a gathered input side, split-contraction partial sums) comes
 * from a static device array of the library instead: 32 MiB per GPU, kept
 * from the first such call on that GPU until the process ends. A layer whose
 * ard_fc_workspace_bytes exceeds 32 MiB is rejected with ARD_ERR_WORKSPACE
 * before any launch. Nothing in the scratch needs to start at zero (a call
 * reads only what it wrote), but every call on one GPU shares that GPU's
 * array: calls that overlap in time on one GPU (other streams, other threads)
 * race and must be serialised by the caller. No call allocates or frees.
 */
int ard_fc_fwd_noalloc(const ard_fc_desc* desc, const void* Xt, const void* W, const float* bias,
                       void* Yt, void* stream);
/* dbias may be NULL. */
int ard_fc_bwd_weight(const ard_fc_desc* desc, const void* Xt, const void* dYt, const void* Yt,
                      float* dW, float* dbias, void* ws, size_t ws_bytes, void* stream);
/*
 * The whole backward of one layer (Sec. III-A applied to both backward
 * products): ard_fc_bwd_data followed by ard_fc_bwd_weight, with the same
 * arguments, layouts, workspace and results, bit for bit. When both products
 * are small enough to take the 32 x 32 output tiles without a split
 * contraction they run as one kernel launch (the tiles of dXt, then those of
 * dW), which saves one launch's fixed cost per layer. dbias may be NULL.
 */
int ard_fc_bwd(const ard_fc_desc* desc, const void* Xt, const void* dYt, const void* Yt, const void* W,
               void* dXt, const void* Xgate, float* dW, float* dbias, void* ws, size_t ws_bytes, void* stream);

/*
 * SGD with momentum restricted to the kept weights of the layer's patterns
 * (the update of a training step around the path; Sec. IV trains with
 * momentum SGD): for every kept output row n and kept input column k,
 *   V[n][k] = momentum * V[n][k] + dW[n][k],  W[n][k] -= lr * V[n][k],
 * and for the kept rows' bias entries the same with Vb, dbias. W is the full
 * [N][K] matrix of the descriptor's dtype, V [N][K] fp32, dW [N][K] fp32, or
 * the compact dWc[kept_out][ldc] when the descriptor's weight_layout is
 * ARD_WEIGHTS_COMPACT_GRAD; with ARD_WEIGHTS_INPUT_MAJOR W, V and dW are all
 * input-major [K][N] and the kept input rows are updated whole. bias, Vb,
 * dbias [N] fp32 (all three given or all NULL).
 * Dropped weights, their momentum and their bias entries are left untouched:
 * they are frozen for the step (the reading of an update restricted to the
 * kept rows). All device, caller-owned.
 */
int ard_fc_sgd_momentum(const ard_fc_desc* desc, void* W, float* V, const float* dW, float* bias, float* Vb,
                        const float* dbias, float lr, float momentum, void* stream);

/* ------------------------------------------------------------------------ */
/* Conventional dropout, the baseline the method replaces (device).         */
/* ------------------------------------------------------------------------ */
/*
 * Sec. II-C: conventional dropout keeps every GEMM dense and multiplies a
 * layer's output by a random 0/1 mask, and the output derivative by the same
 * mask in the backward pass. Element e = j * batch + b of the feature-major
 * Yt[n][batch] (dtype ARD_F32 or ARD_BF16) is kept iff draw e of the
 * counter-based sequence of (seed, stream_id, iter) -- the generator of the
 * pattern sampler -- as a 53-bit uniform is >= p: an independent
 * Bernoulli(1 - p) per element. fwd multiplies Yt in place by scale (kept) or
 * 0 and writes the mask bits (bit e in word e / 32; ceil(n * batch / 32)
 * words, device, caller-owned, 4-byte aligned); bwd multiplies dYt in place by
 * scale * mask. p in [0, 1); stream_id < 2^24, iter < 2^40.
 */
int ard_dropout_fwd(int32_t dtype, int32_t n, int32_t batch, double p, float scale, uint64_t seed,
                    uint32_t stream_id, uint64_t iter, void* Yt, uint32_t* mask, void* stream);
int ard_dropout_bwd(int32_t dtype, int32_t n, int32_t batch, float scale, const uint32_t* mask, void* dYt,
                    void* stream);

/* ------------------------------------------------------------------------ */
/* Layer under a tile pattern (device).                                     */
/* ------------------------------------------------------------------------ */
/*
 * Sec. III-B: with M the kept-tile mask of W expanded to tile x tile blocks,
 *   fwd        Yt  = scale * (W * M) Xt
 *   bwd_data   dXt = scale * (W * M)^T dYt
 *   bwd_weight dW  = scale * M * (dYt Xt^T)
 * Only kept tiles of W are read (fwd, bwd_data) or computed (bwd_weight).
 * Every row of Yt and dXt is written (a row block with no kept tile gets 0);
 * dW outside kept tiles is 0 (ZERO) or untouched (SKIP).
 * Layouts as for the FC layer; in_features = plan->k, out_features = plan->n.
 */
typedef struct {
  int32_t dtype;
  int32_t batch;
  int32_t in_features;
  int32_t out_features;
  float scale;
  int32_t dropped;
} ard_tile_desc;

int ard_tile_fwd(const ard_tile_desc* desc, const ard_tile_plan* plan, const void* Xt,
                 const void* W, void* Yt, void* stream);
int ard_tile_bwd_data(const ard_tile_desc* desc, const ard_tile_plan* plan, const void* dYt,
                      const void* W, void* dXt, void* stream);
int ard_tile_bwd_weight(const ard_tile_desc* desc, const ard_tile_plan* plan, const void* Xt,
                        const void* dYt, float* dW, void* stream);
/*
 * The layer's backward in one call: ard_tile_bwd_data and
 * ard_tile_bwd_weight on the same arguments, with the same results bit for
 * bit. Where both products take the direct-load kernels they run as one
 * launch, the weight-gradient work starting on each compute unit as soon as
 * its bwd_data tile is done; otherwise the two calls one after the other.
 */
int ard_tile_bwd(const ard_tile_desc* desc, const ard_tile_plan* plan, const void* Xt, const void* dYt,
                 const void* W, void* dXt, float* dW, void* stream);

/* ------------------------------------------------------------------------ */
/* LSTM layer with hidden-unit row pattern fixed per sequence (device).     */
/* ------------------------------------------------------------------------ */
/*
 * Sec. IV-C applies the method to LSTM as matrix multiplication. Dropped
 * hidden units are removed for the whole sequence (their h and c stay 0), so
 * the gate GEMMs run on the compact set S: inputs [x_t, h_{t-1}[S]], outputs
 * the four gates of S. Gate order i, f, g, o; W = [W_ih | W_hh]:
 *   z_t = W[:, :I] x_t + W[:, I:] (m * h_{t-1}) + bias
 *   c_t = m * (f * c_{t-1} + i * g),  h_t = m * (o * tanh(c_t))
 * Layouts: X[T][I][B], W[4H][I+H] (dtype), bias[4H] fp32, h0, c0, hT, cT
 * [H][B], Hs[T][H][B]. h0/c0 NULL = zeros. Dropped rows of Hs, hT, cT are 0.
 * The workspace carries the compact weights and the saved gates from fwd to
 * bwd: bwd must get the workspace of the fwd call with the same desc, plan and
 * inputs, unmodified in between. With any other workspace (of sufficient
 * size) the gradients are undefined but every write stays inside the output
 * arrays and the workspace: bwd takes no indices from the workspace.
 * bwd: dHs[T][H][B] (derivative of the loss w.r.t. every h_t), dhT and dcT
 * (extra derivatives of the final state, NULL = 0) -> dX[T][I][B], dW[4H][I+H]
 * fp32, dbias[4H] fp32, dh0 and dc0 [H][B] (each output may be NULL). Entries
 * of dropped units are written 0. Only ARD_F32 is supported.
 * input_plan (stacked layers): the hidden pattern of the layer below, whose
 * dropped units are this layer's dropped inputs. The layer then reads only the
 * kept rows of X (a strided view, no list needed) and compacts the matching
 * input columns of W, so the input products shrink by the kept fraction too;
 * the result is the layer applied to X with dropped input rows taken as 0,
 * and the dX rows and dW input columns of dropped inputs are written 0.
 */
typedef struct {
  int32_t dtype;
  int32_t seq_len;     /* T >= 1 */
  int32_t batch;       /* B >= 1 */
  int32_t input_size;  /* I >= 1 */
  int32_t hidden_size; /* H >= 1 */
  int32_t reserved;
  const ard_row_plan* hidden_plan;  /* n == H, or NULL = no dropout */
  const ard_row_plan* input_plan;   /* n == I, or NULL = every input kept */
} ard_lstm_desc;

size_t ard_lstm_workspace_bytes(const ard_lstm_desc* desc);
int ard_lstm_fwd(const ard_lstm_desc* desc, const void* X, const void* W, const float* bias,
                 const void* h0, const void* c0, void* Hs, void* hT, void* cT, void* ws,
                 size_t ws_bytes, void* stream);
int ard_lstm_bwd(const ard_lstm_desc* desc, const void* X, const void* dHs, const void* dhT,
                 const void* dcT, void* ws, size_t ws_bytes, void* dX, float* dW, float* dbias,
                 void* dh0, void* dc0, void* stream);

/* ------------------------------------------------------------------------ */
/* LSTM layer with a tile pattern on its weights (device).                  */
/* ------------------------------------------------------------------------ */
/*
 * The tile-based pattern (Sec. III-B) applied to an LSTM's matrix products
 * (Sec. IV-C): with M the kept-tile mask of W = [W_ih | W_hh] (4H x (I + H),
 * tiles of weight_plan, built by ard_plan_tiles / ard_plan_tiles_bernoulli
 * over n = 4H, k = I + H), every gate product uses W * M:
 *   z_t = (W * M) [x_t; h_{t-1}] + bias,  i, f, o = sigmoid, g = tanh,
 *   c_t = f * c_{t-1} + i * g,  h_t = o * tanh(c_t)   (every unit kept).
 * Only kept tiles of W are read, and dW = M * dL/d(W * M) is computed on kept
 * tiles only (0 elsewhere). Layouts as for ard_lstm_fwd (fp32 only); 4H and
 * I + H must be multiples of the plan's tile. The workspace
 * (ard_lstm_tile_workspace_bytes) holds the stacked inputs and saved gates
 * from fwd to bwd: bwd must get the fwd call's workspace, unmodified. bwd
 * outputs may be NULL.
 */
typedef struct {
  int32_t dtype;
  int32_t seq_len;
  int32_t batch;
  int32_t input_size;
  int32_t hidden_size;
  int32_t reserved;
  const ard_tile_plan* weight_plan;
} ard_lstm_tile_desc;

size_t ard_lstm_tile_workspace_bytes(const ard_lstm_tile_desc* desc);
int ard_lstm_tile_fwd(const ard_lstm_tile_desc* desc, const void* X, const void* W, const float* bias,
                      const void* h0, const void* c0, void* Hs, void* hT, void* cT, void* ws, size_t ws_bytes,
                      void* stream);
int ard_lstm_tile_bwd(const ard_lstm_tile_desc* desc, const void* W, const void* dHs, const void* dhT,
                      const void* dcT, void* ws, size_t ws_bytes, void* dX, float* dW, float* dbias, void* dh0,
                      void* dc0, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* ARD_H */
