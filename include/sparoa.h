/*
 * sparoa.h -- C ABI of libsparoa.so, the MI355X (gfx950) hot path of SparOA
 * (arXiv 2511.19457): per-operator input-activation sparsity, operator
 * intensity, sparsity x intensity routing, and dense / zero-skipping /
 * bandwidth-bound conv and FC kernels.
 *
 * General conventions
 *   - Every function returns sparoa_status (SPAROA_OK = 0).  On failure a
 *     thread-local message is available from sparoa_last_error().  No C++
 *     exception crosses this boundary.
 *   - Memory: the caller owns every buffer.  Device pointers (suffix _dev,
 *     and every tensor argument of the device calls) point to memory of the
 *     current HIP device.  The library never allocates device memory;
 *     scratch memory comes from a caller workspace sized by the
 *     *_workspace_size queries.
 *   - Streams: device calls are asynchronous and stream-ordered on `stream`
 *     (NULL = the null stream).  Only *_sync calls block.  Output counters
 *     are initialised inside the call: no caller memset is needed.
 *   - Layout: tensors are dense row-major.  Activations NHWC
 *     ([n][h][w][c]); conv weights [c_out][k_h][k_w][c_in/groups];
 *     FC activations [m][k]; FC weights [n][k] (output-feature major), or the
 *     packed layout written by sparoa_fc_pack_weights for the bandwidth
 *     paths.  Output dtype = input dtype; accumulation is fp32.
 *   - Alignment: tensor pointers must be 16-byte aligned; a misaligned
 *     pointer gives SPAROA_ERR_UNSUPPORTED (never a silent slow path).
 *   - Threading: calls are reentrant; the only global state is the
 *     thread-local error message.  Calls on different streams may overlap.
 */
#ifndef SPAROA_H
#define SPAROA_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* 3: the output-measuring calls take their count-commit words as an explicit
 *    argument (y_commit); the workspace queries report the split-K partial
 *    sums only.
 * 4: counts-only output measurement (y_mask NULL in *_routed_measured); a
 *    conv's x bitmap is needed only where its skip kernel reads one
 *    (sparoa_conv2d_reads_mask / sparoa_conv2d_routed_reads_mask). */
#define SPAROA_ABI_VERSION 4u

/* Bytes of the count-commit words of the output-measuring calls (y_commit). */
#define SPAROA_COMMIT_WORDS_BYTES 2048

typedef enum {
  SPAROA_OK = 0,
  SPAROA_ERR_INVALID_ARG = 1, /* null required pointer, bad shape, 0 elements, NaN threshold */
  SPAROA_ERR_UNSUPPORTED = 2, /* valid but not implemented: dtype/path/shape/alignment combo */
  SPAROA_ERR_WORKSPACE = 3,   /* workspace smaller than the *_workspace_size query */
  SPAROA_ERR_HIP = 4          /* a HIP runtime call failed; message has hipGetErrorString */
} sparoa_status;

typedef enum { SPAROA_F32 = 0, SPAROA_F16 = 1, SPAROA_BF16 = 2 } sparoa_dtype;

typedef enum { SPAROA_ACT_NONE = 0, SPAROA_ACT_RELU = 1, SPAROA_ACT_RELU6 = 2 } sparoa_act;

/* bit 0 = skip zero blocks, bit 1 = bandwidth-bound kernel. */
typedef enum {
  SPAROA_PATH_DENSE_MFMA = 0,
  SPAROA_PATH_SKIP_MFMA = 1,
  SPAROA_PATH_DENSE_BW = 2,
  SPAROA_PATH_SKIP_BW = 3
} sparoa_path;

typedef enum { SPAROA_ROUTE_BLOCK = 0, SPAROA_ROUTE_ELEMENT = 1 } sparoa_route_mode;

/* 2-D convolution (cross-correlation).  x NHWC [n][h][w][c_in],
 * w [c_out][kh][kw][c_in/groups], y NHWC [n][ho][wo][c_out] with
 * ho = (h + 2 ph - dh (kh-1) - 1) / sh + 1 (likewise wo). */
typedef struct {
  int64_t n, c_in, h, w, c_out, kh, kw, sh, sw, ph, pw, dh, dw, groups;
  sparoa_dtype dtype;
  int has_bias;
} sparoa_conv_desc;

/* Fully connected y[m][n] = x[m][k] * w[n][k]^T (+ bias[n]). */
typedef struct {
  int64_t m, k, n;
  sparoa_dtype dtype;
  int has_bias;
} sparoa_fc_desc;

/* Sparsity statistics (Eq. 1).  zero_blocks/num_blocks are 0 when no block
 * bitmap was requested. */
typedef struct {
  uint64_t zeros, numel, zero_blocks, num_blocks;
} sparoa_counts;

/* Operator work (Eq. 2): macs = multiply-accumulates, flops = 2 macs,
 * bytes = compulsory traffic, intensity = flops / bytes (FLOP per byte). */
typedef struct {
  uint64_t macs, flops, bytes;
  double intensity;
} sparoa_intensity;

/* Routing thresholds in natural units: sparsity in [0, 1], intensity in
 * FLOP/byte.  mode selects block (default) or element sparsity. */
typedef struct {
  double sparsity_thr, intensity_thr;
  int mode;
} sparoa_thresholds;

uint32_t sparoa_abi_version(void);
const char *sparoa_status_string(sparoa_status s);
/* Detail message of the last failing call on this thread ("" if none). */
const char *sparoa_last_error(void);

/* ------------------------------------------------------------------------
 * Sparsity measurement (SparOA Section 3.1, Eq. 1: rho = zero fraction of an
 * activation tensor; Section 2.1: zero activations may be skipped).
 *
 * x_dev is viewed as a row-major [rows x cols] matrix of `dtype`.  Writes
 * counts_dev->zeros (elements whose magnitude bits are all clear: +0, -0),
 * ->numel = rows*cols.  If mask_dev != NULL and block_rows, block_cols > 0,
 * also writes the nonzero-block bitmap: blocks are block_rows x block_cols
 * tiles (edge tiles clipped); block (bi, bj) has index
 * bi*ceil(cols/block_cols) + bj and sets bit (idx & 31) of mask word idx >> 5
 * iff it holds a nonzero element; unused high bits of the last word are 0;
 * ->zero_blocks / ->num_blocks are filled.  mask_dev must hold
 * sparoa_mask_words() words.  If per_sample_dev != NULL, rows are split into
 * `samples` equal groups (rows % samples == 0, and when a mask is requested
 * (rows/samples) % block_rows == 0) and per_sample_dev[s] = zeros of group s.
 * Asynchronous on `stream`; all outputs are initialised by the call.
 * Errors: INVALID_ARG for rows/cols <= 0, null x/counts, bad samples;
 * UNSUPPORTED for a misaligned x.
 * ---------------------------------------------------------------------- */
sparoa_status sparoa_mask_words(int64_t rows, int64_t cols, int64_t block_rows,
                                int64_t block_cols, int64_t *words);
sparoa_status sparoa_measure_sparsity(const void *x_dev, sparoa_dtype dtype, int64_t rows,
                                      int64_t cols, int64_t block_rows, int64_t block_cols,
                                      int64_t samples, sparoa_counts *counts_dev,
                                      uint32_t *mask_dev, uint64_t *per_sample_dev,
                                      hipStream_t stream);
/* The same measurement (no per-sample counts) into counters the caller has
 * already set to {0, rows*cols, nb, nb} (nb = ceil(rows/block_rows) *
 * ceil(cols/block_cols); a caller resets many counters with one copy): for
 * the block shapes whose bitmap needs no clearing -- 1 row x one 16-byte
 * vector, 1 row x 8 fp32 columns (cols % 8 == 0), 1 row x block_cols >= cols
 * for rows narrower than 16 bytes, or whole columns (block_rows >= rows,
 * block_cols == 1) -- the call is then
 * one launch instead of two.  Other block shapes initialise everything as
 * sparoa_measure_sparsity does.  commit_dev (nullable): zeroed count-commit
 * words (SPAROA_COMMIT_WORDS_BYTES, zero on entry, zero again when the call's
 * kernel finishes; see sparoa_conv2d_routed_measured) through which the
 * one-vector and narrow-row layouts commit their counts instead of one
 * same-address atomic per counter per work-group.  Errors as there. */
sparoa_status sparoa_measure_sparsity_preset(const void *x_dev, sparoa_dtype dtype, int64_t rows,
                                             int64_t cols, int64_t block_rows,
                                             int64_t block_cols, sparoa_counts *counts_dev,
                                             uint32_t *mask_dev, uint64_t *commit_dev,
                                             hipStream_t stream);
/* Same as sparoa_measure_sparsity, then copies the counts into *counts_host
 * and waits for the stream.  counts_dev is caller-provided device scratch of
 * one sparoa_counts. */
sparoa_status sparoa_measure_sparsity_sync(const void *x_dev, sparoa_dtype dtype, int64_t rows,
                                           int64_t cols, int64_t block_rows, int64_t block_cols,
                                           int64_t samples, sparoa_counts *counts_dev,
                                           uint32_t *mask_dev, uint64_t *per_sample_dev,
                                           sparoa_counts *counts_host, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Operator intensity (SparOA Section 3.1, Eq. 2: I = Kh Kw Cin Cout H W),
 * read with H, W = output extents, times the batch, with Cin/groups:
 *   macs  = n * ho * wo * c_out * (c_in/groups) * kh * kw
 *   bytes = size(dtype) * (n c_in h w + c_out (c_in/groups) kh kw
 *                          + n c_out ho wo + has_bias c_out)
 * FC: macs = m k n, bytes = size * (m k + n k + m n + has_bias n).
 * Host-only, pure.  Errors: INVALID_ARG for non-positive sizes, c_in or c_out
 * not divisible by groups, an empty output, or uint64 overflow.
 * ---------------------------------------------------------------------- */
sparoa_status sparoa_op_intensity_conv(const sparoa_conv_desc *desc, sparoa_intensity *out);
sparoa_status sparoa_op_intensity_fc(const sparoa_fc_desc *desc, sparoa_intensity *out);

/* ------------------------------------------------------------------------
 * Routing (SparOA Section 2.2: sparsity and intensity are independent axes
 * giving four quadrants -- sparse/dense x heavy/light; Section 3 opening:
 * fixed-threshold rule).  The CPU/GPU choice of the paper is remapped to
 * kernel paths of one GPU:
 *   skip bit      = rho >= sparsity_thr, rho = zero_blocks/num_blocks (BLOCK
 *                   mode) or zeros/numel (ELEMENT mode), one double division;
 *   bandwidth bit = is_depthwise || intensity < intensity_thr.
 * counts is host memory.  Errors: INVALID_ARG for NaN or negative thresholds
 * or intensity, num_blocks == 0 in BLOCK mode, numel == 0 in ELEMENT mode,
 * counts larger than their totals, an unknown mode.
 * ---------------------------------------------------------------------- */
sparoa_status sparoa_route(const sparoa_counts *counts, const sparoa_intensity *intensity,
                           int is_depthwise, const sparoa_thresholds *thr, sparoa_path *out);

/* ------------------------------------------------------------------------
 * Convolution (the operators of SparOA Sections 1 and 2.1; zero skipping of
 * Section 2.1).  y = act(conv(x, w) + bias + residual), written in dtype (the
 * residual joins before the activation, as in a ResNet bottleneck).
 *   Paths: DENSE_MFMA / SKIP_MFMA : implicit-GEMM on MFMA (groups == 1);
 *          DENSE_BW / SKIP_BW     : depthwise (groups == c_in == c_out) direct
 *                                   kernel; for groups == 1 1x1 convs
 *                                   (16-bit, no padding, c_in <= 256 and
 *                                   % 8 == 0, c_out % 8 == 0, the weights in
 *                                   at most four 48 KB slices, several slices
 *                                   only over >= 32768 output pixels, and not
 *                                   c_in >= 192 with c_in % 64 == 0 and
 *                                   c_out >= 64, nor below 32768 output
 *                                   pixels with c_out >= 64 where the
 *                                   implicit GEMM takes c_in: those are
 *                                   latency-bound) the pointwise kernel: the
 *                                   weights stay in LDS and each activation is
 *                                   read once per slice
 *                                   (sparoa_conv2d_tiling gives (16, 32));
 *                                   any other groups == 1 conv runs the
 *                                   implicit GEMM.
 *   Skip paths of the implicit GEMM need `mask`: the bitmap of x written by
 *   sparoa_measure_sparsity over the [n*h*w, c_in] view with the block shape
 *   returned by sparoa_conv2d_skip_block (one pixel x 8 channels); a
 *   work-group skips every (tile, K chunk) whose gathered input is zero:
 *   those blocks are never loaded nor multiplied.  UNSUPPORTED above
 *   K = 65536 (the routed form then runs dense).  The pointwise and
 *   small-channel kernels test x themselves and take mask == NULL
 *   (sparoa_conv2d_reads_mask tells which).  Dense paths ignore mask.  The
 *   depthwise kernel reads every input once and skips nothing.
 *   bias [c_out] (if desc->has_bias), residual (NHWC, output shape) nullable.
 *   executed_blocks_dev (nullable, skip paths): receives the number of
 *   executed (row tile, tap, channel block) triples; for 16-bit inputs of
 *   at most 4 channels (image stems, served by a direct kernel with tiling
 *   (16, 32)), the number of issued (16-pixel row block, 32-wide k-step)
 *   MFMA steps; on the pointwise kernel, the (16-pixel, 32-channel) blocks
 *   of x holding a nonzero (its skip form skips the others).
 *   Workspace: sparoa_conv2d_workspace_size bytes -- the split-K partial
 *   sums (0 when the GEMM needs no K split); its contents on entry do not
 *   matter and several calls may share one workspace in stream order.
 * Errors: INVALID_ARG for bad shapes, null x/w/y, a null mask on a skip path
 * whose kernel reads it;
 * UNSUPPORTED for grouped non-depthwise convs, unsupported dtype/path;
 * WORKSPACE if ws_bytes is below the partial-sum bytes.
 * ---------------------------------------------------------------------- */
sparoa_status sparoa_conv2d_workspace_size(const sparoa_conv_desc *desc, sparoa_path path,
                                           size_t *bytes);
sparoa_status sparoa_conv2d_skip_block(const sparoa_conv_desc *desc, sparoa_path path,
                                       int64_t *block_rows, int64_t *block_cols);
/* *reads = 1 when the kernel serving `path` reads x's bitmap (the skip
 * paths of the implicit GEMM), 0 otherwise (dense paths; the depthwise,
 * pointwise and small-channel kernels, which test x themselves). */
sparoa_status sparoa_conv2d_reads_mask(const sparoa_conv_desc *desc, sparoa_path path,
                                       int *reads);
/* Work tiling of the implicit-GEMM kernel: rows (output pixels) per tile and
 * K values per chunk, the units executed_blocks_dev counts.  UNSUPPORTED for
 * depthwise convs (not tiled). */
sparoa_status sparoa_conv2d_tiling(const sparoa_conv_desc *desc, sparoa_path path,
                                   int64_t *tile_rows, int64_t *kchunk);
sparoa_status sparoa_conv2d(const sparoa_conv_desc *desc, sparoa_path path, const void *x,
                            const void *w, const void *bias, const void *residual,
                            sparoa_act act, const uint32_t *mask, void *y, void *workspace,
                            size_t ws_bytes, uint64_t *executed_blocks_dev, hipStream_t stream);
/* Fixed-path forms: dense = DENSE_MFMA for groups == 1, DENSE_BW for
 * depthwise; zero_skip = SKIP_MFMA for groups == 1, SKIP_BW for depthwise. */
sparoa_status sparoa_conv2d_dense(const sparoa_conv_desc *desc, const void *x, const void *w,
                                  const void *bias, const void *residual, sparoa_act act,
                                  void *y, void *workspace, size_t ws_bytes, hipStream_t stream);
sparoa_status sparoa_conv2d_zero_skip(const sparoa_conv_desc *desc, const void *x,
                                      const void *w, const void *bias, const void *residual,
                                      sparoa_act act, const uint32_t *mask, void *y,
                                      void *workspace, size_t ws_bytes,
                                      uint64_t *executed_blocks_dev, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Fully connected (SparOA Sections 1 and 2.1).
 * y = act(x w^T + bias + residual); residual [m][n] nullable.
 *   Paths: DENSE_MFMA / SKIP_MFMA : tiled MFMA GEMM, w in [n][k];
 *          DENSE_BW / SKIP_BW     : weight-streaming kernel for 16-bit
 *                                   dtypes, m <= 64 and k <= 16384, w in
 *                                   the packed layout of
 *                                   sparoa_fc_pack_weights, each weight byte
 *                                   read at most once, no workspace; any
 *                                   other FC on a BW path is the 1x1 conv
 *                                   over m pixels (pointwise kernel where it
 *                                   applies, else the implicit GEMM) on
 *                                   w[n][k] (sparoa_fc_uses_packed tells
 *                                   which layout a call takes).
 *   Skip paths need `mask` of x measured over [m, k] with the block shape of
 *   sparoa_fc_skip_block ((1, 8) for the implicit GEMM, (m, 1) for the
 *   weight-streaming kernel):
 *   SKIP_MFMA skips (row tile, K chunk) pairs whose input block is zero;
 *   SKIP_BW skips input columns that are zero in every row, and with them
 *   their weight rows.
 *   executed_blocks_dev (nullable, skip paths): executed (row tile, K block)
 *   pairs (SKIP_MFMA) or nonzero columns (SKIP_BW).
 * Errors as for sparoa_conv2d; UNSUPPORTED for m > 64 on a BW path.
 * ---------------------------------------------------------------------- */
/* Packed weights for the BW paths, 16-column panels in two layouts, one
 * after the other: the skip layout, k-major inside a panel,
 * S[p][k][0..15] = w[16p + 0..15][k] (zero past n; the skip path streams
 * the rows of nonzero input columns), then the dense layout, per 32-k chunk
 * column-major, D[p][c][j][0..31] = w[16p + j][32c + 0..31] (zero past n and
 * k; the dense path loads MFMA operands from it as they are).  Each path
 * reads one layout.  w_packed must hold sparoa_fc_packed_bytes() bytes and
 * must not alias w_nk.  16-bit dtypes. */
sparoa_status sparoa_fc_packed_bytes(const sparoa_fc_desc *desc, size_t *bytes);
sparoa_status sparoa_fc_pack_weights(const sparoa_fc_desc *desc, const void *w_nk,
                                     void *w_packed, hipStream_t stream);
/* *packed = 1 when the call on `path` takes the packed weight layout (the
 * weight-streaming kernel), 0 when it takes w[n][k]. */
sparoa_status sparoa_fc_uses_packed(const sparoa_fc_desc *desc, sparoa_path path, int *packed);
/* Work tiling: (tile_rows, kchunk) = the implicit-GEMM tile rows and K chunk,
 * or (m, 1) for the weight-streaming kernel. */
sparoa_status sparoa_fc_tiling(const sparoa_fc_desc *desc, sparoa_path path, int64_t *tile_rows,
                               int64_t *kchunk);
sparoa_status sparoa_fc_workspace_size(const sparoa_fc_desc *desc, sparoa_path path,
                                       size_t *bytes);
sparoa_status sparoa_fc_skip_block(const sparoa_fc_desc *desc, sparoa_path path,
                                   int64_t *block_rows, int64_t *block_cols);
sparoa_status sparoa_fc(const sparoa_fc_desc *desc, sparoa_path path, const void *x,
                        const void *w_or_packed, const void *bias, const void *residual,
                        sparoa_act act, const uint32_t *mask, void *y, void *workspace,
                        size_t ws_bytes, uint64_t *executed_blocks_dev, hipStream_t stream);
/* Fixed-path forms on the MFMA kernel (w in [n][k]). */
sparoa_status sparoa_fc_dense(const sparoa_fc_desc *desc, const void *x, const void *w_nk,
                              const void *bias, const void *residual, sparoa_act act, void *y,
                              void *workspace, size_t ws_bytes, hipStream_t stream);
sparoa_status sparoa_fc_zero_skip(const sparoa_fc_desc *desc, const void *x, const void *w_nk,
                                  const void *bias, const void *residual, sparoa_act act,
                                  const uint32_t *mask, void *y, void *workspace,
                                  size_t ws_bytes, uint64_t *executed_blocks_dev,
                                  hipStream_t stream);

/* ------------------------------------------------------------------------
 * Device-side routing: the one-GPU form of the paper's asynchronous engine
 * (SparOA Section 5.1 -- execution proceeds without waiting on the host).
 * The bandwidth bit depends on shapes only and is computed on the host from
 * the operator's intensity (Eq. 2) and thr; the skip bit is decided inside
 * the kernel from counts_dev (left in device memory by
 * sparoa_measure_sparsity on the same stream) with the arithmetic of
 * sparoa_route, so the path equals sparoa_route's on the same counts.  No
 * host synchronisation between measurement and execution.
 *   mask: bitmap of x at the block shape of the family's skip path
 *         (sparoa_*_skip_block with SKIP_MFMA or SKIP_BW).  FC: required.
 *         Conv: required where the family's skip kernel reads it
 *         (sparoa_conv2d_routed_reads_mask); the depthwise, pointwise and
 *         small-channel kernels test x themselves and take NULL.
 *   FC: w_nk is used on the MFMA family, w_packed on the BW family; the
 *       other may be NULL.
 *   path_dev (nullable): receives the path taken (a uint32 sparoa_path).
 *   Counts with num_blocks == 0 (BLOCK mode) or numel == 0 (ELEMENT mode)
 *   select the dense path.  Depthwise convs always run the direct kernel;
 *   path_dev still records the decision.
 * Errors: those of sparoa_route (host-checkable thresholds) and of the
 * fixed-path calls.
 * ---------------------------------------------------------------------- */
sparoa_status sparoa_conv2d_routed(const sparoa_conv_desc *desc, const sparoa_thresholds *thr,
                                   const sparoa_counts *counts_dev, const void *x, const void *w,
                                   const void *bias, const void *residual, sparoa_act act,
                                   const uint32_t *mask, void *y, void *workspace,
                                   size_t ws_bytes, uint32_t *path_dev, hipStream_t stream);
/* *reads = 1 when the kernel that serves the routed conv's skip path (the
 * family its intensity and thr->intensity_thr select) reads x's bitmap, 0
 * when it tests x itself (depthwise, pointwise and small-channel kernels)
 * and the call takes mask == NULL. */
sparoa_status sparoa_conv2d_routed_reads_mask(const sparoa_conv_desc *desc,
                                              const sparoa_thresholds *thr, int *reads);
sparoa_status sparoa_fc_routed(const sparoa_fc_desc *desc, const sparoa_thresholds *thr,
                               const sparoa_counts *counts_dev, const void *x, const void *w_nk,
                               const void *w_packed, const void *bias, const void *residual,
                               sparoa_act act, const uint32_t *mask, void *y, void *workspace,
                               size_t ws_bytes, uint32_t *path_dev, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Routed conv / FC that also measures its own output, the next layer's input
 * (the sparsity feature of Eq. 1 is taken on a layer's output activation,
 * SparOA Section 3.1; here the producer emits it instead of a separate pass).
 *   y_counts (device, required), y_mask (device, nullable): afterwards they
 *   hold exactly what sparoa_measure_sparsity(y, dtype, rows, cols, 1, 8, 0,
 *   ...) gives, with rows = n*Ho*Wo, cols = c_out (FC: rows = m, cols = n)
 *   -- the block shape every conv and MFMA-family FC consumer skips at.
 *   y_mask holds sparoa_mask_words(rows, cols, 1, 8) words and needs no
 *   clearing.  y_mask NULL: counts only -- all four counts, no bitmap (for a
 *   consumer that routes on the counts and reads no bitmap); cols % 8 == 0.  The depthwise kernel's counts-only form is its plain
 *   kernel with per-lane counting; with y_mask it runs one output vector
 *   per lane so that a wave's bits are two whole bitmap words.
 *   y_counts must hold {0, rows*cols, nb, nb} on entry, nb = rows*ceil(cols/8):
 *   the fused form adds into it (a caller resets all of a network's counters
 *   with one copy from a template before each pass).
 *   Fused into the producer's epilogue (or its split-K reduction) where the
 *   kernel that serves the layer can (the 64-channel-chunk implicit GEMM --
 *   16-bit, C_in % 64 == 0 or C_in % 8 == 0 with C_in >= 48 -- with
 *   cols % 64 == 0, or cols % 8 == 0 where it splits K and its reduction
 *   writes y; the pointwise kernel with one weight slice; the depthwise
 *   and image-stem kernels, counts only for the stem): no launch of
 *   its own and no second read of y; otherwise the standalone measurement of
 *   y runs after the layer (as sparoa_measure_sparsity_preset with y_commit:
 *   one launch for the block shapes whose bitmap needs no clearing).
 *   y_commit (nullable): SPAROA_COMMIT_WORDS_BYTES of device memory that
 *   must be all zero on entry and is all zero again when the call's kernels
 *   finish (a caller resets it with y_counts).  The fused form then commits
 *   its counts through 8 ticketed words per counter (one atomic per
 *   work-group on a word of its group; the work-group completing a group
 *   adds the group's total to y_counts and clears the word) instead of one
 *   same-address atomic per work-group on y_counts.  NULL: direct commits,
 *   same counts.  Calls that overlap in time must not share y_commit.
 *   Other arguments as for sparoa_conv2d_routed / sparoa_fc_routed.
 * Errors: theirs, and INVALID_ARG for a null y_counts, or a NULL y_mask
 * where cols % 8 != 0.
 * ---------------------------------------------------------------------- */
sparoa_status sparoa_conv2d_routed_measured(const sparoa_conv_desc *desc,
                                            const sparoa_thresholds *thr,
                                            const sparoa_counts *counts_dev, const void *x,
                                            const void *w, const void *bias, const void *residual,
                                            sparoa_act act, const uint32_t *mask, void *y,
                                            void *workspace, size_t ws_bytes, uint32_t *path_dev,
                                            sparoa_counts *y_counts, uint32_t *y_mask,
                                            uint64_t *y_commit, hipStream_t stream);
sparoa_status sparoa_fc_routed_measured(const sparoa_fc_desc *desc, const sparoa_thresholds *thr,
                                        const sparoa_counts *counts_dev, const void *x,
                                        const void *w_nk, const void *w_packed, const void *bias,
                                        const void *residual, sparoa_act act,
                                        const uint32_t *mask, void *y, void *workspace,
                                        size_t ws_bytes, uint32_t *path_dev,
                                        sparoa_counts *y_counts, uint32_t *y_mask,
                                        uint64_t *y_commit, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Split execution of one operator over the zero-skip and dense paths: the
 * on-device reading of the paper's operator split (Algorithm 1 divides an
 * operator's work between two processors by a ratio; here its rows are
 * divided between two kernel paths by their own sparsity).  Every row tile of
 * the skip-capable implicit GEMM (tile rows: sparoa_conv2d_tiling with
 * SKIP_MFMA) takes its own route: the skip path iff
 *     (double)sum(sample_zeros[s0..s1]) / (double)((s1-s0+1) * sample_numel)
 *         >= sparsity_thr,
 * where s0..s1 are the input samples the tile's output rows come from (conv:
 * rows_per_sample = Ho*Wo, sample_numel = H*W*C_in; FC: one sample per row,
 * sample_numel = k).  The output equals the dense path's bit for bit (a
 * skipped chunk is all zeros).
 *   sample_zeros_dev / row_zeros_dev: per-sample zero counts of x
 *     (sparoa_measure_sparsity with samples = n, or = m for an FC).
 *   mask: bitmap of x at block (1, 8).
 *   executed_blocks_dev (nullable): executed (row tile, tap, 64-channel
 *     chunk) triples, every chunk counting on a dense tile (a tap's last
 *     chunk holds C_in mod 64 channels when C_in % 64 != 0).
 * Errors: UNSUPPORTED unless the 16-bit, groups 1 implicit GEMM serves the
 * layer (C_in % 64 == 0, or C_in % 8 == 0 and C_in >= 48); INVALID_ARG for null pointers or a NaN / negative
 * threshold; WORKSPACE as for sparoa_conv2d.
 * ---------------------------------------------------------------------- */
sparoa_status sparoa_conv2d_split(const sparoa_conv_desc *desc, double sparsity_thr,
                                  const uint64_t *sample_zeros_dev, const void *x, const void *w,
                                  const void *bias, const void *residual, sparoa_act act,
                                  const uint32_t *mask, void *y, void *workspace, size_t ws_bytes,
                                  uint64_t *executed_blocks_dev, hipStream_t stream);
sparoa_status sparoa_fc_split(const sparoa_fc_desc *desc, double sparsity_thr,
                              const uint64_t *row_zeros_dev, const void *x, const void *w_nk,
                              const void *bias, const void *residual, sparoa_act act,
                              const uint32_t *mask, void *y, void *workspace, size_t ws_bytes,
                              uint64_t *executed_blocks_dev, hipStream_t stream);

/* ------------------------------------------------------------------------
 * The whole path of one FC operator -- measure, route, execute (SparOA
 * Section 3.1 sparsity feature, Eq. 1; Section 2.2 quadrant routing) -- in
 * one call and no host round trip.
 *   x is measured at the skip granularity of the family that the FC's
 *   intensity (Eq. 2) selects: counts_dev and mask_dev receive exactly what
 *   sparoa_measure_sparsity gives at sparoa_fc_skip_block(desc, family|skip)
 *   (mask_dev: sparoa_mask_words(...) words, caller-owned); the device-routed
 *   FC then runs as in sparoa_fc_routed.  When the weight-streaming kernel
 *   serves the FC and k % 8 == 0, the FC kernel measures its own input and
 *   the call is one kernel launch; otherwise it is the measurement kernel
 *   followed by the routed kernel on the same stream.
 *   Other arguments as for sparoa_fc_routed.
 * Errors: those of sparoa_measure_sparsity and sparoa_fc_routed.
 * ---------------------------------------------------------------------- */
sparoa_status sparoa_fc_measured(const sparoa_fc_desc *desc, const sparoa_thresholds *thr,
                                 const void *x, const void *w_nk, const void *w_packed,
                                 const void *bias, const void *residual, sparoa_act act,
                                 sparoa_counts *counts_dev, uint32_t *mask_dev, void *y,
                                 void *workspace, size_t ws_bytes, uint32_t *path_dev,
                                 hipStream_t stream);

/* ------------------------------------------------------------------------
 * Native executor of independent FC operators: for each op in order,
 * sparoa_fc_measured -- the whole measure -> route -> execute path with one
 * host call per batch (host launch cost instead of one Python call per
 * kernel).  Issues no memset, copy or synchronisation, and no event unless
 * events are given, so a caller may capture it in a HIP graph.  Per op:
 * counts (one sparoa_counts) and mask (sparoa_mask_words words for that
 * granularity) are device scratch; path (nullable) receives the path taken;
 * w_nk / w_packed as for sparoa_fc_routed; thr holds the op's own
 * thresholds (the paper's predictor emits a threshold pair per operator,
 * Section 3, Eq. 5), used when the call's thr argument is NULL.
 * events (nullable): 2n hipEvent_t; events[2i] / events[2i+1] are recorded
 * on `stream` right before op i's first kernel / after its last kernel, and
 * the ops run one after another.  Without events the batch is validated
 * first and its launches are grouped: the self-measuring weight-streaming
 * FCs (16-bit, m <= 64, k % 8 == 0, bandwidth route) run as one launch per
 * 16 ops of a dtype and 16-row-tile count; the ops that measure in a launch
 * of their own are measured together (two launches per 16 ops), then their
 * FC kernels run in op order, then their split-K reductions run together
 * (one launch per 16 ops of a dtype); results are those of op-by-op calls,
 * bit for bit.  A batch in which memory one op writes (y, counts, mask,
 * workspace, path) overlaps memory another op reads or writes runs op by
 * op instead, in order.
 * Every op is validated (as sparoa_fc_measured validates) before the first
 * launch: a batch with an invalid op launches nothing and returns that op's
 * status, with "op <i>: " leading the message.  A HIP failure during the
 * launches returns SPAROA_ERR_HIP at once.
 * ---------------------------------------------------------------------- */
typedef struct {
  sparoa_fc_desc desc;
  const void *x, *w_nk, *w_packed, *bias, *residual;
  sparoa_act act;
  sparoa_counts *counts;
  uint32_t *mask;
  void *y;
  void *workspace;
  size_t ws_bytes;
  uint32_t *path;
  sparoa_thresholds thr;
} sparoa_fc_op;
/* thr: thresholds for every op, or NULL to use each op's own. */
sparoa_status sparoa_fc_ops_run(const sparoa_fc_op *ops, int64_t n, const sparoa_thresholds *thr,
                                hipEvent_t *events, hipStream_t stream);


/* ------------------------------------------------------------------------
 * For callers that cannot allocate device memory -- code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc: the same
 * convolution as sparoa_conv2d (same validation, kernels and output, bit for
 * bit) with no workspace argument.  The split-K partial sums live in a
 * library-owned device array of SPAROA_NOALLOC_SCRATCH_BYTES per GPU,
 * allocated when the library's code object loads and held until the process
 * ends; the call allocates nothing (no hipMalloc, hipFree or allocating
 * library routine).  The array's contents on entry do not matter.
 * Calls that overlap in time on one GPU (other streams, other host threads)
 * share that GPU's array and race; calls ordered on one stream do not.
 * Errors: those of sparoa_conv2d; SPAROA_ERR_WORKSPACE when the shape's
 * split-K partial sums (sparoa_conv2d_workspace_size) exceed the array.
 * ---------------------------------------------------------------------- */
#define SPAROA_NOALLOC_SCRATCH_BYTES (8u << 20)
sparoa_status sparoa_conv2d_noalloc(const sparoa_conv_desc *desc, sparoa_path path, const void *x,
                                    const void *w, const void *bias, const void *residual,
                                    sparoa_act act, const uint32_t *mask, void *y,
                                    uint64_t *executed_blocks_dev, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Network glue (not routed): NHWC max pooling, window k, stride s, padding p.
 * ---------------------------------------------------------------------- */
sparoa_status sparoa_maxpool2d(const void *x, sparoa_dtype dtype, int64_t n, int64_t c,
                               int64_t h, int64_t w, int64_t k, int64_t s, int64_t p, void *y,
                               hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* SPAROA_H */
