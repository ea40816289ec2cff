// extern "C" entry points of libsparoa.so: argument validation, the host-side
// intensity and routing functions, and dispatch to the HIP kernels.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <string>
#include <vector>

#include "common.h"

namespace sparoa {

namespace {
thread_local std::string g_last_error;

bool mul_ok(uint64_t a, uint64_t b, uint64_t *r) { return !__builtin_mul_overflow(a, b, r); }
bool add_ok(uint64_t a, uint64_t b, uint64_t *r) { return !__builtin_add_overflow(a, b, r); }

bool dtype_ok(int d) { return d == SPAROA_F32 || d == SPAROA_F16 || d == SPAROA_BF16; }
bool act_ok(int a) { return a == SPAROA_ACT_NONE || a == SPAROA_ACT_RELU || a == SPAROA_ACT_RELU6; }
bool path_ok(int p) { return p >= SPAROA_PATH_DENSE_MFMA && p <= SPAROA_PATH_SKIP_BW; }

int64_t out_extent(int64_t in, int64_t k, int64_t s, int64_t p, int64_t d) {
  if (in <= 0 || k <= 0 || s <= 0 || p < 0 || d <= 0) return -1;
  const int64_t span = in + 2 * p - d * (k - 1) - 1;
  return span < 0 ? -1 : span / s + 1;
}

sparoa_status check_conv(const sparoa_conv_desc *d, int64_t *ho, int64_t *wo) {
  if (!d) return fail(SPAROA_ERR_INVALID_ARG, "null conv descriptor");
  if (!dtype_ok(d->dtype)) return fail(SPAROA_ERR_INVALID_ARG, "unknown dtype");
  if (d->n <= 0 || d->c_in <= 0 || d->c_out <= 0 || d->groups <= 0 || d->c_in % d->groups ||
      d->c_out % d->groups)
    return fail(SPAROA_ERR_INVALID_ARG, "conv: bad batch/channel/group sizes");
  *ho = out_extent(d->h, d->kh, d->sh, d->ph, d->dh);
  *wo = out_extent(d->w, d->kw, d->sw, d->pw, d->dw);
  if (*ho <= 0 || *wo <= 0) return fail(SPAROA_ERR_INVALID_ARG, "conv: empty output");
  return SPAROA_OK;
}

sparoa_status check_fc(const sparoa_fc_desc *d) {
  if (!d) return fail(SPAROA_ERR_INVALID_ARG, "null fc descriptor");
  if (!dtype_ok(d->dtype)) return fail(SPAROA_ERR_INVALID_ARG, "unknown dtype");
  if (d->m <= 0 || d->k <= 0 || d->n <= 0) return fail(SPAROA_ERR_INVALID_ARG, "fc: sizes must be > 0");
  return SPAROA_OK;
}

bool is_depthwise(const sparoa_conv_desc &d) {
  return d.groups > 1 && d.groups == d.c_in && d.groups == d.c_out;
}

// The 1x1 stride-1 unpadded convolution with the FC's shape.
sparoa_conv_desc fc_as_conv(const sparoa_fc_desc &f) {
  sparoa_conv_desc c;
  c.n = f.m; c.c_in = f.k; c.h = 1; c.w = 1; c.c_out = f.n; c.kh = 1; c.kw = 1;
  c.sh = 1; c.sw = 1; c.ph = 0; c.pw = 0; c.dh = 1; c.dw = 1; c.groups = 1;
  c.dtype = f.dtype; c.has_bias = f.has_bias;
  return c;
}

sparoa_status check_ptrs16(std::initializer_list<const void *> ps) {
  for (const void *p : ps)
    if (p && !aligned16(p)) return fail(SPAROA_ERR_UNSUPPORTED, "pointer not 16-byte aligned");
  return SPAROA_OK;
}

sparoa_status check_measure(const void *x_dev, sparoa_dtype dtype, int64_t rows, int64_t cols,
                            int64_t block_rows, int64_t block_cols, int64_t samples,
                            const sparoa_counts *counts_dev, const uint32_t *mask_dev,
                            const uint64_t *per_sample_dev) {
  if (!x_dev || !counts_dev) return fail(SPAROA_ERR_INVALID_ARG, "measure: null x or counts");
  if (!dtype_ok(dtype)) return fail(SPAROA_ERR_INVALID_ARG, "measure: unknown dtype");
  uint64_t numel;
  if (rows <= 0 || cols <= 0 || !mul_ok((uint64_t)rows, (uint64_t)cols, &numel) ||
      numel > (uint64_t)INT64_MAX / 4)
    return fail(SPAROA_ERR_INVALID_ARG, "measure: rows and cols must be > 0");
  if (mask_dev) {
    int64_t words;
    sparoa_status st = sparoa_mask_words(rows, cols, block_rows, block_cols, &words);
    if (st != SPAROA_OK) return st;
  }
  if (per_sample_dev) {
    if (samples <= 0 || rows % samples)
      return fail(SPAROA_ERR_INVALID_ARG, "measure: rows must split into `samples` groups");
    if (samples > 65535) return fail(SPAROA_ERR_UNSUPPORTED, "measure: more than 65535 samples");
    if (mask_dev && (rows / samples) % block_rows)
      return fail(SPAROA_ERR_INVALID_ARG, "measure: block rows straddle samples");
  }
  if (!aligned16(x_dev)) return fail(SPAROA_ERR_UNSUPPORTED, "measure: x not 16-byte aligned");
  return SPAROA_OK;
}
}  // namespace

sparoa_status fail(sparoa_status s, const std::string &msg) {
  g_last_error = msg;
  return s;
}

sparoa_status hip_fail(hipError_t e, const char *what) {
  g_last_error = std::string(what) + ": " + hipGetErrorString(e);
  return SPAROA_ERR_HIP;
}

}  // namespace sparoa

using namespace sparoa;

extern "C" {

uint32_t sparoa_abi_version(void) { return SPAROA_ABI_VERSION; }

const char *sparoa_status_string(sparoa_status s) {
  switch (s) {
    case SPAROA_OK: return "ok";
    case SPAROA_ERR_INVALID_ARG: return "invalid argument";
    case SPAROA_ERR_UNSUPPORTED: return "unsupported";
    case SPAROA_ERR_WORKSPACE: return "workspace too small";
    case SPAROA_ERR_HIP: return "HIP runtime error";
  }
  return "unknown status";
}

const char *sparoa_last_error(void) { return g_last_error.c_str(); }

// ---------------------------------------------------------------- measure

sparoa_status sparoa_mask_words(int64_t rows, int64_t cols, int64_t block_rows,
                                int64_t block_cols, int64_t *words) {
  g_last_error.clear();
  if (!words || rows <= 0 || cols <= 0 || block_rows <= 0 || block_cols <= 0)
    return fail(SPAROA_ERR_INVALID_ARG, "mask_words: sizes must be > 0");
  uint64_t nb;
  if (!mul_ok((uint64_t)cdiv(rows, block_rows), (uint64_t)cdiv(cols, block_cols), &nb) ||
      nb > ((uint64_t)INT32_MAX) * 32u)
    return fail(SPAROA_ERR_INVALID_ARG, "mask_words: too many blocks");
  *words = (int64_t)((nb + 31) / 32);
  return SPAROA_OK;
}

sparoa_status sparoa_measure_sparsity(const void *x_dev, sparoa_dtype dtype, int64_t rows,
                                      int64_t cols, int64_t block_rows, int64_t block_cols,
                                      int64_t samples, sparoa_counts *counts_dev,
                                      uint32_t *mask_dev, uint64_t *per_sample_dev,
                                      hipStream_t stream) {
  g_last_error.clear();
  sparoa_status st = check_measure(x_dev, dtype, rows, cols, block_rows, block_cols, samples,
                                   counts_dev, mask_dev, per_sample_dev);
  if (st != SPAROA_OK) return st;
  return launch_measure(x_dev, dtype, rows, cols, block_rows, block_cols, samples, counts_dev,
                        mask_dev, per_sample_dev, stream);
}

sparoa_status sparoa_measure_sparsity_preset(const void *x_dev, sparoa_dtype dtype, int64_t rows,
                                             int64_t cols, int64_t block_rows,
                                             int64_t block_cols, sparoa_counts *counts_dev,
                                             uint32_t *mask_dev, uint64_t *commit_dev,
                                             hipStream_t stream) {
  g_last_error.clear();
  sparoa_status st = check_measure(x_dev, dtype, rows, cols, block_rows, block_cols, 0,
                                   counts_dev, mask_dev, nullptr);
  if (st != SPAROA_OK) return st;
  if ((st = check_ptrs16({commit_dev})) != SPAROA_OK) return st;
  return launch_measure(x_dev, dtype, rows, cols, block_rows, block_cols, 0, counts_dev,
                        mask_dev, nullptr, stream, true, commit_dev);
}

sparoa_status sparoa_measure_sparsity_sync(const void *x_dev, sparoa_dtype dtype, int64_t rows,
                                           int64_t cols, int64_t block_rows, int64_t block_cols,
                                           int64_t samples, sparoa_counts *counts_dev,
                                           uint32_t *mask_dev, uint64_t *per_sample_dev,
                                           sparoa_counts *counts_host, hipStream_t stream) {
  if (!counts_host) return fail(SPAROA_ERR_INVALID_ARG, "measure_sync: null host counts");
  sparoa_status st = sparoa_measure_sparsity(x_dev, dtype, rows, cols, block_rows, block_cols,
                                             samples, counts_dev, mask_dev, per_sample_dev,
                                             stream);
  if (st != SPAROA_OK) return st;
  SPAROA_HIP_CHECK(hipMemcpyAsync(counts_host, counts_dev, sizeof(sparoa_counts),
                                  hipMemcpyDeviceToHost, stream));
  SPAROA_HIP_CHECK(hipStreamSynchronize(stream));
  return SPAROA_OK;
}

// -------------------------------------------------------------- intensity

sparoa_status sparoa_op_intensity_conv(const sparoa_conv_desc *d, sparoa_intensity *out) {
  g_last_error.clear();
  int64_t ho, wo;
  sparoa_status st = check_conv(d, &ho, &wo);
  if (st != SPAROA_OK) return st;
  if (!out) return fail(SPAROA_ERR_INVALID_ARG, "null output");
  const uint64_t sz = (uint64_t)elem_size(d->dtype);
  uint64_t t, out_e, taps, macs, w_e, in_e, all, bytes;
  bool ok = mul_ok((uint64_t)d->n, (uint64_t)ho, &t) && mul_ok(t, (uint64_t)wo, &t) &&
            mul_ok(t, (uint64_t)d->c_out, &out_e) &&
            mul_ok((uint64_t)(d->c_in / d->groups), (uint64_t)d->kh, &taps) &&
            mul_ok(taps, (uint64_t)d->kw, &taps) && mul_ok(out_e, taps, &macs) &&
            mul_ok((uint64_t)d->c_out, taps, &w_e) &&
            mul_ok((uint64_t)d->n, (uint64_t)d->c_in, &t) && mul_ok(t, (uint64_t)d->h, &t) &&
            mul_ok(t, (uint64_t)d->w, &in_e) && add_ok(in_e, w_e, &all) &&
            add_ok(all, out_e, &all) &&
            add_ok(all, d->has_bias ? (uint64_t)d->c_out : 0u, &all) && mul_ok(all, sz, &bytes) &&
            macs <= UINT64_MAX / 2;
  if (!ok) return fail(SPAROA_ERR_INVALID_ARG, "conv intensity: uint64 overflow");
  out->macs = macs;
  out->flops = 2 * macs;
  out->bytes = bytes;
  out->intensity = (double)out->flops / (double)bytes;
  return SPAROA_OK;
}

sparoa_status sparoa_op_intensity_fc(const sparoa_fc_desc *d, sparoa_intensity *out) {
  g_last_error.clear();
  sparoa_status st = check_fc(d);
  if (st != SPAROA_OK) return st;
  if (!out) return fail(SPAROA_ERR_INVALID_ARG, "null output");
  const uint64_t sz = (uint64_t)elem_size(d->dtype);
  uint64_t x_e, macs, w_e, y_e, all, bytes;
  bool ok = mul_ok((uint64_t)d->m, (uint64_t)d->k, &x_e) && mul_ok(x_e, (uint64_t)d->n, &macs) &&
            mul_ok((uint64_t)d->n, (uint64_t)d->k, &w_e) &&
            mul_ok((uint64_t)d->m, (uint64_t)d->n, &y_e) && add_ok(x_e, w_e, &all) &&
            add_ok(all, y_e, &all) && add_ok(all, d->has_bias ? (uint64_t)d->n : 0u, &all) &&
            mul_ok(all, sz, &bytes) && macs <= UINT64_MAX / 2;
  if (!ok) return fail(SPAROA_ERR_INVALID_ARG, "fc intensity: uint64 overflow");
  out->macs = macs;
  out->flops = 2 * macs;
  out->bytes = bytes;
  out->intensity = (double)out->flops / (double)bytes;
  return SPAROA_OK;
}

// ------------------------------------------------------------------ route

sparoa_status sparoa_route(const sparoa_counts *c, const sparoa_intensity *in, int is_dw,
                           const sparoa_thresholds *thr, sparoa_path *out) {
  g_last_error.clear();
  if (!c || !in || !thr || !out) return fail(SPAROA_ERR_INVALID_ARG, "route: null argument");
  if (std::isnan(thr->sparsity_thr) || std::isnan(thr->intensity_thr) ||
      std::isnan(in->intensity) || thr->sparsity_thr < 0 || thr->intensity_thr < 0 ||
      in->intensity < 0)
    return fail(SPAROA_ERR_INVALID_ARG, "route: NaN or negative threshold/intensity");
  double rho;
  if (thr->mode == SPAROA_ROUTE_BLOCK) {
    if (c->num_blocks == 0 || c->zero_blocks > c->num_blocks)
      return fail(SPAROA_ERR_INVALID_ARG, "route: block mode needs block counts");
    rho = (double)c->zero_blocks / (double)c->num_blocks;
  } else if (thr->mode == SPAROA_ROUTE_ELEMENT) {
    if (c->numel == 0 || c->zeros > c->numel)
      return fail(SPAROA_ERR_INVALID_ARG, "route: element mode needs numel > 0");
    rho = (double)c->zeros / (double)c->numel;
  } else {
    return fail(SPAROA_ERR_INVALID_ARG, "route: unknown mode");
  }
  const int skip = rho >= thr->sparsity_thr ? 1 : 0;
  const int bw = (is_dw || in->intensity < thr->intensity_thr) ? 1 : 0;
  *out = (sparoa_path)(skip | (bw << 1));
  return SPAROA_OK;
}

// ------------------------------------------------------------------- conv

sparoa_status sparoa_conv2d_workspace_size(const sparoa_conv_desc *d, sparoa_path path,
                                           size_t *bytes) {
  g_last_error.clear();
  int64_t ho, wo;
  sparoa_status st = check_conv(d, &ho, &wo);
  if (st != SPAROA_OK) return st;
  if (!bytes || !path_ok(path)) return fail(SPAROA_ERR_INVALID_ARG, "workspace_size: bad argument");
  *bytes = is_depthwise(*d) ? 0 : gemm_workspace_required(*d, path);
  return SPAROA_OK;
}

sparoa_status sparoa_conv2d_skip_block(const sparoa_conv_desc *d, sparoa_path path,
                                       int64_t *block_rows, int64_t *block_cols) {
  g_last_error.clear();
  int64_t ho, wo;
  sparoa_status st = check_conv(d, &ho, &wo);
  if (st != SPAROA_OK) return st;
  if (!block_rows || !block_cols || !path_ok(path))
    return fail(SPAROA_ERR_INVALID_ARG, "skip_block: bad argument");
  if (is_depthwise(*d)) {
    // The depthwise kernel reads every input once; its bitmap granularity
    // is one pixel x 8 channels (routing statistics only).
    *block_rows = 1;
    *block_cols = 8;
    return SPAROA_OK;
  }
  if (d->groups != 1) return fail(SPAROA_ERR_UNSUPPORTED, "grouped (non-depthwise) conv");
  // The implicit-GEMM skip kernel reads one bit per (pixel, 8 channels).
  *block_rows = 1;
  *block_cols = 8;
  return SPAROA_OK;
}

sparoa_status sparoa_conv2d_tiling(const sparoa_conv_desc *d, sparoa_path path,
                                   int64_t *tile_rows, int64_t *kchunk) {
  g_last_error.clear();
  int64_t ho, wo;
  sparoa_status st = check_conv(d, &ho, &wo);
  if (st != SPAROA_OK) return st;
  if (!tile_rows || !kchunk || !path_ok(path))
    return fail(SPAROA_ERR_INVALID_ARG, "tiling: bad argument");
  if (is_depthwise(*d)) return fail(SPAROA_ERR_UNSUPPORTED, "tiling: depthwise is not tiled");
  if (d->groups != 1) return fail(SPAROA_ERR_UNSUPPORTED, "grouped (non-depthwise) conv");
  GemmTileChoice t = gemm_choose(*d, path);
  *tile_rows = t.bm;
  *kchunk = t.kchunk;
  return SPAROA_OK;
}

sparoa_status sparoa_conv2d(const sparoa_conv_desc *d, sparoa_path path, const void *x,
                            const void *w, const void *bias, const void *residual,
                            sparoa_act act, const uint32_t *mask, void *y, void *workspace,
                            size_t ws_bytes, uint64_t *executed, hipStream_t stream) {
  g_last_error.clear();
  int64_t ho, wo;
  sparoa_status st = check_conv(d, &ho, &wo);
  if (st != SPAROA_OK) return st;
  if (!x || !w || !y || !path_ok(path) || !act_ok(act))
    return fail(SPAROA_ERR_INVALID_ARG, "conv2d: null x/w/y or bad path/act");
  if (d->has_bias && !bias) return fail(SPAROA_ERR_INVALID_ARG, "conv2d: has_bias without bias");
  const bool skip = (path & 1) != 0;
  if (skip && !mask && !is_depthwise(*d) && conv_skip_reads_mask(*d, path))
    return fail(SPAROA_ERR_INVALID_ARG, "conv2d: this skip path's kernel needs x's bitmap");
  if ((st = check_ptrs16({x, w, bias, residual, y, mask, workspace})) != SPAROA_OK) return st;
  if (is_depthwise(*d)) {
    if (!(path & 2)) return fail(SPAROA_ERR_UNSUPPORTED, "depthwise conv runs on the BW path");
    if (executed && (st = launch_set_u64(executed, 0, stream)) != SPAROA_OK) return st;
    return launch_depthwise(*d, x, w, d->has_bias ? bias : nullptr, residual, act, y, stream);
  }
  if (d->groups != 1) return fail(SPAROA_ERR_UNSUPPORTED, "grouped (non-depthwise) conv");
  if (ws_bytes < gemm_workspace_required(*d, path))
    return fail(SPAROA_ERR_WORKSPACE, "conv2d: workspace too small");
  return launch_gemm_conv(*d, path, x, w, d->has_bias ? bias : nullptr, residual, act,
                          skip ? mask : nullptr, y, workspace, ws_bytes, executed, stream);
}

sparoa_status sparoa_conv2d_reads_mask(const sparoa_conv_desc *d, sparoa_path path, int *reads) {
  g_last_error.clear();
  int64_t ho, wo;
  sparoa_status st = check_conv(d, &ho, &wo);
  if (st != SPAROA_OK) return st;
  if (!reads || !path_ok(path)) return fail(SPAROA_ERR_INVALID_ARG, "reads_mask: bad argument");
  *reads = (!is_depthwise(*d) && conv_skip_reads_mask(*d, path)) ? 1 : 0;
  return SPAROA_OK;
}

sparoa_status sparoa_conv2d_dense(const sparoa_conv_desc *d, const void *x, const void *w,
                                  const void *bias, const void *residual, sparoa_act act,
                                  void *y, void *workspace, size_t ws_bytes, hipStream_t stream) {
  const sparoa_path p =
      (d && is_depthwise(*d)) ? SPAROA_PATH_DENSE_BW : SPAROA_PATH_DENSE_MFMA;
  return sparoa_conv2d(d, p, x, w, bias, residual, act, nullptr, y, workspace, ws_bytes,
                       nullptr, stream);
}

sparoa_status sparoa_conv2d_zero_skip(const sparoa_conv_desc *d, const void *x, const void *w,
                                      const void *bias, const void *residual, sparoa_act act,
                                      const uint32_t *mask, void *y, void *workspace,
                                      size_t ws_bytes, uint64_t *executed, hipStream_t stream) {
  const sparoa_path p = (d && is_depthwise(*d)) ? SPAROA_PATH_SKIP_BW : SPAROA_PATH_SKIP_MFMA;
  return sparoa_conv2d(d, p, x, w, bias, residual, act, mask, y, workspace, ws_bytes, executed,
                       stream);
}

// --------------------------------------------------------------------- fc

sparoa_status sparoa_fc_pack_weights(const sparoa_fc_desc *d, const void *w_nk, void *w_packed,
                                     hipStream_t stream) {
  g_last_error.clear();
  sparoa_status st = check_fc(d);
  if (st != SPAROA_OK) return st;
  if (!w_nk || !w_packed || w_nk == w_packed)
    return fail(SPAROA_ERR_INVALID_ARG, "fc_pack_weights: null or aliased buffers");
  if ((st = check_ptrs16({w_nk, w_packed})) != SPAROA_OK) return st;
  return launch_fc_pack(*d, w_nk, w_packed, stream);
}

sparoa_status sparoa_fc_packed_bytes(const sparoa_fc_desc *d, size_t *bytes) {
  g_last_error.clear();
  sparoa_status st = check_fc(d);
  if (st != SPAROA_OK) return st;
  if (!bytes) return fail(SPAROA_ERR_INVALID_ARG, "packed_bytes: null output");
  *bytes = fc_packed_bytes(*d);
  return SPAROA_OK;
}

sparoa_status sparoa_fc_tiling(const sparoa_fc_desc *d, sparoa_path path, int64_t *tile_rows,
                               int64_t *kchunk) {
  g_last_error.clear();
  sparoa_status st = check_fc(d);
  if (st != SPAROA_OK) return st;
  if (!tile_rows || !kchunk || !path_ok(path))
    return fail(SPAROA_ERR_INVALID_ARG, "tiling: bad argument");
  if ((path & 2) && fc_bw_streams(*d)) {
    *tile_rows = d->m;
    *kchunk = 1;
  } else {
    GemmTileChoice t = gemm_choose(fc_as_conv(*d), path);
    *tile_rows = t.bm;
    *kchunk = t.kchunk;
  }
  return SPAROA_OK;
}

sparoa_status sparoa_fc_workspace_size(const sparoa_fc_desc *d, sparoa_path path, size_t *bytes) {
  g_last_error.clear();
  sparoa_status st = check_fc(d);
  if (st != SPAROA_OK) return st;
  if (!bytes || !path_ok(path)) return fail(SPAROA_ERR_INVALID_ARG, "workspace_size: bad argument");
  *bytes = ((path & 2) && fc_bw_streams(*d)) ? fc_bw_workspace(*d, path)
                                              : gemm_workspace_required(fc_as_conv(*d), path);
  return SPAROA_OK;
}

sparoa_status sparoa_fc_uses_packed(const sparoa_fc_desc *d, sparoa_path path, int *packed) {
  g_last_error.clear();
  sparoa_status st = check_fc(d);
  if (st != SPAROA_OK) return st;
  if (!packed || !path_ok(path)) return fail(SPAROA_ERR_INVALID_ARG, "uses_packed: bad argument");
  *packed = ((path & 2) && fc_bw_streams(*d)) ? 1 : 0;
  return SPAROA_OK;
}

sparoa_status sparoa_fc_skip_block(const sparoa_fc_desc *d, sparoa_path path,
                                   int64_t *block_rows, int64_t *block_cols) {
  g_last_error.clear();
  sparoa_status st = check_fc(d);
  if (st != SPAROA_OK) return st;
  if (!block_rows || !block_cols || !path_ok(path))
    return fail(SPAROA_ERR_INVALID_ARG, "skip_block: bad argument");
  if ((path & 2) && fc_bw_streams(*d)) {  // a column is skipped when it is zero in every row
    *block_rows = d->m;
    *block_cols = 1;
  } else {  // the implicit-GEMM skip kernel reads one bit per (row, 8 columns)
    *block_rows = 1;
    *block_cols = 8;
  }
  return SPAROA_OK;
}

sparoa_status sparoa_fc(const sparoa_fc_desc *d, sparoa_path path, const void *x,
                        const void *w, const void *bias, const void *residual, sparoa_act act,
                        const uint32_t *mask, void *y, void *workspace, size_t ws_bytes,
                        uint64_t *executed, hipStream_t stream) {
  g_last_error.clear();
  sparoa_status st = check_fc(d);
  if (st != SPAROA_OK) return st;
  if (!x || !w || !y || !path_ok(path) || !act_ok(act))
    return fail(SPAROA_ERR_INVALID_ARG, "fc: null x/w/y or bad path/act");
  if (d->has_bias && !bias) return fail(SPAROA_ERR_INVALID_ARG, "fc: has_bias without bias");
  const bool skip = (path & 1) != 0;
  if (skip && !mask) return fail(SPAROA_ERR_INVALID_ARG, "fc: skip path needs a mask");
  if ((st = check_ptrs16({x, w, bias, residual, y, mask, workspace})) != SPAROA_OK) return st;
  if ((path & 2) && fc_bw_streams(*d)) {
    if (ws_bytes < fc_bw_workspace(*d, path))
      return fail(SPAROA_ERR_WORKSPACE, "fc: workspace too small");
    return launch_fc_bw(*d, path, x, w, d->has_bias ? bias : nullptr, residual, act,
                        skip ? mask : nullptr, y, workspace, ws_bytes, executed, stream);
  }
  const sparoa_conv_desc c = fc_as_conv(*d);
  if (ws_bytes < gemm_workspace_required(c, path)) return fail(SPAROA_ERR_WORKSPACE, "fc: workspace too small");
  return launch_gemm_conv(c, path, x, w, d->has_bias ? bias : nullptr, residual, act,
                          skip ? mask : nullptr, y, workspace, ws_bytes, executed, stream);
}

sparoa_status sparoa_fc_dense(const sparoa_fc_desc *d, const void *x, const void *w_nk,
                              const void *bias, const void *residual, sparoa_act act, void *y,
                              void *workspace, size_t ws_bytes, hipStream_t stream) {
  return sparoa_fc(d, SPAROA_PATH_DENSE_MFMA, x, w_nk, bias, residual, act, nullptr, y, workspace,
                   ws_bytes, nullptr, stream);
}

sparoa_status sparoa_fc_zero_skip(const sparoa_fc_desc *d, const void *x, const void *w_nk,
                                  const void *bias, const void *residual, sparoa_act act,
                                  const uint32_t *mask, void *y, void *workspace,
                                  size_t ws_bytes, uint64_t *executed, hipStream_t stream) {
  return sparoa_fc(d, SPAROA_PATH_SKIP_MFMA, x, w_nk, bias, residual, act, mask, y, workspace,
                   ws_bytes, executed, stream);
}

// -------------------------------------------------------- device routing

namespace {
sparoa_status check_thr(const sparoa_thresholds *thr) {
  if (!thr) return fail(SPAROA_ERR_INVALID_ARG, "routed: null thresholds");
  if (std::isnan(thr->sparsity_thr) || std::isnan(thr->intensity_thr) || thr->sparsity_thr < 0 ||
      thr->intensity_thr < 0)
    return fail(SPAROA_ERR_INVALID_ARG, "routed: NaN or negative threshold");
  if (thr->mode != SPAROA_ROUTE_BLOCK && thr->mode != SPAROA_ROUTE_ELEMENT)
    return fail(SPAROA_ERR_INVALID_ARG, "routed: unknown mode");
  return SPAROA_OK;
}
}  // namespace

}  // extern "C"

namespace {
// The output measurement of a *_routed_measured call: y_counts with y_mask
// (counts and bitmap), y_counts alone (counts only: cols % 8 == 0), or
// neither.
sparoa_status check_out_measure(const sparoa_counts *y_counts, const uint32_t *y_mask,
                                int64_t cols) {
  if (y_mask && !y_counts)
    return fail(SPAROA_ERR_INVALID_ARG, "routed_measured: y_mask without y_counts");
  if (y_counts && !y_mask && cols % 8 != 0)
    return fail(SPAROA_ERR_INVALID_ARG,
                "routed_measured: counts-only measurement needs cols % 8 == 0");
  return SPAROA_OK;
}
}  // namespace

namespace {
// The routed conv (see sparoa_conv2d_routed).  With y_counts / y_mask
// non-null it also measures y at block (1, 8) over [N*Ho*Wo, C_out]: in the
// GEMM's epilogue where that is fused, else by a standalone pass after it.
sparoa_status conv_routed_impl(const sparoa_conv_desc *d, const sparoa_thresholds *thr,
                               const sparoa_counts *counts_dev, const void *x, const void *w,
                               const void *bias, const void *residual, sparoa_act act,
                               const uint32_t *mask, void *y, void *workspace, size_t ws_bytes,
                               uint32_t *path_dev, sparoa_counts *y_counts, uint32_t *y_mask,
                               uint64_t *y_commit, hipStream_t stream) {
  sparoa_intensity in;
  sparoa_status st = sparoa_op_intensity_conv(d, &in);
  if (st != SPAROA_OK) return st;
  if ((st = check_thr(thr)) != SPAROA_OK) return st;
  if (!counts_dev || !x || !w || !y || !act_ok(act))
    return fail(SPAROA_ERR_INVALID_ARG, "conv2d_routed: null counts/x/w/y or bad act");
  if (d->has_bias && !bias) return fail(SPAROA_ERR_INVALID_ARG, "conv2d_routed: has_bias without bias");
  if ((st = check_ptrs16({x, w, bias, residual, y, mask, workspace, y_counts, y_mask,
                          y_commit})) != SPAROA_OK)
    return st;
  const bool dw = is_depthwise(*d);
  const int bw = (dw || in.intensity < thr->intensity_thr) ? 1 : 0;
  if (!mask && !dw && d->groups == 1 &&
      conv_skip_reads_mask(*d, bw ? SPAROA_PATH_SKIP_BW : SPAROA_PATH_SKIP_MFMA))
    return fail(SPAROA_ERR_INVALID_ARG, "conv2d_routed: this layer's skip kernel needs x's bitmap");
  const DeviceRoute r{counts_dev, thr->sparsity_thr, thr->mode, bw, path_dev};
  int64_t ho = 0, wo = 0;
  if ((st = check_conv(d, &ho, &wo)) != SPAROA_OK) return st;
  const int64_t rows = d->n * ho * wo, cols = d->c_out;
  const bool measure_y = y_counts != nullptr;
  if ((st = check_out_measure(y_counts, y_mask, cols)) != SPAROA_OK) return st;
  auto measure_after = [&]() {
    // y_counts arrive preset ({0, numel, nb, nb}): no init launch where the
    // bitmap needs no clearing
    if (!measure_y) return SPAROA_OK;
    return y_mask ? launch_measure(y, d->dtype, rows, cols, 1, 8, 0, y_counts, y_mask, nullptr,
                                   stream, true, y_commit)
                  : launch_measure_counts8(y, d->dtype, rows, cols, y_counts, y_commit, stream);
  };
  if (dw) {
    if (measure_y && dw_fuses_out_measure(*d)) {   // y_counts arrives initialised
      const OutMeasure om{y_counts, y_mask, reinterpret_cast<unsigned long long *>(y_commit)};
      return launch_depthwise(*d, x, w, d->has_bias ? bias : nullptr, residual, act, y, stream,
                              &r, &om);
    }
    if ((st = launch_depthwise(*d, x, w, d->has_bias ? bias : nullptr, residual, act, y, stream,
                               &r)) != SPAROA_OK)
      return st;
    return measure_after();
  }
  if (d->groups != 1) return fail(SPAROA_ERR_UNSUPPORTED, "grouped (non-depthwise) conv");
  const sparoa_path p = bw ? SPAROA_PATH_SKIP_BW : SPAROA_PATH_SKIP_MFMA;
  if (ws_bytes < gemm_workspace_required(*d, p)) return fail(SPAROA_ERR_WORKSPACE, "conv2d_routed: workspace too small");
  // without a skip kernel for this shape the dense kernel runs and records a dense path
  const bool can_skip = gemm_skip_supported(*d);
  if (measure_y && gemm_fuses_out_measure(*d, p, y_mask != nullptr)) {   // y_counts initialised
    const OutMeasure om{y_counts, y_mask, reinterpret_cast<unsigned long long *>(y_commit)};
    return launch_gemm_conv(*d, p, x, w, d->has_bias ? bias : nullptr, residual, act,
                            can_skip ? mask : nullptr, y, workspace, ws_bytes, nullptr, stream, &r,
                            nullptr, &om);
  }
  if ((st = launch_gemm_conv(*d, p, x, w, d->has_bias ? bias : nullptr, residual, act,
                             can_skip ? mask : nullptr, y, workspace, ws_bytes, nullptr, stream,
                             &r)) != SPAROA_OK)
    return st;
  return measure_after();
}
}  // namespace

extern "C" {

sparoa_status sparoa_conv2d_routed(const sparoa_conv_desc *d, const sparoa_thresholds *thr,
                                   const sparoa_counts *counts_dev, const void *x, const void *w,
                                   const void *bias, const void *residual, sparoa_act act,
                                   const uint32_t *mask, void *y, void *workspace,
                                   size_t ws_bytes, uint32_t *path_dev, hipStream_t stream) {
  g_last_error.clear();
  return conv_routed_impl(d, thr, counts_dev, x, w, bias, residual, act, mask, y, workspace,
                          ws_bytes, path_dev, nullptr, nullptr, nullptr, stream);
}

sparoa_status sparoa_conv2d_routed_reads_mask(const sparoa_conv_desc *d,
                                              const sparoa_thresholds *thr, int *reads) {
  g_last_error.clear();
  sparoa_intensity in;
  sparoa_status st = sparoa_op_intensity_conv(d, &in);
  if (st != SPAROA_OK) return st;
  if ((st = check_thr(thr)) != SPAROA_OK) return st;
  if (!reads) return fail(SPAROA_ERR_INVALID_ARG, "routed_reads_mask: null reads");
  const bool dw = is_depthwise(*d);
  const int bw = (dw || in.intensity < thr->intensity_thr) ? 1 : 0;
  *reads = (!dw && d->groups == 1 &&
            conv_skip_reads_mask(*d, bw ? SPAROA_PATH_SKIP_BW : SPAROA_PATH_SKIP_MFMA))
               ? 1 : 0;
  return SPAROA_OK;
}

sparoa_status sparoa_conv2d_routed_measured(const sparoa_conv_desc *d,
                                            const sparoa_thresholds *thr,
                                            const sparoa_counts *counts_dev, const void *x,
                                            const void *w, const void *bias, const void *residual,
                                            sparoa_act act, const uint32_t *mask, void *y,
                                            void *workspace, size_t ws_bytes, uint32_t *path_dev,
                                            sparoa_counts *y_counts, uint32_t *y_mask,
                                            uint64_t *y_commit, hipStream_t stream) {
  g_last_error.clear();
  if (!y_counts) return fail(SPAROA_ERR_INVALID_ARG, "conv2d_routed_measured: null y_counts");
  return conv_routed_impl(d, thr, counts_dev, x, w, bias, residual, act, mask, y, workspace,
                          ws_bytes, path_dev, y_counts, y_mask, y_commit, stream);
}


}  // extern "C"

namespace {
// Every check of the routed FC, with no device work: the executor runs it on
// a whole batch before its first launch.
sparoa_status fc_routed_check(const sparoa_fc_desc *d, const sparoa_thresholds *thr,
                              const sparoa_counts *counts_dev, const void *x, const void *w_nk,
                              const void *w_packed, const void *bias, const void *residual,
                              sparoa_act act, const uint32_t *mask, void *y, void *workspace,
                              size_t ws_bytes, const sparoa_counts *y_counts,
                              const uint32_t *y_mask, const uint64_t *y_commit) {
  sparoa_intensity in;
  sparoa_status st = sparoa_op_intensity_fc(d, &in);
  if (st != SPAROA_OK) return st;
  if ((st = check_thr(thr)) != SPAROA_OK) return st;
  const int bw = in.intensity < thr->intensity_thr ? 1 : 0;
  const bool streams = bw && fc_bw_streams(*d);
  const void *w = streams ? w_packed : w_nk;
  if (!counts_dev || !x || !w || !y || !mask || !act_ok(act))
    return fail(SPAROA_ERR_INVALID_ARG, "fc_routed: null counts/x/weights/mask/y or bad act");
  if (d->has_bias && !bias) return fail(SPAROA_ERR_INVALID_ARG, "fc_routed: has_bias without bias");
  if ((st = check_ptrs16({x, w, bias, residual, y, mask, workspace, y_counts, y_mask,
                          y_commit})) != SPAROA_OK)
    return st;
  if ((st = check_out_measure(y_counts, y_mask, d->n)) != SPAROA_OK) return st;
  if (!streams) {
    const sparoa_path p = bw ? SPAROA_PATH_SKIP_BW : SPAROA_PATH_SKIP_MFMA;
    if (ws_bytes < gemm_workspace_required(fc_as_conv(*d), p))
      return fail(SPAROA_ERR_WORKSPACE, "fc_routed: workspace too small");
  }
  return SPAROA_OK;
}

// The routed FC (see sparoa_fc_routed); defer as for launch_gemm_conv.
sparoa_status fc_routed_impl(const sparoa_fc_desc *d, const sparoa_thresholds *thr,
                             const sparoa_counts *counts_dev, const void *x, const void *w_nk,
                             const void *w_packed, const void *bias, const void *residual,
                             sparoa_act act, const uint32_t *mask, void *y, void *workspace,
                             size_t ws_bytes, uint32_t *path_dev, hipStream_t stream,
                             SplitReduceJob *defer, sparoa_counts *y_counts = nullptr,
                             uint32_t *y_mask = nullptr, uint64_t *y_commit = nullptr) {
  if (defer) defer->split = 0;
  sparoa_status st = fc_routed_check(d, thr, counts_dev, x, w_nk, w_packed, bias, residual, act,
                                     mask, y, workspace, ws_bytes, y_counts, y_mask, y_commit);
  if (st != SPAROA_OK) return st;
  sparoa_intensity in;
  sparoa_op_intensity_fc(d, &in);
  const int bw = in.intensity < thr->intensity_thr ? 1 : 0;
  const bool streams = bw && fc_bw_streams(*d);
  const void *w = streams ? w_packed : w_nk;
  const bool measure_y = y_counts != nullptr;
  auto measure_after = [&]() {   // y_counts arrive preset
    if (!measure_y) return SPAROA_OK;
    return y_mask ? launch_measure(y, d->dtype, d->m, d->n, 1, 8, 0, y_counts, y_mask, nullptr,
                                   stream, true, y_commit)
                  : launch_measure_counts8(y, d->dtype, d->m, d->n, y_counts, y_commit, stream);
  };
  const DeviceRoute r{counts_dev, thr->sparsity_thr, thr->mode, bw, path_dev};
  if (streams) {
    if ((st = launch_fc_bw(*d, SPAROA_PATH_SKIP_BW, x, w, d->has_bias ? bias : nullptr, residual,
                           act, mask, y, workspace, ws_bytes, nullptr, stream, &r)) != SPAROA_OK)
      return st;
    return measure_after();
  }
  const sparoa_conv_desc c = fc_as_conv(*d);
  const sparoa_path p = bw ? SPAROA_PATH_SKIP_BW : SPAROA_PATH_SKIP_MFMA;
  const bool can_skip = gemm_skip_supported(c);
  if (measure_y && gemm_fuses_out_measure(c, p, y_mask != nullptr)) {   // y_counts initialised
    const OutMeasure om{y_counts, y_mask, reinterpret_cast<unsigned long long *>(y_commit)};
    return launch_gemm_conv(c, p, x, w, d->has_bias ? bias : nullptr, residual, act,
                            can_skip ? mask : nullptr, y, workspace, ws_bytes, nullptr, stream, &r,
                            defer, &om);
  }
  if ((st = launch_gemm_conv(c, p, x, w, d->has_bias ? bias : nullptr, residual, act,
                             can_skip ? mask : nullptr, y, workspace, ws_bytes, nullptr, stream,
                             &r, defer)) != SPAROA_OK)
    return st;
  if (measure_y && defer && defer->split > 1)   // the caller reduces later: cannot measure y now
    return fail(SPAROA_ERR_UNSUPPORTED, "fc_routed_measured: deferred reduction");
  return measure_after();
}

// How sparoa_fc_measured runs one FC: the self-measuring streaming kernel
// (one launch), or a lanebit-layout measurement that an executor may group
// with others, or the standalone measurement; then the routed kernel.
struct FcPlan {
  bool self_measures;
  MeasureJob measure;
};

// Validates the whole call (measurement and routed FC) before any launch.
sparoa_status fc_measured_plan(const sparoa_fc_desc *d, const sparoa_thresholds *thr,
                               const void *x, const void *w_nk, const void *w_packed,
                               const void *bias, const void *residual, sparoa_act act,
                               sparoa_counts *counts_dev, uint32_t *mask_dev, void *y,
                               void *workspace, size_t ws_bytes, FcPlan *p) {
  sparoa_intensity in;
  sparoa_status st = sparoa_op_intensity_fc(d, &in);
  if (st != SPAROA_OK) return st;
  if ((st = check_thr(thr)) != SPAROA_OK) return st;
  const int bw = in.intensity < thr->intensity_thr ? 1 : 0;
  p->self_measures = bw && fc_bw_self_measures(*d);
  if (p->self_measures) {
    if (!counts_dev || !x || !w_packed || !y || !mask_dev || !act_ok(act))
      return fail(SPAROA_ERR_INVALID_ARG, "fc_measured: null counts/x/w_packed/mask/y or bad act");
    if (d->has_bias && !bias) return fail(SPAROA_ERR_INVALID_ARG, "fc_measured: has_bias without bias");
    return check_ptrs16({x, w_packed, bias, residual, y, mask_dev, counts_dev});
  }
  int64_t br, bc;
  const sparoa_path fam = bw ? SPAROA_PATH_SKIP_BW : SPAROA_PATH_SKIP_MFMA;
  if ((st = sparoa_fc_skip_block(d, fam, &br, &bc)) != SPAROA_OK) return st;
  p->measure = MeasureJob{x, d->dtype, d->m, d->k, br, bc, counts_dev, mask_dev};
  if ((st = check_measure(x, d->dtype, d->m, d->k, br, bc, 0, counts_dev, mask_dev, nullptr)) !=
      SPAROA_OK)
    return st;
  return fc_routed_check(d, thr, counts_dev, x, w_nk, w_packed, bias, residual, act, mask_dev, y,
                         workspace, ws_bytes, nullptr, nullptr, nullptr);
}
}  // namespace

extern "C" {

sparoa_status sparoa_fc_routed(const sparoa_fc_desc *d, const sparoa_thresholds *thr,
                               const sparoa_counts *counts_dev, const void *x, const void *w_nk,
                               const void *w_packed, const void *bias, const void *residual,
                               sparoa_act act, const uint32_t *mask, void *y, void *workspace,
                               size_t ws_bytes, uint32_t *path_dev, hipStream_t stream) {
  g_last_error.clear();
  return fc_routed_impl(d, thr, counts_dev, x, w_nk, w_packed, bias, residual, act, mask, y,
                        workspace, ws_bytes, path_dev, stream, nullptr);
}

sparoa_status sparoa_fc_routed_measured(const sparoa_fc_desc *d, const sparoa_thresholds *thr,
                                        const sparoa_counts *counts_dev, const void *x,
                                        const void *w_nk, const void *w_packed, const void *bias,
                                        const void *residual, sparoa_act act,
                                        const uint32_t *mask, void *y, void *workspace,
                                        size_t ws_bytes, uint32_t *path_dev,
                                        sparoa_counts *y_counts, uint32_t *y_mask,
                                        uint64_t *y_commit, hipStream_t stream) {
  g_last_error.clear();
  if (!y_counts) return fail(SPAROA_ERR_INVALID_ARG, "fc_routed_measured: null y_counts");
  return fc_routed_impl(d, thr, counts_dev, x, w_nk, w_packed, bias, residual, act, mask, y,
                        workspace, ws_bytes, path_dev, stream, nullptr, y_counts, y_mask,
                        y_commit);
}

sparoa_status sparoa_fc_measured(const sparoa_fc_desc *d, const sparoa_thresholds *thr,
                                 const void *x, const void *w_nk, const void *w_packed,
                                 const void *bias, const void *residual, sparoa_act act,
                                 sparoa_counts *counts_dev, uint32_t *mask_dev, void *y,
                                 void *workspace, size_t ws_bytes, uint32_t *path_dev,
                                 hipStream_t stream) {
  g_last_error.clear();
  FcPlan p;
  sparoa_status st = fc_measured_plan(d, thr, x, w_nk, w_packed, bias, residual, act, counts_dev,
                                      mask_dev, y, workspace, ws_bytes, &p);
  if (st != SPAROA_OK) return st;
  if (p.self_measures) {
    const int bw = 1;
    const DeviceRoute r{nullptr, thr->sparsity_thr, thr->mode, bw, path_dev};
    return launch_fc_bw_measured(*d, x, w_packed, d->has_bias ? bias : nullptr, residual, act,
                                 counts_dev, mask_dev, y, stream, r);
  }
  const MeasureJob &m = p.measure;
  if ((st = launch_measure(m.x, m.dt, m.rows, m.cols, m.block_rows, m.block_cols, 0, m.counts,
                           m.mask, nullptr, stream)) != SPAROA_OK)
    return st;
  return fc_routed_impl(d, thr, counts_dev, x, w_nk, w_packed, bias, residual, act, mask_dev, y,
                        workspace, ws_bytes, path_dev, stream, nullptr);
}

// ------------------------------------------------------- split execution

}  // extern "C"

namespace {
sparoa_status split_impl(const sparoa_conv_desc &c, double sparsity_thr,
                         const uint64_t *sample_zeros, const void *x, const void *w,
                         const void *bias, const void *residual, sparoa_act act,
                         const uint32_t *mask, void *y, void *workspace, size_t ws_bytes,
                         uint64_t *executed, hipStream_t stream) {
  int64_t ho, wo;
  sparoa_status st = check_conv(&c, &ho, &wo);
  if (st != SPAROA_OK) return st;
  if (!sample_zeros || !x || !w || !y || !mask || !act_ok(act))
    return fail(SPAROA_ERR_INVALID_ARG, "split: null sample_zeros/x/w/mask/y or bad act");
  if (std::isnan(sparsity_thr) || sparsity_thr < 0)
    return fail(SPAROA_ERR_INVALID_ARG, "split: NaN or negative threshold");
  if (c.has_bias && !bias) return fail(SPAROA_ERR_INVALID_ARG, "split: has_bias without bias");
  if ((st = check_ptrs16({x, w, bias, residual, y, mask, workspace})) != SPAROA_OK) return st;
  if (is_depthwise(c) || c.groups != 1 || gemm_choose(c, SPAROA_PATH_SKIP_MFMA).cfg == 0)
    return fail(SPAROA_ERR_UNSUPPORTED,
                "split: needs the 16-bit, C_in % 64 == 0 implicit GEMM (groups 1)");
  if (ws_bytes < gemm_workspace_required(c, SPAROA_PATH_SKIP_MFMA))
    return fail(SPAROA_ERR_WORKSPACE, "split: workspace too small");
  DeviceRoute r{nullptr, sparsity_thr, SPAROA_ROUTE_ELEMENT, 0, nullptr};
  r.sample_zeros = reinterpret_cast<const unsigned long long *>(sample_zeros);
  r.rows_per_sample = ho * wo;
  r.sample_numel = c.h * c.w * c.c_in;
  return launch_gemm_conv(c, SPAROA_PATH_SKIP_MFMA, x, w, c.has_bias ? bias : nullptr, residual,
                          act, mask, y, workspace, ws_bytes, executed, stream, &r);
}
}  // namespace

extern "C" {

sparoa_status sparoa_conv2d_split(const sparoa_conv_desc *d, double sparsity_thr,
                                  const uint64_t *sample_zeros_dev, const void *x, const void *w,
                                  const void *bias, const void *residual, sparoa_act act,
                                  const uint32_t *mask, void *y, void *workspace, size_t ws_bytes,
                                  uint64_t *executed_blocks_dev, hipStream_t stream) {
  g_last_error.clear();
  if (!d) return fail(SPAROA_ERR_INVALID_ARG, "split: null desc");
  return split_impl(*d, sparsity_thr, sample_zeros_dev, x, w, bias, residual, act, mask, y,
                    workspace, ws_bytes, executed_blocks_dev, stream);
}

sparoa_status sparoa_fc_split(const sparoa_fc_desc *d, double sparsity_thr,
                              const uint64_t *row_zeros_dev, const void *x, const void *w_nk,
                              const void *bias, const void *residual, sparoa_act act,
                              const uint32_t *mask, void *y, void *workspace, size_t ws_bytes,
                              uint64_t *executed_blocks_dev, hipStream_t stream) {
  g_last_error.clear();
  sparoa_status st = check_fc(d);
  if (st != SPAROA_OK) return st;
  return split_impl(fc_as_conv(*d), sparsity_thr, row_zeros_dev, x, w_nk, bias, residual, act,
                    mask, y, workspace, ws_bytes, executed_blocks_dev, stream);
}

// ---------------------------------------------------------------- executor

namespace {
// True when some op writes memory that another op reads or writes (an
// output feeding another op's input, or counts, masks, workspaces or path
// words shared between ops -- valid one op after another, but a batch
// measures every op before any op routes and reduces split-K partials after
// later GEMMs): then the ops must run strictly one after another.  Called on
// validated ops.
bool ops_chained(const sparoa_fc_op *ops, int64_t n, const sparoa_thresholds *thr) {
  typedef std::pair<uintptr_t, uintptr_t> Range;
  auto range = [](const void *p, int64_t bytes) {
    const uintptr_t b = reinterpret_cast<uintptr_t>(p);
    return Range(b, b + (uintptr_t)(p ? bytes : 0));
  };
  auto overlap = [](Range a, Range b) { return a.first < b.second && b.first < a.second; };
  std::vector<std::vector<Range>> rd((size_t)n), wr((size_t)n);
  for (int64_t i = 0; i < n; ++i) {
    const sparoa_fc_op &o = ops[i];
    const sparoa_fc_desc &d = o.desc;
    const int64_t e = elem_size(d.dtype);
    const sparoa_thresholds *t = thr ? thr : &o.thr;
    sparoa_intensity in;
    sparoa_op_intensity_fc(&d, &in);
    const sparoa_path fam =
        in.intensity < t->intensity_thr ? SPAROA_PATH_SKIP_BW : SPAROA_PATH_SKIP_MFMA;
    int64_t br = 1, bc = 1, words = 0;
    sparoa_fc_skip_block(&d, fam, &br, &bc);
    sparoa_mask_words(d.m, d.k, br, bc, &words);
    size_t packed = 0;
    sparoa_fc_packed_bytes(&d, &packed);
    rd[i] = {range(o.x, d.m * d.k * e), range(o.residual, d.m * d.n * e),
             range(o.w_nk, d.n * d.k * e), range(o.w_packed, (int64_t)packed),
             range(o.bias, d.n * e)};
    wr[i] = {range(o.y, d.m * d.n * e), range(o.counts, (int64_t)sizeof(sparoa_counts)),
             range(o.mask, words * 4), range(o.workspace, (int64_t)o.ws_bytes),
             range(o.path, 4)};
  }
  for (int64_t i = 0; i < n; ++i)
    for (int64_t j = 0; j < n; ++j) {
      if (i == j) continue;
      for (const Range &w : wr[i]) {
        for (const Range &r : rd[j])
          if (overlap(w, r)) return true;
        for (const Range &r : wr[j])
          if (overlap(w, r)) return true;
      }
    }
  return false;
}

sparoa_status check_ops(const sparoa_fc_op *ops, int64_t n, const sparoa_thresholds *thr) {
  if (!ops || n < 0) return fail(SPAROA_ERR_INVALID_ARG, "fc_ops: null ops or n < 0");
  if (thr) return check_thr(thr);
  for (int64_t i = 0; i < n; ++i) {
    sparoa_status st = check_thr(&ops[i].thr);
    if (st != SPAROA_OK) return st;
  }
  return SPAROA_OK;
}
}  // namespace

sparoa_status sparoa_fc_ops_run(const sparoa_fc_op *ops, int64_t n, const sparoa_thresholds *thr,
                                hipEvent_t *events, hipStream_t stream) {
  g_last_error.clear();
  sparoa_status st = check_ops(ops, n, thr);
  if (st != SPAROA_OK) return st;
  // Every op is validated before the first launch (a batch that fails
  // validation launches nothing), whichever way it then runs.
  std::vector<FcPlan> plan((size_t)n);
  for (int64_t i = 0; i < n; ++i) {
    const sparoa_fc_op &o = ops[i];
    if ((st = fc_measured_plan(&o.desc, thr ? thr : &o.thr, o.x, o.w_nk, o.w_packed, o.bias,
                               o.residual, o.act, o.counts, o.mask, o.y, o.workspace, o.ws_bytes,
                               &plan[i])) != SPAROA_OK) {
      g_last_error = "op " + std::to_string(i) + ": " + g_last_error;
      return st;
    }
  }
  if (events || ops_chained(ops, n, thr)) {  // op by op (each bracketed by its events, if given)
    for (int64_t i = 0; i < n; ++i) {
      const sparoa_fc_op &o = ops[i];
      if (events) SPAROA_HIP_CHECK(hipEventRecord(events[2 * i], stream));
      if ((st = sparoa_fc_measured(&o.desc, thr ? thr : &o.thr, o.x, o.w_nk, o.w_packed, o.bias,
                                   o.residual, o.act, o.counts, o.mask, o.y, o.workspace,
                                   o.ws_bytes, o.path, stream)) != SPAROA_OK)
        return st;
      if (events) SPAROA_HIP_CHECK(hipEventRecord(events[2 * i + 1], stream));
    }
    return SPAROA_OK;
  }
  // Batched: every op is validated first; the measurements of the ops that
  // measure in a launch of their own run grouped (counter init and
  // measurement: two launches per kGroupMax ops of one element size); the
  // self-measuring streaming FCs run grouped (one launch per kGroupMax ops of
  // one dtype and row-tile count); then each other op's FC kernel in op
  // order; then the split-K reductions, grouped per dtype.  Same arithmetic
  // as op-by-op calls, fewer launches.
  for (int esz : {2, 4}) {
    std::vector<MeasureJob> group;
    for (int64_t i = 0; i < n; ++i) {
      const MeasureJob &m = plan[i].measure;
      if (plan[i].self_measures || elem_size(m.dt) != esz) continue;
      if (!measure_groupable(m)) {
        if ((st = launch_measure(m.x, m.dt, m.rows, m.cols, m.block_rows, m.block_cols, 0,
                                 m.counts, m.mask, nullptr, stream)) != SPAROA_OK)
          return st;
        continue;
      }
      group.push_back(m);
      if ((int)group.size() == kGroupMax) {
        if ((st = launch_measure_group(group.data(), kGroupMax, stream)) != SPAROA_OK) return st;
        group.clear();
      }
    }
    if (!group.empty() &&
        (st = launch_measure_group(group.data(), (int)group.size(), stream)) != SPAROA_OK)
      return st;
  }
  // Self-measuring streaming FCs run as grouped launches, one per key (dtype
  // and row tiles) and kGroupMax ops, in op order within a group.
  std::vector<int> keys;
  for (int64_t i = 0; i < n; ++i) {
    if (!plan[i].self_measures) continue;
    const int k = fc_bw_group_key(ops[i].desc);
    if (std::find(keys.begin(), keys.end(), k) == keys.end()) keys.push_back(k);
  }
  for (int key : keys) {
    std::vector<FcBwJob> group;
    for (int64_t i = 0; i < n; ++i) {
      const sparoa_fc_op &o = ops[i];
      if (!plan[i].self_measures || fc_bw_group_key(o.desc) != key) continue;
      const sparoa_thresholds *t = thr ? thr : &o.thr;
      group.push_back(FcBwJob{o.desc, o.x, o.w_packed, o.desc.has_bias ? o.bias : nullptr,
                              o.residual, o.act, o.counts, o.mask, o.y,
                              DeviceRoute{nullptr, t->sparsity_thr, t->mode, 1, o.path}});
      if ((int)group.size() == kGroupMax) {
        if ((st = launch_fc_bw_measured_group(group.data(), kGroupMax, stream)) != SPAROA_OK)
          return st;
        group.clear();
      }
    }
    if (!group.empty() &&
        (st = launch_fc_bw_measured_group(group.data(), (int)group.size(), stream)) != SPAROA_OK)
      return st;
  }
  std::vector<SplitReduceJob> reduces;
  for (int64_t i = 0; i < n; ++i) {
    const sparoa_fc_op &o = ops[i];
    const sparoa_thresholds *t = thr ? thr : &o.thr;
    if (plan[i].self_measures) continue;
    SplitReduceJob job;
    if ((st = fc_routed_impl(&o.desc, t, o.counts, o.x, o.w_nk, o.w_packed, o.bias, o.residual,
                             o.act, o.mask, o.y, o.workspace, o.ws_bytes, o.path, stream,
                             &job)) != SPAROA_OK)
      return st;
    if (job.split > 1) reduces.push_back(job);
  }
  for (sparoa_dtype dt : {SPAROA_F32, SPAROA_F16, SPAROA_BF16}) {
    std::vector<SplitReduceJob> group;
    for (const SplitReduceJob &j : reduces) {
      if (j.dt != dt) continue;
      group.push_back(j);
      if ((int)group.size() == kGroupMax) {
        if ((st = launch_split_reduce_group(group.data(), kGroupMax, stream)) != SPAROA_OK)
          return st;
        group.clear();
      }
    }
    if (!group.empty() &&
        (st = launch_split_reduce_group(group.data(), (int)group.size(), stream)) != SPAROA_OK)
      return st;
  }
  return SPAROA_OK;
}

// ------------------------------------------------------------------- glue

sparoa_status sparoa_maxpool2d(const void *x, sparoa_dtype dtype, int64_t n, int64_t c,
                               int64_t h, int64_t w, int64_t k, int64_t s, int64_t p, void *y,
                               hipStream_t stream) {
  g_last_error.clear();
  if (!x || !y || !dtype_ok(dtype) || n <= 0 || c <= 0)
    return fail(SPAROA_ERR_INVALID_ARG, "maxpool2d: bad argument");
  if (out_extent(h, k, s, p, 1) <= 0 || out_extent(w, k, s, p, 1) <= 0 || p >= k)
    return fail(SPAROA_ERR_INVALID_ARG, "maxpool2d: empty output or padding >= window");
  sparoa_status st = check_ptrs16({x, y});
  if (st != SPAROA_OK) return st;
  return launch_maxpool(x, dtype, n, c, h, w, k, s, p, y, stream);
}

}  // extern "C"
