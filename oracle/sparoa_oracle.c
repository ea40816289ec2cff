/*
 * sparoa_oracle.c -- plain, slow, CPU reference for the SparOA hot path.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, loads or
 * calls this file; only the test suite, the smoke check and the CPU-baseline
 * leg of the benchmark do.  It shares no code, header, table or helper with
 * the HIP library: every decode, index and loop below is written out here.
 *
 * What it computes (paper sections cited per function):
 *   - zero counts, block bitmaps and per-sample counts of an activation
 *     tensor (sparsity, Section 3.1, Eq. 1; zero skipping, Section 2.1);
 *   - the operator intensity closed form (Section 3.1, Eq. 2) generalised
 *     with batch, stride, dilation and groups, plus a MAC counter inside the
 *     direct convolution loop that must agree with it;
 *   - the sparsity x intensity routing rule (Section 2.2 quadrants and the
 *     fixed-threshold rule at the start of Section 3), remapped to kernel
 *     paths on one GPU;
 *   - direct convolution / fully connected operators in double precision,
 *     with the abs-product sum used by the tolerance, and the zero-skipping
 *     variant (Section 1, key insight: skipped zero activations leave the
 *     output unchanged);
 *   - the executed (row-tile, K-block) work count expected from a skipping
 *     kernel, obtained by brute force from the input values;
 *   - 3x3 stride-2 max pooling (network glue, not a routed operator).
 *
 * Floating point inputs are raw IEEE bit patterns (binary32, binary16,
 * bfloat16); they are decoded to double from the format definitions and all
 * arithmetic is in double.  Products of two decoded inputs are exact in
 * double (at most 24+24 significand bits), so skipping an exact-zero term
 * cannot change a double sum.
 *
 * Parity pins: every function here is pinned by tests under tests/ against
 * library routines (numpy, torch CPU float64), closed forms, hand-written
 * golden values and the paper's Table 2.  Routing-threshold optimality is
 * parity unpinned (the paper's thresholds come from a trained predictor that
 * is not available).
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define OR_F32 0
#define OR_F16 1
#define OR_BF16 2

#define OR_OK 0
#define OR_EINVAL 1

#define OR_ACT_NONE 0
#define OR_ACT_RELU 1
#define OR_ACT_RELU6 2

#define OR_ROUTE_BLOCK 0
#define OR_ROUTE_ELEMENT 1

/* ------------------------------------------------------------------------ */
/* Decoding from the format definitions.                                     */
/* ------------------------------------------------------------------------ */

/* IEEE 754 binary16: 1 sign, 5 exponent (bias 15), 10 fraction bits. */
static double dec_f16(uint16_t h) {
  int s = (h >> 15) & 1, e = (h >> 10) & 0x1f, f = h & 0x3ff;
  double v;
  if (e == 0)
    v = ldexp((double)f, -24); /* subnormal: 0.f * 2^-14 */
  else if (e == 31)
    v = f ? NAN : INFINITY;
  else
    v = ldexp((double)(f | 0x400), e - 25); /* 1.f * 2^(e-15) */
  return s ? -v : v;
}

/* bfloat16: 1 sign, 8 exponent (bias 127), 7 fraction bits. */
static double dec_bf16(uint16_t b) {
  int s = (b >> 15) & 1, e = (b >> 7) & 0xff, f = b & 0x7f;
  double v;
  if (e == 0)
    v = ldexp((double)f, -133); /* 0.f * 2^-126 */
  else if (e == 255)
    v = f ? NAN : INFINITY;
  else
    v = ldexp((double)(f | 0x80), e - 134); /* 1.f * 2^(e-127) */
  return s ? -v : v;
}

/* IEEE 754 binary32: 1 sign, 8 exponent (bias 127), 23 fraction bits. */
static double dec_f32(uint32_t u) {
  int s = (u >> 31) & 1, e = (u >> 23) & 0xff;
  uint32_t f = u & 0x7fffffu;
  double v;
  if (e == 0)
    v = ldexp((double)f, -149);
  else if (e == 255)
    v = f ? NAN : INFINITY;
  else
    v = ldexp((double)(f | 0x800000u), e - 150);
  return s ? -v : v;
}

static double elem(const void *p, int dt, int64_t i) {
  if (dt == OR_F32) return dec_f32(((const uint32_t *)p)[i]);
  if (dt == OR_F16) return dec_f16(((const uint16_t *)p)[i]);
  return dec_bf16(((const uint16_t *)p)[i]);
}

/* An element is zero iff its magnitude bits are all clear: +0 and -0 only.
 * Subnormals, NaN and Inf are nonzero. */
static int elem_is_zero(const void *p, int dt, int64_t i) {
  if (dt == OR_F32) return (((const uint32_t *)p)[i] & 0x7fffffffu) == 0;
  return (((const uint16_t *)p)[i] & 0x7fffu) == 0;
}

static int dt_ok(int dt) { return dt == OR_F32 || dt == OR_F16 || dt == OR_BF16; }
static int64_t dt_size(int dt) { return dt == OR_F32 ? 4 : 2; }

/* Exported decoder, so tests can check it against numpy/torch casts. */
double or_decode(const void *p, int dt, int64_t i) { return elem(p, dt, i); }

/* ------------------------------------------------------------------------ */
/* Sparsity (Eq. 1).                                                          */
/* ------------------------------------------------------------------------ */

/*
 * View x as a row-major [rows x cols] matrix.
 * out[0] = zeros z (elements equal to +-0), out[1] = numel n = rows*cols.
 * If mask != NULL and block_rows, block_cols > 0: blocks are block_rows x
 * block_cols tiles, edge tiles clipped to the matrix; block (bi, bj) has
 * linear index bi*ceil(cols/block_cols) + bj and sets bit (idx & 31) of word
 * idx >> 5 iff it holds at least one nonzero element.  out[2] = zero blocks,
 * out[3] = number of blocks.  Without a mask out[2] = out[3] = 0.
 * If per_sample != NULL: rows are split into `samples` equal consecutive
 * groups and per_sample[s] = zeros of group s.
 */
int or_measure(const void *x, int dt, int64_t rows, int64_t cols, int64_t block_rows,
               int64_t block_cols, int64_t samples, uint64_t out[4], uint32_t *mask,
               uint64_t *per_sample) {
  if (!x || !out || !dt_ok(dt) || rows <= 0 || cols <= 0) return OR_EINVAL;
  uint64_t z = 0;
  for (int64_t i = 0; i < rows * cols; ++i) z += (uint64_t)elem_is_zero(x, dt, i);
  out[0] = z;
  out[1] = (uint64_t)(rows * cols);
  out[2] = 0;
  out[3] = 0;
  if (mask) {
    if (block_rows <= 0 || block_cols <= 0) return OR_EINVAL;
    int64_t nbr = (rows + block_rows - 1) / block_rows;
    int64_t nbc = (cols + block_cols - 1) / block_cols;
    int64_t nb = nbr * nbc;
    memset(mask, 0, (size_t)((nb + 31) / 32) * sizeof(uint32_t));
    uint64_t zb = 0;
    for (int64_t bi = 0; bi < nbr; ++bi)
      for (int64_t bj = 0; bj < nbc; ++bj) {
        int nonzero = 0;
        for (int64_t r = bi * block_rows; r < rows && r < (bi + 1) * block_rows; ++r)
          for (int64_t c = bj * block_cols; c < cols && c < (bj + 1) * block_cols; ++c)
            if (!elem_is_zero(x, dt, r * cols + c)) nonzero = 1;
        int64_t idx = bi * nbc + bj;
        if (nonzero)
          mask[idx >> 5] |= 1u << (idx & 31);
        else
          ++zb;
      }
    out[2] = zb;
    out[3] = (uint64_t)nb;
  }
  if (per_sample) {
    if (samples <= 0 || rows % samples) return OR_EINVAL;
    int64_t rs = rows / samples;
    for (int64_t s = 0; s < samples; ++s) {
      uint64_t zs = 0;
      for (int64_t i = s * rs * cols; i < (s + 1) * rs * cols; ++i)
        zs += (uint64_t)elem_is_zero(x, dt, i);
      per_sample[s] = zs;
    }
  }
  return OR_OK;
}

/* rho = z / n: the zero fraction of Eq. 1, evaluated as one division. */
double or_sparsity(uint64_t zeros, uint64_t numel) {
  return numel ? (double)zeros / (double)numel : NAN;
}

/* ------------------------------------------------------------------------ */
/* Intensity (Eq. 2).                                                         */
/* ------------------------------------------------------------------------ */

static int mul_ok(uint64_t a, uint64_t b, uint64_t *r) { return !__builtin_mul_overflow(a, b, r); }
static int add_ok(uint64_t a, uint64_t b, uint64_t *r) { return !__builtin_add_overflow(a, b, r); }

/* Output extent of one spatial dimension; -1 if the window does not fit. */
int64_t or_out_dim(int64_t in, int64_t k, int64_t s, int64_t p, int64_t d) {
  int64_t span = in + 2 * p - d * (k - 1) - 1;
  if (in <= 0 || k <= 0 || s <= 0 || p < 0 || d <= 0 || span < 0) return -1;
  return span / s + 1;
}

/*
 * Eq. 2 with batch and groups: MACs = N * Ho * Wo * Cout * (Cin/g) * Kh * Kw
 * (H, W read as the output extents).  flops = 2 * MACs; bytes = compulsory
 * traffic of input, weights, output (and bias) at the element size.
 * res = {macs, flops, bytes}; *intensity = flops / bytes.
 */
int or_conv_intensity(int64_t n, int64_t cin, int64_t h, int64_t w, int64_t cout, int64_t kh,
                      int64_t kw, int64_t sh, int64_t sw, int64_t ph, int64_t pw, int64_t dh,
                      int64_t dw, int64_t groups, int dt, int has_bias, uint64_t res[3],
                      double *intensity) {
  if (!res || !intensity || !dt_ok(dt) || n <= 0 || cin <= 0 || cout <= 0 || groups <= 0 ||
      cin % groups || cout % groups)
    return OR_EINVAL;
  int64_t ho = or_out_dim(h, kh, sh, ph, dh), wo = or_out_dim(w, kw, sw, pw, dw);
  if (ho <= 0 || wo <= 0) return OR_EINVAL;
  uint64_t macs, t, in_e, w_e, out_e, all, bytes, sz = (uint64_t)dt_size(dt);
  if (!mul_ok((uint64_t)n, (uint64_t)ho, &t) || !mul_ok(t, (uint64_t)wo, &t) ||
      !mul_ok(t, (uint64_t)cout, &out_e))
    return OR_EINVAL;
  if (!mul_ok((uint64_t)(cin / groups), (uint64_t)kh, &t) || !mul_ok(t, (uint64_t)kw, &t) ||
      !mul_ok(out_e, t, &macs) || !mul_ok((uint64_t)cout, t, &w_e))
    return OR_EINVAL;
  if (!mul_ok((uint64_t)n, (uint64_t)cin, &t) || !mul_ok(t, (uint64_t)h, &t) ||
      !mul_ok(t, (uint64_t)w, &in_e))
    return OR_EINVAL;
  if (!add_ok(in_e, w_e, &all) || !add_ok(all, out_e, &all) ||
      !add_ok(all, has_bias ? (uint64_t)cout : 0, &all) || !mul_ok(all, sz, &bytes))
    return OR_EINVAL;
  if (macs > UINT64_MAX / 2) return OR_EINVAL;
  res[0] = macs;
  res[1] = 2 * macs;
  res[2] = bytes;
  *intensity = (double)res[1] / (double)bytes;
  return OR_OK;
}

/* FC y[M,N] = x[M,K] w[N,K]^T: MACs = M*K*N; bytes = x + w + y (+ bias). */
int or_fc_intensity(int64_t m, int64_t k, int64_t n, int dt, int has_bias, uint64_t res[3],
                    double *intensity) {
  if (!res || !intensity || !dt_ok(dt) || m <= 0 || k <= 0 || n <= 0) return OR_EINVAL;
  uint64_t macs, t, x_e, w_e, y_e, all, bytes, sz = (uint64_t)dt_size(dt);
  if (!mul_ok((uint64_t)m, (uint64_t)k, &x_e) || !mul_ok(x_e, (uint64_t)n, &macs) ||
      !mul_ok((uint64_t)n, (uint64_t)k, &w_e) || !mul_ok((uint64_t)m, (uint64_t)n, &y_e))
    return OR_EINVAL;
  if (!add_ok(x_e, w_e, &t) || !add_ok(t, y_e, &all) ||
      !add_ok(all, has_bias ? (uint64_t)n : 0, &all) || !mul_ok(all, sz, &bytes))
    return OR_EINVAL;
  if (macs > UINT64_MAX / 2) return OR_EINVAL;
  res[0] = macs;
  res[1] = 2 * macs;
  res[2] = bytes;
  *intensity = (double)res[1] / (double)bytes;
  return OR_OK;
}

/* ------------------------------------------------------------------------ */
/* Routing (Section 2.2 quadrants; fixed-threshold rule, Section 3).          */
/* ------------------------------------------------------------------------ */

/*
 * Returns the path as two bits, or -1 on invalid input.
 *   bit 0 (skip)      : sparsity >= sparsity_thr   (sparse quadrants)
 *   bit 1 (bandwidth) : depthwise, or intensity < intensity_thr
 *                       (light, memory-bound quadrants)
 * sparsity is zero_blocks/num_blocks in BLOCK mode, zeros/numel in ELEMENT
 * mode.
 */
int or_route(uint64_t zeros, uint64_t numel, uint64_t zero_blocks, uint64_t num_blocks,
             double intensity, int is_depthwise, double sparsity_thr, double intensity_thr,
             int mode) {
  if (isnan(sparsity_thr) || isnan(intensity_thr) || isnan(intensity) || sparsity_thr < 0 ||
      intensity_thr < 0 || intensity < 0)
    return -1;
  double rho;
  if (mode == OR_ROUTE_BLOCK) {
    if (num_blocks == 0 || zero_blocks > num_blocks) return -1;
    rho = (double)zero_blocks / (double)num_blocks;
  } else if (mode == OR_ROUTE_ELEMENT) {
    if (numel == 0 || zeros > numel) return -1;
    rho = (double)zeros / (double)numel;
  } else {
    return -1;
  }
  int skip = rho >= sparsity_thr;
  int bw = is_depthwise || intensity < intensity_thr;
  return skip | (bw << 1);
}

/* ------------------------------------------------------------------------ */
/* Direct convolution and FC (double accumulation).                           */
/* ------------------------------------------------------------------------ */

static double act_apply(double v, int act) {
  if (act == OR_ACT_RELU) return v > 0 ? v : 0.0;
  if (act == OR_ACT_RELU6) return v > 0 ? (v < 6 ? v : 6.0) : 0.0;
  return v;
}

static int mask_bit(const uint32_t *mask, int64_t idx) { return (mask[idx >> 5] >> (idx & 31)) & 1; }

/*
 * 2-D convolution (cross-correlation, as in DNN frameworks).
 *   x : NHWC [n][h][w][cin]             w : [cout][kh][kw][cin/groups]
 *   bias : [cout] or NULL               residual : NHWC [n][ho][wo][cout] or NULL
 *   y = act(bias + sum x*w + residual), evaluated in double (the residual
 *   joins the sum before the activation, as in a ResNet bottleneck).
 *   y_out, a_out : [n][ho][wo][cout]; a_out = |bias| + sum |x*w| (+ |residual|),
 *   the scale of the rounding error of any summation order.
 * skip_mask (or NULL): bitmap over the [n*h*w, cin] view of x with
 *   skip_rows x skip_cols blocks (as or_measure writes it); every product whose
 *   x element lies in a zero block is left out of the sum (zero skipping).
 * *macs counts one MAC per (output element, tap, input channel of the group),
 *   padding taps included: the dense-equivalent work of Eq. 2.
 */
int or_conv2d(int64_t n, int64_t cin, int64_t h, int64_t w, int64_t cout, int64_t kh, int64_t kw,
              int64_t sh, int64_t sw, int64_t ph, int64_t pw, int64_t dh, int64_t dw,
              int64_t groups, int dt, const void *x, const void *wt, const void *bias,
              const void *residual, int act, const uint32_t *skip_mask, int64_t skip_rows,
              int64_t skip_cols, double *y_out, double *a_out, uint64_t *macs) {
  if (!x || !wt || !y_out || !dt_ok(dt) || n <= 0 || cin <= 0 || cout <= 0 || groups <= 0 ||
      cin % groups || cout % groups)
    return OR_EINVAL;
  if (skip_mask && (skip_rows <= 0 || skip_cols <= 0)) return OR_EINVAL;
  int64_t ho_n = or_out_dim(h, kh, sh, ph, dh), wo_n = or_out_dim(w, kw, sw, pw, dw);
  if (ho_n <= 0 || wo_n <= 0) return OR_EINVAL;
  int64_t cin_g = cin / groups, cout_g = cout / groups;
  int64_t nbc = skip_mask ? (cin + skip_cols - 1) / skip_cols : 0;
  uint64_t mac_count = 0;
#pragma omp parallel for collapse(2) schedule(static) reduction(+ : mac_count)
  for (int64_t in = 0; in < n; ++in)
    for (int64_t co = 0; co < cout; ++co) {
      int64_t g = co / cout_g;
      for (int64_t oh = 0; oh < ho_n; ++oh)
        for (int64_t ow = 0; ow < wo_n; ++ow) {
          double acc = bias ? elem(bias, dt, co) : 0.0;
          double mag = fabs(acc);
          for (int64_t r = 0; r < kh; ++r)
            for (int64_t s = 0; s < kw; ++s) {
              mac_count += (uint64_t)cin_g;
              int64_t ih = oh * sh - ph + r * dh, iw = ow * sw - pw + s * dw;
              if (ih < 0 || ih >= h || iw < 0 || iw >= w) continue; /* zero padding */
              int64_t pix = (in * h + ih) * w + iw;
              for (int64_t ci = 0; ci < cin_g; ++ci) {
                int64_t c = g * cin_g + ci;
                if (skip_mask &&
                    !mask_bit(skip_mask, (pix / skip_rows) * nbc + c / skip_cols))
                  continue;
                double p = elem(x, dt, pix * cin + c) *
                           elem(wt, dt, ((co * kh + r) * kw + s) * cin_g + ci);
                acc += p;
                mag += fabs(p);
              }
            }
          int64_t o = ((in * ho_n + oh) * wo_n + ow) * cout + co;
          if (residual) {
            double rv = elem(residual, dt, o);
            acc += rv;
            mag += fabs(rv);
          }
          y_out[o] = act_apply(acc, act);
          if (a_out) a_out[o] = mag;
        }
    }
  if (macs) *macs = mac_count;
  return OR_OK;
}

/*
 * Fully connected: y[m][j] = act(bias[j] + sum_k x[m][k] * w[j][k] + residual[m][j]).
 *   x : [m][k], w : [n][k] (output-feature major), residual : [m][n] or NULL,
 *   y_out, a_out : [m][n].
 * skip_mask (or NULL): bitmap over the [m, k] view of x with skip_rows x
 * skip_cols blocks; terms whose x element lies in a zero block are skipped.
 */
int or_fc(int64_t m, int64_t k, int64_t n, int dt, const void *x, const void *wt,
          const void *bias, const void *residual, int act, const uint32_t *skip_mask,
          int64_t skip_rows, int64_t skip_cols, double *y_out, double *a_out) {
  if (!x || !wt || !y_out || !dt_ok(dt) || m <= 0 || k <= 0 || n <= 0) return OR_EINVAL;
  if (skip_mask && (skip_rows <= 0 || skip_cols <= 0)) return OR_EINVAL;
  int64_t nbc = skip_mask ? (k + skip_cols - 1) / skip_cols : 0;
#pragma omp parallel for collapse(2) schedule(static)
  for (int64_t i = 0; i < m; ++i)
    for (int64_t j = 0; j < n; ++j) {
      double acc = bias ? elem(bias, dt, j) : 0.0;
      double mag = fabs(acc);
      for (int64_t kk = 0; kk < k; ++kk) {
        if (skip_mask && !mask_bit(skip_mask, (i / skip_rows) * nbc + kk / skip_cols)) continue;
        double p = elem(x, dt, i * k + kk) * elem(wt, dt, j * k + kk);
        acc += p;
        mag += fabs(p);
      }
      if (residual) {
        double rv = elem(residual, dt, i * n + j);
        acc += rv;
        mag += fabs(rv);
      }
      y_out[i * n + j] = act_apply(acc, act);
      if (a_out) a_out[i * n + j] = mag;
    }
  return OR_OK;
}

/*
 * Sampled conv outputs: the same definition as or_conv2d, evaluated only at
 * the `count` NHWC output offsets in idx (for checks at full size).
 */
int or_conv2d_at(int64_t n, int64_t cin, int64_t h, int64_t w, int64_t cout, int64_t kh,
                 int64_t kw, int64_t sh, int64_t sw, int64_t ph, int64_t pw, int64_t dh,
                 int64_t dw, int64_t groups, int dt, const void *x, const void *wt,
                 const void *bias, const void *residual, int act, const int64_t *idx,
                 int64_t count, double *y_out, double *a_out) {
  if (!x || !wt || !idx || !y_out || !dt_ok(dt) || n <= 0 || cin <= 0 || cout <= 0 ||
      groups <= 0 || cin % groups || cout % groups || count < 0)
    return OR_EINVAL;
  int64_t ho_n = or_out_dim(h, kh, sh, ph, dh), wo_n = or_out_dim(w, kw, sw, pw, dw);
  if (ho_n <= 0 || wo_n <= 0) return OR_EINVAL;
  int64_t cin_g = cin / groups, cout_g = cout / groups;
  int64_t total = n * ho_n * wo_n * cout;
  for (int64_t t = 0; t < count; ++t)
    if (idx[t] < 0 || idx[t] >= total) return OR_EINVAL;
#pragma omp parallel for schedule(static)
  for (int64_t t = 0; t < count; ++t) {
    int64_t o = idx[t];
    int64_t co = o % cout, ow = (o / cout) % wo_n, oh = (o / cout / wo_n) % ho_n,
            in = o / cout / wo_n / ho_n;
    int64_t g = co / cout_g;
    double acc = bias ? elem(bias, dt, co) : 0.0;
    double mag = fabs(acc);
    for (int64_t r = 0; r < kh; ++r)
      for (int64_t s = 0; s < kw; ++s) {
        int64_t ih = oh * sh - ph + r * dh, iw = ow * sw - pw + s * dw;
        if (ih < 0 || ih >= h || iw < 0 || iw >= w) continue;
        int64_t pix = (in * h + ih) * w + iw;
        for (int64_t ci = 0; ci < cin_g; ++ci) {
          double p = elem(x, dt, pix * cin + g * cin_g + ci) *
                     elem(wt, dt, ((co * kh + r) * kw + s) * cin_g + ci);
          acc += p;
          mag += fabs(p);
        }
      }
    if (residual) {
      double rv = elem(residual, dt, o);
      acc += rv;
      mag += fabs(rv);
    }
    y_out[t] = act_apply(acc, act);
    if (a_out) a_out[t] = mag;
  }
  return OR_OK;
}

/* ------------------------------------------------------------------------ */
/* Executed work of a block-skipping kernel, from the input values.          */
/* ------------------------------------------------------------------------ */

/*
 * FC: number of (row tile, K block) pairs of x[m][k] -- row tiles of
 * tile_rows rows, K blocks of block_k columns, both clipped at the edge --
 * that hold at least one nonzero element.  A kernel that skips all-zero
 * pairs executes exactly this many.
 */
int or_fc_executed_blocks(const void *x, int dt, int64_t m, int64_t k, int64_t tile_rows,
                          int64_t block_k, uint64_t *out) {
  if (!x || !out || !dt_ok(dt) || m <= 0 || k <= 0 || tile_rows <= 0 || block_k <= 0)
    return OR_EINVAL;
  uint64_t cnt = 0;
  for (int64_t t0 = 0; t0 < m; t0 += tile_rows)
    for (int64_t k0 = 0; k0 < k; k0 += block_k) {
      int nz = 0;
      for (int64_t i = t0; i < m && i < t0 + tile_rows; ++i)
        for (int64_t kk = k0; kk < k && kk < k0 + block_k; ++kk)
          if (!elem_is_zero(x, dt, i * k + kk)) nz = 1;
      cnt += (uint64_t)nz;
    }
  *out = cnt;
  return OR_OK;
}

/*
 * Convolution (groups == 1): the implicit-GEMM view has rows = output pixels
 * (n, oh, ow) in NHWC order and K = (r, s, c) taps x channels.  For every
 * tile of tile_rows consecutive output pixels and every (r, s, channel block
 * of block_c channels), the gathered input block is nonzero iff some output
 * pixel of the tile reads an in-bounds input pixel at that tap with a nonzero
 * channel in the block.  *out = number of nonzero (tile, tap, channel block)
 * triples.
 */
int or_conv_executed_blocks(const void *x, int dt, int64_t n, int64_t cin, int64_t h, int64_t w,
                            int64_t kh, int64_t kw, int64_t sh, int64_t sw, int64_t ph,
                            int64_t pw, int64_t dh, int64_t dw, int64_t tile_rows,
                            int64_t block_c, uint64_t *out) {
  if (!x || !out || !dt_ok(dt) || n <= 0 || cin <= 0 || tile_rows <= 0 || block_c <= 0)
    return OR_EINVAL;
  int64_t ho_n = or_out_dim(h, kh, sh, ph, dh), wo_n = or_out_dim(w, kw, sw, pw, dw);
  if (ho_n <= 0 || wo_n <= 0) return OR_EINVAL;
  int64_t rows = n * ho_n * wo_n;
  uint64_t cnt = 0;
  for (int64_t t0 = 0; t0 < rows; t0 += tile_rows)
    for (int64_t r = 0; r < kh; ++r)
      for (int64_t s = 0; s < kw; ++s)
        for (int64_t c0 = 0; c0 < cin; c0 += block_c) {
          int nz = 0;
          for (int64_t p = t0; p < rows && p < t0 + tile_rows && !nz; ++p) {
            int64_t ow = p % wo_n, oh = (p / wo_n) % ho_n, in = p / wo_n / ho_n;
            int64_t ih = oh * sh - ph + r * dh, iw = ow * sw - pw + s * dw;
            if (ih < 0 || ih >= h || iw < 0 || iw >= w) continue;
            for (int64_t c = c0; c < cin && c < c0 + block_c; ++c)
              if (!elem_is_zero(x, dt, ((in * h + ih) * w + iw) * cin + c)) nz = 1;
          }
          cnt += (uint64_t)nz;
        }
  *out = cnt;
  return OR_OK;
}

/*
 * Split execution of one convolution over the skipping and the dense path
 * (the operator split of Algorithm 1, read on one GPU as a split of the
 * operator's row tiles between two kernel paths): the executed (tile, tap,
 * channel block) triples when every tile of tile_rows output pixels is routed
 * on its own.  A tile whose pixels come from input samples s0..s1 skips iff
 *     zeros(x[s0..s1]) / ((s1 - s0 + 1) * h * w * cin) >= sparsity_thr
 * (one double division; zeros counted element by element over the whole
 * samples) and then executes its nonzero triples as above; otherwise it
 * executes all kh * kw * ceil(cin / block_c) of them.  An FC is the case
 * h = w = kh = kw = 1 with one sample per row.
 */
int or_conv_split_executed_blocks(const void *x, int dt, int64_t n, int64_t cin, int64_t h,
                                  int64_t w, int64_t kh, int64_t kw, int64_t sh, int64_t sw,
                                  int64_t ph, int64_t pw, int64_t dh, int64_t dw,
                                  int64_t tile_rows, int64_t block_c, double sparsity_thr,
                                  uint64_t *out) {
  if (!x || !out || !dt_ok(dt) || n <= 0 || cin <= 0 || tile_rows <= 0 || block_c <= 0 ||
      !(sparsity_thr >= 0))
    return OR_EINVAL;
  int64_t ho_n = or_out_dim(h, kh, sh, ph, dh), wo_n = or_out_dim(w, kw, sw, pw, dw);
  if (ho_n <= 0 || wo_n <= 0) return OR_EINVAL;
  const int64_t rows = n * ho_n * wo_n, per = ho_n * wo_n, snum = h * w * cin;
  uint64_t *sz = (uint64_t *)calloc((size_t)n, sizeof(uint64_t));
  if (!sz) return OR_EINVAL;
  for (int64_t s = 0; s < n; ++s)
    for (int64_t e = 0; e < snum; ++e)
      if (elem_is_zero(x, dt, s * snum + e)) ++sz[s];
  const uint64_t all = (uint64_t)(kh * kw) * (uint64_t)((cin + block_c - 1) / block_c);
  uint64_t cnt = 0;
  for (int64_t t0 = 0; t0 < rows; t0 += tile_rows) {
    const int64_t t1 = (t0 + tile_rows < rows ? t0 + tile_rows : rows) - 1;
    const int64_t s0 = t0 / per, s1 = t1 / per;
    uint64_t z = 0;
    for (int64_t s = s0; s <= s1; ++s) z += sz[s];
    const double rho = (double)z / (double)((uint64_t)(s1 - s0 + 1) * (uint64_t)snum);
    if (!(rho >= sparsity_thr)) {
      cnt += all;
      continue;
    }
    for (int64_t r = 0; r < kh; ++r)
      for (int64_t q = 0; q < kw; ++q)
        for (int64_t c0 = 0; c0 < cin; c0 += block_c) {
          int nz = 0;
          for (int64_t p = t0; p <= t1 && !nz; ++p) {
            int64_t ow = p % wo_n, oh = (p / wo_n) % ho_n, in = p / wo_n / ho_n;
            int64_t ih = oh * sh - ph + r * dh, iw = ow * sw - pw + q * dw;
            if (ih < 0 || ih >= h || iw < 0 || iw >= w) continue;
            for (int64_t c = c0; c < cin && c < c0 + block_c; ++c)
              if (!elem_is_zero(x, dt, ((in * h + ih) * w + iw) * cin + c)) nz = 1;
          }
          cnt += (uint64_t)nz;
        }
  }
  free(sz);
  *out = cnt;
  return OR_OK;
}

/* ------------------------------------------------------------------------ */
/* Glue: max pooling (not routed).                                            */
/* ------------------------------------------------------------------------ */

/*
 * NHWC max pooling with a k x k window, stride s, padding p (padding never
 * wins).  y_out : [n][ho][wo][c] in double.
 */
int or_maxpool2d(int64_t n, int64_t c, int64_t h, int64_t w, int64_t k, int64_t s, int64_t p,
                 int dt, const void *x, double *y_out) {
  if (!x || !y_out || !dt_ok(dt) || n <= 0 || c <= 0) return OR_EINVAL;
  int64_t ho_n = or_out_dim(h, k, s, p, 1), wo_n = or_out_dim(w, k, s, p, 1);
  if (ho_n <= 0 || wo_n <= 0) return OR_EINVAL;
  for (int64_t in = 0; in < n; ++in)
    for (int64_t oh = 0; oh < ho_n; ++oh)
      for (int64_t ow = 0; ow < wo_n; ++ow)
        for (int64_t ch = 0; ch < c; ++ch) {
          double best = -INFINITY;
          for (int64_t r = 0; r < k; ++r)
            for (int64_t q = 0; q < k; ++q) {
              int64_t ih = oh * s - p + r, iw = ow * s - p + q;
              if (ih < 0 || ih >= h || iw < 0 || iw >= w) continue;
              double v = elem(x, dt, ((in * h + ih) * w + iw) * c + ch);
              if (v > best) best = v;
            }
          y_out[((in * ho_n + oh) * wo_n + ow) * c + ch] = best;
        }
  return OR_OK;
}

/*
 * Threads of the OpenMP loops above (the CPU-baseline columns time the same
 * loops on one core and on every core).  n <= 0 leaves the setting alone.
 * Returns the thread count now in effect.
 */
int or_set_threads(int n) {
  if (n > 0) omp_set_num_threads(n);
  return omp_get_max_threads();
}
