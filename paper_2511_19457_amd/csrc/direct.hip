// Direct NHWC window kernels: depthwise convolution (the bandwidth path of
// the light quadrant, SparOA Section 2.2 -- a 3x3 depthwise layer does
// 9 MACs per input element, 1.8 - 4.5 FLOP/byte, far below the ridge point)
// and max pooling (network glue).
//
// One lane owns V consecutive channels (one 16-byte vector) of a run of
// kRun consecutive output pixels along a row.  The input columns it needs are
// loaded once per kernel row and reused across the run from registers, the
// per-channel weights stay in registers, accumulation is fp32.  Lanes of a
// wave cover consecutive channel vectors, then consecutive pixels, so every
// load and store is a coalesced 16-byte access; HBM sees each input and
// output byte about once.
#include "common.h"
#include "dtype.h"

namespace sparoa {
namespace {

constexpr int kThreads = 256;
constexpr int kRun = 4;          // output pixels per lane along w
constexpr int kMaxTaps = 25;     // kernel windows up to 5 x 5 in registers

struct DwArgs {
  const char *x, *w, *bias, *residual;
  char *y;
  int64_t N, H, W, C, Ho, Wo;
  int kh, kw, sh, sw, ph, pw, dh, dw;
  int act;
  DeviceRoute route;
};

template <int DT, int V>
__device__ __forceinline__ void load_vec(const char *p, float *out) {
  using E = Elem<DT>;
  using raw = typename E::raw;
  if constexpr (V * E::size == 16) {
    const uint4 q = *reinterpret_cast<const uint4 *>(p);
    raw e[V];
    __builtin_memcpy(e, &q, 16);
#pragma unroll
    for (int i = 0; i < V; ++i) out[i] = E::to_f32(e[i]);
  } else {
    out[0] = E::to_f32(*reinterpret_cast<const raw *>(p));
  }
}

template <int DT, int V>
__device__ __forceinline__ void store_vec(char *p, const float *v) {
  using E = Elem<DT>;
  using raw = typename E::raw;
  if constexpr (V * E::size == 16) {
    raw e[V];
#pragma unroll
    for (int i = 0; i < V; ++i) e[i] = E::from_f32(v[i]);
    uint4 q;
    __builtin_memcpy(&q, e, 16);
    *reinterpret_cast<uint4 *>(p) = q;
  } else {
    *reinterpret_cast<raw *>(p) = E::from_f32(v[0]);
  }
}

// KH, KW > 0: compile-time window (registers only); 0: runtime window.
template <int DT, int V, int KH, int KW>
__global__ __launch_bounds__(kThreads) void depthwise_kernel(DwArgs a) {
  using E = Elem<DT>;
  using raw = typename E::raw;
  constexpr int ESZ = E::size;
  const int64_t cv = a.C / V;                       // channel vectors per pixel
  const int64_t runs = (a.Wo + kRun - 1) / kRun;    // pixel runs per output row
  const int64_t total = a.N * a.Ho * runs * cv;
  const int kh = KH > 0 ? KH : a.kh, kw = KW > 0 ? KW : a.kw;
  const int taps = kh * kw;
  if (a.route.counts && a.route.path_out && blockIdx.x == 0 && threadIdx.x == 0)
    *a.route.path_out = (device_route_skip(a.route) ? 1u : 0u) | ((uint32_t)a.route.bw_bit << 1);
  for (int64_t i = blockIdx.x * (int64_t)kThreads + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * kThreads) {
    const int64_t c0 = (i % cv) * V;
    const int64_t run = (i / cv) % runs;
    const int64_t oh = (i / cv / runs) % a.Ho;
    const int64_t n = i / cv / runs / a.Ho;
    const int64_t ow0 = run * kRun;

    float wv[KH > 0 ? KH * KW : kMaxTaps][V];
#pragma unroll
    for (int t = 0; t < taps; ++t)
#pragma unroll
      for (int j = 0; j < V; ++j)
        wv[t][j] = E::to_f32(reinterpret_cast<const raw *>(a.w)[(c0 + j) * taps + t]);

    float acc[kRun][V];
#pragma unroll
    for (int r = 0; r < kRun; ++r)
#pragma unroll
      for (int j = 0; j < V; ++j)
        acc[r][j] = a.bias ? E::to_f32(reinterpret_cast<const raw *>(a.bias)[c0 + j]) : 0.f;

#pragma unroll
    for (int r = 0; r < kh; ++r) {
      const int64_t ih = oh * a.sh - a.ph + (int64_t)r * a.dh;
      if (ih < 0 || ih >= a.H) continue;
      const char *rowp = a.x + ((n * a.H + ih) * a.W) * a.C * ESZ + c0 * ESZ;
#pragma unroll
      for (int s = 0; s < kw; ++s) {
        const float *wt = wv[r * kw + s];
#pragma unroll
        for (int q = 0; q < kRun; ++q) {
          const int64_t ow = ow0 + q;
          const int64_t iw = ow * a.sw - a.pw + (int64_t)s * a.dw;
          if (ow >= a.Wo || iw < 0 || iw >= a.W) continue;
          float xv[V];
          load_vec<DT, V>(rowp + iw * a.C * ESZ, xv);
#pragma unroll
          for (int j = 0; j < V; ++j) acc[q][j] = fmaf(xv[j], wt[j], acc[q][j]);
        }
      }
    }
#pragma unroll
    for (int q = 0; q < kRun; ++q) {
      const int64_t ow = ow0 + q;
      if (ow >= a.Wo) continue;
      const int64_t o = ((n * a.Ho + oh) * a.Wo + ow) * a.C + c0;
      if (a.residual) {
        float rv[V];
        load_vec<DT, V>(a.residual + o * ESZ, rv);
#pragma unroll
        for (int j = 0; j < V; ++j) acc[q][j] += rv[j];
      }
      float v[V];
#pragma unroll
      for (int j = 0; j < V; ++j) v[j] = apply_act(acc[q][j], a.act);
      store_vec<DT, V>(a.y + o * ESZ, v);
    }
  }
}

// Division by a run-time constant through a multiply-high (Granlund and
// Montgomery, 1994): for 0 <= n < 2^31 and 1 <= d < 2^31,
// n / d == (umulhi(n, m) + n) >> l with l = ceil(log2 d) and
// m = floor(2^32 (2^l - d) / d) + 1.
struct FastDiv {
  uint32_t d, m, l;
};

inline FastDiv make_fastdiv(uint32_t d) {
  uint32_t l = 0;
  while ((1ull << l) < d) ++l;
  const uint64_t m = ((1ull << 32) * ((1ull << l) - d)) / d + 1;
  return FastDiv{d, (uint32_t)m, l};
}

__device__ __forceinline__ uint32_t fdiv(uint32_t n, const FastDiv &f) {
  return (__umulhi(n, f.m) + n) >> f.l;
}

// 3x3 depthwise, padding 1, stride S in both directions, 16-byte channel
// vectors.  An item is (n, oh, run of run3<S>() output pixels, channel vector);
// the grid stride is a multiple of the channel-vector count, so a thread
// keeps one channel vector for its whole life and loads its 9 x V weights
// once (nine 16-byte loads: w[c][3][3] is contiguous over the V channels).
// Per item, the 3 x NC input vectors the run needs are loaded unconditionally
// (clamped addresses, zeroed outside the image) so they are all in flight
// at once; each is decoded once and feeds every (output, tap) pair that
// uses it.  Run length: 4 outputs over 6 input columns at stride 1; 2 outputs
// over 5 columns at stride 2 (more lanes in flight, measured faster there).
template <int S>
constexpr int run3() { return S == 1 ? 4 : 2; }

template <int DT, int S>
__global__ __launch_bounds__(kThreads) void dw3x3_kernel(DwArgs a, FastDiv fcv, FastDiv fruns, FastDiv fho) {
  using E = Elem<DT>;
  using raw = typename E::raw;
  constexpr int ESZ = E::size;
  constexpr int V = 16 / ESZ;
  constexpr int R = run3<S>();
  constexpr int NC = (R - 1) * S + 3;  // input columns per kernel row
  const int64_t cv = a.C / V;
  const int64_t runs = (a.Wo + R - 1) / R;
  const int64_t total = a.N * a.Ho * runs * cv;
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  if (a.route.counts && a.route.path_out && blockIdx.x == 0 && threadIdx.x == 0)
    *a.route.path_out = (device_route_skip(a.route) ? 1u : 0u) | ((uint32_t)a.route.bw_bit << 1);
  int64_t i = blockIdx.x * (int64_t)kThreads + threadIdx.x;
  if (i >= total) return;
  const int64_t c0 = (int64_t)((uint32_t)i - fdiv((uint32_t)i, fcv) * (uint32_t)cv) * V;
  float wv[9][V];
  {
    raw we[9 * V];
#pragma unroll
    for (int t = 0; t < 9; ++t) {
      const uint4 q = *reinterpret_cast<const uint4 *>(a.w + (c0 * 9 + t * V) * ESZ);
      __builtin_memcpy(&we[t * V], &q, 16);
    }
#pragma unroll
    for (int j = 0; j < V; ++j)
#pragma unroll
      for (int t = 0; t < 9; ++t) wv[t][j] = E::to_f32(we[j * 9 + t]);
  }
  float bv[V];
  if (a.bias) {
    load_vec<DT, V>(a.bias + c0 * ESZ, bv);
  } else {
#pragma unroll
    for (int j = 0; j < V; ++j) bv[j] = 0.f;
  }
  const int H = (int)a.H, W = (int)a.W;
  for (; i < total; i += stride) {
    const uint32_t rest = fdiv((uint32_t)i, fcv);
    const uint32_t rest2 = fdiv(rest, fruns);
    const int run = (int)(rest - rest2 * (uint32_t)runs);
    const uint32_t n32 = fdiv(rest2, fho);
    const int oh = (int)(rest2 - n32 * (uint32_t)a.Ho);
    const int64_t n = n32;
    const int ow0 = run * R;
    const int ih0 = oh * S - 1, iw0 = ow0 * S - 1;
    uint4 xin[3][NC];
#pragma unroll
    for (int r = 0; r < 3; ++r) {
      const int ih = ih0 + r;
      const bool rv = ih >= 0 && ih < H;
      const int ihc = min(max(ih, 0), H - 1);
      const char *rowp = a.x + (((n * H + ihc) * W) * a.C + c0) * ESZ;
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        const int iw = iw0 + c;
        const bool v = rv && iw >= 0 && iw < W;
        const int iwc = min(max(iw, 0), W - 1);
        const uint4 q = *reinterpret_cast<const uint4 *>(rowp + (int64_t)iwc * a.C * ESZ);
        xin[r][c] = v ? q : make_uint4(0u, 0u, 0u, 0u);
      }
    }
    float acc[R][V];
#pragma unroll
    for (int q = 0; q < R; ++q)
#pragma unroll
      for (int j = 0; j < V; ++j) acc[q][j] = bv[j];
#pragma unroll
    for (int r = 0; r < 3; ++r)
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        raw e[V];
        __builtin_memcpy(e, &xin[r][c], 16);
        float xv[V];
#pragma unroll
        for (int j = 0; j < V; ++j) xv[j] = E::to_f32(e[j]);
#pragma unroll
        for (int q = 0; q < R; ++q) {
          const int s = c - q * S;  // tap column that reads input column c for output q
          if (s < 0 || s > 2) continue;
#pragma unroll
          for (int j = 0; j < V; ++j) acc[q][j] = fmaf(xv[j], wv[r * 3 + s][j], acc[q][j]);
        }
      }
#pragma unroll
    for (int q = 0; q < R; ++q) {
      const int ow = ow0 + q;
      if (ow >= a.Wo) continue;
      const int64_t o = ((n * a.Ho + oh) * a.Wo + ow) * a.C + c0;
      if (a.residual) {
        float rv[V];
        load_vec<DT, V>(a.residual + o * ESZ, rv);
#pragma unroll
        for (int j = 0; j < V; ++j) acc[q][j] += rv[j];
      }
      float v[V];
#pragma unroll
      for (int j = 0; j < V; ++j) v[j] = apply_act(acc[q][j], a.act);
      store_vec<DT, V>(a.y + o * ESZ, v);
    }
  }
}

template <int DT, int V>
__global__ __launch_bounds__(kThreads) void maxpool_kernel(const char *x, char *y, int64_t N,
                                                           int64_t C, int64_t H, int64_t W,
                                                           int64_t Ho, int64_t Wo, int k, int s,
                                                           int p) {
  using E = Elem<DT>;
  constexpr int ESZ = E::size;
  const int64_t cv = C / V;
  const int64_t total = N * Ho * Wo * cv;
  for (int64_t i = blockIdx.x * (int64_t)kThreads + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * kThreads) {
    const int64_t c0 = (i % cv) * V, pix = i / cv;
    const int64_t ow = pix % Wo, oh = (pix / Wo) % Ho, n = pix / Wo / Ho;
    float best[V];
#pragma unroll
    for (int j = 0; j < V; ++j) best[j] = -INFINITY;
    for (int r = 0; r < k; ++r) {
      const int64_t ih = oh * s - p + r;
      if (ih < 0 || ih >= H) continue;
      for (int q = 0; q < k; ++q) {
        const int64_t iw = ow * s - p + q;
        if (iw < 0 || iw >= W) continue;
        float v[V];
        load_vec<DT, V>(x + (((n * H + ih) * W + iw) * C + c0) * ESZ, v);
#pragma unroll
        for (int j = 0; j < V; ++j) best[j] = v[j] > best[j] ? v[j] : best[j];
      }
    }
    store_vec<DT, V>(y + (pix * C + c0) * ESZ, best);
  }
}

template <int DT>
sparoa_status dw_dispatch(const DwArgs &a, hipStream_t st) {
  constexpr int VV = 16 / Elem<DT>::size;
  const bool vec = a.C % VV == 0;
  const int V = vec ? VV : 1;
  const int64_t total = a.N * a.Ho * cdiv(a.Wo, kRun) * (a.C / V);
  int64_t blocks = cdiv(total, kThreads);
  if (blocks > 65536) blocks = 65536;
  const bool k3 = a.kh == 3 && a.kw == 3;
  const bool fast3 = vec && k3 && a.ph == 1 && a.pw == 1 && a.dh == 1 && a.dw == 1 &&
                     a.sh == a.sw && (a.sh == 1 || a.sh == 2);
  const int64_t cv = a.C / VV;
  const int64_t runs = cdiv(a.Wo, a.sh == 1 ? run3<1>() : run3<2>());
  const int64_t items = a.N * a.Ho * runs * cv;
  // item indices and the grid stride stay below 2^31 (32-bit divisions)
  if (fast3 && items < (1ll << 30)) {
    // the grid stride must be a multiple of the channel-vector count
    int64_t g = 256, c = cv;
    while (c) { const int64_t t = g % c; g = c; c = t; }  // gcd(256, cv)
    const int64_t q = cv / g;
    int64_t nb = cdiv(items, kThreads);
    if (nb > 4096) nb = 4096;
    nb = cdiv(nb, q) * q;
    const FastDiv fcv = make_fastdiv((uint32_t)cv), fruns = make_fastdiv((uint32_t)runs),
                  fho = make_fastdiv((uint32_t)a.Ho);
    if (a.sh == 1)
      hipLaunchKernelGGL((dw3x3_kernel<DT, 1>), dim3((unsigned)nb), dim3(kThreads), 0, st, a, fcv, fruns, fho);
    else
      hipLaunchKernelGGL((dw3x3_kernel<DT, 2>), dim3((unsigned)nb), dim3(kThreads), 0, st, a, fcv, fruns, fho);
    SPAROA_LAUNCH_CHECK("dw3x3_kernel");
    return SPAROA_OK;
  }
  if (vec && k3)
    hipLaunchKernelGGL((depthwise_kernel<DT, VV, 3, 3>), dim3((unsigned)blocks), dim3(kThreads), 0, st, a);
  else if (vec)
    hipLaunchKernelGGL((depthwise_kernel<DT, VV, 0, 0>), dim3((unsigned)blocks), dim3(kThreads), 0, st, a);
  else
    hipLaunchKernelGGL((depthwise_kernel<DT, 1, 0, 0>), dim3((unsigned)blocks), dim3(kThreads), 0, st, a);
  SPAROA_LAUNCH_CHECK("depthwise_kernel");
  return SPAROA_OK;
}

template <int DT>
sparoa_status mp_dispatch(const void *x, void *y, int64_t n, int64_t c, int64_t h, int64_t w,
                          int64_t ho, int64_t wo, int k, int s, int p, hipStream_t st) {
  constexpr int VV = 16 / Elem<DT>::size;
  const bool vec = c % VV == 0;
  const int64_t total = n * ho * wo * (c / (vec ? VV : 1));
  int64_t blocks = cdiv(total, kThreads);
  if (blocks > 65536) blocks = 65536;
  const char *xp = static_cast<const char *>(x);
  char *yp = static_cast<char *>(y);
  if (vec)
    hipLaunchKernelGGL((maxpool_kernel<DT, VV>), dim3((unsigned)blocks), dim3(kThreads), 0, st, xp,
                       yp, n, c, h, w, ho, wo, k, s, p);
  else
    hipLaunchKernelGGL((maxpool_kernel<DT, 1>), dim3((unsigned)blocks), dim3(kThreads), 0, st, xp,
                       yp, n, c, h, w, ho, wo, k, s, p);
  SPAROA_LAUNCH_CHECK("maxpool_kernel");
  return SPAROA_OK;
}

}  // namespace

sparoa_status launch_depthwise(const sparoa_conv_desc &d, const void *x, const void *w,
                               const void *bias, const void *residual, sparoa_act act, void *y,
                               hipStream_t stream, const DeviceRoute *route) {
  if (d.kh * d.kw > kMaxTaps) return fail(SPAROA_ERR_UNSUPPORTED, "depthwise window above 5x5");
  DwArgs a;
  a.x = static_cast<const char *>(x);
  a.w = static_cast<const char *>(w);
  a.bias = static_cast<const char *>(bias);
  a.residual = static_cast<const char *>(residual);
  a.y = static_cast<char *>(y);
  a.N = d.n; a.H = d.h; a.W = d.w; a.C = d.c_in;
  a.Ho = (d.h + 2 * d.ph - d.dh * (d.kh - 1) - 1) / d.sh + 1;
  a.Wo = (d.w + 2 * d.pw - d.dw * (d.kw - 1) - 1) / d.sw + 1;
  a.kh = (int)d.kh; a.kw = (int)d.kw; a.sh = (int)d.sh; a.sw = (int)d.sw;
  a.ph = (int)d.ph; a.pw = (int)d.pw; a.dh = (int)d.dh; a.dw = (int)d.dw;
  a.act = act;
  a.route = route ? *route : DeviceRoute{nullptr, 0.0, 0, 0, nullptr};
  switch (d.dtype) {
    case SPAROA_BF16: return dw_dispatch<SPAROA_BF16>(a, stream);
    case SPAROA_F16: return dw_dispatch<SPAROA_F16>(a, stream);
    case SPAROA_F32: return dw_dispatch<SPAROA_F32>(a, stream);
  }
  return fail(SPAROA_ERR_INVALID_ARG, "depthwise: dtype");
}

sparoa_status launch_maxpool(const void *x, sparoa_dtype dt, int64_t n, int64_t c, int64_t h,
                             int64_t w, int64_t k, int64_t s, int64_t p, void *y,
                             hipStream_t stream) {
  const int64_t ho = (h + 2 * p - k) / s + 1, wo = (w + 2 * p - k) / s + 1;
  switch (dt) {
    case SPAROA_BF16: return mp_dispatch<SPAROA_BF16>(x, y, n, c, h, w, ho, wo, (int)k, (int)s, (int)p, stream);
    case SPAROA_F16: return mp_dispatch<SPAROA_F16>(x, y, n, c, h, w, ho, wo, (int)k, (int)s, (int)p, stream);
    case SPAROA_F32: return mp_dispatch<SPAROA_F32>(x, y, n, c, h, w, ho, wo, (int)k, (int)s, (int)p, stream);
  }
  return fail(SPAROA_ERR_INVALID_ARG, "maxpool: dtype");
}

}  // namespace sparoa
