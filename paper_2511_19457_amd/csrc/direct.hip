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
#include "commit.h"
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
  sparoa_counts *om_counts = nullptr;   // non-null: measure y (fused; see dw3x3_kernel)
  uint32_t *om_mask = nullptr;
  unsigned long long *om_words = nullptr;
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
// vectors.  An item is (n, oh, run of R output pixels, channel vector), R
// dividing Wo so runs never cross a row (pixel-run pr = item / cv covers
// pixels pr * R .. pr * R + R - 1); a thread keeps one channel vector for its
// whole life and loads its 9 x V weights once (nine 16-byte loads: w[c][3][3]
// is contiguous over the V channels).  Per item, the 3 x NC input vectors the
// run needs are loaded unconditionally (clamped addresses, zeroed outside the
// image) so they are all in flight at once; each is decoded once and feeds
// every (output, tap) pair that uses it.
template <int DT>
struct Dw3Lane {
  static constexpr int V = 16 / Elem<DT>::size;
  // weights stay in their 16-bit form (half the registers of fp32 copies);
  // fp16 products then map to mixed-precision FMAs with no conversions
  typename Elem<DT>::raw wv[9][V];
  float bv[V];
  __device__ __forceinline__ void load(const DwArgs &a, int64_t c0) {
    using E = Elem<DT>;
    using raw = typename E::raw;
    raw we[9 * V];
#pragma unroll
    for (int t = 0; t < 9; ++t) {
      const uint4 q = *reinterpret_cast<const uint4 *>(a.w + (c0 * 9 + t * V) * E::size);
      __builtin_memcpy(&we[t * V], &q, 16);
    }
#pragma unroll
    for (int j = 0; j < V; ++j)
#pragma unroll
      for (int t = 0; t < 9; ++t) wv[t][j] = we[j * 9 + t];
    if (a.bias) {
      load_vec<DT, V>(a.bias + c0 * E::size, bv);
    } else {
#pragma unroll
      for (int j = 0; j < V; ++j) bv[j] = 0.f;
    }
  }
};

// One item in flight: its output position and its NR x NC input vectors.  An
// item is RH output rows x a run of R output pixels of one channel vector;
// with RH = 2 at stride 1 the two rows share two of their four input rows,
// so an output takes 3 instead of 4.5 loads at R = 4.
template <int S, int R, int RH>
struct Dw3Item {
  static constexpr int NC = (R - 1) * S + 3;   // input columns per kernel row
  static constexpr int NR = (RH - 1) * S + 3;  // input rows
  int64_t o;            // element offset of the item's first output vector
  uint4 xin[NR][NC];
};

// Issues the input loads of item i (buffer loads: a tap outside the image
// takes an offset past the descriptor's range and reads zero without a
// memory access -- no branch, no select; x is under 2^31 bytes).
// fho divides by Ho / RH (row groups per image).
template <int DT, int S, int R, int RH>
__device__ __forceinline__ void dw3_fetch(const DwArgs &a, __amdgpu_buffer_rsrc_t xrs, uint32_t i,
                                          int64_t c0, const FastDiv &fcv, const FastDiv &fruns,
                                          const FastDiv &fho, Dw3Item<S, R, RH> &it) {
  constexpr int ESZ = Elem<DT>::size;
  constexpr int NC = Dw3Item<S, R, RH>::NC, NR = Dw3Item<S, R, RH>::NR;
  const int H = (int)a.H, W = (int)a.W;
  const uint32_t runs = (uint32_t)(a.Wo / R), groups = (uint32_t)(a.Ho / RH);
  const uint32_t rest = fdiv(i, fcv);   // pixel-run
  const uint32_t rest2 = fdiv(rest, fruns);
  const int run = (int)(rest - rest2 * runs);
  const uint32_t n32 = fdiv(rest2, fho);
  const int oh = (int)(rest2 - n32 * groups) * RH;
  const int64_t n = n32;
  const int ow0 = run * R;
  const int ih0 = oh * S - 1, iw0 = ow0 * S - 1;
  it.o = ((n * a.Ho + oh) * a.Wo + ow0) * a.C + c0;
  const uint32_t pix_bytes = (uint32_t)(a.C * ESZ);
#pragma unroll
  for (int r = 0; r < NR; ++r) {
    const int ih = ih0 + r;
    const bool rv = ih >= 0 && ih < H;
    const uint32_t row_off = (uint32_t)((n * H + ih) * W) * pix_bytes + (uint32_t)(c0 * ESZ);
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const int iw = iw0 + c;
      const bool v = rv && iw >= 0 && iw < W;
      const uint32_t off = v ? row_off + (uint32_t)iw * pix_bytes : 0x80000000u;
      it.xin[r][c] =
          __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(xrs, off, 0, 0));
    }
  }
}

// Computes and stores the item's RH x R output vectors.  Returns bit
// rh R + q set iff output vector (rh, q) has a nonzero element; adds its
// zero elements to *zeros.
template <int DT, int S, int R, int RH, bool COUNT>
__device__ __forceinline__ uint32_t dw3_finish(const DwArgs &a, const Dw3Lane<DT> &l,
                                               const Dw3Item<S, R, RH> &it, uint32_t *zeros) {
  using E = Elem<DT>;
  using raw = typename E::raw;
  constexpr int ESZ = E::size;
  constexpr int V = Dw3Lane<DT>::V;
  constexpr int NC = Dw3Item<S, R, RH>::NC, NR = Dw3Item<S, R, RH>::NR;
  float acc[RH][R][V];
#pragma unroll
  for (int h = 0; h < RH; ++h)
#pragma unroll
    for (int q = 0; q < R; ++q)
#pragma unroll
      for (int j = 0; j < V; ++j) acc[h][q][j] = l.bv[j];
  uint32_t nzbits = 0;
  // Input rows in order; output row h is complete after input row h S + 2
  // and is stored there, so its accumulators die before the next rows.
#pragma unroll
  for (int rr = 0; rr < NR; ++rr) {
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      raw e[V];
      __builtin_memcpy(e, &it.xin[rr][c], 16);
      float xv[V];
#pragma unroll
      for (int j = 0; j < V; ++j) xv[j] = E::to_f32(e[j]);
#pragma unroll
      for (int h = 0; h < RH; ++h) {
        const int r = rr - h * S;   // kernel row that reads input row rr for output row h
        if (r < 0 || r > 2) continue;
#pragma unroll
        for (int q = 0; q < R; ++q) {
          const int s = c - q * S;  // kernel column that reads input column c for output q
          if (s < 0 || s > 2) continue;
#pragma unroll
          for (int j = 0; j < V; ++j)
            acc[h][q][j] = fmaf(xv[j], E::to_f32(l.wv[r * 3 + s][j]), acc[h][q][j]);
        }
      }
    }
#pragma unroll
    for (int h = 0; h < RH; ++h) {
      if (h * S + 2 != rr) continue;
#pragma unroll
      for (int q = 0; q < R; ++q) {
        const int64_t o = it.o + (h * a.Wo + q) * a.C;
        if (a.residual) {
          float rv[V];
          load_vec<DT, V>(a.residual + o * ESZ, rv);
#pragma unroll
          for (int j = 0; j < V; ++j) acc[h][q][j] += rv[j];
        }
        raw t[V];
        uint32_t any = 0;   // OR of the magnitudes
#pragma unroll
        for (int j = 0; j < V; ++j) {
          t[j] = E::from_f32(apply_act(acc[h][q][j], a.act));
          if (COUNT) {
            // zero test in plain integer arithmetic (m - 1 wraps to bit 31 iff
            // m == 0; m < 2^31), so no compare masks occupy scalar registers
            const uint32_t m = (uint32_t)t[j] & E::mag_mask;   // 0 for +0 and -0
            *zeros += (m - 1u) >> 31;
            any |= m;
          }
        }
        if (COUNT) nzbits |= (((any - 1u) >> 31) ^ 1u) << (h * R + q);
        uint4 qv;
        __builtin_memcpy(&qv, t, 16);
        *reinterpret_cast<uint4 *>(a.y + o * ESZ) = qv;
      }
    }
  }
  return nzbits;
}

template <int DT>
__device__ __forceinline__ __amdgpu_buffer_rsrc_t dw3_x_rsrc(const DwArgs &a) {
  return __builtin_amdgcn_make_buffer_rsrc((void *)a.x, (short)0,
                                           (int)(a.N * a.H * a.W * a.C * Elem<DT>::size),
                                           kBufDword3);
}

// Work-groups are dispatched to the 8 XCDs round robin (b -> XCD b % 8), each
// XCD with its own L2.  With nb % 8 == 0 this maps them to logical blocks so
// that each XCD walks one contiguous eighth of the items: adjacent output
// rows, which read two of their three input rows in common, then share an L2
// (consecutive ids would put them on different XCDs and fetch every input
// row three times from HBM).  A bijection on [0, nb) either way.
__device__ __forceinline__ int64_t xcd_block(int64_t b, int64_t nb) {
  return (nb & 7) ? b : (b & 7) * (nb >> 3) + (b >> 3);
}

// Plain walk: a grid of up to 4096 work-groups (most lanes get a single
// item) striding over items by a multiple of cv, so a thread's channel
// vector never changes.  The first item's inputs are requested before the
// lane's weights, so both arrive in one round trip.  COUNT: the counts-only
// output measurement (Section 3.1, Eq. 1, at block (1 pixel, 8 channels) =
// one output vector, no bitmap): zeros and nonzero vectors per lane, one
// ticketed commit per work-group.  Two waves per SIMD at least: the
// counting form of the 2 x 4 item would otherwise take 258 registers and one
// wave; capped at 256 it spills a few bytes per lane and is still 10-15%
// faster than 1 x 4 items on the stride-1 MobileNetV2 layers.
template <int DT, int S, int R, int RH, bool COUNT>
__global__ __launch_bounds__(kThreads, 2) void dw3x3_kernel(DwArgs a, FastDiv fcv, FastDiv fruns,
                                                        FastDiv fho) {
  const int64_t cv = a.C / Dw3Lane<DT>::V;
  const int64_t total = a.N * (a.Ho / RH) * (a.Wo / R) * cv;
  SPAROA_ARGS_UP_FRONT("s"(a.x), "s"(a.w), "s"(a.bias), "s"(a.residual), "s"(a.y), "s"(a.N),
                       "s"(a.H), "s"(a.W), "s"(a.C), "s"(a.Ho), "s"(a.Wo), "s"(a.act),
                       "s"(a.om_counts), "s"(a.route.counts), "s"(gridDim.x), "s"(fcv.m),
                       "s"(fcv.l), "s"(fruns.m), "s"(fruns.l), "s"(fho.m), "s"(fho.l));
  // the route's counts are requested with the first item's loads; work-group
  // 0 records the path once they are in (behind no other work-group's start)
  const RouteCountsReq rq = route_counts_request(a.route);
  int64_t i = xcd_block(blockIdx.x, gridDim.x) * kThreads + threadIdx.x;
  if (!COUNT && i >= total) return;   // (COUNT: every thread reaches the commit)
  uint32_t zeros = 0, nz = 0;
  if (i < total) {
    const int64_t c0 = (int64_t)((uint32_t)i - fdiv((uint32_t)i, fcv) * (uint32_t)cv) *
                       Dw3Lane<DT>::V;
    const __amdgpu_buffer_rsrc_t xrs = dw3_x_rsrc<DT>(a);
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    Dw3Item<S, R, RH> it;
    dw3_fetch<DT, S, R, RH>(a, xrs, (uint32_t)i, c0, fcv, fruns, fho, it);
    Dw3Lane<DT> l;
    l.load(a, c0);
    if (a.route.counts && a.route.path_out && blockIdx.x == 0 && threadIdx.x == 0)
      *a.route.path_out = (route_counts_skip(rq, a.route) ? 1u : 0u) | ((uint32_t)a.route.bw_bit << 1);
    for (;;) {
      const uint32_t bits = dw3_finish<DT, S, R, RH, COUNT>(a, l, it, &zeros);
      if (COUNT) nz += (uint32_t)__popc(bits);
      i += stride;
      if (i >= total) break;
      dw3_fetch<DT, S, R, RH>(a, xrs, (uint32_t)i, c0, fcv, fruns, fho, it);
    }
  }
  if (COUNT) om_commit(zeros, nz, a.om_counts, a.om_words, blockIdx.x, gridDim.x);
}

// Measured walk with the bitmap: the same convolution with the output
// measurement of Section 3.1 (Eq. 1) on y, bitmap at block (1 pixel, 8
// channels) = one output vector.  One output vector per lane (runs of 1), so
// the item index is the block index and a wave's 64 items, starting at a
// multiple of 64, are two whole bitmap words: the wave ballots them and two
// lanes store them (no atomics, no clearing).  The grid stride (as in the
// plain walk, up to 4096 work-groups) is a multiple of 64 and of cv.
template <int DT, int S>
__global__ __launch_bounds__(kThreads) void dw3x3_measured_kernel(DwArgs a, FastDiv fcv,
                                                                 FastDiv fwo, FastDiv fho,
                                                                 int64_t om_words) {
  const int lane = threadIdx.x & 63;
  const int64_t cv = a.C / Dw3Lane<DT>::V;
  const int64_t total = a.N * a.Ho * a.Wo * cv;
  SPAROA_ARGS_UP_FRONT("s"(a.x), "s"(a.w), "s"(a.bias), "s"(a.residual), "s"(a.y), "s"(a.N),
                       "s"(a.H), "s"(a.W), "s"(a.C), "s"(a.Ho), "s"(a.Wo), "s"(a.act),
                       "s"(a.om_counts), "s"(a.route.counts), "s"(gridDim.x), "s"(fcv.m),
                       "s"(fcv.l), "s"(fwo.m), "s"(fwo.l), "s"(fho.m), "s"(fho.l));
  // the route's counts are requested with the first item's loads; work-group
  // 0 records the path once they are in (behind no other work-group's start)
  const RouteCountsReq rq = route_counts_request(a.route);
  const int64_t first = xcd_block(blockIdx.x, gridDim.x) * kThreads + threadIdx.x;
  const int64_t c0 = (int64_t)((uint32_t)first - fdiv((uint32_t)first, fcv) * (uint32_t)cv) *
                     Dw3Lane<DT>::V;
  const __amdgpu_buffer_rsrc_t xrs = dw3_x_rsrc<DT>(a);
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  uint32_t zeros = 0, nz = 0;
  Dw3Item<S, 1, 1> it;
  if (first < total) dw3_fetch<DT, S, 1, 1>(a, xrs, (uint32_t)first, c0, fcv, fwo, fho, it);
  Dw3Lane<DT> l;
  l.load(a, c0);
  if (a.route.counts && a.route.path_out && blockIdx.x == 0 && threadIdx.x == 0)
    *a.route.path_out = (route_counts_skip(rq, a.route) ? 1u : 0u) | ((uint32_t)a.route.bw_bit << 1);
  for (int64_t base = first - lane; base < total; base += stride) {   // wave-uniform
    const int64_t i = base + lane;
    uint32_t bits = 0;
    if (i < total) bits = dw3_finish<DT, S, 1, 1, true>(a, l, it, &zeros);
    const uint64_t bal = __ballot(bits != 0u);
    const int64_t w0 = base >> 5;
    if (lane == 0 && w0 < om_words) a.om_mask[w0] = (uint32_t)bal;
    if (lane == 32 && w0 + 1 < om_words) a.om_mask[w0 + 1] = (uint32_t)(bal >> 32);
    nz += lane == 0 ? (uint32_t)__popcll(bal) : 0u;
    if (i + stride < total)
      dw3_fetch<DT, S, 1, 1>(a, xrs, (uint32_t)(i + stride), c0, fcv, fwo, fho, it);
  }
  om_commit(zeros, nz, a.om_counts, a.om_words, blockIdx.x, gridDim.x);
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

// The same pooling with 32-bit indices (items and x below 2^31 elements):
// the item decomposes by multiply-shift divisions (a 64-bit division per
// item made the general kernel ALU-bound at about 3.4 TB/s), one item per
// lane.
template <int DT, int V>
__global__ __launch_bounds__(kThreads) void maxpool32_kernel(const char *x, char *y, int C, int H,
                                                             int W, int Ho, int Wo, int k, int s,
                                                             int p, uint32_t total, FastDiv fcv,
                                                             FastDiv fwo, FastDiv fho) {
  SPAROA_ARGS_UP_FRONT("s"(x), "s"(y), "s"(C), "s"(H), "s"(W), "s"(total), "s"(fcv.m),
                       "s"(fcv.l), "s"(fwo.m), "s"(fwo.l), "s"(fho.m), "s"(fho.l));
  using E = Elem<DT>;
  constexpr int ESZ = E::size;
  const uint32_t i = blockIdx.x * (uint32_t)kThreads + threadIdx.x;
  if (i >= total) return;
  const uint32_t pix = fdiv(i, fcv), t = fdiv(pix, fwo), n = fdiv(t, fho);
  const int c0 = (int)(i - pix * fcv.d) * V;
  const int ow = (int)(pix - t * fwo.d), oh = (int)(t - n * fho.d);
  float best[V];
#pragma unroll
  for (int j = 0; j < V; ++j) best[j] = -INFINITY;
  for (int r = 0; r < k; ++r) {
    const int ih = oh * s - p + r;
    if (ih < 0 || ih >= H) continue;
    for (int q = 0; q < k; ++q) {
      const int iw = ow * s - p + q;
      if (iw < 0 || iw >= W) continue;
      float v[V];
      load_vec<DT, V>(x + (size_t)((((int)n * H + ih) * W + iw) * C + c0) * ESZ, v);
#pragma unroll
      for (int j = 0; j < V; ++j) best[j] = v[j] > best[j] ? v[j] : best[j];
    }
  }
  store_vec<DT, V>(y + (size_t)((int)pix * C + c0) * ESZ, best);
}

// Run length of the 3x3 kernel: 4 outputs along w at stride 1 where 4
// divides Wo, else 2 where Wo is even, else 1 (a run never crosses a row).
// Longer runs re-read fewer input columns per output.
int dw_run(int64_t wo, int64_t s) {
  if (s == 1 && wo % 4 == 0) return 4;
  return wo % 2 == 0 ? 2 : 1;
}

bool dw_fast3(const DwArgs &a, int esz) {
  return a.C % (16 / esz) == 0 && a.kh == 3 && a.kw == 3 && a.ph == 1 && a.pw == 1 &&
         a.dh == 1 && a.dw == 1 && a.sh == a.sw && (a.sh == 1 || a.sh == 2);
}

int64_t gcd64(int64_t a, int64_t b) {
  while (b) { const int64_t t = a % b; a = b; b = t; }
  return a;
}

// Work-group count of a walk over `items` whose stride (nb x 256 items) must
// be a multiple of cv: a multiple of q = cv / gcd(256, cv) and of 8 (XCD
// mapping), at most `cap` unless one multiple is more.
int64_t dw_grid(int64_t items, int64_t cv, int64_t cap) {
  const int64_t q = cv / gcd64(kThreads, cv);
  const int64_t unit = q * 8 / gcd64(q, 8);
  int64_t nb = cdiv(items, kThreads);
  if (nb > cap) nb = cap;
  nb = cdiv(nb, unit) * unit;
  return nb;
}

template <int DT, int S, int R, int RH>
sparoa_status launch_dw3(const DwArgs &a, hipStream_t st, const FastDiv &fcv, int64_t cv) {
  const int64_t runs = a.Wo / R;
  const int64_t items = a.N * (a.Ho / RH) * runs * cv;
  const FastDiv fruns = make_fastdiv((uint32_t)runs), fho = make_fastdiv((uint32_t)(a.Ho / RH));
  const int64_t nb = dw_grid(items, cv, 4096);
  if (a.om_counts)   // counts only (no bitmap)
    hipLaunchKernelGGL((dw3x3_kernel<DT, S, R, RH, true>), dim3((unsigned)nb), dim3(kThreads), 0,
                       st, a, fcv, fruns, fho);
  else
    hipLaunchKernelGGL((dw3x3_kernel<DT, S, R, RH, false>), dim3((unsigned)nb), dim3(kThreads),
                       0, st, a, fcv, fruns, fho);
  SPAROA_LAUNCH_CHECK("dw3x3_kernel");
  return SPAROA_OK;
}

template <int DT, int S>
sparoa_status launch_dw3_measured(const DwArgs &a, hipStream_t st, const FastDiv &fcv,
                                  int64_t cv) {
  const int64_t items = a.N * a.Ho * a.Wo * cv;
  const int64_t nb = dw_grid(items, cv, 4096);
  const int64_t om_words = cdiv(items, 32);
  hipLaunchKernelGGL((dw3x3_measured_kernel<DT, S>), dim3((unsigned)nb), dim3(kThreads), 0, st,
                     a, fcv, make_fastdiv((uint32_t)a.Wo), make_fastdiv((uint32_t)a.Ho),
                     om_words);
  SPAROA_LAUNCH_CHECK("dw3x3_measured_kernel");
  return SPAROA_OK;
}

// The 3x3 fast path's limits: item indices and the grid stride stay below
// 2^31 (32-bit divisions), x below 2^31 bytes (32-bit buffer offsets).
bool dw3_fits(const DwArgs &a, int esz) {
  return dw_fast3(a, esz) && a.N * a.Ho * a.Wo * (a.C / (16 / esz)) < (1ll << 30) &&
         a.N * a.H * a.W * a.C * esz < (1ll << 31);
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
  if (dw3_fits(a, Elem<DT>::size)) {
    const int64_t cv = a.C / VV;
    const FastDiv fcv = make_fastdiv((uint32_t)cv);
    if (a.om_counts) {
      if constexpr (Elem<DT>::size == 2) {
        if (a.om_mask)   // the bitmap too: one output vector per lane
          return a.sh == 1 ? launch_dw3_measured<DT, 1>(a, st, fcv, cv)
                           : launch_dw3_measured<DT, 2>(a, st, fcv, cv);
      } else {
        return fail(SPAROA_ERR_UNSUPPORTED, "depthwise: no fused output measurement");
      }
    }
    const int R = dw_run(a.Wo, a.sh);
    if (a.sh == 1) {
      // two output rows per item where Ho is even (stride 1: 3 loads per
      // output at runs of 4 instead of 4.5)
      const bool rows2 = a.Ho % 2 == 0;
      if (R == 4)
        return rows2 ? launch_dw3<DT, 1, 4, 2>(a, st, fcv, cv) : launch_dw3<DT, 1, 4, 1>(a, st, fcv, cv);
      if (R == 2)
        return rows2 ? launch_dw3<DT, 1, 2, 2>(a, st, fcv, cv) : launch_dw3<DT, 1, 2, 1>(a, st, fcv, cv);
      return rows2 ? launch_dw3<DT, 1, 1, 2>(a, st, fcv, cv) : launch_dw3<DT, 1, 1, 1>(a, st, fcv, cv);
    }
    if (R == 2) return launch_dw3<DT, 2, 2, 1>(a, st, fcv, cv);
    return launch_dw3<DT, 2, 1, 1>(a, st, fcv, cv);
  }
  if (a.om_counts) return fail(SPAROA_ERR_UNSUPPORTED, "depthwise: no fused output measurement");
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
  if (vec && total < (1ll << 31) && n * h * w * c < (1ll << 31) && n * ho * wo * c < (1ll << 31)) {
    const uint32_t cv = (uint32_t)(c / VV);
    hipLaunchKernelGGL((maxpool32_kernel<DT, VV>), dim3((unsigned)cdiv(total, kThreads)),
                       dim3(kThreads), 0, st, xp, yp, (int)c, (int)h, (int)w, (int)ho, (int)wo, k,
                       s, p, (uint32_t)total, make_fastdiv(cv), make_fastdiv((uint32_t)wo),
                       make_fastdiv((uint32_t)ho));
    SPAROA_LAUNCH_CHECK("maxpool32_kernel");
    return SPAROA_OK;
  }
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

namespace {
DwArgs dw_args(const sparoa_conv_desc &d) {
  DwArgs a;
  a.N = d.n; a.H = d.h; a.W = d.w; a.C = d.c_in;
  a.Ho = (d.h + 2 * d.ph - d.dh * (d.kh - 1) - 1) / d.sh + 1;
  a.Wo = (d.w + 2 * d.pw - d.dw * (d.kw - 1) - 1) / d.sw + 1;
  a.kh = (int)d.kh; a.kw = (int)d.kw; a.sh = (int)d.sh; a.sw = (int)d.sw;
  a.ph = (int)d.ph; a.pw = (int)d.pw; a.dh = (int)d.dh; a.dw = (int)d.dw;
  return a;
}
}  // namespace

bool dw_fuses_out_measure(const sparoa_conv_desc &d) {
  return elem_size(d.dtype) == 2 && dw3_fits(dw_args(d), 2);   // one output vector = one block
}

sparoa_status launch_depthwise(const sparoa_conv_desc &d, const void *x, const void *w,
                               const void *bias, const void *residual, sparoa_act act, void *y,
                               hipStream_t stream, const DeviceRoute *route,
                               const OutMeasure *om) {
  if (om && !dw_fuses_out_measure(d))
    return fail(SPAROA_ERR_UNSUPPORTED, "depthwise: no fused output measurement for this shape");
  if (d.kh * d.kw > kMaxTaps) return fail(SPAROA_ERR_UNSUPPORTED, "depthwise window above 5x5");
  DwArgs a = dw_args(d);
  a.x = static_cast<const char *>(x);
  a.w = static_cast<const char *>(w);
  a.bias = static_cast<const char *>(bias);
  a.residual = static_cast<const char *>(residual);
  a.y = static_cast<char *>(y);
  a.act = act;
  a.route = route ? *route : DeviceRoute{nullptr, 0.0, 0, 0, nullptr};
  if (om) {
    a.om_counts = om->counts;
    a.om_mask = om->mask;
    a.om_words = om->words;
  }
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
