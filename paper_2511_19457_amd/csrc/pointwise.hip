// Pointwise (1x1) convolution on the bandwidth path: the light, memory-bound
// operators of the sparsity x intensity quadrants (SparOA Section 2.2) --
// MobileNet's expand and project convs, low-intensity 1x1 convs and FCs
// over many rows -- where a compute tile that re-reads activations once per
// output-channel tile wastes HBM bytes.
//
// A work-group holds its whole slice of the weights (all C_out channels when
// they fit, else at most four equal slices) in LDS for the life of the
// kernel and walks 64R-pixel tiles of the output: each activation byte
// crosses HBM once per slice, each output byte once, and the weights stay
// on chip.  The contraction still runs on the matrix cores, transposed so
// the output layout suits NHWC: D[oc][pix] = sum_k W[oc][k] X[pix][k] with
// v_mfma_f32_16x16x32_{bf16,f16}; the A operand (16 output channels x 32 k)
// comes from LDS, the B operand (32 k x 16 pixels) straight from global
// memory -- lane (pixel p, group g) loads the 16 bytes of channels
// 8g..8g+7 of its pixel, so a wave's load is 16 pixel rows of 64 contiguous
// bytes -- and each lane ends with 4 consecutive output channels of one
// pixel; lanes g and g ^ 1 then swap halves so each finishes 8 consecutive
// channels of its pixel with 16-byte residual loads and stores.  K (= C_in)
// is at most 256: all of a tile's activation loads are issued before its
// first MFMA, and the next tile's while the current one computes.
//
// Zero skipping (Section 2.1): in the skip form an MFMA group whose B
// operand is zero in all 64 lanes -- a 16-pixel x 32-channel block of zero
// activations -- is not issued; it would add exact zeros, so the output
// equals the dense form's.  executed_blocks counts the (16-pixel block,
// 32-channel block) pairs that ran.
//
// Output measurement (Section 3.1, Eq. 1, taken on the layer's output): with
// one slice the epilogue also counts the zeros of y and builds its bitmap at
// block (1 pixel, 8 channels); a tile's bitmap words meet in LDS (tiles start
// on 32-bit word boundaries) and leave as whole-word stores.
#include "commit.h"
#include "common.h"
#include "dtype.h"

namespace sparoa {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kPwThreads = 256;          // 4 waves
constexpr int kPwMaxK = 256;             // C_in limit: all k-steps of a tile in flight
constexpr int kPwLdsBytes = 48 * 1024;   // weight slice bound (three work-groups per CU)
constexpr int kPwMaxSlices = 4;          // activations read at most 4 times
constexpr int kPwMaxWords = 256 * 32 / 32;   // bitmap words of a tile: 256 pixels x 32 blocks

struct PwArgs {
  const char *x, *w, *bias, *residual;
  char *y;
  unsigned long long *executed;
  int M, K, Cout, H, W, Ho, Wo, sh, sw;
  int ks;           // 32-wide k-steps
  int bn;           // output channels per slice (multiple of 16)
  int slices;
  int tiles;        // pixel tiles per slice
  int row_bytes;    // LDS bytes per weight row (K padded to 32, plus 16)
  int x_bytes;      // buffer range of x
  float inv_wo, inv_ho;
  int act, mode;    // mode: 0 dense, 1 skip, 2 device route
  DeviceRoute route;
  sparoa_counts *om_counts;  // non-null: measure y (one slice only)
  uint32_t *om_mask;
  unsigned long long *om_words;
  int64_t om_mask_words;
};

__device__ __forceinline__ void divmod_f(int n, int d, float inv_d, int &q, int &r) {
  const int q0 = (int)((float)n * inv_d);
  const int r0 = n - q0 * d;
  const bool lo = r0 < 0, hi = r0 >= d;   // one correction, as selects
  q = lo ? q0 - 1 : (hi ? q0 + 1 : q0);
  r = lo ? r0 + d : (hi ? r0 - d : r0);
}

template <int DT, int NB, int R, int KS>
__global__ __launch_bounds__(kPwThreads) void pointwise_kernel(PwArgs a) {
  using E = Elem<DT>;
  using raw = typename E::raw;
  constexpr int P = 64 * R;              // output pixels per tile
  extern __shared__ __attribute__((aligned(16))) char wl[];   // [NB * 16][row_bytes]
  __shared__ uint32_t ombits[kPwMaxWords];
  __shared__ unsigned long long exec_part[4];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, rl = lane & 15;
  const int slice = (int)(blockIdx.x % (unsigned)a.slices);
  const int wg_in_slice = (int)(blockIdx.x / (unsigned)a.slices);
  const int wgs_per_slice = (int)(gridDim.x / (unsigned)a.slices);
  const int c0 = slice * a.bn;

  SPAROA_ARGS_UP_FRONT("s"(a.x), "s"(a.w), "s"(a.y), "s"(a.M), "s"(a.K), "s"(a.Cout),
                       "s"(a.bn), "s"(a.slices), "s"(a.row_bytes), "s"(a.x_bytes), "s"(a.mode),
                       "s"(a.route.counts));
  // the device route's counts are requested now and decided on once the
  // weight slice is staged (nothing before needs the decision)
  const RouteCountsReq rq = route_counts_request(a.route);

  // ---- weight slice -> LDS, zero past C_out and past K (16-byte vectors;
  // K % 8 == 0, so a vector never straddles two rows).  Eight independent
  // loads per thread in flight per round (addresses clamped, values masked).
  const raw *w = reinterpret_cast<const raw *>(a.w);
  const int vpr = a.row_bytes / 16;     // vectors per LDS row (the last is padding)
  const int nv = NB * 16 * vpr;
  for (int v0 = tid; v0 < nv; v0 += kPwThreads * 8) {
    uint4 q[8];
    bool ok[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int v = v0 + kPwThreads * u;
      const int row = v / vpr, kv = v - row * vpr;
      const int oc = c0 + row, k = kv * 8;
      ok[u] = v < nv && oc < a.Cout && row < a.bn && k < a.K;
      q[u] = *reinterpret_cast<const uint4 *>(w + (ok[u] ? (int64_t)oc * a.K + k : 0));
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int v = v0 + kPwThreads * u;
      if (v < nv)
        *reinterpret_cast<uint4 *>(wl + (size_t)v * 16) =
            ok[u] ? q[u] : make_uint4(0u, 0u, 0u, 0u);
    }
  }
  __syncthreads();
  bool skip = a.mode == 1;
  if (a.mode == 2) {
    skip = route_counts_skip(rq, a.route);
    if (a.route.path_out && blockIdx.x == 0 && tid == 0)
      *a.route.path_out = (skip ? 1u : 0u) | ((uint32_t)a.route.bw_bit << 1);
  }

  const __amdgpu_buffer_rsrc_t xr =
      __builtin_amdgcn_make_buffer_rsrc((void *)a.x, (short)0, a.x_bytes, kBufDword3);
  const bool om = a.om_counts != nullptr;
  const int C8 = a.Cout / 8;
  uint32_t om_zeros = 0, om_nz = 0;
  unsigned long long executed = 0;
  const raw *bias = reinterpret_cast<const raw *>(a.bias);
  const raw *res = reinterpret_cast<const raw *>(a.residual);
  raw *y = reinterpret_cast<raw *>(a.y);
  const bool unit_stride = a.sh == 1 && a.sw == 1;

  // activations of one tile: every k-step of the R pixel blocks (lane:
  // pixel rl, channels 8g..8g+7 of each 32-wide k-step), straight loads
  auto load_tile = [&](int tile, u32x4 (&bx)[R][KS]) __attribute__((always_inline)) {
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int m = tile * P + (wave * R + r) * 16 + rl;
      int pixel = m;
      if (!unit_stride) {
        const int mm = m < a.M ? m : 0;
        int t1, ow, n, oh;
        divmod_f(mm, a.Wo, a.inv_wo, t1, ow);
        divmod_f(t1, a.Ho, a.inv_ho, n, oh);
        pixel = (n * a.H + oh * a.sh) * a.W + ow * a.sw;
      }
      const int off = (pixel * a.K + 8 * g) * 2;
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        const bool ok = m < a.M && 32 * s + 8 * g < a.K;
        bx[r][s] = __builtin_amdgcn_raw_buffer_load_b128(xr, ok ? off + 64 * s : (int)0x80000000,
                                                          0, 0);
      }
    }
  };

  // Finishes 8 consecutive output channels c0 + oc8 .. + 7 of pixel m (one
  // bitmap block): bias, residual, activation, one 16-byte store, and the
  // block's zero count and nonzero bit.
  auto finish8 = [&](int m, int p0, int oc8, const float (&v)[8]) __attribute__((always_inline)) {
    if (m >= a.M || oc8 >= a.bn || c0 + oc8 >= a.Cout) return;
    const int oc = c0 + oc8;
    float o[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] = v[e];
    raw t[8];
    if (bias) {
      const uint4 q = *reinterpret_cast<const uint4 *>(bias + oc);
      __builtin_memcpy(t, &q, 16);
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] += E::to_f32(t[e]);
    }
    if (res) {
      const uint4 q = *reinterpret_cast<const uint4 *>(res + (int64_t)m * a.Cout + oc);
      __builtin_memcpy(t, &q, 16);
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] += E::to_f32(t[e]);
    }
    uint32_t nz = 0;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      t[e] = E::from_f32(apply_act(o[e], a.act));
      const bool z = (t[e] & 0x7FFFu) == 0u;
      om_zeros += (om && z) ? 1u : 0u;
      nz |= z ? 0u : 1u;
    }
    uint4 q;
    __builtin_memcpy(&q, t, 16);
    *reinterpret_cast<uint4 *>(y + (int64_t)m * a.Cout + oc) = q;
    if (om && nz) {
      const int bit = (m - p0) * C8 + oc / 8;
      atomicOr(&ombits[bit >> 5], 1u << (bit & 31));
      om_nz += 1;
    }
  };

  u32x4 cur[R][KS], nxt[R][KS];
  int tile = wg_in_slice;
  if (tile < a.tiles) load_tile(tile, cur);
  for (; tile < a.tiles; tile += wgs_per_slice) {
    const int p0 = tile * P;
    const int next = tile + wgs_per_slice;
    if (next < a.tiles) load_tile(next, nxt);   // the next tile's loads fly during this one
    f32x4 acc[R][NB];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int j = 0; j < NB; ++j) acc[r][j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      bool run[R];
#pragma unroll
      for (int r = 0; r < R; ++r) {
        run[r] = true;
        if (skip) {
          const u32x4 v = cur[r][s];
          run[r] = __ballot((v[0] | v[1] | v[2] | v[3]) != 0u) != 0ull;
          executed += run[r] && slice == 0 ? 1u : 0u;   // each pair once, not once per slice
        }
      }
#pragma unroll
      for (int j = 0; j < NB; ++j) {
        const u32x4 av = *reinterpret_cast<const u32x4 *>(wl + (size_t)(j * 16 + rl) * a.row_bytes +
                                                          64 * s + 16 * g);
#pragma unroll
        for (int r = 0; r < R; ++r) {
          if (!run[r]) continue;
          if constexpr (DT == SPAROA_BF16)
            acc[r][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(bf16x8, av), __builtin_bit_cast(bf16x8, cur[r][s]), acc[r][j],
                0, 0, 0);
          else
            acc[r][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(
                __builtin_bit_cast(f16x8, av), __builtin_bit_cast(f16x8, cur[r][s]), acc[r][j],
                0, 0, 0);
        }
      }
      // keep each k-step's weight reads next to its MFMAs (hoisting every
      // step's reads ahead held KS * NB fragments in registers)
      __builtin_amdgcn_sched_barrier(0);
    }

    // ---- epilogue.  Lane (pixel rl, group g) holds channels 16 j + 4 g .. + 3
    // of block j.  For a block pair (j, j + 1) lanes g and g ^ 1 swap halves so
    // each lane holds 8 consecutive channels of its pixel: even g channels
    // 32 jp + 8 (g / 2) .., odd g channels 32 jp + 16 + 8 (g / 2) ..
    if (om) {
      for (int i = tid; i < P * C8 / 32; i += kPwThreads) ombits[i] = 0u;
      __syncthreads();
    }
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int m = p0 + (wave * R + r) * 16 + rl;
#pragma unroll
      for (int jp = 0; jp + 1 < NB; jp += 2) {
        const bool odd = (g & 1) != 0;
        float v[8];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float send = odd ? acc[r][jp][e] : acc[r][jp + 1][e];
          const float recv = __shfl_xor(send, 16, 64);
          v[e] = odd ? recv : acc[r][jp][e];
          v[4 + e] = odd ? acc[r][jp + 1][e] : recv;
        }
        finish8(m, p0, 16 * jp + (odd ? 16 : 0) + 8 * (g >> 1), v);
      }
      if constexpr (NB % 2 == 1) {
        // the last block alone: lanes g and g ^ 1 hold channels 8 (g / 2) ..;
        // the even lane takes the odd lane's four
        constexpr int j = NB - 1;
        float v[8];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float recv = __shfl_xor(acc[r][j][e], 16, 64);
          v[e] = acc[r][j][e];
          v[4 + e] = recv;
        }
        if ((g & 1) == 0) finish8(m, p0, 16 * j + 8 * (g >> 1), v);
      }
    }
    if (om) {
      __syncthreads();
      const int64_t w0 = (int64_t)p0 * C8 / 32;
      for (int i = tid; i < P * C8 / 32; i += kPwThreads)
        if (w0 + i < a.om_mask_words) a.om_mask[w0 + i] = ombits[i];
      __syncthreads();
    }
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int s = 0; s < KS; ++s) cur[r][s] = nxt[r][s];
  }

  if (a.executed && skip) {
    if (lane == 0) exec_part[wave] = executed;
    __syncthreads();
    if (tid == 0) {
      const unsigned long long tot = exec_part[0] + exec_part[1] + exec_part[2] + exec_part[3];
      if (tot) atomicAdd(a.executed, tot);
    }
  }
  if (om) om_commit(om_zeros, om_nz, a.om_counts, a.om_words, blockIdx.x, gridDim.x);
}

struct PwChoice {
  int nb, r, bn, slices, ks, ksi, row_bytes;
};

bool pw_choose(const sparoa_conv_desc &d, PwChoice *c) {
  if (d.dtype == SPAROA_F32 || d.groups != 1 || d.kh != 1 || d.kw != 1 || d.ph || d.pw)
    return false;
  if (d.c_in % 8 || d.c_out % 8 || d.c_in > kPwMaxK) return false;
  // measured on ResNet-50 / MobileNetV2 shapes (N = 32): with K >= 192 and
  // at least 64 output channels the 64-channel-chunk implicit GEMM is faster
  // (256 -> 64 at 56 x 56: 28 vs 34 us; 192 -> 64 at 14 x 14: 11.5 vs 14 us)
  if (d.c_in >= 192 && d.c_in % 64 == 0 && d.c_out >= 64) return false;
  const int64_t ho = (d.h - 1) / d.sh + 1, wo = (d.w - 1) / d.sw + 1;
  const int64_t M = d.n * ho * wo;
  if (M >= ((int64_t)1 << 24) || d.n * d.h * d.w * d.c_in * 2 >= ((int64_t)1 << 31)) return false;
  // below 32768 pixels the layer is latency-bound and the implicit GEMM's
  // tiles finish sooner wherever it takes the channel count and there are
  // 64 output channels or more (ResNet-50 stage 1 at N = 1, 64 -> 256: 4.8
  // vs 8.8 us; N = 8, 64 -> 64: 5.7 vs 7.6 us); from 100352 pixels the
  // pointwise kernel wins (N = 32, 64 -> 256: 26 vs 36 us)
  if (M < 32768 && d.c_out >= 64 && (d.c_in % 64 == 0 || d.c_in >= 48)) return false;
  const int ks = (int)cdiv(d.c_in, 32);
  // instantiated k-step counts; LDS rows hold all of them (zero past K)
  const int ksi = ks <= 2 ? ks : (ks <= 4 ? 4 : 8);
  const int row_bytes = ksi * 64 + 16;
  const int64_t nb_all = cdiv(d.c_out, 16);
  // fewest slices whose 16-channel blocks, rounded up to an instantiated
  // count, fit the LDS bound
  static const int kNb[] = {1, 2, 4, 6, 8, 12, 16};
  int64_t slices = 1;
  int nb = 0, nbi = 0;
  for (; slices <= kPwMaxSlices; ++slices) {
    nb = (int)cdiv(nb_all, slices);
    nbi = 0;
    for (int v : kNb)
      if (v >= nb) { nbi = v; break; }
    if (nbi && (int64_t)nbi * 16 * row_bytes <= kPwLdsBytes) break;
  }
  if (slices > kPwMaxSlices) return false;
  // several slices re-read x once per slice: only where the tiles of one
  // slice alone fill the chip (else the implicit GEMM does better)
  if (slices > 1 && cdiv(M, 128) < 256) return false;
  // activation registers (current and next tile) R * KS * 8 VGPRs <= 64,
  // accumulators R * NB * 4 <= 64
  if (ksi == 8 && nbi < 12 && nbi > 4) return false;   // (not instantiated)
  int r = 4;
  while (r > 1 && (r * ksi > 8 || r * nbi > 16)) r /= 2;
  if (r * ksi > 8 || r * nbi > 16) return false;
  c->nb = nbi;
  c->r = r;
  c->ksi = ksi;
  c->bn = nb * 16;
  c->slices = (int)slices;
  c->ks = ks;
  c->row_bytes = row_bytes;
  return true;
}

template <int DT, int NB, int R, int KS>
const void *pw_fn() {
  return reinterpret_cast<const void *>(&pointwise_kernel<DT, NB, R, KS>);
}

// The (NB, KS) pairs pw_choose can select, R fixed by them.
template <int DT, int NB>
const void *pw_kernel_nb(int r, int ks) {
  constexpr int R1 = NB <= 4 ? 4 : (NB <= 8 ? 2 : 1);      // KS = 1, 2
  constexpr int R4 = NB <= 8 ? 2 : 1;                      // KS = 4
  if (ks == 1 && r == R1) return pw_fn<DT, NB, R1, 1>();
  if (ks == 2 && r == R1) return pw_fn<DT, NB, R1, 2>();
  if (ks == 4 && r == R4) return pw_fn<DT, NB, R4, 4>();
  if constexpr (NB <= 4 || NB >= 12)
    if (ks == 8 && r == 1) return pw_fn<DT, NB, 1, 8>();
  return nullptr;
}

template <int DT>
const void *pw_kernel(int nb, int r, int ks) {
  switch (nb) {
    case 1: return pw_kernel_nb<DT, 1>(r, ks);
    case 2: return pw_kernel_nb<DT, 2>(r, ks);
    case 4: return pw_kernel_nb<DT, 4>(r, ks);
    case 6: return pw_kernel_nb<DT, 6>(r, ks);
    case 8: return pw_kernel_nb<DT, 8>(r, ks);
    case 12: return pw_kernel_nb<DT, 12>(r, ks);
    case 16: return pw_kernel_nb<DT, 16>(r, ks);
  }
  return nullptr;
}

// Work-groups of `fn` that fit on the current device at once (occupancy
// query, cached per device, kernel and LDS size).
}  // namespace

bool pw_eligible(const sparoa_conv_desc &d) {
  PwChoice c;
  return pw_choose(d, &c);
}

bool pw_fuses_out_measure(const sparoa_conv_desc &d) {
  PwChoice c;
  return pw_choose(d, &c) && c.slices == 1 && 64 * c.r * (d.c_out / 8) / 32 <= kPwMaxWords;
}

sparoa_status launch_pointwise(const sparoa_conv_desc &d, const void *x, const void *w,
                               const void *bias, const void *residual, sparoa_act act, void *y,
                               bool skip, uint64_t *executed, hipStream_t stream,
                               const DeviceRoute *route, const OutMeasure *om) {
  PwChoice c;
  if (!pw_choose(d, &c)) return fail(SPAROA_ERR_UNSUPPORTED, "pointwise: shape not eligible");
  if (om && !pw_fuses_out_measure(d))
    return fail(SPAROA_ERR_UNSUPPORTED, "pointwise: no fused output measurement for this shape");
  PwArgs a;
  const int64_t ho = (d.h - 1) / d.sh + 1, wo = (d.w - 1) / d.sw + 1;
  a.x = static_cast<const char *>(x);
  a.w = static_cast<const char *>(w);
  a.bias = static_cast<const char *>(bias);
  a.residual = static_cast<const char *>(residual);
  a.y = static_cast<char *>(y);
  a.executed = reinterpret_cast<unsigned long long *>(skip ? executed : nullptr);
  a.M = (int)(d.n * ho * wo);
  a.K = (int)d.c_in;
  a.Cout = (int)d.c_out;
  a.H = (int)d.h; a.W = (int)d.w; a.Ho = (int)ho; a.Wo = (int)wo;
  a.sh = (int)d.sh; a.sw = (int)d.sw;
  a.ks = c.ks;
  a.bn = c.bn;
  a.slices = c.slices;
  const int P = 64 * c.r;
  a.tiles = (int)cdiv(a.M, P);
  a.row_bytes = c.row_bytes;
  a.x_bytes = (int)(d.n * d.h * d.w * d.c_in * 2);
  a.inv_wo = 1.0f / (float)wo;
  a.inv_ho = 1.0f / (float)ho;
  a.act = act;
  a.mode = route && route->counts ? 2 : (skip ? 1 : 0);
  a.route = route ? *route : DeviceRoute{nullptr, 0.0, 0, 0, nullptr};
  a.om_counts = om ? om->counts : nullptr;
  a.om_mask = om ? om->mask : nullptr;
  a.om_words = om ? om->words : nullptr;
  a.om_mask_words = a.om_mask ? (a.M * (int64_t)(d.c_out / 8) + 31) / 32 : 0;   // null: counts only
  const unsigned lds = (unsigned)(c.nb * 16 * c.row_bytes);
  const void *fn = d.dtype == SPAROA_BF16 ? pw_kernel<SPAROA_BF16>(c.nb, c.r, c.ksi)
                                          : pw_kernel<SPAROA_F16>(c.nb, c.r, c.ksi);
  if (!fn) return fail(SPAROA_ERR_UNSUPPORTED, "pointwise: tile configuration");
  // persistent work-groups, as many as are resident at once, each bound to
  // one slice: every work-group stages its weights once for many tiles
  int resident = 0;
  if (sparoa_status st = resident_blocks(fn, kPwThreads, lds, &resident); st != SPAROA_OK)
    return st;
  int64_t per_slice = resident / c.slices;
  if (per_slice < 1) per_slice = 1;
  if (per_slice > a.tiles) per_slice = a.tiles;
  const dim3 grid((unsigned)(per_slice * c.slices));
  // (executed_blocks was zeroed by the caller, launch_gemm_conv)
  void *args[] = {&a};
  SPAROA_HIP_CHECK(hipLaunchKernel(fn, grid, dim3(kPwThreads), args, lds, stream));
  return SPAROA_OK;
}

}  // namespace sparoa
