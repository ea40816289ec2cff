// Implicit-GEMM convolution on the gfx950 matrix cores (MFMA), dense and
// zero-skipping.  Fully connected layers run through the same kernel as a
// 1x1 convolution over m "pixels".
//
// GEMM view of conv (NHWC activations, [c_out][kh][kw][c_in] weights):
//   rows  m = (n, oh, ow)                      M = n * ho * wo
//   cols  j = output channel                   N = c_out
//   depth k = (r, s, c) = (r*kw + s)*c_in + c  K = kh * kw * c_in
//   A[m][k] = x[n][oh*sh - ph + r*dh][ow*sw - pw + s*dw][c]  (0 outside)
//   B[j][k] = w[j][r][s][c]                     (row j of w, contiguous in k)
//
// Work-group = 256 threads = 4 waves in a 2 x 2 layout; the tile is
// BM x BN with BM = 32*TM, BN = 32*TN, each wave owning (BM/2) x (BN/2) as
// TM x TN MFMA 16x16 blocks.  The K loop walks chunks of 32 k values; A and B
// chunks are staged global -> registers -> LDS (double buffered, one barrier
// per chunk) and fed to v_mfma_f32_16x16x32_{bf16,f16} (one per block per
// chunk) or v_mfma_f32_16x16x4_f32 (eight per block per chunk).
//
// Zero skipping (SparOA Section 2.1: zero activations can be skipped without
// changing the output): the skip variant reads the activation bitmap written
// by the measurement kernel at one bit per (pixel, 8 channels).  At start-up
// each work-group ORs, for every pixel its tile gathers at every tap, those
// bits into an LDS bit vector over K/8 (the nonzero 8-wide K slices of its
// tile), turns it into one flag per 32-wide chunk, and compacts the nonzero
// chunk indices into an LDS list (ballot + popcount prefix).  The main loop
// then walks only that list: skipped chunks cost neither global/LDS traffic
// nor MFMA issue.  Because the chunk order and the MFMA block decomposition
// are those of the dense variant, and a skipped chunk would only have added
// exact zeros, the skip output equals the dense output bit for bit (for
// finite weights).
#include "common.h"
#include "dtype.h"

namespace sparoa {
namespace {

constexpr int kThreads = 256;
constexpr int kBK = 32;            // K values per chunk (skip granularity)
constexpr int kMaxChunks = 2048;   // K <= 65536 on the skip path
constexpr int kMaxVecWords = kMaxChunks * kBK / 8 / 32;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

struct GemmArgs {
  const char *x;
  const char *w;
  const char *bias;
  const char *residual;
  char *y;
  float *partial;
  const uint32_t *mask;
  unsigned long long *executed;
  int64_t M, N, K;
  int64_t H, W, Cin, Ho, Wo, Kw, sh, sw, ph, pw, dh, dw, taps;
  int64_t nchunks, chunks_per_split;
  int act;
  int split;
  DeviceRoute route;
};

template <int DT>
__device__ __forceinline__ f32x4 mfma_chunk(const char *a_row, const char *b_row, f32x4 acc,
                                            int g) {
  if constexpr (DT == SPAROA_BF16) {
    const bf16x8 a = *reinterpret_cast<const bf16x8 *>(a_row + 16 * g);
    const bf16x8 b = *reinterpret_cast<const bf16x8 *>(b_row + 16 * g);
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc, 0, 0, 0);
  } else if constexpr (DT == SPAROA_F16) {
    const f16x8 a = *reinterpret_cast<const f16x8 *>(a_row + 16 * g);
    const f16x8 b = *reinterpret_cast<const f16x8 *>(b_row + 16 * g);
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, acc, 0, 0, 0);
  } else {
    // Lane group g holds k = 16h + 4g + e of both operands; the four MFMAs
    // over e cover the 16 k values of half h.
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const f32x4 a = *reinterpret_cast<const f32x4 *>(a_row + 64 * h + 16 * g);
      const f32x4 b = *reinterpret_cast<const f32x4 *>(b_row + 64 * h + 16 * g);
#pragma unroll
      for (int e = 0; e < 4; ++e) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[e], b[e], acc, 0, 0, 0);
    }
    return acc;
  }
}

// Reads n <= 32 bits starting at bit `pos` of a bitmap.
__device__ __forceinline__ uint32_t read_bits(const uint32_t *m, int64_t pos, int n) {
  const int64_t wd = pos >> 5;
  const int off = (int)(pos & 31);
  uint32_t v = m[wd] >> off;
  if (off + n > 32) v |= m[wd + 1] << (32 - off);
  return n == 32 ? v : (v & ((1u << n) - 1u));
}

// ORs n <= 32 bits into an LDS bitmap at bit `pos`.
__device__ __forceinline__ void lds_or_bits(uint32_t *m, int pos, uint32_t v, int n) {
  if (!v) return;
  const int wd = pos >> 5, off = pos & 31;
  atomicOr(m + wd, v << off);
  if (off && off + n > 32) atomicOr(m + wd + 1, v >> (32 - off));
}

template <int DT, int TM, int TN, bool VEC, bool SKIP>
__global__ __launch_bounds__(kThreads) void gemm_kernel(GemmArgs a) {
  using E = Elem<DT>;
  constexpr int ESZ = E::size;
  constexpr int BM = 32 * TM, BN = 32 * TN;
  constexpr int ROWB = kBK * ESZ + 16;   // LDS row stride (padding: conflict-free reads)
  constexpr int VPR = kBK * ESZ / 16;    // 16-byte vectors per chunk row
  constexpr int EPV = 16 / ESZ;          // elements per vector
  constexpr int AV = BM * VPR / kThreads;  // A vectors per thread
  constexpr int BV = BN * VPR / kThreads;  // B vectors per thread
  static_assert(AV >= 1 && BV >= 1, "tile too small for the work-group");

  __shared__ __attribute__((aligned(16))) char smem[2][(BM + BN) * ROWB];
  __shared__ int list[SKIP ? kMaxChunks : 1];
  __shared__ uint32_t nzvec[SKIP ? kMaxVecWords : 1];
  __shared__ int list_len;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int64_t m0 = (int64_t)blockIdx.x * BM, n0 = (int64_t)blockIdx.y * BN;
  const int64_t c_begin = (int64_t)blockIdx.z * a.chunks_per_split;
  const int64_t c_end = min(c_begin + a.chunks_per_split, a.nchunks);

  // ---- per-thread A rows (fixed over the K loop) --------------------------
  // A vector q = tid + kThreads*u covers row q / VPR, vector column q % VPR.
  int64_t a_pix[AV];  // n * H * W, or -1 when the row is past M
  int a_h0[AV], a_w0[AV];
  const uint32_t cin = (uint32_t)a.Cin, kw = (uint32_t)a.Kw, kdim = (uint32_t)a.K;
  const int H = (int)a.H, W = (int)a.W, dh = (int)a.dh, dw = (int)a.dw;
#pragma unroll
  for (int u = 0; u < AV; ++u) {
    const int q = tid + kThreads * u;
    const int64_t m = m0 + q / VPR;
    if (m < a.M) {
      const int64_t ow = m % a.Wo, oh = (m / a.Wo) % a.Ho, nn = m / (a.Wo * a.Ho);
      a_pix[u] = nn * a.H * a.W;
      a_h0[u] = (int)(oh * a.sh - a.ph);
      a_w0[u] = (int)(ow * a.sw - a.pw);
    } else {
      a_pix[u] = -1;
      a_h0[u] = a_w0[u] = 0;
    }
  }

  // ---- chunk list (skip variant) -------------------------------------------
  int64_t count = c_end - c_begin;
  bool use_list = SKIP;
  if constexpr (SKIP) {
    if (a.route.counts) {
      use_list = device_route_skip(a.route);
      if (a.route.path_out && blockIdx.x == 0 && blockIdx.y == 0 && blockIdx.z == 0 && tid == 0)
        *a.route.path_out = (use_list ? 1u : 0u) | ((uint32_t)a.route.bw_bit << 1);
    }
  }
  if constexpr (!SKIP) {
    if (a.route.path_out && blockIdx.x == 0 && blockIdx.y == 0 && blockIdx.z == 0 && tid == 0)
      *a.route.path_out = (uint32_t)a.route.bw_bit << 1;
  }
  if (SKIP && use_list) {
    const int cpg = (int)((a.Cin + 7) / 8);  // bitmap blocks per pixel
    const int kv_words = (int)((a.taps * cpg + 31) / 32);
    for (int i = tid; i < kv_words; i += kThreads) nzvec[i] = 0u;
    __syncthreads();
    for (int64_t p = tid; p < (int64_t)BM * a.taps; p += kThreads) {
      const int r_in = (int)(p / a.taps);
      const int tap = (int)(p - (int64_t)r_in * a.taps);
      const int64_t m = m0 + r_in;
      if (m >= a.M) continue;
      const int64_t ow = m % a.Wo, oh = (m / a.Wo) % a.Ho, nn = m / (a.Wo * a.Ho);
      const int64_t r = tap / a.Kw, s = tap - r * a.Kw;
      const int64_t ih = oh * a.sh - a.ph + r * a.dh, iw = ow * a.sw - a.pw + s * a.dw;
      if (ih < 0 || ih >= a.H || iw < 0 || iw >= a.W) continue;
      const int64_t pix = (nn * a.H + ih) * a.W + iw;
      for (int b = 0; b < cpg; b += 32) {
        const int nb = min(32, cpg - b);
        lds_or_bits(nzvec, tap * cpg + b, read_bits(a.mask, pix * cpg + b, nb), nb);
      }
    }
    __syncthreads();
    if (wave == 0) {
      int total = 0;
      for (int64_t base = c_begin; base < c_end; base += 64) {
        const int64_t j = base + lane;
        bool nz = false;
        if (j < c_end) {
          // walk the chunk's k range one (tap, 8-channel block) run at a time
          uint32_t k = (uint32_t)(j * kBK);
          const uint32_t kend = (uint32_t)min(j * kBK + kBK, a.K);
          while (k < kend) {
            const uint32_t tap = k / cin, c = k - tap * cin;
            const uint32_t bit = tap * (uint32_t)cpg + c / 8;
            nz |= (nzvec[bit >> 5] >> (bit & 31)) & 1u;
            const uint32_t cnext = (c / 8 + 1) * 8;
            k = tap * cin + (cnext < cin ? cnext : cin);
          }
        }
        const uint64_t bal = __ballot(nz);
        const int before = __popcll(bal & ((1ull << lane) - 1ull));
        if (nz) list[total + before] = (int)j;
        total += __popcll(bal);
      }
      if (lane == 0) {
        list_len = total;
        if (a.executed && blockIdx.y == 0 && total)
          atomicAdd(a.executed, (unsigned long long)total);
      }
    }
    __syncthreads();
    count = list_len;
  }

  // ---- global -> register staging of one chunk -----------------------------
  uint4 ra[AV], rb[BV];
  auto load_chunk = [&](int64_t j) {
    const int64_t kbase = j * kBK;
#pragma unroll
    for (int u = 0; u < AV; ++u) {
      const int q = tid + kThreads * u;
      uint4 v = make_uint4(0, 0, 0, 0);
      if constexpr (VEC) {
        const uint32_t k = (uint32_t)kbase + (uint32_t)(q % VPR) * EPV;
        if (a_pix[u] >= 0 && k < kdim) {
          const uint32_t tap = k / cin, c = k - tap * cin;
          const uint32_t r = tap / kw, s = tap - r * kw;
          const int ih = a_h0[u] + (int)r * dh, iw = a_w0[u] + (int)s * dw;
          if (ih >= 0 && ih < H && iw >= 0 && iw < W)
            v = *reinterpret_cast<const uint4 *>(
                a.x + ((a_pix[u] + (int64_t)ih * W + iw) * a.Cin + c) * ESZ);
        }
      } else {
        typename E::raw e[EPV];
#pragma unroll
        for (int t = 0; t < EPV; ++t) {
          e[t] = 0;
          const uint32_t k = (uint32_t)kbase + (uint32_t)(q % VPR) * EPV + t;
          if (a_pix[u] >= 0 && k < kdim) {
            const uint32_t tap = k / cin, c = k - tap * cin;
            const uint32_t r = tap / kw, s = tap - r * kw;
            const int ih = a_h0[u] + (int)r * dh, iw = a_w0[u] + (int)s * dw;
            if (ih >= 0 && ih < H && iw >= 0 && iw < W)
              e[t] = reinterpret_cast<const typename E::raw *>(
                  a.x)[(a_pix[u] + (int64_t)ih * W + iw) * a.Cin + c];
          }
        }
        __builtin_memcpy(&v, e, 16);
      }
      ra[u] = v;
    }
#pragma unroll
    for (int u = 0; u < BV; ++u) {
      const int q = tid + kThreads * u;
      const int64_t jn = n0 + q / VPR;
      const int64_t k = kbase + (q % VPR) * EPV;
      uint4 v = make_uint4(0, 0, 0, 0);
      if constexpr (VEC) {
        if (jn < a.N && k < a.K) v = *reinterpret_cast<const uint4 *>(a.w + (jn * a.K + k) * ESZ);
      } else {
        typename E::raw e[EPV];
#pragma unroll
        for (int t = 0; t < EPV; ++t)
          e[t] = (jn < a.N && k + t < a.K)
                     ? reinterpret_cast<const typename E::raw *>(a.w)[jn * a.K + k + t]
                     : (typename E::raw)0;
        __builtin_memcpy(&v, e, 16);
      }
      rb[u] = v;
    }
  };
  auto store_chunk = [&](int buf) {
#pragma unroll
    for (int u = 0; u < AV; ++u) {
      const int q = tid + kThreads * u;
      *reinterpret_cast<uint4 *>(&smem[buf][(q / VPR) * ROWB + (q % VPR) * 16]) = ra[u];
    }
#pragma unroll
    for (int u = 0; u < BV; ++u) {
      const int q = tid + kThreads * u;
      *reinterpret_cast<uint4 *>(&smem[buf][(BM + q / VPR) * ROWB + (q % VPR) * 16]) = rb[u];
    }
  };

  f32x4 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto chunk_at = [&](int64_t i) -> int64_t {
    return (SKIP && use_list) ? (int64_t)list[i] : c_begin + i;
  };

  const int g = lane >> 4, rl = lane & 15;
  if (count > 0) {
    load_chunk(chunk_at(0));
    store_chunk(0);
    __syncthreads();
    for (int64_t i = 0; i < count; ++i) {
      const int buf = (int)(i & 1);
      const bool more = i + 1 < count;
      if (more) load_chunk(chunk_at(i + 1));
      const char *As = &smem[buf][0];
      const char *Bs = &smem[buf][BM * ROWB];
#pragma unroll
      for (int tm = 0; tm < TM; ++tm) {
        const char *arow = As + (wm * (BM / 2) + tm * 16 + rl) * ROWB;
#pragma unroll
        for (int tn = 0; tn < TN; ++tn) {
          const char *brow = Bs + (wn * (BN / 2) + tn * 16 + rl) * ROWB;
          acc[tm][tn] = mfma_chunk<DT>(arow, brow, acc[tm][tn], g);
        }
      }
      if (more) store_chunk(buf ^ 1);
      __syncthreads();
    }
  }

  // ---- epilogue ------------------------------------------------------------
  // MFMA 16x16 output layout: lane holds rows 4*(lane/16) + v, column lane%16.
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int tn = 0; tn < TN; ++tn)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int64_t row = m0 + wm * (BM / 2) + tm * 16 + 4 * g + v;
        const int64_t col = n0 + wn * (BN / 2) + tn * 16 + rl;
        if (row >= a.M || col >= a.N) continue;
        const float val = acc[tm][tn][v];
        if (a.split > 1) {
          a.partial[((int64_t)blockIdx.z * a.M + row) * a.N + col] = val;
        } else {
          float o = val;
          if (a.bias) o += E::to_f32(reinterpret_cast<const typename E::raw *>(a.bias)[col]);
          if (a.residual)
            o += E::to_f32(reinterpret_cast<const typename E::raw *>(a.residual)[row * a.N + col]);
          reinterpret_cast<typename E::raw *>(a.y)[row * a.N + col] = E::from_f32(apply_act(o, a.act));
        }
      }
}

// Sums the K-split partials in split order, adds bias and residual, then
// applies the activation.
template <int DT>
__global__ __launch_bounds__(256) void split_reduce(const float *__restrict__ partial, int split,
                                                    int64_t M, int64_t N, const char *bias,
                                                    const char *residual, int act, char *y) {
  using E = Elem<DT>;
  const int64_t total = M * N;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    float o = 0.f;
    for (int z = 0; z < split; ++z) o += partial[z * total + i];
    const int64_t col = i % N;
    if (bias) o += E::to_f32(reinterpret_cast<const typename E::raw *>(bias)[col]);
    if (residual) o += E::to_f32(reinterpret_cast<const typename E::raw *>(residual)[i]);
    reinterpret_cast<typename E::raw *>(y)[i] = E::from_f32(apply_act(o, act));
  }
}

__global__ void set_u64(unsigned long long *p, unsigned long long v) { *p = v; }

template <int DT, int TM, int TN, bool VEC, bool SKIP>
void launch_tile(dim3 grid, hipStream_t st, const GemmArgs &a) {
  hipLaunchKernelGGL((gemm_kernel<DT, TM, TN, VEC, SKIP>), grid, dim3(kThreads), 0, st, a);
}

template <int DT, bool VEC, bool SKIP>
bool dispatch_tile(int bm, int bn, dim3 grid, hipStream_t st, const GemmArgs &a) {
  if constexpr (DT == SPAROA_F32) {  // fp32 tiles: 64 x 64 (LDS budget)
    if (bm != 64 || bn != 64) return false;
    launch_tile<DT, 2, 2, VEC, SKIP>(grid, st, a);
    return true;
  }
  if (bm == 128 && bn == 128) launch_tile<DT, 4, 4, VEC, SKIP>(grid, st, a);
  else if (bm == 128 && bn == 64) launch_tile<DT, 4, 2, VEC, SKIP>(grid, st, a);
  else if (bm == 64 && bn == 128) launch_tile<DT, 2, 4, VEC, SKIP>(grid, st, a);
  else if (bm == 64 && bn == 64) launch_tile<DT, 2, 2, VEC, SKIP>(grid, st, a);
  else return false;
  return true;
}

template <int DT>
bool dispatch(int bm, int bn, bool vec, bool skip, dim3 grid, hipStream_t st, const GemmArgs &a) {
  if (vec)
    return skip ? dispatch_tile<DT, true, true>(bm, bn, grid, st, a)
                : dispatch_tile<DT, true, false>(bm, bn, grid, st, a);
  return skip ? dispatch_tile<DT, false, true>(bm, bn, grid, st, a)
              : dispatch_tile<DT, false, false>(bm, bn, grid, st, a);
}

struct Shape {
  int64_t M, N, K, ho, wo;
};

Shape shape_of(const sparoa_conv_desc &d) {
  Shape s;
  s.ho = (d.h + 2 * d.ph - d.dh * (d.kh - 1) - 1) / d.sh + 1;
  s.wo = (d.w + 2 * d.pw - d.dw * (d.kw - 1) - 1) / d.sw + 1;
  s.M = d.n * s.ho * s.wo;
  s.N = d.c_out;
  s.K = d.kh * d.kw * d.c_in;
  return s;
}

}  // namespace

sparoa_status launch_set_u64(uint64_t *p, uint64_t v, hipStream_t stream) {
  hipLaunchKernelGGL(set_u64, dim3(1), dim3(1), 0, stream, reinterpret_cast<unsigned long long *>(p),
                     (unsigned long long)v);
  SPAROA_LAUNCH_CHECK("set_u64");
  return SPAROA_OK;
}

sparoa_status launch_split_reduce(sparoa_dtype dt, const float *partial, int split, int64_t M,
                                  int64_t N, const void *bias, const void *residual,
                                  sparoa_act act, void *y, hipStream_t stream) {
  const int64_t total = M * N;
  int64_t blocks = cdiv(total, 256);
  if (blocks > 4096) blocks = 4096;
  const char *b = static_cast<const char *>(bias);
  const char *r = static_cast<const char *>(residual);
  char *o = static_cast<char *>(y);
  switch (dt) {
    case SPAROA_BF16:
      hipLaunchKernelGGL(split_reduce<SPAROA_BF16>, dim3((unsigned)blocks), dim3(256), 0, stream,
                         partial, split, M, N, b, r, (int)act, o);
      break;
    case SPAROA_F16:
      hipLaunchKernelGGL(split_reduce<SPAROA_F16>, dim3((unsigned)blocks), dim3(256), 0, stream,
                         partial, split, M, N, b, r, (int)act, o);
      break;
    case SPAROA_F32:
      hipLaunchKernelGGL(split_reduce<SPAROA_F32>, dim3((unsigned)blocks), dim3(256), 0, stream,
                         partial, split, M, N, b, r, (int)act, o);
      break;
  }
  SPAROA_LAUNCH_CHECK("split_reduce");
  return SPAROA_OK;
}

bool gemm_skip_supported(const sparoa_conv_desc &d) {
  const Shape s = shape_of(d);
  const int64_t bits = d.kh * d.kw * cdiv(d.c_in, 8);
  return cdiv(s.K, kBK) <= kMaxChunks && bits <= (int64_t)kMaxVecWords * 32;
}

GemmTileChoice gemm_choose(const sparoa_conv_desc &d, sparoa_path) {
  const Shape s = shape_of(d);
  GemmTileChoice t;
  t.kchunk = kBK;
  if (d.dtype == SPAROA_F32) {
    t.bm = 64;
    t.bn = 64;
  } else {
    t.bn = s.N <= 64 ? 64 : 128;
    t.bm = 128;
    if (cdiv(s.M, t.bm) * cdiv(s.N, t.bn) < 256) t.bm = 64;
    if (cdiv(s.M, t.bm) * cdiv(s.N, t.bn) < 256) t.bn = 64;
  }
  const int64_t tiles = cdiv(s.M, t.bm) * cdiv(s.N, t.bn);
  const int64_t nchunks = cdiv(s.K, kBK);
  int64_t split = 1;
  if (tiles < 192) {
    split = cdiv(512, tiles);
    if (split > 8) split = 8;
    if (split > nchunks / 8) split = nchunks / 8;
    if (split < 1) split = 1;
  }
  t.split_k = (int)split;
  return t;
}

size_t gemm_workspace(const sparoa_conv_desc &d, sparoa_path path) {
  const GemmTileChoice t = gemm_choose(d, path);
  if (t.split_k <= 1) return 0;
  const Shape s = shape_of(d);
  return (size_t)t.split_k * (size_t)s.M * (size_t)s.N * sizeof(float);
}

sparoa_status launch_gemm_conv(const sparoa_conv_desc &d, sparoa_path path, const void *x,
                               const void *w, const void *bias, const void *residual,
                               sparoa_act act, const uint32_t *mask, void *y, void *ws,
                               size_t ws_bytes, uint64_t *executed, hipStream_t stream,
                               const DeviceRoute *route) {
  const Shape s = shape_of(d);
  const GemmTileChoice t = gemm_choose(d, path);
  const int epv = d.dtype == SPAROA_F32 ? 4 : 8;
  const bool vec = d.c_in % epv == 0;
  const bool skip = mask != nullptr;
  const int64_t nchunks = cdiv(s.K, kBK);
  if (skip && !gemm_skip_supported(d))
    return fail(SPAROA_ERR_UNSUPPORTED, "zero-skip conv: K above the skip kernel's 65536");
  if (s.M > INT32_MAX || s.N > INT32_MAX) return fail(SPAROA_ERR_UNSUPPORTED, "GEMM too large");

  GemmArgs a;
  a.x = static_cast<const char *>(x);
  a.w = static_cast<const char *>(w);
  a.bias = static_cast<const char *>(bias);
  a.residual = static_cast<const char *>(residual);
  a.y = static_cast<char *>(y);
  a.partial = static_cast<float *>(ws);
  a.mask = mask;
  a.executed = reinterpret_cast<unsigned long long *>(skip ? executed : nullptr);
  a.M = s.M; a.N = s.N; a.K = s.K;
  a.H = d.h; a.W = d.w; a.Cin = d.c_in; a.Ho = s.ho; a.Wo = s.wo; a.Kw = d.kw;
  a.sh = d.sh; a.sw = d.sw; a.ph = d.ph; a.pw = d.pw; a.dh = d.dh; a.dw = d.dw;
  a.taps = d.kh * d.kw;
  a.nchunks = nchunks;
  a.split = t.split_k;
  a.chunks_per_split = cdiv(nchunks, t.split_k);
  a.act = act;
  a.route = route ? *route : DeviceRoute{nullptr, 0.0, 0, 0, nullptr};
  const int64_t gz = cdiv(nchunks, a.chunks_per_split);
  a.split = (int)gz;
  if (gz > 1 && ws_bytes < (size_t)gz * s.M * s.N * sizeof(float))
    return fail(SPAROA_ERR_WORKSPACE, "GEMM split-K workspace too small");

  if (executed) {
    hipLaunchKernelGGL(set_u64, dim3(1), dim3(1), 0, stream,
                       reinterpret_cast<unsigned long long *>(executed), 0ull);
    SPAROA_LAUNCH_CHECK("set_u64");
  }
  dim3 grid((unsigned)cdiv(s.M, t.bm), (unsigned)cdiv(s.N, t.bn), (unsigned)gz);
  bool ok = false;
  switch (d.dtype) {
    case SPAROA_BF16: ok = dispatch<SPAROA_BF16>(t.bm, t.bn, vec, skip, grid, stream, a); break;
    case SPAROA_F16: ok = dispatch<SPAROA_F16>(t.bm, t.bn, vec, skip, grid, stream, a); break;
    case SPAROA_F32: ok = dispatch<SPAROA_F32>(t.bm, t.bn, vec, skip, grid, stream, a); break;
  }
  if (!ok) return fail(SPAROA_ERR_UNSUPPORTED, "GEMM tile shape");
  SPAROA_LAUNCH_CHECK("gemm_kernel");
  if (gz > 1)
    return launch_split_reduce(d.dtype, a.partial, a.split, s.M, s.N, bias, residual, act, y,
                               stream);
  return SPAROA_OK;
}

}  // namespace sparoa
