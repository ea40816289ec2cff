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
#include "commit.h"
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
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

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
  int64_t x_bytes, w_bytes;  // buffer-descriptor ranges (second-generation kernel)
  float inv_wo, inv_ho;      // 1 / Wo, 1 / Ho rounded once on the host (float divmod)
  // 32-bit tile walk of the second-generation kernel (every value below
  // 2^24; the host checks the tile count): column tiles, row x column tiles
  // per split, chunks per tap, kernel rows, and the reciprocals of the
  // divisors rounded once (float divmod)
  int ntn32, ntmn32, cpt32, kh32;
  float inv_ntn, inv_ntmn, inv_cpt, inv_kw, inv_dh, inv_dw;
  int act;
  int split;
  DeviceRoute route;
  sparoa_counts *om_counts;  // non-null: the epilogue measures y (OutMeasure)
  uint32_t *om_mask;
  unsigned long long *om_words;  // grouped count commit words, or null
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

__device__ __forceinline__ int64_t cdiv_dev(int64_t a, int64_t b) { return (a + b - 1) / b; }

// q = n / d, r = n % d for 0 <= n < 2^24 and 0 < d < 2^24: the float
// quotient is within one of the true one, then one integer correction,
// written as selects (no branch: a kernel's start keeps one basic block, so
// its kernel-argument loads are issued together rather than one round trip
// per block)
__device__ __forceinline__ void divmod_small(int n, int d, float inv_d, int &q, int &r) {
  const int q0 = (int)((float)n * inv_d);
  const int r0 = n - q0 * d;
  const bool lo = r0 < 0, hi = r0 >= d;
  q = lo ? q0 - 1 : (hi ? q0 + 1 : q0);
  r = lo ? r0 + d : (hi ? r0 - d : r0);
}


// Bit t set for the taps t of [0, k) whose input coordinate o + t d lies in
// [0, n): t from ceil(-o / d) to ceil((n - o) / d), clipped to [0, k <= 32)
// (no branch; inv_d = 1 / d rounded once).
__device__ __forceinline__ uint32_t taps_inside(int o, int n, int k, int d, float inv_d) {
  int lo, hi, rem;
  divmod_small(max(-o, 0) + d - 1, d, inv_d, lo, rem);
  divmod_small(max(n - o, 0) + d - 1, d, inv_d, hi, rem);
  lo = min(lo, k);
  hi = min(hi, k);
  const uint32_t mhi = hi >= 32 ? ~0u : (1u << hi) - 1u;
  const uint32_t mlo = lo >= 32 ? ~0u : (1u << lo) - 1u;
  return hi > lo ? mhi & ~mlo : 0u;
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
// applies the activation.  Grouped form: up to kGroupMax reductions of one
// dtype in one launch, work-groups dealt to the jobs in proportion to their
// size.  A thread finishes 8 consecutive outputs (16-byte partial, bias and
// residual loads, one 16-byte store) when N % 8 == 0, else one.
struct ReduceGroup {
  int n;
  int wg_begin[kGroupMax + 1];
  const float *partial[kGroupMax];
  int split[kGroupMax];
  int64_t M[kGroupMax], N[kGroupMax];
  const char *bias[kGroupMax], *residual[kGroupMax];
  int act[kGroupMax];
  char *y[kGroupMax];
  sparoa_counts *om_counts[kGroupMax];  // non-null: measure y (16-bit, N % 8 == 0)
  uint32_t *om_mask[kGroupMax];
  unsigned long long *om_words[kGroupMax];
};

template <int DT>
__global__ __launch_bounds__(256) void split_reduce_group(ReduceGroup g) {
  using E = Elem<DT>;
  using raw = typename E::raw;
  // this work-group's job: the starts at or below blockIdx.x, counted over
  // fixed indices (their loads are issued together, not one per step)
  int j = 0;
#pragma unroll
  for (int q = 1; q < kGroupMax; ++q) j += (q < g.n && (int)blockIdx.x >= g.wg_begin[q]) ? 1 : 0;
  const int64_t b0 = blockIdx.x - g.wg_begin[j], nb = g.wg_begin[j + 1] - g.wg_begin[j];
  const int64_t M = g.M[j], N = g.N[j], total = M * N;
  const float *partial = g.partial[j];
  const int split = g.split[j], act = g.act[j];
  const raw *bias = reinterpret_cast<const raw *>(g.bias[j]);
  const raw *res = reinterpret_cast<const raw *>(g.residual[j]);
  raw *y = reinterpret_cast<raw *>(g.y[j]);
  // output measurement: vector v = block v at (1 row, 8 channels); a wave's
  // 64 consecutive vectors are two whole bitmap words (as in measure_lanebit)
  sparoa_counts *om = E::size == 2 ? g.om_counts[j] : nullptr;
  uint32_t *om_mask = g.om_mask[j];   // null: counts only
  const int lane = threadIdx.x & 63;
  const int64_t om_words = om_mask ? (total / 8 + 31) / 32 : 0;
  uint32_t om_zeros = 0, om_nz = 0;
  if (N % 8 == 0) {
    // the column advances by a fixed step mod N (one division per thread)
    const int64_t step = nb * 256;
    int64_t col = ((b0 * 256 + threadIdx.x) * 8) % N;
    const int64_t col_step = (step * 8) % N;
    for (int64_t v = b0 * 256 + threadIdx.x; v < total / 8;
         v += step, col = col + col_step >= N ? col + col_step - N : col + col_step) {
      const int64_t i = v * 8;
      float o[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
      // the slices' partial sums added in slice order (the rounding of the
      // reduction is fixed), four slices' loads in flight at a time
      int z = 0;
      for (; z + 4 <= split; z += 4) {
        float4 lo[4], hi[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          lo[u] = *reinterpret_cast<const float4 *>(partial + (z + u) * total + i);
          hi[u] = *reinterpret_cast<const float4 *>(partial + (z + u) * total + i + 4);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          o[0] += lo[u].x; o[1] += lo[u].y; o[2] += lo[u].z; o[3] += lo[u].w;
          o[4] += hi[u].x; o[5] += hi[u].y; o[6] += hi[u].z; o[7] += hi[u].w;
        }
      }
      for (; z < split; ++z) {
        const float4 lo = *reinterpret_cast<const float4 *>(partial + z * total + i);
        const float4 hi = *reinterpret_cast<const float4 *>(partial + z * total + i + 4);
        o[0] += lo.x; o[1] += lo.y; o[2] += lo.z; o[3] += lo.w;
        o[4] += hi.x; o[5] += hi.y; o[6] += hi.z; o[7] += hi.w;
      }
      raw t[8];
      if (bias) {
        if constexpr (E::size == 2) {
          const uint4 q = *reinterpret_cast<const uint4 *>(bias + col);
          __builtin_memcpy(t, &q, 16);
        } else {
          for (int e = 0; e < 8; ++e) t[e] = bias[col + e];
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) o[e] += E::to_f32(t[e]);
      }
      if (res) {
        if constexpr (E::size == 2) {
          const uint4 q = *reinterpret_cast<const uint4 *>(res + i);
          __builtin_memcpy(t, &q, 16);
        } else {
          for (int e = 0; e < 8; ++e) t[e] = res[i + e];
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) o[e] += E::to_f32(t[e]);
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) t[e] = E::from_f32(apply_act(o[e], act));
      if constexpr (E::size == 2) {
        uint4 q;
        __builtin_memcpy(&q, t, 16);
        *reinterpret_cast<uint4 *>(y + i) = q;
        if (om) {
          uint32_t nzb = 0;
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const bool z = (t[e] & 0x7FFFu) == 0u;
            om_zeros += z ? 1u : 0u;
            nzb |= z ? 0u : 1u;
          }
          om_nz += nzb;
          const uint64_t bal = __ballot(nzb != 0u);
          const int64_t w0 = (v - lane) >> 5;
          if (lane == 0 && w0 < om_words) om_mask[w0] = (uint32_t)bal;
          if (lane == 32 && w0 + 1 < om_words) om_mask[w0 + 1] = (uint32_t)(bal >> 32);
        }
      } else {
        for (int e = 0; e < 8; ++e) y[i + e] = t[e];
      }
    }
    if (om) om_commit(om_zeros, om_nz, om, g.om_words[j], b0, nb);
  } else {
    for (int64_t i = b0 * 256 + threadIdx.x; i < total; i += nb * 256) {
      float o = 0.f;
      for (int z = 0; z < split; ++z) o += partial[z * total + i];
      const int64_t col = i % N;
      if (bias) o += E::to_f32(bias[col]);
      if (res) o += E::to_f32(res[i]);
      y[i] = E::from_f32(apply_act(o, act));
    }
  }
}

// ---------------------------------------------------------------------------
// Second-generation implicit GEMM for the common case: 16-bit data, groups 1,
// C_in % 64 == 0.  A K chunk is 64 channels of one tap, so the tap and
// channel offset of a chunk are work-group-uniform scalars (no per-vector
// division), and a thread's gathered pixels only move by the tap offset.
// Work-group = WGM x WGN waves; a wave owns WTM x WTN MFMA 16x16 blocks,
// which sets the LDS bytes read per MFMA.  Chunks are staged global ->
// registers -> LDS (swizzled 128-byte rows: conflict-free 16-byte reads and
// writes), double-buffered, one barrier per
// 64-wide chunk (two MFMA k-steps).  Gathers are branch-free (out-of-image
// taps read a valid address and are zeroed) so all of a thread's loads are
// in flight together.  Tiles are ordered so that each XCD works on a
// contiguous range of output rows (neighbouring tiles share input halos in
// that XCD's L2).  The skip form walks only the (tap, 64-channel) chunks in
// which some gathered pixel of the tile is nonzero, in dense order, so its
// output equals the dense form's bit for bit.
constexpr int kBK2 = 64;
constexpr int kMaxChunks2 = 1024;          // K <= 65536 on the skip path

// PART: C_in % 64 != 0, a tap's last chunk is partial (a separate
// instantiation: the per-lane channel test and the per-chunk weight offset
// cost the whole-chunk kernels up to 10 %).
template <int DT, int WGM, int WGN, int WTM, int WTN, int PF, int KS, bool SKIP, bool PART>
__global__ __launch_bounds__(64 * WGM * WGN, 2) void igemm_kernel(GemmArgs a) {
  constexpr int NT = 64 * WGM * WGN;   // threads per work-group
  constexpr int BKC = 32 * KS;         // channels per chunk (KS MFMA k-steps)
  // LDS rows of 128 bytes with 16-byte vector v of row r stored at slot
  // v ^ (r & 7): the vectors of one column in any 8 consecutive rows sit in
  // distinct banks, so the 16-byte writes and MFMA-operand reads are free of
  // bank conflicts without padding (measured as fast as 160-byte padded rows
  // and 20 % smaller).
  constexpr int ROW = BKC * 2;
  constexpr int VPR = BKC / 8;         // 16-byte vectors per chunk row
  using E = Elem<DT>;
  static_assert(E::size == 2, "16-bit types");
  static_assert(VPR == 8, "swizzle of 8-vector rows");
  constexpr int BM = WGM * 16 * WTM, BN = WGN * 16 * WTN;
  constexpr int AV = BM * VPR / NT;  // 16-byte A vectors per thread per chunk
  constexpr int BV = BN * VPR / NT;
  constexpr int RPU = NT / VPR;       // rows covered by one vector slot u
  static_assert(AV >= 1 && BV >= 1, "tile too small");
  static_assert(RPU % 8 == 0, "a thread's rows agree mod 8");
  constexpr int CS = BN + 4;  // fp32 row stride of the epilogue's staged tile
  constexpr int STAGE = 2 * (BM + BN) * ROW;
  constexpr int SMEM = STAGE > BM * CS * 4 ? STAGE : BM * CS * 4;

  __shared__ __attribute__((aligned(16))) char smem_raw[SMEM];
  auto stage = [&](int buf) __attribute__((always_inline)) -> char * {
    return smem_raw + buf * ((BM + BN) * ROW);
  };
  // the chunks this tile walks, in order, each packed as
  // j | cb << 10 | r << 20 | s << 25 (chunk id, channel block within the
  // tap, kernel row and column): the walk needs no division per chunk
  __shared__ int list[kMaxChunks2];
  __shared__ uint32_t nzvec[SKIP ? kMaxVecWords + 1 : 1];
  __shared__ int list_len;
  __shared__ uint8_t ombytes[BM * (BN / 64 > 0 ? BN / 64 : 1)];   // output bitmap bytes of the tile

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WGN, wn = wave % WGN;
  // XCD-aware order on a 1-D grid: work-groups are dealt round-robin to the 8
  // XCDs, so XCD i gets the i-th contiguous range of tile ids, and a tile id
  // walks (split, row tile, column tile) with the column tiles innermost: the
  // tiles that gather the same input rows run together in one XCD's L2.
  // (tile arithmetic in 32 bits with float-reciprocal division: a 64-bit
  // division by a runtime value is a long scalar sequence on the critical
  // path of every work-group's start)
  // The set-up's kernel arguments are requested in one round trip: this
  // empty statement needs them at the top (the compiler otherwise loads each
  // group just before its first use, behind branches, one round trip each).
  asm volatile("" ::"s"(a.M), "s"(a.N), "s"(a.H), "s"(a.W), "s"(a.Cin), "s"(a.Ho), "s"(a.Wo),
               "s"(a.Kw), "s"(a.sh), "s"(a.sw), "s"(a.ph), "s"(a.pw), "s"(gridDim.x),
               "s"(a.route.counts), "s"(a.route.path_out), "s"(a.om_counts));
  const int ntiles = (int)gridDim.x;   // row tiles x column tiles x splits
  const bool om = BN % 64 == 0 && a.om_counts != nullptr;
  // the device route's counts, requested first as vector loads (in-order
  // counters: waiting for them later does not wait for the loads behind
  // them; a scalar load would make the first kernel-argument use wait for
  // it): their latency overlaps the tile's offset arithmetic and the dense
  // walk's list writes
  u32x4 rcq[2] = {u32x4{0u, 0u, 0u, 0u}, u32x4{0u, 0u, 0u, 0u}};
  if (SKIP && !a.route.sample_zeros && a.route.counts) {
    const __amdgpu_buffer_rsrc_t cr = __builtin_amdgcn_make_buffer_rsrc(
        (void *)a.route.counts, (short)0, (int)sizeof(sparoa_counts), kBufDword3);
    rcq[0] = __builtin_amdgcn_raw_buffer_load_b128(cr, 0, 0, 0);
    rcq[1] = __builtin_amdgcn_raw_buffer_load_b128(cr, 16, 0, 0);
  }
  // one tile; returns its output's zero count and nonzero-block count
  auto tile_body = [&](const int vid) __attribute__((always_inline)) -> uint2 {
  // (XCD i holds the i-th range: q + 1 tiles for the first r XCDs, q after)
  const int tile = (vid & 7) * (ntiles >> 3) + min(vid & 7, ntiles & 7) + (vid >> 3);
  int zsplit_, rest, mt, nt;
  divmod_small(tile, a.ntmn32, a.inv_ntmn, zsplit_, rest);
  divmod_small(rest, a.ntn32, a.inv_ntn, mt, nt);
  const int64_t zsplit = zsplit_;
  const int64_t m0 = (int64_t)mt * BM, n0 = (int64_t)nt * BN;
  const bool first_tile = tile == 0;
  const bool first_col = nt == 0;
  const int cps = (int)a.chunks_per_split;
  const int c_begin = zsplit_ * cps;
  const int c_end = min(c_begin + cps, (int)a.nchunks);
  const int cpt = a.cpt32;   // chunks per tap
  const float inv_cpt = a.inv_cpt, inv_kw_ = a.inv_kw;
  auto pack_chunk = [&](int j) __attribute__((always_inline)) -> int {
    int t, cb, r, sx;
    divmod_small(j, cpt, inv_cpt, t, cb);
    divmod_small(t, (int)a.Kw, inv_kw_, r, sx);
    return j | (cb << 10) | (r << 20) | (sx << 25);
  };
  const int cg = tid % VPR;             // this thread's 16-byte column of a chunk row
  const int rr = tid / VPR;             // this thread's first chunk row

  // ---- gathered pixels of this thread's A rows (fixed over the K loop).
  // Loads go through buffer descriptors: a 32-bit byte offset per lane, and
  // an offset past the end (taps in the padding) reads 0 without touching
  // memory.  vt[u] has bit t set when tap t of row u lies inside the image.
  const __amdgpu_buffer_rsrc_t xr =
      __builtin_amdgcn_make_buffer_rsrc((void *)a.x, (short)0, (int)a.x_bytes, kBufDword3);
  const __amdgpu_buffer_rsrc_t wr =
      __builtin_amdgcn_make_buffer_rsrc((void *)a.w, (short)0, (int)a.w_bytes, kBufDword3);
  int a_offb[AV];      // byte offset of (n, h0, w0, channel cg*8)
  uint32_t vrow[AV], vcol[AV];  // bit r / s: kernel row r / column s lies inside the image
  const int H = (int)a.H, W = (int)a.W, Ho = (int)a.Ho, Wo = (int)a.Wo, Cin = (int)a.Cin;
  const int kw = (int)a.Kw, dh = (int)a.dh, dw = (int)a.dw;
  const float inv_wo = a.inv_wo, inv_ho = a.inv_ho;
#pragma unroll
  for (int u = 0; u < AV; ++u) {
    const int m = (int)m0 + rr + RPU * u;
    const int mm = m < (int)a.M ? m : 0;
    int t1, ow, nn, oh;
    divmod_small(mm, Wo, inv_wo, t1, ow);
    divmod_small(t1, Ho, inv_ho, nn, oh);
    const int h0 = oh * (int)a.sh - (int)a.ph, w0 = ow * (int)a.sw - (int)a.pw;
    a_offb[u] = (((nn * H + h0) * W + w0) * Cin + cg * 8) * 2;
    vrow[u] = taps_inside(h0, H, a.kh32, dh, a.inv_dh);
    vcol[u] = taps_inside(w0, W, kw, dw, a.inv_dw);
  }
  int b_offb[BV];
#pragma unroll
  for (int u = 0; u < BV; ++u) {
    const int jn = (int)n0 + rr + RPU * u;
    b_offb[u] = ((jn < (int)a.N ? jn : 0) * (int)a.K + cg * 8) * 2;
  }

  // ---- skip list ---------------------------------------------------------
  int count = c_end - c_begin;
  bool use_list = SKIP;
  bool prefilled = false;   // the list already holds the dense walk
  if constexpr (SKIP) {
    if (a.route.sample_zeros) {
      // split execution: this tile's own route, from the zero counts of the
      // samples its rows come from (one double division, >=, as sparoa_route)
      const int64_t last = min(m0 + BM, a.M) - 1;
      const int64_t s0 = m0 / a.route.rows_per_sample, s1 = last / a.route.rows_per_sample;
      unsigned long long z = 0;
      for (int64_t q = s0; q <= s1; ++q) z += a.route.sample_zeros[q];
      const double n = (double)((unsigned long long)(s1 - s0 + 1) *
                                (unsigned long long)a.route.sample_numel);
      use_list = (double)z / n >= a.route.sparsity_thr;
      if (!use_list && a.executed && first_col && tid == 0 && count)
        atomicAdd(a.executed, (unsigned long long)count);  // a dense tile runs every chunk
    } else if (a.route.counts) {
      // the dense walk is written while the route's counts are in flight
      // (a dense-routed tile then waits for them only once); a skip-routed
      // tile overwrites it with its list
      for (int i = tid; i < (int)count; i += NT) list[i] = pack_chunk((int)c_begin + i);
      prefilled = true;
      uint32_t rw[8];   // the same in every lane: scalars, so the route is uniform
#pragma unroll
      for (int q = 0; q < 8; ++q) rw[q] = __builtin_amdgcn_readfirstlane(rcq[q >> 2][q & 3]);
      sparoa_counts rc;
      __builtin_memcpy(&rc, rw, sizeof(rc));
      use_list = route_skip_counts(rc, a.route.sparsity_thr, a.route.mode);
      if (a.route.path_out && first_tile && tid == 0)
        *a.route.path_out = (use_list ? 1u : 0u) | ((uint32_t)a.route.bw_bit << 1);
    }
  }
  if constexpr (!SKIP) {
    if (a.route.path_out && first_tile && tid == 0)
      *a.route.path_out = (uint32_t)a.route.bw_bit << 1;
  }
  if (SKIP && use_list) {
    const int cpg = (int)(a.Cin / 8);  // bitmap blocks per pixel
    const int kv_words = (int)((a.taps * cpg + 31) / 32) + 1;   // + the window's spare word
    for (int i = tid; i < kv_words; i += NT) nzvec[i] = 0u;
    __syncthreads();
    // (32-bit index arithmetic with float-reciprocal division: pixel
    // indices are below 2^24 on this kernel)
    const int taps = (int)a.taps, ntp = BM * taps;
    const float inv_taps = 1.0f / (float)taps, inv_kw = 1.0f / (float)kw;
    for (int p = tid; p < ntp; p += NT) {
      int r_in, tap, t1, ow, nn, oh, r, sx;
      divmod_small(p, taps, inv_taps, r_in, tap);
      const int m = (int)m0 + r_in;
      if (m >= (int)a.M) continue;
      divmod_small(m, Wo, inv_wo, t1, ow);
      divmod_small(t1, Ho, inv_ho, nn, oh);
      divmod_small(tap, kw, inv_kw, r, sx);
      const int ih = oh * (int)a.sh - (int)a.ph + r * dh, iw = ow * (int)a.sw - (int)a.pw + sx * dw;
      if (ih < 0 || ih >= H || iw < 0 || iw >= W) continue;
      const int64_t pix = ((int64_t)nn * H + ih) * W + iw;
      for (int b = 0; b < cpg; b += 32) {
        const int nb = min(32, cpg - b);
        lds_or_bits(nzvec, tap * cpg + b, read_bits(a.mask, pix * cpg + b, nb), nb);
      }
    }
    __syncthreads();
    if (wave == 0) {
      int total = 0;
      for (int base = c_begin; base < c_end; base += 64) {
        const int j = base + lane;
        bool nz = false;
        if (j < c_end) {
          // chunk j = channels [BKC cb, min(BKC cb + BKC, Cin)) of tap t:
          // up to BKC / 8 bitmap bits from bit t cpg + (BKC / 8) cb, read
          // through a 64-bit window (with cpg % 8 != 0 they may straddle a
          // word; the word past the last is cleared)
          // (whole chunks: BKC / 8 bits at a multiple of BKC / 8, inside
          // one word)
          static_assert(BKC / 8 <= 32, "chunk bits in a 64-bit window");
          int t, cb;
          divmod_small(j, cpt, inv_cpt, t, cb);
          const int pos = t * cpg + (BKC / 8) * cb;
          if constexpr (PART) {
            const int nb = min(BKC / 8, cpg - (BKC / 8) * cb);
            const uint64_t win =
                (uint64_t)nzvec[pos >> 5] | ((uint64_t)nzvec[(pos >> 5) + 1] << 32);
            nz = ((win >> (pos & 31)) & ((1ull << nb) - 1ull)) != 0ull;
          } else {
            constexpr uint32_t kBits = BKC / 8 >= 32 ? 0xFFFFFFFFu : ((1u << (BKC / 8)) - 1u);
            nz = ((nzvec[pos >> 5] >> (pos & 31)) & kBits) != 0u;
          }
        }
        const uint64_t bal = __ballot(nz);
        const int before = __popcll(bal & ((1ull << lane) - 1ull));
        if (nz) list[total + before] = pack_chunk(j);
        total += __popcll(bal);
      }
      if (lane == 0) {
        list_len = total;
        if (a.executed && first_col && total)
          atomicAdd(a.executed, (unsigned long long)total);
      }
    }
    __syncthreads();
    count = list_len;
  }

  // ---- staging: a ring of PF chunks in registers, two chunks in LDS --------
  u32x4 ra[PF][AV], rb[PF][BV];  // native vectors: no struct copies, stays in VGPRs
  // valid == false: every offset out of range, the loads return zeros without
  // touching memory -- the prologue issues its PF + 1 loads unconditionally,
  // so the compiler can count the loads in flight at the loop head (a
  // conditional prologue load made it wait for the whole ring there)
  auto load_chunk = [&](int info, u32x4 (&ra_s)[AV], u32x4 (&rb_s)[BV], bool valid)
                        __attribute__((always_inline)) {
    const int j = info & 1023, cb = (info >> 10) & 1023;
    const int r = (info >> 20) & 31, sx = (info >> 25) & 31;
    const int tap_offb = ((r * dh * W + sx * dw) * Cin + cb * BKC) * 2;
    // PART: this lane's 8 channels of the chunk exist (channels past C_in in
    // the last chunk of a tap read zero on both sides), and the chunk starts
    // at K index (r kw + sx) C_in + BKC cb of a weight row (whole chunks:
    // at BKC j)
    const bool col = PART ? valid && cb * BKC + cg * 8 < Cin : valid;
    const int kofs = PART ? ((r * kw + sx) * Cin + cb * BKC) * 2 : j * (BKC * 2);
#pragma unroll
    for (int u = 0; u < AV; ++u) {
      const bool in_img = col && ((vrow[u] >> r) & (vcol[u] >> sx) & 1u);
      const int off = in_img ? a_offb[u] + tap_offb : (int)0x80000000;
      ra_s[u] = __builtin_amdgcn_raw_buffer_load_b128(xr, off, 0, 0);
    }
#pragma unroll
    for (int u = 0; u < BV; ++u)
      rb_s[u] = __builtin_amdgcn_raw_buffer_load_b128(wr, col ? b_offb[u] : (int)0x80000000,
                                                      valid ? kofs : 0, 0);
  };
  // every row a thread stores is rr mod 8 (RPU and BM are multiples of 8)
  const int st_col = 16 * (cg ^ (rr & 7));
  auto store_chunk = [&](int buf, const u32x4 (&ra_s)[AV], const u32x4 (&rb_s)[BV])
                         __attribute__((always_inline)) {
    char *s = stage(buf);
#pragma unroll
    for (int u = 0; u < AV; ++u)
      *reinterpret_cast<u32x4 *>(s + (rr + RPU * u) * ROW + st_col) = ra_s[u];
#pragma unroll
    for (int u = 0; u < BV; ++u)
      *reinterpret_cast<u32x4 *>(s + (BM + rr + RPU * u) * ROW + st_col) = rb_s[u];
  };

  f32x4 acc[WTM][WTN];
#pragma unroll
  for (int i = 0; i < WTM; ++i)
#pragma unroll
    for (int j = 0; j < WTN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int g = lane >> 4, rl = lane & 15;
  // operand rows of a lane are rl mod 16, so their swizzle is rl & 7
  int ks_col[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) ks_col[ks] = 16 * ((4 * ks + g) ^ (rl & 7));
  auto compute = [&](int buf) __attribute__((always_inline)) {
    const char *As = stage(buf) + (wm * WTM * 16 + rl) * ROW;
    const char *Bs = stage(buf) + (BM + wn * WTN * 16 + rl) * ROW;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      u32x4 af[WTM], bfr[WTN];
#pragma unroll
      for (int tm = 0; tm < WTM; ++tm)
        af[tm] = *reinterpret_cast<const u32x4 *>(As + tm * 16 * ROW + ks_col[ks]);
#pragma unroll
      for (int tn = 0; tn < WTN; ++tn)
        bfr[tn] = *reinterpret_cast<const u32x4 *>(Bs + tn * 16 * ROW + ks_col[ks]);
#pragma unroll
      for (int tm = 0; tm < WTM; ++tm)
#pragma unroll
        for (int tn = 0; tn < WTN; ++tn) {
          if constexpr (DT == SPAROA_BF16)
            acc[tm][tn] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(bf16x8, af[tm]), __builtin_bit_cast(bf16x8, bfr[tn]),
                acc[tm][tn], 0, 0, 0);
          else
            acc[tm][tn] = __builtin_amdgcn_mfma_f32_16x16x32_f16(
                __builtin_bit_cast(f16x8, af[tm]), __builtin_bit_cast(f16x8, bfr[tn]),
                acc[tm][tn], 0, 0, 0);
        }
    }
  };
  // Chunk i lives in register slot i % PF until it is stored to LDS buffer
  // i & 1 (one iteration ahead of its use); the slot is then refilled with
  // chunk i + PF, so PF chunks of loads are always in flight.  The loop body
  // is written out once per slot so every slot index is a constant and the
  // ring stays in registers.
  static_assert(PF >= 2 && PF <= 4, "register ring depth");
  const int n = (int)count;
  // dense walks (the dense kernel, and a dense-routed tile of the skip
  // kernel) fill the list in dense order: no branch on the route inside the
  // main loop
  if (!SKIP || !use_list) {
    if (!prefilled)
      for (int i = tid; i < (int)count; i += NT) list[i] = pack_chunk((int)c_begin + i);
    __syncthreads();
  }
  // (the list entry is the same in every lane: read it as a scalar, so the
  // weight loads take it as their scalar offset -- an LDS value the
  // compiler must treat as divergent made it wrap every weight load in a
  // readfirstlane loop)
  auto chunk_at = [&](int i) __attribute__((always_inline)) -> int {
    return __builtin_amdgcn_readfirstlane(list[i]);
  };
  if (n > 0) {
    // chunk 0 alone first (every work-group starts at once: a deep prologue
    // would queue each one's first chunk behind all the others' prefetch)
    // (chunks past the last are not loaded: short K -- a 1x1 conv over 64
    // channels is one chunk -- would otherwise re-read its chunks PF times)
    load_chunk(chunk_at(0), ra[0], rb[0], true);
    store_chunk(0, ra[0], rb[0]);
    load_chunk(chunk_at(min(1, n - 1)), ra[1], rb[1], 1 < n);
    if constexpr (PF > 2)
      load_chunk(chunk_at(min(2, n - 1)), ra[PF > 2 ? 2 : 0], rb[PF > 2 ? 2 : 0], 2 < n);
    if constexpr (PF > 3)
      load_chunk(chunk_at(min(3, n - 1)), ra[PF > 3 ? 3 : 0], rb[PF > 3 ? 3 : 0], 3 < n);
    load_chunk(chunk_at(min(PF, n - 1)), ra[0], rb[0], PF < n);
    __syncthreads();
  // Steady state: groups of PF straight-line steps (no branch inside a step,
  // so the compiler's load counters stay exact and PF chunks stay in flight);
  // the refill past the end re-reads the last chunk.  The last group runs
  // the guarded form.
#define SPAROA_IG_STEP(D, GUARD)                                                   \
  {                                                                                \
    constexpr int sn = ((D) + 1) % PF;                                             \
    const int i = i0 + (D);                                                        \
    if (!(GUARD) || i < n) {                                                       \
      const int jn = chunk_at(min(i + 1 + PF, n - 1)); /* read before the MFMAs */ \
      compute(i & 1);                                                              \
      if (!(GUARD) || i + 1 < n) store_chunk((i + 1) & 1, ra[sn], rb[sn]); \
      if (!(GUARD) || i + 1 + PF < n) load_chunk(jn, ra[sn], rb[sn], true);      \
      __syncthreads();                                                             \
    }                                                                              \
  }
    int i0 = 0;
    for (; i0 + PF < n; i0 += PF) {
      SPAROA_IG_STEP(0, false)
      SPAROA_IG_STEP(1, false)
      if constexpr (PF > 2) SPAROA_IG_STEP(2, false)
      if constexpr (PF > 3) SPAROA_IG_STEP(3, false)
    }
    for (; i0 < n; i0 += PF) {
      SPAROA_IG_STEP(0, true)
      SPAROA_IG_STEP(1, true)
      if constexpr (PF > 2) SPAROA_IG_STEP(2, true)
      if constexpr (PF > 3) SPAROA_IG_STEP(3, true)
    }
#undef SPAROA_IG_STEP
  }

  // ---- epilogue: the fp32 tile goes through LDS (a lane holds rows
  // 4*(lane/16) + v, column lane % 16 of each MFMA block), then each thread
  // finishes 8 consecutive columns of a row: bias and residual as 16-byte
  // loads, one 16-byte store.
  using raw = typename E::raw;
  float *ct = reinterpret_cast<float *>(smem_raw);
  __syncthreads();
#pragma unroll
  for (int tm = 0; tm < WTM; ++tm)
#pragma unroll
    for (int tn = 0; tn < WTN; ++tn)
#pragma unroll
      for (int v = 0; v < 4; ++v)
        ct[(wm * WTM * 16 + tm * 16 + 4 * g + v) * CS + wn * WTN * 16 + tn * 16 + rl] =
            acc[tm][tn][v];
  __syncthreads();
  constexpr int C8 = BN / 8;
  constexpr int EIT = BM * C8 / NT;   // epilogue rows per thread
  static_assert(BM * C8 % NT == 0 && NT % C8 == 0, "epilogue mapping");
  const bool vec_n = a.N % 8 == 0;
  // A thread's 8 columns are the same in every epilogue row (NT is a
  // multiple of C8): its bias vector is loaded once, and the residual
  // vectors of all its rows are requested before its first store (a load
  // issued behind stores waits for them here, which serialised the rows).
  const int c_t = (tid % C8) * 8;
  const bool vec_t = vec_n && a.split == 1 && n0 + c_t < a.N;
  using raw_t = typename E::raw;
  uint4 bias_q = {0u, 0u, 0u, 0u};
  if (a.bias && vec_t)
    bias_q = *reinterpret_cast<const uint4 *>(reinterpret_cast<const raw_t *>(a.bias) + n0 + c_t);
  uint4 res_q[EIT];
#pragma unroll
  for (int it = 0; it < EIT; ++it) {
    const int64_t row = m0 + (tid + it * NT) / C8;
    res_q[it] = uint4{0u, 0u, 0u, 0u};
    if (a.residual && vec_t && row < a.M)
      res_q[it] = *reinterpret_cast<const uint4 *>(reinterpret_cast<const raw_t *>(a.residual) +
                                                   row * a.N + n0 + c_t);
  }
  // Output measurement (host: no split, N % 64 == 0, and N % BN == 0 for
  // wider tiles): each 8 consecutive lanes of a tile row hold one bitmap byte
  // (8 channel blocks of 8); every lane stays in the loop for the ballot.
  uint32_t om_zeros = 0, om_nz = 0;
#pragma unroll
  for (int it = 0; it < EIT; ++it) {
    const int q = tid + it * NT;
    const int r = q / C8, c = (q % C8) * 8;
    const int64_t row = m0 + r, col = n0 + c;
    if (om) {
      const bool valid = row < a.M;
      uint32_t nzb = 0;
      if (valid) {
        float o[8];
        const float4 lo = *reinterpret_cast<const float4 *>(&ct[r * CS + c]);
        const float4 hi = *reinterpret_cast<const float4 *>(&ct[r * CS + c + 4]);
        o[0] = lo.x; o[1] = lo.y; o[2] = lo.z; o[3] = lo.w;
        o[4] = hi.x; o[5] = hi.y; o[6] = hi.z; o[7] = hi.w;
        raw t[8], out[8];
        if (a.bias) {
          __builtin_memcpy(t, &bias_q, 16);
#pragma unroll
          for (int e = 0; e < 8; ++e) o[e] += E::to_f32(t[e]);
        }
        if (a.residual) {
          __builtin_memcpy(t, &res_q[it], 16);
#pragma unroll
          for (int e = 0; e < 8; ++e) o[e] += E::to_f32(t[e]);
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          out[e] = E::from_f32(apply_act(o[e], a.act));
          const bool z = (out[e] & 0x7FFFu) == 0u;
          om_zeros += z ? 1u : 0u;
          nzb |= z ? 0u : 1u;
        }
        uint4 q4;
        __builtin_memcpy(&q4, out, 16);
        *reinterpret_cast<uint4 *>(reinterpret_cast<raw *>(a.y) + row * a.N + col) = q4;
      }
      om_nz += nzb;
      const uint64_t bal = __ballot(nzb != 0u);
      // the tile's bitmap bytes (8 channel blocks of 8 per byte) meet in LDS
      // and each row's BN / 64 bytes leave as one store below
      if ((lane & 7) == 0) ombytes[r * (BN / 64) + c / 64] = valid ? (uint8_t)(bal >> (lane & ~7)) : 0;
      continue;
    }
    if (row >= a.M || col >= a.N) continue;
    float o[8];
    {
      const float4 lo = *reinterpret_cast<const float4 *>(&ct[r * CS + c]);
      const float4 hi = *reinterpret_cast<const float4 *>(&ct[r * CS + c + 4]);
      o[0] = lo.x; o[1] = lo.y; o[2] = lo.z; o[3] = lo.w;
      o[4] = hi.x; o[5] = hi.y; o[6] = hi.z; o[7] = hi.w;
    }
    const int ne = (int)min((int64_t)8, a.N - col);
    if (a.split > 1) {
      float *dst = a.partial + (zsplit * a.M + row) * a.N + col;
      if (vec_n) {
        *reinterpret_cast<float4 *>(dst) = make_float4(o[0], o[1], o[2], o[3]);
        *reinterpret_cast<float4 *>(dst + 4) = make_float4(o[4], o[5], o[6], o[7]);
      } else {
        for (int e = 0; e < ne; ++e) dst[e] = o[e];
      }
      continue;
    }
    raw *dst = reinterpret_cast<raw *>(a.y) + row * a.N + col;
    if (vec_n) {
      raw bv[8], rv[8], out[8];
      if (a.bias) {
        __builtin_memcpy(bv, &bias_q, 16);
#pragma unroll
        for (int e = 0; e < 8; ++e) o[e] += E::to_f32(bv[e]);
      }
      if (a.residual) {
        __builtin_memcpy(rv, &res_q[it], 16);
#pragma unroll
        for (int e = 0; e < 8; ++e) o[e] += E::to_f32(rv[e]);
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) out[e] = E::from_f32(apply_act(o[e], a.act));
      uint4 q4;
      __builtin_memcpy(&q4, out, 16);
      *reinterpret_cast<uint4 *>(dst) = q4;
    } else {
      for (int e = 0; e < ne; ++e) {
        float v = o[e];
        if (a.bias) v += E::to_f32(reinterpret_cast<const raw *>(a.bias)[col + e]);
        if (a.residual) v += E::to_f32(reinterpret_cast<const raw *>(a.residual)[row * a.N + col + e]);
        dst[e] = E::from_f32(apply_act(v, a.act));
      }
    }
  }
  if (om) {
    __syncthreads();
    // rows past M still clear their bytes when they lie inside the bitmap's
    // last word (bits past the last block are 0)
    const int64_t mbytes = a.om_mask ? 4 * ((a.M * (a.N / 8) + 31) / 32) : 0;   // null: counts only
    for (int r = tid; r < BM; r += NT) {
      const int64_t row = m0 + r, byte = row * (a.N / 64) + n0 / 64;
      if (byte >= mbytes) continue;   // (BN / 64 bytes of a row lie in one word)
      if constexpr (BN == 256) {      // n0 / 64 and N / 64 multiples of 4: 4-byte aligned
        const uint32_t v = (uint32_t)ombytes[4 * r] | ((uint32_t)ombytes[4 * r + 1] << 8) |
                           ((uint32_t)ombytes[4 * r + 2] << 16) |
                           ((uint32_t)ombytes[4 * r + 3] << 24);
        *reinterpret_cast<uint32_t *>(reinterpret_cast<uint8_t *>(a.om_mask) + byte) = v;
      } else if constexpr (BN == 128) {  // n0 / 64 and N / 64 even: 2-byte aligned
        const uint16_t v = (uint16_t)(ombytes[2 * r] | (ombytes[2 * r + 1] << 8));
        *reinterpret_cast<uint16_t *>(reinterpret_cast<uint8_t *>(a.om_mask) + byte) = v;
      } else {
        reinterpret_cast<uint8_t *>(a.om_mask)[byte] = ombytes[r];
      }
    }
  }
  return make_uint2(om_zeros, om_nz);
  };
  // (one tile per work-group; the lambda form measured fewer scalar-register
  // spills than straight-line code)
  const uint2 t = tile_body((int)blockIdx.x);
  if (om) om_commit(t.x, t.y, a.om_counts, a.om_words, blockIdx.x, gridDim.x);
}

// ---------------------------------------------------------------------------
// Direct MFMA conv for inputs with at most 4 channels (image stems: ResNet's
// 7x7/2 and MobileNetV2's 3x3/2 over RGB), where the implicit GEMM's 8- or
// 64-channel K chunks would be mostly padding and its gathers scalar.  A
// work-group computes one output row (all Wo pixels, all C_out <= 64
// channels).  It stages the kh input rows the row needs, zero-padded on both
// sides, in LDS as [kh][PW][4] (channels padded to 4 with zeros), so K is
// laid out as (kernel row r, tap pair j, tap parity, channel): an 8-element
// block of K is two taps x 4 channels, contiguous and 8-byte aligned in the
// patch.  K = kh * ceil(kw/2) blocks, four per v_mfma_f32_16x16x32 k-step;
// a tap past kw (odd kw) and blocks past the last kernel row read zero.  The
// B operands (weights, zero-padded the same way) stay in registers.  Waves
// split C_out into 16-channel column blocks and the Wo pixels into 16-pixel
// row blocks.  Skip form: an MFMA whose A operand is zero in all 64 lanes is
// not issued (it would add exact zeros), so the skip output equals the dense
// output bit for bit; executed_blocks counts the issued (row block, k-step)
// pairs.  The fp32 tile goes through LDS to 16-byte stores with bias,
// residual and activation; each thread's 8 output channels of a pixel are one
// (1, 8) block of the output, so the epilogue also counts zeros and nonzero
// blocks when asked (counts-only measurement of y, one ticketed commit per
// work-group).
constexpr int kScMaxKSteps = 8;
constexpr int kScMaxRB = 8;            // Wo <= 128
constexpr int kScPatchBytes = 48 * 1024;  // LDS bound of the eligible shapes

struct SmallCArgs {
  const char *x, *w, *bias, *residual;
  char *y;
  unsigned long long *executed;
  int N, H, W, C, Ho, Wo, Cout, kh, kw, sh, sw, ph, pw;
  int PW, PWP, bpr, ksteps, act;   // PWP = PW + 1: patch row pitch in pixels
  int raw_elems, w_elems;  // LDS elements of the raw rows and the weights (each % 8 == 0)
  int c_w;                 // weight elements (Cout * kh * kw * C)
  int region_off;          // LDS byte offset of the weights / raw rows / tile region
  float inv_bpr, inv_rv, inv_rowe;   // 1 / bpr, 1 / (W*C/8), 1 / (W*C), rounded once
  int vec;                 // rows and weights are whole 16-byte vectors
  int mode;  // 0 dense, 1 skip, 2 device route
  DeviceRoute route;
  // counts-only output measurement at block (1 pixel, 8 channels): non-null
  // om_counts holds {0, numel, nb, nb} on entry; om_words: count-commit words
  sparoa_counts *om_counts;
  unsigned long long *om_words;
};

template <int DT, int KS>
__global__ __launch_bounds__(256) void conv_small_c_kernel(SmallCArgs a) {
  using E = Elem<DT>;
  using raw = typename E::raw;
  extern __shared__ __attribute__((aligned(16))) char smem[];   // small_c_lds_bytes
  __shared__ unsigned long long exec_part[4];
  __shared__ uint4 sink;   // target of the staging stores of out-of-range lanes
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nwn = a.Cout / 16, nwm = 4 / nwn;   // waves over column / row blocks
  const int wn = wave % nwn, wm = wave / nwn;
  const int g = lane >> 4, rl = lane & 15;
  SPAROA_ARGS_UP_FRONT("s"(a.x), "s"(a.w), "s"(a.H), "s"(a.W), "s"(a.C), "s"(a.Ho), "s"(a.Cout),
                       "s"(a.kh), "s"(a.sh), "s"(a.ph), "s"(a.w_elems), "s"(a.c_w),
                       "s"(a.region_off), "s"(a.inv_rv), "s"(a.vec), "s"(a.mode),
                       "s"(a.route.counts));
  const int img = (int)(blockIdx.x / (unsigned)a.Ho), oh = (int)(blockIdx.x % (unsigned)a.Ho);
  // the device route's counts are requested now and decided on once the
  // weights and input rows are staged (nothing before needs the decision)
  const RouteCountsReq rq = route_counts_request(a.route);
  // LDS: patch [kh][PWP][4] | region: weights [Cout*kh*kw*C], raw input rows
  // [kh][W*C] while the operands are built, then the fp32 output tile
  raw *patch = reinterpret_cast<raw *>(smem);
  char *region = smem + a.region_off;
  raw *wl = reinterpret_cast<raw *>(region);
  raw *rawx = wl + a.w_elems;
  float *ct = reinterpret_cast<float *>(region);
  const raw *x = reinterpret_cast<const raw *>(a.x);
  const raw *w = reinterpret_cast<const raw *>(a.w);
  const int rowe = a.W * a.C;
  const int ih0 = oh * a.sh - a.ph;
  const int64_t img_base = (int64_t)img * a.H * rowe;

  // ---- weights and the kh input rows -> LDS: loads unconditional (clamped
  // addresses; rows outside the image are zeroed by the patch below) and
  // independent, stores unconditional (no branch to sink the loads into)
  if (a.vec) {
    const int wv = a.w_elems / 8, rv = rowe / 8, nv = a.kh * rv;
    for (int v0 = tid; v0 < wv + nv; v0 += 256 * 4) {
      uint4 q[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int v = min(v0 + 256 * u, wv + nv - 1);
        int r, cv;
        divmod_small(max(v - wv, 0), rv, a.inv_rv, r, cv);
        const int ih = min(max(ih0 + r, 0), a.H - 1);
        const raw *src = v < wv ? w + (int64_t)v * 8
                                : x + img_base + (int64_t)ih * rowe + (int64_t)cv * 8;
        q[u] = *reinterpret_cast<const uint4 *>(src);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int v = v0 + 256 * u;
        *(v < wv + nv ? reinterpret_cast<uint4 *>(wl + (size_t)v * 8) : &sink) = q[u];
      }
    }
  } else {
    const int ne = a.kh * rowe;
    for (int e0 = tid; e0 < a.c_w + ne; e0 += 256 * 8) {
      raw q[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int e = min(e0 + 256 * u, a.c_w + ne - 1);
        int r, ce;
        divmod_small(max(e - a.c_w, 0), rowe, a.inv_rowe, r, ce);
        const int ih = min(max(ih0 + r, 0), a.H - 1);
        q[u] = e < a.c_w ? w[e] : x[img_base + (int64_t)ih * rowe + ce];
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int e = e0 + 256 * u;
        raw *dst = e < a.c_w ? wl + e : rawx + (e - a.c_w);
        *(e < a.c_w + ne ? dst : reinterpret_cast<raw *>(&sink)) = q[u];
      }
    }
  }
  __syncthreads();
  bool skip = a.mode == 1;
  if (a.mode == 2) {
    skip = route_counts_skip(rq, a.route);
    if (a.route.path_out && blockIdx.x == 0 && tid == 0)
      *a.route.path_out = (skip ? 1u : 0u) | ((uint32_t)a.route.bw_bit << 1);
  }

  // ---- padded patch patch[r][q][c4] (q = input column + pw; zero outside
  // the image and for channels >= C; one column past PW keeps every operand
  // read in range): a thread owns columns, kernel rows inner
  for (int q = tid; q < a.PWP; q += 256) {
    const int iw = q - a.pw;
    const bool col_in = iw >= 0 && iw < a.W;
    const int iwc = min(max(iw, 0), a.W - 1) * a.C;
    for (int r = 0; r < a.kh; ++r) {
      const int ih = ih0 + r;
      const bool in = col_in && ih >= 0 && ih < a.H;
      const raw *src = rawx + r * rowe + iwc;
      raw v[4];
#pragma unroll
      for (int c = 0; c < 4; ++c) {    // unconditional reads (clamped), then masked
        const raw t = src[min(c, a.C - 1)];
        v[c] = in && c < a.C ? t : (raw)0;
      }
      uint2 q2;
      __builtin_memcpy(&q2, v, 8);
      *reinterpret_cast<uint2 *>(patch + (size_t)(r * a.PWP + q) * 4) = q2;
    }
  }
  // ---- B operands (registers): lane (column rl, group g) at k-step t holds
  // K block b = 4t + g = (kernel row b / bpr, tap pair b % bpr); the A side
  // keeps each block's patch offset and all-ones / zero masks of its taps
  const int co = wn * 16 + rl;
  int koff[KS];
  uint32_t mlo[KS], mhi[KS];
  u32x4 bop[KS];
#pragma unroll
  for (int t = 0; t < KS; ++t) {
    int r, j;
    divmod_small(4 * t + g, a.bpr, a.inv_bpr, r, j);
    const int rc = min(r, a.kh - 1);
    const bool lo_ok = r < a.kh, hi_ok = lo_ok && 2 * j + 1 < a.kw;
    mlo[t] = lo_ok ? 0xFFFFFFFFu : 0u;
    mhi[t] = hi_ok ? 0xFFFFFFFFu : 0u;
    koff[t] = (rc * a.PWP + 2 * j) * 4;
    const raw *wr = wl + ((co * a.kh + rc) * a.kw + 2 * j) * a.C;
    const int s1 = min(2 * j + 1, a.kw - 1) - 2 * j;   // second tap (clamped)
    raw v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int c = e & 3;
      const raw wv = wr[(e >> 2) * s1 * a.C + min(c, a.C - 1)];
      v[e] = (e < 4 ? lo_ok : hi_ok) && c < a.C ? wv : (raw)0;
    }
    __builtin_memcpy(&bop[t], v, 16);
  }
  __syncthreads();   // patch complete; weights and raw rows dead: the tile may reuse them

  // ---- MFMAs, one 16-pixel row block at a time (this wave's rb = wm, wm +
  // nwm, ...); each block's fp32 result goes straight to the tile
  const int RB = (a.Wo + 15) / 16;
  const int CS = a.Cout + 4;
  unsigned long long executed = 0;
  for (int rb = wm; rb < RB; rb += nwm) {
    const int ow = min(rb * 16 + rl, a.Wo - 1);  // rows past Wo read a valid pixel, unused
    const int pix = ow * a.sw * 4;
    u32x4 aops[KS];
#pragma unroll
    for (int t = 0; t < KS; ++t) {   // all reads first
      // two 8-byte reads: a block starts on an 8-byte (not 16-byte) boundary
      const uint2 lo = *reinterpret_cast<const uint2 *>(patch + koff[t] + pix);
      const uint2 hi = *reinterpret_cast<const uint2 *>(patch + koff[t] + pix + 4);
      aops[t] = u32x4{lo.x & mlo[t], lo.y & mlo[t], hi.x & mhi[t], hi.y & mhi[t]};
    }
    f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int t = 0; t < KS; ++t) {
      const u32x4 aop = aops[t];
      if (skip && __ballot((aop[0] | aop[1] | aop[2] | aop[3]) != 0u) == 0ull) continue;  // exact
      executed += 1;
      if constexpr (DT == SPAROA_BF16)
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, aop),
                                                      __builtin_bit_cast(bf16x8, bop[t]), acc,
                                                      0, 0, 0);
      else
        acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, aop),
                                                     __builtin_bit_cast(f16x8, bop[t]), acc,
                                                     0, 0, 0);
    }
#pragma unroll
    for (int v = 0; v < 4; ++v) ct[(rb * 16 + 4 * g + v) * CS + wn * 16 + rl] = acc[v];
  }
  if (a.executed && skip && wn == 0 && lane == 0) exec_part[wm] = executed;
  __syncthreads();

  // ---- epilogue: 8 channels per thread, 16-byte stores
  const int C8 = a.Cout / 8, lc8 = C8 == 8 ? 3 : (C8 == 4 ? 2 : 1);   // Cout in {16, 32, 64}
  const raw *bias = reinterpret_cast<const raw *>(a.bias);
  uint32_t om_zeros = 0, om_nz = 0;
  const int64_t row0 = (int64_t)blockIdx.x * a.Wo;
  for (int q = tid; q < a.Wo * C8; q += 256) {
    const int ow = q >> lc8, c = (q & (C8 - 1)) * 8;
    const int64_t orow = row0 + ow;
    float o[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] = ct[ow * CS + c + e];
    raw t8[8];
    if (bias) {
      const uint4 q4 = *reinterpret_cast<const uint4 *>(bias + c);
      __builtin_memcpy(t8, &q4, 16);
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] += E::to_f32(t8[e]);
    }
    if (a.residual) {
      const uint4 q4 = *reinterpret_cast<const uint4 *>(
          reinterpret_cast<const raw *>(a.residual) + orow * a.Cout + c);
      __builtin_memcpy(t8, &q4, 16);
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] += E::to_f32(t8[e]);
    }
    uint32_t any = 0;   // OR of the magnitudes
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      t8[e] = E::from_f32(apply_act(o[e], a.act));
      // zero test in integer arithmetic (m - 1 wraps to bit 31 iff m == 0)
      const uint32_t m = (uint32_t)t8[e] & E::mag_mask;
      om_zeros += (m - 1u) >> 31;
      any |= m;
    }
    om_nz += ((any - 1u) >> 31) ^ 1u;
    uint4 q4;
    __builtin_memcpy(&q4, t8, 16);
    *reinterpret_cast<uint4 *>(reinterpret_cast<raw *>(a.y) + orow * a.Cout + c) = q4;
  }
  if (a.executed && skip && tid == 0) {
    unsigned long long tot = 0;
    for (int i = 0; i < nwm; ++i) tot += exec_part[i];
    if (tot) atomicAdd(a.executed, tot);
  }
  if (a.om_counts) om_commit(om_zeros, om_nz, a.om_counts, a.om_words, blockIdx.x, gridDim.x);
}

template <int DT, int WGM, int WGN, int WTM, int WTN, int PF, int KS, bool SKIP, bool PART>
void launch_ig(dim3 grid, hipStream_t st, const GemmArgs &a) {
  hipLaunchKernelGGL((igemm_kernel<DT, WGM, WGN, WTM, WTN, PF, KS, SKIP, PART>), grid,
                     dim3(64 * WGM * WGN), 0, st, a);
}

// Tile configurations of the second-generation kernel (BM x BN) and the
// chunks each keeps in flight in registers.
enum IgCfg { kIg128x64 = 1, kIg64x64, kIg128x128, kIg128x256 };

// 64-channel chunks: two MFMA k-steps per barrier (four measured slower:
// more LDS and registers per work-group for the same latency per step).
template <int DT, bool SKIP>
bool dispatch_ig(int cfg, int kchunk, bool part, dim3 grid, hipStream_t st, const GemmArgs &a) {
  if (kchunk != kBK2) return false;
  if (part) {   // partial chunks: the two tiles the chooser takes for them
    switch (cfg) {
      case kIg128x64: launch_ig<DT, 2, 2, 4, 2, 4, 2, SKIP, true>(grid, st, a); return true;
      case kIg64x64: launch_ig<DT, 2, 2, 2, 2, 4, 2, SKIP, true>(grid, st, a); return true;
    }
    return false;
  }
  switch (cfg) {
    case kIg128x64: launch_ig<DT, 2, 2, 4, 2, 4, 2, SKIP, false>(grid, st, a); return true;
    case kIg64x64: launch_ig<DT, 2, 2, 2, 2, 4, 2, SKIP, false>(grid, st, a); return true;
    case kIg128x128: launch_ig<DT, 2, 2, 4, 4, 3, 2, SKIP, false>(grid, st, a); return true;
    case kIg128x256: launch_ig<DT, 2, 4, 4, 4, 3, 2, SKIP, false>(grid, st, a); return true;
  }
  return false;
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

sparoa_status launch_split_reduce_group(const SplitReduceJob *jobs, int n, hipStream_t stream) {
  if (n < 1 || n > kGroupMax) return fail(SPAROA_ERR_INVALID_ARG, "split reduce: group size");
  ReduceGroup g;
  g.n = n;
  int64_t wg = 0;
  for (int j = 0; j < n; ++j) {
    const SplitReduceJob &r = jobs[j];
    if (r.dt != jobs[0].dt) return fail(SPAROA_ERR_INVALID_ARG, "split reduce: mixed dtypes");
    // 16-byte vectors need N % 8 == 0 and 16-byte aligned rows of bias / residual / y
    const int64_t items = r.N % 8 == 0 ? r.M * r.N / 8 : r.M * r.N;
    int64_t blocks = cdiv(items, 256);
    if (blocks > 2048) blocks = 2048;
    g.wg_begin[j] = (int)wg;
    g.partial[j] = r.partial;
    g.split[j] = r.split;
    g.M[j] = r.M;
    g.N[j] = r.N;
    g.bias[j] = static_cast<const char *>(r.bias);
    g.residual[j] = static_cast<const char *>(r.residual);
    g.act[j] = (int)r.act;
    g.y[j] = static_cast<char *>(r.y);
    g.om_counts[j] = r.om_counts;
    g.om_mask[j] = r.om_mask;
    g.om_words[j] = r.om_words;
    if (r.om_counts && (elem_size(r.dt) != 2 || r.N % 8 != 0))
      return fail(SPAROA_ERR_UNSUPPORTED, "split reduce: output measurement needs 16-bit, N % 8 == 0");
    wg += blocks;
  }
  g.wg_begin[n] = (int)wg;
  switch (jobs[0].dt) {
    case SPAROA_BF16:
      hipLaunchKernelGGL(split_reduce_group<SPAROA_BF16>, dim3((unsigned)wg), dim3(256), 0, stream, g);
      break;
    case SPAROA_F16:
      hipLaunchKernelGGL(split_reduce_group<SPAROA_F16>, dim3((unsigned)wg), dim3(256), 0, stream, g);
      break;
    case SPAROA_F32:
      hipLaunchKernelGGL(split_reduce_group<SPAROA_F32>, dim3((unsigned)wg), dim3(256), 0, stream, g);
      break;
  }
  SPAROA_LAUNCH_CHECK("split_reduce_group");
  return SPAROA_OK;
}

sparoa_status launch_split_reduce(const SplitReduceJob &job, hipStream_t stream) {
  return launch_split_reduce_group(&job, 1, stream);
}

namespace {
// LDS of the direct small-channel kernel: raw input rows, weights (each
// rounded up to whole 16-byte vectors) and the padded patch.
int64_t small_c_raw_elems(const sparoa_conv_desc &d) { return cdiv(d.kh * d.w * d.c_in, 8) * 8; }
int64_t small_c_w_elems(const sparoa_conv_desc &d) {
  return cdiv(d.c_out * d.kh * d.kw * d.c_in, 8) * 8;
}
// LDS layout: patch [kh][PW + 1][4] | region: weights and raw rows, later the
// fp32 output tile [16 * ceil(Wo / 16)][Cout + 4]
int64_t small_c_region_off(const sparoa_conv_desc &d) {
  const Shape s = shape_of(d);
  return cdiv(d.kh * (d.sw * (s.wo - 1) + d.kw + 1) * 8, 16) * 16;
}
int64_t small_c_lds_bytes(const sparoa_conv_desc &d) {
  const Shape s = shape_of(d);
  const int64_t staged = 2 * (small_c_raw_elems(d) + small_c_w_elems(d));
  const int64_t tile = 16 * cdiv(s.wo, 16) * (d.c_out + 4) * 4;
  return small_c_region_off(d) + (staged > tile ? staged : tile);
}

// Shapes the direct small-channel kernel serves (image stems).
bool small_c_eligible(const sparoa_conv_desc &d) {
  if (d.dtype == SPAROA_F32 || d.groups != 1 || d.dh != 1 || d.dw != 1) return false;
  if (d.c_in > 4 || d.kw > 8 || d.kh > 32) return false;
  if (!(d.c_out == 16 || d.c_out == 32 || d.c_out == 64)) return false;
  const Shape s = shape_of(d);
  if (s.wo > 16 * kScMaxRB || d.n * s.ho >= ((int64_t)1 << 31)) return false;
  if (cdiv(d.kh * ((d.kw + 1) / 2), 4) > kScMaxKSteps) return false;
  return small_c_lds_bytes(d) <= kScPatchBytes;
}

sparoa_status launch_small_c(const sparoa_conv_desc &d, const void *x, const void *w,
                             const void *bias, const void *residual, sparoa_act act, void *y,
                             bool skip, uint64_t *executed, hipStream_t stream,
                             const DeviceRoute *route, const OutMeasure *om) {
  if (om && om->mask)
    return fail(SPAROA_ERR_UNSUPPORTED, "small-channel conv: fused measurement is counts-only");
  const Shape s = shape_of(d);
  SmallCArgs a;
  a.x = static_cast<const char *>(x);
  a.w = static_cast<const char *>(w);
  a.bias = static_cast<const char *>(bias);
  a.residual = static_cast<const char *>(residual);
  a.y = static_cast<char *>(y);
  a.executed = reinterpret_cast<unsigned long long *>(skip ? executed : nullptr);
  a.N = (int)d.n; a.H = (int)d.h; a.W = (int)d.w; a.C = (int)d.c_in;
  a.Ho = (int)s.ho; a.Wo = (int)s.wo; a.Cout = (int)d.c_out;
  a.kh = (int)d.kh; a.kw = (int)d.kw; a.sh = (int)d.sh; a.sw = (int)d.sw;
  a.ph = (int)d.ph; a.pw = (int)d.pw;
  a.PW = (int)(d.sw * (s.wo - 1) + d.kw);
  a.PWP = a.PW + 1;
  a.bpr = (int)((d.kw + 1) / 2);
  a.ksteps = (int)cdiv(d.kh * a.bpr, 4);
  a.raw_elems = (int)small_c_raw_elems(d);
  a.w_elems = (int)small_c_w_elems(d);
  a.c_w = (int)(d.c_out * d.kh * d.kw * d.c_in);
  // whole vectors: each input row and the weight tensor a multiple of 8 elements
  a.vec = (d.w * d.c_in) % 8 == 0 && (d.c_out * d.kh * d.kw * d.c_in) % 8 == 0;
  a.inv_bpr = 1.0f / (float)a.bpr;
  a.inv_rv = a.vec ? 1.0f / (float)(d.w * d.c_in / 8) : 0.0f;
  a.inv_rowe = 1.0f / (float)(d.w * d.c_in);
  a.region_off = (int)small_c_region_off(d);
  a.act = act;
  a.mode = route && route->counts ? 2 : (skip ? 1 : 0);
  a.route = route ? *route : DeviceRoute{nullptr, 0.0, 0, 0, nullptr};
  a.om_counts = om ? om->counts : nullptr;
  a.om_words = om ? om->words : nullptr;
  const dim3 grid((unsigned)(d.n * s.ho));
  const unsigned lds = (unsigned)small_c_lds_bytes(d);   // <= kScPatchBytes (eligibility)
  switch (a.ksteps) {
#define SPAROA_SC(K)                                                                         \
  case K:                                                                                  \
    if (d.dtype == SPAROA_BF16)                                                            \
      hipLaunchKernelGGL((conv_small_c_kernel<SPAROA_BF16, K>), grid, dim3(256), lds, stream, a); \
    else                                                                                   \
      hipLaunchKernelGGL((conv_small_c_kernel<SPAROA_F16, K>), grid, dim3(256), lds, stream, a);  \
    break;
    SPAROA_SC(1) SPAROA_SC(2) SPAROA_SC(3) SPAROA_SC(4)
    SPAROA_SC(5) SPAROA_SC(6) SPAROA_SC(7) SPAROA_SC(8)
#undef SPAROA_SC
    default: return fail(SPAROA_ERR_UNSUPPORTED, "small-channel conv: k-steps");
  }
  SPAROA_LAUNCH_CHECK("conv_small_c_kernel");
  return SPAROA_OK;
}

// The second-generation kernel takes 16-bit convs whose channel count is a
// multiple of its 64-wide K chunk.
bool ig_eligible(const sparoa_conv_desc &d) {
  // 32-bit byte offsets into x and w; pixel indices below 2^24 (float divmod)
  if (d.n * d.h * d.w * d.c_in >= ((int64_t)1 << 30)) return false;
  if (shape_of(d).M >= ((int64_t)1 << 24) || d.kw > 32 || d.kh > 32) return false;
  if (d.c_out * d.kh * d.kw * d.c_in >= ((int64_t)1 << 30)) return false;
  // C_in a multiple of 8 (16-byte vectors); a tap's last chunk may be
  // partial (its channels past C_in read zero), from 48 channels up (below,
  // most of a chunk would be padding)
  return d.dtype != SPAROA_F32 && d.groups == 1 &&
         (d.c_in % kBK2 == 0 || (d.c_in % 8 == 0 && d.c_in >= 48)) &&
         d.kh * d.kw * cdiv(d.c_in, kBK2) <= kMaxChunks2 &&
         d.kh * d.kw * (d.c_in / 8) <= (int64_t)kMaxVecWords * 32;
}

// Tile of the second-generation kernel: the largest tile that still gives
// every CU a work-group, else the smallest with split-K.
GemmTileChoice ig_choose(const Shape &s, int64_t c_in) {
  auto tiles = [&](int bm, int bn) { return cdiv(s.M, bm) * cdiv(s.N, bn); };
  GemmTileChoice t;
  t.kchunk = kBK2;
  const bool one_tap = s.K == c_in;  // 1 x 1 kernel: a plain GEMM over channels
  // 128 x 64 (waves of 64 x 32, two work-groups per CU) wherever it fills
  // the chip: it beat 128 x 128 (one work-group per CU) by 10 - 25% on 3x3
  // convs at N = 32 (638 vs 506 TFLOP/s at 256 channels, 56 x 56)
  // 128 x 128 (waves of 64 x 64: half the LDS reads per MFMA, two
  // work-groups per CU) where it still gives each CU several tiles: 19-23 %
  // faster on 3x3 convs with 256-512 channels at 56 x 56, N = 32; with fewer
  // tiles the chip runs part-empty and 128 x 64 wins
  // 128 x 256 (eight waves of 64 x 64, one work-group per CU) for 1 x 1
  // kernels with enough tiles: each A row is gathered once per 256 output
  // channels instead of 128; 7 - 13 % faster on 1 x 1 convs and GEMMs with
  // N >= 1024 (FFN 2048 x 768 -> 3072: 28.2 -> 25.8 us), 2 - 9 % slower on
  // 3 x 3 convs with 256-512 channels, which keep 128 x 128
  // (partial chunks, C_in % 64 != 0: 128 x 64 or 64 x 64 only)
  const bool whole = c_in % t.kchunk == 0;
  if (whole && one_tap && s.N % 256 == 0 && tiles(128, 256) >= 192) {
    t.cfg = kIg128x256; t.bm = 128; t.bn = 256;
  } else if (whole && s.N % 128 == 0 && tiles(128, 128) >= 384) {
    t.cfg = kIg128x128; t.bm = 128; t.bn = 128;
  } else if (tiles(128, 64) >= 240) {
    t.cfg = kIg128x64; t.bm = 128; t.bn = 64;
  } else {
    t.cfg = kIg64x64; t.bm = 64; t.bn = 64;
  }
  // chunks: whole or partial 64-channel blocks of each tap
  const int64_t tl = tiles(t.bm, t.bn), nchunks = (s.K / c_in) * cdiv(c_in, t.kchunk);
  int64_t split = 1;
  if (tl < 192) {
    // about one work-group per CU: more splits cost more partial traffic than
    // they gain (FC 64 x 4096 x 4096: split 4 15.1 us, split 8 17.8 us)
    split = cdiv(256, tl);
    if (split > 8) split = 8;
    if (split > nchunks / 4) split = nchunks / 4;
    if (split < 1) split = 1;
    // the reduction is a launch of its own (about 6 us on small outputs):
    // split only where the chunks it takes off a tile's walk (about 0.3 us
    // each on these under-filled grids) are worth more
    if (split > 1 && nchunks * (split - 1) < 20 * split) split = 1;
  }
  t.split_k = (int)split;
  return t;
}
}  // namespace

bool gemm_skip_supported(const sparoa_conv_desc &d) {
  const Shape s = shape_of(d);
  if (ig_eligible(d) || small_c_eligible(d)) return true;
  const int64_t bits = d.kh * d.kw * cdiv(d.c_in, 8);
  return cdiv(s.K, kBK) <= kMaxChunks && bits <= (int64_t)kMaxVecWords * 32;
}


bool conv_skip_reads_mask(const sparoa_conv_desc &d, sparoa_path path) {
  if (!(path & 1) || d.groups != 1 || !gemm_skip_supported(d)) return false;
  const GemmTileChoice t = gemm_choose(d, path);
  return !(t.pointwise || t.small_c);
}

GemmTileChoice gemm_choose(const sparoa_conv_desc &d, sparoa_path path) {
  const Shape s = shape_of(d);
  GemmTileChoice t;
  if ((path & 2) && pw_eligible(d)) {   // bandwidth path, 1x1: weights in LDS, x read once
    t.cfg = 0;
    t.bm = 16;      // skip unit: 16-pixel x 32-channel activation blocks
    t.bn = 16;
    t.kchunk = 32;
    t.split_k = 1;
    t.pointwise = true;
    return t;
  }
  if (ig_eligible(d)) return ig_choose(s, d.c_in);
  if (small_c_eligible(d)) {   // one output row per work-group, 16-pixel row blocks
    t.cfg = 0;
    t.bm = 16;
    t.bn = 16;
    t.kchunk = 32;
    t.split_k = 1;
    t.small_c = true;
    return t;
  }
  t.cfg = 0;
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

bool gemm_fuses_out_measure(const sparoa_conv_desc &d, sparoa_path path, bool bitmap) {
  const GemmTileChoice t = gemm_choose(d, path);
  // the pointwise kernel measures whole tiles of one weight slice
  if (t.pointwise) return pw_fuses_out_measure(d);
  // the small-channel kernel counts (no bitmap)
  if (t.small_c) return !bitmap;
  // the second-generation kernel (64-column tiles) writes whole bitmap bytes
  // when C_out % 64 == 0; its split-K reduction measures 16-byte vectors (a
  // wave's 64 vectors are two whole bitmap words), any C_out % 8 == 0
  if (t.cfg == 0 || elem_size(d.dtype) != 2) return false;
  if (d.c_out % 64 == 0) return true;
  // the K splits the launch will take (as launch_gemm_conv counts them)
  const int64_t nchunks = d.kh * d.kw * cdiv(d.c_in, t.kchunk);
  const int64_t gz = cdiv(nchunks, cdiv(nchunks, t.split_k));
  return gz > 1 && d.c_out % 8 == 0;
}

size_t gemm_workspace_required(const sparoa_conv_desc &d, sparoa_path path) {
  const GemmTileChoice t = gemm_choose(d, path);
  if (t.split_k <= 1) return 0;
  const Shape s = shape_of(d);
  return (size_t)t.split_k * (size_t)s.M * (size_t)s.N * sizeof(float);
}


sparoa_status launch_gemm_conv(const sparoa_conv_desc &d, sparoa_path path, const void *x,
                               const void *w, const void *bias, const void *residual,
                               sparoa_act act, const uint32_t *mask, void *y, void *ws,
                               size_t ws_bytes, uint64_t *executed, hipStream_t stream,
                               const DeviceRoute *route, SplitReduceJob *defer,
                               const OutMeasure *om) {
  const Shape s = shape_of(d);
  const GemmTileChoice t = gemm_choose(d, path);
  if (om && !gemm_fuses_out_measure(d, path, om->mask != nullptr))
    return fail(SPAROA_ERR_UNSUPPORTED, "GEMM: no fused output measurement for this shape");
  const int epv = d.dtype == SPAROA_F32 ? 4 : 8;
  const bool vec = d.c_in % epv == 0;
  // the skip form: x's bitmap given, or a skip path on a kernel that tests x
  // itself (the pointwise and small-channel kernels read no bitmap)
  const bool skip = mask != nullptr || ((path & 1) && (t.pointwise || t.small_c));
  // (the second-generation kernel's chunks are per tap: whole or partial
  // 64-channel blocks)
  const int64_t nchunks =
      t.cfg ? d.kh * d.kw * cdiv(d.c_in, t.kchunk) : cdiv(s.K, t.kchunk);
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
  a.x_bytes = d.n * d.h * d.w * d.c_in * elem_size(d.dtype);
  a.w_bytes = s.N * s.K * elem_size(d.dtype);
  a.inv_wo = 1.0f / (float)s.wo;
  a.inv_ho = 1.0f / (float)s.ho;
  a.nchunks = nchunks;
  a.kh32 = (int)d.kh;
  a.inv_kw = 1.0f / (float)d.kw;
  a.inv_dh = 1.0f / (float)d.dh;
  a.inv_dw = 1.0f / (float)d.dw;
  a.split = t.split_k;
  a.chunks_per_split = cdiv(nchunks, t.split_k);
  a.act = act;
  a.route = route ? *route : DeviceRoute{nullptr, 0.0, 0, 0, nullptr};
  const int64_t gz = cdiv(nchunks, a.chunks_per_split);
  a.split = (int)gz;
  // the epilogue measures y when it writes y; with split-K the reduction does
  a.om_counts = om && gz == 1 ? om->counts : nullptr;
  a.om_mask = om && gz == 1 ? om->mask : nullptr;
  // grouped count commit when the caller gives the words
  unsigned long long *om_words = om ? om->words : nullptr;
  a.om_words = gz == 1 ? om_words : nullptr;
  if (gz > 1 && ws_bytes < (size_t)gz * s.M * s.N * sizeof(float))
    return fail(SPAROA_ERR_WORKSPACE, "GEMM split-K workspace too small");

  if (executed) {
    hipLaunchKernelGGL(set_u64, dim3(1), dim3(1), 0, stream,
                       reinterpret_cast<unsigned long long *>(executed), 0ull);
    SPAROA_LAUNCH_CHECK("set_u64");
  }
  if (t.small_c) {
    if (defer) *defer = SplitReduceJob{d.dtype, nullptr, 0, s.M, s.N, bias, residual, act, y,
                                       nullptr, nullptr, nullptr};
    return launch_small_c(d, x, w, bias, residual, act, y, skip, executed, stream, route, om);
  }
  if (t.pointwise) {
    if (defer) *defer = SplitReduceJob{d.dtype, nullptr, 0, s.M, s.N, bias, residual, act, y,
                                       nullptr, nullptr, nullptr};
    return launch_pointwise(d, x, w, bias, residual, act, y, skip, executed, stream, route, om);
  }
  dim3 grid((unsigned)cdiv(s.M, t.bm), (unsigned)cdiv(s.N, t.bn), (unsigned)gz);
  if (t.cfg) {
    const int64_t ntn = cdiv(s.N, t.bn), ntmn = cdiv(s.M, t.bm) * ntn;
    if (ntmn * gz >= (int64_t)1 << 24)
      return fail(SPAROA_ERR_UNSUPPORTED, "GEMM: 2^24 tiles or more");
    grid = dim3((unsigned)(ntmn * gz));
    a.ntn32 = (int)ntn;
    a.ntmn32 = (int)ntmn;
    a.inv_ntn = 1.0f / (float)ntn;
    a.inv_ntmn = 1.0f / (float)ntmn;
    a.cpt32 = (int)cdiv(d.c_in, t.kchunk);
    a.inv_cpt = 1.0f / (float)a.cpt32;
  }
  bool ok = false;
  const bool part = d.c_in % kBK2 != 0;   // a tap's last chunk is partial
  if (t.cfg) {
    switch (d.dtype) {
      case SPAROA_BF16:
        ok = skip ? dispatch_ig<SPAROA_BF16, true>(t.cfg, t.kchunk, part, grid, stream, a)
                  : dispatch_ig<SPAROA_BF16, false>(t.cfg, t.kchunk, part, grid, stream, a);
        break;
      case SPAROA_F16:
        ok = skip ? dispatch_ig<SPAROA_F16, true>(t.cfg, t.kchunk, part, grid, stream, a)
                  : dispatch_ig<SPAROA_F16, false>(t.cfg, t.kchunk, part, grid, stream, a);
        break;
      default: break;
    }
  } else switch (d.dtype) {
    case SPAROA_BF16: ok = dispatch<SPAROA_BF16>(t.bm, t.bn, vec, skip, grid, stream, a); break;
    case SPAROA_F16: ok = dispatch<SPAROA_F16>(t.bm, t.bn, vec, skip, grid, stream, a); break;
    case SPAROA_F32: ok = dispatch<SPAROA_F32>(t.bm, t.bn, vec, skip, grid, stream, a); break;
  }
  if (!ok) return fail(SPAROA_ERR_UNSUPPORTED, "GEMM tile shape");
  SPAROA_LAUNCH_CHECK("gemm_kernel");
  const SplitReduceJob job{d.dtype, a.partial, gz > 1 ? (int)gz : 0, s.M, s.N, bias, residual,
                           act, y, om && gz > 1 ? om->counts : nullptr,
                           om && gz > 1 ? om->mask : nullptr, gz > 1 ? om_words : nullptr};
  if (defer) {
    *defer = job;
    return SPAROA_OK;
  }
  if (gz > 1) return launch_split_reduce(job, stream);
  return SPAROA_OK;
}

}  // namespace sparoa
