// Weight-streaming FC for small m (m <= 64): the bandwidth path of the
// light quadrants (SparOA Section 2.2) and its zero-skipping form (Section
// 2.1).  At m <= 64 an FC has intensity <= ~62 FLOP/byte, far below the
// MI355X ridge point, so its time is the time to stream the weights once.
//
// Weights are packed once (sparoa_fc_pack_weights) into 64-column panels,
// k-major inside a panel: Wp[p][k][0..63] = w[64p + 0..63][k] (zero past n).
// One input column k then owns one contiguous 128-byte (16-bit) row of every
// panel, so skipping a column that is zero in all m rows skips whole cache
// lines of weights: the skip granularity is one column, the HBM saving is
// exact.
//
// Work-group = 256 threads; it owns one panel and a range of k (split-K).
// It first lists the k of its range that it will visit (all of them, or --
// skip variant -- the nonzero columns read from the column bitmap, compacted
// with ballot + popcount), then walks that list 64 entries at a time: the 64
// weight rows are loaded with 16-byte coalesced loads and written transposed
// into LDS, the matching x[:, k] values are gathered into LDS, and each wave
// runs MFMA 16x16x32 over its 16 output columns for all m (padded to 16).
// Partial sums of a split go to the workspace; a reduction kernel adds them
// in split order and applies bias and activation.
#include "common.h"
#include "dtype.h"

namespace sparoa {
namespace {

constexpr int kThreads = 256;
constexpr int kPanel = 64;     // output columns per panel
constexpr int kCh = 64;        // list entries per step
constexpr int kMaxRange = 4096;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

struct FcBwArgs {
  const char *x;
  const char *wp;
  const char *bias;
  const char *residual;
  char *y;
  float *partial;
  const uint32_t *mask;
  unsigned long long *executed;
  int64_t M, K, N, krange;
  int splits;
  int act;
};

template <int DT, int MT, bool SKIP>
__global__ __launch_bounds__(kThreads) void fc_bw_kernel(FcBwArgs a) {
  using E = Elem<DT>;
  using raw = typename E::raw;
  static_assert(E::size == 2, "16-bit types only");
  constexpr int ROWB = (kCh + 8) * 2;  // LDS row stride, bytes
  __shared__ __attribute__((aligned(16))) char As[2][MT * 16 * ROWB];
  __shared__ __attribute__((aligned(16))) char Bt[2][kPanel * ROWB];
  __shared__ unsigned short list[SKIP ? kMaxRange : 1];
  __shared__ int list_len;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t p = blockIdx.x;
  const int64_t kb = (int64_t)blockIdx.y * a.krange;
  const int64_t ke = min(kb + a.krange, a.K);

  int count = (int)(ke - kb);
  if constexpr (SKIP) {
    if (wave == 0) {
      int total = 0;
      for (int64_t base = kb; base < ke; base += 64) {
        const int64_t k = base + lane;
        const bool nz = k < ke && ((a.mask[k >> 5] >> (k & 31)) & 1u);
        const uint64_t bal = __ballot(nz);
        if (nz) list[total + __popcll(bal & ((1ull << lane) - 1ull))] = (unsigned short)(k - kb);
        total += __popcll(bal);
      }
      if (lane == 0) {
        list_len = total;
        if (a.executed && p == 0 && total) atomicAdd(a.executed, (unsigned long long)total);
      }
    }
    __syncthreads();
    count = list_len;
  }

  uint4 rw[2];
  raw rx[MT * 4];
  auto entry_k = [&](int e) -> int64_t {  // k of list entry e, or -1 past the end
    if (e >= count) return -1;
    return SKIP ? kb + (int64_t)list[e] : kb + e;
  };
  auto load_step = [&](int s0) {
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int v = tid + kThreads * u;
      const int64_t k = entry_k(s0 + v / 8);
      rw[u] = k >= 0 ? *reinterpret_cast<const uint4 *>(
                           a.wp + ((p * a.K + k) * kPanel + 8 * (v % 8)) * 2)
                     : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int u = 0; u < MT * 4; ++u) {
      const int v = tid + kThreads * u;
      const int m = v / kCh;
      const int64_t k = entry_k(s0 + v % kCh);
      rx[u] = (m < a.M && k >= 0) ? reinterpret_cast<const raw *>(a.x)[m * a.K + k] : (raw)0;
    }
  };
  auto store_step = [&](int buf) {
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int v = tid + kThreads * u;
      const int e = v / 8, c0 = 8 * (v % 8);
      const raw *h = reinterpret_cast<const raw *>(&rw[u]);
#pragma unroll
      for (int i = 0; i < 8; ++i)
        *reinterpret_cast<raw *>(&Bt[buf][(c0 + i) * ROWB + 2 * e]) = h[i];
    }
#pragma unroll
    for (int u = 0; u < MT * 4; ++u) {
      const int v = tid + kThreads * u;
      *reinterpret_cast<raw *>(&As[buf][(v / kCh) * ROWB + 2 * (v % kCh)]) = rx[u];
    }
  };

  f32x4 acc[MT];
#pragma unroll
  for (int i = 0; i < MT; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int g = lane >> 4, rl = lane & 15;
  const int steps = (count + kCh - 1) / kCh;
  if (steps > 0) {
    load_step(0);
    store_step(0);
    __syncthreads();
    for (int st = 0; st < steps; ++st) {
      const int buf = st & 1;
      const bool more = st + 1 < steps;
      if (more) load_step((st + 1) * kCh);
      const char *brow = &Bt[buf][(16 * wave + rl) * ROWB];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          const char *arow = &As[buf][(mt * 16 + rl) * ROWB];
          if constexpr (DT == SPAROA_BF16) {
            const bf16x8 av = *reinterpret_cast<const bf16x8 *>(arow + 64 * h + 16 * g);
            const bf16x8 bv = *reinterpret_cast<const bf16x8 *>(brow + 64 * h + 16 * g);
            acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bv, acc[mt], 0, 0, 0);
          } else {
            const f16x8 av = *reinterpret_cast<const f16x8 *>(arow + 64 * h + 16 * g);
            const f16x8 bv = *reinterpret_cast<const f16x8 *>(brow + 64 * h + 16 * g);
            acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(av, bv, acc[mt], 0, 0, 0);
          }
        }
      }
      if (more) store_step(buf ^ 1);
      __syncthreads();
    }
  }

  const int64_t col = p * kPanel + 16 * wave + rl;
  if (col >= a.N) return;
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int64_t row = mt * 16 + 4 * g + v;
      if (row >= a.M) continue;
      if (a.splits > 1) {
        a.partial[((int64_t)blockIdx.y * a.M + row) * a.N + col] = acc[mt][v];
      } else {
        float o = acc[mt][v];
        if (a.bias) o += E::to_f32(reinterpret_cast<const raw *>(a.bias)[col]);
        if (a.residual) o += E::to_f32(reinterpret_cast<const raw *>(a.residual)[row * a.N + col]);
        reinterpret_cast<raw *>(a.y)[row * a.N + col] = E::from_f32(apply_act(o, a.act));
      }
    }
}

// Packs w[n][k] into 64-column k-major panels, zero-filled past n.
template <typename raw>
__global__ void fc_pack_kernel(const raw *__restrict__ w, raw *__restrict__ wp, int64_t K,
                               int64_t N, int64_t panels) {
  const int64_t total = panels * K * (kPanel / 8);
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t q = i % (kPanel / 8), k = (i / (kPanel / 8)) % K, p = i / (kPanel / 8) / K;
    raw v[8];
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const int64_t n = p * kPanel + 8 * q + t;
      v[t] = n < N ? w[n * K + k] : (raw)0;
    }
    uint4 out;
    __builtin_memcpy(&out, v, 16);
    *reinterpret_cast<uint4 *>(wp + (p * K + k) * kPanel + 8 * q) = out;
  }
}

struct BwPlan {
  int64_t panels, krange;
  int splits;
};

BwPlan plan(const sparoa_fc_desc &d) {
  BwPlan pl;
  pl.panels = cdiv(d.n, kPanel);
  int64_t ks = cdiv(1024, pl.panels);
  if (ks > 16) ks = 16;
  if (d.m > 16 && ks > 8) ks = 8;
  if (ks < 1) ks = 1;
  int64_t kr = cdiv(cdiv(d.k, ks), 64) * 64;
  if (kr > kMaxRange) kr = kMaxRange;
  pl.krange = kr;
  pl.splits = (int)cdiv(d.k, kr);
  return pl;
}

template <int DT, bool SKIP>
bool launch_mt(int mt, dim3 grid, hipStream_t st, const FcBwArgs &a) {
  switch (mt) {
    case 1: hipLaunchKernelGGL((fc_bw_kernel<DT, 1, SKIP>), grid, dim3(kThreads), 0, st, a); break;
    case 2: hipLaunchKernelGGL((fc_bw_kernel<DT, 2, SKIP>), grid, dim3(kThreads), 0, st, a); break;
    case 3: hipLaunchKernelGGL((fc_bw_kernel<DT, 3, SKIP>), grid, dim3(kThreads), 0, st, a); break;
    case 4: hipLaunchKernelGGL((fc_bw_kernel<DT, 4, SKIP>), grid, dim3(kThreads), 0, st, a); break;
    default: return false;
  }
  return true;
}

__global__ void zero_u64(unsigned long long *p) { *p = 0ull; }

}  // namespace

size_t fc_packed_bytes(const sparoa_fc_desc &d) {
  return (size_t)cdiv(d.n, kPanel) * kPanel * (size_t)d.k * (size_t)elem_size(d.dtype);
}

size_t fc_bw_workspace(const sparoa_fc_desc &d, sparoa_path) {
  const BwPlan pl = plan(d);
  return pl.splits > 1 ? (size_t)pl.splits * d.m * d.n * sizeof(float) : 0;
}

sparoa_status launch_fc_pack(const sparoa_fc_desc &d, const void *w_nk, void *w_packed,
                             hipStream_t stream) {
  if (d.dtype == SPAROA_F32) return fail(SPAROA_ERR_UNSUPPORTED, "fc bandwidth path: fp32");
  const int64_t panels = cdiv(d.n, kPanel);
  const int64_t total = panels * d.k * (kPanel / 8);
  int64_t blocks = cdiv(total, 256);
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL(fc_pack_kernel<uint16_t>, dim3((unsigned)blocks), dim3(256), 0, stream,
                     static_cast<const uint16_t *>(w_nk), static_cast<uint16_t *>(w_packed), d.k,
                     d.n, panels);
  SPAROA_LAUNCH_CHECK("fc_pack_kernel");
  return SPAROA_OK;
}

sparoa_status launch_fc_bw(const sparoa_fc_desc &d, sparoa_path path, const void *x,
                           const void *w_packed, const void *bias, const void *residual,
                           sparoa_act act,
                           const uint32_t *mask, void *y, void *ws, size_t ws_bytes,
                           uint64_t *executed, hipStream_t stream) {
  if (d.dtype == SPAROA_F32) return fail(SPAROA_ERR_UNSUPPORTED, "fc bandwidth path: fp32");
  if (d.m > 64) return fail(SPAROA_ERR_UNSUPPORTED, "fc bandwidth path: m > 64");
  const BwPlan pl = plan(d);
  if (pl.splits > 1 && ws_bytes < fc_bw_workspace(d, path))
    return fail(SPAROA_ERR_WORKSPACE, "fc bandwidth path: workspace too small");
  const bool skip = mask != nullptr;
  FcBwArgs a;
  a.x = static_cast<const char *>(x);
  a.wp = static_cast<const char *>(w_packed);
  a.bias = static_cast<const char *>(bias);
  a.residual = static_cast<const char *>(residual);
  a.y = static_cast<char *>(y);
  a.partial = static_cast<float *>(ws);
  a.mask = mask;
  a.executed = reinterpret_cast<unsigned long long *>(skip ? executed : nullptr);
  a.M = d.m; a.K = d.k; a.N = d.n; a.krange = pl.krange;
  a.splits = pl.splits;
  a.act = act;
  if (a.executed) {
    hipLaunchKernelGGL(zero_u64, dim3(1), dim3(1), 0, stream, a.executed);
    SPAROA_LAUNCH_CHECK("zero_u64");
  }
  const int mt = (int)cdiv(d.m, 16);
  dim3 grid((unsigned)pl.panels, (unsigned)pl.splits);
  bool ok;
  if (d.dtype == SPAROA_BF16)
    ok = skip ? launch_mt<SPAROA_BF16, true>(mt, grid, stream, a)
              : launch_mt<SPAROA_BF16, false>(mt, grid, stream, a);
  else
    ok = skip ? launch_mt<SPAROA_F16, true>(mt, grid, stream, a)
              : launch_mt<SPAROA_F16, false>(mt, grid, stream, a);
  if (!ok) return fail(SPAROA_ERR_UNSUPPORTED, "fc bandwidth path: m");
  SPAROA_LAUNCH_CHECK("fc_bw_kernel");
  if (pl.splits > 1)
    return launch_split_reduce(d.dtype, a.partial, pl.splits, d.m, d.n, bias, residual, act, y,
                               stream);
  return SPAROA_OK;
}

}  // namespace sparoa
