// Weight-streaming FC for small m (m <= 64): the bandwidth path of the
// light quadrants (SparOA Section 2.2) and its zero-skipping form (Section
// 2.1).  At m <= 64 an FC has intensity <= ~62 FLOP/byte, far below the
// MI355X ridge point, so its time is the time to stream the weights once.
//
// Weights are packed once (sparoa_fc_pack_weights) into 16-column panels,
// k-major inside a panel: Wp[p][k][0..15] = w[16p + 0..15][k] (zero past n).
// A panel is one contiguous stream of k rows of 32 bytes; an input column k
// that is zero in all m rows owns exactly one such row per panel, so the
// skip variant drops it from the stream (skip granularity: one column).
//
// One work-group streams one panel over all of K (no cross-work-group
// reduction, no device-scope fences).  Its waves (16 for m <= 32, else 8)
// split K into contiguous slices.  A wave walks its slice -- all of it, or,
// in the skip variant, the nonzero columns listed from the column bitmap by a
// popcount prefix sum -- in chunks of 32 entries, keeping 4 to 8 chunks of
// weight rows (16-byte loads, two lanes per row) and input values
// in flight in registers.  Dense input rows are read with 16-byte loads; the
// skip variant gathers input pairs spread over all lanes (one 4-byte load
// when the pair's columns are adjacent).  Each chunk goes
// through a wave-private LDS tile (weights transposed on the way in) into
// v_mfma_f32_16x16x32 over all m (padded to 16) and the panel's 16 columns.
// The waves' fp32 partials are added in wave order through LDS
// (deterministic), then bias, residual, activation and the cast to dtype.
//
// Self-measuring form (measure -> route -> execute in one launch): every
// work-group reads all of x anyway, so before streaming it counts the zeros
// of x and builds the column bitmap in LDS (16-byte loads, a lane per group
// of 8 columns over all rows), takes the route decision from those counts
// with the same arithmetic as the host route, and uses the LDS bitmap for its
// column list; work-group 0 also stores the counts, the bitmap and the path.
#include "common.h"
#include "dtype.h"

namespace sparoa {
namespace {

constexpr int kPanel = 16;          // output columns per panel / work-group
constexpr int kCh = 32;             // entries per chunk = one MFMA k-step
constexpr int kMaxWaveK = 1024;     // K values per wave slice
constexpr int kRowB = (kCh + 8) * 2;  // LDS row stride in bytes (80: conflict-free b128 reads)

// Waves per work-group and chunks in flight per wave for MT row tiles.
template <int MT>
struct Shape {
  static constexpr int waves = MT <= 2 ? 16 : 8;
  static constexpr int depth = MT == 1 ? 8 : (MT == 2 ? 5 : 4);  // within the VGPR budget
};

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

struct FcBwArgs {
  const char *x;
  const char *wp;
  const char *bias;
  const char *residual;
  char *y;
  const uint32_t *mask;
  unsigned long long *executed;
  int64_t M, K, N, slice;
  int act;
  int xvec;
  DeviceRoute route;
  sparoa_counts *mcounts;  // self-measuring form: outputs of the measurement
  uint32_t *mmask;
};

constexpr int kMaxColWords = kMaxWaveK * 16 / 32;  // bitmap words for the largest K

// LDS of one wave: transposed weight tile [16 cols][32 entries], input tile
// [16*MT rows][32 entries], and the wave's list of columns.
template <int MT, bool SKIP>
struct WaveLds {
  char wt[kPanel * kRowB];
  char xs[MT * 16 * kRowB];
  unsigned short list[SKIP ? kMaxWaveK : 8];
};

template <int DT, int MT, bool SKIP, bool XVEC, bool MEASURE = false>
__global__ __launch_bounds__(64 * Shape<MT>::waves) void fc_bw_kernel(FcBwArgs a) {
  static_assert(!MEASURE || SKIP, "the self-measuring form may skip");
  constexpr int NW = Shape<MT>::waves;
  constexpr int kDepth = Shape<MT>::depth;
  constexpr int kThreads = 64 * NW;
  using E = Elem<DT>;
  using raw = typename E::raw;
  static_assert(E::size == 2, "16-bit types only");
  using Lds = WaveLds<MT, SKIP>;
  // gfx950 addresses 160 KB of LDS per work-group
  static_assert(sizeof(Lds) * NW <= 160 * 1024, "LDS budget");
  static_assert(sizeof(Lds) * NW >= NW * MT * 16 * kPanel * 4, "reduction space");
  __shared__ __attribute__((aligned(16))) char lds_raw[sizeof(Lds) * NW];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  Lds &L = reinterpret_cast<Lds *>(lds_raw)[wave];
  const int64_t p = blockIdx.x;
  const int64_t kb = (int64_t)wave * a.slice;
  const int64_t ke = min(kb + a.slice, a.K);
  const char *wpanel = a.wp + p * a.K * kPanel * 2;

  int count = ke > kb ? (int)(ke - kb) : 0;
  bool use_list = SKIP;
  const uint32_t *colbits = a.mask;
  if constexpr (SKIP) {
    __shared__ uint32_t mbits[MEASURE ? kMaxColWords : 1];
    if constexpr (MEASURE) {
      // Thread t owns column groups t, t + kThreads, ... (8 columns = one
      // bitmap byte; K % 8 == 0): it ORs the group's nonzero flags over all
      // rows (kMR row loads in flight), counts zeros, and stores the byte;
      // bytes past K up to the last whole word are stored as 0.  The waves'
      // sums meet in LDS: one barrier.
      constexpr int kMR = MT == 1 ? 8 : (MT == 2 ? 16 : 32);
      __shared__ unsigned wsum[NW][2];
      const int ng = (int)(a.K / 8);
      const int nbytes = 4 * (int)((a.K + 31) / 32);
      unsigned zeros = 0, ones = 0;
      for (int g = tid; g < nbytes; g += kThreads) {
        uint32_t nzb = 0;
        if (g < ng) {
          const char *px = a.x + (int64_t)g * 16;
          for (int m0 = 0; m0 < a.M; m0 += kMR) {
            // unconditional loads (rows past M re-read row M - 1 and are
            // masked below), so all kMR stay in flight
            uint4 q[kMR];
#pragma unroll
            for (int u = 0; u < kMR; ++u) {
              const int64_t r = min((int64_t)(m0 + u), a.M - 1);
              q[u] = *reinterpret_cast<const uint4 *>(px + r * a.K * 2);
            }
#pragma unroll
            for (int u = 0; u < kMR; ++u) {
              const uint32_t wv[4] = {q[u].x, q[u].y, q[u].z, q[u].w};
              uint32_t b = 0;
#pragma unroll
              for (int h = 0; h < 4; ++h) {
                b |= ((wv[h] & 0x7FFFu) != 0u ? 1u : 0u) << (2 * h);
                b |= ((wv[h] & 0x7FFF0000u) != 0u ? 1u : 0u) << (2 * h + 1);
              }
              const bool valid = m0 + u < a.M;
              zeros += valid ? 8u - (unsigned)__popc(b) : 0u;
              nzb |= valid ? b : 0u;
            }
          }
          ones += (unsigned)__popc(nzb);
        }
        reinterpret_cast<unsigned char *>(mbits)[g] = (unsigned char)nzb;
      }
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) {
        zeros += __shfl_xor(zeros, o, 64);
        ones += __shfl_xor(ones, o, 64);
      }
      if (lane == 0) {
        wsum[wave][0] = zeros;
        wsum[wave][1] = ones;
      }
      __syncthreads();
      zeros = 0;
      ones = 0;
#pragma unroll
      for (int w = 0; w < NW; ++w) {
        zeros += wsum[w][0];
        ones += wsum[w][1];
      }
      const int nwords = nbytes / 4;
      sparoa_counts c;
      c.zeros = zeros;
      c.numel = (uint64_t)a.M * (uint64_t)a.K;
      c.zero_blocks = (uint64_t)a.K - ones;
      c.num_blocks = (uint64_t)a.K;
      use_list = route_skip_counts(c, a.route.sparsity_thr, a.route.mode);
      if (p == 0) {
        for (int i = tid; i < nwords; i += kThreads) a.mmask[i] = mbits[i];
        if (tid == 0) {
          *a.mcounts = c;
          if (a.route.path_out)
            *a.route.path_out = (use_list ? 1u : 0u) | ((uint32_t)a.route.bw_bit << 1);
        }
      }
      colbits = mbits;
    } else if (a.route.counts) {
      use_list = device_route_skip(a.route);
      if (a.route.path_out && p == 0 && tid == 0)
        *a.route.path_out = (use_list ? 1u : 0u) | ((uint32_t)a.route.bw_bit << 1);
    }
  }
  if (SKIP && use_list) {
    // The slice's bitmap words (at most 32: one per lane) are loaded at once;
    // an exclusive prefix sum of their popcounts gives each lane its place
    // in the list, then each lane writes the offsets of its set bits.
    const int nw = (count + 31) / 32;
    uint32_t wv = 0;
    if (lane < nw) {
      wv = colbits[(kb >> 5) + lane];
      const int tail = count - 32 * lane;
      if (tail < 32) wv &= (1u << tail) - 1u;
    }
    const int cnt = __popc(wv);
    int incl = cnt;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int t = __shfl_up(incl, o, 64);
      if (lane >= o) incl += t;
    }
    int pos = incl - cnt;
    while (wv) {
      const int b = __ffs(wv) - 1;
      L.list[pos++] = (unsigned short)(32 * lane + b);
      wv &= wv - 1u;
    }
    const int total = __shfl(incl, 63, 64);
    count = total;
    if (a.executed && p == 0 && lane == 0 && total)
      atomicAdd(a.executed, (unsigned long long)total);
  }
  const int nch = (count + kCh - 1) / kCh;

  // entry -> column k (or -1 past the end of the wave's list)
  auto entry_k = [&](int e) -> int64_t {
    if (e >= count) return -1;
    if (SKIP && use_list) return kb + (int64_t)L.list[e];
    return kb + e;
  };
  // Register staging of one chunk: weight row e = lane / 2, half lane % 2.
  // Input, vector form: (row m, 8 entries) per v = lane + 64 j, one 16-byte
  // load when the 8 columns are contiguous (dense order);
  // pair form (skip order): (row m, entries 2q, 2q + 1) per v = lane + 64 j,
  // one 4-byte load when the two columns are adjacent, else two gathers.
  // Both forms use the same 4 * MT registers.
  const bool vecform = !SKIP || !use_list;
  const bool xvec = XVEC || (SKIP && a.xvec);  // rows 16-byte aligned
  struct Stage {
    uint4 w;
    uint32_t xr[4 * MT];
  };
  auto load = [&](int c, Stage &s) {
    const int64_t k = entry_k(c * kCh + (lane >> 1));
    s.w = k >= 0 ? *reinterpret_cast<const uint4 *>(wpanel + (k * kPanel + 8 * (lane & 1)) * 2)
                 : make_uint4(0, 0, 0, 0);
    if (vecform) {
#pragma unroll
      for (int j = 0; j < MT; ++j) {
        const int v = lane + 64 * j;
        const int m = v >> 2, e0 = c * kCh + 8 * (v & 3);
        uint4 q = make_uint4(0, 0, 0, 0);
        if (m < a.M) {
          if (xvec && e0 + 8 <= count) {
            q = *reinterpret_cast<const uint4 *>(a.x + (m * a.K + kb + e0) * 2);
          } else {
            raw t[8];
#pragma unroll
            for (int i = 0; i < 8; ++i)
              t[i] = e0 + i < count ? reinterpret_cast<const raw *>(a.x)[m * a.K + kb + e0 + i]
                                    : (raw)0;
            __builtin_memcpy(&q, t, 16);
          }
        }
        __builtin_memcpy(&s.xr[4 * j], &q, 16);
      }
    } else {
#pragma unroll
      for (int j = 0; j < 4 * MT; ++j) {
        const int v = lane + 64 * j;
        const int m = v >> 4, e0 = c * kCh + 2 * (v & 15);
        uint32_t pr = 0;
        if (m < a.M) {
          const int64_t k0 = entry_k(e0), k1 = entry_k(e0 + 1);
          const raw *xr = reinterpret_cast<const raw *>(a.x) + m * a.K;
          if (k0 >= 0 && k1 == k0 + 1 && ((m * a.K + k0) & 1) == 0) {  // 4-byte aligned pair
            pr = *reinterpret_cast<const uint32_t *>(xr + k0);
          } else {
            const uint32_t lo = k0 >= 0 ? xr[k0] : 0u, hi = k1 >= 0 ? xr[k1] : 0u;
            pr = lo | (hi << 16);
          }
        }
        s.xr[j] = pr;
      }
    }
  };
  auto stash = [&](const Stage &s) {
    // weights: lane holds columns 8h..8h+7 of entry e; write them transposed
    const int e = lane >> 1, c0 = 8 * (lane & 1);
    raw h[8];
    __builtin_memcpy(h, &s.w, 16);
#pragma unroll
    for (int i = 0; i < 8; ++i) *reinterpret_cast<raw *>(&L.wt[(c0 + i) * kRowB + 2 * e]) = h[i];
    if (vecform) {
#pragma unroll
      for (int j = 0; j < MT; ++j) {
        const int v = lane + 64 * j;
        uint4 q;
        __builtin_memcpy(&q, &s.xr[4 * j], 16);
        *reinterpret_cast<uint4 *>(&L.xs[(v >> 2) * kRowB + 16 * (v & 3)]) = q;
      }
    } else {
#pragma unroll
      for (int j = 0; j < 4 * MT; ++j) {
        const int v = lane + 64 * j;
        *reinterpret_cast<uint32_t *>(&L.xs[(v >> 4) * kRowB + 4 * (v & 15)]) = s.xr[j];
      }
    }
  };

  f32x4 acc[MT];
#pragma unroll
  for (int i = 0; i < MT; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int g = lane >> 4, rl = lane & 15;

  Stage st[kDepth];
#pragma unroll
  for (int j = 0; j < kDepth; ++j)
    if (j < nch) load(j, st[j]);
  for (int c0 = 0; c0 < nch; c0 += kDepth) {
#pragma unroll
    for (int j = 0; j < kDepth; ++j) {
      const int c = c0 + j;
      if (c < nch) {
        // LDS operations of one wave execute in order: the tile written here
        // is the one read below, and the reads finish before the next write.
        stash(st[j]);
        const char *brow = &L.wt[rl * kRowB + 16 * g];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          const char *arow = &L.xs[(mt * 16 + rl) * kRowB + 16 * g];
          if constexpr (DT == SPAROA_BF16)
            acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                *reinterpret_cast<const bf16x8 *>(arow), *reinterpret_cast<const bf16x8 *>(brow),
                acc[mt], 0, 0, 0);
          else
            acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(
                *reinterpret_cast<const f16x8 *>(arow), *reinterpret_cast<const f16x8 *>(brow),
                acc[mt], 0, 0, 0);
        }
        if (c + kDepth < nch) load(c + kDepth, st[j]);
      }
    }
  }

  // Cross-wave reduction in wave order through LDS (reuses the tiles).
  __syncthreads();
  float *red = reinterpret_cast<float *>(lds_raw);  // [wave][16*MT][16]
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int v = 0; v < 4; ++v)
      red[(wave * MT * 16 + mt * 16 + 4 * g + v) * kPanel + rl] = acc[mt][v];
  __syncthreads();
  for (int e = tid; e < MT * 16 * kPanel; e += kThreads) {
    const int64_t row = e / kPanel, col = p * kPanel + e % kPanel;
    if (row >= a.M || col >= a.N) continue;
    float o = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) o += red[w * MT * 16 * kPanel + e];
    if (a.bias) o += E::to_f32(reinterpret_cast<const raw *>(a.bias)[col]);
    if (a.residual) o += E::to_f32(reinterpret_cast<const raw *>(a.residual)[row * a.N + col]);
    reinterpret_cast<raw *>(a.y)[row * a.N + col] = E::from_f32(apply_act(o, a.act));
  }
}

// Packs w[n][k] into 16-column k-major panels, zero-filled past n.
template <typename raw>
__global__ void fc_pack_kernel(const raw *__restrict__ w, raw *__restrict__ wp, int64_t K,
                               int64_t N, int64_t panels) {
  const int64_t total = panels * K * 2;  // (panel, k, half-row of 8 columns)
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t h = i & 1, k = (i >> 1) % K, p = (i >> 1) / K;
    raw v[8];
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const int64_t n = p * kPanel + 8 * h + t;
      v[t] = n < N ? w[n * K + k] : (raw)0;
    }
    uint4 out;
    __builtin_memcpy(&out, v, 16);
    *reinterpret_cast<uint4 *>(wp + (p * K + k) * kPanel + 8 * h) = out;
  }
}

template <int DT, int MT, bool SKIP, bool XVEC, bool MEASURE>
void launch_one(dim3 grid, hipStream_t st, const FcBwArgs &a) {
  hipLaunchKernelGGL((fc_bw_kernel<DT, MT, SKIP, XVEC, MEASURE>), grid,
                     dim3(64 * Shape<MT>::waves), 0, st, a);
}

template <int DT, bool SKIP, bool XVEC, bool MEASURE = false>
bool launch_mt(int mt, dim3 grid, hipStream_t st, const FcBwArgs &a) {
  switch (mt) {
    case 1: launch_one<DT, 1, SKIP, XVEC, MEASURE>(grid, st, a); break;
    case 2: launch_one<DT, 2, SKIP, XVEC, MEASURE>(grid, st, a); break;
    case 3: launch_one<DT, 3, SKIP, XVEC, MEASURE>(grid, st, a); break;
    case 4: launch_one<DT, 4, SKIP, XVEC, MEASURE>(grid, st, a); break;
    default: return false;
  }
  return true;
}

template <int DT>
bool launch_dt(int mt, bool skip, bool xvec, dim3 grid, hipStream_t st, const FcBwArgs &a) {
  if (skip) return launch_mt<DT, true, false>(mt, grid, st, a);
  return xvec ? launch_mt<DT, false, true>(mt, grid, st, a)
              : launch_mt<DT, false, false>(mt, grid, st, a);
}

int waves_for(int64_t m) { return m <= 32 ? Shape<1>::waves : Shape<3>::waves; }

int64_t slice_for(const sparoa_fc_desc &d) {
  return cdiv(cdiv(d.k, waves_for(d.m)), 64) * 64;
}

}  // namespace

bool fc_bw_streams(const sparoa_fc_desc &d) {
  return d.dtype != SPAROA_F32 && d.m <= 64 && slice_for(d) <= kMaxWaveK;
}

size_t fc_packed_bytes(const sparoa_fc_desc &d) {
  return (size_t)cdiv(d.n, kPanel) * kPanel * (size_t)d.k * (size_t)elem_size(d.dtype);
}

size_t fc_bw_workspace(const sparoa_fc_desc &, sparoa_path) { return 0; }

sparoa_status launch_fc_pack(const sparoa_fc_desc &d, const void *w_nk, void *w_packed,
                             hipStream_t stream) {
  if (d.dtype == SPAROA_F32) return fail(SPAROA_ERR_UNSUPPORTED, "fc bandwidth path: fp32");
  const int64_t panels = cdiv(d.n, kPanel);
  const int64_t total = panels * d.k * 2;
  int64_t blocks = cdiv(total, 256);
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL(fc_pack_kernel<uint16_t>, dim3((unsigned)blocks), dim3(256), 0, stream,
                     static_cast<const uint16_t *>(w_nk), static_cast<uint16_t *>(w_packed), d.k,
                     d.n, panels);
  SPAROA_LAUNCH_CHECK("fc_pack_kernel");
  return SPAROA_OK;
}

sparoa_status launch_fc_bw(const sparoa_fc_desc &d, sparoa_path, const void *x,
                           const void *w_packed, const void *bias, const void *residual,
                           sparoa_act act, const uint32_t *mask, void *y, void *, size_t,
                           uint64_t *executed, hipStream_t stream, const DeviceRoute *route) {
  if (!fc_bw_streams(d))
    return fail(SPAROA_ERR_UNSUPPORTED, "weight-streaming FC: needs 16-bit, m <= 64, k <= 16384");
  const bool skip = mask != nullptr;
  FcBwArgs a;
  a.x = static_cast<const char *>(x);
  a.wp = static_cast<const char *>(w_packed);
  a.bias = static_cast<const char *>(bias);
  a.residual = static_cast<const char *>(residual);
  a.y = static_cast<char *>(y);
  a.mask = mask;
  a.executed = reinterpret_cast<unsigned long long *>(skip ? executed : nullptr);
  a.M = d.m; a.K = d.k; a.N = d.n; a.slice = slice_for(d);
  a.act = act;
  a.route = route ? *route : DeviceRoute{nullptr, 0.0, 0, 0, nullptr};
  a.mcounts = nullptr;
  a.mmask = nullptr;
  if (a.executed) {
    sparoa_status st = launch_set_u64(executed, 0, stream);
    if (st != SPAROA_OK) return st;
  }
  const int mt = (int)cdiv(d.m, 16);
  // dense x rows are read as 16-byte vectors: needs every row 16-byte aligned
  const bool xvec = d.k % 8 == 0;
  a.xvec = xvec ? 1 : 0;
  dim3 grid((unsigned)cdiv(d.n, kPanel));
  const bool ok = d.dtype == SPAROA_BF16 ? launch_dt<SPAROA_BF16>(mt, skip, xvec, grid, stream, a)
                                         : launch_dt<SPAROA_F16>(mt, skip, xvec, grid, stream, a);
  if (!ok) return fail(SPAROA_ERR_UNSUPPORTED, "fc bandwidth path: m");
  SPAROA_LAUNCH_CHECK("fc_bw_kernel");
  return SPAROA_OK;
}

bool fc_bw_self_measures(const sparoa_fc_desc &d) { return fc_bw_streams(d) && d.k % 8 == 0; }

sparoa_status launch_fc_bw_measured(const sparoa_fc_desc &d, const void *x, const void *w_packed,
                                    const void *bias, const void *residual, sparoa_act act,
                                    sparoa_counts *counts, uint32_t *mask, void *y,
                                    hipStream_t stream, const DeviceRoute &route) {
  if (!fc_bw_self_measures(d))
    return fail(SPAROA_ERR_UNSUPPORTED, "self-measuring FC: needs the streaming kernel and k % 8 == 0");
  FcBwArgs a;
  a.x = static_cast<const char *>(x);
  a.wp = static_cast<const char *>(w_packed);
  a.bias = static_cast<const char *>(bias);
  a.residual = static_cast<const char *>(residual);
  a.y = static_cast<char *>(y);
  a.mask = nullptr;
  a.executed = nullptr;
  a.M = d.m; a.K = d.k; a.N = d.n; a.slice = slice_for(d);
  a.act = act;
  a.xvec = 1;
  a.route = route;
  a.route.counts = nullptr;
  a.mcounts = counts;
  a.mmask = mask;
  const int mt = (int)cdiv(d.m, 16);
  dim3 grid((unsigned)cdiv(d.n, kPanel));
  const bool ok = d.dtype == SPAROA_BF16
                      ? launch_mt<SPAROA_BF16, true, false, true>(mt, grid, stream, a)
                      : launch_mt<SPAROA_F16, true, false, true>(mt, grid, stream, a);
  if (!ok) return fail(SPAROA_ERR_UNSUPPORTED, "fc bandwidth path: m");
  SPAROA_LAUNCH_CHECK("fc_bw_kernel (self-measuring)");
  return SPAROA_OK;
}

}  // namespace sparoa
