// Weight-streaming FC for small m (m <= 64): the bandwidth path of the
// light quadrants (SparOA Section 2.2) and its zero-skipping form (Section
// 2.1).  At m <= 64 an FC has intensity <= ~62 FLOP/byte, far below the
// MI355X ridge point, so its time is the time to stream the weights once.
//
// Weights are packed once (sparoa_fc_pack_weights) into 16-column panels in
// two layouts.  Skip layout, k-major inside a panel: S[p][k][0..15] =
// w[16p + 0..15][k] (zero past n): a panel is one contiguous stream of k rows
// of 32 bytes, and an input column k that is zero in all m rows owns exactly
// one such row per panel, so the skip variant drops it from the stream (skip
// granularity: one column).  Dense layout, per 32-k chunk column-major:
// D[p][c][j][0..31] = w[16p + j][32c + 0..31] (zero past n and k): the 16
// bytes a lane loads are its MFMA B operand as they are (8 consecutive k of
// one column), so the dense order needs no transpose through LDS.
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

#include <algorithm>
#include <type_traits>

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
  // ring depth (chunks in flight), dense and skip order, within the VGPR
  // budget without spills (a skip-order chunk holds twice the input registers)
  static constexpr int depth = MT == 1 ? 8 : 4;
  static constexpr int list_depth = MT == 1 ? 6 : (MT == 4 ? 2 : 3);
};

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

struct FcBwArgs {
  const char *x;
  const char *wp;  // skip layout
  const char *wd;  // dense layout
  const char *bias;
  const char *residual;
  char *y;
  const uint32_t *mask;
  unsigned long long *executed;
  int64_t M, K, N, slice;
  int act;
  DeviceRoute route;
  sparoa_counts *mcounts;  // self-measuring form: outputs of the measurement
  uint32_t *mmask;
};

constexpr int kMaxColWords = kMaxWaveK * 16 / 32;  // bitmap words for the largest K

// LDS of one wave: transposed weight tile [16 cols][32 entries] and input
// tile [16*MT rows][32 entries] of the chunk in flight to the MFMA.
template <int MT>
struct WaveTiles {
  char wt[kPanel * kRowB];
  char xs[MT * 16 * kRowB];
};

// LDS of one wave in the grouped kernel: the transposed weight tile only (the
// input is staged per work-group).
struct WeightTile {
  char wt[kPanel * kRowB];
};

// ---- pieces shared by the single-operator and the grouped kernels --------

// Measurement of x by one work-group of NW waves (the self-measuring forms):
// zero count and the column bitmap at block (m, 1) into mbits (LDS), the
// route decision from those counts with the host route's arithmetic.  When
// store, the counts, the bitmap and the path also go to a.mcounts / a.mmask /
// path_out.  Thread t owns column groups t, t + 64 NW, ... (8 columns = one
// bitmap byte; K % 8 == 0): it ORs the group's nonzero flags over all rows
// (kMR row loads in flight), counts zeros, and stores the byte; bytes past K
// up to the last whole word are stored as 0.  The waves' sums meet in LDS.
// Returns the skip decision (the same in every lane).
template <int MT, int NW>
__device__ __forceinline__ bool fc_measure_route(const FcBwArgs &a, bool store, uint32_t *mbits) {
  constexpr int kThreads = 64 * NW;
  constexpr int kMR = MT == 1 ? 8 : (MT == 2 ? 16 : 32);
  __shared__ unsigned wsum[NW][2];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int ng = (int)(a.K / 8);
  const int nbytes = 4 * (int)((a.K + 31) / 32);
  unsigned zeros = 0, ones = 0;
  for (int g = tid; g < nbytes; g += kThreads) {
    uint32_t nzb = 0;
    if (g < ng) {
      const char *px = a.x + (int64_t)g * 16;
      for (int m0 = 0; m0 < a.M; m0 += kMR) {
        // unconditional loads (rows past M re-read row M - 1 and are masked
        // below), so all kMR stay in flight
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
  sparoa_counts c;
  c.zeros = zeros;
  c.numel = (uint64_t)a.M * (uint64_t)a.K;
  c.zero_blocks = (uint64_t)a.K - ones;
  c.num_blocks = (uint64_t)a.K;
  const bool skip = __builtin_amdgcn_readfirstlane(
                        route_skip_counts(c, a.route.sparsity_thr, a.route.mode) ? 1 : 0) != 0;
  if (store) {
    for (int i = tid; i < nbytes / 4; i += kThreads) a.mmask[i] = mbits[i];
    if (tid == 0) {
      *a.mcounts = c;
      if (a.route.path_out)
        *a.route.path_out = (skip ? 1u : 0u) | ((uint32_t)a.route.bw_bit << 1);
    }
  }
  return skip;
}

// The same measurement and route for any m, rows split over threads (the
// grouped kernel, where m reaches 64): tpg threads per column group (a power
// of two, tpg * groups <= 64 NW, tpg <= m), each ORs its rows' nonzero flags
// into the group's bitmap byte with an LDS atomic and counts their zeros;
// the nonzero-column count is taken from the finished bitmap.
template <int NW>
__device__ __forceinline__ bool fc_measure_route_rows(const FcBwArgs &a, bool store,
                                                      uint32_t *mbits) {
  constexpr int kThreads = 64 * NW;
  constexpr int kMR = 8;
  __shared__ unsigned wsum[NW][2];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int M = (int)a.M;
  const int ng = (int)(a.K / 8);
  const int nwords = (int)((a.K + 31) / 32);
  for (int i = tid; i < nwords; i += kThreads) mbits[i] = 0u;
  __syncthreads();
  int lt = 0;  // log2 of tpg
  while ((2 << lt) * ng <= kThreads && (2 << lt) <= M) ++lt;
  const int tpg = 1 << lt;
  unsigned zeros = 0;
  for (int t = tid; t < ng * tpg; t += kThreads) {
    const int g = t >> lt, ph = t & (tpg - 1);
    const char *px = a.x + (int64_t)g * 16;
    uint32_t nzb = 0;
    for (int m0 = ph * kMR; m0 < M; m0 += tpg * kMR) {
      // unconditional loads (rows past M re-read row M - 1 and are masked
      // below), so all kMR stay in flight
      uint4 q[kMR];
#pragma unroll
      for (int u = 0; u < kMR; ++u) {
        const int64_t r = min(m0 + u, M - 1);
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
        const bool valid = m0 + u < M;
        zeros += valid ? 8u - (unsigned)__popc(b) : 0u;
        nzb |= valid ? b : 0u;
      }
    }
    if (nzb) atomicOr(&mbits[g >> 2], nzb << (8 * (g & 3)));
  }
  __syncthreads();
  unsigned ones = 0;
  for (int i = tid; i < nwords; i += kThreads) ones += (unsigned)__popc(mbits[i]);
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
  sparoa_counts c;
  c.zeros = zeros;
  c.numel = (uint64_t)a.M * (uint64_t)a.K;
  c.zero_blocks = (uint64_t)a.K - ones;
  c.num_blocks = (uint64_t)a.K;
  const bool skip = __builtin_amdgcn_readfirstlane(
                        route_skip_counts(c, a.route.sparsity_thr, a.route.mode) ? 1 : 0) != 0;
  if (store) {
    for (int i = tid; i < nwords; i += kThreads) a.mmask[i] = mbits[i];
    if (tid == 0) {
      *a.mcounts = c;
      if (a.route.path_out)
        *a.route.path_out = (skip ? 1u : 0u) | ((uint32_t)a.route.bw_bit << 1);
    }
  }
  return skip;
}

// List of the nonzero columns of slice [kb, kb + count) (offsets from kb, in
// order) built by one wave from the column bitmap: the slice's bitmap words
// (at most 32: one per lane) are loaded at once, an exclusive prefix sum of
// their popcounts gives each lane its place, then each lane writes the
// offsets of its set bits.  Returns the list length (the same in every lane).
__device__ __forceinline__ int fc_build_list(const uint32_t *colbits, int64_t kb, int count,
                                             unsigned short *list, int lane) {
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
    list[pos++] = (unsigned short)(32 * lane + b);
    wv &= wv - 1u;
  }
  return __builtin_amdgcn_readfirstlane(__shfl(incl, 63, 64));
}

// Register staging of one chunk: weight row e = lane / 2, half lane % 2;
// the input as 4 * MT pairs (dense order: packed), or in skip order as
// 8 * MT 16-bit gathers, each in a register of its own (two loads into the
// halves of one register would make the second wait for the first).
template <int MT, bool LIST>
struct Stage {
  uint4 w;
  uint32_t xr[LIST ? 8 * MT : 4 * MT];
};

// Entry e of a slice walk -> column k, or -1 past its end.  LIST: the skip
// order (list of nonzero columns of the slice), else dense order.
// Branch-free: the list read is clamped and the result selected.
template <bool LIST>
__device__ __forceinline__ int fc_entry_k(const unsigned short *list, int kb, int count, int e) {
  int k;
  if constexpr (LIST) k = kb + (int)list[max(0, min(e, count - 1))];
  else k = kb + e;
  return e < count ? k : -1;
}

constexpr int kOob = (int)0x80000000;  // a buffer offset past every descriptor's size

// Loads chunk c of the slice [kb, kb + count) of one 16-column panel (wrs:
// its k-major weights).  Input, dense order: (row m, 8 entries) per
// v = lane + 64 j, one 16-byte load (rows 16-byte aligned: XVEC) or eight
// 2-byte loads; skip order: (row m, entries 2q, 2q + 1) per v = lane + 64 j,
// two 2-byte gathers.  Both forms use the same 4 * MT registers.  Every load
// is a buffer load issued unconditionally: an entry past the end, a row past
// M or a ring slot past the last chunk (live false) reads zero from an
// out-of-range offset without touching memory, so the compiler's load
// counters stay exact and the ring stays in flight.
template <int DT, int MT, bool LIST, bool XVEC>
__device__ __forceinline__ void fc_load_chunk(Stage<MT, LIST> &s, __amdgpu_buffer_rsrc_t wrs,
                                              __amdgpu_buffer_rsrc_t xrs, int r0, int Mi, int Ki,
                                              int kb,
                                              int count, const unsigned short *list, int c,
                                              bool live, int lane) {
  using raw = typename Elem<DT>::raw;
  if constexpr (LIST) {  // skip layout (wrs): row k, half lane % 2, transposed later
    const int k = fc_entry_k<LIST>(list, kb, count, c * kCh + (lane >> 1));
    s.w = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(
        wrs, live && k >= 0 ? (k * kPanel + 8 * (lane & 1)) * 2 : kOob, 0, 0));
  } else {  // dense layout (wrs): the B operand, column lane % 16, k 8 (lane / 16) + 0..7
    s.w = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(
        wrs, live && c * kCh < count ? (((kb >> 5) + c) * 16 + (lane & 15)) * 64 + 16 * (lane >> 4)
                                      : kOob, 0, 0));
  }
  if constexpr (!LIST) {
#pragma unroll
    for (int j = 0; j < MT; ++j) {
      const int v = lane + 64 * j;
      const int m = r0 + (v >> 2), e0 = c * kCh + 8 * (v & 3);
      const int row = (m * Ki + kb + e0) * 2;
      uint4 q;
      if constexpr (XVEC) {  // count % 8 == 0: e0 < count covers all 8 entries
        q = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(
            xrs, live && m < Mi && e0 < count ? row : kOob, 0, 0));
      } else {
        raw t[8];
#pragma unroll
        for (int i = 0; i < 8; ++i)
          t[i] = __builtin_bit_cast(raw, __builtin_amdgcn_raw_buffer_load_b16(
              xrs, live && m < Mi && e0 + i < count ? row + 2 * i : kOob, 0, 0));
        __builtin_memcpy(&q, t, 16);
      }
      __builtin_memcpy(&s.xr[4 * j], &q, 16);
    }
  } else {
#pragma unroll
    for (int j = 0; j < 4 * MT; ++j) {
      const int v = lane + 64 * j;
      const int m = r0 + (v >> 4), e0 = c * kCh + 2 * (v & 15);
      const int k0 = fc_entry_k<true>(list, kb, count, e0);
      const int k1 = fc_entry_k<true>(list, kb, count, e0 + 1);
      const bool ok = live && m < Mi;
      s.xr[2 * j] = __builtin_bit_cast(uint16_t, __builtin_amdgcn_raw_buffer_load_b16(
          xrs, ok && k0 >= 0 ? (m * Ki + k0) * 2 : kOob, 0, 0));
      s.xr[2 * j + 1] = __builtin_bit_cast(uint16_t, __builtin_amdgcn_raw_buffer_load_b16(
          xrs, ok && k1 >= 0 ? (m * Ki + k1) * 2 : kOob, 0, 0));
    }
  }
}

// One staged chunk through the wave's LDS tiles (weights transposed on the
// way in) into v_mfma_f32_16x16x32 over all m (padded to 16) and the
// panel's 16 columns.  LDS operations of one wave execute in order: the
// tile written here is the one read back, and the reads finish before the
// next chunk's writes.
template <int DT, int MT, bool LIST>
__device__ __forceinline__ void fc_mma_chunk(const Stage<MT, LIST> &s, WaveTiles<MT> &T,
                                             f32x4 (&acc)[MT], int lane) {
  using raw = typename Elem<DT>::raw;
  if constexpr (LIST) {  // skip layout: weights transposed through the wave's tile
    const int e = lane >> 1, c0 = 8 * (lane & 1);
    raw h[8];
    __builtin_memcpy(h, &s.w, 16);
#pragma unroll
    for (int i = 0; i < 8; ++i) *reinterpret_cast<raw *>(&T.wt[(c0 + i) * kRowB + 2 * e]) = h[i];
  }
  if constexpr (!LIST) {
#pragma unroll
    for (int j = 0; j < MT; ++j) {
      const int v = lane + 64 * j;
      uint4 q;
      __builtin_memcpy(&q, &s.xr[4 * j], 16);
      *reinterpret_cast<uint4 *>(&T.xs[(v >> 2) * kRowB + 16 * (v & 3)]) = q;
    }
  } else {
#pragma unroll
    for (int j = 0; j < 4 * MT; ++j) {
      const int v = lane + 64 * j;
      *reinterpret_cast<uint32_t *>(&T.xs[(v >> 4) * kRowB + 4 * (v & 15)]) =
          s.xr[2 * j] | (s.xr[2 * j + 1] << 16);
    }
  }
  const int g = lane >> 4, rl = lane & 15;
  u32x4 bq;
  if constexpr (LIST) bq = *reinterpret_cast<const u32x4 *>(&T.wt[rl * kRowB + 16 * g]);
  else bq = __builtin_bit_cast(u32x4, s.w);  // dense layout: already the B operand
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    const u32x4 aq = *reinterpret_cast<const u32x4 *>(&T.xs[(mt * 16 + rl) * kRowB + 16 * g]);
    if constexpr (DT == SPAROA_BF16)
      acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, aq),
                                                        __builtin_bit_cast(bf16x8, bq),
                                                        acc[mt], 0, 0, 0);
    else
      acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, aq),
                                                       __builtin_bit_cast(f16x8, bq),
                                                       acc[mt], 0, 0, 0);
  }
}

// Output element (row, col) from its fp32 sum: bias, residual, activation,
// cast (the same order in both kernels).
template <int DT>
__device__ __forceinline__ void fc_store(const FcBwArgs &a, int64_t row, int64_t col, float o) {
  using E = Elem<DT>;
  using raw = typename E::raw;
  if (a.bias) o += E::to_f32(reinterpret_cast<const raw *>(a.bias)[col]);
  if (a.residual) o += E::to_f32(reinterpret_cast<const raw *>(a.residual)[row * a.N + col]);
  reinterpret_cast<raw *>(a.y)[row * a.N + col] = E::from_f32(apply_act(o, a.act));
}

// Panel p's weights in the skip layout (LIST) or the dense layout.
template <bool LIST>
__device__ __forceinline__ __amdgpu_buffer_rsrc_t fc_panel_rsrc(const FcBwArgs &a, int64_t p) {
  if constexpr (LIST)
    return __builtin_amdgcn_make_buffer_rsrc((void *)(a.wp + p * a.K * kPanel * 2), (short)0,
                                             (int)(a.K * kPanel * 2), kBufDword3);
  const int64_t bytes = (a.K + kCh - 1) / kCh * kPanel * kCh * 2;
  return __builtin_amdgcn_make_buffer_rsrc((void *)(a.wd + p * bytes), (short)0, (int)bytes,
                                           kBufDword3);
}

// ---- single operator: one work-group per panel ----------------------------
// Wave w walks K slice w ([w * slice, (w + 1) * slice) ∩ [0, K)); the waves'
// fp32 partials meet in LDS and are added in wave order (deterministic).
template <int DT, int MT, bool SKIP, bool XVEC, bool MEASURE = false>
__global__ __launch_bounds__(64 * Shape<MT>::waves) void fc_bw_kernel(FcBwArgs a) {
  static_assert(!MEASURE || SKIP, "the self-measuring form may skip");
  constexpr int NW = Shape<MT>::waves;
  constexpr int kDepth = Shape<MT>::depth;
  constexpr int kThreads = 64 * NW;
  static_assert(Elem<DT>::size == 2, "16-bit types only");
  __shared__ WaveTiles<MT> tiles[NW];
  __shared__ unsigned short lists[SKIP ? NW : 1][SKIP ? kMaxWaveK : 1];
  __shared__ float red[NW * MT * 16 * kPanel];  // [wave][16*MT][16] partials
  __shared__ uint32_t mbits[MEASURE ? kMaxColWords : 1];
  // gfx950 addresses 160 KB of LDS per work-group
  static_assert(sizeof(tiles) + sizeof(lists) + sizeof(red) + sizeof(mbits) <= 160 * 1024,
                "LDS budget");

  // wave, count, use_list: the same in every lane of a wave; readfirstlane
  // tells the compiler, so descriptors and loop bounds live in scalar
  // registers (no per-lane loops around buffer loads, no divergent branches)
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int64_t p = blockIdx.x;
  const int kb = (int)(wave * a.slice);
  int count = (int)max((int64_t)0, min(a.slice, a.K - kb));
  bool use_list = SKIP;
  const uint32_t *colbits = a.mask;
  if constexpr (MEASURE) {
    use_list = fc_measure_route<MT, NW>(a, p == 0, mbits);
    colbits = mbits;
  } else if constexpr (SKIP) {
    if (a.route.counts) {
      use_list = device_route_skip(a.route);
      if (a.route.path_out && p == 0 && tid == 0)
        *a.route.path_out = (use_list ? 1u : 0u) | ((uint32_t)a.route.bw_bit << 1);
    }
  }
  const unsigned short *list = lists[SKIP ? wave : 0];
  if (SKIP && use_list) {
    count = fc_build_list(colbits, kb, count, lists[wave], lane);
    if (a.executed && p == 0 && lane == 0 && count)
      atomicAdd(a.executed, (unsigned long long)count);
  }
  // Chunk c sits in register slot c % D (the ring depth); ring slots past the last chunk
  // load nothing.
  const int nch = (count + kCh - 1) / kCh;
  const __amdgpu_buffer_rsrc_t xrs = __builtin_amdgcn_make_buffer_rsrc(
      (void *)a.x, (short)0, (int)(a.M * a.K * 2), kBufDword3);
  const int Mi = (int)a.M, Ki = (int)a.K;
  f32x4 acc[MT];
#pragma unroll
  for (int i = 0; i < MT; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};

  // the walk, with the order (dense or skip list) fixed outside the loop
  auto run = [&](auto list_tag) __attribute__((always_inline)) {
    constexpr bool LIST = decltype(list_tag)::value;
    constexpr int D = LIST ? Shape<MT>::list_depth : kDepth;
    const __amdgpu_buffer_rsrc_t wrs = fc_panel_rsrc<LIST>(a, p);
    Stage<MT, LIST> st[D];
#pragma unroll
    for (int j = 0; j < D; ++j) {
      fc_load_chunk<DT, MT, LIST, XVEC>(st[j], wrs, xrs, 0, Mi, Ki, kb, count, list, j, j < nch,
                                        lane);
      __builtin_amdgcn_sched_barrier(0);  // slot order, as in the steady state
    }
    // steady state: straight-line groups of D chunks; then the last
    // (partial) group, whose chunks are all loaded already
    int c0 = 0;
    for (; c0 + D <= nch; c0 += D) {
#pragma unroll
      for (int j = 0; j < D; ++j) {
        fc_mma_chunk<DT, MT, LIST>(st[j], tiles[wave], acc, lane);
        const int cn = c0 + j + D;
        fc_load_chunk<DT, MT, LIST, XVEC>(st[j], wrs, xrs, 0, Mi, Ki, kb, count, list, cn, cn < nch,
                                          lane);
        // keep the steps in order: hoisting later steps' LDS staging would
        // wait for all the ring's chunks at once and drain it
        __builtin_amdgcn_sched_barrier(0);
      }
    }
#pragma unroll
    for (int j = 0; j < D; ++j)
      if (c0 + j < nch) fc_mma_chunk<DT, MT, LIST>(st[j], tiles[wave], acc, lane);
  };
  if (SKIP && use_list) run(std::true_type{});
  else run(std::false_type{});

  __syncthreads();
  const int g = lane >> 4, rl = lane & 15;
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
    fc_store<DT>(a, row, col, o);
  }
}

// ---- several operators in one launch --------------------------------------
// The G_j = start[j + 1] - start[j] work-groups of FC j each take 16
// consecutive panels, one per wave.  A wave walks every K slice of the
// single-operator kernel in slice order (the same chunks, lists and MFMA
// sequence), keeps each slice's partial apart and adds it to its sum at the
// slice's end: the sums are those of the single-operator kernel bit for bit.
// The work-group measures x once, and its waves build the slice lists
// together (wave s: slice s).  The input is staged once per work-group, SC
// chunks at a time, in double-buffered LDS that all 16 waves read their MFMA
// A operands from (x is read from L2 once per work-group, not once per
// wave); the weights stream through a per-wave register ring that runs on
// across the stage barriers.
struct FcBwGroup {
  FcBwArgs op[kGroupMax];
  int start[kGroupMax + 1];
  int n;
};
static_assert(sizeof(FcBwGroup) <= 4096, "kernel argument space");

// A copy of v held in scalar registers: v is the same in every lane, but the
// compiler cannot see that for a kernel-argument entry picked by a computed
// index (it would wrap each buffer load in a loop over distinct descriptors).
template <typename T>
__device__ __forceinline__ T uniform_copy(const T &v) {
  static_assert(sizeof(T) % 4 == 0, "whole dwords");
  uint32_t w[sizeof(T) / 4];
  __builtin_memcpy(w, &v, sizeof(T));
#pragma unroll
  for (int i = 0; i < (int)(sizeof(T) / 4); ++i) w[i] = __builtin_amdgcn_readfirstlane(w[i]);
  T out;
  __builtin_memcpy(&out, w, sizeof(T));
  return out;
}


// Waves (= panels) per work-group: 8, so that two work-groups share a CU
// and the dispatcher rebalances as work-groups of skipped (short) operators
// finish; chunks per x stage SC >= ring depth D, so that waiting for a
// stage's x loads (issued SC chunks earlier) leaves the ring in flight.
// Chunks per x stage SC = chunks in flight D: dense order 8; skip order,
// whose gathers take a register per 2-byte value, 8, 4 for m > 16 -- so
// that m <= 32 fits two work-groups per CU (128 VGPRs, 80 KB of LDS).  For
// m > 48 the staged rows take 96 KB at 8 chunks, so one work-group per CU
// (the dispatcher spreads such launches one per CU anyway); eight m = 64
// FCs of 4096 x 4096 take 5 % less time than with 4 chunks in flight.
template <int MT, bool LIST = false>
struct GroupShape {
  static constexpr int NW = 8;
  static constexpr int SC = LIST ? (MT == 1 ? 8 : 4) : 8;
  static constexpr int D = SC;                                 // weight ring depth (chunks)
  static constexpr int U = SC;                                 // steps per loop iteration
  static constexpr int XROW = SC * kCh * 2 + 16;               // LDS bytes per staged x row
  static constexpr int XVEC = MT * 16 * SC * 4;                // 16-byte vectors per stage
  static constexpr int XVAL = MT * 16 * SC * kCh;              // 2-byte values per stage
  static constexpr int NXVEC = (XVEC + 64 * NW - 1) / (64 * NW);  // per thread
  static constexpr int NXV = (XVAL + 64 * NW - 1) / (64 * NW);    // per thread
};

// (at least four waves per SIMD -- two work-groups per CU -- for m <= 48)
template <int DT, int MT>
__global__ __launch_bounds__(64 * GroupShape<MT>::NW, MT == 4 ? 2 : 4) void fc_bw_measured_group(
    FcBwGroup grp) {
  constexpr int NW = GroupShape<MT>::NW;
  constexpr int kThreads = 64 * NW;
  constexpr int XROWMAX = GroupShape<MT>::XROW;  // the dense stage is the larger
  using raw = typename Elem<DT>::raw;
  __shared__ WeightTile wtiles[NW];  // each wave's transposed weight chunk
  __shared__ __attribute__((aligned(16))) char xst[2][MT * 16 * XROWMAX];
  constexpr int kMaxSlices = Shape<MT>::waves;  // K slices of the single-operator kernel
  __shared__ unsigned short lists[kMaxSlices][kMaxWaveK];
  __shared__ int slice_count[kMaxSlices];
  __shared__ uint32_t mbits[kMaxColWords];
  // m <= 32: two work-groups per CU; larger m holds one (registers bound it)
  static_assert(sizeof(wtiles) + sizeof(xst) + sizeof(lists) + sizeof(mbits) <=
                    (MT <= 2 ? 80 : 160) * 1024,
                "LDS budget");

  // this work-group's operator: the starts at or below blockIdx.x, counted
  // over fixed indices (their loads are issued together, not one per step)
  int j = 0;
#pragma unroll
  for (int q = 1; q < kGroupMax; ++q) j += (q < grp.n && (int)blockIdx.x >= grp.start[q]) ? 1 : 0;
  const FcBwArgs a = uniform_copy(grp.op[j]);
  const int wg = (int)blockIdx.x - grp.start[j];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

  const bool use_list = fc_measure_route_rows<NW>(a, wg == 0, mbits);
  const int nslices = (int)((a.K + a.slice - 1) / a.slice);  // <= kMaxSlices
  for (int sl = wave; sl < nslices; sl += NW) {
    const int kb = (int)(sl * a.slice);
    int count = (int)min(a.slice, a.K - kb);
    if (use_list) count = fc_build_list(mbits, kb, count, lists[sl], lane);
    if (lane == 0) slice_count[sl] = count;
  }
  __syncthreads();

  // this wave's panel; waves past the last one still stage x and meet the
  // barriers, but load no weights and store nothing
  const int64_t p = (int64_t)wg * NW + wave;
  const bool pvalid = p < (a.N + kPanel - 1) / kPanel;
  const __amdgpu_buffer_rsrc_t xrs = __builtin_amdgcn_make_buffer_rsrc(
      (void *)a.x, (short)0, (int)(a.M * a.K * 2), kBufDword3);
  const int Mi = (int)a.M, Ki = (int)a.K, slice = (int)a.slice;

  // The walk: every slice in slice order, each as nchu chunks (the most any
  // slice has; chunks past a slice's entries load nothing and add zeros, so
  // the slice partials are those of the single-operator kernel).  Chunk i =
  // chunk i % nchu of slice i / nchu; x stage t holds chunks [t SC, t SC + SC).
  int nchu = 1;  // at least one (all-empty slices: every chunk loads nothing)
  for (int sl = 0; sl < nslices; ++sl)
    nchu = max(nchu, __builtin_amdgcn_readfirstlane((slice_count[sl] + kCh - 1) / kCh));
  const int total = nslices * nchu;
  f32x4 acc[MT], sum[MT];
#pragma unroll
  for (int i = 0; i < MT; ++i) acc[i] = sum[i] = f32x4{0.f, 0.f, 0.f, 0.f};

  // ALIGNED: nchu % U == 0 (dense slices of 8 or 16 chunks), so a slice ends
  // only at an iteration's last step and the partial's selects run there
  auto run = [&](auto list_tag, auto aligned_tag) __attribute__((always_inline)) {
    constexpr bool LIST = decltype(list_tag)::value;
    constexpr bool ALIGNED = decltype(aligned_tag)::value;
    using GS = GroupShape<MT, LIST>;
    constexpr int SC = GS::SC, D = GS::D, U = GS::U, XROW = GS::XROW;
    const __amdgpu_buffer_rsrc_t wrs = fc_panel_rsrc<LIST>(a, pvalid ? p : 0);
    constexpr int NXVEC = GS::NXVEC;  // staged 16-byte x vectors per thread (dense order)
    constexpr int NXV = GS::NXV;      // staged 2-byte x values per thread (skip order)
    static_assert(U % SC == 0 && U % D == 0 && SC >= D, "whole stages and ring cycles");
    static_assert((LIST ? GS::XVAL : GS::XVEC) % kThreads == 0,
                  "every thread stages whole vectors / values");
    // Column of entry e of chunk i (-1 past the slice's entries or the walk).
    // Everything is computed unconditionally and selected (a short-circuit
    // here becomes a branch inside the ring, which drains it).
    // column_at: the same for chunk c of slice sl (sl >= nslices: past the
    // walk), which the ring's look-ahead tracks with counters instead of a
    // division per step.
    auto column_at = [&](int sl, int c, int e) __attribute__((always_inline)) -> int {
      const int slc = min(sl, nslices - 1);
      const int ee = c * kCh + e;
      int k, cnt;
      if constexpr (LIST) {
        cnt = slice_count[slc];
        k = slc * slice + (int)lists[slc][max(0, min(ee, cnt - 1))];
      } else {  // every column of the slice (no LDS read: no wait in the ring)
        cnt = min(slice, Ki - slc * slice);
        k = slc * slice + ee;
      }
      const bool ok = (sl < nslices) & (ee < cnt);
      return ok ? k : -1;
    };
    auto column = [&](int i, int e) __attribute__((always_inline)) -> int {
      if constexpr (!LIST) {
        // dense: the chunks tile K in order (a slice is nchu whole chunks, or
        // the only slice), so chunk i starts at column 32 i
        const int k = i * kCh + e;
        return (i < total) & (k < Ki) ? k : -1;
      }
      const int ic = min(i, total - 1);
      const int sl = ic / nchu, c = ic - sl * nchu;
      return column_at(i < total ? sl : nslices, c, e);
    };
    // x stage t -> registers: dense, NXVEC 16-byte vectors (row, 8 entries)
    // per thread; skip order, NXV 2-byte gathers per thread.
    uint4 xv[NXVEC];
    uint32_t xh[NXV];
    auto stage_load = [&](int t) __attribute__((always_inline)) {
      // rows past M read row M - 1: their outputs are never stored, and an
      // MFMA output row depends on its own A row only (no per-lane test
      // here, which the compiler would turn into a branch in the ring)
      if constexpr (!LIST) {
#pragma unroll
        for (int u = 0; u < NXVEC; ++u) {
          const int v = tid + kThreads * u;
          const int r = v / (SC * 4), eg = v - r * (SC * 4);
          const int k = column(t * SC + (eg >> 2), 8 * (eg & 3));
          xv[u] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(
              xrs, k >= 0 ? (min(r, Mi - 1) * Ki + k) * 2 : kOob, 0, 0));
        }
      } else {
#pragma unroll
        for (int u = 0; u < NXV; ++u) {
          const int v = tid + kThreads * u;
          const int r = v / (SC * kCh), ev = v - r * (SC * kCh);
          const int k = column(t * SC + ev / kCh, ev % kCh);
          xh[u] = __builtin_bit_cast(uint16_t, __builtin_amdgcn_raw_buffer_load_b16(
              xrs, k >= 0 ? (min(r, Mi - 1) * Ki + k) * 2 : kOob, 0, 0));
        }
      }
    };
    auto stage_store = [&](int t) __attribute__((always_inline)) {
      char *buf = xst[t & 1];
      if constexpr (!LIST) {
#pragma unroll
        for (int u = 0; u < NXVEC; ++u) {
          const int v = tid + kThreads * u;
          const int r = v / (SC * 4), eg = v - r * (SC * 4);
          *reinterpret_cast<uint4 *>(&buf[r * XROW + 16 * eg]) = xv[u];
        }
      } else {
#pragma unroll
        for (int u = 0; u < NXV; ++u) {
          const int v = tid + kThreads * u;
          const int r = v / (SC * kCh), ev = v - r * (SC * kCh);
          *reinterpret_cast<raw *>(&buf[r * XROW + 2 * ev]) = (raw)xh[u];
        }
      }
    };
    // weight ring: chunk i's 32 entries; skip layout: lane = (entry lane / 2,
    // half lane % 2); dense layout: the B operand (column lane % 16, entries
    // 8 (lane / 16) + 0..7) of the slice's k chunk
    auto wload = [&](uint4 &w, int i, int sl, int c) __attribute__((always_inline)) {
      int off;
      if constexpr (LIST) {
        const int k = column_at(sl, c, lane >> 1);
        off = pvalid && k >= 0 ? (k * kPanel + 8 * (lane & 1)) * 2 : kOob;
      } else {
        const int k = column(i, 0);  // the chunk's first column, -1 past the walk
        off = pvalid && k >= 0 ? ((k >> 5) * 16 + (lane & 15)) * 64 + 16 * (lane >> 4) : kOob;
      }
      w = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(wrs, off, 0, 0));
    };
    int cc = 0;  // chunks done in the current slice
    auto step = [&](const uint4 &w, int i, bool last) __attribute__((always_inline)) {
      // weights transposed into the wave's tile, then MT MFMAs whose A
      // operands come straight from the staged x
      const int g = lane >> 4, rl = lane & 15;
      u32x4 bq;
      if constexpr (LIST) {
        WeightTile &T = wtiles[wave];
        const int e = lane >> 1, c0 = 8 * (lane & 1);
        raw h[8];
        __builtin_memcpy(h, &w, 16);
#pragma unroll
        for (int q = 0; q < 8; ++q)
          *reinterpret_cast<raw *>(&T.wt[(c0 + q) * kRowB + 2 * e]) = h[q];
        bq = *reinterpret_cast<const u32x4 *>(&T.wt[rl * kRowB + 16 * g]);
      } else {
        bq = __builtin_bit_cast(u32x4, w);  // dense layout: already the B operand
      }
      const char *xa = &xst[(i / SC) & 1][rl * XROW + ((i % SC) * kCh + 8 * g) * 2];
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const u32x4 aq = *reinterpret_cast<const u32x4 *>(xa + mt * 16 * XROW);
        if constexpr (DT == SPAROA_BF16)
          acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, aq),
                                                            __builtin_bit_cast(bf16x8, bq),
                                                            acc[mt], 0, 0, 0);
        else
          acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, aq),
                                                           __builtin_bit_cast(f16x8, bq),
                                                           acc[mt], 0, 0, 0);
      }
      // at a slice's end its partial joins the sum (selects, no branch)
      if (ALIGNED && !last) return;
      const bool end = ALIGNED ? (i + 1) % nchu == 0 : ++cc == nchu;
      if (!ALIGNED) cc = end ? 0 : cc;
#pragma unroll
      for (int r = 0; r < MT; ++r) {
        const f32x4 t = sum[r] + acc[r];
        sum[r] = end ? t : sum[r];
        acc[r] = end ? f32x4{0.f, 0.f, 0.f, 0.f} : acc[r];
      }
    };

    uint4 ring[D];
    stage_load(0);
    stage_store(0);
#pragma unroll
    for (int q = 0; q < D; ++q) {
      const int qc = min(q, total - 1);
      wload(ring[q], q, q < total ? qc / nchu : nslices, qc % nchu);
      __builtin_amdgcn_sched_barrier(0);  // slot order, as in the loop
    }
    __syncthreads();
    // (slice, chunk) of the look-ahead chunk i + D in skip order, advanced
    // one per step (the dense order computes its columns directly)
    int la_sl = D / nchu, la_c = D % nchu;
    const int iters = (total + U - 1) / U;  // loop iterations of U steps
    for (int it = 0; it < iters; ++it) {
#pragma unroll
      for (int q = 0; q < U; ++q) {
        const int i = it * U + q;
        if (q % SC == 0) stage_load(i / SC + 1);  // the next stage, during this one
        step(ring[q % D], i, q == U - 1);
        wload(ring[q % D], i + D, la_sl, la_c);
        if constexpr (LIST) {
          ++la_c;
          const bool wrap = la_c == nchu;
          la_c = wrap ? 0 : la_c;
          la_sl += wrap ? 1 : 0;
        }
        if (q % SC == SC - 1) {
          stage_store(i / SC + 1);
          __syncthreads();  // next stage staged; this stage's readers done
        }
        __builtin_amdgcn_sched_barrier(0);  // keep the steps in order
      }
    }
  };
  if (use_list) run(std::true_type{}, std::false_type{});
  else if (nchu % GroupShape<MT>::U == 0) run(std::false_type{}, std::true_type{});
  else run(std::false_type{}, std::false_type{});

  if (!pvalid) return;
  const int g = lane >> 4, rl = lane & 15;
  const int64_t col = p * kPanel + rl;
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int64_t row = mt * 16 + 4 * g + v;
      if (row < a.M && col < a.N) fc_store<DT>(a, row, col, sum[mt][v]);
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

// Packs w[n][k] into the dense layout: vector v = (panel, chunk, column j,
// group g) holds w[16 panel + j][32 chunk + 8 g + 0..7], zero past n and k.
__global__ void fc_pack_dense_kernel(const uint16_t *__restrict__ w, uint16_t *__restrict__ wd,
                                     int64_t K, int64_t N, int64_t chunks, int64_t vecs) {
  for (int64_t v = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; v < vecs;
       v += (int64_t)gridDim.x * blockDim.x) {
    const int64_t g = v & 3, j = (v >> 2) % kPanel, pc = (v >> 2) / kPanel;
    const int64_t c = pc % chunks, p = pc / chunks;
    const int64_t n = p * kPanel + j, k0 = c * kCh + 8 * g;
    uint16_t t[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) t[i] = n < N && k0 + i < K ? w[n * K + k0 + i] : (uint16_t)0;
    uint4 out;
    __builtin_memcpy(&out, t, 16);
    *reinterpret_cast<uint4 *>(wd + 8 * v) = out;
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
  if (skip)
    return xvec ? launch_mt<DT, true, true>(mt, grid, st, a)
                : launch_mt<DT, true, false>(mt, grid, st, a);
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

// Skip layout, then the dense layout (k rounded up to whole 32-k chunks).
size_t fc_skip_layout_bytes(const sparoa_fc_desc &d) {
  return (size_t)cdiv(d.n, kPanel) * kPanel * (size_t)d.k * (size_t)elem_size(d.dtype);
}

size_t fc_packed_bytes(const sparoa_fc_desc &d) {
  return fc_skip_layout_bytes(d) +
         (size_t)cdiv(d.n, kPanel) * kPanel * (size_t)(cdiv(d.k, kCh) * kCh) *
             (size_t)elem_size(d.dtype);
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
  const int64_t chunks = cdiv(d.k, kCh);
  const int64_t vecs = panels * chunks * kPanel * 4;  // 16-byte vectors of the dense layout
  blocks = std::min<int64_t>(cdiv(vecs, 256), 8192);
  hipLaunchKernelGGL(fc_pack_dense_kernel, dim3((unsigned)blocks), dim3(256), 0, stream,
                     static_cast<const uint16_t *>(w_nk),
                     reinterpret_cast<uint16_t *>(static_cast<char *>(w_packed) +
                                                  fc_skip_layout_bytes(d)),
                     d.k, d.n, chunks, vecs);
  SPAROA_LAUNCH_CHECK("fc_pack_dense_kernel");
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
  a.wd = static_cast<const char *>(w_packed) + fc_skip_layout_bytes(d);
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
  a.wd = static_cast<const char *>(w_packed) + fc_skip_layout_bytes(d);
  a.bias = static_cast<const char *>(bias);
  a.residual = static_cast<const char *>(residual);
  a.y = static_cast<char *>(y);
  a.mask = nullptr;
  a.executed = nullptr;
  a.M = d.m; a.K = d.k; a.N = d.n; a.slice = slice_for(d);
  a.act = act;
  a.route = route;
  a.route.counts = nullptr;
  a.mcounts = counts;
  a.mmask = mask;
  const int mt = (int)cdiv(d.m, 16);
  dim3 grid((unsigned)cdiv(d.n, kPanel));
  const bool ok = d.dtype == SPAROA_BF16
                      ? launch_mt<SPAROA_BF16, true, true, true>(mt, grid, stream, a)
                      : launch_mt<SPAROA_F16, true, true, true>(mt, grid, stream, a);
  if (!ok) return fail(SPAROA_ERR_UNSUPPORTED, "fc bandwidth path: m");
  SPAROA_LAUNCH_CHECK("fc_bw_kernel (self-measuring)");
  return SPAROA_OK;
}

int fc_bw_group_key(const sparoa_fc_desc &d) {
  return fc_bw_self_measures(d) ? (int)d.dtype * 8 + (int)cdiv(d.m, 16) : -1;
}

sparoa_status launch_fc_bw_measured_group(const FcBwJob *jobs, int n, hipStream_t stream) {
  if (n < 1 || n > kGroupMax) return fail(SPAROA_ERR_INVALID_ARG, "fc group: size");
  const int key = fc_bw_group_key(jobs[0].d);
  FcBwGroup g;
  g.n = n;
  int64_t wg = 0;
  for (int j = 0; j < n; ++j) {
    const FcBwJob &o = jobs[j];
    if (fc_bw_group_key(o.d) != key || key < 0)
      return fail(SPAROA_ERR_INVALID_ARG, "fc group: mixed dtypes or row tiles");
    FcBwArgs &a = g.op[j];
    a.x = static_cast<const char *>(o.x);
    a.wp = static_cast<const char *>(o.w_packed);
    a.wd = static_cast<const char *>(o.w_packed) + fc_skip_layout_bytes(o.d);
    a.bias = static_cast<const char *>(o.bias);
    a.residual = static_cast<const char *>(o.residual);
    a.y = static_cast<char *>(o.y);
    a.mask = nullptr;
    a.executed = nullptr;
    a.M = o.d.m; a.K = o.d.k; a.N = o.d.n; a.slice = slice_for(o.d);
    a.act = o.act;
    a.route = o.route;
    a.route.counts = nullptr;
    a.mcounts = o.counts;
    a.mmask = o.mask;
    g.start[j] = (int)wg;
    wg += cdiv(cdiv(o.d.n, kPanel), (int64_t)GroupShape<1>::NW);  // a wave per panel
    if (wg > (int64_t)1 << 30) return fail(SPAROA_ERR_UNSUPPORTED, "fc group: too many panels");
  }
  g.start[n] = (int)wg;
  const dim3 grid((unsigned)wg), block(64 * GroupShape<1>::NW);
  const bool bf = jobs[0].d.dtype == SPAROA_BF16;
  switch ((int)cdiv(jobs[0].d.m, 16)) {
#define SPAROA_FCG(MT)                                                                        \
  case MT:                                                                                    \
    if (bf)                                                                                   \
      hipLaunchKernelGGL((fc_bw_measured_group<SPAROA_BF16, MT>), grid, block, 0, stream, g); \
    else                                                                                      \
      hipLaunchKernelGGL((fc_bw_measured_group<SPAROA_F16, MT>), grid, block, 0, stream, g);  \
    break;
    SPAROA_FCG(1)
    SPAROA_FCG(2)
    SPAROA_FCG(3)
    SPAROA_FCG(4)
#undef SPAROA_FCG
    default: return fail(SPAROA_ERR_UNSUPPORTED, "fc group: m");
  }
  SPAROA_LAUNCH_CHECK("fc_bw_measured_group");
  return SPAROA_OK;
}

}  // namespace sparoa
