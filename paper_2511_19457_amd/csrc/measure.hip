// Sparsity measurement (SparOA Section 3.1, Eq. 1): zero count, nonzero-block
// bitmap and per-sample zero counts of an activation tensor, in one coalesced
// pass over HBM.
//
// Work item = (block row, chunk of up to 4 of its rows, group of V consecutive
// columns).  A lane loads the V elements of its group (one 16-byte load for
// V = 16 / element size) in each row of its chunk, tests the raw magnitude
// bits (+0 and -0 are zero; subnormals, NaN and Inf are not; no float
// compare, so FTZ/DAZ cannot matter) and keeps a V-bit "nonzero seen" flag.  Consecutive lanes hold
// consecutive items, so a wave covers a contiguous run of bitmap bits: the
// wave ORs its bits per bitmap word across lanes (shuffles) and one lane per
// word issues the atomicOr.  The old word returned by atomicOr tells which
// bits were newly set, so each nonzero block is counted exactly once and the
// zero-block count needs no second pass.  Integer sums are order-independent,
// so every output is deterministic.
//
// Counts leave a work-group through one atomic per counter: atomics on one
// address serialise device-wide (~10 ns each on MI355X), so grids stay at a
// few hundred work-groups that loop over the tensor.
#include "commit.h"
#include "common.h"

namespace sparoa {
namespace {

constexpr int kThreads = 256;
constexpr int kUnroll = 4;    // items per lane in flight
constexpr int kRowChunk = 4;  // rows of one block handled by one lane

__global__ void measure_init(sparoa_counts *counts, uint64_t numel, uint64_t nb, uint32_t *mask,
                             int64_t words, uint64_t *per_sample, int64_t samples) {
  int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  int64_t stride = (int64_t)gridDim.x * blockDim.x;
  if (i == 0) {
    counts->zeros = 0;
    counts->numel = numel;
    counts->zero_blocks = nb;  // nonzero blocks are subtracted as they are found
    counts->num_blocks = nb;
  }
  for (int64_t j = i; j < words; j += stride) mask[j] = 0u;
  for (int64_t j = i; j < samples; j += stride) per_sample[j] = 0ull;
}

__device__ __forceinline__ uint32_t wave_or(uint32_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v |= __shfl_xor(v, o, 64);
  return v;
}

__device__ __forceinline__ uint64_t wave_sum(uint64_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Adds the work-group's zero count and nonzero-block count to the totals
// (and the zero count to a per-sample slot): the waves' sums meet in LDS and
// one lane issues one atomic per counter.  Every thread must call it.
template <int NT>
__device__ __forceinline__ void wg_commit(uint64_t zeros, uint64_t nonzero, sparoa_counts *counts,
                                          uint64_t *sample_zeros) {
  __shared__ unsigned long long part[2][NT / 64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint64_t wz = wave_sum(zeros), wn = wave_sum(nonzero);
  if (lane == 0) {
    part[0][wave] = wz;
    part[1][wave] = wn;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    unsigned long long z = 0, n = 0;
#pragma unroll
    for (int i = 0; i < NT / 64; ++i) {
      z += part[0][i];
      n += part[1][i];
    }
    if (z) {
      atomicAdd((unsigned long long *)&counts->zeros, z);
      if (sample_zeros) atomicAdd((unsigned long long *)sample_zeros, z);
    }
    if (n) atomicAdd((unsigned long long *)&counts->zero_blocks, 0ull - n);
  }
}

// ORs (word, bits) pairs of the lanes into the bitmap, one atomic per distinct
// word; returns (in the issuing lanes) how many bits were newly set.
__device__ __forceinline__ uint32_t wave_flush(bool has, int word, uint32_t bits,
                                               uint32_t *mask) {
  const int lane = threadIdx.x & 63;
  uint32_t newly = 0;
  uint64_t pending = __ballot(has);
  while (pending) {
    int leader = __ffsll((unsigned long long)pending) - 1;
    int w = __shfl(word, leader, 64);
    bool mine = has && word == w;
    uint32_t v = wave_or(mine ? bits : 0u);
    if (lane == leader) {
      uint32_t old = atomicOr(mask + w, v);
      newly += __popc(v & ~old);
    }
    pending &= ~__ballot(mine);
  }
  return newly;
}

template <int ESZ>
struct Raw;
template <>
struct Raw<2> {
  using T = uint16_t;
  static constexpr uint32_t kMag = 0x7fffu;
};
template <>
struct Raw<4> {
  using T = uint32_t;
  static constexpr uint32_t kMag = 0x7fffffffu;
};

// Loads the V elements at p and returns a V-bit mask of nonzero elements.
template <int ESZ, int V>
__device__ __forceinline__ uint32_t nonzero_bits(const char *p) {
  uint32_t nz = 0;
  if constexpr (V * ESZ == 16) {
    const uint4 q = *reinterpret_cast<const uint4 *>(p);
    const uint32_t w[4] = {q.x, q.y, q.z, q.w};
    if constexpr (ESZ == 2) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        nz |= ((w[i] & 0x7fffu) != 0u) << (2 * i);
        nz |= ((w[i] & 0x7fff0000u) != 0u) << (2 * i + 1);
      }
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) nz |= ((w[i] & 0x7fffffffu) != 0u) << i;
    }
  } else {
    static_assert(V == 1, "vector width");
    nz = (*reinterpret_cast<const typename Raw<ESZ>::T *>(p) & Raw<ESZ>::kMag) != 0u;
  }
  return nz;
}

// The V elements of one lanebit item (one block of 1 x V): a 16-byte vector,
// or two of them for fp32 blocks of 8 (32 contiguous bytes per lane).
template <int ESZ, int V>
__device__ __forceinline__ uint32_t item_nonzero_bits(const char *p) {
  if constexpr (V * ESZ == 32)
    return nonzero_bits<ESZ, V / 2>(p) | (nonzero_bits<ESZ, V / 2>(p + 16) << (V / 2));
  else
    return nonzero_bits<ESZ, V>(p);
}

// grid = (x: work-groups per sample, y: samples).  Sample s covers rows
// [s*rs, s*rs + rs); its block rows are numbered s*nbr_s + local index.
// Work item = (block row, chunk of kRowChunk rows inside it, column group):
// chunks of one block OR their flags into the same bitmap bits, so tall
// blocks still spread over many lanes.  The kUnroll item slots of a lane are
// a grid-width apart, keeping each wave on a contiguous run of items.
template <int ESZ, int V>
__global__ __launch_bounds__(kThreads) void measure_main(
    const char *__restrict__ x, int64_t cols, int64_t rs, int64_t br, int64_t bc, int64_t nbc,
    int64_t nbr_s, int64_t cpb, int64_t gpr, uint32_t *__restrict__ mask, sparoa_counts *counts,
    uint64_t *per_sample) {
  const int64_t s = blockIdx.y;
  const int64_t per_block = cpb * gpr;
  const int64_t items = nbr_s * per_block;
  const int64_t row_bytes = cols * ESZ;
  const int64_t slot = (int64_t)gridDim.x * kThreads;
  uint64_t zeros = 0;
  uint32_t newly = 0;
  for (int64_t base = (int64_t)blockIdx.x * kThreads; base < items;
       base += slot * kUnroll) {
    uint32_t nz[kUnroll];
    int64_t bitpos[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t item = base + u * slot + threadIdx.x;
      nz[u] = 0;
      bitpos[u] = -1;
      if (item < items) {
        const int64_t bi = item / per_block, rem = item - bi * per_block;
        const int64_t rc = rem / gpr, g = rem - rc * gpr;
        const int64_t blk0 = s * rs + bi * br;
        const int64_t r0 = blk0 + rc * kRowChunk;
        const int64_t r1 = min(min(r0 + kRowChunk, blk0 + br), s * rs + rs);
        const char *p = x + r0 * row_bytes + g * V * ESZ;
#pragma unroll
        for (int64_t r = r0; r < r1; ++r, p += row_bytes) {
          const uint32_t b = nonzero_bits<ESZ, V>(p);
          zeros += V - __popc(b);
          nz[u] |= b;
        }
        bitpos[u] = (s * nbr_s + bi) * nbc + (g * V) / bc;
      }
    }
    if (mask) {
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        int word = 0;
        uint32_t lo = 0, hi = 0;
        if (bitpos[u] >= 0) {
          uint32_t lbits;
          if (V == 1 || bc % V == 0) {  // the V columns lie in one block
            lbits = nz[u] != 0u;
          } else {  // V % bc == 0: V / bc blocks per lane
            lbits = 0;
            const uint32_t bm = (1u << bc) - 1u;
            for (int j = 0; j < V / bc; ++j) lbits |= ((nz[u] >> (j * bc)) & bm ? 1u : 0u) << j;
          }
          word = (int)(bitpos[u] >> 5);
          const uint64_t sh = (uint64_t)lbits << (bitpos[u] & 31);
          lo = (uint32_t)sh;
          hi = (uint32_t)(sh >> 32);
        }
        newly += wave_flush(lo != 0u, word, lo, mask);
        newly += wave_flush(hi != 0u, word + 1, hi, mask);
      }
    }
  }
  wg_commit<kThreads>(zeros, (uint64_t)newly, counts, per_sample ? per_sample + s : nullptr);
}

// One bitmap bit per lane (block = 1 row x V columns, V = elements per
// 16-byte vector): item index == block index, so the 64 items of a wave slot
// are two whole bitmap words.  The wave ballots its bits and two lanes store
// the words: no atomics, and the bitmap needs no clearing.  The grid's slots
// start at multiples of 64 items, which keeps the words aligned.
constexpr int kLanebitThreads = 1024;  // one work-group per CU, 16 waves
constexpr int kLanebitUnroll = 4;

// Work-group `bid` of `nblk` measuring one tensor.
template <int ESZ, int V>
__device__ __forceinline__ void lanebit_pass(const char *__restrict__ x, int64_t items,
                                             int64_t words, uint32_t *__restrict__ mask,
                                             sparoa_counts *counts, int64_t bid, int64_t nblk,
                                             unsigned long long *commit = nullptr) {
  constexpr int NT = kLanebitThreads;
  const int lane = threadIdx.x & 63;
  const int64_t slot = nblk * NT;
  uint64_t zeros = 0, nonzero = 0;
  for (int64_t base = bid * NT; base < items; base += slot * kLanebitUnroll) {
    // unconditional loads (items past the end re-read the last item and are
    // masked), so all kLanebitUnroll stay in flight
    uint32_t nz[kLanebitUnroll];
#pragma unroll
    for (int u = 0; u < kLanebitUnroll; ++u) {
      const int64_t item = base + u * slot + threadIdx.x;
      nz[u] = item_nonzero_bits<ESZ, V>(x + min(item, items - 1) * (V * ESZ));
    }
#pragma unroll
    for (int u = 0; u < kLanebitUnroll; ++u) {
      const bool valid = base + u * slot + threadIdx.x < items;
      nz[u] = valid ? nz[u] : 0u;
      zeros += valid ? (uint64_t)(V - __popc(nz[u])) : 0ull;
    }
#pragma unroll
    for (int u = 0; u < kLanebitUnroll; ++u) {
      const uint64_t bal = __ballot(nz[u] != 0u);
      const int64_t w0 = (base + u * slot + (threadIdx.x & ~63)) >> 5;
      if (lane == 0 && w0 < words) mask[w0] = (uint32_t)bal;
      if (lane == 32 && w0 + 1 < words) mask[w0 + 1] = (uint32_t)(bal >> 32);
      nonzero += lane == 0 ? (uint64_t)__popcll(bal) : 0ull;
    }
  }
  // with commit words: ticketed commits over 16 addresses instead of one
  // same-address atomic per counter per work-group
  if (commit) om_commit((uint32_t)zeros, (uint32_t)nonzero, counts, commit, bid, nblk);
  else wg_commit<NT>(zeros, nonzero, counts, nullptr);
}

template <int ESZ, int V>
__global__ __launch_bounds__(kLanebitThreads) void measure_lanebit(const char *__restrict__ x,
                                                                   int64_t items, int64_t words,
                                                                   uint32_t *__restrict__ mask,
                                                                   sparoa_counts *counts,
                                                                   unsigned long long *commit) {
  SPAROA_ARGS_UP_FRONT("s"(x), "s"(items), "s"(words), "s"(mask), "s"(counts), "s"(commit),
                       "s"(gridDim.x));
  lanebit_pass<ESZ, V>(x, items, words, mask, counts, blockIdx.x, gridDim.x, commit);
}

// One bitmap bit per row (block = 1 row x block_cols >= cols) for rows
// narrower than one 16-byte vector, e.g. a 3-channel image in NHWC: a lane
// owns 8 consecutive rows, i.e. 8 * cols contiguous elements starting at a
// multiple of 16 bytes (cols * ESZ / 2 vectors), so a wave owns 512 rows =
// 16 whole bitmap words: no atomics on the bitmap and no clearing.  The one
// lane whose rows run past the end reads its elements one at a time (the
// tensor's byte size need not be a multiple of 16).
template <int ESZ>
__global__ __launch_bounds__(kLanebitThreads) void measure_rowbit(const char *__restrict__ x,
                                                                  int64_t rows, int cols,
                                                                  int64_t words,
                                                                  uint32_t *__restrict__ mask,
                                                                  sparoa_counts *counts,
                                                                  unsigned long long *commit) {
  SPAROA_ARGS_UP_FRONT("s"(x), "s"(rows), "s"(cols), "s"(words), "s"(mask), "s"(counts),
                       "s"(commit), "s"(gridDim.x));
  constexpr int EPV = 16 / ESZ;  // elements per 16-byte vector
  const int lane = threadIdx.x & 63;
  const int nv = cols * ESZ / 2;  // vectors per 8 rows
  const int64_t groups = (rows + 7) / 8;
  const int64_t numel = rows * cols;
  const int64_t stride = (int64_t)gridDim.x * kLanebitThreads;
  uint64_t zeros = 0, nonzero = 0;
  // wave-uniform loop: a wave's 64 groups start at a multiple of 64
  for (int64_t base = (int64_t)blockIdx.x * kLanebitThreads + (threadIdx.x & ~63);
       base < groups; base += stride) {
    const int64_t gi = base + lane;
    const int64_t e0 = gi * 8 * cols;
    uint32_t rowbits = 0;
    if (gi < groups) {
      int r = 0, k = 0;  // row within the group, column within the row
      if (e0 + 8 * cols <= numel) {
        const char *p = x + e0 * ESZ;
        for (int v = 0; v < nv; ++v) {
          const uint32_t nzv = nonzero_bits<ESZ, EPV>(p + 16 * v);
          zeros += (uint64_t)(EPV - __popc(nzv));
#pragma unroll
          for (int e = 0; e < EPV; ++e) {
            rowbits |= ((nzv >> e) & 1u) << r;
            if (++k == cols) { k = 0; ++r; }
          }
        }
      } else {
        for (int64_t e = e0; e < numel; ++e) {
          const uint32_t nz = nonzero_bits<ESZ, 1>(x + e * ESZ);
          zeros += 1u - nz;
          rowbits |= nz << r;
          if (++k == cols) { k = 0; ++r; }
        }
      }
    }
    nonzero += (uint64_t)__popc(rowbits);
    // lanes 4q .. 4q + 3 hold the 32 rows of bitmap word base / 4 + q
    const uint32_t word = rowbits | (__shfl_down(rowbits, 1, 64) << 8) |
                          (__shfl_down(rowbits, 2, 64) << 16) |
                          (__shfl_down(rowbits, 3, 64) << 24);
    const int64_t w = base / 4 + lane / 4;
    if ((lane & 3) == 0 && w < words) mask[w] = word;
  }
  if (commit) om_commit((uint32_t)zeros, (uint32_t)nonzero, counts, commit, blockIdx.x, gridDim.x);
  else wg_commit<kLanebitThreads>(zeros, nonzero, counts, nullptr);
}

// Several tensors of one element size in the lanebit layout, one launch:
// work-groups are dealt to the tensors in proportion to their size.
struct LanebitGroup {
  int n;
  int wg_begin[kGroupMax + 1];
  const char *x[kGroupMax];
  int64_t items[kGroupMax];
  uint32_t *mask[kGroupMax];
  sparoa_counts *counts[kGroupMax];
};

template <int V>
__global__ void measure_init_group(LanebitGroup g) {
  const int j = threadIdx.x;
  if (j < g.n) {
    g.counts[j]->zeros = 0;
    g.counts[j]->numel = (uint64_t)g.items[j] * V;
    g.counts[j]->zero_blocks = (uint64_t)g.items[j];  // nonzero blocks are subtracted
    g.counts[j]->num_blocks = (uint64_t)g.items[j];
  }
}

template <int ESZ, int V>
__global__ __launch_bounds__(kLanebitThreads) void measure_lanebit_group(LanebitGroup g) {
  // this work-group's tensor: the starts at or below blockIdx.x, counted
  // over fixed indices (their loads are issued together, not one per step)
  int j = 0;
#pragma unroll
  for (int q = 1; q < kGroupMax; ++q) j += (q < g.n && (int)blockIdx.x >= g.wg_begin[q]) ? 1 : 0;
  lanebit_pass<ESZ, V>(g.x[j], g.items[j], (g.items[j] + 31) / 32, g.mask[j], g.counts[j],
                       blockIdx.x - g.wg_begin[j], g.wg_begin[j + 1] - g.wg_begin[j]);
}

// The lanebit layout measured by one work-group that also writes all four
// counts (no init launch, no atomics): for small tensors, where two launches
// cost more than the pass.  Each wave reduces its slots in registers; the
// waves' sums meet in LDS.
template <int ESZ, int V>
__global__ __launch_bounds__(1024) void measure_lanebit_wg(const char *__restrict__ x,
                                                          int64_t items, int64_t words,
                                                          uint32_t *__restrict__ mask,
                                                          sparoa_counts *counts) {
  constexpr int NT = 1024, U = 8;
  __shared__ unsigned long long part[2][NT / 64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint64_t zeros = 0, nonzero = 0;
  for (int64_t base = 0; base < items; base += (int64_t)NT * U) {
    uint32_t nz[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {  // unconditional loads, masked past the end
      const int64_t item = base + u * NT + threadIdx.x;
      nz[u] = item_nonzero_bits<ESZ, V>(x + min(item, items - 1) * (V * ESZ));
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t w0 = (base + u * NT + (threadIdx.x & ~63)) >> 5;
      const bool valid = base + u * NT + threadIdx.x < items;
      const uint32_t b = valid ? nz[u] : 0u;
      zeros += valid ? (uint64_t)(V - __popc(b)) : 0ull;
      const uint64_t bal = __ballot(b != 0u);
      if (lane == 0 && w0 < words) mask[w0] = (uint32_t)bal;
      if (lane == 32 && w0 + 1 < words) mask[w0 + 1] = (uint32_t)(bal >> 32);
      nonzero += lane == 0 ? (uint64_t)__popcll(bal) : 0ull;
    }
  }
  const uint64_t wz = wave_sum(zeros), wn = wave_sum(nonzero);
  if (lane == 0) {
    part[0][wave] = wz;
    part[1][wave] = wn;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    unsigned long long z = 0, n = 0;
#pragma unroll
    for (int i = 0; i < NT / 64; ++i) {
      z += part[0][i];
      n += part[1][i];
    }
    counts->zeros = z;
    counts->numel = (uint64_t)items * V;
    counts->zero_blocks = (uint64_t)items - n;
    counts->num_blocks = (uint64_t)items;
  }
}

// Column strips: a single block row covering all rows, one column per block
// (the "column is zero in every row" bitmap).  A work-group owns 64 column
// groups (64 V columns = 2 V whole bitmap words); its 4 waves take every
// 4th row of the strip, their flags are ORed in LDS, and wave 0 assembles and
// stores the words: no atomics, no clearing.
template <int ESZ, int V>
__global__ __launch_bounds__(kThreads) void measure_strips(const char *__restrict__ x,
                                                           int64_t rows, int64_t cols,
                                                           int64_t words,
                                                           uint32_t *__restrict__ mask,
                                                           sparoa_counts *counts) {
  static_assert(32 % V == 0, "lanes per word");
  __shared__ uint32_t flags[kThreads];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t gpr = cols / V;
  const int64_t g = (int64_t)blockIdx.x * 64 + lane;
  const int64_t row_bytes = cols * ESZ;
  uint64_t zeros = 0;
  uint32_t nz = 0;
  if (g < gpr) {
    const char *p = x + g * V * ESZ;
    int64_t r = wave;
    for (; r + 12 < rows; r += 16) {  // four rows of this wave in flight
      const uint32_t b0 = nonzero_bits<ESZ, V>(p + r * row_bytes);
      const uint32_t b1 = nonzero_bits<ESZ, V>(p + (r + 4) * row_bytes);
      const uint32_t b2 = nonzero_bits<ESZ, V>(p + (r + 8) * row_bytes);
      const uint32_t b3 = nonzero_bits<ESZ, V>(p + (r + 12) * row_bytes);
      zeros += 4 * V - __popc(b0) - __popc(b1) - __popc(b2) - __popc(b3);
      nz |= b0 | b1 | b2 | b3;
    }
    for (; r < rows; r += 4) {
      const uint32_t b = nonzero_bits<ESZ, V>(p + r * row_bytes);
      zeros += V - __popc(b);
      nz |= b;
    }
  }
  flags[threadIdx.x] = nz;
  __syncthreads();
  uint64_t nonzero = 0;
  if (wave == 0) {
    const uint32_t f = flags[lane] | flags[64 + lane] | flags[128 + lane] | flags[192 + lane];
    constexpr int kLanesPerWord = 32 / V;
    uint32_t word = 0;
#pragma unroll
    for (int j = 0; j < kLanesPerWord; ++j) word |= __shfl(f, (lane & ~(kLanesPerWord - 1)) + j, 64) << (j * V);
    const int64_t w = ((int64_t)blockIdx.x * 64 + lane) / kLanesPerWord;
    if (lane % kLanesPerWord == 0 && w < words) {
      mask[w] = word;
      nonzero = __popc(word);
    }
  }
  wg_commit<kThreads>(zeros, nonzero, counts, nullptr);
}

// Column strips that fit one work-group (at most 16 x 64 column groups): 16
// waves in ceil(groups / 64) sets, the waves of a set taking interleaved
// rows; flags and counts combine in LDS and the work-group writes the bitmap
// and all four counts itself -- one launch, no atomics, no clearing.
template <int ESZ, int V>
__global__ __launch_bounds__(1024) void measure_strips_wg(const char *__restrict__ x, int64_t rows,
                                                           int64_t cols, int64_t words,
                                                           uint32_t *__restrict__ mask,
                                                           sparoa_counts *counts) {
  static_assert(32 % V == 0, "lanes per word");
  __shared__ uint32_t flags[16][64];
  __shared__ unsigned long long zsum[16], nzsum[16];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t gpr = cols / V;
  const int sets = (int)((gpr + 63) / 64);
  const int wps = 16 / sets;  // waves per set
  const int set = wave / wps, sub = wave - set * wps;
  const int64_t g = (int64_t)set * 64 + lane;
  const int64_t row_bytes = cols * ESZ;
  uint64_t zeros = 0;
  uint32_t nz = 0;
  if (set < sets && g < gpr) {
    const char *p = x + g * V * ESZ;
    int64_t r = sub;
    for (; r + 3 * wps < rows; r += 4 * wps) {  // four rows in flight
      const uint32_t b0 = nonzero_bits<ESZ, V>(p + r * row_bytes);
      const uint32_t b1 = nonzero_bits<ESZ, V>(p + (r + wps) * row_bytes);
      const uint32_t b2 = nonzero_bits<ESZ, V>(p + (r + 2 * wps) * row_bytes);
      const uint32_t b3 = nonzero_bits<ESZ, V>(p + (r + 3 * wps) * row_bytes);
      zeros += 4 * V - __popc(b0) - __popc(b1) - __popc(b2) - __popc(b3);
      nz |= b0 | b1 | b2 | b3;
    }
    for (; r < rows; r += wps) {
      const uint32_t b = nonzero_bits<ESZ, V>(p + r * row_bytes);
      zeros += V - __popc(b);
      nz |= b;
    }
  }
  flags[wave][lane] = nz;
  const uint64_t wz = wave_sum(zeros);
  if (lane == 0) zsum[wave] = wz;
  __syncthreads();
  uint64_t nonzero = 0;
  if (set < sets && sub == 0) {
    uint32_t f = 0;
    for (int i = 0; i < wps; ++i) f |= flags[wave + i][lane];
    constexpr int kLanesPerWord = 32 / V;
    uint32_t word = 0;
#pragma unroll
    for (int j = 0; j < kLanesPerWord; ++j)
      word |= __shfl(f, (lane & ~(kLanesPerWord - 1)) + j, 64) << (j * V);
    const int64_t w = ((int64_t)set * 64 + lane) / kLanesPerWord;
    if (lane % kLanesPerWord == 0 && w < words) {
      mask[w] = word;
      nonzero = __popc(word);
    }
  }
  const uint64_t wn = wave_sum(nonzero);
  if (lane == 0) nzsum[wave] = wn;
  __syncthreads();
  if (threadIdx.x == 0) {
    unsigned long long z = 0, n = 0;
    for (int i = 0; i < 16; ++i) {
      z += zsum[i];
      n += nzsum[i];
    }
    counts->zeros = z;
    counts->numel = (uint64_t)(rows * cols);
    counts->zero_blocks = (uint64_t)cols - n;
    counts->num_blocks = (uint64_t)cols;
  }
}

template <int ESZ, int V>
void launch_main(dim3 grid, hipStream_t st, const void *x, int64_t cols, int64_t rs, int64_t br,
                 int64_t bc, int64_t nbc, int64_t nbr_s, int64_t cpb, uint32_t *mask,
                 sparoa_counts *counts, uint64_t *per_sample) {
  hipLaunchKernelGGL((measure_main<ESZ, V>), grid, dim3(kThreads), 0, st,
                     static_cast<const char *>(x), cols, rs, br, bc, nbc, nbr_s, cpb, cols / V,
                     mask, counts, per_sample);
}

}  // namespace

bool measure_groupable(const MeasureJob &j) {
  const int vw = 16 / (int)elem_size(j.dt);
  return j.mask && j.cols % vw == 0 && j.block_rows == 1 && j.block_cols == vw;
}

sparoa_status launch_measure_group(const MeasureJob *jobs, int n, hipStream_t stream) {
  if (n < 1 || n > kGroupMax) return fail(SPAROA_ERR_INVALID_ARG, "measure group: size");
  const int esz = (int)elem_size(jobs[0].dt);
  LanebitGroup g;
  g.n = n;
  int64_t wg = 0;
  for (int j = 0; j < n; ++j) {
    const MeasureJob &m = jobs[j];
    if (!measure_groupable(m) || (int)elem_size(m.dt) != esz)
      return fail(SPAROA_ERR_INVALID_ARG, "measure group: layout or element size");
    g.wg_begin[j] = (int)wg;
    g.x[j] = static_cast<const char *>(m.x);
    g.items[j] = m.rows * (m.cols / (16 / esz));
    g.mask[j] = m.mask;
    g.counts[j] = m.counts;
    int64_t b = cdiv(g.items[j], (int64_t)kLanebitThreads);
    if (b > 256) b = 256;
    if (b < 1) b = 1;
    wg += b;
  }
  g.wg_begin[n] = (int)wg;
  if (esz == 2) {
    hipLaunchKernelGGL(measure_init_group<8>, dim3(1), dim3(64), 0, stream, g);
    SPAROA_LAUNCH_CHECK("measure_init_group");
    hipLaunchKernelGGL((measure_lanebit_group<2, 8>), dim3((unsigned)wg), dim3(kLanebitThreads), 0,
                       stream, g);
  } else {
    hipLaunchKernelGGL(measure_init_group<4>, dim3(1), dim3(64), 0, stream, g);
    SPAROA_LAUNCH_CHECK("measure_init_group");
    hipLaunchKernelGGL((measure_lanebit_group<4, 4>), dim3((unsigned)wg), dim3(kLanebitThreads), 0,
                       stream, g);
  }
  SPAROA_LAUNCH_CHECK("measure_lanebit_group");
  return SPAROA_OK;
}

sparoa_status launch_measure_counts8(const void *x, sparoa_dtype dt, int64_t rows, int64_t cols,
                                    sparoa_counts *counts, uint64_t *commit_words,
                                    hipStream_t stream) {
  if (cols % 8 != 0)
    return fail(SPAROA_ERR_INVALID_ARG, "counts-only measurement: cols % 8 == 0");
  // the lanebit layout with no bitmap words: item = block = 8 elements
  const int64_t items = rows * (cols / 8);
  const char *xc = static_cast<const char *>(x);
  const bool h = elem_size(dt) == 2;
  if (items <= 4096) {   // one work-group writes all four counts
    if (h)
      hipLaunchKernelGGL((measure_lanebit_wg<2, 8>), dim3(1), dim3(1024), 0, stream, xc, items,
                         (int64_t)0, (uint32_t *)nullptr, counts);
    else
      hipLaunchKernelGGL((measure_lanebit_wg<4, 8>), dim3(1), dim3(1024), 0, stream, xc, items,
                         (int64_t)0, (uint32_t *)nullptr, counts);
    SPAROA_LAUNCH_CHECK("measure_lanebit_wg");
    return SPAROA_OK;
  }
  int64_t gx = cdiv(items, (int64_t)kLanebitThreads);
  if (gx > 256) gx = 256;
  unsigned long long *cw = reinterpret_cast<unsigned long long *>(commit_words);
  if (h)
    hipLaunchKernelGGL((measure_lanebit<2, 8>), dim3((unsigned)gx), dim3(kLanebitThreads), 0,
                       stream, xc, items, (int64_t)0, (uint32_t *)nullptr, counts, cw);
  else
    hipLaunchKernelGGL((measure_lanebit<4, 8>), dim3((unsigned)gx), dim3(kLanebitThreads), 0,
                       stream, xc, items, (int64_t)0, (uint32_t *)nullptr, counts, cw);
  SPAROA_LAUNCH_CHECK("measure_lanebit");
  return SPAROA_OK;
}

sparoa_status launch_measure(const void *x, sparoa_dtype dt, int64_t rows, int64_t cols,
                             int64_t block_rows, int64_t block_cols, int64_t samples,
                             sparoa_counts *counts, uint32_t *mask, uint64_t *per_sample,
                             hipStream_t stream, bool preset, uint64_t *commit_words) {
  // commit words serve the layouts whose counts arrive preset
  unsigned long long *commit =
      preset ? reinterpret_cast<unsigned long long *>(commit_words) : nullptr;
  const int esz = (int)elem_size(dt);
  const int vw = 16 / esz;
  const bool want_mask = mask != nullptr;
  const int64_t br = want_mask ? block_rows : 1;
  const int64_t bc = want_mask ? block_cols : 1;
  const int64_t S = per_sample ? samples : 1;
  const int64_t rs = rows / S;
  const int64_t nbr_s = cdiv(rs, br);
  const int64_t nbc = cdiv(cols, bc);
  const int64_t nb = want_mask ? cdiv(rows, br) * nbc : 0;
  const int64_t words = want_mask ? cdiv(nb, 32) : 0;

  const bool vec = cols % vw == 0 && (!want_mask || bc % vw == 0 || vw % bc == 0);
  // fast paths that own whole bitmap words (no atomics, no clearing)
  // lanebit items: one 16-byte vector, or two for fp32 blocks of 8
  const int lv = (esz == 4 && bc == 8 && cols % 8 == 0) ? 8 : vw;
  const bool lanebit = want_mask && vec && br == 1 && bc == lv && !per_sample;
  const bool strips = want_mask && vec && bc == 1 && !per_sample && br >= rows;
  const bool rowbit = want_mask && br == 1 && bc >= cols && cols * esz < 16 && !per_sample;

  if (lanebit && rows * (cols / lv) <= 4096) {  // one work-group measures it all
    const int64_t items = rows * (cols / lv);
    if (esz == 2)
      hipLaunchKernelGGL((measure_lanebit_wg<2, 8>), dim3(1), dim3(1024), 0, stream,
                         static_cast<const char *>(x), items, words, mask, counts);
    else if (lv == 8)
      hipLaunchKernelGGL((measure_lanebit_wg<4, 8>), dim3(1), dim3(1024), 0, stream,
                         static_cast<const char *>(x), items, words, mask, counts);
    else
      hipLaunchKernelGGL((measure_lanebit_wg<4, 4>), dim3(1), dim3(1024), 0, stream,
                         static_cast<const char *>(x), items, words, mask, counts);
    SPAROA_LAUNCH_CHECK("measure_lanebit_wg");
    return SPAROA_OK;
  }
  if (strips && cols / vw <= 16 * 64) {  // one work-group measures it all
    if (esz == 2)
      hipLaunchKernelGGL((measure_strips_wg<2, 8>), dim3(1), dim3(1024), 0, stream,
                         static_cast<const char *>(x), rows, cols, words, mask, counts);
    else
      hipLaunchKernelGGL((measure_strips_wg<4, 4>), dim3(1), dim3(1024), 0, stream,
                         static_cast<const char *>(x), rows, cols, words, mask, counts);
    SPAROA_LAUNCH_CHECK("measure_strips_wg");
    return SPAROA_OK;
  }

  // counters the caller already set and no bitmap to clear: no init launch
  if (!(preset && (lanebit || strips || rowbit))) {
    const int64_t zw = (lanebit || strips || rowbit) ? 0 : words;   // words to clear
    const int64_t work = zw > S ? zw : S;
    const int64_t g = work < 1 ? 1 : (cdiv(work, 256) < 1024 ? cdiv(work, 256) : 1024);
    hipLaunchKernelGGL(measure_init, dim3((unsigned)g), dim3(256), 0, stream, counts,
                       (uint64_t)(rows * cols), (uint64_t)nb, mask, zw, per_sample,
                       per_sample ? S : 0);
    SPAROA_LAUNCH_CHECK("measure_init");
  }

  if (lanebit) {
    const int64_t items = rows * (cols / lv);
    // one work-group per CU where the tensor fills them (one item per lane
    // at the least); with commit words a work-group's commit costs two
    // returning atomics spread over 16 addresses, so a small tensor is spread
    // over as many compute units as it has 1024-item slots
    int64_t gx = cdiv(items, (int64_t)kLanebitThreads);
    if (gx > 256) gx = 256;
    if (esz == 2)
      hipLaunchKernelGGL((measure_lanebit<2, 8>), dim3((unsigned)gx), dim3(kLanebitThreads), 0,
                         stream, static_cast<const char *>(x), items, words, mask, counts, commit);
    else if (lv == 8)
      hipLaunchKernelGGL((measure_lanebit<4, 8>), dim3((unsigned)gx), dim3(kLanebitThreads), 0,
                         stream, static_cast<const char *>(x), items, words, mask, counts, commit);
    else
      hipLaunchKernelGGL((measure_lanebit<4, 4>), dim3((unsigned)gx), dim3(kLanebitThreads), 0,
                         stream, static_cast<const char *>(x), items, words, mask, counts, commit);
    SPAROA_LAUNCH_CHECK("measure_lanebit");
    return SPAROA_OK;
  }
  if (rowbit) {
    int64_t gx = cdiv(cdiv(rows, 8), (int64_t)kLanebitThreads);
    if (gx > 256) gx = 256;
    if (esz == 2)
      hipLaunchKernelGGL(measure_rowbit<2>, dim3((unsigned)gx), dim3(kLanebitThreads), 0, stream,
                         static_cast<const char *>(x), rows, (int)cols, words, mask, counts,
                         commit);
    else
      hipLaunchKernelGGL(measure_rowbit<4>, dim3((unsigned)gx), dim3(kLanebitThreads), 0, stream,
                         static_cast<const char *>(x), rows, (int)cols, words, mask, counts,
                         commit);
    SPAROA_LAUNCH_CHECK("measure_rowbit");
    return SPAROA_OK;
  }
  if (strips) {
    const int64_t gx = cdiv(cols / vw, 64);
    if (esz == 2)
      hipLaunchKernelGGL((measure_strips<2, 8>), dim3((unsigned)gx), dim3(kThreads), 0, stream,
                         static_cast<const char *>(x), rows, cols, words, mask, counts);
    else
      hipLaunchKernelGGL((measure_strips<4, 4>), dim3((unsigned)gx), dim3(kThreads), 0, stream,
                         static_cast<const char *>(x), rows, cols, words, mask, counts);
    SPAROA_LAUNCH_CHECK("measure_strips");
    return SPAROA_OK;
  }

  const int V = vec ? vw : 1;
  const int64_t cpb = cdiv(br < rs ? br : rs, kRowChunk);   // row chunks per block row
  const int64_t items_s = nbr_s * cpb * (cols / V);
  int64_t gx = cdiv(items_s, (int64_t)kThreads);
  const int64_t cap = cdiv(512, S);
  if (gx > cap) gx = cap;
  if (gx < 1) gx = 1;
  dim3 grid((unsigned)gx, (unsigned)S);
  if (esz == 2) {
    if (vec)
      launch_main<2, 8>(grid, stream, x, cols, rs, br, bc, nbc, nbr_s, cpb, mask, counts, per_sample);
    else
      launch_main<2, 1>(grid, stream, x, cols, rs, br, bc, nbc, nbr_s, cpb, mask, counts, per_sample);
  } else {
    if (vec)
      launch_main<4, 4>(grid, stream, x, cols, rs, br, bc, nbc, nbr_s, cpb, mask, counts, per_sample);
    else
      launch_main<4, 1>(grid, stream, x, cols, rs, br, bc, nbc, nbr_s, cpb, mask, counts, per_sample);
  }
  SPAROA_LAUNCH_CHECK("measure_main");
  return SPAROA_OK;
}

}  // namespace sparoa
