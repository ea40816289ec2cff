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
  const uint64_t wz = wave_sum(zeros);
  const uint64_t wn = wave_sum((uint64_t)newly);
  if ((threadIdx.x & 63) == 0) {
    if (wz) {
      atomicAdd((unsigned long long *)&counts->zeros, (unsigned long long)wz);
      if (per_sample) atomicAdd((unsigned long long *)(per_sample + s), (unsigned long long)wz);
    }
    if (wn) atomicAdd((unsigned long long *)&counts->zero_blocks, (unsigned long long)(0ull - wn));
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

sparoa_status launch_measure(const void *x, sparoa_dtype dt, int64_t rows, int64_t cols,
                             int64_t block_rows, int64_t block_cols, int64_t samples,
                             sparoa_counts *counts, uint32_t *mask, uint64_t *per_sample,
                             hipStream_t stream) {
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

  {
    const int64_t work = words > S ? words : S;
    const int64_t g = work < 1 ? 1 : (cdiv(work, 256) < 1024 ? cdiv(work, 256) : 1024);
    hipLaunchKernelGGL(measure_init, dim3((unsigned)g), dim3(256), 0, stream, counts,
                       (uint64_t)(rows * cols), (uint64_t)nb, mask, words, per_sample,
                       per_sample ? S : 0);
    SPAROA_LAUNCH_CHECK("measure_init");
  }

  const bool vec = cols % vw == 0 && (!want_mask || bc % vw == 0 || vw % bc == 0);
  const int V = vec ? vw : 1;
  const int64_t cpb = cdiv(br < rs ? br : rs, kRowChunk);   // row chunks per block row
  const int64_t items_s = nbr_s * cpb * (cols / V);
  int64_t gx = cdiv(items_s, (int64_t)kThreads);
  const int64_t cap = cdiv(2048, S);
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
