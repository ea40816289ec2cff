// Count commit of an output measurement fused into a producer kernel: the
// work-groups' zero counts and nonzero-block counts reach the sparoa_counts of
// the output without one same-address atomic per work-group.
#pragma once

#include <hip/hip_runtime.h>

#include "sparoa.h"

namespace sparoa {

// Words of the grouped count commit: kOmGroups groups x 2 counters, one
// 128-byte line each.
constexpr int kOmGroups = 8;
constexpr int kOmDirectMax = 64;   // grids up to this many work-groups commit directly
static_assert(2 * kOmGroups * 128 == SPAROA_COMMIT_WORDS_BYTES, "commit word layout");

// Adds a work-group's zero count and nonzero-block count into counts
// (zero_blocks starts at nb).  Same-address atomics serialise device-wide
// (13-17 ns per work-group measured with one atomic per counter), so with
// `words` (the caller's zeroed count-commit words) work-group b of nwg is
// a member of group b % kOmGroups: each member adds (1 << 40) + its count to
// its group's word with one returning atomic, and the member whose add
// completes the group adds the group's total to counts and clears the word
// for the next call.  Without `words`, or for a grid of at most
// kOmDirectMax work-groups: one atomic per counter per work-group (the words
// are left untouched).
__device__ __forceinline__ void om_commit(uint32_t zeros, uint32_t nz, sparoa_counts *counts,
                                          unsigned long long *words, int64_t b, int64_t nwg) {
  __shared__ uint32_t part[2][16];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    zeros += __shfl_xor(zeros, o, 64);
    nz += __shfl_xor(nz, o, 64);
  }
  if (lane == 0) {
    part[0][wave] = zeros;
    part[1][wave] = nz;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    unsigned long long z = 0, n = 0;
    for (int i = 0; i < (int)(blockDim.x >> 6); ++i) {
      z += part[0][i];
      n += part[1][i];
    }
    // small grids commit directly: the ticket's returning atomic is a memory
    // round trip on every work-group's path (about 1 us), more than up to 64
    // work-groups' serialised same-address atomics (measured: 64 work-groups
    // 1 us faster direct, 98 work-groups 0.25 us slower)
    if (!words || nwg <= kOmDirectMax) {
      if (z) atomicAdd((unsigned long long *)&counts->zeros, z);
      if (n) atomicAdd((unsigned long long *)&counts->zero_blocks, 0ull - n);
      return;
    }
    constexpr unsigned long long kTicket = 1ull << 40;  // sums < 2^40, members < 2^24
    const int64_t g = b % kOmGroups;
    const unsigned long long members =
        (unsigned long long)(nwg / kOmGroups + (g < nwg % kOmGroups ? 1 : 0));
    unsigned long long *wz = words + g * 32, *wn = words + g * 32 + 16;
    const unsigned long long oz = atomicAdd(wz, kTicket + z);
    const unsigned long long on = atomicAdd(wn, kTicket + n);
    if ((oz >> 40) == members - 1) {
      const unsigned long long tz = (oz & (kTicket - 1)) + z;
      if (tz) atomicAdd((unsigned long long *)&counts->zeros, tz);
      atomicExch(wz, 0ull);
    }
    if ((on >> 40) == members - 1) {
      const unsigned long long tn = (on & (kTicket - 1)) + n;
      if (tn) atomicAdd((unsigned long long *)&counts->zero_blocks, 0ull - tn);
      atomicExch(wn, 0ull);
    }
  }
}

}  // namespace sparoa
