// Internal declarations shared by the HIP sources of libsparoa.so.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <map>
#include <mutex>
#include <string>
#include <tuple>

#include "sparoa.h"

namespace sparoa {

// Thread-local error message plumbing (defined in abi.cpp).
sparoa_status fail(sparoa_status s, const std::string &msg);
sparoa_status hip_fail(hipError_t e, const char *what);

#define SPAROA_HIP_CHECK(call)                                  \
  do {                                                          \
    hipError_t e_ = (call);                                     \
    if (e_ != hipSuccess) return ::sparoa::hip_fail(e_, #call); \
  } while (0)

// Checks the launch of the kernel just enqueued.
#define SPAROA_LAUNCH_CHECK(what)                               \
  do {                                                          \
    hipError_t e_ = hipGetLastError();                          \
    if (e_ != hipSuccess) return ::sparoa::hip_fail(e_, what);  \
  } while (0)

inline int64_t elem_size(sparoa_dtype d) { return d == SPAROA_F32 ? 4 : 2; }
inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Work-groups of kernel `fn` (`threads` threads, `lds` bytes of dynamic LDS)
// resident on the whole current device at once: the occupancy query times the
// compute-unit count, cached per (device, kernel, threads, LDS).  Sizes the
// grids of persistent kernels.
inline sparoa_status resident_blocks(const void *fn, int threads, unsigned lds, int *out) {
  static std::mutex mu;
  static std::map<std::tuple<int, const void *, int, unsigned>, int> cache;
  int dev = 0;
  SPAROA_HIP_CHECK(hipGetDevice(&dev));
  const auto key = std::make_tuple(dev, fn, threads, lds);
  std::lock_guard<std::mutex> lock(mu);
  auto it = cache.find(key);
  if (it == cache.end()) {
    int per_cu = 0, cus = 0;
    SPAROA_HIP_CHECK(hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, threads, lds));
    SPAROA_HIP_CHECK(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
    it = cache.emplace(key, (per_cu > 0 ? per_cu : 1) * (cus > 0 ? cus : 1)).first;
  }
  *out = it->second;
  return SPAROA_OK;
}

// Word 3 of a raw buffer descriptor on gfx9-family GPUs (32-bit data format;
// untyped loads ignore the rest).  Buffer loads at an offset past the
// descriptor's size return zero without a memory access.
constexpr int kBufDword3 = 0x00020000;

// Device-side routing: the skip decision is taken inside the kernel from the
// counts the measurement kernel left in device memory (no host round trip);
// the bandwidth bit depends on shapes only and is fixed by the host.
struct DeviceRoute {
  const sparoa_counts *counts;  // nullptr: the host already chose the path
  double sparsity_thr;
  int mode;
  int bw_bit;
  uint32_t *path_out;  // nullable: receives the path taken
  // Split execution (one operator over both paths): when non-null, every row
  // tile of the skip-capable GEMM takes its own route -- the skip path iff
  // the zero fraction of the input samples its output rows come from is at
  // least sparsity_thr.  sample_zeros[s] = zeros of input sample s, which
  // holds sample_numel elements and yields rows_per_sample output rows.
  const unsigned long long *sample_zeros = nullptr;
  int64_t rows_per_sample = 0, sample_numel = 0;
};

#ifdef __HIPCC__
// Same arithmetic as sparoa_route: one double division, >= comparison.
__device__ __forceinline__ bool route_skip_counts(const sparoa_counts &c, double thr, int mode) {
  double rho;
  if (mode == SPAROA_ROUTE_BLOCK) {
    if (c.num_blocks == 0 || c.zero_blocks > c.num_blocks) return false;
    rho = (double)c.zero_blocks / (double)c.num_blocks;
  } else {
    if (c.numel == 0 || c.zeros > c.numel) return false;
    rho = (double)c.zeros / (double)c.numel;
  }
  return rho >= thr;
}
__device__ __forceinline__ bool device_route_skip(const DeviceRoute &r) {
  return route_skip_counts(*r.counts, r.sparsity_thr, r.mode);
}

// The route's counts as two 16-byte vector loads, requested at a kernel's top
// and decided on later (their memory round trip then overlaps the kernel's
// own start).  Vector loads, not scalar ones: the scalar-load counter
// completes in order, so a scalar load of the counts would make every later
// kernel-argument use wait for it.  Null counts read zeros (a descriptor of
// size 0) and route dense.
struct RouteCountsReq {
  __attribute__((ext_vector_type(4))) unsigned int q[2];
};
__device__ __forceinline__ RouteCountsReq route_counts_request(const DeviceRoute &r) {
  const __amdgpu_buffer_rsrc_t cr = __builtin_amdgcn_make_buffer_rsrc(
      (void *)r.counts, (short)0, r.counts ? (int)sizeof(sparoa_counts) : 0, kBufDword3);
  RouteCountsReq q;
  q.q[0] = __builtin_amdgcn_raw_buffer_load_b128(cr, 0, 0, 0);
  q.q[1] = __builtin_amdgcn_raw_buffer_load_b128(cr, 16, 0, 0);
  return q;
}
__device__ __forceinline__ bool route_counts_skip(const RouteCountsReq &q, const DeviceRoute &r) {
  uint32_t w[8];   // the same in every lane: scalars, so the decision is uniform
#pragma unroll
  for (int i = 0; i < 8; ++i) w[i] = __builtin_amdgcn_readfirstlane(q.q[i >> 2][i & 3]);
  sparoa_counts c;
  __builtin_memcpy(&c, w, sizeof(c));
  return r.counts != nullptr && route_skip_counts(c, r.sparsity_thr, r.mode);
}
#endif

// Kernel arguments a kernel's start needs, requested together: an empty asm
// statement that reads them from scalar registers makes the compiler issue
// their loads at the kernel's top in one memory round trip.  Left alone, it
// loads each group just before its first use, and a group behind a branch
// costs a round trip of its own (about 0.5 us at the start of every
// work-group, measured on the implicit GEMM).
#define SPAROA_ARGS_UP_FRONT(...) asm volatile("" ::__VA_ARGS__)

// ---- launchers (validated arguments; defined in the .hip files) ---------

// preset: counts already hold {0, numel, nb, nb}; layouts whose bitmap needs
// no clearing (block 1 x one 16-byte vector, one block per row narrower than
// 16 bytes, whole-column strips) then skip the init launch.
// commit_words (preset only, nullable): zeroed count-commit words for the
// layouts that commit per work-group (lanebit, rowbit), left zero.
sparoa_status launch_measure(const void *x, sparoa_dtype dt, int64_t rows, int64_t cols,
                             int64_t block_rows, int64_t block_cols, int64_t samples,
                             sparoa_counts *counts, uint32_t *mask, uint64_t *per_sample,
                             hipStream_t stream, bool preset = false,
                             uint64_t *commit_words = nullptr);
// Counts only, at block (1, 8) over [rows, cols] (16-bit, cols % 8 == 0):
// all four counts, no bitmap.  counts arrive preset {0, numel, nb, nb}
// (commit_words as for the preset measurement).
sparoa_status launch_measure_counts8(const void *x, sparoa_dtype dt, int64_t rows, int64_t cols,
                                    sparoa_counts *counts, uint64_t *commit_words,
                                    hipStream_t stream);

constexpr int kGroupMax = 16;  // jobs per grouped launch

// Several measurements in the lanebit layout (block 1 x one 16-byte vector,
// a mask given), all of one element size, in two launches (counter init,
// measurement) for up to kGroupMax tensors.
struct MeasureJob {
  const void *x;
  sparoa_dtype dt;
  int64_t rows, cols, block_rows, block_cols;
  sparoa_counts *counts;
  uint32_t *mask;
};
bool measure_groupable(const MeasureJob &j);
sparoa_status launch_measure_group(const MeasureJob *jobs, int n, hipStream_t stream);

// Sums split-K fp32 partials [split][M][N] in split order, adds bias and
// residual, applies the activation, and writes y in dtype.
struct SplitReduceJob {
  sparoa_dtype dt;
  const float *partial;
  int split;          // 0: nothing to reduce
  int64_t M, N;
  const void *bias, *residual;
  sparoa_act act;
  void *y;
  sparoa_counts *om_counts;  // non-null: measure y (see OutMeasure)
  uint32_t *om_mask;
  unsigned long long *om_words;  // non-null: grouped count commit (OutMeasure::words)
};
sparoa_status launch_split_reduce(const SplitReduceJob &job, hipStream_t stream);
// Several reductions of one dtype in one launch (n <= kGroupMax).
sparoa_status launch_split_reduce_group(const SplitReduceJob *jobs, int n, hipStream_t stream);

// Measurement of a producer's output in its own epilogue (the next layer's
// input): counts and the bitmap at block (1 row, 8 channels) of y viewed as
// [M = N*Ho*Wo, C_out] -- exactly what launch_measure gives for that view.
// counts must hold {0, numel, nb, nb} before the producer runs (the caller
// resets them); the bitmap needs no clearing.
// words: SPAROA_COMMIT_WORDS_BYTES of zeroed count-commit words (ticketed
// commit, left zero), or null for one atomic per work-group on counts.
struct OutMeasure {
  sparoa_counts *counts;
  uint32_t *mask;
  unsigned long long *words = nullptr;
};

// Implicit-GEMM MFMA conv (groups == 1); FC runs through it as a 1x1 conv.
struct GemmTileChoice {
  int cfg;          // 0: general kernel; else a tile of the 64-channel-chunk kernel
  int bm, bn;       // output tile rows (pixels) x cols (channels)
  int kchunk;       // K elements per main-loop step == skip granularity (channels)
  int split_k;      // number of K splits (1 = none)
  bool small_c = false;  // the direct kernel for C_in <= 4 (image stems), cfg 0
  bool pointwise = false;  // the bandwidth-path 1x1 kernel (weights in LDS), cfg 0
};
// Whether the kernel of a groups == 1 conv's skip path reads x's bitmap
// (false for dense paths, the pointwise and small-channel kernels, which test
// x themselves, and shapes without a skip kernel).
bool conv_skip_reads_mask(const sparoa_conv_desc &d, sparoa_path path);
GemmTileChoice gemm_choose(const sparoa_conv_desc &d, sparoa_path path);
bool gemm_skip_supported(const sparoa_conv_desc &d);
// Workspace bytes a GEMM call needs (split-K partials).
size_t gemm_workspace_required(const sparoa_conv_desc &d, sparoa_path path);
sparoa_status launch_gemm_conv(const sparoa_conv_desc &d, sparoa_path path, const void *x,
                               const void *w, const void *bias, const void *residual,
                               sparoa_act act, const uint32_t *mask, void *y, void *ws,
                               size_t ws_bytes, uint64_t *executed, hipStream_t stream,
                               const DeviceRoute *route = nullptr,
                               SplitReduceJob *defer = nullptr,
                               const OutMeasure *om = nullptr);
// defer: when non-null, a split-K reduction is described there (split > 1)
// instead of launched; split = 0 when the GEMM needs none.
// om: measure y in the epilogue (or in the split-K reduction); only when
// gemm_fuses_out_measure(d, path, om->mask != nullptr) -- otherwise the call
// fails.  bitmap: the measurement also writes y's bitmap (the small-channel
// kernel only counts).
bool gemm_fuses_out_measure(const sparoa_conv_desc &d, sparoa_path path, bool bitmap);

// Pointwise (1x1) kernel of the bandwidth path: 16-bit, groups 1, no
// padding, C_in <= 256 and % 8 == 0, C_out % 8 == 0, the weights in at most
// four LDS slices.  Skip form: MFMAs over all-zero 16-pixel x 32-channel
// activation blocks are not issued.  om: fused output measurement (only when
// pw_fuses_out_measure).
bool pw_eligible(const sparoa_conv_desc &d);
bool pw_fuses_out_measure(const sparoa_conv_desc &d);
sparoa_status launch_pointwise(const sparoa_conv_desc &d, const void *x, const void *w,
                               const void *bias, const void *residual, sparoa_act act, void *y,
                               bool skip, uint64_t *executed, hipStream_t stream,
                               const DeviceRoute *route, const OutMeasure *om);

// Writes v to *p on the stream with a one-lane kernel (no memset node).
sparoa_status launch_set_u64(uint64_t *p, uint64_t v, hipStream_t stream);

// Depthwise direct conv (groups == c_in == c_out); om: measure y in the
// kernel (only when dw_fuses_out_measure).
bool dw_fuses_out_measure(const sparoa_conv_desc &d);
sparoa_status launch_depthwise(const sparoa_conv_desc &d, const void *x, const void *w,
                               const void *bias, const void *residual, sparoa_act act, void *y,
                               hipStream_t stream, const DeviceRoute *route = nullptr,
                               const OutMeasure *om = nullptr);

// FC weight-streaming (bandwidth) kernel over k-major packed weights.
size_t fc_packed_bytes(const sparoa_fc_desc &d);
// The weight-streaming kernel takes 16-bit FCs with m <= 64 and k <= 16384;
// every other bandwidth-path FC runs the implicit GEMM on w[n][k].
bool fc_bw_streams(const sparoa_fc_desc &d);
size_t fc_bw_workspace(const sparoa_fc_desc &d, sparoa_path path);
sparoa_status launch_fc_pack(const sparoa_fc_desc &d, const void *w_nk, void *w_packed,
                             hipStream_t stream);
sparoa_status launch_fc_bw(const sparoa_fc_desc &d, sparoa_path path, const void *x,
                           const void *w_packed, const void *bias, const void *residual,
                           sparoa_act act,
                           const uint32_t *mask, void *y, void *ws, size_t ws_bytes,
                           uint64_t *executed, hipStream_t stream,
                           const DeviceRoute *route = nullptr);
// The weight-streaming kernel can also measure its own input (zero count and
// the column bitmap at block (m, 1)) before routing: needs k % 8 == 0.
bool fc_bw_self_measures(const sparoa_fc_desc &d);
// Measures x into counts/mask (what sparoa_measure_sparsity gives at block
// (m, 1)), takes the skip decision from those counts and runs the FC, in one
// launch.  route->counts is ignored; its thresholds, bw bit and path_out apply.
sparoa_status launch_fc_bw_measured(const sparoa_fc_desc &d, const void *x, const void *w_packed,
                                    const void *bias, const void *residual, sparoa_act act,
                                    sparoa_counts *counts, uint32_t *mask, void *y,
                                    hipStream_t stream, const DeviceRoute &route);

// One self-measuring streaming FC of a grouped launch (route.counts unused).
struct FcBwJob {
  sparoa_fc_desc d;
  const void *x, *w_packed, *bias, *residual;
  sparoa_act act;
  sparoa_counts *counts;
  uint32_t *mask;
  void *y;
  DeviceRoute route;
};
// FCs with equal keys (>= 0: dtype and 16-row tiles) can share a grouped
// launch; -1: not self-measuring.
int fc_bw_group_key(const sparoa_fc_desc &d);
// Up to kGroupMax independent self-measuring FCs (no FC reads another's
// output) of one key in one launch; per FC, the same arithmetic and outputs
// as launch_fc_bw_measured.
sparoa_status launch_fc_bw_measured_group(const FcBwJob *jobs, int n, hipStream_t stream);

sparoa_status launch_maxpool(const void *x, sparoa_dtype dt, int64_t n, int64_t c, int64_t h,
                             int64_t w, int64_t k, int64_t s, int64_t p, void *y,
                             hipStream_t stream);

}  // namespace sparoa
