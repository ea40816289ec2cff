// sparoa_conv2d_noalloc: the fixed-path convolution for callers that cannot
// allocate device memory (code under HIP graph capture, tight serving loops,
// harnesses that forbid hipMalloc).  It runs the kernels of sparoa_conv2d;
// the split-K partial sums that sparoa_conv2d takes from the caller's
// workspace live instead in a file-scope device array of fixed size, one copy
// per GPU, held until the process ends.
//
// The partial sums need no clearing: every (split, row, column) of a call's
// partial planes is written by exactly one work-group before the reduction
// reads it.  Calls that overlap in time on one GPU (different streams, or
// different host threads) share the array and race; calls ordered on one
// stream do not.
#include <mutex>

#include "common.h"

namespace sparoa {
namespace {

constexpr size_t kScratchBytes = size_t(8) << 20;   // SPAROA_NOALLOC_SCRATCH_BYTES
static_assert(kScratchBytes == SPAROA_NOALLOC_SCRATCH_BYTES, "documented limit");
constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};

// Device address of `scratch` on the current device.  The array's name is a
// host-side stand-in; only the address hipGetSymbolAddress returns for a
// device may reach a kernel.  Looked up once per device, on that device's
// first call.
sparoa_status scratch_on_current_device(void **out) {
  int dev = -1;
  SPAROA_HIP_CHECK(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) return fail(SPAROA_ERR_UNSUPPORTED, "noalloc: device index");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *p = nullptr;
    SPAROA_HIP_CHECK(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p) return fail(SPAROA_ERR_HIP, "noalloc: no device address for the scratch array");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return SPAROA_OK;
}

}  // namespace
}  // namespace sparoa

using namespace sparoa;

extern "C" sparoa_status sparoa_conv2d_noalloc(const sparoa_conv_desc *d, sparoa_path path,
                                               const void *x, const void *w, const void *bias,
                                               const void *residual, sparoa_act act,
                                               const uint32_t *mask, void *y,
                                               uint64_t *executed_blocks_dev,
                                               hipStream_t stream) {
  size_t need = 0;
  sparoa_status st = sparoa_conv2d_workspace_size(d, path, &need);   // validates desc and path
  if (st != SPAROA_OK) return st;
  if (need > kScratchBytes)
    return fail(SPAROA_ERR_WORKSPACE,
                "conv2d_noalloc: the split-K partial sums of this shape need " +
                    std::to_string(need) + " bytes, above the " + std::to_string(kScratchBytes) +
                    "-byte scratch array (use sparoa_conv2d with a workspace)");
  void *ws = nullptr;
  if (need > 0 && (st = scratch_on_current_device(&ws)) != SPAROA_OK) return st;
  return sparoa_conv2d(d, path, x, w, bias, residual, act, mask, y, ws, need > 0 ? kScratchBytes : 0,
                       executed_blocks_dev, stream);
}
