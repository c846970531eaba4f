// hypic_build_segment_noalloc: the segment build for callers that cannot
// allocate device memory.  Its only scratch, the longest-first order of a
// build of more than kInlineOrder segments, lives in a fixed device array of
// this file instead of a caller's workspace.
//
// Each GPU the library runs on holds its own copy of the array until the
// process ends.  Its address on the current device is looked up once per
// device (hipGetSymbolAddress, with that device current) and kept; host code
// uses that address, never the array's name, which on the host is only a
// stand-in symbol.  Every call on a GPU shares that GPU's array: calls that
// overlap on one GPU (on different streams, or from different threads before
// the first has run) race on it.  The order kernel writes every one of the
// n_seg entries it needs, so nothing has to start at zero.

#include <hip/hip_runtime.h>
#include <mutex>
#include <stdint.h>

#include "../../include/hypic.h"
#include "api_impl.hpp"
#include "scan.hpp"

namespace {

static_assert(HYPIC_NOALLOC_MAX_SEGMENTS > hypic::kInlineOrder, "scratch below the inline order");

// the longest-first order of one build: HYPIC_NOALLOC_MAX_SEGMENTS int32 (256 KiB)
static __device__ __align__(256) int32_t scratch[HYPIC_NOALLOC_MAX_SEGMENTS];

constexpr int kMaxDevices = 256;
std::mutex g_scratch_mu;
int32_t* g_scratch[kMaxDevices];  // device address of `scratch`, per device

// The current device's copy of `scratch`: hipGetSymbolAddress on the first use
// on a device (that device current), the kept address afterwards.
int32_t current_scratch(int32_t** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return HYPIC_EHIP;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch[dev] == nullptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr)
      return HYPIC_EHIP;
    g_scratch[dev] = static_cast<int32_t*>(p);
  }
  *out = g_scratch[dev];
  return HYPIC_OK;
}

}  // namespace

extern "C" int32_t hypic_build_segment_noalloc(const hypic_dims* dims, const void* q,
                                               const void* k, const void* v,
                                               const float* beta, const float* log_alpha,
                                               int32_t n_tokens, const int32_t* cu_seqlens,
                                               const int32_t* cu_seqlens_host, int32_t n_seg,
                                               void* o, float* S_seg, float* P_hat,
                                               float* log_decay, void* stream) {
  if (n_seg > HYPIC_NOALLOC_MAX_SEGMENTS) return HYPIC_EWORKSPACE;
  int32_t* order = nullptr;
  size_t order_bytes = 0;
  if (n_seg > hypic::kInlineOrder) {
    const int32_t st = current_scratch(&order);
    if (st != HYPIC_OK) return st;
    order_bytes = sizeof(int32_t) * HYPIC_NOALLOC_MAX_SEGMENTS;
  }
  return hypic::build_segment_impl(dims, q, k, v, beta, log_alpha, n_tokens, cu_seqlens,
                                   cu_seqlens_host, n_seg, o, S_seg, P_hat, log_decay, order,
                                   order_bytes, stream);
}
