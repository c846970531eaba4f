// Launch interface between the C ABI layer and the scan / compose kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hypic {

// Builds of at most this many segments carry their longest-first order in the
// kernel arguments; larger builds compute it on the device into the workspace.
constexpr int kInlineOrder = 128;

// Arguments of the chunked scan kernel (segment build when mode == 0, seam
// rescan when mode == 1).  All pointers are device pointers.
struct ScanArgs {
  const void* q;
  const void* k;
  const void* v;
  const float* beta;
  const float* log_alpha;
  int32_t h_qk, h_v, group;  // group = h_v / h_qk
  int32_t n_tokens;
  int32_t mode;              // 0 build, 1 seam
  int32_t n_roles;           // 1: state only, 2: state and operator
  const int32_t* cu_seqlens; // build: segment offsets
  const int32_t* order;      // build: longest-first segment order (n_inline == 0)
  const int32_t* tok_start;  // seam: first token of each entry
  const int32_t* tok_len;    // seam: segment length of each entry
  int32_t w;                 // seam width
  int32_t n_entries;         // seam: number of entries
  int32_t group_e;           // seam: entries per workgroup (w <= chunk: run back to back)
  const float* S_in;         // seam: incoming states
  void* o;                   // outputs (build: [T,h_v,d_v]; seam: [n,w,h_v,d_v])
  float* S_out;              // build: S_seg; seam: S_post (may be null)
  float* P_hat;              // build, role 1
  float* log_decay;          // build, may be null
  int32_t n_inline;          // build: > 0 when the order is held in order_inline
  uint16_t order_inline[kInlineOrder];
};

// Segment scheduled at position `rank` of the longest-first order.
__device__ __forceinline__ int32_t segment_of_rank(const ScanArgs& a, int rank) {
  return a.n_inline > 0 ? static_cast<int32_t>(a.order_inline[rank]) : a.order[rank];
}

struct ComposeArgs {
  const float* P_hat;
  const float* log_decay;
  const float* S_seg;
  const int32_t* seg_ids;
  const int32_t* req_offsets;
  const float* S_prefix;
  float* S_out;
  float* S_incoming;
  int32_t h_v;
};

// Transition families of the scalar / diagonal family scan and compose.
constexpr int FAM_SCALAR = 1;
constexpr int FAM_DIAGONAL = 2;

// Arguments of the family scan kernel (segment build when mode == 0, seam
// rescan when mode == 1).  gate: [T, h_v] (scalar) or [T, h_v, d_k] (diagonal).
struct FamArgs {
  const void* q;
  const void* k;
  const void* v;
  const float* gate;
  int32_t h_qk, h_v, group;
  int32_t n_tokens;
  int32_t mode;
  const int32_t* cu_seqlens;  // build: segment offsets
  const int32_t* order;       // build: longest-first order (n_inline == 0)
  const int32_t* tok_start;   // seam: first token of each entry
  const int32_t* tok_len;     // seam: segment length of each entry
  int32_t w;                  // seam width
  const float* S_in;          // seam: incoming states
  void* o;                    // build: [T,h_v,d_v]; seam: [n,w,h_v,d_v]
  float* S_out;               // build: S_seg; seam: S_post (may be null)
  float* log_decay;           // build: [n,h_v] or [n,h_v,d_k], may be null
  int32_t n_inline;
  uint16_t order_inline[kInlineOrder];
};

struct FamComposeArgs {
  const float* log_decay;  // [n_pool,h_v] or [n_pool,h_v,d_k]
  const float* S_seg;
  const int32_t* seg_ids;
  const int32_t* req_offsets;
  const float* S_prefix;
  float* S_out;
  float* S_incoming;
  int32_t h_v;
};

hipError_t launch_family_scan(const FamArgs& a, int family, int bf16, int d_k, int d_v,
                              int n_chains, hipStream_t s);
hipError_t launch_family_compose(const FamComposeArgs& a, int family, int d_k, int d_v,
                                 int n_req, hipStream_t s);

hipError_t launch_rope_state(const float* S_in, float* S_out, const int32_t* delta, int n,
                             int h_v, int d_k, int d_v, double base, hipStream_t s);
hipError_t launch_rope_keys(const void* k_in, void* k_out, int bf16, const int32_t* cu,
                            const int32_t* delta, int n_seg, int max_len, int heads, int d,
                            double base, hipStream_t s);
hipError_t launch_causal_conv(const void* x, const float* w, int bf16, const int32_t* cu,
                              int n_seg, int max_len, const float* state_in, void* y,
                              float* state_out, int C, int K, int silu, hipStream_t s);

hipError_t launch_lpt_order(const int32_t* cu, int n, int32_t* order, hipStream_t s);
// Launches the scan over n_chains (segments or seam entries) x h_v heads;
// returns hipErrorInvalidValue if the grid would exceed 2^31 - 1 workgroups.
hipError_t launch_scan(const ScanArgs& a, int bf16, int d_k, int d_v, int chunk,
                       int n_chains, hipStream_t s);
// Workgroups per (chain, head) of the bf16 chunk-64 scan.
int scan_bf16_items_per_head(int d_k, int d_v, int with_operator);
hipError_t launch_scan_bf16(const ScanArgs& a, int d_k, int d_v, int n_items, hipStream_t s);
hipError_t launch_compose(const ComposeArgs& a, int f32, int d_k, int d_v, int n_req,
                          hipStream_t s);

}  // namespace hypic
