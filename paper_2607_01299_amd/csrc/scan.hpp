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
  const int32_t* out_entry;  // seam: output entry of each entry (NULL: the same)
  // mode 2, composition with seams in one pass: a chain is one (request, head);
  // chunk c is the request's c-th listed pool entry, whose seam tokens are
  // tok_start[i], min(w, tok_len[i]) with i = seg_ids[req_offsets[r] + c]; after
  // the seam the state composes with that entry's tuple.  The request order
  // (longest first) is held in order / order_inline.
  const int32_t* seg_ids;      // [nnz] pool entry of each listed segment
  const int32_t* req_offsets;  // [n_req + 1] CSR offsets
  const float* pool_P;         // [n_pool, h_v, d_k, d_k]
  const float* pool_ld;        // [n_pool, h_v]
  const float* pool_S;         // [n_pool, h_v, d_k, d_v]
  const float* S_prefix;       // [n_req, h_v, d_k, d_v] or NULL (zero)
  float* S_final;              // [n_req, h_v, d_k, d_v]
  int32_t advance;             // 1: the seam advances the state (Sec. 4.3); 0: it does not
};

// Entry of the seam output o[n, w, h_v, d_v] that seam entry e writes.
__device__ __forceinline__ int32_t seam_out_entry(const ScanArgs& a, int e) {
  return a.out_entry != nullptr ? a.out_entry[e] : e;
}

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

hipError_t launch_lpt_order(const int32_t* cu, int n, int32_t* order, hipStream_t s);
// Launches the scan over n_chains (segments or seam entries) x h_v heads;
// returns hipErrorInvalidValue if the grid would exceed 2^31 - 1 workgroups.
hipError_t launch_scan(const ScanArgs& a, int bf16, int d_k, int d_v, int chunk,
                       int n_chains, hipStream_t s);
// Workgroups per (chain, head) of the bf16 chunk-64 scan.
int scan_bf16_items_per_head(int d_k, int d_v, int with_operator);
hipError_t launch_scan_bf16(const ScanArgs& a, int d_k, int d_v, int n_items, hipStream_t s);
// Mode 2 (bf16 tokens, seam w <= 64, no operator): one workgroup per (request,
// head), n_req x h_v workgroups.
hipError_t launch_seam_compose_fused(const ScanArgs& a, int d_k, int d_v, int n_req,
                                     hipStream_t s);
hipError_t launch_compose(const ComposeArgs& a, int f32, int d_k, int d_v, int n_req,
                          hipStream_t s);

}  // namespace hypic
