// Launch interface between the C ABI layer and the kernels of the scalar and
// diagonal transition families and of the reuse-time steps next to the cache.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "scan.hpp"

namespace hypic {

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

// The software-pipelined builds of the diagonal and scalar families
// (gated_pipe.hip): bf16 inputs, d_k = 128, d_v = 64 or 128, segment build only.
bool diag_pipe_supported(int bf16, int d_k, int d_v, int mode);
hipError_t launch_diag_pipe(const FamArgs& a, int d_v, int n_chains, hipStream_t s);
hipError_t launch_scalar_pipe(const FamArgs& a, int d_v, int n_chains, hipStream_t s);

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

hipError_t launch_seam_steps(const int32_t* order, const int32_t* req_offsets,
                             const int32_t* seg_ids, const int32_t* seam_start,
                             const int32_t* seam_len, int n_req, int max_n, int32_t* ts,
                             int32_t* tl, int32_t* sid, int32_t* orow, int32_t* iota,
                             hipStream_t s);
hipError_t launch_permute_states(const float* src, float* dst, const int32_t* order, int n,
                                 long floats, int scatter, hipStream_t s);

}  // namespace hypic
