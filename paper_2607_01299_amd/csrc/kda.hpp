// Launch interface of the chunked scan for the KDA row of Tab. 1 (kda.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "scan.hpp"

namespace hypic {

struct KdaArgs {
  const void* q;
  const void* k;
  const void* v;
  const float* beta;          // [T, h_v]
  const float* gate;          // [T, h_v, d_k], natural-log units
  int32_t h_qk, h_v, group;
  int32_t n_tokens;
  int32_t mode;               // 0 build, 1 seam
  const int32_t* cu_seqlens;  // build: segment offsets
  const int32_t* order;       // build: longest-first order (n_inline == 0)
  const int32_t* tok_start;   // seam: first token of each entry
  const int32_t* tok_len;     // seam: segment length of each entry
  int32_t w;                  // seam width
  const float* S_in;          // seam: incoming states
  void* o;                    // build: [T,h_v,d_v]; seam: [n,w,h_v,d_v]; may be null
  float* S_out;               // build: S_seg; seam: S_post (may be null)
  float* P_hat;               // build: [n,h_v,d_k,d_k] or null (no operator)
  float* log_decay;           // build: [n,h_v], written with P_hat
  int32_t n_inline;
  uint16_t order_inline[kInlineOrder];
};

// State columns (and, in a build with P_hat, operator columns) of n_chains
// (segment or seam entry, v-head) chains.
hipError_t launch_kda_scan(const KdaArgs& a, int bf16, int d_k, int d_v, int n_chains,
                           hipStream_t s);

}  // namespace hypic
