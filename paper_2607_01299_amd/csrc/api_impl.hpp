// Internal entry points shared by the C ABI's variants (not exported).
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "../../include/hypic.h"

namespace hypic {

// hypic_build_segment with its workspace: validation, order, scan launch.
int32_t build_segment_impl(const hypic_dims* dims, const void* q, const void* k,
                           const void* v, const float* beta, const float* log_alpha,
                           int32_t n_tokens, const int32_t* cu_seqlens,
                           const int32_t* cu_seqlens_host, int32_t n_seg, void* o,
                           float* S_seg, float* P_hat, float* log_decay, void* workspace,
                           size_t workspace_bytes, void* stream);

}  // namespace hypic
