// C ABI of libhypic.so: argument validation on the host, workspace sizing and
// kernel dispatch.  Nothing is enqueued unless every check passes.

#include <algorithm>
#include <cmath>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/hypic.h"
#include "api_impl.hpp"
#include "family.hpp"
#include "kda.hpp"
#include "scan.hpp"

namespace {

constexpr size_t kAlign = 256;

size_t round_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Checks shared by every entry point.  Returns HYPIC_OK or an error code.
int32_t check_dims(const hypic_dims* d) {
  if (d == nullptr) return HYPIC_EINVAL;
  if (d->h_qk < 1 || d->h_v < 1) return HYPIC_EINVAL;
  if (d->h_v % d->h_qk != 0) return HYPIC_EINVAL;
  if (d->d_k != 64 && d->d_k != 128) return HYPIC_EUNSUPPORTED;
  if (d->d_v != 64 && d->d_v != 128) return HYPIC_EUNSUPPORTED;
  if (d->chunk != 16 && d->chunk != 32 && d->chunk != 64) return HYPIC_EUNSUPPORTED;
  if (d->dtype != HYPIC_F32 && d->dtype != HYPIC_BF16) return HYPIC_EUNSUPPORTED;
  return HYPIC_OK;
}

int32_t hip_status(hipError_t e) { return e == hipSuccess ? HYPIC_OK : HYPIC_EHIP; }

// Segment offsets of a build: 0 = cu[0] <= cu[1] <= ... <= cu[n_seg] <= n_tokens,
// so every segment lies inside the packed token arrays.
bool check_segment_offsets(const int32_t* cu_host, int32_t n_seg, int32_t n_tokens) {
  if (cu_host[0] != 0) return false;
  for (int32_t s = 0; s < n_seg; ++s)
    if (cu_host[s + 1] < cu_host[s]) return false;
  return cu_host[n_seg] <= n_tokens;
}

}  // namespace

extern "C" {

const char* hypic_status_str(int32_t status) {
  switch (status) {
    case HYPIC_OK: return "ok";
    case HYPIC_EINVAL: return "invalid argument (pointer, size, offset or index)";
    case HYPIC_EUNSUPPORTED: return "unsupported dims (d_k, d_v in {64,128}; chunk in {16,32,64}; dtype F32 or BF16)";
    case HYPIC_EWORKSPACE: return "workspace missing or too small";
    case HYPIC_EHIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

size_t hypic_workspace_bytes(int32_t op, const hypic_dims* dims, int64_t n) {
  if (check_dims(dims) != HYPIC_OK || n <= 0) return 0;
  if ((op == HYPIC_OP_BUILD || op == HYPIC_OP_COMPOSE_RESCAN) && n > hypic::kInlineOrder)
    return round_up(static_cast<size_t>(n) * sizeof(int32_t));
  return 0;
}

int32_t hypic_build_segment(const hypic_dims* dims, const void* q, const void* k,
                            const void* v, const float* beta, const float* log_alpha,
                            int32_t n_tokens, const int32_t* cu_seqlens,
                            const int32_t* cu_seqlens_host,
                            int32_t n_seg, void* o, float* S_seg, float* P_hat,
                            float* log_decay, void* workspace, size_t workspace_bytes,
                            void* stream) {
  return hypic::build_segment_impl(dims, q, k, v, beta, log_alpha, n_tokens, cu_seqlens,
                                   cu_seqlens_host, n_seg, o, S_seg, P_hat, log_decay,
                                   workspace, workspace_bytes, stream);
}

}  // extern "C"

namespace hypic {

// The segment build behind hypic_build_segment and hypic_build_segment_noalloc:
// host validation, then the longest-first order (in the kernel arguments, or
// on the device into `workspace`) and the scan launch.
int32_t build_segment_impl(const hypic_dims* dims, const void* q, const void* k,
                           const void* v, const float* beta, const float* log_alpha,
                           int32_t n_tokens, const int32_t* cu_seqlens,
                           const int32_t* cu_seqlens_host, int32_t n_seg, void* o,
                           float* S_seg, float* P_hat, float* log_decay, void* workspace,
                           size_t workspace_bytes, void* stream) {
  int32_t st = check_dims(dims);
  if (st != HYPIC_OK) return st;
  if (n_seg < 0 || n_tokens < 0) return HYPIC_EINVAL;
  if (n_seg == 0) return HYPIC_OK;
  if (!q || !k || !v || !beta || !log_alpha || !cu_seqlens || !cu_seqlens_host || !S_seg)
    return HYPIC_EINVAL;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || (o && !aligned16(o)))
    return HYPIC_EINVAL;
  if (!check_segment_offsets(cu_seqlens_host, n_seg, n_tokens)) return HYPIC_EINVAL;
  const int64_t n_items = static_cast<int64_t>(n_seg) * dims->h_v * 4;
  if (n_items > 0x7fffffff) return HYPIC_EINVAL;
  const size_t need = hypic_workspace_bytes(HYPIC_OP_BUILD, dims, n_seg);
  if (need > 0 && (workspace == nullptr || workspace_bytes < need)) return HYPIC_EWORKSPACE;

  hipStream_t s = static_cast<hipStream_t>(stream);
  hypic::ScanArgs a{};
  if (n_seg <= hypic::kInlineOrder) {
    // Eq. (9) list order, longest first, ties by index, from the host offsets.
    int32_t idx[hypic::kInlineOrder];
    for (int32_t i = 0; i < n_seg; ++i) idx[i] = i;
    std::stable_sort(idx, idx + n_seg, [&](int32_t x, int32_t y) {
      return cu_seqlens_host[x + 1] - cu_seqlens_host[x] >
             cu_seqlens_host[y + 1] - cu_seqlens_host[y];
    });
    for (int32_t i = 0; i < n_seg; ++i) a.order_inline[i] = static_cast<uint16_t>(idx[i]);
    a.n_inline = n_seg;
    a.order = nullptr;
  } else {
    int32_t* order = static_cast<int32_t*>(workspace);
    st = hip_status(hypic::launch_lpt_order(cu_seqlens, n_seg, order, s));
    if (st != HYPIC_OK) return st;
    a.order = order;
  }
  a.q = q;
  a.k = k;
  a.v = v;
  a.beta = beta;
  a.log_alpha = log_alpha;
  a.h_qk = dims->h_qk;
  a.h_v = dims->h_v;
  a.group = dims->h_v / dims->h_qk;
  a.n_tokens = n_tokens;
  a.mode = 0;
  a.n_roles = P_hat ? 2 : 1;
  a.cu_seqlens = cu_seqlens;
  a.o = o;
  a.S_out = S_seg;
  a.P_hat = P_hat;
  a.log_decay = log_decay;
  return hip_status(hypic::launch_scan(a, dims->dtype == HYPIC_BF16, dims->d_k, dims->d_v,
                                       dims->chunk, n_seg, s));
}

}  // namespace hypic

extern "C" {

int32_t hypic_compose_segments(const hypic_dims* dims, const float* P_hat,
                               const float* log_decay, const float* S_seg, int32_t n_pool,
                               const int32_t* seg_ids, const int32_t* seg_ids_host,
                               const int32_t* req_offsets, const int32_t* req_offsets_host,
                               int32_t n_req, const float* S_prefix, float* S_out,
                               float* S_incoming, void* workspace, size_t workspace_bytes,
                               void* stream) {
  (void)workspace;
  (void)workspace_bytes;
  int32_t st = check_dims(dims);
  if (st != HYPIC_OK) return st;
  if (n_req < 0 || n_pool < 0) return HYPIC_EINVAL;
  if (n_req == 0) return HYPIC_OK;
  if (!req_offsets || !req_offsets_host || !S_out) return HYPIC_EINVAL;
  if (req_offsets_host[0] != 0) return HYPIC_EINVAL;
  for (int32_t r = 0; r < n_req; ++r)
    if (req_offsets_host[r + 1] < req_offsets_host[r]) return HYPIC_EINVAL;
  const int32_t nnz = req_offsets_host[n_req];
  if (!aligned16(S_out) || (S_prefix && !aligned16(S_prefix)) ||
      (S_incoming && !aligned16(S_incoming)))
    return HYPIC_EINVAL;
  if (nnz > 0) {
    if (!P_hat || !log_decay || !S_seg || !seg_ids || !seg_ids_host) return HYPIC_EINVAL;
    if (!aligned16(P_hat) || !aligned16(S_seg)) return HYPIC_EINVAL;
    for (int32_t j = 0; j < nnz; ++j)
      if (seg_ids_host[j] < 0 || seg_ids_host[j] >= n_pool) return HYPIC_EINVAL;
  }
  if (static_cast<int64_t>(n_req) * dims->h_v > 0x7fffffff) return HYPIC_EINVAL;

  hypic::ComposeArgs a{};
  a.P_hat = P_hat;
  a.log_decay = log_decay;
  a.S_seg = S_seg;
  a.seg_ids = seg_ids;
  a.req_offsets = req_offsets;
  a.S_prefix = S_prefix;
  a.S_out = S_out;
  a.S_incoming = S_incoming;
  a.h_v = dims->h_v;
  return hip_status(hypic::launch_compose(a, dims->dtype == HYPIC_F32, dims->d_k, dims->d_v,
                                          n_req, static_cast<hipStream_t>(stream)));
}

int32_t hypic_seam_rescan(const hypic_dims* dims, const void* q, const void* k,
                          const void* v, const float* beta, const float* log_alpha,
                          int32_t n_tokens, const int32_t* tok_start, const int32_t* tok_len,
                          const int32_t* tok_start_host, const int32_t* tok_len_host,
                          int32_t n_entries, int32_t w, const float* S_in, void* o_seam,
                          float* S_post, void* workspace, size_t workspace_bytes,
                          void* stream) {
  (void)workspace;
  (void)workspace_bytes;
  int32_t st = check_dims(dims);
  if (st != HYPIC_OK) return st;
  if (n_entries < 0 || n_tokens < 0 || w < 1) return HYPIC_EINVAL;
  if (n_entries == 0) return HYPIC_OK;
  if (!q || !k || !v || !beta || !log_alpha || !tok_start || !tok_len || !tok_start_host ||
      !tok_len_host || !S_in || !o_seam)
    return HYPIC_EINVAL;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o_seam))
    return HYPIC_EINVAL;
  for (int32_t e = 0; e < n_entries; ++e) {
    const int64_t len = tok_len_host[e];
    const int64_t start = tok_start_host[e];
    if (len < 1 || start < 0) return HYPIC_EINVAL;
    const int64_t w_eff = len < w ? len : w;
    if (start + w_eff > n_tokens) return HYPIC_EINVAL;
  }
  if (static_cast<int64_t>(n_entries) * dims->h_v * 4 > 0x7fffffff) return HYPIC_EINVAL;

  hypic::ScanArgs a{};
  a.q = q;
  a.k = k;
  a.v = v;
  a.beta = beta;
  a.log_alpha = log_alpha;
  a.h_qk = dims->h_qk;
  a.h_v = dims->h_v;
  a.group = dims->h_v / dims->h_qk;
  a.n_tokens = n_tokens;
  a.mode = 1;
  a.n_roles = 1;
  a.tok_start = tok_start;
  a.tok_len = tok_len;
  a.w = w;
  a.S_in = S_in;
  a.o = o_seam;
  a.S_out = S_post;
  return hip_status(hypic::launch_scan(a, dims->dtype == HYPIC_BF16, dims->d_k, dims->d_v,
                                       dims->chunk, n_entries, static_cast<hipStream_t>(stream)));
}

// ---------------------------------------------------------------------------
// scalar and diagonal transition families
// ---------------------------------------------------------------------------

int32_t hypic_family_build(const hypic_dims* dims, int32_t family, const void* q,
                           const void* k, const void* v, const float* gate, int32_t n_tokens,
                           const int32_t* cu_seqlens, const int32_t* cu_seqlens_host,
                           int32_t n_seg, void* o, float* S_seg, float* log_decay,
                           void* workspace, size_t workspace_bytes, void* stream) {
  int32_t st = check_dims(dims);
  if (st != HYPIC_OK) return st;
  if (family != HYPIC_FAMILY_SCALAR && family != HYPIC_FAMILY_DIAGONAL) return HYPIC_EUNSUPPORTED;
  if (n_seg < 0 || n_tokens < 0) return HYPIC_EINVAL;
  if (n_seg == 0) return HYPIC_OK;
  if (!q || !k || !v || !gate || !cu_seqlens || !cu_seqlens_host || !S_seg) return HYPIC_EINVAL;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v)) return HYPIC_EINVAL;
  if (!check_segment_offsets(cu_seqlens_host, n_seg, n_tokens)) return HYPIC_EINVAL;
  if (static_cast<int64_t>(n_seg) * dims->h_v * 2 > 0x7fffffff) return HYPIC_EINVAL;
  const size_t need = hypic_workspace_bytes(HYPIC_OP_BUILD, dims, n_seg);
  if (need > 0 && (workspace == nullptr || workspace_bytes < need)) return HYPIC_EWORKSPACE;

  hipStream_t s = static_cast<hipStream_t>(stream);
  hypic::FamArgs a{};
  if (n_seg <= hypic::kInlineOrder) {
    int32_t idx[hypic::kInlineOrder];
    for (int32_t i = 0; i < n_seg; ++i) idx[i] = i;
    std::stable_sort(idx, idx + n_seg, [&](int32_t x, int32_t y) {
      return cu_seqlens_host[x + 1] - cu_seqlens_host[x] >
             cu_seqlens_host[y + 1] - cu_seqlens_host[y];
    });
    for (int32_t i = 0; i < n_seg; ++i) a.order_inline[i] = static_cast<uint16_t>(idx[i]);
    a.n_inline = n_seg;
  } else {
    int32_t* order = static_cast<int32_t*>(workspace);
    st = hip_status(hypic::launch_lpt_order(cu_seqlens, n_seg, order, s));
    if (st != HYPIC_OK) return st;
    a.order = order;
  }
  a.q = q;
  a.k = k;
  a.v = v;
  a.gate = gate;
  a.h_qk = dims->h_qk;
  a.h_v = dims->h_v;
  a.group = dims->h_v / dims->h_qk;
  a.n_tokens = n_tokens;
  a.mode = 0;
  a.cu_seqlens = cu_seqlens;
  a.o = o;
  a.S_out = S_seg;
  a.log_decay = log_decay;
  return hip_status(hypic::launch_family_scan(a, family, dims->dtype == HYPIC_BF16, dims->d_k,
                                              dims->d_v, n_seg, s));
}

int32_t hypic_family_compose(const hypic_dims* dims, int32_t family, const float* log_decay,
                             const float* S_seg, int32_t n_pool, const int32_t* seg_ids,
                             const int32_t* seg_ids_host, const int32_t* req_offsets,
                             const int32_t* req_offsets_host, int32_t n_req,
                             const float* S_prefix, float* S_out, float* S_incoming,
                             void* workspace, size_t workspace_bytes, void* stream) {
  (void)workspace;
  (void)workspace_bytes;
  int32_t st = check_dims(dims);
  if (st != HYPIC_OK) return st;
  if (family != HYPIC_FAMILY_SCALAR && family != HYPIC_FAMILY_DIAGONAL) return HYPIC_EUNSUPPORTED;
  if (n_req < 0 || n_pool < 0) return HYPIC_EINVAL;
  if (n_req == 0) return HYPIC_OK;
  if (!req_offsets || !req_offsets_host || !S_out) return HYPIC_EINVAL;
  if (!aligned16(S_out) || (S_prefix && !aligned16(S_prefix)) ||
      (S_incoming && !aligned16(S_incoming)))
    return HYPIC_EINVAL;
  if (req_offsets_host[0] != 0) return HYPIC_EINVAL;
  for (int32_t r = 0; r < n_req; ++r)
    if (req_offsets_host[r + 1] < req_offsets_host[r]) return HYPIC_EINVAL;
  const int32_t nnz = req_offsets_host[n_req];
  if (nnz > 0) {
    if (!log_decay || !S_seg || !seg_ids || !seg_ids_host || !aligned16(S_seg))
      return HYPIC_EINVAL;
    for (int32_t j = 0; j < nnz; ++j)
      if (seg_ids_host[j] < 0 || seg_ids_host[j] >= n_pool) return HYPIC_EINVAL;
  }
  if (static_cast<int64_t>(n_req) * dims->h_v * 4 > 0x7fffffff) return HYPIC_EINVAL;

  hypic::FamComposeArgs a{};
  a.log_decay = log_decay;
  a.S_seg = S_seg;
  a.seg_ids = seg_ids;
  a.req_offsets = req_offsets;
  a.S_prefix = S_prefix;
  a.S_out = S_out;
  a.S_incoming = S_incoming;
  a.h_v = dims->h_v;
  return hip_status(hypic::launch_family_compose(a, family, dims->d_k, dims->d_v, n_req,
                                                 static_cast<hipStream_t>(stream)));
}

int32_t hypic_family_seam(const hypic_dims* dims, int32_t family, const void* q, const void* k,
                          const void* v, const float* gate, int32_t n_tokens,
                          const int32_t* tok_start, const int32_t* tok_len,
                          const int32_t* tok_start_host, const int32_t* tok_len_host,
                          int32_t n_entries, int32_t w, const float* S_in, void* o_seam,
                          float* S_post, void* workspace, size_t workspace_bytes,
                          void* stream) {
  (void)workspace;
  (void)workspace_bytes;
  int32_t st = check_dims(dims);
  if (st != HYPIC_OK) return st;
  if (family != HYPIC_FAMILY_SCALAR && family != HYPIC_FAMILY_DIAGONAL) return HYPIC_EUNSUPPORTED;
  if (n_entries < 0 || n_tokens < 0 || w < 1) return HYPIC_EINVAL;
  if (n_entries == 0) return HYPIC_OK;
  if (!q || !k || !v || !gate || !tok_start || !tok_len || !tok_start_host || !tok_len_host ||
      !S_in || !o_seam)
    return HYPIC_EINVAL;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v)) return HYPIC_EINVAL;
  for (int32_t e = 0; e < n_entries; ++e) {
    const int64_t len = tok_len_host[e];
    const int64_t start = tok_start_host[e];
    if (len < 1 || start < 0) return HYPIC_EINVAL;
    const int64_t w_eff = len < w ? len : w;
    if (start + w_eff > n_tokens) return HYPIC_EINVAL;
  }
  if (static_cast<int64_t>(n_entries) * dims->h_v * 2 > 0x7fffffff) return HYPIC_EINVAL;

  hypic::FamArgs a{};
  a.q = q;
  a.k = k;
  a.v = v;
  a.gate = gate;
  a.h_qk = dims->h_qk;
  a.h_v = dims->h_v;
  a.group = dims->h_v / dims->h_qk;
  a.n_tokens = n_tokens;
  a.mode = 1;
  a.tok_start = tok_start;
  a.tok_len = tok_len;
  a.w = w;
  a.S_in = S_in;
  a.o = o_seam;
  a.S_out = S_post;
  return hip_status(hypic::launch_family_scan(a, family, dims->dtype == HYPIC_BF16, dims->d_k,
                                              dims->d_v, n_entries,
                                              static_cast<hipStream_t>(stream)));
}

// ---------------------------------------------------------------------------
// the KDA row of Tab. 1
// ---------------------------------------------------------------------------

int32_t hypic_kda_build(const hypic_dims* dims, const void* q, const void* k, const void* v,
                        const float* beta, const float* gate, int32_t n_tokens,
                        const int32_t* cu_seqlens, const int32_t* cu_seqlens_host, int32_t n_seg, void* o, float* S_seg,
                        float* P_hat, float* log_decay, void* workspace, size_t workspace_bytes,
                        void* stream) {
  int32_t st = check_dims(dims);
  if (st != HYPIC_OK) return st;
  if (n_seg < 0 || n_tokens < 0) return HYPIC_EINVAL;
  if (n_seg == 0) return HYPIC_OK;
  if (!q || !k || !v || !beta || !gate || !cu_seqlens || !cu_seqlens_host || !S_seg)
    return HYPIC_EINVAL;
  if (P_hat != nullptr && log_decay == nullptr) return HYPIC_EINVAL;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v)) return HYPIC_EINVAL;
  if (!check_segment_offsets(cu_seqlens_host, n_seg, n_tokens)) return HYPIC_EINVAL;
  if (static_cast<int64_t>(n_seg) * dims->h_v * 2 > 0x7fffffff) return HYPIC_EINVAL;
  const size_t need = hypic_workspace_bytes(HYPIC_OP_BUILD, dims, n_seg);
  if (need > 0 && (workspace == nullptr || workspace_bytes < need)) return HYPIC_EWORKSPACE;

  hipStream_t s = static_cast<hipStream_t>(stream);
  hypic::KdaArgs a{};
  if (n_seg <= hypic::kInlineOrder) {
    int32_t idx[hypic::kInlineOrder];
    for (int32_t i = 0; i < n_seg; ++i) idx[i] = i;
    std::stable_sort(idx, idx + n_seg, [&](int32_t x, int32_t y) {
      return cu_seqlens_host[x + 1] - cu_seqlens_host[x] >
             cu_seqlens_host[y + 1] - cu_seqlens_host[y];
    });
    for (int32_t i = 0; i < n_seg; ++i) a.order_inline[i] = static_cast<uint16_t>(idx[i]);
    a.n_inline = n_seg;
  } else {
    int32_t* order = static_cast<int32_t*>(workspace);
    st = hip_status(hypic::launch_lpt_order(cu_seqlens, n_seg, order, s));
    if (st != HYPIC_OK) return st;
    a.order = order;
  }
  a.q = q;
  a.k = k;
  a.v = v;
  a.beta = beta;
  a.gate = gate;
  a.h_qk = dims->h_qk;
  a.h_v = dims->h_v;
  a.group = dims->h_v / dims->h_qk;
  a.n_tokens = n_tokens;
  a.mode = 0;
  a.cu_seqlens = cu_seqlens;
  a.o = o;
  a.S_out = S_seg;
  a.P_hat = P_hat;
  a.log_decay = log_decay;
  return hip_status(
      hypic::launch_kda_scan(a, dims->dtype == HYPIC_BF16, dims->d_k, dims->d_v, n_seg, s));
}

int32_t hypic_kda_seam(const hypic_dims* dims, const void* q, const void* k, const void* v,
                       const float* beta, const float* gate, int32_t n_tokens,
                       const int32_t* tok_start, const int32_t* tok_len,
                       const int32_t* tok_start_host, const int32_t* tok_len_host,
                       int32_t n_entries, int32_t w, const float* S_in, void* o_seam,
                       float* S_post, void* workspace, size_t workspace_bytes, void* stream) {
  (void)workspace;
  (void)workspace_bytes;
  int32_t st = check_dims(dims);
  if (st != HYPIC_OK) return st;
  if (n_entries < 0 || n_tokens < 0 || w < 1) return HYPIC_EINVAL;
  if (n_entries == 0) return HYPIC_OK;
  if (!q || !k || !v || !beta || !gate || !tok_start || !tok_len || !tok_start_host ||
      !tok_len_host || !S_in || !o_seam)
    return HYPIC_EINVAL;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v)) return HYPIC_EINVAL;
  for (int32_t e = 0; e < n_entries; ++e) {
    const int64_t len = tok_len_host[e];
    const int64_t start = tok_start_host[e];
    if (len < 1 || start < 0) return HYPIC_EINVAL;
    const int64_t w_eff = len < w ? len : w;
    if (start + w_eff > n_tokens) return HYPIC_EINVAL;
  }
  if (static_cast<int64_t>(n_entries) * dims->h_v * 2 > 0x7fffffff) return HYPIC_EINVAL;

  hypic::KdaArgs a{};
  a.q = q;
  a.k = k;
  a.v = v;
  a.beta = beta;
  a.gate = gate;
  a.h_qk = dims->h_qk;
  a.h_v = dims->h_v;
  a.group = dims->h_v / dims->h_qk;
  a.n_tokens = n_tokens;
  a.mode = 1;
  a.tok_start = tok_start;
  a.tok_len = tok_len;
  a.w = w;
  a.S_in = S_in;
  a.o = o_seam;
  a.S_out = S_post;
  return hip_status(hypic::launch_kda_scan(a, dims->dtype == HYPIC_BF16, dims->d_k, dims->d_v,
                                           n_entries, static_cast<hipStream_t>(stream)));
}

// ---------------------------------------------------------------------------
// reuse with seam windows that advance the state (Sec. 4.3)
// ---------------------------------------------------------------------------

namespace {

struct SeamComposeLayout {
  size_t states, order, lists, total;  // byte offsets of the parts, total size
};

SeamComposeLayout seam_compose_layout(const hypic_dims* d, int64_t n_req, int64_t max_n) {
  SeamComposeLayout l{};
  const size_t state = static_cast<size_t>(d->h_v) * d->d_k * d->d_v * sizeof(float);
  l.states = 0;
  l.order = round_up(2 * static_cast<size_t>(n_req) * state);
  l.lists = l.order + round_up(static_cast<size_t>(n_req) * sizeof(int32_t));
  l.total = l.lists + round_up((4 * static_cast<size_t>(max_n) * n_req + n_req + 1) *
                               sizeof(int32_t));
  return l;
}

}  // namespace

namespace {

// Host validation shared by the two seam-composition calls; max_n gets the
// longest request's entry count.
int32_t check_seam_compose(const hypic_dims* dims, const float* P_hat, const float* log_decay,
                           const float* S_seg, int32_t n_pool, const void* q, const void* k,
                           const void* v, const float* beta, const float* log_alpha,
                           int32_t n_tokens, const int32_t* seam_start,
                           const int32_t* seam_start_host, const int32_t* seam_len,
                           const int32_t* seam_len_host, int32_t w, const int32_t* seg_ids,
                           const int32_t* seg_ids_host, const int32_t* req_offsets,
                           const int32_t* req_offsets_host, int32_t n_req,
                           const float* S_prefix, float* S_out, void* o_seam, int32_t* max_n_out) {
  int32_t st = check_dims(dims);
  if (st != HYPIC_OK) return st;
  if (n_req < 0 || n_pool < 0 || n_tokens < 0 || w < 1) return HYPIC_EINVAL;
  if (n_req == 0) return HYPIC_OK;
  if (!req_offsets || !req_offsets_host || !S_out || !aligned16(S_out) ||
      (S_prefix && !aligned16(S_prefix)))
    return HYPIC_EINVAL;
  if (req_offsets_host[0] != 0) return HYPIC_EINVAL;
  int32_t max_n = 0;
  for (int32_t r = 0; r < n_req; ++r) {
    const int32_t n = req_offsets_host[r + 1] - req_offsets_host[r];
    if (n < 0) return HYPIC_EINVAL;
    max_n = n > max_n ? n : max_n;
  }
  const int32_t nnz = req_offsets_host[n_req];
  if (nnz > 0) {
    if (!P_hat || !log_decay || !S_seg || !seg_ids || !seg_ids_host || !q || !k || !v || !beta ||
        !log_alpha || !seam_start || !seam_start_host || !seam_len || !seam_len_host || !o_seam)
      return HYPIC_EINVAL;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o_seam) ||
        !aligned16(P_hat) || !aligned16(S_seg))
      return HYPIC_EINVAL;
    for (int32_t j = 0; j < nnz; ++j)
      if (seg_ids_host[j] < 0 || seg_ids_host[j] >= n_pool) return HYPIC_EINVAL;
    for (int32_t i = 0; i < n_pool; ++i) {
      const int64_t len = seam_len_host[i], start = seam_start_host[i];
      if (len < 1 || start < 0) return HYPIC_EINVAL;
      if (start + (len < w ? len : w) > n_tokens) return HYPIC_EINVAL;
    }
  }
  if (static_cast<int64_t>(n_req) * dims->h_v * 4 > 0x7fffffff ||
      static_cast<int64_t>(max_n) * n_req > 0x7fffffff)
    return HYPIC_EINVAL;
  *max_n_out = max_n;
  return HYPIC_OK;
}

// The one-pass composition with seams runs on the bf16 chunk-64 scan: bf16
// tokens, chunk 64, a seam of at most one chunk.
bool fusable(const hypic_dims* dims, int32_t w) {
  return dims->dtype == HYPIC_BF16 && dims->chunk == 64 && w <= 64;
}

// One launch: requests longest first (Eq. (9) list order, ties by index; in
// the kernel arguments up to kInlineOrder requests, else on the device into
// order_ws), one workgroup per (request, head).
int32_t launch_fused(const hypic_dims* dims, const float* P_hat, const float* log_decay,
                     const float* S_seg, const void* q, const void* k, const void* v,
                     const float* beta, const float* log_alpha, int32_t n_tokens,
                     const int32_t* seam_start, const int32_t* seam_len, int32_t w,
                     const int32_t* seg_ids, const int32_t* req_offsets,
                     const int32_t* req_offsets_host, int32_t n_req, const float* S_prefix,
                     float* S_out, void* o_seam, int32_t advance, int32_t* order_ws,
                     hipStream_t s) {
  hypic::ScanArgs a{};
  if (n_req <= hypic::kInlineOrder) {
    int32_t idx[hypic::kInlineOrder];
    for (int32_t i = 0; i < n_req; ++i) idx[i] = i;
    std::stable_sort(idx, idx + n_req, [&](int32_t x, int32_t y) {
      return req_offsets_host[x + 1] - req_offsets_host[x] >
             req_offsets_host[y + 1] - req_offsets_host[y];
    });
    for (int32_t i = 0; i < n_req; ++i) a.order_inline[i] = static_cast<uint16_t>(idx[i]);
    a.n_inline = n_req;
  } else {
    const int32_t st = hip_status(hypic::launch_lpt_order(req_offsets, n_req, order_ws, s));
    if (st != HYPIC_OK) return st;
    a.order = order_ws;
  }
  a.q = q;
  a.k = k;
  a.v = v;
  a.beta = beta;
  a.log_alpha = log_alpha;
  a.h_qk = dims->h_qk;
  a.h_v = dims->h_v;
  a.group = dims->h_v / dims->h_qk;
  a.n_tokens = n_tokens;
  a.mode = 2;
  a.n_roles = 1;
  a.tok_start = seam_start;
  a.tok_len = seam_len;
  a.w = w;
  a.o = o_seam;
  a.seg_ids = seg_ids;
  a.req_offsets = req_offsets;
  a.pool_P = P_hat;
  a.pool_ld = log_decay;
  a.pool_S = S_seg;
  a.S_prefix = S_prefix;
  a.S_final = S_out;
  a.advance = advance;
  return hip_status(hypic::launch_seam_compose_fused(a, dims->d_k, dims->d_v, n_req, s));
}

}  // namespace

size_t hypic_seam_compose_workspace_bytes(const hypic_dims* dims, int32_t n_req,
                                          int32_t max_per_request) {
  if (check_dims(dims) != HYPIC_OK || n_req <= 0 || max_per_request < 0) return 0;
  return seam_compose_layout(dims, n_req, max_per_request).total;
}

int32_t hypic_compose_with_seams(const hypic_dims* dims, const float* P_hat,
                                 const float* log_decay, const float* S_seg, int32_t n_pool,
                                 const void* q, const void* k, const void* v, const float* beta,
                                 const float* log_alpha, int32_t n_tokens,
                                 const int32_t* seam_start, const int32_t* seam_start_host,
                                 const int32_t* seam_len, const int32_t* seam_len_host, int32_t w,
                                 const int32_t* seg_ids, const int32_t* seg_ids_host,
                                 const int32_t* req_offsets, const int32_t* req_offsets_host,
                                 int32_t n_req, const float* S_prefix, float* S_out,
                                 void* o_seam, void* workspace, size_t workspace_bytes,
                                 void* stream) {
  int32_t max_n = 0;
  int32_t st = check_seam_compose(dims, P_hat, log_decay, S_seg, n_pool, q, k, v, beta,
                                  log_alpha, n_tokens, seam_start, seam_start_host, seam_len,
                                  seam_len_host, w, seg_ids, seg_ids_host, req_offsets,
                                  req_offsets_host, n_req, S_prefix, S_out, o_seam, &max_n);
  if (st != HYPIC_OK || n_req == 0) return st;
  const SeamComposeLayout l = seam_compose_layout(dims, n_req, max_n);
  if (workspace == nullptr || workspace_bytes < l.total) return HYPIC_EWORKSPACE;

  hipStream_t s = static_cast<hipStream_t>(stream);
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  if (fusable(dims, w)) {
    // one pass: each (request, head) keeps its running state on chip across
    // its entries (seam, then the tail tuple)
    return launch_fused(dims, P_hat, log_decay, S_seg, q, k, v, beta, log_alpha, n_tokens,
                        seam_start, seam_len, w, seg_ids, req_offsets, req_offsets_host, n_req,
                        S_prefix, S_out, o_seam, 1, reinterpret_cast<int32_t*>(ws + l.order), s);
  }
  const long state_floats = static_cast<long>(dims->h_v) * dims->d_k * dims->d_v;
  float* cur = reinterpret_cast<float*>(ws + l.states);
  float* tmp = cur + static_cast<long>(n_req) * state_floats;
  int32_t* order = reinterpret_cast<int32_t*>(ws + l.order);
  int32_t* lists = reinterpret_cast<int32_t*>(ws + l.lists);
  const long plane = static_cast<long>(max_n) * n_req;
  int32_t *ts = lists, *tl = lists + plane, *sid = lists + 2 * plane, *orow = lists + 3 * plane;
  int32_t* iota = lists + 4 * plane;

  // requests longest first (Eq. (9) list order, ties by index): the requests
  // still running at step j are ranks 0 .. A_j - 1
  st = hip_status(hypic::launch_lpt_order(req_offsets, n_req, order, s));
  if (st == HYPIC_OK && max_n > 0)
    st = hip_status(hypic::launch_seam_steps(order, req_offsets, seg_ids, seam_start, seam_len,
                                             n_req, max_n, ts, tl, sid, orow, iota, s));
  if (st == HYPIC_OK)
    st = hip_status(hypic::launch_permute_states(S_prefix, cur, order, n_req, state_floats, 0, s));
  for (int32_t j = 0; j < max_n && st == HYPIC_OK; ++j) {
    int32_t active = 0;  // A_j: requests with more than j entries
    for (int32_t r = 0; r < n_req; ++r)
      active += (req_offsets_host[r + 1] - req_offsets_host[r]) > j;
    // seam: the running state of each active request through its entry's
    // first w tokens, outputs to the entry's CSR row
    hypic::ScanArgs a{};
    a.q = q;
    a.k = k;
    a.v = v;
    a.beta = beta;
    a.log_alpha = log_alpha;
    a.h_qk = dims->h_qk;
    a.h_v = dims->h_v;
    a.group = dims->h_v / dims->h_qk;
    a.n_tokens = n_tokens;
    a.mode = 1;
    a.n_roles = 1;
    a.tok_start = ts + static_cast<long>(j) * n_req;
    a.tok_len = tl + static_cast<long>(j) * n_req;
    a.w = w;
    a.S_in = cur;
    a.o = o_seam;
    a.S_out = tmp;
    a.out_entry = orow + static_cast<long>(j) * n_req;
    st = hip_status(hypic::launch_scan(a, dims->dtype == HYPIC_BF16, dims->d_k, dims->d_v,
                                       dims->chunk, active, s));
    if (st != HYPIC_OK) break;
    // the entry's tail tuple, Eq. (4)
    hypic::ComposeArgs c{};
    c.P_hat = P_hat;
    c.log_decay = log_decay;
    c.S_seg = S_seg;
    c.seg_ids = sid + static_cast<long>(j) * n_req;
    c.req_offsets = iota;
    c.S_prefix = tmp;
    c.S_out = cur;
    c.S_incoming = nullptr;
    c.h_v = dims->h_v;
    st = hip_status(hypic::launch_compose(c, dims->dtype == HYPIC_F32, dims->d_k, dims->d_v,
                                          active, s));
  }
  if (st == HYPIC_OK)
    st = hip_status(hypic::launch_permute_states(cur, S_out, order, n_req, state_floats, 1, s));
  return st;
}

int32_t hypic_compose_and_rescan(const hypic_dims* dims, const float* P_hat,
                                 const float* log_decay, const float* S_seg, int32_t n_pool,
                                 const void* q, const void* k, const void* v, const float* beta,
                                 const float* log_alpha, int32_t n_tokens,
                                 const int32_t* seam_start, const int32_t* seam_start_host,
                                 const int32_t* seam_len, const int32_t* seam_len_host, int32_t w,
                                 const int32_t* seg_ids, const int32_t* seg_ids_host,
                                 const int32_t* req_offsets, const int32_t* req_offsets_host,
                                 int32_t n_req, const float* S_prefix, float* S_out,
                                 void* o_seam, void* workspace, size_t workspace_bytes,
                                 void* stream) {
  int32_t max_n = 0;
  int32_t st = check_seam_compose(dims, P_hat, log_decay, S_seg, n_pool, q, k, v, beta,
                                  log_alpha, n_tokens, seam_start, seam_start_host, seam_len,
                                  seam_len_host, w, seg_ids, seg_ids_host, req_offsets,
                                  req_offsets_host, n_req, S_prefix, S_out, o_seam, &max_n);
  if (st != HYPIC_OK || n_req == 0) return st;
  if (!fusable(dims, w)) return HYPIC_EUNSUPPORTED;
  const size_t need = hypic_workspace_bytes(HYPIC_OP_COMPOSE_RESCAN, dims, n_req);
  if (need > 0 && (workspace == nullptr || workspace_bytes < need)) return HYPIC_EWORKSPACE;
  return launch_fused(dims, P_hat, log_decay, S_seg, q, k, v, beta, log_alpha, n_tokens,
                      seam_start, seam_len, w, seg_ids, req_offsets, req_offsets_host, n_req,
                      S_prefix, S_out, o_seam, 0, static_cast<int32_t*>(workspace),
                      static_cast<hipStream_t>(stream));
}

// ---------------------------------------------------------------------------
// reuse-time steps next to the cache: RoPE state shift, key re-rotation, conv
// ---------------------------------------------------------------------------

namespace {

// cu[0] == 0, non-decreasing; returns the longest segment or -1
int64_t check_offsets(const int32_t* cu_host, int32_t n_seg) {
  if (cu_host[0] != 0) return -1;
  int64_t longest = 0;
  for (int32_t s = 0; s < n_seg; ++s) {
    const int64_t len = static_cast<int64_t>(cu_host[s + 1]) - cu_host[s];
    if (len < 0) return -1;
    longest = len > longest ? len : longest;
  }
  return longest;
}

bool good_base(double base) { return std::isfinite(base) && base > 0.0; }

}  // namespace

int32_t hypic_rope_shift_state(const hypic_dims* dims, const float* S_in, float* S_out,
                               int32_t n, const int32_t* delta, double base, void* stream) {
  int32_t st = check_dims(dims);
  if (st != HYPIC_OK) return st;
  if (n < 0 || !good_base(base)) return HYPIC_EINVAL;
  if (n == 0) return HYPIC_OK;
  if (!S_in || !S_out || !delta || !aligned16(S_in) || !aligned16(S_out)) return HYPIC_EINVAL;
  if (static_cast<int64_t>(n) * dims->h_v > 0x7fffffff) return HYPIC_EINVAL;
  return hip_status(hypic::launch_rope_state(S_in, S_out, delta, n, dims->h_v, dims->d_k,
                                             dims->d_v, base, static_cast<hipStream_t>(stream)));
}

int32_t hypic_rope_rerotate_keys(const hypic_dims* dims, const void* k_in, void* k_out,
                                 const int32_t* cu_seqlens, const int32_t* cu_seqlens_host,
                                 int32_t n_seg, const int32_t* delta, double base,
                                 void* stream) {
  int32_t st = check_dims(dims);
  if (st != HYPIC_OK) return st;
  if (n_seg < 0 || !good_base(base)) return HYPIC_EINVAL;
  if (n_seg == 0) return HYPIC_OK;
  if (!k_in || !k_out || !cu_seqlens || !cu_seqlens_host || !delta) return HYPIC_EINVAL;
  if (!aligned16(k_in) || !aligned16(k_out)) return HYPIC_EINVAL;
  const int64_t longest = check_offsets(cu_seqlens_host, n_seg);
  if (longest < 0 || (longest + 63) / 64 > 65535) return HYPIC_EINVAL;
  return hip_status(hypic::launch_rope_keys(k_in, k_out, dims->dtype == HYPIC_BF16, cu_seqlens,
                                            delta, n_seg, static_cast<int>(longest), dims->h_qk,
                                            dims->d_k, base, static_cast<hipStream_t>(stream)));
}

int32_t hypic_causal_conv(int32_t dtype, int32_t channels, int32_t width, const void* x,
                          const float* weight, const int32_t* cu_seqlens,
                          const int32_t* cu_seqlens_host, int32_t n_seg, const float* state_in,
                          void* y, float* state_out, int32_t silu, void* stream) {
  if (dtype != HYPIC_F32 && dtype != HYPIC_BF16) return HYPIC_EUNSUPPORTED;
  if (width < 1 || width > 8) return HYPIC_EUNSUPPORTED;
  if (channels < 1 || n_seg < 0) return HYPIC_EINVAL;
  if (n_seg == 0) return HYPIC_OK;
  if (!x || !weight || !y || !cu_seqlens || !cu_seqlens_host) return HYPIC_EINVAL;
  if (x == y || !aligned16(x) || !aligned16(y)) return HYPIC_EINVAL;
  const int64_t longest = check_offsets(cu_seqlens_host, n_seg);
  if (longest < 0 || (longest + 63) / 64 > 65535 || (channels + 255) / 256 > 65535)
    return HYPIC_EINVAL;
  return hip_status(hypic::launch_causal_conv(x, weight, dtype == HYPIC_BF16, cu_seqlens, n_seg,
                                              static_cast<int>(longest), state_in, y, state_out,
                                              channels, width, silu ? 1 : 0,
                                              static_cast<hipStream_t>(stream)));
}

}  // extern "C"
