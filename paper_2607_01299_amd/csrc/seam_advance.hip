// Helpers of reuse with seam windows that advance the state (Sec. 4.3): the
// requests are ranked longest first, so the requests still running at step j
// are ranks 0 .. A_j - 1 and every step's seam and composition work on
// contiguous state slots; these kernels lay out the per-step entry lists and
// move states between request order and rank order.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "family.hpp"

namespace hypic {

namespace {

// entry (step j, rank e) of the step-major lists, stride n_req per step
__global__ void seam_steps_kernel(const int32_t* order, const int32_t* req_offsets,
                                  const int32_t* seg_ids, const int32_t* seam_start,
                                  const int32_t* seam_len, int n_req, int max_n, int32_t* ts,
                                  int32_t* tl, int32_t* sid, int32_t* orow, int32_t* iota) {
  const long idx = static_cast<long>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (idx <= n_req) iota[idx] = static_cast<int32_t>(idx);
  if (idx >= static_cast<long>(max_n) * n_req) return;
  const int j = static_cast<int>(idx / n_req), e = static_cast<int>(idx % n_req);
  const int r = order[e];
  const int p = req_offsets[r] + j;
  if (p >= req_offsets[r + 1]) return;
  const int id = seg_ids[p];
  ts[idx] = seam_start[id];
  tl[idx] = seam_len[id];
  sid[idx] = id;
  orow[idx] = p;
}

// gather (dst[e] = src[order[e]], zeros when src is NULL) or scatter
// (dst[order[e]] = src[e]) of n states of `floats` floats each
__global__ void permute_states_kernel(const float* src, float* dst, const int32_t* order, int n,
                                      long floats, int scatter) {
  const long per = floats / 4;
  const long idx = static_cast<long>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (idx >= per * n) return;
  const int e = static_cast<int>(idx / per);
  const long f = idx % per;
  const long from = scatter ? e : order[e];
  const long to = scatter ? order[e] : e;
  const float4 v = src ? reinterpret_cast<const float4*>(src)[from * per + f]
                       : make_float4(0.f, 0.f, 0.f, 0.f);
  reinterpret_cast<float4*>(dst)[to * per + f] = v;
}

}  // namespace

hipError_t launch_seam_steps(const int32_t* order, const int32_t* req_offsets,
                             const int32_t* seg_ids, const int32_t* seam_start,
                             const int32_t* seam_len, int n_req, int max_n, int32_t* ts,
                             int32_t* tl, int32_t* sid, int32_t* orow, int32_t* iota,
                             hipStream_t s) {
  const long total = static_cast<long>(max_n) * n_req;
  const long items = (total > n_req + 1) ? total : n_req + 1;
  hipLaunchKernelGGL(seam_steps_kernel, dim3((items + 255) / 256), dim3(256), 0, s, order,
                     req_offsets, seg_ids, seam_start, seam_len, n_req, max_n, ts, tl, sid, orow,
                     iota);
  return hipGetLastError();
}

hipError_t launch_permute_states(const float* src, float* dst, const int32_t* order, int n,
                                 long floats, int scatter, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const long items = floats / 4 * n;
  hipLaunchKernelGGL(permute_states_kernel, dim3((items + 255) / 256), dim3(256), 0, s, src,
                     dst, order, n, floats, scatter);
  return hipGetLastError();
}

}  // namespace hypic
