// Segment composition, Eq. (6), for gfx950.
//
// One workgroup of d_k / 16 waves per (request, v-head).  The running state S
// (d_k x d_v, float32) stays on chip for the whole request: each wave owns a
// band of 16 rows as matrix-core accumulators, and a transposed copy of the
// full state sits in LDS as the shared B operand.  Per listed segment i
// every wave streams its rows of P_hat_i and S_seg_i straight from HBM into
// registers (each byte of the pool tuple is read once) and computes
//     S[band] <- exp(log_decay_i) * (P_hat_i[band, :] @ S) + S_seg_i[band]
// which is the two-segment true splice of Eq. (4) applied in list order.
// The state entering each segment is optionally written out for the seam.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mfma.hpp"
#include "scan.hpp"

namespace hypic {

namespace {

template <int DK, int DV, int P>
__global__ __launch_bounds__(DK * 4) void compose_kernel(ComposeArgs args) {
  constexpr int RW = 16;           // rows per wave
  constexpr int MT = 1;
  constexpr int NT = DV / 16;
  constexpr int LDT = DK + 4;      // transposed state row stride (floats)
  __shared__ float st_t[DV * LDT];  // st_t[n * LDT + k] = S[k][n]

  const int tid = threadIdx.x;
  const int wave = tid / 64, lane = tid % 64;
  const int g = lane / 16, ln = lane % 16;
  const int req = blockIdx.x / args.h_v;
  const int h = blockIdx.x % args.h_v;
  const int row0 = wave * RW;
  const long state_sz = static_cast<long>(DK) * DV;

  f32x4 s[MT][NT];
  const float* pre = args.S_prefix ? args.S_prefix + (static_cast<long>(req) * args.h_v + h) * state_sz
                                   : nullptr;
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        s[mt][nt][i] = pre ? pre[(row0 + mt * 16 + 4 * g + i) * DV + nt * 16 + ln] : 0.f;

  auto publish = [&]() {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
        *reinterpret_cast<f32x4*>(&st_t[(nt * 16 + ln) * LDT + row0 + mt * 16 + 4 * g]) =
            s[mt][nt];
  };
  publish();
  __syncthreads();

  // The pool tuple of step j + 1 is loaded into registers while step j
  // computes (software pipelining), so the HBM latency hides behind the
  // matrix-core work and the barriers.
  const int j0 = args.req_offsets[req], j1 = args.req_offsets[req + 1];
  float nP[MT][DK / 32][8];
  f32x4 nS[MT][NT];
  float nE = 0.f;
  auto load_step = [&](int j) __attribute__((always_inline)) {
    const long sh = static_cast<long>(args.seg_ids[j]) * args.h_v + h;
    const float* Pi = args.P_hat + sh * DK * DK;
    const float* Si = args.S_seg + sh * state_sz;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int kb = 0; kb < DK / 32; ++kb) frag_kcontig(Pi, DK, row0 + mt * 16 + ln, kb * 32, g, nP[mt][kb]);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          nS[mt][nt][i] = Si[(row0 + mt * 16 + 4 * g + i) * DV + nt * 16 + ln];
    nE = __expf(args.log_decay[sh]);
  };
  if (j0 < j1) load_step(j0);
  for (int j = j0; j < j1; ++j) {
    float cP[MT][DK / 32][8];
    f32x4 cS[MT][NT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
      for (int kb = 0; kb < DK / 32; ++kb)
#pragma unroll
        for (int e = 0; e < 8; ++e) cP[mt][kb][e] = nP[mt][kb][e];
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) cS[mt][nt] = nS[mt][nt];
    }
    const float e = nE;
    if (j + 1 < j1) load_step(j + 1);
    if (args.S_incoming != nullptr) {
      float* dst = args.S_incoming + (static_cast<long>(j) * args.h_v + h) * state_sz;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            dst[(row0 + mt * 16 + 4 * g + i) * DV + nt * 16 + ln] = s[mt][nt][i];
    }
    f32x4 prod[MT][NT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) prod[mt][nt] = zero4();
#pragma unroll
    for (int kb = 0; kb < DK / 32; ++kb) {
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        float fb[8];
        frag_kcontig(st_t, LDT, nt * 16 + ln, kb * 32, g, fb);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) mma_blk<P>(prod[mt][nt], cP[mt][kb], fb);
      }
    }
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) s[mt][nt] = prod[mt][nt] * e + cS[mt][nt];
    __syncthreads();  // every wave has read the old state
    publish();
    __syncthreads();
  }

  float* out = args.S_out + (static_cast<long>(req) * args.h_v + h) * state_sz;
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        out[(row0 + mt * 16 + 4 * g + i) * DV + nt * 16 + ln] = s[mt][nt][i];
}

template <int DK, int DV>
hipError_t launch_compose_d(const ComposeArgs& a, int f32, int n_req, hipStream_t s) {
  const dim3 grid(static_cast<unsigned>(n_req) * a.h_v);
  const dim3 block(DK * 4);  // one wave per 16 state rows
  if (f32)
    hipLaunchKernelGGL((compose_kernel<DK, DV, P_F32>), grid, block, 0, s, a);
  else
    hipLaunchKernelGGL((compose_kernel<DK, DV, P_SPLIT>), grid, block, 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_compose(const ComposeArgs& a, int f32, int d_k, int d_v, int n_req,
                          hipStream_t s) {
  if (n_req <= 0) return hipSuccess;
  if (d_k == 64 && d_v == 64) return launch_compose_d<64, 64>(a, f32, n_req, s);
  if (d_k == 64 && d_v == 128) return launch_compose_d<64, 128>(a, f32, n_req, s);
  if (d_k == 128 && d_v == 64) return launch_compose_d<128, 64>(a, f32, n_req, s);
  return launch_compose_d<128, 128>(a, f32, n_req, s);
}

}  // namespace hypic
