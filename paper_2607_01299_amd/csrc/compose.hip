// Segment composition, Eq. (6), for gfx950.
//
// One workgroup of d_k / 16 waves per (request, v-head).  The running state S
// (d_k x d_v, float32) stays on chip for the whole request.  Per listed segment
// i every wave updates its band of 16 state rows,
//     S[band] <- exp(log_decay_i) * (P_hat_i[band, :] @ S) + S_seg_i[band],
// which is the two-segment true splice of Eq. (4) applied in list order.
//
// The product is formed transposed, S^T P_hat^T, so that the accumulator
// layout gives each lane four consecutive columns of one state row: every
// access to HBM (P_hat rows, S_seg, the optional prefix, S_incoming, S_out)
// is then a 16-byte load or store per lane, 64 contiguous bytes per row per
// instruction.  The A operand (S^T) is read from a column-major copy of the
// state in LDS; the B operand (P_hat^T) is P_hat's own rows.  Each byte of the
// pool tuple is read once.  The tuple of step j + 1 is loaded into registers
// while step j computes.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mfma.hpp"
#include "scan.hpp"

namespace hypic {

namespace {

template <int DK, int DV, int P>
__global__ __launch_bounds__(DK * 4) void compose_kernel(ComposeArgs args) {
  constexpr int KB = DK / 32;     // 32-wide contraction blocks
  constexpr int NT = DV / 16;     // 16-column tiles of the state
  constexpr int LDT = DK + 4;     // column stride (floats) of the LDS copy
  __shared__ float st_t[DV * LDT];  // st_t[c * LDT + d] = S[d][c]

  const int tid = threadIdx.x;
  const int wave = tid / 64, lane = tid % 64;
  const int g = lane / 16, ln = lane % 16;
  const int req = blockIdx.x / args.h_v;
  const int h = blockIdx.x % args.h_v;
  const int row = wave * 16 + ln;  // this lane's state row
  const long state_sz = static_cast<long>(DK) * DV;
  const long hs = static_cast<long>(req) * args.h_v + h;

  // s[mt][i] = S[row][16 mt + 4 g + i]
  f32x4 s[NT];
  if (args.S_prefix != nullptr) {
    const float* pre = args.S_prefix + hs * state_sz + static_cast<long>(row) * DV + 4 * g;
#pragma unroll
    for (int mt = 0; mt < NT; ++mt) s[mt] = *reinterpret_cast<const f32x4*>(pre + 16 * mt);
  } else {
#pragma unroll
    for (int mt = 0; mt < NT; ++mt) s[mt] = zero4();
  }

  auto publish = [&]() {
#pragma unroll
    for (int mt = 0; mt < NT; ++mt)
#pragma unroll
      for (int i = 0; i < 4; ++i) st_t[(16 * mt + 4 * g + i) * LDT + row] = s[mt][i];
  };
  publish();
  __syncthreads();

  // pool tuple of one step: this lane's row of P_hat as B fragments (k slots
  // kap(g, .) of each 32-block) and its four S_seg columns per tile
  const int j0 = args.req_offsets[req], j1 = args.req_offsets[req + 1];
  float nP[KB][8];
  f32x4 nS[NT];
  float nE = 0.f;
  auto load_step = [&](int j) __attribute__((always_inline)) {
    const long sh = static_cast<long>(args.seg_ids[j]) * args.h_v + h;
    const float* Pi = args.P_hat + sh * DK * DK + static_cast<long>(row) * DK + 4 * g;
    const float* Si = args.S_seg + sh * state_sz + static_cast<long>(row) * DV + 4 * g;
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      const float4 lo = *reinterpret_cast<const float4*>(Pi + 32 * kb);
      const float4 hi = *reinterpret_cast<const float4*>(Pi + 32 * kb + 16);
      nP[kb][0] = lo.x; nP[kb][1] = lo.y; nP[kb][2] = lo.z; nP[kb][3] = lo.w;
      nP[kb][4] = hi.x; nP[kb][5] = hi.y; nP[kb][6] = hi.z; nP[kb][7] = hi.w;
    }
#pragma unroll
    for (int mt = 0; mt < NT; ++mt) nS[mt] = *reinterpret_cast<const f32x4*>(Si + 16 * mt);
    nE = __expf(args.log_decay[sh]);
  };
  if (j0 < j1) load_step(j0);
  for (int j = j0; j < j1; ++j) {
    float cP[KB][8];
    f32x4 cS[NT];
#pragma unroll
    for (int kb = 0; kb < KB; ++kb)
#pragma unroll
      for (int e = 0; e < 8; ++e) cP[kb][e] = nP[kb][e];
#pragma unroll
    for (int mt = 0; mt < NT; ++mt) cS[mt] = nS[mt];
    const float e = nE;
    if (j + 1 < j1) load_step(j + 1);
    if (args.S_incoming != nullptr) {
      float* dst = args.S_incoming + (static_cast<long>(j) * args.h_v + h) * state_sz +
                   static_cast<long>(row) * DV + 4 * g;
#pragma unroll
      for (int mt = 0; mt < NT; ++mt) *reinterpret_cast<f32x4*>(dst + 16 * mt) = s[mt];
    }
#pragma unroll
    for (int mt = 0; mt < NT; ++mt) {
      f32x4 prod = zero4();
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
        // A = S^T: column 16 mt + ln of the state, rows 32 kb + kap(g, .)
        float fa[8];
        const float* src = st_t + (16 * mt + ln) * LDT + 32 * kb + 4 * g;
        const float4 lo = *reinterpret_cast<const float4*>(src);
        const float4 hi = *reinterpret_cast<const float4*>(src + 16);
        fa[0] = lo.x; fa[1] = lo.y; fa[2] = lo.z; fa[3] = lo.w;
        fa[4] = hi.x; fa[5] = hi.y; fa[6] = hi.z; fa[7] = hi.w;
        mma_blk<P>(prod, fa, cP[kb]);
      }
      s[mt] = prod * e + cS[mt];
    }
    __syncthreads();  // every wave has read the old state
    publish();
    __syncthreads();
  }

  float* out = args.S_out + hs * state_sz + static_cast<long>(row) * DV + 4 * g;
#pragma unroll
  for (int mt = 0; mt < NT; ++mt) *reinterpret_cast<f32x4*>(out + 16 * mt) = s[mt];
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
