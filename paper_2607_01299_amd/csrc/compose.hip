// Segment composition, Eq. (6), for gfx950.
//
// For every request r and v-head h, S starts at the prefix (or zero) and for
// each listed segment i in order
//     S_incoming[j] = S;   S <- exp(log_decay_i) * (P_hat_i @ S) + S_seg_i,
// which is the two-segment true splice of Eq. (4) applied in list order.
//
// One workgroup of d_k / 16 waves runs one (request, v-head, column block):
// the state S (all d_k rows, NC = d_v / NCB columns) stays on chip for the
// whole request, wave w owning rows 16w .. 16w+15.  Per listed segment:
//   * each wave streams its 16 rows of P_hat_i from HBM (16 rows x 64
//     contiguous bytes per load instruction), split once into bf16 hi + lo,
//     the A operand of P_hat S;
//   * the B operand is S itself: a wave's 16 x 16 accumulator tiles are
//     exactly half of a 32-deep B fragment (rows 4g .. 4g+3 of column n in
//     lane (g, n)), so publishing the state is one 8-byte LDS store of its hi
//     and one of its lo part per tile, and every wave reads the fragments it
//     needs with 16-byte loads;
//   * the product runs in three bf16 passes (hi hi, hi lo, lo hi) or on the
//     float32 matrix cores, then S <- e^g (P_hat S) + S_seg in float32.
// The tuple of a later step is loaded into registers while a step computes
// (two steps ahead on split grids, one on full-width ones).
// Small grids split the columns of each head over NCB = 8 or 4 workgroups (numbered
// so that they land on one XCD and share its L2 for P_hat); large grids keep
// one workgroup per head, so each byte of the pool tuple is read once, ordered
// head-major so that concurrent requests share one head's pool slice in the
// memory-side cache.  The incoming states are written with non-temporal
// stores, which keep them from displacing that slice.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mfma.hpp"
#include "scan.hpp"

namespace hypic {

namespace {

typedef unsigned short u16;
typedef u16 u16x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ u16 bf16_bits(float x) {
  return __builtin_bit_cast(u16, static_cast<__bf16>(x));
}

template <int DK, int DV, int P, int NCB>
__global__ __launch_bounds__(DK * 4) void compose_kernel(ComposeArgs args) {
  constexpr int KB = DK / 32;        // 32-deep contraction blocks
  constexpr int NC = DV / NCB;       // state columns of this workgroup
  constexpr int NT = NC / 16;        // 16-column tiles
  constexpr bool SPLIT = P != P_F32;
  // B fragments of S: (kb, mt) -> 64 lanes x 8 values, as bf16 hi + lo or float32
  constexpr int FRAG_U32 = SPLIT ? 64 * 4 * 2 : 64 * 8;  // 32-bit words per fragment
  __shared__ __align__(16) uint32_t sb[KB * NT * FRAG_U32];

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int g = lane >> 4, ln = lane & 15;

  // work item: n_heads chains of NCB column blocks, the blocks of one chain
  // numbered to land on one XCD back to back (workgroups are dealt to the 8
  // XCDs round-robin); chains past the last full group of 8 keep linear order
  const int n_chains = static_cast<int>(gridDim.x) / NCB;
  const int full = (n_chains / 8) * 8 * NCB;
  int chain, cb;
  if (static_cast<int>(blockIdx.x) < full) {
    const int slot = blockIdx.x / 8;
    chain = (slot / NCB) * 8 + blockIdx.x % 8;
    cb = slot % NCB;
  } else {
    const int b = blockIdx.x - full;
    chain = full / NCB + b / NCB;
    cb = b % NCB;
  }
  // Split grids are request-major.  Full-width grids are head-major: the
  // workgroups resident at one time then draw on one head's slice of the pool
  // (n_pool x 128 KiB at d = 128), which the memory-side cache can keep while
  // the incoming states stream past it (written non-temporally, below).
  const int n_req = n_chains / args.h_v;
  const int req = (NCB == 1) ? chain % n_req : chain / args.h_v;
  const int h = (NCB == 1) ? chain / n_req : chain % args.h_v;
  const int c0 = cb * NC;
  const long state_sz = static_cast<long>(DK) * DV;
  const long hs = static_cast<long>(req) * args.h_v + h;
  const int row0 = wave * 16;  // this wave's state rows

  // element (mt, i) of a state tile: S[row0 + 4g + i][c0 + 16mt + ln]
  auto tile_ptr = [&](const float* base, int mt) __attribute__((always_inline)) {
    return base + static_cast<long>(row0 + 4 * g) * DV + c0 + 16 * mt + ln;
  };

  f32x4 s[NT];
  if (args.S_prefix != nullptr) {
    const float* pre = args.S_prefix + hs * state_sz;
#pragma unroll
    for (int mt = 0; mt < NT; ++mt)
#pragma unroll
      for (int i = 0; i < 4; ++i) s[mt][i] = tile_ptr(pre, mt)[i * DV];
  } else {
#pragma unroll
    for (int mt = 0; mt < NT; ++mt) s[mt] = zero4();
  }

  // publish: tile mt of wave w fills slots 4(w % 2) .. +3 of fragment (w / 2, mt)
  auto publish = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int mt = 0; mt < NT; ++mt) {
      uint32_t* f = sb + ((wave >> 1) * NT + mt) * FRAG_U32;
      if constexpr (SPLIT) {
        u16x4 hi, lo;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const __bf16 hb = static_cast<__bf16>(s[mt][i]);
          hi[i] = __builtin_bit_cast(u16, hb);
          lo[i] = bf16_bits(s[mt][i] - static_cast<float>(hb));
        }
        *reinterpret_cast<u16x4*>(f + lane * 4 + 2 * (wave & 1)) = hi;
        *reinterpret_cast<u16x4*>(f + 64 * 4 + lane * 4 + 2 * (wave & 1)) = lo;
      } else {
        *reinterpret_cast<float4*>(f + lane * 8 + 4 * (wave & 1)) =
            make_float4(s[mt][0], s[mt][1], s[mt][2], s[mt][3]);
      }
    }
  };
  publish();
  lds_barrier();  // (no wave reads what another writes to HBM: loads stay in flight)

  // Pool tuple of one step: this lane's row of P_hat as A fragments (k slots
  // kap(g, .) of each 32-block), the S_seg tile elements and log_decay.
  // LOOK register sets: the tuple of step j + LOOK is loaded while step j
  // computes.  Split grids are latency-bound and look two steps ahead; the
  // full-width state of an unsplit grid leaves registers for one.
  constexpr int LOOK = (NCB > 1) ? 2 : 1;
  struct Tuple {
    float p[KB][8];
    f32x4 s[NT];
    float e;
  };
  const int j0 = args.req_offsets[req], j1 = args.req_offsets[req + 1];
  // the request's first 64 segment ids, one per lane, so that a step's tuple
  // address does not wait for a load of its id
  const int my_id = (j0 + lane < j1) ? args.seg_ids[j0 + lane] : 0;
  auto load_step = [&](Tuple& t, int j) __attribute__((always_inline)) {
    const int id = (j - j0 < 64) ? __builtin_amdgcn_readlane(my_id, j - j0) : args.seg_ids[j];
    const long sh = static_cast<long>(id) * args.h_v + h;
    const float* Pi = args.P_hat + sh * DK * DK + static_cast<long>(row0 + ln) * DK + 4 * g;
    const float* Si = args.S_seg + sh * state_sz;
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      const float4 a = *reinterpret_cast<const float4*>(Pi + 32 * kb);
      const float4 b = *reinterpret_cast<const float4*>(Pi + 32 * kb + 16);
      t.p[kb][0] = a.x; t.p[kb][1] = a.y; t.p[kb][2] = a.z; t.p[kb][3] = a.w;
      t.p[kb][4] = b.x; t.p[kb][5] = b.y; t.p[kb][6] = b.z; t.p[kb][7] = b.w;
    }
#pragma unroll
    for (int mt = 0; mt < NT; ++mt)
#pragma unroll
      for (int i = 0; i < 4; ++i) t.s[mt][i] = tile_ptr(Si, mt)[i * DV];
    // the exponential is taken when the step uses it: taking it here would
    // make the wave wait for this load, and with it (loads complete in order)
    // for every row of the tuple just requested
    t.e = args.log_decay[sh];
  };
  // one composition step with the tuple t (step j), then the load of step
  // j + LOOK into t
  auto step = [&](Tuple& t, int j) __attribute__((always_inline)) {
    // A operand of this step, split once
    bf16x8 ah[KB], al[KB];
    float af[KB][8];
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      if constexpr (SPLIT) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          ah[kb][e] = static_cast<__bf16>(t.p[kb][e]);
          al[kb][e] = static_cast<__bf16>(t.p[kb][e] - static_cast<float>(ah[kb][e]));
        }
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) af[kb][e] = t.p[kb][e];
      }
    }
    f32x4 cS[NT];
#pragma unroll
    for (int mt = 0; mt < NT; ++mt) cS[mt] = t.s[mt];
    const float e = __expf(t.e);
    if (j + LOOK < j1) load_step(t, j + LOOK);
    if (args.S_incoming != nullptr) {
      float* dst = args.S_incoming + (static_cast<long>(j) * args.h_v + h) * state_sz;
#pragma unroll
      for (int mt = 0; mt < NT; ++mt)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          __builtin_nontemporal_store(s[mt][i], const_cast<float*>(tile_ptr(dst, mt)) + i * DV);
    }
#pragma unroll
    for (int mt = 0; mt < NT; ++mt) {
      f32x4 acc = zero4();
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
        const uint32_t* f = sb + (kb * NT + mt) * FRAG_U32;
        if constexpr (SPLIT) {
          const bf16x8 bh = *reinterpret_cast<const bf16x8*>(f + lane * 4);
          const bf16x8 bl = *reinterpret_cast<const bf16x8*>(f + 64 * 4 + lane * 4);
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah[kb], bh, acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah[kb], bl, acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al[kb], bh, acc, 0, 0, 0);
        } else {
          const float4 b0 = *reinterpret_cast<const float4*>(f + lane * 8);
          const float4 b1 = *reinterpret_cast<const float4*>(f + lane * 8 + 4);
          const float bv[8] = {b0.x, b0.y, b0.z, b0.w, b1.x, b1.y, b1.z, b1.w};
#pragma unroll
          for (int q = 0; q < 8; ++q)
            acc = __builtin_amdgcn_mfma_f32_16x16x4f32(af[kb][q], bv[q], acc, 0, 0, 0);
        }
      }
      s[mt] = acc * e + cS[mt];
    }
    lds_barrier();  // every wave has read the old state
    publish();
    lds_barrier();
  };
  if constexpr (LOOK == 2) {
    Tuple ta, tb;
    if (j0 < j1) load_step(ta, j0);
    if (j0 + 1 < j1) load_step(tb, j0 + 1);
    for (int j = j0; j < j1; j += 2) {
      step(ta, j);
      if (j + 1 < j1) step(tb, j + 1);
    }
  } else {
    Tuple ta;
    if (j0 < j1) load_step(ta, j0);
    for (int j = j0; j < j1; ++j) step(ta, j);
  }

  float* out = args.S_out + hs * state_sz;
#pragma unroll
  for (int mt = 0; mt < NT; ++mt)
#pragma unroll
    for (int i = 0; i < 4; ++i) const_cast<float*>(tile_ptr(out, mt))[i * DV] = s[mt][i];
}

template <int DK, int DV, int P>
hipError_t launch_compose_p(const ComposeArgs& a, int n_req, hipStream_t s) {
  const long heads = static_cast<long>(n_req) * a.h_v;
  const dim3 block(DK * 4);  // one wave per 16 state rows
  // split the columns of each head over 8 (d_v = 128) or 4 workgroups while
  // that keeps the grid within two workgroups per compute unit: a short
  // request's chain of dependent steps then runs on more compute units (8
  // blocks take the 8-segment, 16-head chain from 28.8 to 26.0 us)
  if constexpr (DV >= 128) {
    if (heads * 8 <= 512) {
      hipLaunchKernelGGL((compose_kernel<DK, DV, P, 8>), dim3(heads * 8), block, 0, s, a);
      return hipGetLastError();
    }
  }
  if (heads * 4 <= 512) {
    hipLaunchKernelGGL((compose_kernel<DK, DV, P, 4>), dim3(heads * 4), block, 0, s, a);
  } else {
    hipLaunchKernelGGL((compose_kernel<DK, DV, P, 1>), dim3(heads), block, 0, s, a);
  }
  return hipGetLastError();
}

template <int DK, int DV>
hipError_t launch_compose_d(const ComposeArgs& a, int f32, int n_req, hipStream_t s) {
  if (f32) return launch_compose_p<DK, DV, P_F32>(a, n_req, s);
  return launch_compose_p<DK, DV, P_SPLIT>(a, n_req, s);
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
