// Matrix-core helpers for gfx950 (CDNA4): 16x16 output tiles contracted over
// blocks of 32 k-values, in four precisions.
//
// Fragment convention.  A 64-lane wave is split into 4 lane groups
// g = lane / 16; r = lane % 16 names the tile row (A operand) or tile column
// (B operand).  For one 32-wide k block, element j (0..7) of a lane holds the
// k index kap(g, j):
//     j < 4 : 4 g + j           j >= 4 : 16 + 4 g + (j - 4)
// A operand: a[j] = A[row r][kb + kap(g, j)];  B operand: b[j] = B[kb + kap(g, j)][col r].
// The matrix core pairs element j of lane group g of A with the same slot of B,
// so any bijection works as long as A and B agree; this one makes the
// accumulator layout of two stacked 16x16 result tiles (lane (g, n) holds rows
// 4g..4g+3 of column n) directly usable as a B operand (or a transposed A
// operand) of the next product, with no data movement.
//
// Accumulator layout (16x16 f32 tile, both instruction shapes used here):
// lane (g, n) holds C[4 g + i][n], i = 0..3.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hypic {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

// Precision of one 16x16x32 product block.
enum Prec : int {
  P_F32 = 0,      // float32 matrix cores (v_mfma_f32_16x16x4_f32), 8 steps
  P_BF16 = 1,     // both operands rounded to bf16, one bf16 pass
  P_SPLIT_A = 2,  // A split hi+lo, B exact in bf16: 2 passes
  P_SPLIT_B = 3,  // B split hi+lo, A exact in bf16: 2 passes
  P_SPLIT = 4     // both split: hi*hi + hi*lo + lo*hi, 3 passes
};

__device__ __forceinline__ int kap(int g, int j) {
  return (j < 4) ? (4 * g + j) : (12 + 4 * g + j);
}

__device__ __forceinline__ float bf16_bits_to_f32(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// Element load with conversion to float from either storage type.
__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(uint16_t x) { return bf16_bits_to_f32(x); }

template <int P>
__device__ __forceinline__ void mma_blk(f32x4& acc, const float (&a)[8],
                                        const float (&b)[8]) {
  if constexpr (P == P_F32) {
#pragma unroll
    for (int j = 0; j < 8; ++j)
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[j], b[j], acc, 0, 0, 0);
  } else {
    bf16x8 ah, bh;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      ah[j] = static_cast<__bf16>(a[j]);
      bh[j] = static_cast<__bf16>(b[j]);
    }
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bh, acc, 0, 0, 0);
    if constexpr (P == P_SPLIT || P == P_SPLIT_B) {
      bf16x8 bl;
#pragma unroll
      for (int j = 0; j < 8; ++j)
        bl[j] = static_cast<__bf16>(b[j] - static_cast<float>(bh[j]));
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bl, acc, 0, 0, 0);
    }
    if constexpr (P == P_SPLIT || P == P_SPLIT_A) {
      bf16x8 al;
#pragma unroll
      for (int j = 0; j < 8; ++j)
        al[j] = static_cast<__bf16>(a[j] - static_cast<float>(ah[j]));
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, bh, acc, 0, 0, 0);
    }
  }
}

// a[j] = M[row * ld + kb + kap(g, j)]   (k contiguous in memory)
template <typename T>
__device__ __forceinline__ void frag_kcontig(const T* M, int ld, int row, int kb,
                                             int g, float (&a)[8]) {
  const T* p = M + static_cast<long>(row) * ld + kb + 4 * g;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    a[j] = to_f32(p[j]);
    a[4 + j] = to_f32(p[16 + j]);
  }
}

// b[j] = M[(kb + kap(g, j)) * ld + col]   (k strided in memory)
template <typename T>
__device__ __forceinline__ void frag_kstrided(const T* M, int ld, int col, int kb,
                                              int g, float (&b)[8]) {
#pragma unroll
  for (int j = 0; j < 8; ++j)
    b[j] = to_f32(M[static_cast<long>(kb + kap(g, j)) * ld + col]);
}

// Operand from two accumulator tiles covering k rows kb..kb+15 (lo) and
// kb+16..kb+31 (hi) of one 16-column tile.
__device__ __forceinline__ void frag_from_acc(const f32x4& lo, const f32x4& hi,
                                              float (&b)[8]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    b[i] = lo[i];
    b[4 + i] = hi[i];
  }
}

// Workgroup barrier for hand-offs through LDS only: waits for this wave's own
// LDS traffic, then meets the other waves.  Unlike __syncthreads() it does not
// drain outstanding global loads and stores, so register prefetches and result
// stores stay in flight across it.  Only for kernels in which no wave reads
// global memory that another wave of the same launch writes.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

__device__ __forceinline__ f32x4 zero4() {
  f32x4 z = {0.f, 0.f, 0.f, 0.f};
  return z;
}

}  // namespace hypic
