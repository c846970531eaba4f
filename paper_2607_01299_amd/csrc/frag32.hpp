// Matrix-core operand helpers of the pipelined chunk scans on gfx950.
//
// Products are v_mfma_f32_32x32x16_bf16 (state-side) and
// v_mfma_f32_16x16x32_bf16 (chunk-local tiles).  Operands are stored
// "fragment major": a 32 x 16 operand block is 64 lanes x 8 bf16 in lane
// order, read with one 16-byte load per lane.  Within a 16-deep contraction
// step, slot (g2, j) of lane group g2 = lane / 32 carries index
// 8(j / 4) + 4 g2 + j % 4, which is exactly the row set a 32 x 32 accumulator
// holds in elements 8h .. 8h+7, so accumulators feed the next product as
// operands with no data movement.  Rows of a state are kept in the order rho
// (true row = rho with bits 2 and 3 swapped): a 16-deep step over rho then
// covers 8 contiguous true rows per lane group, which is how q and k rows
// arrive from HBM (16 contiguous bytes per lane).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mfma.hpp"

namespace hypic {
namespace f32frag {

constexpr int FR = 512;  // u16 elements of one fragment (64 lanes x 8 bf16)

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned short u16;
typedef u16 u16x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f32x16 zero16() {
  f32x16 z;
#pragma unroll
  for (int i = 0; i < 16; ++i) z[i] = 0.f;
  return z;
}
__device__ __forceinline__ f32x16 mma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
// 16 x 16 x 32: lane (g, n) of A holds A[n][8g .. 8g+7], of B holds B^T[n][8g ..
// 8g+7]; the result lane (g, n) holds (A B)[4g + e][n], i.e. sum_k A[4g+e][k] B^T[n][k]
__device__ __forceinline__ f32x4 mma16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// a float32 operand held as bf16 hi + lo (about 2^-16 relative)
struct Split8 {
  bf16x8 h, l;
};
__device__ __forceinline__ Split8 split8(const float (&x)[8]) {
  Split8 r;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    r.h[j] = static_cast<__bf16>(x[j]);
    r.l[j] = static_cast<__bf16>(x[j] - static_cast<float>(r.h[j]));
  }
  return r;
}
// three bf16 passes (hi*hi + hi*lo + lo*hi) of a 16 x 16 x 32 product
__device__ __forceinline__ f32x4 mma16_x3(const Split8& a, const Split8& b, f32x4 c) {
  c = mma16(a.h, b.h, c);
  c = mma16(a.h, b.l, c);
  return mma16(a.l, b.h, c);
}

// elements 8h .. 8h+7 of a 32 x 32 accumulator: one 16-deep operand step
__device__ __forceinline__ bf16x8 frag_of(const f32x16& a, int h) {
  bf16x8 r;
#pragma unroll
  for (int j = 0; j < 8; ++j) r[j] = static_cast<__bf16>(a[8 * h + j]);
  return r;
}
__device__ __forceinline__ void split_of(const f32x16& a, int h, bf16x8& hi, bf16x8& lo) {
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const float x = a[8 * h + j];
    hi[j] = static_cast<__bf16>(x);
    lo[j] = static_cast<__bf16>(x - static_cast<float>(hi[j]));
  }
}

__device__ __forceinline__ bf16x8 ldf(const u16* base, int f, int lane) {
  return *reinterpret_cast<const bf16x8*>(base + f * FR + lane * 8);
}
__device__ __forceinline__ void stf(u16* base, int f, int lane, bf16x8 v) {
  *reinterpret_cast<bf16x8*>(base + f * FR + lane * 8) = v;
}

__device__ __forceinline__ uint4 mask4(uint4 w, bool keep) {
  const uint32_t m = keep ? 0xffffffffu : 0u;
  return make_uint4(w.x & m, w.y & m, w.z & m, w.w & m);
}
__device__ __forceinline__ bf16x8 as_bf(uint4 w) { return __builtin_bit_cast(bf16x8, w); }
__device__ __forceinline__ bf16x8 masked(uint4 w, bool keep) { return as_bf(mask4(w, keep)); }

__device__ __forceinline__ u16 bf16_bits(float x) {
  __bf16 h = static_cast<__bf16>(x);
  return __builtin_bit_cast(u16, h);
}
// the 8 bf16 of a 16-byte load as float32
__device__ __forceinline__ void unpack8(uint4 w, float (&x)[8]) {
  const uint32_t d[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    x[2 * i] = __uint_as_float(d[i] << 16);
    x[2 * i + 1] = __uint_as_float(d[i] & 0xffff0000u);
  }
}

// true row of element (tile m, element e) held by lane group g2 of a state
// accumulator: rho = 32m + 8(e/4) + 4 g2 + e%4 with bits 2, 3 swapped
__device__ __forceinline__ int true_row(int m, int e, int g2) {
  const int b = e >> 2;
  return 32 * m + 16 * (b >> 1) + 8 * g2 + 4 * (b & 1) + (e & 3);
}
// token (or contraction index) carried by slot j of lane group g2 in step s
__device__ __forceinline__ int slot_idx(int s, int g2, int j) {
  return 16 * s + 8 * (j >> 2) + 4 * g2 + (j & 3);
}
// index of fragment (row tile t, step s) in the 6-fragment lower-triangular
// sets (t = 0: s = 0, 1; t = 1: s = 0..3)
__device__ __forceinline__ int tri_idx(int t, int s) { return (t == 0) ? s : 2 + s; }

// u16 offset of the four slots 4(g/2) .. +3 of lane 32(g%2) + 16h + n in
// fragment f: where lane (g, n) of a 16 x 16 accumulator tile (rows 4g + e)
// lands in a 32x32-layout operand fragment whose 16-deep step is that tile's
// rows and whose 32-wide side holds the tile's columns at offset 16h
__device__ __forceinline__ int scatter_off(int f, int h, int lane) {
  const int g = lane >> 4, n = lane & 15;
  return f * FR + (32 * (g & 1) + 16 * h + n) * 8 + 4 * (g >> 1);
}
__device__ __forceinline__ u16x4 pack4(float a, float b, float c, float d) {
  u16x4 r;
  r[0] = bf16_bits(a);
  r[1] = bf16_bits(b);
  r[2] = bf16_bits(c);
  r[3] = bf16_bits(d);
  return r;
}

// raw 16-byte loads of the 32x32-layout fragments of one token tile of a
// token-major bf16 matrix: lane (g2, r) gets row 32t + r, columns 16u + 8g2 ..
// +7 for u = 0 .. NU-1 (rows past the chunk are clamped; zeroed at use)
template <int NU>
__device__ __forceinline__ void load_tile32(uint4 (&dst)[NU], const u16* base, long rs, int c0,
                                            int n, int t, int lane) {
  const int tok = 32 * t + (lane & 31);
  const int tc = (tok < n) ? tok : n - 1;
  const u16* p = base + static_cast<long>(c0 + tc) * rs + 8 * (lane >> 5);
#pragma unroll
  for (int u = 0; u < NU; ++u) dst[u] = *reinterpret_cast<const uint4*>(p + 16 * u);
}

// DPP row operation (16-lane rows) on a float: CTRL 0x111.. row_shr, 0x15F
// row_newbcast:15; lanes without a source read zero
template <int CTRL>
__device__ __forceinline__ float dpp_row(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xf, 0xf, true));
}
// inclusive prefix sum over the 16 lanes of each row
__device__ __forceinline__ float row_scan16(float v) {
  v += dpp_row<0x111>(v);
  v += dpp_row<0x112>(v);
  v += dpp_row<0x114>(v);
  v += dpp_row<0x118>(v);
  return v;
}
// lane 15 of each row, to every lane of the row
__device__ __forceinline__ float row_last(float v) { return dpp_row<0x15F>(v); }

}  // namespace f32frag
}  // namespace hypic
