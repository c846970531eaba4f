// Fragment, LDS and buffer helpers shared by the chunked scans of the
// transition families (family.hip) and of the KDA row of Tab. 1 (kda.hip).
//
// Fragments follow the convention of mfma.hpp: for one 32-wide k block, slot j
// of lane group g = lane / 16 holds k index kb + kap(g, j), and lane % 16 names
// the row (A operand) or the column (B operand).  Operands are bf16 bit
// patterns (u16) or float32; the float32 form runs on the float32 matrix cores.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mfma.hpp"

namespace hypic {
namespace {

typedef unsigned short u16;
typedef u16 u16x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float ldv(const u16* p) { return bf16_bits_to_f32(*p); }
__device__ __forceinline__ float ldv(const float* p) { return *p; }
__device__ __forceinline__ void stv(u16* p, float x) {
  *p = __builtin_bit_cast(u16, static_cast<__bf16>(x));
}
__device__ __forceinline__ void stv(float* p, float x) { *p = x; }

// A 16x16x32 operand in the native type of the matrix-core path: slot j of lane
// group g carries contraction index kap(g, j) (see mfma.hpp).
template <typename ST>
struct Frag;
template <>
struct Frag<u16> {
  bf16x8 x;
  __device__ void set(int j, float v) { x[j] = static_cast<__bf16>(v); }
};
template <>
struct Frag<float> {
  float x[8];
  __device__ void set(int j, float v) { x[j] = v; }
};

__device__ __forceinline__ f32x4 mma(const Frag<u16>& a, const Frag<u16>& b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a.x, b.x, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mma(const Frag<float>& a, const Frag<float>& b, f32x4 c) {
#pragma unroll
  for (int j = 0; j < 8; ++j) c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.x[j], b.x[j], c, 0, 0, 0);
  return c;
}

// slot j = M[row][kb + kap(g, j)]: two 8-byte (bf16) or 16-byte (float) loads
__device__ __forceinline__ Frag<u16> frag_row(const u16* M, int ld, int row, int kb, int g) {
  const u16* p = M + row * ld + kb + 4 * g;
  const u16x4 lo = *reinterpret_cast<const u16x4*>(p);
  const u16x4 hi = *reinterpret_cast<const u16x4*>(p + 16);
  Frag<u16> f;
  f.x = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
  return f;
}
__device__ __forceinline__ Frag<float> frag_row(const float* M, int ld, int row, int kb, int g) {
  const float* p = M + row * ld + kb + 4 * g;
  const float4 lo = *reinterpret_cast<const float4*>(p);
  const float4 hi = *reinterpret_cast<const float4*>(p + 16);
  Frag<float> f;
  f.x[0] = lo.x; f.x[1] = lo.y; f.x[2] = lo.z; f.x[3] = lo.w;
  f.x[4] = hi.x; f.x[5] = hi.y; f.x[6] = hi.z; f.x[7] = hi.w;
  return f;
}
// frag_row over a token-minor operand stored with its 4-token groups permuted:
// token t of the row sits at t ^ x (x a multiple of 8, uniform over the wave)
__device__ __forceinline__ Frag<u16> frag_row_sw(const u16* M, int ld, int row, int kb, int g,
                                                 int x) {
  const u16* p = M + row * ld;
  const u16x4 lo = *reinterpret_cast<const u16x4*>(p + ((kb + 4 * g) ^ x));
  const u16x4 hi = *reinterpret_cast<const u16x4*>(p + ((kb + 16 + 4 * g) ^ x));
  Frag<u16> f;
  f.x = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
  return f;
}
// slot j = M[row][kb + kap(g, j)] * s[kb + kap(g, j)]
template <typename ST>
__device__ __forceinline__ Frag<ST> frag_row_scaled(const ST* M, int ld, int row, int kb, int g,
                                                    const float* s) {
  const Frag<ST> raw = frag_row(M, ld, row, kb, g);
  const float4 s0 = *reinterpret_cast<const float4*>(s + kb + 4 * g);
  const float4 s1 = *reinterpret_cast<const float4*>(s + kb + 16 + 4 * g);
  const float sv[8] = {s0.x, s0.y, s0.z, s0.w, s1.x, s1.y, s1.z, s1.w};
  Frag<ST> f;
#pragma unroll
  for (int j = 0; j < 8; ++j) f.set(j, static_cast<float>(raw.x[j]) * sv[j]);
  return f;
}

// Split-bf16 operands: a float32 value x is carried as hi = bf16(x) and
// lo = bf16(x - hi), about 2^-16 relative together, and a product of two such
// operands runs as three bf16 passes (hi hi + hi lo + lo hi).  Used where one
// bf16 rounding of a gate-scaled operand is too coarse: an intra-chunk score
// q_t . k_i that nearly cancels.
__device__ __forceinline__ float bf16_round(float x) {
  return static_cast<float>(static_cast<__bf16>(x));
}
struct SplitFrag {
  Frag<u16> h, l;
};
__device__ __forceinline__ f32x4 mma3(const SplitFrag& a, const SplitFrag& b, f32x4 c) {
  c = mma(a.h, b.h, c);
  c = mma(a.h, b.l, c);
  return mma(a.l, b.h, c);
}
// slot j = M[row][kb + kap(g, j)] with M held as hi + lo arrays of one layout
__device__ __forceinline__ SplitFrag frag_row_split(const u16* Mh, const u16* Ml, int ld, int row,
                                                    int kb, int g) {
  SplitFrag f;
  f.h = frag_row(Mh, ld, row, kb, g);
  f.l = frag_row(Ml, ld, row, kb, g);
  return f;
}
// slot j = (Mh + Ml)[row][kb + kap(g, j)] * s[kb + kap(g, j)], split again
__device__ __forceinline__ SplitFrag frag_row_split_scaled(const u16* Mh, const u16* Ml, int ld,
                                                           int row, int kb, int g,
                                                           const float* s) {
  const Frag<u16> rh = frag_row(Mh, ld, row, kb, g), rl = frag_row(Ml, ld, row, kb, g);
  const float4 s0 = *reinterpret_cast<const float4*>(s + kb + 4 * g);
  const float4 s1 = *reinterpret_cast<const float4*>(s + kb + 16 + 4 * g);
  const float sv[8] = {s0.x, s0.y, s0.z, s0.w, s1.x, s1.y, s1.z, s1.w};
  SplitFrag f;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const float x = (static_cast<float>(rh.x[j]) + static_cast<float>(rl.x[j])) * sv[j];
    const float xh = bf16_round(x);
    f.h.set(j, xh);
    f.l.set(j, x - xh);
  }
  return f;
}
// slot j = (Mh + Ml)[row][kb + kap(g, j)] * s[kb + kap(g, j)], rounded once
__device__ __forceinline__ Frag<u16> frag_row_sum_scaled(const u16* Mh, const u16* Ml, int ld,
                                                         int row, int kb, int g,
                                                         const float* s) {
  const Frag<u16> rh = frag_row(Mh, ld, row, kb, g), rl = frag_row(Ml, ld, row, kb, g);
  const float4 s0 = *reinterpret_cast<const float4*>(s + kb + 4 * g);
  const float4 s1 = *reinterpret_cast<const float4*>(s + kb + 16 + 4 * g);
  const float sv[8] = {s0.x, s0.y, s0.z, s0.w, s1.x, s1.y, s1.z, s1.w};
  Frag<u16> f;
#pragma unroll
  for (int j = 0; j < 8; ++j)
    f.set(j, (static_cast<float>(rh.x[j]) + static_cast<float>(rl.x[j])) * sv[j]);
  return f;
}

// index of the tile pair (tq, tk), tk < tq, in fx
__device__ __forceinline__ int pair_idx(int tq, int tk) { return tq * (tq - 1) / 2 + tk; }

// eight consecutive elements of one row, packed for one 16-byte (bf16) or two
// 16-byte (float) LDS stores
__device__ __forceinline__ void st8(u16* p, const float (&x)[8]) {
  bf16x8 b;
#pragma unroll
  for (int j = 0; j < 8; ++j) b[j] = static_cast<__bf16>(x[j]);
  *reinterpret_cast<bf16x8*>(p) = b;
}
__device__ __forceinline__ void st8(float* p, const float (&x)[8]) {
  *reinterpret_cast<float4*>(p) = make_float4(x[0], x[1], x[2], x[3]);
  *reinterpret_cast<float4*>(p + 4) = make_float4(x[4], x[5], x[6], x[7]);
}
// element e of a 16-byte register load of the input type, and its raw bits
__device__ __forceinline__ uint32_t word_of(const uint4& w, int i) {
  return (i == 0) ? w.x : ((i == 1) ? w.y : ((i == 2) ? w.z : w.w));
}
__device__ __forceinline__ float elem(const uint4& w, int e, const u16*) {
  const uint32_t word = word_of(w, e >> 1);
  return __uint_as_float((e & 1) ? (word & 0xffff0000u) : (word << 16));
}
__device__ __forceinline__ float elem(const uint4& w, int e, const float*) {
  return __uint_as_float(word_of(w, e));
}
// element e of two bf16 rows, a in the low half and b in the high half
__device__ __forceinline__ uint32_t pair_raw(const uint4& a, const uint4& b, int e) {
  const uint32_t wa = word_of(a, e >> 1), wb = word_of(b, e >> 1);
  return (e & 1) ? ((wa >> 16) | (wb & 0xffff0000u)) : ((wa & 0xffffu) | (wb << 16));
}
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
  return static_cast<uint32_t>(__builtin_bit_cast(u16, static_cast<__bf16>(lo))) |
         (static_cast<uint32_t>(__builtin_bit_cast(u16, static_cast<__bf16>(hi))) << 16);
}
__device__ __forceinline__ void put_raw(u16* p, const uint4& w, int e) {
  const uint32_t word = word_of(w, e >> 1);
  *p = static_cast<u16>((e & 1) ? (word >> 16) : (word & 0xffffu));
}
__device__ __forceinline__ void put_raw(float* p, const uint4& w, int e) {
  *p = __uint_as_float(word_of(w, e));
}

// Buffer resources over [base, base + bytes): loads past the end return zero and
// stores past it are dropped by the hardware, so a partial chunk needs no
// branch around its memory operations (and every iteration issues the same
// number of them, which keeps the compiler's waits on earlier loads partial).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* base, long bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0,
                                           static_cast<int>(bytes > 0 ? bytes : 0), 0x00020000);
}
__device__ __forceinline__ uint4 bload16(__amdgpu_buffer_rsrc_t r, int off) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}
__device__ __forceinline__ float bload4(__amdgpu_buffer_rsrc_t r, int off) {
  return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
}
__device__ __forceinline__ void bstore(__amdgpu_buffer_rsrc_t r, int off, float x, u16*) {
  __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(u16, static_cast<__bf16>(x)), r, off,
                                        0, 0);
}
__device__ __forceinline__ void bstore(__amdgpu_buffer_rsrc_t r, int off, float x, float*) {
  __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(x), r, off, 0, 0);
}

// Inclusive prefix sum over the 64 lanes of a wave with DPP moves (no LDS
// round trip): shifts by 1, 2, 4, 8 inside each row of 16 lanes, then the last
// lane of row 0 is added to row 1 (and of row 2 to row 3), then the last lane
// of row 1 to rows 2 and 3.  Lanes whose DPP source falls outside the row, or
// whose row is masked off, add zero.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ float dpp_add(float x) {
  const int v = __builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, ROW_MASK, 0xf, true);
  return x + __int_as_float(v);
}
__device__ __forceinline__ float wave_inclusive_sum(float x) {
  x = dpp_add<0x111, 0xf>(x);  // row_shr:1
  x = dpp_add<0x112, 0xf>(x);  // row_shr:2
  x = dpp_add<0x114, 0xf>(x);  // row_shr:4
  x = dpp_add<0x118, 0xf>(x);  // row_shr:8
  x = dpp_add<0x142, 0xa>(x);  // row_bcast:15 into rows 1 and 3
  x = dpp_add<0x143, 0xc>(x);  // row_bcast:31 into rows 2 and 3
  return x;
}

}  // namespace
}  // namespace hypic
