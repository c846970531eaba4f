// Reuse-time steps next to the linear-attention cache on gfx950:
//   * the state RoPE shift of Eq. (7): S <- R(delta) S for a cached state whose
//     keys carried rotary position embeddings (scalar-transition models);
//   * the key re-rotation of Eq. (8): K_b = R(b - a) K_a for cached keys;
//   * the causal depthwise convolution with a carried conv state (Sec. 4.2
//     warm-up): each segment starts from the K - 1 raw inputs before it (zero
//     when cached alone) and hands its last K - 1 inputs on.
// R(p) rotates channel pairs (2i, 2i + 1) by p * base^(-2i/d).  Angles are
// formed and reduced in float64 (positions reach 1e5 and more, where a float32
// angle is off by far more than the result's precision), then applied in
// float32.  All three are elementwise streams: 16-byte accesses per lane where
// the layout allows, bounded by HBM bandwidth.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "scan.hpp"

namespace hypic {

namespace {

typedef unsigned short u16;

__device__ __forceinline__ float to_float(float x) { return x; }
__device__ __forceinline__ float to_float(u16 x) {
  return __uint_as_float(static_cast<uint32_t>(x) << 16);
}
__device__ __forceinline__ void from_float(float* p, float x) { *p = x; }
__device__ __forceinline__ void from_float(u16* p, float x) {
  *p = __builtin_bit_cast(u16, static_cast<__bf16>(x));
}

// cos / sin of delta * base^(-2i/d) for the d/2 pairs, into LDS (float64 angle)
__device__ __forceinline__ void rope_table(float* cs, float* sn, int d, long delta, double base) {
  for (int i = threadIdx.x; i < d / 2; i += blockDim.x) {
    const double theta = pow(base, -2.0 * static_cast<double>(i) / static_cast<double>(d));
    double s, c;
    sincos(static_cast<double>(delta) * theta, &s, &c);
    cs[i] = static_cast<float>(c);
    sn[i] = static_cast<float>(s);
  }
  __syncthreads();
}

// ---------------------------------------------------------------------------
// Eq. (7): S_out[e, h] = R(delta[e]) S_in[e, h]; one workgroup per (entry, head),
// each thread a pair of rows times four columns per step
// ---------------------------------------------------------------------------
template <int DK, int DV>
__global__ __launch_bounds__(256) void rope_state_kernel(const float* S_in, float* S_out,
                                                         const int32_t* delta, int h_v,
                                                         double base) {
  __shared__ float cs[DK / 2], sn[DK / 2];
  const int e = blockIdx.x / h_v;
  rope_table(cs, sn, DK, delta[e], base);
  const long off = static_cast<long>(blockIdx.x) * DK * DV;
  const float* src = S_in + off;
  float* dst = S_out + off;
  constexpr int NQ = DV / 4;                 // float4 per row
  for (int idx = threadIdx.x; idx < (DK / 2) * NQ; idx += 256) {
    const int i = idx / NQ, c4 = idx % NQ;
    const float4 a = *reinterpret_cast<const float4*>(src + (2 * i) * DV + 4 * c4);
    const float4 b = *reinterpret_cast<const float4*>(src + (2 * i + 1) * DV + 4 * c4);
    const float c = cs[i], s = sn[i];
    *reinterpret_cast<float4*>(dst + (2 * i) * DV + 4 * c4) =
        make_float4(c * a.x - s * b.x, c * a.y - s * b.y, c * a.z - s * b.z, c * a.w - s * b.w);
    *reinterpret_cast<float4*>(dst + (2 * i + 1) * DV + 4 * c4) =
        make_float4(s * a.x + c * b.x, s * a.y + c * b.y, s * a.z + c * b.z, s * a.w + c * b.w);
  }
}

// ---------------------------------------------------------------------------
// Eq. (8): k_out[t, h] = R(delta[s]) k_in[t, h] for the tokens t of segment s;
// grid (segment, 64-token block): blocks past a segment's end exit at once
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ __launch_bounds__(256) void rope_keys_kernel(const T* k_in, T* k_out,
                                                        const int32_t* cu, const int32_t* delta,
                                                        int heads, double base) {
  __shared__ float cs[D / 2], sn[D / 2];
  const int s = blockIdx.x;
  const int t0 = cu[s] + 64 * static_cast<int>(blockIdx.y);
  const int t1 = min(t0 + 64, cu[s + 1]);
  if (t0 >= t1) return;  // uniform across the workgroup
  rope_table(cs, sn, D, delta[s], base);
  const int pairs = heads * (D / 2);
  const long row = static_cast<long>(heads) * D;
  for (int idx = threadIdx.x; idx < (t1 - t0) * pairs; idx += 256) {
    const int t = t0 + idx / pairs, r = idx % pairs;
    const int hh = r / (D / 2), i = r % (D / 2);
    const long o = t * row + hh * D + 2 * i;
    const float a = to_float(k_in[o]), b = to_float(k_in[o + 1]);
    from_float(k_out + o, cs[i] * a - sn[i] * b);
    from_float(k_out + o + 1, sn[i] * a + cs[i] * b);
  }
}

// ---------------------------------------------------------------------------
// causal depthwise convolution over packed segments with carried conv state:
//   y[t, c] = act(sum_j w[c, j] xx[t + j, c]),  xx = concat(state_in[s], x[segment s])
// grid (segment, 64-token block, 256-channel block)
// ---------------------------------------------------------------------------
constexpr int kMaxWidth = 8;

template <typename T>
__global__ __launch_bounds__(256) void conv_kernel(const T* x, const float* w, const int32_t* cu,
                                                   const float* state_in, T* y, float* state_out,
                                                   int C, int K, int silu) {
  const int s = blockIdx.x;
  const int c = blockIdx.z * 256 + threadIdx.x;
  const int lo = cu[s], hi = cu[s + 1];
  const int t0 = lo + 64 * static_cast<int>(blockIdx.y);
  if (c >= C) return;
  float wk[kMaxWidth], win[kMaxWidth];
#pragma unroll
  for (int j = 0; j < kMaxWidth; ++j) wk[j] = (j < K) ? w[static_cast<long>(c) * K + j] : 0.f;
  // raw input at position p of xx (p < K - 1: the carried state)
  auto xx = [&](int p) -> float {
    if (p >= K - 1) return to_float(x[static_cast<long>(lo + p - (K - 1)) * C + c]);
    return state_in ? state_in[(static_cast<long>(s) * (K - 1) + p) * C + c] : 0.f;
  };
  if (t0 < hi) {
    const int r0 = t0 - lo;  // first output row of this block within the segment
    // window: xx[r0 .. r0 + K - 2] precede the first output's own input
#pragma unroll
    for (int j = 0; j < kMaxWidth - 1; ++j) win[j] = (j < K - 1) ? xx(r0 + j) : 0.f;
    const int t1 = min(t0 + 64, hi);
    for (int t = t0; t < t1; ++t) {
      const float cur = to_float(x[static_cast<long>(t) * C + c]);
      float acc = 0.f;
#pragma unroll
      for (int j = 0; j < kMaxWidth - 1; ++j)
        if (j < K - 1) acc += wk[j] * win[j];
      // the newest input takes tap K - 1
#pragma unroll
      for (int j = 0; j < kMaxWidth; ++j)
        if (j == K - 1) acc += wk[j] * cur;
      if (silu) acc = acc / (1.f + __expf(-acc));
      from_float(y + static_cast<long>(t) * C + c, acc);
#pragma unroll
      for (int j = 0; j < kMaxWidth - 2; ++j) win[j] = win[j + 1];
#pragma unroll
      for (int j = 0; j < kMaxWidth - 1; ++j)
        if (j == K - 2) win[j] = cur;
    }
  }
  // the block that holds the segment's first tokens hands on its last K - 1 inputs
  if (state_out != nullptr && blockIdx.y == 0) {
    const int L = hi - lo;
    for (int i = 0; i < K - 1; ++i)
      state_out[(static_cast<long>(s) * (K - 1) + i) * C + c] = xx(L + i);
  }
}

template <int DK>
hipError_t launch_rope_state_d(const float* S_in, float* S_out, const int32_t* delta, int n,
                               int h_v, int d_v, double base, hipStream_t st) {
  const dim3 grid(static_cast<unsigned>(n) * h_v);
  if (d_v == 64)
    hipLaunchKernelGGL((rope_state_kernel<DK, 64>), grid, dim3(256), 0, st, S_in, S_out, delta,
                       h_v, base);
  else
    hipLaunchKernelGGL((rope_state_kernel<DK, 128>), grid, dim3(256), 0, st, S_in, S_out, delta,
                       h_v, base);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_rope_keys_t(const void* k_in, void* k_out, const int32_t* cu,
                              const int32_t* delta, int n_seg, int max_len, int heads, int d,
                              double base, hipStream_t st) {
  const dim3 grid(n_seg, (max_len + 63) / 64);
  if (d == 64)
    hipLaunchKernelGGL((rope_keys_kernel<T, 64>), grid, dim3(256), 0, st,
                       static_cast<const T*>(k_in), static_cast<T*>(k_out), cu, delta, heads,
                       base);
  else
    hipLaunchKernelGGL((rope_keys_kernel<T, 128>), grid, dim3(256), 0, st,
                       static_cast<const T*>(k_in), static_cast<T*>(k_out), cu, delta, heads,
                       base);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_rope_state(const float* S_in, float* S_out, const int32_t* delta, int n,
                             int h_v, int d_k, int d_v, double base, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (d_k == 64) return launch_rope_state_d<64>(S_in, S_out, delta, n, h_v, d_v, base, s);
  return launch_rope_state_d<128>(S_in, S_out, delta, n, h_v, d_v, base, s);
}

hipError_t launch_rope_keys(const void* k_in, void* k_out, int bf16, const int32_t* cu,
                            const int32_t* delta, int n_seg, int max_len, int heads, int d,
                            double base, hipStream_t s) {
  if (n_seg <= 0 || max_len <= 0) return hipSuccess;
  if (bf16)
    return launch_rope_keys_t<u16>(k_in, k_out, cu, delta, n_seg, max_len, heads, d, base, s);
  return launch_rope_keys_t<float>(k_in, k_out, cu, delta, n_seg, max_len, heads, d, base, s);
}

hipError_t launch_causal_conv(const void* x, const float* w, int bf16, const int32_t* cu,
                              int n_seg, int max_len, const float* state_in, void* y,
                              float* state_out, int C, int K, int silu, hipStream_t s) {
  if (n_seg <= 0) return hipSuccess;
  const dim3 grid(n_seg, max_len > 0 ? (max_len + 63) / 64 : 1, (C + 255) / 256);
  if (bf16)
    hipLaunchKernelGGL((conv_kernel<u16>), grid, dim3(256), 0, s, static_cast<const u16*>(x), w,
                       cu, state_in, static_cast<u16*>(y), state_out, C, K, silu);
  else
    hipLaunchKernelGGL((conv_kernel<float>), grid, dim3(256), 0, s, static_cast<const float*>(x),
                       w, cu, state_in, static_cast<float*>(y), state_out, C, K, silu);
  return hipGetLastError();
}

}  // namespace hypic
