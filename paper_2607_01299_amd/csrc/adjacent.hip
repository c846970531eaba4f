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
// float32.  All three are elementwise streams with 16-byte accesses per lane,
// bounded by HBM bandwidth.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "family.hpp"

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
// grid (segment, 64-token block): blocks past a segment's end exit at once.
// Each lane moves 16 bytes (VEC elements, VEC / 2 channel pairs).
// ---------------------------------------------------------------------------
template <typename T>
struct alignas(16) Vec16 {
  static constexpr int N = 16 / static_cast<int>(sizeof(T));
  T v[N];
};

template <typename T, int D>
__global__ __launch_bounds__(256) void rope_keys_kernel(const T* k_in, T* k_out,
                                                        const int32_t* cu, const int32_t* delta,
                                                        int heads, double base) {
  constexpr int VEC = Vec16<T>::N;
  __shared__ float cs[D / 2], sn[D / 2];
  const int s = blockIdx.x;
  const int t0 = cu[s] + 64 * static_cast<int>(blockIdx.y);
  const int t1 = min(t0 + 64, cu[s + 1]);
  if (t0 >= t1) return;  // uniform across the workgroup
  rope_table(cs, sn, D, delta[s], base);
  const int per_row = heads * D / VEC;  // 16-byte pieces per token
  const long row = static_cast<long>(heads) * D;
  for (int idx = threadIdx.x; idx < (t1 - t0) * per_row; idx += 256) {
    const int t = t0 + idx / per_row, r = idx % per_row;
    const long o = t * row + static_cast<long>(r) * VEC;
    const int i0 = (r * VEC) % D / 2;  // first channel pair of this piece
    const Vec16<T> a = *reinterpret_cast<const Vec16<T>*>(k_in + o);
    Vec16<T> b;
#pragma unroll
    for (int p = 0; p < VEC / 2; ++p) {
      const float x = to_float(a.v[2 * p]), y = to_float(a.v[2 * p + 1]);
      const float c = cs[i0 + p], sv = sn[i0 + p];
      from_float(&b.v[2 * p], c * x - sv * y);
      from_float(&b.v[2 * p + 1], sv * x + c * y);
    }
    *reinterpret_cast<Vec16<T>*>(k_out + o) = b;
  }
}

// ---------------------------------------------------------------------------
// causal depthwise convolution over packed segments with carried conv state:
//   y[t, c] = act(sum_j w[c, j] xx[t + j, c]),  xx = concat(state_in[s], x[segment s])
// grid (segment, 64-token block, channel block); each lane carries VEC
// consecutive channels (one 16-byte load and store per token when the rows
// allow it, VEC = 1 otherwise) and slides a register window of the width - 1
// previous inputs down the block's tokens, loading eight tokens at a time.
// ---------------------------------------------------------------------------
constexpr int kMaxWidth = 8;

template <typename T, int VEC>
struct alignas(VEC * sizeof(T)) Piece {
  T v[VEC];
};

template <typename T, int VEC, int K>
__global__ __launch_bounds__(256) void conv_kernel(const T* x, const float* w, const int32_t* cu,
                                                   const float* state_in, T* y, float* state_out,
                                                   int C, int silu) {
  constexpr int TB = 8;  // tokens loaded together
  static_assert(TB >= K - 1, "the window must fit one batch");
  const int s = blockIdx.x;
  const int c0 = (blockIdx.z * 256 + threadIdx.x) * VEC;  // first channel of this lane
  const int lo = cu[s], hi = cu[s + 1];
  const int t0 = lo + 64 * static_cast<int>(blockIdx.y);
  if (c0 >= C) return;  // C is a multiple of VEC
  float wk[K][VEC];
#pragma unroll
  for (int j = 0; j < K; ++j)
#pragma unroll
    for (int e = 0; e < VEC; ++e) wk[j][e] = w[static_cast<long>(c0 + e) * K + j];
  auto load_x = [&](int t, float (&out)[VEC]) __attribute__((always_inline)) {
    const Piece<T, VEC> a =
        *reinterpret_cast<const Piece<T, VEC>*>(x + static_cast<long>(t) * C + c0);
#pragma unroll
    for (int e = 0; e < VEC; ++e) out[e] = to_float(a.v[e]);
  };
  // raw inputs at position p of xx (p < K - 1: the carried state)
  auto xx = [&](int p, float (&out)[VEC]) __attribute__((always_inline)) {
    if (p >= K - 1) {
      load_x(lo + p - (K - 1), out);
    } else {
#pragma unroll
      for (int e = 0; e < VEC; ++e)
        out[e] = state_in ? state_in[(static_cast<long>(s) * (K - 1) + p) * C + c0 + e] : 0.f;
    }
  };
  if (t0 < hi) {
    const int r0 = t0 - lo;  // first output row of this block within the segment
    // win[j]: the input K - 1 - j tokens before the next output's own input
    float win[K > 1 ? K - 1 : 1][VEC];
#pragma unroll
    for (int j = 0; j < K - 1; ++j) xx(r0 + j, win[j]);
    const int t1 = min(t0 + 64, hi);
    for (int tb = t0; tb < t1; tb += TB) {
      float cur[TB][VEC];
#pragma unroll
      for (int u = 0; u < TB; ++u) load_x((tb + u < t1) ? tb + u : t1 - 1, cur[u]);
#pragma unroll
      for (int u = 0; u < TB; ++u) {
        Piece<T, VEC> out;
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
          float acc = 0.f;
#pragma unroll
          for (int j = 0; j < K; ++j) {
            const int idx = u - (K - 1) + j;  // batch position of tap j's input
            acc += wk[j][e] * ((idx >= 0) ? cur[idx >= 0 ? idx : 0][e]
                                          : win[idx >= 0 ? 0 : K - 1 + idx][e]);
          }
          if (silu) acc = acc * __builtin_amdgcn_rcpf(1.f + __expf(-acc));
          from_float(&out.v[e], acc);
        }
        if (tb + u < t1)
          *reinterpret_cast<Piece<T, VEC>*>(y + static_cast<long>(tb + u) * C + c0) = out;
      }
      // the last K - 1 inputs of this batch precede the next one
#pragma unroll
      for (int j = 0; j < K - 1; ++j)
#pragma unroll
        for (int e = 0; e < VEC; ++e) win[j][e] = cur[TB - (K - 1) + j][e];
    }
  }
  // the block that holds the segment's first tokens hands on its last K - 1 inputs
  if (state_out != nullptr && blockIdx.y == 0) {
    const int L = hi - lo;
    for (int i = 0; i < K - 1; ++i) {
      float v[VEC];
      xx(L + i, v);
#pragma unroll
      for (int e = 0; e < VEC; ++e)
        state_out[(static_cast<long>(s) * (K - 1) + i) * C + c0 + e] = v[e];
    }
  }
}

template <typename T, int VEC>
hipError_t launch_conv_v(const T* x, const float* w, const int32_t* cu, const float* state_in,
                         T* y, float* state_out, int C, int K, int silu, dim3 grid,
                         hipStream_t s) {
  switch (K) {
#define HYPIC_CONV_CASE(KK)                                                                 \
  case KK:                                                                                  \
    hipLaunchKernelGGL((conv_kernel<T, VEC, KK>), grid, dim3(256), 0, s, x, w, cu, state_in, \
                       y, state_out, C, silu);                                              \
    break;
    HYPIC_CONV_CASE(1)
    HYPIC_CONV_CASE(2)
    HYPIC_CONV_CASE(3)
    HYPIC_CONV_CASE(4)
    HYPIC_CONV_CASE(5)
    HYPIC_CONV_CASE(6)
    HYPIC_CONV_CASE(7)
    HYPIC_CONV_CASE(8)
#undef HYPIC_CONV_CASE
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
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
  if (K < 1 || K > kMaxWidth) return hipErrorInvalidValue;
  // 16 bytes per lane when every row starts 16-byte aligned, one channel otherwise
  const int vec = (C % (bf16 ? 8 : 4) == 0) ? (bf16 ? 8 : 4) : 1;
  const dim3 grid(n_seg, max_len > 0 ? (max_len + 63) / 64 : 1, (C + 256 * vec - 1) / (256 * vec));
  if (bf16) {
    const u16* xi = static_cast<const u16*>(x);
    u16* yo = static_cast<u16*>(y);
    return (vec == 8) ? launch_conv_v<u16, 8>(xi, w, cu, state_in, yo, state_out, C, K, silu, grid, s)
                      : launch_conv_v<u16, 1>(xi, w, cu, state_in, yo, state_out, C, K, silu, grid, s);
  }
  const float* xi = static_cast<const float*>(x);
  float* yo = static_cast<float*>(y);
  return (vec == 4) ? launch_conv_v<float, 4>(xi, w, cu, state_in, yo, state_out, C, K, silu, grid, s)
                    : launch_conv_v<float, 1>(xi, w, cu, state_in, yo, state_out, C, K, silu, grid, s);
}

}  // namespace hypic
