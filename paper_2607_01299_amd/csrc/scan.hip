// Chunked gated-delta-rule scan for gfx950: segment build and seam rescan.
//
// One workgroup (4 waves) runs one (segment, v-head, role) chain over the
// segment's chunks in order.  Role S carries the state S (d_k x d_v) and emits
// the outputs; role P carries the decay-free operator P_hat (d_k x d_k).  Both
// roles recompute the chunk's Gram matrix and triangular solve, so the two
// chains of one head run on different compute units at the same time.
//
// Per chunk of C tokens (chunk-local index r = 0..C-1, incoming state S0),
// with b_r = sum_{s<=r} a_s, gamma_r = exp(b_r), Gamma_ri = exp(b_r - b_i) for
// i <= r (never above 1):
//   L   = strictly-lower part of diag(beta) K K^T
//   A1  = (I + L)^{-1}                         (decay-free UT transform)
//   W   = A1 diag(beta) K                      (decay-free WY factor)
//   W'  = diag(gamma) W,   U = (A1 . Gamma) diag(beta) V
//   Vn  = U - W' S0                            (the delta-rule corrected values)
//   O   = diag(gamma) Q S0 + (tril(Q K^T) . Gamma) Vn
//   S   <- gamma_{C-1} S0 + K^T diag(exp(b_{C-1} - b)) Vn
//   P   <- P0 - K^T (W P0)
// which is the token recurrence of Eq. (2) with the GDN transition of Tab. 1
// applied C times; (A1 . Gamma) is the gated UT transform because
// diag(gamma) A1 diag(gamma)^{-1} = A1 . Gamma elementwise.  P follows the
// identity-start construction of Sec. 5 with the gate factored out (Tab. 3).
//
// Precision: q, k, v are exact in bf16, so K K^T, Q K^T and every product with
// K as one operand lose nothing in the bf16 matrix cores.  The state path
// rounds its float32 operands to bf16 (the decay keeps that rounding from
// accumulating).  The operator path has no decay, so its float32 operands are
// split into bf16 hi + lo terms.  float32 inputs use float32 matrix cores.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mfma.hpp"
#include "scan.hpp"

namespace hypic {

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = 4;

template <typename TIn>
struct IoTraits;
template <>
struct IoTraits<uint16_t> {
  static constexpr int kVec = 8;  // elements per 16-byte load
  static constexpr int kPad = 8;  // row padding (elements) in LDS
  static constexpr int kQK = P_BF16;
  static constexpr int kS = P_BF16;       // state-path products
  static constexpr int kWop = P_SPLIT_A;  // W for the operator path (K exact)
  static constexpr int kP = P_SPLIT;      // W P0
  static constexpr int kKX = P_SPLIT_B;   // K^T X (K exact)
  __device__ static void store(uint16_t* p, float x) {
    __bf16 h = static_cast<__bf16>(x);
    *p = *reinterpret_cast<uint16_t*>(&h);
  }
};
template <>
struct IoTraits<float> {
  static constexpr int kVec = 4;
  static constexpr int kPad = 4;
  static constexpr int kQK = P_F32;
  static constexpr int kS = P_F32;
  static constexpr int kWop = P_F32;
  static constexpr int kP = P_F32;
  static constexpr int kKX = P_F32;
  __device__ static void store(float* p, float x) { *p = x; }
};

template <typename TIn, int DK, int DV, int C>
struct Smem {
  static constexpr int CP = (C < 32) ? 32 : C;  // padded token extent
  static constexpr int PADI = IoTraits<TIn>::kPad;
  static constexpr int LDK = DK + PADI;  // K, Q rows (input type)
  static constexpr int LDV = DV + PADI;  // V rows (input type)
  static constexpr int LDW = DK + 4;     // W rows (float)
  static constexpr int LDC = CP + 4;     // chunk x chunk matrices (float)
  static constexpr int QW_BYTES =
      (CP * LDW * 4 > CP * LDK * static_cast<int>(sizeof(TIn)))
          ? CP * LDW * 4
          : CP * LDK * static_cast<int>(sizeof(TIn));
  TIn k[CP * LDK];
  TIn v[CP * LDV];
  // Q (input type) during the first half of a chunk, then W or W' (float)
  alignas(16) unsigned char qw[QW_BYTES];
  float L[CP * LDC];   // strictly-lower diag(beta) K K^T
  float A[CP * LDC];   // (I + L)^{-1}
  float X[CP * LDC];   // tril(Q K^T) . Gamma
  float T[3 * 256];    // solve scratch
  float beta[CP];
  float b[CP];
};

// Blocked inverse of the unit lower-triangular I + L (16x16 diagonal blocks by
// forward substitution, off-diagonal blocks by
// A_ij = -A_ii sum_{k=j}^{i-1} L_ik A_kj, one block diagonal at a time).
template <int CP, int LDC>
__device__ void unit_lower_inverse(const float* L, float* A, float* T, int tid) {
  constexpr int NB = CP / 16;
  // diagonal blocks: thread (blk, j) solves column j of block blk
  if (tid < NB * 16) {
    const int blk = tid / 16, j = tid % 16;
    const int o = blk * 16;
    float x[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      float acc = (r == j) ? 1.f : 0.f;
#pragma unroll
      for (int i = 0; i < r; ++i) acc -= L[(o + r) * LDC + o + i] * x[i];
      x[r] = (r < j) ? 0.f : acc;
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) A[(o + r) * LDC + o + j] = x[r];
  }
  // strictly upper blocks are zero
  for (int idx = tid; idx < CP * CP; idx += kThreads) {
    const int r = idx / CP, c = idx % CP;
    if ((c / 16) > (r / 16)) A[r * LDC + c] = 0.f;
  }
  __syncthreads();
  for (int dist = 1; dist < NB; ++dist) {
    const int nblk = NB - dist;
    for (int idx = tid; idx < nblk * 256; idx += kThreads) {
      const int bl = idx / 256, e = idx % 256;
      const int bi = dist + bl, bj = bl;
      const int r = e / 16, c = e % 16;
      float acc = 0.f;
      for (int bk = bj; bk < bi; ++bk) {
#pragma unroll
        for (int m = 0; m < 16; ++m)
          acc += L[(bi * 16 + r) * LDC + bk * 16 + m] * A[(bk * 16 + m) * LDC + bj * 16 + c];
      }
      T[bl * 256 + e] = acc;
    }
    __syncthreads();
    for (int idx = tid; idx < nblk * 256; idx += kThreads) {
      const int bl = idx / 256, e = idx % 256;
      const int bi = dist + bl, bj = bl;
      const int r = e / 16, c = e % 16;
      float acc = 0.f;
#pragma unroll
      for (int m = 0; m < 16; ++m)
        acc += A[(bi * 16 + r) * LDC + bi * 16 + m] * T[bl * 256 + m * 16 + c];
      A[(bi * 16 + r) * LDC + bj * 16 + c] = -acc;
    }
    __syncthreads();
  }
}

// Copy `n` valid rows of a [rows, D] token tile from global (row stride `gstride`
// elements) into LDS (row stride LD); rows n..CP-1 are zero-filled.
template <typename TIn, int D, int LD, int CP>
__device__ void load_tile(TIn* dst, const TIn* src, long gstride, int n, int tid) {
  constexpr int VEC = IoTraits<TIn>::kVec;
  constexpr int PER_ROW = D / VEC;
  for (int idx = tid; idx < CP * PER_ROW; idx += kThreads) {
    const int r = idx / PER_ROW, cv = idx % PER_ROW;
    uint4 val = make_uint4(0u, 0u, 0u, 0u);
    if (r < n) val = *reinterpret_cast<const uint4*>(src + r * gstride + cv * VEC);
    *reinterpret_cast<uint4*>(dst + r * LD + cv * VEC) = val;
  }
}

template <typename TIn, int DK, int DV, int C>
__global__ __launch_bounds__(kThreads) void scan_kernel(ScanArgs args) {
  using SM = Smem<TIn, DK, DV, C>;
  using IO = IoTraits<TIn>;
  constexpr int CP = SM::CP;
  constexpr int LDK = SM::LDK, LDV = SM::LDV, LDW = SM::LDW, LDC = SM::LDC;
  constexpr int MTC = CP / 16;  // token tiles
  constexpr int MTK = DK / 16;  // d_k tiles (state rows)
  constexpr int SV = DV / kWaves, NTS = SV / 16;  // state columns per wave
  constexpr int SP = DK / kWaves, NTP = SP / 16;  // operator columns per wave
  constexpr int NTA = (NTS > NTP) ? NTS : NTP;
  static_assert(SV % 16 == 0 && SP % 16 == 0, "slab must be whole tiles");
  static_assert(sizeof(SM) <= 160 * 1024, "LDS budget");

  __shared__ SM sm;
  TIn* q_s = reinterpret_cast<TIn*>(sm.qw);
  float* w_s = reinterpret_cast<float*>(sm.qw);

  const int tid = threadIdx.x;
  const int wave = tid / 64, lane = tid % 64;
  const int g = lane / 16, ln = lane % 16;

  // ---- work item --------------------------------------------------------
  const int per_item = args.n_roles * args.h_v;
  const int rank = blockIdx.x / per_item;
  const int rem = blockIdx.x % per_item;
  const int role = rem % args.n_roles;  // 0: state, 1: operator
  const int h = rem / args.n_roles;
  const int hk = h / args.group;
  int seg, lo, hi;
  if (args.mode == 0) {
    seg = segment_of_rank(args, rank);
    lo = args.cu_seqlens[seg];
    hi = args.cu_seqlens[seg + 1];
  } else {
    seg = rank;
    lo = args.tok_start[seg];
    const int len = args.tok_len[seg];
    hi = lo + ((len < args.w) ? len : args.w);
  }
  lo = (lo < 0) ? 0 : ((lo > args.n_tokens) ? args.n_tokens : lo);
  hi = (hi < lo) ? lo : ((hi > args.n_tokens) ? args.n_tokens : hi);

  const TIn* kg = static_cast<const TIn*>(args.k);
  const TIn* qg = static_cast<const TIn*>(args.q);
  const TIn* vg = static_cast<const TIn*>(args.v);
  const long qk_stride = static_cast<long>(args.h_qk) * DK;
  const long v_stride = static_cast<long>(args.h_v) * DV;

  // ---- chain state: rows = d_k tiles, columns = this wave's slab ------------
  f32x4 st[MTK][NTA];
  const int col0 = wave * ((role == 0) ? SV : SP);
  const long sh = static_cast<long>(seg) * args.h_v + h;
  if (role == 0) {
    const float* s_in = (args.mode == 1) ? args.S_in + sh * DK * DV : nullptr;
#pragma unroll
    for (int mt = 0; mt < MTK; ++mt)
#pragma unroll
      for (int nt = 0; nt < NTS; ++nt)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          st[mt][nt][i] = s_in ? s_in[(mt * 16 + 4 * g + i) * DV + col0 + nt * 16 + ln] : 0.f;
  } else {
#pragma unroll
    for (int mt = 0; mt < MTK; ++mt)
#pragma unroll
      for (int nt = 0; nt < NTP; ++nt)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          st[mt][nt][i] = (mt * 16 + 4 * g + i == col0 + nt * 16 + ln) ? 1.f : 0.f;
  }
  float log_decay = 0.f;

  for (int c0 = lo; c0 < hi; c0 += C) {
    const int n = (hi - c0 < C) ? (hi - c0) : C;

    // ---- A: stage the chunk's tokens ----------------------------------------
    load_tile<TIn, DK, LDK, CP>(sm.k, kg + c0 * qk_stride + hk * DK, qk_stride, n, tid);
    if (role == 0) {
      load_tile<TIn, DK, LDK, CP>(q_s, qg + c0 * qk_stride + hk * DK, qk_stride, n, tid);
      load_tile<TIn, DV, LDV, CP>(sm.v, vg + c0 * v_stride + h * DV, v_stride, n, tid);
    }
    if (wave == 0) {
      float a = 0.f, bt = 0.f;
      if (lane < n) {
        const long idx = static_cast<long>(c0 + lane) * args.h_v + h;
        a = args.log_alpha[idx];
        bt = args.beta[idx];
      }
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const float u = __shfl_up(a, off, 64);
        if (lane >= off) a += u;
      }
      if (lane < CP) {
        sm.b[lane] = a;
        sm.beta[lane] = bt;
      }
    }
    __syncthreads();
    const float b_last = sm.b[CP - 1];
    log_decay += b_last;

    // ---- B: Gram / query-key tiles; Q S0 ------------------------------------
    {
      constexpr int NLT = MTC * (MTC + 1) / 2;  // lower tiles incl. diagonal
      const int nmat = (role == 0) ? 2 : 1;
      for (int t = wave; t < NLT * nmat; t += kWaves) {
        const int which = t / NLT;  // 0: K K^T, 1: Q K^T
        int lt = t % NLT, ti = 0;
        while (lt > ti) { lt -= ti + 1; ++ti; }
        const int tj = lt;
        const TIn* amat = (which == 0) ? sm.k : q_s;
        f32x4 acc = zero4();
#pragma unroll
        for (int kb = 0; kb < DK; kb += 32) {
          float fa[8], fb[8];
          frag_kcontig(amat, LDK, ti * 16 + ln, kb, g, fa);
          frag_kcontig(sm.k, LDK, tj * 16 + ln, kb, g, fb);
          mma_blk<IO::kQK>(acc, fa, fb);
        }
        const int ci = tj * 16 + ln;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int r = ti * 16 + 4 * g + i;
          if (which == 0) {
            sm.L[r * LDC + ci] = (ci < r) ? sm.beta[r] * acc[i] : 0.f;
          } else {
            sm.X[r * LDC + ci] = (ci <= r) ? acc[i] * __expf(sm.b[r] - sm.b[ci]) : 0.f;
          }
        }
      }
      // zero the strictly-upper tiles
      for (int idx = tid; idx < CP * CP; idx += kThreads) {
        const int r = idx / CP, c = idx % CP;
        if ((c / 16) > (r / 16)) {
          sm.L[r * LDC + c] = 0.f;
          sm.X[r * LDC + c] = 0.f;
        }
      }
    }
    f32x4 oq[MTC][NTS];
    if (role == 0) {
#pragma unroll
      for (int mt = 0; mt < MTC; ++mt)
#pragma unroll
        for (int nt = 0; nt < NTS; ++nt) {
          f32x4 acc = zero4();
#pragma unroll
          for (int kt = 0; kt < MTK / 2; ++kt) {
            float fa[8], fb[8];
            frag_kcontig(q_s, LDK, mt * 16 + ln, kt * 32, g, fa);
            frag_from_acc(st[2 * kt][nt], st[2 * kt + 1][nt], fb);
            mma_blk<IO::kS>(acc, fa, fb);
          }
          oq[mt][nt] = acc;
        }
    }
    __syncthreads();

    // ---- C: UT transform ------------------------------------------------------
    unit_lower_inverse<CP, LDC>(sm.L, sm.A, sm.T, tid);

    // ---- D: W (or W') into LDS; U for this wave's slab -----------------------
    {
      constexpr int NWT = MTC * MTK;
      for (int t = wave; t < NWT; t += kWaves) {
        const int ti = t / MTK, tk = t % MTK;
        f32x4 acc = zero4();
#pragma unroll
        for (int kb = 0; kb < CP; kb += 32) {
          float fa[8], fb[8];
          frag_kcontig(sm.A, LDC, ti * 16 + ln, kb, g, fa);
#pragma unroll
          for (int j = 0; j < 8; ++j) fa[j] *= sm.beta[kb + kap(g, j)];
          frag_kstrided(sm.k, LDK, tk * 16 + ln, kb, g, fb);
          if (role == 0)
            mma_blk<IO::kS>(acc, fa, fb);
          else
            mma_blk<IO::kWop>(acc, fa, fb);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int r = ti * 16 + 4 * g + i;
          const float scale = (role == 0) ? __expf(sm.b[r]) : 1.f;
          w_s[r * LDW + tk * 16 + ln] = scale * acc[i];
        }
      }
    }
    f32x4 vn[MTC][NTS];
    if (role == 0) {
#pragma unroll
      for (int mt = 0; mt < MTC; ++mt)
#pragma unroll
        for (int nt = 0; nt < NTS; ++nt) {
          f32x4 acc = zero4();
          const int r = mt * 16 + ln;
          const float br = sm.b[r];
#pragma unroll
          for (int kb = 0; kb < CP; kb += 32) {
            float fa[8], fb[8];
            frag_kcontig(sm.A, LDC, r, kb, g, fa);
#pragma unroll
            for (int j = 0; j < 8; ++j) {
              const int i = kb + kap(g, j);
              fa[j] = (i <= r) ? fa[j] * sm.beta[i] * __expf(br - sm.b[i]) : 0.f;
            }
            frag_kstrided(sm.v, LDV, col0 + nt * 16 + ln, kb, g, fb);
            mma_blk<IO::kS>(acc, fa, fb);
          }
          vn[mt][nt] = acc;
        }
    }
    __syncthreads();

    // ---- E: chain update ---------------------------------------------------------
    if (role == 0) {
      // Vn = U - W' S0
#pragma unroll
      for (int mt = 0; mt < MTC; ++mt)
#pragma unroll
        for (int nt = 0; nt < NTS; ++nt) {
          f32x4 acc = zero4();
#pragma unroll
          for (int kt = 0; kt < MTK / 2; ++kt) {
            float fa[8], fb[8];
            frag_kcontig(w_s, LDW, mt * 16 + ln, kt * 32, g, fa);
            frag_from_acc(st[2 * kt][nt], st[2 * kt + 1][nt], fb);
            mma_blk<IO::kS>(acc, fa, fb);
          }
          vn[mt][nt] -= acc;
        }
      // O = diag(gamma) Q S0 + X Vn
#pragma unroll
      for (int mt = 0; mt < MTC; ++mt)
#pragma unroll
        for (int nt = 0; nt < NTS; ++nt) {
          f32x4 acc = oq[mt][nt];
#pragma unroll
          for (int i = 0; i < 4; ++i) acc[i] *= __expf(sm.b[mt * 16 + 4 * g + i]);
#pragma unroll
          for (int kt = 0; kt < MTC / 2; ++kt) {
            float fa[8], fb[8];
            frag_kcontig(sm.X, LDC, mt * 16 + ln, kt * 32, g, fa);
            frag_from_acc(vn[2 * kt][nt], vn[2 * kt + 1][nt], fb);
            mma_blk<IO::kS>(acc, fa, fb);
          }
          oq[mt][nt] = acc;
        }
      if (args.o != nullptr) {
        TIn* og = static_cast<TIn*>(args.o);
#pragma unroll
        for (int mt = 0; mt < MTC; ++mt)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int r = mt * 16 + 4 * g + i;
            if (r < n) {
              long row;
              if (args.mode == 0)
                row = c0 + r;
              else
                row = static_cast<long>(seam_out_entry(args, seg)) * args.w + (c0 - lo) + r;
              TIn* orow = og + row * v_stride + h * DV + col0;
#pragma unroll
              for (int nt = 0; nt < NTS; ++nt) IO::store(orow + nt * 16 + ln, oq[mt][nt][i]);
            }
          }
      }
      // S <- gamma_last S0 + K^T diag(exp(b_last - b)) Vn
      const float g_last = __expf(b_last);
#pragma unroll
      for (int kt = 0; kt < MTC / 2; ++kt)
#pragma unroll
        for (int nt = 0; nt < NTS; ++nt)
#pragma unroll
          for (int half = 0; half < 2; ++half)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int r = kt * 32 + half * 16 + 4 * g + i;
              vn[2 * kt + half][nt][i] *= __expf(b_last - sm.b[r]);
            }
#pragma unroll
      for (int mt = 0; mt < MTK; ++mt)
#pragma unroll
        for (int nt = 0; nt < NTS; ++nt) {
          f32x4 acc = st[mt][nt] * g_last;
#pragma unroll
          for (int kt = 0; kt < MTC / 2; ++kt) {
            float fa[8], fb[8];
            frag_kstrided(sm.k, LDK, mt * 16 + ln, kt * 32, g, fa);
            frag_from_acc(vn[2 * kt][nt], vn[2 * kt + 1][nt], fb);
            mma_blk<IO::kS>(acc, fa, fb);
          }
          st[mt][nt] = acc;
        }
    } else {
      // X = W P0 ;  P <- P0 - K^T X
      f32x4 x[MTC][NTP];
#pragma unroll
      for (int mt = 0; mt < MTC; ++mt)
#pragma unroll
        for (int nt = 0; nt < NTP; ++nt) {
          f32x4 acc = zero4();
#pragma unroll
          for (int kt = 0; kt < MTK / 2; ++kt) {
            float fa[8], fb[8];
            frag_kcontig(w_s, LDW, mt * 16 + ln, kt * 32, g, fa);
            frag_from_acc(st[2 * kt][nt], st[2 * kt + 1][nt], fb);
            mma_blk<IO::kP>(acc, fa, fb);
          }
          x[mt][nt] = -acc;
        }
#pragma unroll
      for (int mt = 0; mt < MTK; ++mt)
#pragma unroll
        for (int nt = 0; nt < NTP; ++nt) {
          f32x4 acc = st[mt][nt];
#pragma unroll
          for (int kt = 0; kt < MTC / 2; ++kt) {
            float fa[8], fb[8];
            frag_kstrided(sm.k, LDK, mt * 16 + ln, kt * 32, g, fa);
            frag_from_acc(x[2 * kt][nt], x[2 * kt + 1][nt], fb);
            mma_blk<IO::kKX>(acc, fa, fb);
          }
          st[mt][nt] = acc;
        }
    }
    __syncthreads();
  }

  // ---- write the chain's result ------------------------------------------------
  if (role == 0) {
    if (args.S_out != nullptr) {
      float* so = args.S_out + sh * DK * DV;
#pragma unroll
      for (int mt = 0; mt < MTK; ++mt)
#pragma unroll
        for (int nt = 0; nt < NTS; ++nt)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            so[(mt * 16 + 4 * g + i) * DV + col0 + nt * 16 + ln] = st[mt][nt][i];
    }
    if (args.log_decay != nullptr && tid == 0) args.log_decay[sh] = log_decay;
  } else {
    float* po = args.P_hat + sh * DK * DK;
#pragma unroll
    for (int mt = 0; mt < MTK; ++mt)
#pragma unroll
      for (int nt = 0; nt < NTP; ++nt)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          po[(mt * 16 + 4 * g + i) * DK + col0 + nt * 16 + ln] = st[mt][nt][i];
  }
}

// Longest-first order of the segments (Eq. (9) LPT list order; ties by index).
__global__ void lpt_order_kernel(const int32_t* cu, int n, int32_t* order) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int li = cu[i + 1] - cu[i];
  int rank = 0;
  for (int j = 0; j < n; ++j) {
    const int lj = cu[j + 1] - cu[j];
    rank += (lj > li) || (lj == li && j < i);
  }
  order[rank] = i;
}

template <typename TIn, int DK, int DV, int C>
hipError_t launch_scan_t(const ScanArgs& a, int n_items, hipStream_t stream) {
  hipLaunchKernelGGL((scan_kernel<TIn, DK, DV, C>), dim3(n_items), dim3(kThreads), 0,
                     stream, a);
  return hipGetLastError();
}

template <typename TIn, int DK, int DV>
hipError_t launch_scan_c(const ScanArgs& a, int chunk, int n_items, hipStream_t s) {
  switch (chunk) {
    case 16: return launch_scan_t<TIn, DK, DV, 16>(a, n_items, s);
    case 32: return launch_scan_t<TIn, DK, DV, 32>(a, n_items, s);
    default: return launch_scan_t<TIn, DK, DV, 64>(a, n_items, s);
  }
}

template <typename TIn>
hipError_t launch_scan_d(const ScanArgs& a, int d_k, int d_v, int chunk, int n_items,
                         hipStream_t s) {
  if (d_k == 64 && d_v == 64) return launch_scan_c<TIn, 64, 64>(a, chunk, n_items, s);
  if (d_k == 64 && d_v == 128) return launch_scan_c<TIn, 64, 128>(a, chunk, n_items, s);
  if (d_k == 128 && d_v == 64) return launch_scan_c<TIn, 128, 64>(a, chunk, n_items, s);
  return launch_scan_c<TIn, 128, 128>(a, chunk, n_items, s);
}

}  // namespace

hipError_t launch_lpt_order(const int32_t* cu, int n, int32_t* order, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(lpt_order_kernel, dim3((n + 255) / 256), dim3(256), 0, s, cu, n, order);
  return hipGetLastError();
}

hipError_t launch_scan(const ScanArgs& a, int bf16, int d_k, int d_v, int chunk,
                       int n_chains, hipStream_t s) {
  if (n_chains <= 0) return hipSuccess;
  const bool fast = bf16 && chunk == 64;
  const int64_t per_head =
      fast ? scan_bf16_items_per_head(d_k, d_v, a.n_roles == 2) : a.n_roles;
  if (fast) {
    // Seams of at most one chunk run back to back through one workgroup's
    // pipeline, up to 16 entries of one head per workgroup: as many as make
    // the launch a single round of workgroups over the 256 compute units, so
    // that a workgroup of g entries takes g + 2 iterations (the pipeline's
    // fill) once rather than two rounds of g / 2 + 2.
    ScanArgs b = a;
    b.n_entries = n_chains;
    b.group_e = 1;
    if (a.mode == 1 && a.w <= 64) {
      const int64_t pairs = static_cast<int64_t>(n_chains) * a.h_v;
      const int64_t ge = (pairs + 255) / 256;
      b.group_e = static_cast<int>((ge < 1) ? 1 : ((ge > 16) ? 16 : ge));
    }
    const int64_t groups = (n_chains + b.group_e - 1) / b.group_e;
    const int64_t n_items = groups * a.h_v * per_head;
    if (n_items > 0x7fffffff) return hipErrorInvalidValue;
    return launch_scan_bf16(b, d_k, d_v, static_cast<int>(n_items), s);
  }
  const int64_t n_items = static_cast<int64_t>(n_chains) * a.h_v * per_head;
  if (n_items > 0x7fffffff) return hipErrorInvalidValue;
  if (bf16)
    return launch_scan_d<uint16_t>(a, d_k, d_v, chunk, static_cast<int>(n_items), s);
  return launch_scan_d<float>(a, d_k, d_v, chunk, static_cast<int>(n_items), s);
}

}  // namespace hypic
