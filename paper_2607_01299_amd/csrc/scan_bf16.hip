// Chunked gated-delta-rule scan, bf16 inputs, chunk 64: the production path
// of the segment build and the seam rescan on gfx950.
//
// Same mathematics as scan.hip (per chunk: Gram matrix, unit-lower-triangular
// inverse A1 = (I + L)^{-1}, WY factor W, then the state / operator update),
// organised for the CDNA4 matrix cores:
//
// * Work split.  One workgroup of 8 waves runs one (segment, v-head, column
//   block) chain: waves 0-3 own 16 columns each of a 64-column block of the
//   state S (and emit those output columns), waves 4-7 own the same 64 columns
//   of the operator P_hat.  The chunk's Gram matrix, inverse and W are computed
//   once per workgroup and shared by both halves; each SIMD runs one state
//   wave and one operator wave, so one's matrix-core work hides the other's
//   latency.
// * Operand layout.  Every matrix-core operand is staged in LDS "fragment
//   major": a 16 x 32 (rows x contraction) tile is 64 lanes x 8 bf16 stored in
//   lane order, so a lane reads its fragment with one 16-byte load and a wave
//   reads 1 KiB of consecutive bytes.  Products whose result feeds another
//   product are computed transposed where that makes the accumulator tile
//   already be the next operand's fragment (W^T = K^T (A1 diag beta)^T,
//   K Q^T, O^T), and states are used as operands straight from registers.
// * Gates are exponentiated once per chunk (b = prefix sum of log alpha,
//   gamma = exp(b), exp(b_last - b)); every decay factor is exp of a
//   non-positive number.
// * The inverse: the four 16 x 16 diagonal blocks by column-parallel
//   substitution in one wave (one 16-lane row per block, coefficients shared
//   by DPP row broadcasts), overlapping the other waves' Gram and K Q^T tiles;
//   then the off-diagonal blocks
//   A_ij = -sum_k N_ik A_kj with N_ik = A_ii L_ik on float32 matrix cores, one
//   block diagonal at a time.
// * The next chunk's q, k, v, beta, log alpha are loaded into registers while
//   the current chunk computes.
// * Precision: W is formed in two bf16 passes (A1 diag(beta) split hi + lo, K
//   exact) and kept as hi + lo; the state path uses single bf16 passes (its
//   decay keeps rounding from accumulating); the operator path, which has no
//   decay, uses W hi + lo and splits P0 (three passes for W P0, two for K^T X).

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mfma.hpp"
#include "scan.hpp"

namespace hypic {

namespace {

constexpr int kThreads = 512;
constexpr int kGateWave = 1;  // loads and exponentiates the gates of each chunk
constexpr int C = 64;        // tokens per chunk
constexpr int NCOL = 64;     // state / operator columns per workgroup
constexpr int KTC = C / 32;  // 32-wide contraction blocks over the chunk's tokens
constexpr int LDC = C + 4;   // row stride (floats) of the float32 chunk x chunk matrices
constexpr int LDD = 20;      // row stride (floats) of the staged diagonal blocks of A1

typedef unsigned short u16;
typedef u16 u16x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));

// ---- fragment-major layout -------------------------------------------------
// logical R x K matrix (contraction over K), KT = K / 32 blocks per row tile.
__device__ __forceinline__ int frag_slot(int rt, int kt, int KT, int lane) {
  return ((rt * KT + kt) * 64 + lane) * 8;
}
__device__ __forceinline__ bf16x8 ld_frag(const u16* base, int slot) {
  return *reinterpret_cast<const bf16x8*>(base + slot);
}
__device__ __forceinline__ void st_frag(u16* base, int slot, bf16x8 v) {
  *reinterpret_cast<bf16x8*>(base + slot) = v;
}

__device__ __forceinline__ f32x4 mma(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 pack(const f32x4& lo, const f32x4& hi) {
  bf16x8 r;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    r[i] = static_cast<__bf16>(lo[i]);
    r[4 + i] = static_cast<__bf16>(hi[i]);
  }
  return r;
}
__device__ __forceinline__ void pack_split(const f32x4& lo, const f32x4& hi, bf16x8& h,
                                           bf16x8& l) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    h[i] = static_cast<__bf16>(lo[i]);
    h[4 + i] = static_cast<__bf16>(hi[i]);
    l[i] = static_cast<__bf16>(lo[i] - static_cast<float>(h[i]));
    l[4 + i] = static_cast<__bf16>(hi[i] - static_cast<float>(h[4 + i]));
  }
}

// float32 16x16x16 product on matrix cores: a[s] = A[m][4g+s], b[s] = B[4g+s][n]
__device__ __forceinline__ f32x4 mma16_f32(const float4& a, const float4& b, f32x4 c) {
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.x, b.x, c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.y, b.y, c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.z, b.z, c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.w, b.w, c, 0, 0, 0);
  return c;
}

__device__ __forceinline__ u16 bf16_of(float x) {
  __bf16 h = static_cast<__bf16>(x);
  return *reinterpret_cast<u16*>(&h);
}

// Step I of the column-parallel unit-lower substitution on 16-lane rows: lane
// 16b + c holds column c of the solution (x) and column c of -L (lcol); the
// coefficient -L[r][I] comes from lane I of the same row (DPP row_newbcast:I).
template <int I>
__device__ __forceinline__ void unit_lower_solve_step(float (&x)[16], const float (&lcol)[16]) {
  if constexpr (I < 15) {
    float nl[16];
#pragma unroll
    for (int r = I + 1; r < 16; ++r)
      nl[r] = __builtin_bit_cast(
          float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, lcol[r]), 0x150 + I, 0xF, 0xF,
                                          false));
#pragma unroll
    for (int r = I + 1; r < 16; ++r) x[r] = __builtin_fmaf(nl[r], x[I], x[r]);
    unit_lower_solve_step<I + 1>(x, lcol);
  }
}

// Row order of the d_k dimension inside the kernel.  q and k are loaded 16
// contiguous bytes per lane (lane (g, m) of a 32-column block holds columns
// 8g .. 8g+7), which makes a matrix-core slot (g, j) carry column 8g + j.  The
// transposed K tiles, and with them the state and operator rows, are laid out
// so that packing row tiles (2kb, 2kb+1) from accumulators gives exactly that
// slot order: row m of d_k tile dt is d = d_perm(dt, m).  Rows are mapped back
// to their true index only where a state or operator enters or leaves HBM.
__device__ __forceinline__ int d_perm(int dt, int m) {
  return 32 * (dt >> 1) + 8 * (m >> 2) + 4 * (dt & 1) + (m & 3);
}

// lower-triangle tile t in 0..9 -> (row tile, column tile) with column <= row
__device__ __forceinline__ int tri_row(int t) { return (t < 1) ? 0 : (t < 3) ? 1 : (t < 6) ? 2 : 3; }
__device__ __forceinline__ int tri_col(int t) { return t - tri_row(t) * (tri_row(t) + 1) / 2; }

// owner wave and register slot of K Q^T tile t (query tile tri_row(t), key tile
// tri_col(t)): wave w holds the tiles of key tile w in slot (query - key); the
// tile (query 3, key 0) goes to wave 3, slot 1
__device__ __forceinline__ int kq_owner(int t) { return (t == 6) ? 3 : tri_col(t); }
__device__ __forceinline__ int kq_slot(int t) { return (t == 6) ? 1 : tri_row(t) - tri_col(t); }

// ---- LDS plan (bytes); regions are reused across the phases of a chunk ------
// Phase 0 of chunk c + 1 runs in the same barrier interval as the chain update
// of chunk c, so everything that update reads and phase 0 writes is kept
// apart: K over tokens and the gates are double-buffered, W hi and the
// (Q K^T . Gamma) fragments have regions of their own.
template <int DK>
struct Lds {
  static constexpr int FK = C * DK * 2;     // bytes of a 64 x DK bf16 fragment matrix
  static constexpr int F32M = C * LDC * 4;  // padded 64 x 64 float32 matrix
  static constexpr int RA = (FK > F32M) ? FK : F32M;
  static constexpr int GATES = 4 * C * 4;
  static constexpr int O_KD = 0;            // K over d -> A1 (f32)
  static constexpr int O_Q = O_KD + RA;     // Q over d -> A1^T -> (A1 . Gamma) beta
  static constexpr int O_KT = O_Q + RA;     // K over tokens, two buffers
  static constexpr int O_L = O_KT + 2 * FK;  // L^T (f32) + N blocks -> A1 beta hi / lo
  static constexpr int O_WS = O_L + F32M;   // gamma W (state path)
  static constexpr int O_WL = O_WS + FK;    // staged A1 diagonal blocks -> W lo (operator path)
  static constexpr int O_WH = O_WL + FK;    // W hi (operator path)
  static constexpr int O_QK = O_WH + FK;    // (Q K^T . Gamma)
  static constexpr int O_G = O_QK + C * C * 2;  // gates, two buffers
  static constexpr int TOTAL = O_G + 2 * GATES;
  static_assert(2 * C * C * 2 <= F32M, "A1 beta hi + lo fit the L region");
  static_assert(C * C * 2 <= RA, "(A1 . Gamma) beta fits the Q region");
  static_assert(C * LDD * 4 <= FK, "staged diagonal blocks fit the W lo region");
  static_assert(TOTAL <= 160 * 1024, "LDS budget");
};

template <int DK, int DV>
__global__ __launch_bounds__(kThreads, 1) void scan_bf16_kernel(ScanArgs args) {
  using LP = Lds<DK>;
  constexpr int KTD = DK / 32;  // contraction blocks over d_k
  constexpr int DT = DK / 16;   // d_k row tiles of the state
  constexpr int NS = DV / NCOL;
  constexpr int NP = DK / NCOL;

  extern __shared__ __align__(16) unsigned char smem[];
  u16* fKd = reinterpret_cast<u16*>(smem + LP::O_KD);
  float* A1 = reinterpret_cast<float*>(smem + LP::O_KD);
  u16* fQ = reinterpret_cast<u16*>(smem + LP::O_Q);
  float* A1t = reinterpret_cast<float*>(smem + LP::O_Q);
  u16* fAgb = reinterpret_cast<u16*>(smem + LP::O_Q);
  float* Lt = reinterpret_cast<float*>(smem + LP::O_L);
  u16* fAbh = reinterpret_cast<u16*>(smem + LP::O_L);
  u16* fAbl = fAbh + C * C;
  u16* fWs = reinterpret_cast<u16*>(smem + LP::O_WS);
  u16* fWl = reinterpret_cast<u16*>(smem + LP::O_WL);
  u16* fWh = reinterpret_cast<u16*>(smem + LP::O_WH);
  u16* fQK = reinterpret_cast<u16*>(smem + LP::O_QK);
  float* Dg = reinterpret_cast<float*>(smem + LP::O_WL);  // diagonal blocks of A1 (phase 1-2)
  // buffer set par of the double-buffered regions
  auto kt_buf = [&](int par) { return reinterpret_cast<u16*>(smem + LP::O_KT + par * LP::FK); };
  auto gate_buf = [&](int par) {
    return reinterpret_cast<float*>(smem + LP::O_G + par * LP::GATES);
  };

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int lane = tid & 63;
  const int g = lane >> 4, ln = lane & 15;
  const int lane0 = lane, g0 = g, ln0 = ln;  // for the prefetch (outside the chunk loop)
  // With the operator requested, waves 0-3 carry 64 state columns and waves
  // 4-7 the same 64 operator columns.  Without it, all 8 waves carry state
  // columns (128 per workgroup).
  const bool with_op = args.n_roles == 2;
  const bool sw = !with_op || wave < 4;  // state wave (else operator wave)
  const int wq = with_op ? (wave & 3) : wave;  // column tile within the block
  const int span = with_op ? NCOL : 2 * NCOL;  // state columns per workgroup

  // ---- work item ----------------------------------------------------------
  const int n_cb = with_op ? ((NP > NS) ? NP : NS) : (DV + span - 1) / span;
  // Workgroups are dealt to the 8 XCDs round-robin; the n_cb column blocks of a
  // chain are numbered so that they land on one XCD back to back and share its
  // L2 for q and k.  Chains past the last full group of 8 keep linear order.
  const int n_chains = static_cast<int>(gridDim.x) / n_cb;
  const int full = (n_chains / 8) * 8 * n_cb;
  int chain, cb;
  if (static_cast<int>(blockIdx.x) < full) {
    const int slot = blockIdx.x / 8;
    chain = (slot / n_cb) * 8 + blockIdx.x % 8;
    cb = slot % n_cb;
  } else {
    const int b = blockIdx.x - full;
    chain = full / n_cb + b / n_cb;
    cb = b % n_cb;
  }
  const int rank = chain / args.h_v;
  const int h = chain % args.h_v;
  const int col0 = cb * span + wq * 16;  // this wave's 16 columns (of S or P_hat)
  const bool has_state = cb * span < DV;           // the block holds state columns
  const bool has_op = with_op && (cb < NP);
  const bool wave_cols = sw ? (col0 < DV) : has_op;  // does this wave own columns?
  int seg, lo, hi;
  if (args.mode == 0) {
    seg = args.order[rank];
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

  const int hk = h / args.group;
  const u16* kg = static_cast<const u16*>(args.k);
  const u16* qg = static_cast<const u16*>(args.q);
  const u16* vg = static_cast<const u16*>(args.v);
  const long qk_stride = static_cast<long>(args.h_qk) * DK;
  const long v_stride = static_cast<long>(args.h_v) * DV;
  const long sh = static_cast<long>(seg) * args.h_v + h;

  // ---- chain state: 16 columns per wave, all d_k rows ------------------------
  f32x4 st[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) st[dt] = zero4();
  if (sw) {
    if (args.mode == 1 && wave_cols) {
      const float* s_in = args.S_in + sh * DK * DV;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int i = 0; i < 4; ++i) st[dt][i] = s_in[d_perm(dt, 4 * g + i) * DV + col0 + ln];
    }
  } else {
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int i = 0; i < 4; ++i) st[dt][i] = (d_perm(dt, 4 * g + i) == col0 + ln) ? 1.f : 0.f;
  }
  float log_decay = 0.f;

  // ---- prefetch of one chunk's tokens into registers -------------------------
  // Tokens are loaded as matrix-core A-operand fragments straight from HBM:
  // lane (g, m) of fragment (token tile tt, column block kb) holds the 8
  // columns kb*32 + 8g .. kb*32 + 8g + 7 of token tt*16 + m (one 16-byte load).
  // A "pair job" loads the two token tiles 2*kt, 2*kt + 1 of one column block.
  //   K: pair job (kb, kt) on wave kb + KTD*kt      (waves [0, 2*KTD))
  //   Q: pair job (kb, kt) on wave 8 - 2*KTD + ...  (waves [8 - 2*KTD, 8))
  //   V: every state wave loads its own 16 columns, lane (g, m) of token tile tt
  //      holding columns col0 + 4g .. col0 + 4g + 3 of token tt*16 + m
  const bool k_job = wave < 2 * KTD;
  const int kjb = wave % KTD, kjt = wave / KTD;
  const bool q_job = wave >= 8 - 2 * KTD;
  const int qjb = (wave - (8 - 2 * KTD)) % KTD, qjt = (wave - (8 - 2 * KTD)) / KTD;
  const bool v_job = sw && wave_cols;
  // Raw loads only: every use of the loaded words (the tail mask included)
  // waits until phase 0 of the next chunk, so the loads stay in flight while
  // phases 4 and 5 compute.  Element [2t + h] holds half h of token tile 2kt + t.
  uint4 pk[2], pq[2];
  uint2 pv[4];
  bf16x8 vB[KTC];  // state waves: this chunk's V columns as B fragments (phase 0 -> 4)
  float pa = 0.f, pbeta = 0.f;
  auto load_pair = [&](uint4 (&dst)[2], const u16* base, long rs, int col, int kt, int c0,
                       int n) __attribute__((always_inline)) {
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const int tok = (2 * kt + t) * 16 + ln0;
      const int tc = (tok < n) ? tok : n - 1;  // clamped (valid) token; zeroed on use
      dst[t] = *reinterpret_cast<const uint4*>(base + (c0 + tc) * rs + col + 8 * g0);
    }
  };
  auto prefetch = [&](int c0) __attribute__((always_inline)) {
    const int n = (hi - c0 < C) ? (hi - c0) : C;  // n >= 1
    if (k_job) load_pair(pk, kg + hk * DK, qk_stride, kjb * 32, kjt, c0, n);
    if (q_job) load_pair(pq, qg + hk * DK, qk_stride, qjb * 32, qjt, c0, n);
    if (v_job) {
#pragma unroll
      for (int tt = 0; tt < 4; ++tt) {
        const int tok = tt * 16 + ln0;
        const int tc = (tok < n) ? tok : n - 1;
        pv[tt] = *reinterpret_cast<const uint2*>(vg + (c0 + tc) * v_stride + h * DV + col0 +
                                                 4 * g0);
      }
    }
    if (wave == kGateWave) {
      const int tc = (lane0 < n) ? lane0 : n - 1;
      const long idx = static_cast<long>(c0 + tc) * args.h_v + h;
      pa = args.log_alpha[idx];
      pbeta = args.beta[idx];
    }
  };

  // ---- phase 0 of the chunk at c0n into buffer set par: fragments -> LDS
  //      (lane-contiguous); transposed copies of K and V by exact identity
  //      products on the matrix cores; gates -------------------------------------
  auto phase0 = [&](int c0n, int par, int lane, int g, int ln) __attribute__((always_inline)) {
    const int n = (hi - c0n < C) ? (hi - c0n) : C;
    u16* fKt = kt_buf(par);
    float* gb = gate_buf(par);
    float* gbeta = gb + C;
    float* ggam = gb + 2 * C;
    float* gdec = gb + 3 * C;
  {
    // selector B operands: slot (g', j') of lane (g', n) holds column
    // 8g' + j' of the loaded 32-column block, so eye[half] = 1 exactly where
    // 8g' + j' = d_perm(half, n) and (X eye[half])[m][n] = X[m][d_perm(half, n)]
    bf16x8 eye[2];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      eye[0][j] = static_cast<__bf16>((g == (ln >> 2) && j == (ln & 3)) ? 1.f : 0.f);
      eye[1][j] = static_cast<__bf16>((g == (ln >> 2) && j == 4 + (ln & 3)) ? 1.f : 0.f);
    }
    // fragment t of a prefetched pair, with tokens past the chunk's end zeroed
    auto take = [&](const uint4 (&src)[2], int kt, int t) __attribute__((always_inline)) {
      const uint32_t keep = ((2 * kt + t) * 16 + ln < n) ? 0xffffffffu : 0u;
      const uint4 w = src[t];
      return __builtin_bit_cast(bf16x8,
                                make_uint4(w.x & keep, w.y & keep, w.z & keep, w.w & keep));
    };
    auto transpose_pair = [&](bf16x8 f0, bf16x8 f1, u16* dst, int row_tile0, int kt)
        __attribute__((always_inline)) {
      // f0, f1: A fragments of token tiles 2kt, 2kt+1 over a 32-column block
      // whose two 16-column halves become row tiles row_tile0 and row_tile0 + 1
      // of the token-contraction fragments
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        const f32x4 c_lo = mma(f0, eye[half], zero4());
        const f32x4 c_hi = mma(f1, eye[half], zero4());
        st_frag(dst, frag_slot(row_tile0 + half, kt, KTC, lane), pack(c_lo, c_hi));
      }
    };
    if (k_job) {
      const bf16x8 f0 = take(pk, kjt, 0), f1 = take(pk, kjt, 1);
      st_frag(fKd, frag_slot(2 * kjt, kjb, KTD, lane), f0);
      st_frag(fKd, frag_slot(2 * kjt + 1, kjb, KTD, lane), f1);
      transpose_pair(f0, f1, fKt, 2 * kjb, kjt);
    }
    if (q_job) {
      st_frag(fQ, frag_slot(2 * qjt, qjb, KTD, lane), take(pq, qjt, 0));
      st_frag(fQ, frag_slot(2 * qjt + 1, qjb, KTD, lane), take(pq, qjt, 1));
    }
    if (v_job) {
      // this wave's V columns as token-contraction B fragments, by exact
      // 16x16x16 identity products: (V_tt I)[m][n] lands in lane (g, n) as
      // rows 4g .. 4g+3, i.e. tokens along the contraction
      s16x4 eye16;
#pragma unroll
      for (int j = 0; j < 4; ++j) eye16[j] = (4 * g + j == ln) ? short(0x3F80) : short(0);
      f32x4 vt[4];
#pragma unroll
      for (int tt = 0; tt < 4; ++tt) {
        const uint32_t keep = (tt * 16 + ln < n) ? 0xffffffffu : 0u;
        const uint2 w2 = make_uint2(pv[tt].x & keep, pv[tt].y & keep);
        vt[tt] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(s16x4, w2),
                                                           eye16, zero4(), 0, 0, 0);
      }
      vB[0] = pack(vt[0], vt[1]);
      vB[1] = pack(vt[2], vt[3]);
    }
  }
  if (wave == kGateWave) {
    float b = (lane < n) ? pa : 0.f;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const float u = __shfl_up(b, off, 64);
      if (lane >= off) b += u;
    }
    const float b_last = __shfl(b, 63, 64);
    gb[lane] = b;
    gbeta[lane] = (lane < n) ? pbeta : 0.f;
    ggam[lane] = __expf(b);
    gdec[lane] = __expf(b_last - b);
  }
  };

  if (lo < hi) {
    prefetch(lo);
    phase0(lo, 0, lane0, g0, ln0);
    lds_barrier();
  }

  for (int c0 = lo; c0 < hi; c0 += C) {
    const int n = (hi - c0 < C) ? (hi - c0) : C;
    // an opaque copy of the thread index keeps the compiler from hoisting every
    // loop-invariant fragment address out of the chunk loop (each would pin a
    // register for the whole loop); they are cheap to recompute per chunk
    int tid = threadIdx.x;
    asm volatile("" : "+v"(tid));
    const int lane = tid & 63;
    const int g = lane >> 4, ln = lane & 15;
    const int par = ((c0 - lo) / C) & 1;  // buffer set of this chunk
    const u16* fKt = kt_buf(par);
    const float* gb = gate_buf(par);
    const float* gbeta = gb + C;
    const float* ggam = gb + 2 * C;
    const float* gdec = gb + 3 * C;

    const float b_last = gb[C - 1];
    log_decay += b_last;

    // ---- phase 1: Gram tiles; diagonal blocks of A1 = (I + L)^{-1}; K Q^T; (Q S0)^T --
    // Wave 4 forms the four diagonal Gram tiles, gathers column c of G_bb into
    // lane 16b + c by cross-row lane swaps (no LDS round trip) and inverts all
    // four blocks at once by unit-lower substitution, one lane per column: the
    // coefficient L[r][i] reaches every lane of row b by a DPP row broadcast
    // from lane i.
    f32x4 kq[3];
    f32x4 oq[4];
    float xd[16];  // wave 4, lane 16b + c: column c of the inverse diagonal block b
    if (wave == 4) {
      // the inverse is this phase's longest path: its instructions win issue
      // arbitration until it is done
      __builtin_amdgcn_s_setprio(2);
      f32x4 gd[4];  // diagonal Gram tiles; lane (g, n) of tile b holds G_b[4g + i][n]
#pragma unroll
      for (int bd = 0; bd < 4; ++bd) {
        gd[bd] = zero4();
#pragma unroll
        for (int kb = 0; kb < KTD; ++kb) {
          const bf16x8 f = ld_frag(fKd, frag_slot(bd, kb, KTD, lane));
          gd[bd] = mma(f, f, gd[bd]);
        }
      }
      // exchange (tile b, lane row g) <-> (tile g, lane row b) with two rounds of
      // row swaps: afterwards lane 16b + c of tile g holds G_b[4g + i][c], so
      // lane 16b + c has all of column c of G_b
#pragma unroll
      for (int i = 0; i < 4; ++i) {
#pragma unroll
        for (int b2 = 0; b2 < 2; ++b2) {  // upper half of tile b2 <-> lower half of b2 + 2
          const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(gd[b2][i]),
                                                          __float_as_uint(gd[b2 + 2][i]), false,
                                                          false);
          // the two results are copied out one by one before any bit cast
          const unsigned r0 = r[0], r1 = r[1];
          gd[b2][i] = __uint_as_float(r0);
          gd[b2 + 2][i] = __uint_as_float(r1);
        }
#pragma unroll
        for (int b2 = 0; b2 < 4; b2 += 2) {  // odd rows of tile b2 <-> even rows of b2 + 1
          const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(gd[b2][i]),
                                                          __float_as_uint(gd[b2 + 1][i]), false,
                                                          false);
          const unsigned r0 = r[0], r1 = r[1];
          gd[b2][i] = __uint_as_float(r0);
          gd[b2 + 1][i] = __uint_as_float(r1);
        }
      }
      const int ob = (lane >> 4) * 16;
      float lcol[16];  // -L[r][ln] = -beta_r G[r][ln] of block lane / 16 (used for r > ln)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const float4 bb = *reinterpret_cast<const float4*>(gbeta + ob + 4 * q4);
        lcol[4 * q4] = -bb.x * gd[q4][0];
        lcol[4 * q4 + 1] = -bb.y * gd[q4][1];
        lcol[4 * q4 + 2] = -bb.z * gd[q4][2];
        lcol[4 * q4 + 3] = -bb.w * gd[q4][3];
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) xd[r] = (r == ln) ? 1.f : 0.f;
      unit_lower_solve_step<0>(xd, lcol);
#pragma unroll
      for (int r = 0; r < 16; ++r) Dg[(ob + r) * LDD + ln] = xd[r];
      __builtin_amdgcn_s_setprio(0);
    }
    // off-diagonal Gram tiles (1,0) (2,0) (2,1) (3,0) (3,1) (3,2), all on wave 5,
    // which loads each K fragment once
    if (wave == 5) {
      f32x4 go[6];
#pragma unroll
      for (int j = 0; j < 6; ++j) go[j] = zero4();
#pragma unroll
      for (int kb = 0; kb < KTD; ++kb) {
        bf16x8 kf[4];
#pragma unroll
        for (int t4 = 0; t4 < 4; ++t4) kf[t4] = ld_frag(fKd, frag_slot(t4, kb, KTD, lane));
#pragma unroll
        for (int j = 0; j < 6; ++j) {
          const int ti = (j < 1) ? 1 : (j < 3) ? 2 : 3;
          const int tj = (j < 1) ? 0 : (j < 3) ? j - 1 : j - 3;
          go[j] = mma(kf[ti], kf[tj], go[j]);
        }
      }
#pragma unroll
      for (int j = 0; j < 6; ++j) {
        const int ti = (j < 1) ? 1 : (j < 3) ? 2 : 3;
        const int tj = (j < 1) ? 0 : (j < 3) ? j - 1 : j - 3;
        // L^T[c][r] = beta_r G[r][c]  (c < r throughout an off-diagonal tile)
        const int c = tj * 16 + ln;
        const float4 bb = *reinterpret_cast<const float4*>(gbeta + ti * 16 + 4 * g);
        *reinterpret_cast<float4*>(Lt + c * LDC + ti * 16 + 4 * g) =
            make_float4(bb.x * go[j][0], bb.y * go[j][1], bb.z * go[j][2], bb.w * go[j][3]);
      }
    }
    // (Q S0)^T = S0^T Q^T on every state wave (lane (g, n) holds four consecutive
    // state columns of query token n).  Waves 0-3 also form the K Q^T tiles from
    // the same Q fragments: wave w the tiles of key tile w, wave 3 also (0, 3).
    {
      const bool do_oq = sw && wave_cols;
      bf16x8 s0h[KTD];
#pragma unroll
      for (int kb = 0; kb < KTD; ++kb) s0h[kb] = pack(st[2 * kb], st[2 * kb + 1]);
#pragma unroll
      for (int rt = 0; rt < 4; ++rt) oq[rt] = zero4();
#pragma unroll
      for (int sl = 0; sl < 3; ++sl) kq[sl] = zero4();
#pragma unroll
      for (int w = 0; w < 5; ++w) {
        // w < 4: wave w; w == 4: any other state wave
        if ((w < 4) ? (w != wave) : (wave < 4 || !do_oq)) continue;
#pragma unroll
        for (int kb = 0; kb < KTD; ++kb) {
          bf16x8 qf[4];
#pragma unroll
          for (int rt = 0; rt < 4; ++rt) qf[rt] = ld_frag(fQ, frag_slot(rt, kb, KTD, lane));
          if (do_oq) {
#pragma unroll
            for (int rt = 0; rt < 4; ++rt) oq[rt] = mma(s0h[kb], qf[rt], oq[rt]);
          }
          if (w < 4) {
            const bf16x8 ka = ld_frag(fKd, frag_slot(w, kb, KTD, lane));
#pragma unroll
            for (int sl = 0; sl < 3; ++sl)
              if (w + sl < 4) kq[sl] = mma(ka, qf[w + sl], kq[sl]);
            if (w == 3) kq[1] = mma(ld_frag(fKd, frag_slot(0, kb, KTD, lane)), qf[3], kq[1]);
          }
        }
      }
    }
    // (Q K^T . Gamma) as A-operand fragments over key tokens for query rows
#pragma unroll
    for (int t = 0; t < 10; ++t) {
      if (kq_owner(t) != wave) continue;
      const int tr = tri_row(t), ti = tri_col(t);
      const int r = tr * 16 + ln;
      const float br = gb[r];
      const f32x4 a = kq[kq_slot(t)];
      u16x4 val;
#pragma unroll
      for (int i4 = 0; i4 < 4; ++i4) {
        const int i = ti * 16 + 4 * g + i4;
        val[i4] = bf16_of((i <= r) ? a[i4] * __expf(br - gb[i]) : 0.f);
      }
      *reinterpret_cast<u16x4*>(fQK + frag_slot(tr, ti >> 1, KTC, lane) + (ti & 1) * 4) = val;
    }
    // zero halves (key tile > query tile): (1,0) (2,0) (3,0) (2,1) (3,1) (3,2)
#pragma unroll
    for (int t = 0; t < 6; ++t) {
      if (((t < 4) ? t : t + 1) != wave) continue;  // waves 0-3, 5, 6
      const int ti = (t < 3) ? t + 1 : ((t == 5) ? 3 : t - 1);
      const int tr = (t < 3) ? 0 : ((t == 5) ? 2 : 1);
      *reinterpret_cast<uint2*>(fQK + frag_slot(tr, ti >> 1, KTC, lane) + (ti & 1) * 4) =
          make_uint2(0u, 0u);
    }
    // The next chunk's tokens load while this chunk computes.  Issuing the loads
    // keeps the CU's load path busy for ~1.5k cycles, so they are issued where
    // the waves would otherwise wait: waves 0-2 here, waves 3-7 (idle while
    // the off-diagonal blocks of A1 are merged) once the merges begin.
    if (wave < 3 && c0 + C < hi) prefetch(c0 + C);
    lds_barrier();

    // ---- phase 2: the rest of A1 -------------------------------------------------------
    // (a) the diagonal blocks move from their staging copy into A1 and A1^T
    if (wave == 4) {
      const int o = (lane >> 4) * 16;
#pragma unroll
      for (int r = 0; r < 16; ++r) A1[(o + r) * LDC + o + ln] = xd[r];
      float4* tp = reinterpret_cast<float4*>(A1t + (o + ln) * LDC + o);
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4)
        tp[q4] = make_float4(xd[4 * q4], xd[4 * q4 + 1], xd[4 * q4 + 2], xd[4 * q4 + 3]);
    }
    // (b) N_ik = A_ii L_ik for i > k, written row-major into the unused
    //     lower-left block positions (i, k) of the L^T storage
#pragma unroll
    for (int p = 0; p < 6; ++p) {
      if (p != wave) continue;
      // pairs (1,0) (2,1) (3,2) (2,0) (3,1) (3,0)
      const int bi = 16 * ((p < 3) ? p + 1 : ((p == 5) ? 3 : p - 1));
      const int bk = 16 * ((p < 3) ? p : ((p == 4) ? 1 : 0));
      const float4 a = *reinterpret_cast<const float4*>(Dg + (bi + ln) * LDD + 4 * g);
      const float4 b = *reinterpret_cast<const float4*>(Lt + (bk + ln) * LDC + bi + 4 * g);
      const f32x4 acc = mma16_f32(a, b, zero4());
#pragma unroll
      for (int i = 0; i < 4; ++i) Lt[(bi + 4 * g + i) * LDC + bk + ln] = acc[i];
    }
    lds_barrier();
    // (c)-(e) A_ij = -sum_{k=j}^{i-1} N_ik A_kj, one block diagonal at a time
    if (wave >= 3 && c0 + C < hi) prefetch(c0 + C);
#pragma unroll
    for (int dist = 1; dist < 4; ++dist) {
#pragma unroll
      for (int bj = 0; bj < 4 - dist; ++bj) {
        if (bj != wave) continue;
        const int bi = bj + dist;
        f32x4 acc = zero4();
#pragma unroll
        for (int bk = bj; bk < bi; ++bk) {
          const float4 a =
              *reinterpret_cast<const float4*>(Lt + (bi * 16 + ln) * LDC + bk * 16 + 4 * g);
          const float4 b =
              *reinterpret_cast<const float4*>(A1t + (bj * 16 + ln) * LDC + bk * 16 + 4 * g);
          acc = mma16_f32(a, b, acc);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) A1[(bi * 16 + 4 * g + i) * LDC + bj * 16 + ln] = -acc[i];
        *reinterpret_cast<float4*>(A1t + (bj * 16 + ln) * LDC + bi * 16 + 4 * g) =
            make_float4(-acc[0], -acc[1], -acc[2], -acc[3]);
      }
      lds_barrier();
    }

    // ---- phase 3: fragments of A1 diag(beta) (hi, lo), (A1 . Gamma) diag(beta) and
    //               (Q K^T . Gamma) -------------------------------------------------------
    {
      // 512 slots of a 64 x 64 fragment matrix, one per thread
      const int s = tid;
      const int sl = s & 63, tile = s >> 6;
      const int rt = tile / KTC, kt = tile % KTC;
      const int sg = sl >> 4, r = rt * 16 + (sl & 15);
      const int k0 = kt * 32 + 4 * sg;
      const float4 a0 = *reinterpret_cast<const float4*>(A1 + r * LDC + k0);
      const float4 a1 = *reinterpret_cast<const float4*>(A1 + r * LDC + k0 + 16);
      const float4 b0 = *reinterpret_cast<const float4*>(gbeta + k0);
      const float4 b1 = *reinterpret_cast<const float4*>(gbeta + k0 + 16);
      const float4 e0 = *reinterpret_cast<const float4*>(gb + k0);
      const float4 e1 = *reinterpret_cast<const float4*>(gb + k0 + 16);
      const float av[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
      const float bv[8] = {b0.x, b0.y, b0.z, b0.w, b1.x, b1.y, b1.z, b1.w};
      const float ev[8] = {e0.x, e0.y, e0.z, e0.w, e1.x, e1.y, e1.z, e1.w};
      const float br = gb[r];
      bf16x8 hh, ll, gg;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int i = k0 + ((j < 4) ? j : 12 + j);
        const bool keep = (i <= r);
        const float ab = keep ? av[j] * bv[j] : 0.f;
        hh[j] = static_cast<__bf16>(ab);
        ll[j] = static_cast<__bf16>(ab - static_cast<float>(hh[j]));
        gg[j] = static_cast<__bf16>(keep ? ab * __expf(br - ev[j]) : 0.f);
      }
      st_frag(fAbh, s * 8, hh);
      st_frag(fAbl, s * 8, ll);
      st_frag(fAgb, s * 8, gg);
    }
    lds_barrier();

    // ---- phase 4: W^T tiles -> fragments (gamma W, W hi, W lo); U ---------------------
    // wave (rt, dg): query-token tile rt = wave % 4, d_k tiles 4*dg .. 4*dg + 3; the
    // A1 diag(beta) fragments of tile rt are loaded once for all four products
    {
      constexpr int NG = DT / 4;  // groups of four d_k tiles
      if (wave < 4 * NG) {
        const int rt = wave & 3, dg = wave >> 2;
        bf16x8 ah[KTC], al[KTC];
#pragma unroll
        for (int kt = 0; kt < KTC; ++kt) {
          ah[kt] = ld_frag(fAbh, frag_slot(rt, kt, KTC, lane));
          al[kt] = ld_frag(fAbl, frag_slot(rt, kt, KTC, lane));
        }
        f32x4 w4[4];
#pragma unroll
        for (int d = 0; d < 4; ++d) {
          f32x4 acc = zero4();
#pragma unroll
          for (int kt = 0; kt < KTC; ++kt) {
            const bf16x8 a = ld_frag(fKt, frag_slot(4 * dg + d, kt, KTC, lane));
            acc = mma(a, ah[kt], acc);
            acc = mma(a, al[kt], acc);
          }
          w4[d] = acc;
        }
        const float gam = ggam[rt * 16 + ln];
#pragma unroll
        for (int p = 0; p < 2; ++p) {
          const int kb = 2 * dg + p;
          bf16x8 hh, ll;
          pack_split(w4[2 * p], w4[2 * p + 1], hh, ll);
          st_frag(fWh, frag_slot(rt, kb, KTD, lane), hh);
          st_frag(fWl, frag_slot(rt, kb, KTD, lane), ll);
          st_frag(fWs, frag_slot(rt, kb, KTD, lane), pack(w4[2 * p] * gam, w4[2 * p + 1] * gam));
        }
      }
    }
    f32x4 u[4];
    if (sw && wave_cols) {
#pragma unroll
      for (int rt = 0; rt < 4; ++rt) {
        f32x4 acc = zero4();
#pragma unroll
        for (int kt = 0; kt < KTC; ++kt)
          acc = mma(ld_frag(fAgb, frag_slot(rt, kt, KTC, lane)),
                    vB[kt], acc);
        u[rt] = acc;
      }
    }
    lds_barrier();

    // ---- phase 5: chain update -----------------------------------------------------------
    if (sw && wave_cols) {
      bf16x8 s0h[KTD];
#pragma unroll
      for (int kb = 0; kb < KTD; ++kb) s0h[kb] = pack(st[2 * kb], st[2 * kb + 1]);
      // Vn = U - W' S0
#pragma unroll
      for (int rt = 0; rt < 4; ++rt) {
        f32x4 acc = zero4();
#pragma unroll
        for (int kb = 0; kb < KTD; ++kb)
          acc = mma(ld_frag(fWs, frag_slot(rt, kb, KTD, lane)), s0h[kb], acc);
        u[rt] -= acc;
      }
      bf16x8 vnf[KTC];
#pragma unroll
      for (int kt = 0; kt < KTC; ++kt) vnf[kt] = pack(u[2 * kt], u[2 * kt + 1]);
      // O^T = (Q S0)^T diag(gamma) + Vn^T (Q K^T . Gamma)^T; lane (g, n) holds
      // O[token rt*16 + n][col0 + 4g .. col0 + 4g + 3]
      u16* og = static_cast<u16*>(args.o);
      const long orow0 = (args.mode == 0) ? static_cast<long>(c0)
                                          : static_cast<long>(seg) * args.w + (c0 - lo);
#pragma unroll
      for (int rt = 0; rt < 4; ++rt) {
        f32x4 acc = oq[rt] * ggam[rt * 16 + ln];
#pragma unroll
        for (int kt = 0; kt < KTC; ++kt)
          if (2 * kt <= rt) acc = mma(vnf[kt], ld_frag(fQK, frag_slot(rt, kt, KTC, lane)), acc);
        const int r = rt * 16 + ln;
        if (og != nullptr && r < n) {
          u16x4 o4;
#pragma unroll
          for (int i = 0; i < 4; ++i) o4[i] = bf16_of(acc[i]);
          *reinterpret_cast<u16x4*>(og + (orow0 + r) * v_stride + h * DV + col0 + 4 * g) = o4;
        }
      }
      // S <- gamma_last S0 + K^T diag(exp(b_last - b)) Vn
#pragma unroll
      for (int kt = 0; kt < KTC; ++kt) {
        const float4 d0 = *reinterpret_cast<const float4*>(gdec + kt * 32 + 4 * g);
        const float4 d1 = *reinterpret_cast<const float4*>(gdec + kt * 32 + 16 + 4 * g);
        f32x4 x0 = u[2 * kt], x1 = u[2 * kt + 1];
        x0[0] *= d0.x;
        x0[1] *= d0.y;
        x0[2] *= d0.z;
        x0[3] *= d0.w;
        x1[0] *= d1.x;
        x1[1] *= d1.y;
        x1[2] *= d1.z;
        x1[3] *= d1.w;
        vnf[kt] = pack(x0, x1);
      }
      const float g_last = __expf(b_last);
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        f32x4 acc = st[dt] * g_last;
#pragma unroll
        for (int kt = 0; kt < KTC; ++kt)
          acc = mma(ld_frag(fKt, frag_slot(dt, kt, KTC, lane)), vnf[kt], acc);
        st[dt] = acc;
      }
    } else if (!sw && has_op) {
      // X = W P0 (three passes);  P <- P0 - K^T X (two passes, K exact)
      bf16x8 p0h[KTD], p0l[KTD];
#pragma unroll
      for (int kb = 0; kb < KTD; ++kb) pack_split(st[2 * kb], st[2 * kb + 1], p0h[kb], p0l[kb]);
      f32x4 x[4];
#pragma unroll
      for (int rt = 0; rt < 4; ++rt) {
        f32x4 acc = zero4();
#pragma unroll
        for (int kb = 0; kb < KTD; ++kb) {
          const bf16x8 wh = ld_frag(fWh, frag_slot(rt, kb, KTD, lane));
          const bf16x8 wl = ld_frag(fWl, frag_slot(rt, kb, KTD, lane));
          acc = mma(wh, p0h[kb], acc);
          acc = mma(wh, p0l[kb], acc);
          acc = mma(wl, p0h[kb], acc);
        }
        x[rt] = -acc;
      }
      bf16x8 xh[KTC], xl[KTC];
#pragma unroll
      for (int kt = 0; kt < KTC; ++kt) pack_split(x[2 * kt], x[2 * kt + 1], xh[kt], xl[kt]);
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        f32x4 acc = st[dt];
#pragma unroll
        for (int kt = 0; kt < KTC; ++kt) {
          const bf16x8 a = ld_frag(fKt, frag_slot(dt, kt, KTC, lane));
          acc = mma(a, xh[kt], acc);
          acc = mma(a, xl[kt], acc);
        }
        st[dt] = acc;
      }
    }
    // phase 0 of the next chunk shares this interval with the update above
    if (c0 + C < hi) phase0(c0 + C, par ^ 1, lane, g, ln);
    lds_barrier();
  }

  // ---- results ------------------------------------------------------------------------
  if (!wave_cols) return;
  if (sw) {
    if (args.S_out != nullptr) {
      float* so = args.S_out + sh * DK * DV;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int i = 0; i < 4; ++i) so[d_perm(dt, 4 * g + i) * DV + col0 + ln] = st[dt][i];
    }
    if (args.log_decay != nullptr && cb == 0 && tid == 0) args.log_decay[sh] = log_decay;
  } else {
    float* po = args.P_hat + sh * DK * DK;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int i = 0; i < 4; ++i) po[d_perm(dt, 4 * g + i) * DK + col0 + ln] = st[dt][i];
  }
}

template <int DK, int DV>
hipError_t launch_t(const ScanArgs& a, int n_items, hipStream_t s) {
  constexpr int bytes = Lds<DK>::TOTAL;
  // one-time (thread-safe static initialisation) opt-in to more than 64 KiB of LDS
  static const hipError_t attr = hipFuncSetAttribute(
      reinterpret_cast<const void*>(&scan_bf16_kernel<DK, DV>),
      hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL((scan_bf16_kernel<DK, DV>), dim3(n_items), dim3(kThreads), bytes, s, a);
  return hipGetLastError();
}

}  // namespace

int scan_bf16_items_per_head(int d_k, int d_v, int with_operator) {
  const int ns = d_v / NCOL, np = d_k / NCOL;
  if (!with_operator) return (d_v + 2 * NCOL - 1) / (2 * NCOL);
  return (np > ns) ? np : ns;
}

hipError_t launch_scan_bf16(const ScanArgs& a, int d_k, int d_v, int n_items, hipStream_t s) {
  if (n_items <= 0) return hipSuccess;
  if (d_k == 64 && d_v == 64) return launch_t<64, 64>(a, n_items, s);
  if (d_k == 64 && d_v == 128) return launch_t<64, 128>(a, n_items, s);
  if (d_k == 128 && d_v == 64) return launch_t<128, 64>(a, n_items, s);
  return launch_t<128, 128>(a, n_items, s);
}

}  // namespace hypic
