// Chunked gated-delta-rule scan, bf16 inputs, chunk 64: the production path
// of the segment build and the seam rescan on gfx950.
//
// Mathematics (per chunk of 64 tokens, incoming state S0; b = prefix sum of
// log alpha inside the chunk, gamma = exp(b), Gamma_ri = exp(b_r - b_i)):
//   L  = strictly-lower part of diag(beta) K K^T,   A1 = (I + L)^{-1}
//   W  = A1 diag(beta) K,       U = (A1 . Gamma) diag(beta) V
//   Vn = U - diag(gamma) W S0
//   O  = diag(gamma) Q S0 + (tril(Q K^T) . Gamma) Vn
//   S  <- gamma_last S0 + K^T diag(exp(b_last - b)) Vn
//   P  <- P0 - K^T (W P0)                         (decay-free operator)
// i.e. the token recurrence of Eq. (2) with the GDN transition of Tab. 1
// applied 64 times (diag(gamma) A1 diag(gamma)^{-1} = A1 . Gamma turns the
// decay-free UT transform into the gated one), and the identity-start operator
// construction of Sec. 5 with the gate factored out as in Tab. 3.
//
// Organisation on CDNA4.  One workgroup of 8 waves runs one (segment, v-head,
// 64-column block) chain.  The waves have fixed roles and the chunk loop is
// software-pipelined three deep, so the chunk-local work (which does not
// depend on the state) runs ahead of the sequential state update:
//   waves 0-1  state columns (32 each): U, Vn, outputs, S update for chunk c;
//   waves 2-3  operator columns (32 each): X = W P0, P update for chunk c
//              (without the operator they carry state columns too);
//              W (hi + lo) of chunk c + 1 is formed after the first barrier by
//              the four waves on SIMDs 2 and 3 (waves 2, 6, 3, 7), one 32-row
//              rho block of d_k each;
//   wave 4     inverse of chunk c + 2: Gram matrix, the four diagonal 16 x 16
//              blocks of A1 by column-parallel substitution (DPP row
//              broadcasts), the off-diagonal blocks of -A1 diag(beta) by
//              split-bf16 products (three passes), all in registers, written
//              as float32 matrix-core fragments;
//   waves 5-7  chunk c + 1: gates, K Q^T masked with Gamma and the Q
//              fragments (wave 5, which loads K and Q once per workgroup);
//              K^T, -A1 diag(beta) split into bf16 hi + lo, and
//              (A1 . Gamma) diag(beta) (waves 6, 7: one half each).
// A seam of w <= 64 tokens is one chunk: up to 16 entries of one head then run
// back to back through the same pipeline, one entry per iteration, each state
// wave storing the finished state and loading the next entry's incoming state
// between iterations.
// Each iteration has two LDS-only barriers: the consumers' state-independent
// products read the previous iteration's fragments before the first, their
// K^T products follow it; the producers write K^T, Q and gates for c + 1
// before the first barrier (double-buffered) and W, (A1 . Gamma) beta and
// (Q K^T . Gamma) after it (single-buffered, the consumers are done with them).
//
// Products are v_mfma_f32_32x32x16_bf16 wherever an operand comes from LDS
// (twice the work of a 16x16x32 product per byte of operand traffic).  Every
// operand is stored "fragment major": a 32 x 16 operand block is 64 lanes x 8
// bf16 in lane order, read with one 16-byte load per lane.  Within a 16-deep
// contraction step, slot (g2, j) of lane group g2 = lane / 32 carries index
// 8(j / 4) + 4 g2 + j % 4, which is exactly the row set a 32 x 32 accumulator
// holds in elements 8h .. 8h+7: accumulators feed the next product as
// operands with no data movement.  Rows of the state and the operator are kept
// in the matching order rho (true row d = rho with bits 2 and 3 swapped), so
// operands loaded straight from HBM (q, k rows: 16 contiguous bytes per lane)
// meet them without shuffles; rows are mapped back only at the HBM boundary.
//
// Precision: q, k, v are exact in bf16.  W is formed from A1 diag(beta)
// split into bf16 hi + lo (K exact) and kept as hi + lo; the state path uses
// single bf16 operands (its decay keeps rounding from accumulating); the
// operator path, which has no decay, splits its float32 operands (three
// passes for W P0, two for K^T X).

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "frag32.hpp"
#include "mfma.hpp"
#include "scan.hpp"

namespace hypic {

namespace {

using namespace f32frag;

constexpr int kThreads = 512;
constexpr int C = 64;     // tokens per chunk
constexpr int NCOL = 64;  // state / operator columns per workgroup (with the operator)

typedef short s16x4 __attribute__((ext_vector_type(4)));
// 16 x 16 x 16 product of float32 operands on the bf16 matrix cores, split
// into hi + lo terms (hi*hi + hi*lo + lo*hi): a[s] = A[r][4g + s],
// b[s] = B[4g + s][n]; lane (g, n) of the result holds C[4g + e][n]
__device__ __forceinline__ void split4(const f32x4& x, s16x4& hi, s16x4& lo) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const __bf16 h = static_cast<__bf16>(x[i]);
    hi[i] = __builtin_bit_cast(short, h);
    lo[i] = __builtin_bit_cast(short, static_cast<__bf16>(x[i] - static_cast<float>(h)));
  }
}
struct Split4 {
  s16x4 h, l;
};
__device__ __forceinline__ Split4 split4(const f32x4& x) {
  Split4 r;
  split4(x, r.h, r.l);
  return r;
}
__device__ __forceinline__ f32x4 mma16_x3(const Split4& a, const Split4& b, f32x4 c) {
  c = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a.h, b.h, c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a.h, b.l, c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a.l, b.h, c, 0, 0, 0);
  return c;
}

// Step I of the column-parallel unit-lower substitution on 16-lane rows: lane
// 16b + c holds column c of the solution (x) and column c of -L (lcol); the
// coefficient -L[r][I] comes from lane I of the same row (DPP row_newbcast:I).
// The broadcast and the multiply-add are one instruction (v_fmac_f32 with a
// DPP source operand).  lcol is written well before its first use as a DPP
// source, so no extra wait states are needed beyond the one nop in front.
template <int I>
__device__ __forceinline__ void unit_lower_solve_step(float (&x)[16], const float (&lcol)[16]) {
  if constexpr (I < 15) {
#pragma unroll
    for (int r = I + 1; r < 16; ++r)
      asm("v_fmac_f32_dpp %0, %1, %2 row_newbcast:%3 row_mask:0xf bank_mask:0xf"
          : "+v"(x[r])
          : "v"(lcol[r]), "v"(x[I]), "n"(I));
    unit_lower_solve_step<I + 1>(x, lcol);
  }
}


// ---- LDS plan (bytes) --------------------------------------------------------
template <int DK>
struct Lds {
  static constexpr int FB = FR * 2;            // bytes of one fragment
  static constexpr int NKT = (DK / 32) * 4;    // K^T fragments (rho tile m, token step s)
  static constexpr int NW = 2 * (DK / 16);     // W / Q fragments (token tile t, d step u)
  static constexpr int O_KT = 0;                       // K^T, two buffers
  static constexpr int O_WH = O_KT + 2 * NKT * FB;     // W hi
  static constexpr int O_WL = O_WH + NW * FB;          // W lo (operator path)
  static constexpr int O_Q = O_WL + NW * FB;           // Q, two buffers
  static constexpr int O_QK = O_Q + 2 * NW * FB;       // (Q K^T . Gamma)^T, 6 fragments
  static constexpr int O_AG = O_QK + 6 * FB;           // (A1 . Gamma) diag(beta), 6 fragments
  static constexpr int O_AB = O_AG + 6 * FB;           // -A1 diag(beta) as bf16 hi + lo
  static constexpr int O_AF = O_AB + 12 * FB;          // -A1 diag(beta) in float32, two buffers
  static constexpr int AFB = 6 * 2 * FB;               // bytes of one float32 buffer
  static constexpr int O_G = O_AF + 2 * AFB;           // gates b, beta, gamma, dec; two buffers
  static constexpr int O_BS = O_G + 2 * 4 * C * 4;     // inverse wave: beta
  static constexpr int TOTAL = O_BS + C * 4;
  static_assert(TOTAL <= 160 * 1024, "LDS budget");
};

// Shared description of the chain a workgroup runs: the chunks of one
// segment (build) or seam entry, or, for seams of at most one chunk, the
// seam entries e0 .. e0 + nc - 1 of one head back to back (one chunk each).
struct Chain {
  int seg, h, hk, lo, hi, nc, cb;
  long sh;            // seg * h_v + h
  long qk_stride;     // elements between token rows of q, k
  long v_stride;      // elements between token rows of v, o
  bool with_op, need_state, need_op;
  bool batched;       // one seam entry per chunk
  int e0, w, n_tok;
  const int32_t* tok_start;
  const int32_t* tok_len;
  const int32_t* ids;  // fused composition: pool entry of listed segment e0 + c
  // batched entries: lane l holds the first token and token count of entry
  // e0 + l (l < 64), read once per workgroup, so that no iteration waits on a
  // chain of dependent loads for its token range
  int pre_t, pre_n;
  int pre_id;    // fused: lane l holds the pool entry of listed segment e0 + l
  float pre_ld;  // fused: lane l holds that entry's log_decay (this head)
};

// token range of seam entry e0 + c (through the request's pool ids when fused)
__device__ __forceinline__ int entry_of(const Chain& ch, int c) {
  return ch.ids != nullptr ? ch.ids[ch.e0 + c] : ch.e0 + c;
}
__device__ __forceinline__ int entry_start(const Chain& ch, int c) {
  const int t = ch.tok_start[entry_of(ch, c)];
  return (t < 0) ? 0 : ((t >= ch.n_tok) ? ch.n_tok - 1 : t);
}
__device__ __forceinline__ int entry_len(const Chain& ch, int c, int t) {
  const int l = ch.tok_len[entry_of(ch, c)];
  int n = (l < ch.w) ? l : ch.w;
  n = (n > ch.n_tok - t) ? ch.n_tok - t : n;
  return (n < 1) ? 1 : n;
}
__device__ __forceinline__ int chunk_start(const Chain& ch, int c) {
  if (!ch.batched) return ch.lo + c * C;
  return (c < 64) ? __builtin_amdgcn_readlane(ch.pre_t, c) : entry_start(ch, c);
}
__device__ __forceinline__ int chunk_len(const Chain& ch, int c) {
  if (!ch.batched) {
    const int r = ch.hi - (ch.lo + c * C);
    return (r < C) ? r : C;
  }
  return (c < 64) ? __builtin_amdgcn_readlane(ch.pre_n, c) : entry_len(ch, c, entry_start(ch, c));
}

// The fused composition (mode 2) adds DK / 32 - 1 barriers to every iteration
// that composes an entry (compose_entry): three producer waves stage P_hat's
// A operands into LDS one output tile at a time, the first before the
// iteration's first barrier and each later one before a barrier of its own
// (producer_compose_first, producer_compose), and a wave without a part in it
// passes the same barriers after its own work.
template <int DK>
__device__ __forceinline__ int compose_barriers(const ScanArgs& args) {
  return args.mode == 2 ? DK / 32 - 1 : 0;
}
__device__ __forceinline__ void pass_barriers(const Chain& ch, int it, int n) {
  if (it >= 0 && it < ch.nc)
    for (int i = 0; i < n; ++i) lds_barrier();
}

// A stager's share of one entry's P_hat A operands: for every output tile m
// (32 rows, order rho) the steps u = FIRST .. FIRST + US - 1 of lane (g2, r):
// true row rho^-1(32 m + r), true columns 16 u + 8 g2 .. +7 in float32.  The
// stagers are the Q K producer (SLOT 0) and the two K^T producers (SLOT 1, 2);
// the inverse wave, the one with no registers to spare, takes no share.  A
// ring of D tiles: the first D are loaded an iteration before they are staged,
// each later one D rounds before.
template <int DK, int SLOT>
struct PShare {
  static constexpr int NM = DK / 32, NU = DK / 16, D = (NM < 2) ? NM : 2;
  // steps per stager: 2, 3, 3 at d_k = 128; 1, 2, 1 at d_k = 64
  static constexpr int US = (NU == 8) ? (SLOT == 0 ? 2 : 3) : (SLOT == 1 ? 2 : 1);
  static constexpr int FIRST = (NU == 8) ? (SLOT == 0 ? 0 : (SLOT == 1 ? 2 : 5))
                                         : (SLOT == 0 ? 0 : (SLOT == 1 ? 1 : 3));
  float4 p[D][US][2];
  const float* pr;  // this lane's first element of the entry's share
};

template <int DK, int SLOT>
__device__ __forceinline__ void share_load_tile(PShare<DK, SLOT>& sh, int m) {
  constexpr int US = PShare<DK, SLOT>::US, D = PShare<DK, SLOT>::D;
#pragma unroll
  for (int k = 0; k < US; ++k) {
    sh.p[m % D][k][0] = *reinterpret_cast<const float4*>(sh.pr + 32 * m * DK + 16 * k);
    sh.p[m % D][k][1] = *reinterpret_cast<const float4*>(sh.pr + 32 * m * DK + 16 * k + 4);
  }
}

template <int DK, int SLOT>
__device__ __forceinline__ void share_load(PShare<DK, SLOT>& sh, const ScanArgs& args,
                                           const Chain& ch, int c, int lane) {
  constexpr int D = PShare<DK, SLOT>::D, FIRST = PShare<DK, SLOT>::FIRST;
  const int id = (c < 64) ? __builtin_amdgcn_readlane(ch.pre_id, c) : entry_of(ch, c);
  const int g2 = lane >> 5, n32 = lane & 31;
  const int prow = (n32 & ~12) | ((n32 & 4) << 1) | ((n32 & 8) >> 1);  // rho -> true row
  sh.pr = args.pool_P + (static_cast<long>(id) * args.h_v + ch.h) * DK * DK + prow * DK +
          8 * g2 + 16 * FIRST;
#pragma unroll
  for (int m = 0; m < D; ++m) share_load_tile<DK, SLOT>(sh, m);
}

// Stage output tile m's share, split into bf16 hi + lo, as fragments 2u (hi)
// and 2u + 1 (lo) of buffer m % 2, then load the share of tile m + D into the
// ring.  The buffers are regions idle during a fused composition: W lo (no
// operator columns) and the Q fragments of chunk c (free once the iteration's
// first barrier has passed, so tile 0, staged before it, goes to W lo).
template <int DK, int SLOT>
__device__ __forceinline__ void share_stage(PShare<DK, SLOT>& sh, unsigned char* smem, int par,
                                            int m, int lane) {
  using LP = Lds<DK>;
  constexpr int NM = PShare<DK, SLOT>::NM, US = PShare<DK, SLOT>::US, D = PShare<DK, SLOT>::D;
  constexpr int FIRST = PShare<DK, SLOT>::FIRST;
  u16* buf = reinterpret_cast<u16*>((m & 1) ? smem + LP::O_Q + par * LP::NW * LP::FB
                                            : smem + LP::O_WL);
#pragma unroll
  for (int k = 0; k < US; ++k) {
    const float4 p0 = sh.p[m % D][k][0], p1 = sh.p[m % D][k][1];
    f32x16 a;
    a[0] = p0.x; a[1] = p0.y; a[2] = p0.z; a[3] = p0.w;
    a[4] = p1.x; a[5] = p1.y; a[6] = p1.z; a[7] = p1.w;
    bf16x8 ah, al;
    split_of(a, 0, ah, al);
    stf(buf, 2 * (FIRST + k), lane, ah);
    stf(buf, 2 * (FIRST + k) + 1, lane, al);
  }
  if (m + D < NM) share_load_tile<DK, SLOT>(sh, m + D);
}

// A stager's part of the fused composition of entry it: tile 0 at the start of
// the iteration (before its first barrier, so the state waves can multiply it
// as soon as they reach it) ...
template <int DK, int SLOT, bool FUSED>
__device__ __forceinline__ void producer_compose_first(PShare<DK, SLOT>& sh, const Chain& ch,
                                                       unsigned char* smem, int it, int lane) {
  if constexpr (FUSED) {
    if (it >= 0 && it < ch.nc) share_stage<DK, SLOT>(sh, smem, it & 1, 0, lane);
  }
}

// ... and at its end the later tiles, one per barrier, then the loads of entry
// it + 1's first tiles.
template <int DK, int SLOT, bool FUSED>
__device__ __forceinline__ void producer_compose(PShare<DK, SLOT>& sh, const ScanArgs& args,
                                                 const Chain& ch, unsigned char* smem, int it,
                                                 int lane) {
  if constexpr (FUSED) {
    if (it >= 0 && it < ch.nc) {
#pragma unroll
      for (int m = 1; m < PShare<DK, SLOT>::NM; ++m) {
        share_stage<DK, SLOT>(sh, smem, it & 1, m, lane);
        lds_barrier();
      }
    }
    if (it + 1 >= 0 && it + 1 < ch.nc) share_load<DK, SLOT>(sh, args, ch, it + 1, lane);
  }
}

// =============================================================================
// wave 4: A1 diag(beta) of chunk c + 2
// =============================================================================
// Exchange (tile b, 16-lane row g) <-> (tile g, 16-lane row b) of four 16 x 16
// tiles held one f32x4 per lane: an involution on (tile, lane row) pairs, done
// with cross-row lane swaps.
__device__ __forceinline__ void exchange_tiles(f32x4 (&x)[4]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
#pragma unroll
    for (int b2 = 0; b2 < 2; ++b2) {  // upper half of tile b2 <-> lower half of b2 + 2
      const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x[b2][i]),
                                                      __float_as_uint(x[b2 + 2][i]), false, false);
      // the two results are copied out one by one before any bit cast
      const unsigned r0 = r[0], r1 = r[1];
      x[b2][i] = __uint_as_float(r0);
      x[b2 + 2][i] = __uint_as_float(r1);
    }
#pragma unroll
    for (int b2 = 0; b2 < 4; b2 += 2) {  // odd rows of tile b2 <-> even rows of b2 + 1
      const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x[b2][i]),
                                                      __float_as_uint(x[b2 + 1][i]), false, false);
      const unsigned r0 = r[0], r1 = r[1];
      x[b2][i] = __uint_as_float(r0);
      x[b2 + 1][i] = __uint_as_float(r1);
    }
  }
}

// X^T of a 16 x 16 float32 tile in accumulator form (lane (g, n): X[4g + e][n]):
// the tile used as an A operand is X^T, multiplied by the identity in two
// exact bf16 passes (hi, lo)
__device__ __forceinline__ f32x4 transpose16(const Split4& x, const s16x4& eye) {
  f32x4 c = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(x.h, eye, zero4(), 0, 0, 0);
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(x.l, eye, c, 0, 0, 0);
}

template <int DK, int DV, bool FUSED>
__device__ __forceinline__ void inverse_wave(const ScanArgs& args, const Chain& ch,
                                             unsigned char* smem, int lane) {
  using LP = Lds<DK>;
  constexpr int KTD = DK / 32;
  const int g = lane >> 4, n16 = lane & 15;
  float* bs = reinterpret_cast<float*>(smem + LP::O_BS);
  const u16* kg = static_cast<const u16*>(args.k) + ch.hk * DK;

  s16x4 eye;  // 16 x 16 identity as a B operand: lane (g, n) slot j is 1 where 4g + j == n
#pragma unroll
  for (int j = 0; j < 4; ++j) eye[j] = (4 * g + j == n16) ? short(0x3F80) : short(0);

  // Row-form block (i, jb) of -A1 diag(beta) (lane (g, n): row 16i + n,
  // columns 16jb + 4g + e) into the float32 fragments (t, s) of -A1 diag(beta):
  // lane (g2, r) of fragment (t, s) holds columns 16s + 8(j/4) + 4g2 + j%4 of
  // row 32t + r, so this lane's four values are slots 4(g/2) .. +3 of lane
  // 32(g%2) + 16(i%2) + n of fragment (i/2, jb).
  auto emit = [&](float* af, int i, int jb, const f32x4& x) __attribute__((always_inline)) {
    const int lane_f = 32 * (g & 1) + 16 * (i & 1) + n16;
    *reinterpret_cast<float4*>(af + (tri_idx(i >> 1, jb) * 64 + lane_f) * 8 + 4 * (g >> 1)) =
        make_float4(x[0], x[1], x[2], x[3]);
  };

  // 16x16x32 A fragments of K: lane (g, r) holds K[16t + r][32u + 8g .. +7]
  uint4 kr[4][KTD];
  float pb = 0.f;
  auto prefetch = [&](int c) __attribute__((always_inline)) {
    const int c0 = chunk_start(ch, c), n = chunk_len(ch, c);
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int tok = 16 * t + n16;
      const int tc = (tok < n) ? tok : n - 1;
      const u16* p = kg + static_cast<long>(c0 + tc) * ch.qk_stride + 8 * g;
#pragma unroll
      for (int u = 0; u < KTD; ++u) kr[t][u] = *reinterpret_cast<const uint4*>(p + 32 * u);
    }
    const int tc = (lane < n) ? lane : n - 1;
    pb = args.beta[static_cast<long>(c0 + tc) * args.h_v + ch.h];
  };
  if (ch.nc > 0) prefetch(0);
  // The fragments hold the blocks above the diagonal (0,1) and (2,3) too; they
  // stay zero (per chunk only blocks on or below the diagonal are written).
#pragma unroll
  for (int par = 0; par < 2; ++par) {
    float* af = reinterpret_cast<float*>(smem + LP::O_AF + par * LP::AFB);
    emit(af, 0, 1, zero4());
    emit(af, 2, 3, zero4());
  }

  for (int it = -2; it < ch.nc; ++it) {
    const int c = it + 2;
    const bool active = c < ch.nc;
    f32x4 gu[6];      // upper Gram tiles (k, i), k < i: rows of L_ik once scaled by beta
    f32x4 dc[4], dr[4];  // diagonal blocks D_b of A1: accumulator form, row form
    if (active) {
      const int n = chunk_len(ch, c);
      const float beta = (lane < n) ? pb : 0.f;
      bs[lane] = beta;
      if (n < C) {
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
          for (int u = 0; u < KTD; ++u) kr[t][u] = mask4(kr[t][u], 16 * t + n16 < n);
      }
      f32x4 gd[4];
#pragma unroll
      for (int bd = 0; bd < 4; ++bd) {
        gd[bd] = zero4();
#pragma unroll
        for (int u = 0; u < KTD; ++u) gd[bd] = mma16(as_bf(kr[bd][u]), as_bf(kr[bd][u]), gd[bd]);
      }
#pragma unroll
      for (int p = 0; p < 6; ++p) {
        // pairs (0,1) (0,2) (0,3) (1,2) (1,3) (2,3)
        const int k = (p < 3) ? 0 : ((p < 5) ? 1 : 2);
        const int i = (p < 3) ? p + 1 : ((p < 5) ? p - 1 : 3);
        gu[p] = zero4();
#pragma unroll
        for (int u = 0; u < KTD; ++u) gu[p] = mma16(as_bf(kr[k][u]), as_bf(kr[i][u]), gu[p]);
      }
      if (c + 1 < ch.nc) prefetch(c + 1);
      // afterwards lane 16b + c of tile q holds G_b[4q + e][c]: lane 16b + c has
      // column c of the diagonal Gram block b
      exchange_tiles(gd);
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // beta visible to the wave
      const int ob = g * 16;
      float lcol[16];  // -L[r][c] = -beta_r G[r][c] of block g (used for r > c)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const float4 bb = *reinterpret_cast<const float4*>(bs + ob + 4 * q4);
        lcol[4 * q4] = -bb.x * gd[q4][0];
        lcol[4 * q4 + 1] = -bb.y * gd[q4][1];
        lcol[4 * q4 + 2] = -bb.z * gd[q4][2];
        lcol[4 * q4 + 3] = -bb.w * gd[q4][3];
      }
      float xd[16];  // lane 16b + c: column c of D_b
#pragma unroll
      for (int r = 0; r < 16; ++r) xd[r] = (r == n16) ? 1.f : 0.f;
      asm volatile("s_nop 1" ::: "memory");
      unit_lower_solve_step<0>(xd, lcol);
      // the same exchange turns the columns into accumulator form
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4)
        dc[q4] = f32x4{xd[4 * q4], xd[4 * q4 + 1], xd[4 * q4 + 2], xd[4 * q4 + 3]};
      exchange_tiles(dc);
#pragma unroll
      for (int bd = 0; bd < 4; ++bd) dr[bd] = transpose16(split4(dc[bd]), eye);
    }
    lds_barrier();
    if (active) {
      float* af = reinterpret_cast<float*>(smem + LP::O_AF + (c & 1) * LP::AFB);
      // L_ik as A operand: lane (g, r): beta_{16i + r} G[16i + r][16k + 4g + s];
      // every operand is split into bf16 hi + lo once
      auto Lr = [&](int i, int k) __attribute__((always_inline)) {
        const int p = (k == 0) ? i - 1 : ((k == 1) ? i + 1 : 5);
        return split4(gu[p] * bs[16 * i + n16]);
      };
      const Split4 L10 = Lr(1, 0), L20 = Lr(2, 0), L21 = Lr(2, 1);
      const Split4 L30 = Lr(3, 0), L31 = Lr(3, 1), L32 = Lr(3, 2);
      // Y = -A1 diag(beta) block by block: Y_jj = D_j diag(-beta_j),
      // Y_ij = -D_i sum_{k=j}^{i-1} L_ik Y_kj (the column scaling commutes
      // with the recursion)
      f32x4 yd[3];
#pragma unroll
      for (int j = 0; j < 3; ++j) yd[j] = dc[j] * -bs[16 * j + n16];
      const Split4 Y0 = split4(yd[0]), Y1 = split4(yd[1]), Y2 = split4(yd[2]);
      const Split4 R1 = split4(dr[1]), R2 = split4(dr[2]), R3 = split4(dr[3]);
      // T_ij = sum_k L_ik Y_kj; Y_ij = -D_i T_ij in accumulator form where a later
      // product needs it, and its row form -T_ij^T D_i^T (T as the A operand is
      // T^T, the row form of D_i as the B operand is D_i^T) for the fragments
      const Split4 T10 = split4(mma16_x3(L10, Y0, zero4()));
      const Split4 T21 = split4(mma16_x3(L21, Y1, zero4()));
      const Split4 T32 = split4(mma16_x3(L32, Y2, zero4()));
      const Split4 Y10 = split4(-mma16_x3(R1, T10, zero4()));
      const Split4 Y21 = split4(-mma16_x3(R2, T21, zero4()));
      const Split4 T20 = split4(mma16_x3(L21, Y10, mma16_x3(L20, Y0, zero4())));
      const Split4 T31 = split4(mma16_x3(L32, Y21, mma16_x3(L31, Y1, zero4())));
      const Split4 Y20 = split4(-mma16_x3(R2, T20, zero4()));
      const Split4 T30 =
          split4(mma16_x3(L32, Y20, mma16_x3(L31, Y10, mma16_x3(L30, Y0, zero4()))));
      // every block on or below the diagonal, in row form, into the fragments
#pragma unroll
      for (int bd = 0; bd < 4; ++bd) {
        const float4 bb = *reinterpret_cast<const float4*>(bs + 16 * bd + 4 * g);
        emit(af, bd, bd, dr[bd] * f32x4{-bb.x, -bb.y, -bb.z, -bb.w});
      }
      emit(af, 1, 0, -mma16_x3(T10, R1, zero4()));
      emit(af, 2, 1, -mma16_x3(T21, R2, zero4()));
      emit(af, 3, 2, -mma16_x3(T32, R3, zero4()));
      emit(af, 2, 0, -mma16_x3(T20, R2, zero4()));
      emit(af, 3, 1, -mma16_x3(T31, R3, zero4()));
      emit(af, 3, 0, -mma16_x3(T30, R3, zero4()));
    }
    pass_barriers(ch, it, compose_barriers<DK>(args));
    lds_barrier();
  }
}

// =============================================================================
// waves 5-7: the state-independent fragments of chunk c + 1
// =============================================================================
// W^T tiles (rho tile m, token tile t) = K^T (A1 diag beta)^T in two passes,
// from the negated A1 diag(beta) fragments, so the tiles hold -W^T; the
// accumulator halves are the fragments (t, u = 2m + h) of -W, kept as hi + lo.
// Formed after the first barrier of iteration c for chunk c + 1 by the waves
// that share SIMDs 2 and 3 (the least loaded after that barrier): waves 2, 6,
// 3, 7 take rho tiles 0, 1, 2, 3.
// rho tile of W formed by consumer slot w (waves 0-3), or -1
__device__ __forceinline__ int w_tile(int w) { return (w == 2) ? 0 : ((w == 3) ? 2 : -1); }

template <int DK>
__device__ __forceinline__ void emit_w(const Chain& ch, unsigned char* smem, int lane, int par,
                                       int m) {
  using LP = Lds<DK>;
  constexpr int NU = DK / 16;
  if (m < 0 || m >= DK / 32) return;
  const u16* fKt = reinterpret_cast<const u16*>(smem + LP::O_KT + par * LP::NKT * LP::FB);
  const u16* ab = reinterpret_cast<const u16*>(smem + LP::O_AB);
  u16* fWh = reinterpret_cast<u16*>(smem + LP::O_WH);
  u16* fWl = reinterpret_cast<u16*>(smem + LP::O_WL);
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    f32x16 acc = zero16();
#pragma unroll
    for (int s = 0; s < 2 * t + 2; ++s) {
      const bf16x8 a = ldf(fKt, m * 4 + s, lane);
      acc = mma32(a, ldf(ab, tri_idx(t, s), lane), acc);
      acc = mma32(a, ldf(ab, 6 + tri_idx(t, s), lane), acc);
    }
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      bf16x8 hi, lo;
      split_of(acc, h, hi, lo);
      stf(fWh, t * NU + 2 * m + h, lane, hi);
      if (ch.need_op) stf(fWl, t * NU + 2 * m + h, lane, lo);
    }
  }
}

// raw 16-byte loads of the 16x16x32-layout fragments of one 16-token tile of a
// token-major bf16 matrix: lane (g, r) gets row 16t + r, columns 32u + 8g ..
// +7 for u = 0 .. NB-1 (16 rows x 64 contiguous bytes per instruction; rows
// past the chunk are clamped and zeroed at use)
template <int NB>
__device__ __forceinline__ void load_tile16(uint4 (&dst)[NB], const u16* base, long rs, int c0,
                                            int n, int t, int lane) {
  const int tok = 16 * t + (lane & 15);
  const int tc = (tok < n) ? tok : n - 1;
  const u16* p = base + static_cast<long>(c0 + tc) * rs + 8 * (lane >> 4);
#pragma unroll
  for (int u = 0; u < NB; ++u) dst[u] = *reinterpret_cast<const uint4*>(p + 32 * u);
}

// Wave 5: loads all of K and Q of the chunk (one copy per workgroup) and the
// gates; forms K Q^T masked with Gamma, the Q fragments and its share of W.
template <int DK, int DV, bool FUSED>
__device__ __forceinline__ void producer_qk_wave(const ScanArgs& args, const Chain& ch,
                                                 unsigned char* smem, int lane) {
  using LP = Lds<DK>;
  PShare<DK, 0> psh;  // fused composition: this wave's share of the next entry's P_hat
  constexpr int NU = DK / 16;
  constexpr int KTD = DK / 32;
  const int g = lane >> 4, n16 = lane & 15;
  const u16* kg = static_cast<const u16*>(args.k) + ch.hk * DK;
  const u16* qg = static_cast<const u16*>(args.q) + ch.hk * DK;
  u16* fQK = reinterpret_cast<u16*>(smem + LP::O_QK);

  // K Q^T tiles (k tile 1, q tile 0) and (3, 2) lie above the diagonal inside
  // fragments that are read; they stay zero
  *reinterpret_cast<u16x4*>(fQK + scatter_off(tri_idx(0, 1), 0, lane)) = pack4(0.f, 0.f, 0.f, 0.f);
  *reinterpret_cast<u16x4*>(fQK + scatter_off(tri_idx(1, 3), 0, lane)) = pack4(0.f, 0.f, 0.f, 0.f);

  uint4 kr[4][KTD], qr[4][KTD];
  float pa = 0.f, pbeta = 0.f;
  auto prefetch = [&](int c) __attribute__((always_inline)) {
    const int c0 = chunk_start(ch, c), n = chunk_len(ch, c);
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      load_tile16<KTD>(kr[t], kg, ch.qk_stride, c0, n, t, lane);
      load_tile16<KTD>(qr[t], qg, ch.qk_stride, c0, n, t, lane);
    }
    const int tc = (lane < n) ? lane : n - 1;
    const long idx = static_cast<long>(c0 + tc) * args.h_v + ch.h;
    pa = args.log_alpha[idx];
    pbeta = args.beta[idx];
  };
  if (ch.nc > 0) prefetch(0);

  for (int it = -2; it < ch.nc; ++it) {
    producer_compose_first<DK, 0, FUSED>(psh, ch, smem, it, lane);
    const int p = it + 1;
    const bool active = p >= 0 && p < ch.nc;
    const int par = p & 1;
    f32x4 kq[10];  // K Q^T 16 x 16 tiles (k tile tk <= q tile tq), in order of tq then tk
    if (active) {
      const int n = chunk_len(ch, p);
      float* gb = reinterpret_cast<float*>(smem + LP::O_G + par * 4 * C * 4);
      // gates: b = prefix sum of log alpha (stored in log2 units, b2 = b
      // log2(e), so every decay factor is one exp2), beta, gamma = exp(b),
      // exp(b_last - b)
      {
        float b = (lane < n) ? pa * 1.44269504088896341f : 0.f;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
          const float u = __shfl_up(b, off, 64);
          if (lane >= off) b += u;
        }
        const float b_last = __shfl(b, 63, 64);
        gb[lane] = b;
        gb[C + lane] = (lane < n) ? pbeta : 0.f;
        gb[2 * C + lane] = __builtin_amdgcn_exp2f(b);
        gb[3 * C + lane] = __builtin_amdgcn_exp2f(b_last - b);
      }
      if (n < C) {
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
          for (int u = 0; u < KTD; ++u) {
            kr[t][u] = mask4(kr[t][u], 16 * t + n16 < n);
            qr[t][u] = mask4(qr[t][u], 16 * t + n16 < n);
          }
      }
      if (ch.need_state) {
        u16* fQ = reinterpret_cast<u16*>(smem + LP::O_Q + par * LP::NW * LP::FB);
#pragma unroll
        for (int tq = 0, i = 0; tq < 4; ++tq)
#pragma unroll
          for (int tk = 0; tk <= tq; ++tk, ++i) {
            kq[i] = zero4();
#pragma unroll
            for (int u = 0; u < KTD; ++u) kq[i] = mma16(as_bf(kr[tk][u]), as_bf(qr[tq][u]), kq[i]);
          }
        // Q fragments for the consumers' (Q S0)^T: the 16 bytes of lane (g, r)
        // of tile (t, u) are slot group g%2 of lane 16(t%2) + r of fragment
        // (t/2, 2u + g/2)
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
          for (int u = 0; u < KTD; ++u)
            *reinterpret_cast<uint4*>(fQ + ((t >> 1) * NU + 2 * u + (g >> 1)) * FR +
                                      (32 * (g & 1) + 16 * (t & 1) + n16) * 8) = qr[t][u];
      }
    }
    lds_barrier();
    if (active) {
      if (p + 1 < ch.nc) prefetch(p + 1);
      if (ch.need_state) {
        const float* gb = reinterpret_cast<const float*>(smem + LP::O_G + par * 4 * C * 4);
        // (Q K^T . Gamma)^T as B fragments (key step s, query tile): the tile
        // (tk, tq) holds (K Q^T)[16tk + 4g + e][16tq + n]; kept where key <= query,
        // times exp(b_q - b_k)
#pragma unroll
        for (int tq = 0, i = 0; tq < 4; ++tq) {
          const float bq = gb[16 * tq + n16];
#pragma unroll
          for (int tk = 0; tk <= tq; ++tk, ++i) {
            const float4 bk = *reinterpret_cast<const float4*>(gb + 16 * tk + 4 * g);
            const float bkv[4] = {bk.x, bk.y, bk.z, bk.w};
            float v[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              // computed for every slot, then selected: no divergent branch
              const float x = kq[i][e] * __builtin_amdgcn_exp2f(bq - bkv[e]);
              v[e] = (tk < tq || 4 * g + e <= n16) ? x : 0.f;
            }
            *reinterpret_cast<u16x4*>(fQK + scatter_off(tri_idx(tq >> 1, tk), tq & 1, lane)) =
                pack4(v[0], v[1], v[2], v[3]);
          }
        }
      }
    }
    producer_compose<DK, 0, FUSED>(psh, args, ch, smem, it, lane);
    lds_barrier();
  }
}

// Waves 6, 7: load one d_k half of K (HALF = 0, 1) and form its K^T
// fragments; then (A1 . Gamma) diag(beta) and a share of W.
template <int DK, int DV, int HALF, bool FUSED>
__device__ __forceinline__ void producer_kt_wave(const ScanArgs& args, const Chain& ch,
                                                 unsigned char* smem, int lane) {
  using LP = Lds<DK>;
  PShare<DK, 1 + HALF> psh;  // fused composition: this wave's share of the next entry's P_hat
  constexpr int NH = DK / 64;  // 32-wide d_k blocks of this half
  const int g = lane >> 4, n16 = lane & 15;
  const int g2 = lane >> 5, n32 = lane & 31;
  const u16* kg = static_cast<const u16*>(args.k) + ch.hk * DK + HALF * (DK / 2);
  u16* fAG = reinterpret_cast<u16*>(smem + LP::O_AG);

  // selectors for K^T over one 32-wide d block: B operand of 16x16x32, lane
  // (g, n) slot j is 1 where 8g + j == 16h + n with bits 2, 3 swapped
  bf16x8 esel[2];
  {
    const int pn = (n16 & ~12) | ((n16 & 4) << 1) | ((n16 & 8) >> 1);
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int j = 0; j < 8; ++j)
        esel[h][j] = static_cast<__bf16>((8 * g + j == 16 * h + pn) ? 1.f : 0.f);
  }
  uint4 kr[4][NH];
  auto prefetch = [&](int c) __attribute__((always_inline)) {
    const int c0 = chunk_start(ch, c), n = chunk_len(ch, c);
#pragma unroll
    for (int t = 0; t < 4; ++t) load_tile16<NH>(kr[t], kg, ch.qk_stride, c0, n, t, lane);
  };
  if (ch.nc > 0) prefetch(0);

  for (int it = -2; it < ch.nc; ++it) {
    producer_compose_first<DK, 1 + HALF, FUSED>(psh, ch, smem, it, lane);
    const int p = it + 1;
    const bool active = p >= 0 && p < ch.nc;
    const int par = p & 1;
    if (active) {
      const int n = chunk_len(ch, p);
      u16* fKt = reinterpret_cast<u16*>(smem + LP::O_KT + par * LP::NKT * LP::FB);
      if (n < C) {
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
          for (int u = 0; u < NH; ++u) kr[t][u] = mask4(kr[t][u], 16 * t + n16 < n);
      }
      // K^T: the 16 x 16 tile (token tile t, rho tile mt) is K times a 0/1
      // selector; lane (g, n) holds K[16t + 4g + e][true row of rho 16mt + n],
      // which are slots 4(g/2) .. +3 of lane 32(g%2) + 16(mt%2) + n of the
      // fragment (rho tile mt/2, token step t)
#pragma unroll
      for (int u = 0; u < NH; ++u)
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int mt = 2 * (HALF * NH + u) + h;
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            const f32x4 x = mma16(as_bf(kr[t][u]), esel[h], zero4());
            *reinterpret_cast<u16x4*>(fKt + scatter_off((mt >> 1) * 4 + t, mt & 1, lane)) =
                pack4(x[0], x[1], x[2], x[3]);
          }
        }
      {
        // -A1 diag(beta) of this chunk as bf16 hi + lo fragments for W: wave 6
        // the fragments 0-2, wave 7 the fragments 3-5
        const float* af = reinterpret_cast<const float*>(smem + LP::O_AF + par * LP::AFB);
        u16* ab = reinterpret_cast<u16*>(smem + LP::O_AB);
#pragma unroll
        for (int f = 3 * HALF; f < 3 * HALF + 3; ++f) {
          const float4 v0 = *reinterpret_cast<const float4*>(af + (f * 64 + lane) * 8);
          const float4 v1 = *reinterpret_cast<const float4*>(af + (f * 64 + lane) * 8 + 4);
          f32x16 x;
          x[0] = v0.x; x[1] = v0.y; x[2] = v0.z; x[3] = v0.w;
          x[4] = v1.x; x[5] = v1.y; x[6] = v1.z; x[7] = v1.w;
          bf16x8 hi, lo;
          split_of(x, 0, hi, lo);
          stf(ab, f, lane, hi);
          stf(ab, 6 + f, lane, lo);
        }
      }
      if (p + 1 < ch.nc) prefetch(p + 1);
    }
    lds_barrier();
    if (active) {
      const float* af = reinterpret_cast<const float*>(smem + LP::O_AF + par * LP::AFB);
      const float* gb = reinterpret_cast<const float*>(smem + LP::O_G + par * 4 * C * 4);
      if (ch.need_state) {
        // (A1 . Gamma) diag(beta) as A fragments (t, s): lane (g2, r) holds
        // exp(b_r - b_i) A1[r][i] beta_i, r = 32t + r, i = slot; wave 6 the
        // fragments 0-3, wave 7 the fragments 4, 5
#pragma unroll
        for (int f = (HALF == 0) ? 0 : 4; f < ((HALF == 0) ? 4 : 6); ++f) {
          const int t = (f < 2) ? 0 : 1, s = (f < 2) ? f : f - 2;
          const int row = 32 * t + n32;
          const float br = gb[row];
          const float4 b0 = *reinterpret_cast<const float4*>(gb + 16 * s + 4 * g2);
          const float4 b1 = *reinterpret_cast<const float4*>(gb + 16 * s + 8 + 4 * g2);
          const float bi[8] = {b0.x, b0.y, b0.z, b0.w, b1.x, b1.y, b1.z, b1.w};
          const float4 v0 = *reinterpret_cast<const float4*>(af + (f * 64 + lane) * 8);
          const float4 v1 = *reinterpret_cast<const float4*>(af + (f * 64 + lane) * 8 + 4);
          const float av[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
          bf16x8 o;
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            // the fragments hold -A1 diag(beta)
            const float x = av[j] * -__builtin_amdgcn_exp2f(br - bi[j]);
            o[j] = static_cast<__bf16>((slot_idx(s, g2, j) <= row) ? x : 0.f);
          }
          stf(fAG, f, lane, o);
        }
      }
      emit_w<DK>(ch, smem, lane, par, 1 + 2 * HALF);
    }
    producer_compose<DK, 1 + HALF, FUSED>(psh, args, ch, smem, it, lane);
    lds_barrier();
  }
}

// =============================================================================
// waves 0-3: the chain update of chunk c
// =============================================================================

// One Eq. (4) step of the fused composition, S <- exp(g) P S + S_i, for a
// state wave's 32 columns (all d_k rows, order rho).  P's A operands (lane
// (g2, r) of step u: true row rho^-1(32 m + r), true columns 16 u + 8 g2 ..
// +7, the slot order of a state B fragment mapped back to 8 contiguous
// columns, split into bf16 hi + lo) are staged once per workgroup by the four
// producer waves into two LDS buffers in turn, tile 0 before the iteration's
// first barrier and each later tile before a barrier of its own; the producers
// load them ahead.  The B operand is exp(g) S from the accumulators, split
// once; S_i's tiles are loaded at the start and added to each tile's product;
// three passes.  d_k / 32 - 1 barriers.
template <int DK, int DV>
__device__ __forceinline__ void compose_entry(f32x16 (&st)[DK / 32], const float* Si, float e,
                                              int col0, int lane, const u16* buf0,
                                              const u16* buf1) {
  constexpr int NM = DK / 32, NU = DK / 16;
  const int g2 = lane >> 5;
  bf16x8 bh[NU], bl[NU];
#pragma unroll
  for (int u = 0; u < NU; ++u) {
    const f32x16 es = st[u >> 1] * e;
    split_of(es, u & 1, bh[u], bl[u]);
  }
  // S_i's tiles of this wave's columns (the state registers are free now)
  const float* sr = Si + col0 + (lane & 31);
#pragma unroll
  for (int m = 0; m < NM; ++m)
#pragma unroll
    for (int x = 0; x < 16; ++x) st[m][x] = sr[true_row(m, x, g2) * DV];
#pragma unroll
  for (int m = 0; m < NM; ++m) {
    if (m > 0) lds_barrier();  // tile m is staged (tile 0 before the iteration's first barrier)
    const u16* cur = (m & 1) ? buf1 : buf0;
    f32x16 acc = zero16();
#pragma unroll
    for (int u = 0; u < NU; ++u) {
      const bf16x8 ah = ldf(cur, 2 * u, lane), al = ldf(cur, 2 * u + 1, lane);
      acc = mma32(ah, bh[u], acc);
      acc = mma32(ah, bl[u], acc);
      acc = mma32(al, bh[u], acc);
    }
    st[m] += acc;
  }
}

template <int DK, int DV, bool FUSED>
__device__ __forceinline__ void state_wave(const ScanArgs& args, const Chain& ch,
                                           unsigned char* smem, int lane, int col0, int wslot) {
  using LP = Lds<DK>;
  constexpr int NU = DK / 16;
  constexpr int NM = DK / 32;
  const int g2 = lane >> 5, n32 = lane & 31;
  const u16* fWh = reinterpret_cast<const u16*>(smem + LP::O_WH);
  const u16* fQK = reinterpret_cast<const u16*>(smem + LP::O_QK);
  const u16* fAG = reinterpret_cast<const u16*>(smem + LP::O_AG);
  const u16* vg = static_cast<const u16*>(args.v) + ch.h * DV + col0;
  u16* og = static_cast<u16*>(args.o);

  // state columns col0 .. col0 + 31, all d_k rows (order rho)
  f32x16 st[NM];
#pragma unroll
  for (int m = 0; m < NM; ++m) st[m] = zero16();
  const float* s_first = FUSED ? args.S_prefix : (args.mode == 1 ? args.S_in : nullptr);
  if (s_first != nullptr) {
    const float* s_in = s_first + ch.sh * DK * DV + col0 + n32;
#pragma unroll
    for (int m = 0; m < NM; ++m)
#pragma unroll
      for (int e = 0; e < 16; ++e) st[m][e] = s_in[true_row(m, e, g2) * DV];
  }
  // identity selector for the V transposes: slot j of step u is 1 where
  // 16u + 8g2 + j == n
  bf16x8 isel[2];
#pragma unroll
  for (int u = 0; u < 2; ++u)
#pragma unroll
    for (int j = 0; j < 8; ++j)
      isel[u][j] = static_cast<__bf16>((16 * u + 8 * g2 + j == n32) ? 1.f : 0.f);

  uint4 vr[2][2];
  auto prefetch = [&](int c) __attribute__((always_inline)) {
    const int c0 = chunk_start(ch, c), n = chunk_len(ch, c);
    load_tile32<2>(vr[0], vg, ch.v_stride, c0, n, 0, lane);
    load_tile32<2>(vr[1], vg, ch.v_stride, c0, n, 1, lane);
  };
  if (ch.nc > 0) prefetch(0);
  float log_decay = 0.f;

  const int lane_in = lane;
  for (int it = -2; it < ch.nc; ++it) {
    // an opaque copy of the lane index keeps the compiler from hoisting every
    // loop-invariant fragment address out of the chunk loop (each would pin a
    // register); they are cheap to recompute per chunk
    int lane = lane_in;
    asm volatile("" : "+v"(lane));
    const int g2 = lane >> 5, n32 = lane & 31;
    const int c = it;
    const bool active = c >= 0;
    const int par = c & 1;
    const float* gb = reinterpret_cast<const float*>(smem + LP::O_G + par * 4 * C * 4);
    bf16x8 dvn[4];
    if (active) {
      const int c0 = chunk_start(ch, c), n = chunk_len(ch, c);
      const float* ggam = gb + 2 * C;
      const float* gdec = gb + 3 * C;
      const u16* fQ = reinterpret_cast<const u16*>(smem + LP::O_Q + par * LP::NW * LP::FB);
      // V (this wave's columns) as B fragments over tokens, by exact
      // products with the identity: lane (g2, n) holds V[slot][col0 + n]
      bf16x8 vB[4];
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const bool keep = n == C || 32 * t + n32 < n;
        f32x16 acc = mma32(masked(vr[t][0], keep), isel[0], zero16());
        acc = mma32(masked(vr[t][1], keep), isel[1], acc);
        vB[2 * t] = frag_of(acc, 0);
        vB[2 * t + 1] = frag_of(acc, 1);
      }
      if (c + 1 < ch.nc) prefetch(c + 1);
      // U = (A1 . Gamma) diag(beta) V
      f32x16 vn[2];
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        vn[t] = zero16();
#pragma unroll
        for (int s = 0; s < 2 * t + 2; ++s)
          vn[t] = mma32(ldf(fAG, tri_idx(t, s), lane), vB[s], vn[t]);
      }
      // S0 as bf16 operands (step u over rho); shared by W S0 and (Q S0)^T
      bf16x8 s0[NU];
#pragma unroll
      for (int u = 0; u < NU; ++u) s0[u] = frag_of(st[u >> 1], u & 1);
      // Vn = U - diag(gamma) W S0 (the W fragments hold -W)
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        f32x16 ws = zero16();
#pragma unroll
        for (int u = 0; u < NU; ++u) ws = mma32(ldf(fWh, t * NU + u, lane), s0[u], ws);
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          const float4 gm = *reinterpret_cast<const float4*>(ggam + 32 * t + 8 * b + 4 * g2);
          vn[t][4 * b] += gm.x * ws[4 * b];
          vn[t][4 * b + 1] += gm.y * ws[4 * b + 1];
          vn[t][4 * b + 2] += gm.z * ws[4 * b + 2];
          vn[t][4 * b + 3] += gm.w * ws[4 * b + 3];
        }
      }
      // O^T = (S0^T Q^T) diag(gamma) + Vn^T (Q K^T . Gamma)^T; lane (g2, n)
      // holds O[token 32tq + n][col0 + 8b + 4g2 + i]
      bf16x8 vA[4];
#pragma unroll
      for (int s = 0; s < 4; ++s) vA[s] = frag_of(vn[s >> 1], s & 1);
      const long orow0 = (args.mode == 0) ? static_cast<long>(c0)
                         : ch.batched ? static_cast<long>(seam_out_entry(args, ch.e0 + c)) * args.w
                                      : static_cast<long>(seam_out_entry(args, ch.seg)) * args.w +
                                            (c0 - ch.lo);
#pragma unroll
      for (int tq = 0; tq < 2; ++tq) {
        f32x16 acc = zero16();
#pragma unroll
        for (int u = 0; u < NU; ++u) acc = mma32(s0[u], ldf(fQ, tq * NU + u, lane), acc);
        acc *= ggam[32 * tq + n32];
#pragma unroll
        for (int s = 0; s < 2 * tq + 2; ++s)
          acc = mma32(vA[s], ldf(fQK, tri_idx(tq, s), lane), acc);
        const int r = 32 * tq + n32;
        if (og != nullptr && r < n) {
          u16* dst = og + (orow0 + r) * ch.v_stride + ch.h * DV + col0 + 4 * g2;
#pragma unroll
          for (int b = 0; b < 4; ++b) {
            u16x4 o4;
#pragma unroll
            for (int i = 0; i < 4; ++i) o4[i] = bf16_bits(acc[4 * b + i]);
            *reinterpret_cast<u16x4*>(dst + 8 * b) = o4;
          }
        }
      }
      // diag(exp(b_last - b)) Vn as B fragments over tokens
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        const float4 d0 = *reinterpret_cast<const float4*>(gdec + 16 * s + 4 * g2);
        const float4 d1 = *reinterpret_cast<const float4*>(gdec + 16 * s + 8 + 4 * g2);
        const float dv[8] = {d0.x, d0.y, d0.z, d0.w, d1.x, d1.y, d1.z, d1.w};
        bf16x8 f;
#pragma unroll
        for (int j = 0; j < 8; ++j) f[j] = static_cast<__bf16>(vn[s >> 1][8 * (s & 1) + j] * dv[j]);
        dvn[s] = f;
      }
    }
    lds_barrier();
    // the seam advances the state, except in a fused composition that reads
    // the seam from the incoming state only
    if (active && (!FUSED || args.advance)) {
      const u16* fKt = reinterpret_cast<const u16*>(smem + LP::O_KT + par * LP::NKT * LP::FB);
      const float b_last = gb[C - 1];  // log2 units
      log_decay += b_last * 0.693147180559945309f;
      const float g_last = __builtin_amdgcn_exp2f(b_last);
#pragma unroll
      for (int m = 0; m < NM; ++m) {
        f32x16 acc = st[m] * g_last;
#pragma unroll
        for (int s = 0; s < 4; ++s) acc = mma32(ldf(fKt, m * 4 + s, lane), dvn[s], acc);
        st[m] = acc;
      }
    }
    if constexpr (FUSED) {
      // Eq. (4) with the listed segment's tuple
      if (active) {
        const int id = (c < 64) ? __builtin_amdgcn_readlane(ch.pre_id, c) : entry_of(ch, c);
        const long ih = static_cast<long>(id) * args.h_v + ch.h;
        const float ld = (c < 64) ? __builtin_amdgcn_readlane(__float_as_int(ch.pre_ld), c)
                                  : __float_as_int(args.pool_ld[ih]);
        compose_entry<DK, DV>(st, args.pool_S + ih * DK * DV, __expf(__int_as_float(ld)), col0,
                              lane, reinterpret_cast<const u16*>(smem + LP::O_WL),
                              reinterpret_cast<const u16*>(smem + LP::O_Q + par * LP::NW * LP::FB));
      }
    } else if (active && ch.batched) {
      // one seam entry per chunk: its state after the seam, then the state
      // entering the next entry
      const long eh = static_cast<long>(ch.e0 + c) * args.h_v + ch.h;
      // an opaque copy of the row stride keeps the compiler from hoisting all
      // 64 row offsets out of the loop (each would pin a register)
      int dv = DV;
      asm volatile("" : "+v"(dv));
      __builtin_amdgcn_sched_barrier(0);
      if (args.S_out != nullptr) {
        float* so = args.S_out + eh * DK * DV + col0 + n32;
#pragma unroll
        for (int m = 0; m < NM; ++m)
#pragma unroll
          for (int e = 0; e < 16; ++e) so[true_row(m, e, g2) * dv] = st[m][e];
      }
      __builtin_amdgcn_sched_barrier(0);
      if (c + 1 < ch.nc) {
        const float* s_in = args.S_in + (eh + args.h_v) * DK * DV + col0 + n32;
#pragma unroll
        for (int m = 0; m < NM; ++m)
#pragma unroll
          for (int e = 0; e < 16; ++e) st[m][e] = s_in[true_row(m, e, g2) * dv];
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    if (it + 1 >= 0 && it + 1 < ch.nc) emit_w<DK>(ch, smem, lane, (it + 1) & 1, w_tile(wslot));
    lds_barrier();
  }

  float* s_last = FUSED ? args.S_final : (ch.batched ? nullptr : args.S_out);
  if (s_last != nullptr) {
    float* so = s_last + ch.sh * DK * DV + col0 + n32;
#pragma unroll
    for (int m = 0; m < NM; ++m)
#pragma unroll
      for (int e = 0; e < 16; ++e) so[true_row(m, e, g2) * DV] = st[m][e];
  }
  if (args.log_decay != nullptr && ch.cb == 0 && col0 == 0 && lane == 0)
    args.log_decay[ch.sh] = log_decay;
}

template <int DK, int DV>
__device__ __forceinline__ void operator_wave(const ScanArgs& args, const Chain& ch,
                                              unsigned char* smem, int lane, int col0, int wslot) {
  using LP = Lds<DK>;
  constexpr int NU = DK / 16;
  constexpr int NM = DK / 32;
  const int g2 = lane >> 5, n32 = lane & 31;
  const u16* fWh = reinterpret_cast<const u16*>(smem + LP::O_WH);
  const u16* fWl = reinterpret_cast<const u16*>(smem + LP::O_WL);

  // operator columns col0 .. col0 + 31, all d_k rows (order rho); P_hat = I
  f32x16 st[NM];
#pragma unroll
  for (int m = 0; m < NM; ++m)
#pragma unroll
    for (int e = 0; e < 16; ++e) st[m][e] = (true_row(m, e, g2) == col0 + n32) ? 1.f : 0.f;

  for (int it = -2; it < ch.nc; ++it) {
    const int c = it;
    const bool active = c >= 0;
    bf16x8 xh[4], xl[4];
    if (active) {
      // -X = (-W) P0 in three passes (W hi + lo, P0 hi + lo)
      bf16x8 ph[NU], pl[NU];
#pragma unroll
      for (int u = 0; u < NU; ++u) split_of(st[u >> 1], u & 1, ph[u], pl[u]);
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        f32x16 acc = zero16();
#pragma unroll
        for (int u = 0; u < NU; ++u) {
          const bf16x8 wh = ldf(fWh, t * NU + u, lane);
          acc = mma32(wh, ph[u], acc);
          acc = mma32(wh, pl[u], acc);
          acc = mma32(ldf(fWl, t * NU + u, lane), ph[u], acc);
        }
        split_of(acc, 0, xh[2 * t], xl[2 * t]);
        split_of(acc, 1, xh[2 * t + 1], xl[2 * t + 1]);
      }
    }
    lds_barrier();
    if (active) {
      // P <- P0 - K^T X = P0 + K^T (-X) (K exact, X hi + lo)
      const u16* fKt =
          reinterpret_cast<const u16*>(smem + LP::O_KT + (c & 1) * LP::NKT * LP::FB);
#pragma unroll
      for (int m = 0; m < NM; ++m) {
        f32x16 acc = st[m];
#pragma unroll
        for (int s = 0; s < 4; ++s) {
          const bf16x8 a = ldf(fKt, m * 4 + s, lane);
          acc = mma32(a, xh[s], acc);
          acc = mma32(a, xl[s], acc);
        }
        st[m] = acc;
      }
    }
    if (it + 1 >= 0 && it + 1 < ch.nc) emit_w<DK>(ch, smem, lane, (it + 1) & 1, w_tile(wslot));
    lds_barrier();
  }

  float* po = args.P_hat + ch.sh * DK * DK + col0 + n32;
#pragma unroll
  for (int m = 0; m < NM; ++m)
#pragma unroll
    for (int e = 0; e < 16; ++e) po[true_row(m, e, g2) * DK] = st[m][e];
}

// every wave of the workgroup runs the same number of iterations and barriers;
// a consumer slot without columns still forms its share of W
template <int DK, int DV>
__device__ __forceinline__ void idle_wave(const Chain& ch, unsigned char* smem, int lane,
                                          int wslot, int xb) {
  for (int it = -2; it < ch.nc; ++it) {
    lds_barrier();
    pass_barriers(ch, it, xb);
    if (it + 1 >= 0 && it + 1 < ch.nc) emit_w<DK>(ch, smem, lane, (it + 1) & 1, w_tile(wslot));
    lds_barrier();
  }
}

// FUSED: mode 2, composition with seams (no operator columns)
template <int DK, int DV, bool FUSED>
__global__ __launch_bounds__(kThreads, 1) void scan_bf16_kernel(ScanArgs args) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int lane = tid & 63;

  Chain ch;
  ch.with_op = args.n_roles == 2;
  constexpr int NP = DK / NCOL, NS = DV / NCOL;
  const int n_cb = ch.with_op ? ((NP > NS) ? NP : NS) : (DV + 2 * NCOL - 1) / (2 * NCOL);
  // Workgroups are dealt to the 8 XCDs round-robin.  A unit is every
  // workgroup that reads one q/k head's tokens: the n_cb column blocks of each
  // of the group's v-head chains (chains G u .. G u + G - 1, G = h_v / h_qk).
  // A unit's workgroups are numbered to land on one XCD back to back, so they
  // share its L2 for q and k; units past the last full group of 8 keep linear
  // order.
  const int n_chains = static_cast<int>(gridDim.x) / n_cb;
  const int G = args.group;
  const int U = G * n_cb;
  const int full = (n_chains / G / 8) * 8 * U;
  int chain, cb;
  if (static_cast<int>(blockIdx.x) < full) {
    const int slot = blockIdx.x / 8;
    const int within = slot % U;
    chain = ((slot / U) * 8 + blockIdx.x % 8) * G + within / n_cb;
    cb = within % n_cb;
  } else {
    const int b = blockIdx.x - full;
    chain = full / n_cb + b / n_cb;
    cb = b % n_cb;
  }
  const int rank = chain / args.h_v;
  ch.h = chain % args.h_v;
  ch.cb = cb;
  int lo, hi;
  ch.batched = args.mode == 1 && args.w <= C;
  ch.w = args.w;
  ch.n_tok = args.n_tokens;
  ch.tok_start = args.tok_start;
  ch.tok_len = args.tok_len;
  ch.e0 = 0;
  ch.ids = nullptr;
  if (FUSED) {
    // one (request, head): the request's listed segments, one seam each
    const int r = segment_of_rank(args, rank);
    ch.batched = true;
    ch.ids = args.seg_ids;
    ch.e0 = args.req_offsets[r];
    ch.seg = r;
    lo = hi = 0;
  } else if (args.mode == 0) {
    ch.seg = segment_of_rank(args, rank);
    lo = args.cu_seqlens[ch.seg];
    hi = args.cu_seqlens[ch.seg + 1];
  } else if (ch.batched) {
    ch.e0 = rank * args.group_e;
    ch.seg = ch.e0;
    lo = hi = 0;
  } else {
    ch.seg = rank;
    lo = args.tok_start[ch.seg];
    const int len = args.tok_len[ch.seg];
    hi = lo + ((len < args.w) ? len : args.w);
  }
  lo = (lo < 0) ? 0 : ((lo > args.n_tokens) ? args.n_tokens : lo);
  hi = (hi < lo) ? lo : ((hi > args.n_tokens) ? args.n_tokens : hi);
  ch.lo = lo;
  ch.hi = hi;
  if (FUSED) {
    ch.nc = args.req_offsets[ch.seg + 1] - ch.e0;
  } else if (ch.batched) {
    const int e1 = ch.e0 + args.group_e;
    ch.nc = ((e1 < args.n_entries) ? e1 : args.n_entries) - ch.e0;
  } else {
    ch.nc = (hi - lo + C - 1) / C;
  }
  ch.hk = ch.h / args.group;
  ch.sh = static_cast<long>(ch.seg) * args.h_v + ch.h;
  ch.qk_stride = static_cast<long>(args.h_qk) * DK;
  ch.v_stride = static_cast<long>(args.h_v) * DV;
  ch.pre_t = ch.pre_n = ch.pre_id = 0;
  ch.pre_ld = 0.f;
  if (ch.batched && lane < ch.nc) {
    ch.pre_t = entry_start(ch, lane);
    ch.pre_n = entry_len(ch, lane, ch.pre_t);
    ch.pre_id = entry_of(ch, lane);
    if (FUSED) ch.pre_ld = args.pool_ld[static_cast<long>(ch.pre_id) * args.h_v + ch.h];
  }
  ch.need_state = ch.with_op ? (cb * NCOL < DV) : true;
  ch.need_op = ch.with_op && (cb * NCOL < DK);

  if (wave < 4) {
    int col0;
    bool state_role;
    if (ch.with_op) {
      state_role = wave < 2;
      col0 = cb * NCOL + 32 * (wave & 1);
    } else {
      state_role = true;
      col0 = cb * 2 * NCOL + 32 * wave;
    }
    if (state_role && col0 < DV)
      state_wave<DK, DV, FUSED>(args, ch, smem, lane, col0, wave);
    else if (!state_role && ch.need_op)
      operator_wave<DK, DV>(args, ch, smem, lane, col0, wave);
    else
      idle_wave<DK, DV>(ch, smem, lane, wave, compose_barriers<DK>(args));
  } else if (wave == 4) {
    inverse_wave<DK, DV, FUSED>(args, ch, smem, lane);
  } else if (wave == 5) {
    producer_qk_wave<DK, DV, FUSED>(args, ch, smem, lane);
  } else if (wave == 6) {
    producer_kt_wave<DK, DV, 0, FUSED>(args, ch, smem, lane);
  } else {
    producer_kt_wave<DK, DV, 1, FUSED>(args, ch, smem, lane);
  }
}

template <int DK, int DV, bool FUSED = false>
hipError_t launch_t(const ScanArgs& a, int n_items, hipStream_t s) {
  constexpr int bytes = Lds<DK>::TOTAL;
  // one-time (thread-safe static initialisation) opt-in to more than 64 KiB of LDS
  static const hipError_t attr = hipFuncSetAttribute(
      reinterpret_cast<const void*>(&scan_bf16_kernel<DK, DV, FUSED>),
      hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL((scan_bf16_kernel<DK, DV, FUSED>), dim3(n_items), dim3(kThreads), bytes, s,
                     a);
  return hipGetLastError();
}

}  // namespace

int scan_bf16_items_per_head(int d_k, int d_v, int with_operator) {
  const int ns = d_v / NCOL, np = d_k / NCOL;
  if (!with_operator) return (d_v + 2 * NCOL - 1) / (2 * NCOL);
  return (np > ns) ? np : ns;
}

hipError_t launch_seam_compose_fused(const ScanArgs& a, int d_k, int d_v, int n_req,
                                     hipStream_t s) {
  // no operator columns: one workgroup carries every state column of a head
  const int64_t n_items = static_cast<int64_t>(n_req) * a.h_v * scan_bf16_items_per_head(d_k, d_v, 0);
  if (n_items <= 0) return hipSuccess;
  if (n_items > 0x7fffffff || a.n_roles != 1 || a.mode != 2 || a.w > C) return hipErrorInvalidValue;
  const int n = static_cast<int>(n_items);
  if (d_k == 64 && d_v == 64) return launch_t<64, 64, true>(a, n, s);
  if (d_k == 64 && d_v == 128) return launch_t<64, 128, true>(a, n, s);
  if (d_k == 128 && d_v == 64) return launch_t<128, 64, true>(a, n, s);
  return launch_t<128, 128, true>(a, n, s);
}

hipError_t launch_scan_bf16(const ScanArgs& a, int d_k, int d_v, int n_items, hipStream_t s) {
  if (n_items <= 0) return hipSuccess;
  if (d_k == 64 && d_v == 64) return launch_t<64, 64>(a, n_items, s);
  if (d_k == 64 && d_v == 128) return launch_t<64, 128>(a, n_items, s);
  if (d_k == 128 && d_v == 64) return launch_t<128, 64>(a, n_items, s);
  return launch_t<128, 128>(a, n_items, s);
}

}  // namespace hypic
