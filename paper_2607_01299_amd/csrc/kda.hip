// Segment build and seam rescan for the KDA row of Tab. 1 on gfx950: the delta
// rule with a per-channel gate,
//   S_t = (I - beta_t k_t k_t^T) diag(exp(g_t)) S_{t-1} + beta_t k_t v_t^T,
//   o_t = S_t^T q_t                      (Eq. (2); the token reads its own write),
// and its Tab. 3 operator T_C = prod_t (I - beta_t k_t k_t^T) diag(exp(g_t)),
// stored as T_C = exp(log_decay) P_hat.  log_decay is the sum over the
// segment's 64-token chunks of each chunk's largest per-channel gate sum; it
// keeps P_hat within float32 range and leaves the tuple in the format that the
// GDN composition (Eq. (6)) reads.
//
// Chunked form (C = 64 tokens, incoming state S0, B = per-channel prefix sum
// of the gate inside the chunk, inclusive).  With nu_t the corrected value
// beta_t (v_t - S'_t^T k_t) of token t (S'_t the gated state before its
// write), unrolling the recurrence over the chunk gives
//   G_ti = sum_c k_tc k_ic exp(B_tc - B_ic)              (i < t)
//   N    = (I + diag(beta) G)^-1 diag(beta) (V - (K . exp(B)) S0)
//   O    = (Q . exp(B)) S0 + A N,  A_ti = sum_c q_tc k_ic exp(B_tc - B_ic) (i <= t)
//   S   <- exp(B_last) . S0 + (K . exp(B_last - B))^T N.
// The operator is the same update of d_k extra state columns with V = 0 from
// S0 = I, rescaled by exp(-m) after each chunk (m = the chunk's largest channel
// gate sum, accumulated into log_decay).
//
// Gates inside G and A are referred to 16-token tiles as in the diagonal family
// (family.hip): K and Q are stored once as K . exp(B - Bbar) (query side) and
// K . exp(Bbar - B) (key side), Bbar the cumulative gate before the token's
// tile, and each tile pair is completed by the channel vector
// exp(Bbar_tq - Bbar_tk) <= 1.  Every channel's gate sum over 16 consecutive
// tokens must stay above about -80 (float32 range), as for the diagonal family.
// With bf16 operands the state columns form each decayed key
// exp(B_last - B_t) k_t with one exponential; otherwise (float32 state columns,
// operator columns) it is the key side times the decay from its tile to the
// chunk end, which can lose key contributions below about exp(-7) of the
// chunk's largest where a channel decays by more than 87 within one chunk.
//
// Organisation: one 8-wave workgroup runs one (segment or seam entry, v-head,
// 64-column block) chain over its chunks; each wave holds 16 columns x half the
// d_k rows of the block's state in registers.  State columns use the input
// precision on the matrix cores (bf16 operands with float32 accumulation for
// bf16 inputs), except the intra-chunk scores G and A, whose tile-referred
// gate-scaled operands are kept as bf16 hi + lo pairs (three passes): a score
// q_t . k_i that nearly cancels would otherwise be dominated by one bf16
// rounding of its operands.  Operator columns always keep float32 operands in
// LDS and run their products as three-pass split bf16, so that the
// normalised operator does not pick up a one-pass bf16 rounding per chunk.  The 64 x 64 inverse
// runs in float32: the four diagonal
// 16 x 16 blocks by forward substitution (one lane per column), then block row
// by block row, T_ij = -X_i sum_k L_ik T_kj, on the float32 matrix cores.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "frag_common.hpp"
#include "kda.hpp"
#include "mfma.hpp"

namespace hypic {

namespace {

constexpr int kKT = 512;  // threads of a workgroup (8 waves)
constexpr int KC = 64;    // tokens per chunk
constexpr int KNC = 64;   // columns per workgroup
constexpr int NCG = KNC / 16;  // column groups of 16 (waves per row group)
constexpr int LTD = KC + 4;    // row stride of the float32 64 x 64 matrices

template <typename ST, int DK, bool OP>
struct KdaLds {
  static constexpr int PAD = (sizeof(ST) == 2) ? 8 : 4;
  static constexpr int LDK = DK + PAD;  // token-major rows of Q and K
  static constexpr int LDV = KC + PAD;  // V^T rows, and rows of the channel-major keys
  // K . exp(B - Bbar) (G and Y), then Q . exp(B - Bbar) (outputs)
  alignas(16) ST qk[KC * LDK];
  alignas(16) ST kk[KC * LDK];    // K, then K . exp(Bbar - B)
  alignas(16) float lt[KC * LTD]; // diag(beta) G (strict lower) -> its inverse T (in place) -> A
  // state columns only: V^T of the block's columns (read in stage 3 only;
  // with bf16 operands the A tiles of stage 7 reuse it).  With bf16 operands
  // (PRE) also (K . exp(B_last - B))^T channel-major (float32 operands form it
  // on the fly: no LDS left for it), and (SPL) the bf16 remainders of the
  // query-side and key-side operands, so that the scores G and A run on hi + lo
  // operands: a q_t . k_i that nearly cancels keeps its float32 accuracy
  static constexpr bool PRE = !OP && sizeof(ST) == 2;
  static constexpr bool SPL = PRE;
  alignas(16) ST vt[OP ? 1 : KNC * LDV];
  alignas(16) ST kdt[PRE ? DK * LDV : 1];
  alignas(16) ST qlo[SPL ? KC * LDK : 8];  // remainders of qk
  alignas(16) ST klo[SPL ? KC * LDK : 8];  // remainders of kk
  // the off-diagonal 16 x 16 blocks of the inverse, kept apart from L (TB:
  // bf16 state columns and operator columns; float32 state columns write them
  // into lt, which takes a second barrier per block row)
  static constexpr bool TB = PRE || OP;
  static constexpr int TBS = SPL ? 16 : 20;  // row stride of a block
  alignas(16) float tb[TB ? 6 * 16 * TBS : 4];
  // bf16 state columns (NS): N republished into a second fragment buffer and
  // A formed into vt (free after stage 3), in one stage
  static constexpr bool NS = PRE;
  alignas(16) Frag<ST> rf2[NS ? NCG * 2 * 64 : 1];
  // S0 as B fragments: column group, 32-row block, lane
  alignas(16) Frag<ST> s0f[NCG][DK / 32][64];
  alignas(16) Frag<ST> rf[NCG][2][64];         // diag(beta) R, then N, as B fragments over tokens
  // per (token part, channel) gate totals: part pt of channel c at pt d_k + c
  alignas(16) float part[kKT];
  alignas(16) float fx[6 * DK];     // exp(Bbar_tq - Bbar_tk), tk < tq
  alignas(16) float hx[4 * DK];     // exp(Bbar) per tile
  alignas(16) float gl[4 * DK];     // exp(B_last - Bbar) per tile
  alignas(16) float lx[DK];         // exp(B_last)
  alignas(16) float beta[KC];
  alignas(16) float bmax[2];        // per-wave maxima of the channel totals
};

__device__ __forceinline__ int pair_ix(int tq, int tk) { return tq * (tq - 1) / 2 + tk; }

// One 32-deep product block.  Operator columns (SPLIT) run their float32
// operands as three bf16 passes (hi hi + hi lo + lo hi: about 2^-16 relative
// per product, against 2^-9 for one bf16 pass), a sixth of the float32
// matrix-core time; every other product runs in its operand type.
template <bool SPLIT>
__device__ __forceinline__ f32x4 mmk(const Frag<float>& a, const Frag<float>& b, f32x4 c) {
  if constexpr (SPLIT) {
    mma_blk<P_SPLIT>(c, a.x, b.x);
    return c;
  } else {
    return mma(a, b, c);
  }
}
template <bool SPLIT>
__device__ __forceinline__ f32x4 mmk(const Frag<u16>& a, const Frag<u16>& b, f32x4 c) {
  return mma(a, b, c);
}

// A-operand fragment of a float32 matrix in the operand type ST
template <typename ST>
__device__ __forceinline__ Frag<ST> frag_f32(const float* M, int ld, int row, int kb, int g) {
  if constexpr (sizeof(ST) == 4) {
    return frag_row(M, ld, row, kb, g);
  } else {
    const float4 lo = *reinterpret_cast<const float4*>(M + row * ld + kb + 4 * g);
    const float4 hi = *reinterpret_cast<const float4*>(M + row * ld + kb + 16 + 4 * g);
    Frag<ST> f;
    f.set(0, lo.x); f.set(1, lo.y); f.set(2, lo.z); f.set(3, lo.w);
    f.set(4, hi.x); f.set(5, hi.y); f.set(6, hi.z); f.set(7, hi.w);
    return f;
  }
}

// A-operand fragment of (K . exp(B_last - B))^T: row = channel c, k = tokens
// kb .. kb + 31 of the token-major key-side K (tiles 2 kb/32 and 2 kb/32 + 1)
template <typename ST, int DK>
__device__ __forceinline__ Frag<ST> frag_kdec(const ST* kk, int ldk, int c, int kb, int g,
                                              const float* gl) {
  const float g0 = gl[(kb >> 4) * DK + c], g1 = gl[((kb >> 4) + 1) * DK + c];
  Frag<ST> f;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int t = kb + kap(g, j);
    f.set(j, ldv(kk + t * ldk + c) * ((j < 4) ? g0 : g1));
  }
  return f;
}

// acc += A B over 16 k (float32 matrix cores): 16 x 16 row-major float32
// blocks at A (row stride lda) and B (row stride ldb)
__device__ __forceinline__ f32x4 mm16p(const float* A, int lda, const float* B, int ldb,
                                       f32x4 acc, int g, int ln) {
  const float4 a = *reinterpret_cast<const float4*>(A + ln * lda + 4 * g);
  const float av[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
  for (int j = 0; j < 4; ++j)
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av[j], B[(4 * g + j) * ldb + ln], acc, 0, 0, 0);
  return acc;
}

// A-operand fragment of the inverse T (row tile mt, k tokens 32 kt .. +31)
// when its off-diagonal blocks are kept apart: the diagonal block from lt, the
// blocks left of it from tb, zero right of it
template <typename ST, int TBS>
__device__ __forceinline__ Frag<ST> frag_T(const float* lt, const float* tb, int mt, int kt,
                                           int g, int ln) {
  Frag<ST> f;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int tk = 2 * kt + h;
    float4 v = {0.f, 0.f, 0.f, 0.f};
    if (tk == mt)
      v = *reinterpret_cast<const float4*>(lt + (16 * mt + ln) * LTD + 16 * tk + 4 * g);
    else if (tk < mt)
      v = *reinterpret_cast<const float4*>(tb + pair_ix(mt, tk) * 16 * TBS + ln * TBS + 4 * g);
    f.set(4 * h, v.x);
    f.set(4 * h + 1, v.y);
    f.set(4 * h + 2, v.z);
    f.set(4 * h + 3, v.w);
  }
  return f;
}

// One 16 x 16 score tile (query tile tq, key tile tk <= tq) over all d_k
// channels from the tile-referred operands: sum_c qk[t][c] kk[i][c], with
// the query side scaled by exp(Bbar_tq - Bbar_tk) for tk < tq.  SPL: both
// operands as hi + lo, three bf16 passes.
template <typename ST, int DK, bool OP, bool SPL>
__device__ __forceinline__ f32x4 score_tile(const ST* qk, const ST* qlo, const ST* kk,
                                            const ST* klo, const float* fx, int tq, int tk,
                                            int g, int ln) {
  constexpr int LDK = DK + ((sizeof(ST) == 2) ? 8 : 4);
  f32x4 acc = zero4();
  if constexpr (SPL) {
#pragma unroll
    for (int kb = 0; kb < DK; kb += 32) {
      const SplitFrag fa =
          (tk < tq) ? frag_row_split_scaled(qk, qlo, LDK, tq * 16 + ln, kb, g,
                                            fx + pair_ix(tq, tk) * DK)
                    : frag_row_split(qk, qlo, LDK, tq * 16 + ln, kb, g);
      acc = mma3(fa, frag_row_split(kk, klo, LDK, tk * 16 + ln, kb, g), acc);
    }
  } else {
#pragma unroll
    for (int kb = 0; kb < DK; kb += 32) {
      Frag<ST> fa;
      if (tk < tq)
        fa = frag_row_scaled(qk, LDK, tq * 16 + ln, kb, g, fx + pair_ix(tq, tk) * DK);
      else
        fa = frag_row(qk, LDK, tq * 16 + ln, kb, g);
      acc = mmk<OP>(fa, frag_row(kk, LDK, tk * 16 + ln, kb, g), acc);
    }
  }
  return acc;
}

// A-operand fragment of the query-side operand times exp(Bbar) of its tile
// (K . exp(B) in stage 3, Q . exp(B) in stage 8); SPL: from hi + lo, rounded once
template <typename ST, bool SPL>
__device__ __forceinline__ Frag<ST> frag_decayed(const ST* qk, const ST* qlo, int ld, int row,
                                                 int kb, int g, const float* s) {
  if constexpr (SPL)
    return frag_row_sum_scaled(qk, qlo, ld, row, kb, g, s);
  else
    return frag_row_scaled(qk, ld, row, kb, g, s);
}

__device__ __forceinline__ int kda_segment_of_rank(const KdaArgs& a, int rank) {
  return a.n_inline > 0 ? static_cast<int>(a.order_inline[rank]) : a.order[rank];
}

// TIN: storage type of q, k, v; ST: operand type; OP: operator columns
template <typename TIN, typename ST, bool OP, int DK, int DV>
__global__ __launch_bounds__(kKT) void kda_scan_kernel(KdaArgs args) {
  using L = KdaLds<ST, DK, OP>;
  constexpr int LDK = L::LDK, LDV = L::LDV;
  constexpr int NRG = 8 / NCG;                            // row groups
  constexpr int VEC = 16 / static_cast<int>(sizeof(TIN)); // elements per 16-byte load
  constexpr int NQ = KC * DK / (VEC * kKT);               // 16-byte loads of Q (and K)
  constexpr int NV = (KC * KNC + VEC * kKT - 1) / (VEC * kKT);
  constexpr int NMH = DK / (16 * NRG);                    // state row tiles per wave
  constexpr int NPT = kKT / DK;                           // gate threads per channel
  constexpr int TPT = KC / NPT;                           // tokens per gate thread
  static_assert(NQ >= 1 && NMH % 2 == 0 && NRG == 2, "tile split");
  static_assert(TPT == 16 || TPT == 8, "gate split");
  static_assert(sizeof(L) <= 160 * 1024, "LDS budget");
  constexpr bool PRE = L::PRE, TB = L::TB, NS = L::NS, SPL = L::SPL;
  constexpr int TBS = L::TBS;
  static_assert(KNC == KC, "A reuses the V^T array");

  extern __shared__ __align__(16) unsigned char smem_raw[];
  L& sm = *reinterpret_cast<L*>(smem_raw);
  ST* const la = sm.vt;  // A (NS): stages 7-8, after V^T's last read in stage 3

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63;
  const int g = lane >> 4, ln = lane & 15;
  const int cg = wave % NCG, rgrp = wave / NCG;

  // ---- work item: XCD-aware numbering of the column blocks of one chain ----
  constexpr int n_cb = OP ? DK / KNC : DV / KNC;
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
  const int hk = h / args.group;
  int seg, lo, hi;
  if (args.mode == 0) {
    seg = kda_segment_of_rank(args, rank);
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

  const long qk_stride = static_cast<long>(args.h_qk) * DK;
  const long v_stride = static_cast<long>(args.h_v) * DV;
  const TIN* qg = static_cast<const TIN*>(args.q) + hk * DK;
  const TIN* kg = static_cast<const TIN*>(args.k) + hk * DK;
  const TIN* vg = static_cast<const TIN*>(args.v) + h * DV + cb * KNC;
  const long sh = static_cast<long>(seg) * args.h_v + h;
  const int col16 = 16 * cg;
  const int col = cb * KNC + col16;      // column of the state (or of the operator)
  const int row0 = rgrp * (DK / NRG);    // this wave's first state row

  // ---- state: rows row0 .. row0 + DK/2 - 1, columns col .. col + 15 ----
  f32x4 st[NMH];
#pragma unroll
  for (int mt = 0; mt < NMH; ++mt) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = row0 + mt * 16 + 4 * g + i;
      if constexpr (OP)
        st[mt][i] = (r == col + ln) ? 1.f : 0.f;
      else
        st[mt][i] = (args.mode == 1) ? args.S_in[(sh * DK + r) * DV + col + ln] : 0.f;
    }
  }

  // the upper 16 x 16 tiles of L read with its rows, (0, 1) and (2, 3), stay
  // zero (those of A in vt are cleared per chunk, in stage 7)
  {
    const int t = tid >> 8, e = tid & 255;
    sm.lt[(32 * t + (e >> 4)) * LTD + 32 * t + 16 + (e & 15)] = 0.f;
  }

  // ---- register prefetch of one chunk ----
  uint4 rq[OP ? 1 : NQ], rk[NQ], rv[OP ? 1 : NV];
  float rg[TPT], rb = 0.f;
  const int pc = tid % DK, pt = tid / DK;  // gate thread: channel, token part
  auto prefetch = [&](int c0, int n) __attribute__((always_inline)) {
    constexpr int SZ = static_cast<int>(sizeof(TIN));
    const auto rsk = rsrc(kg + static_cast<long>(c0) * qk_stride, n * qk_stride * SZ);
#pragma unroll
    for (int u = 0; u < NQ; ++u) {
      const int idx = u * kKT + tid;
      const int r = idx / (DK / VEC), cv = idx % (DK / VEC);
      rk[u] = bload16(rsk, static_cast<int>((r * qk_stride + cv * VEC) * SZ));
    }
    if constexpr (!OP) {
      const auto rsq = rsrc(qg + static_cast<long>(c0) * qk_stride, n * qk_stride * SZ);
      const auto rsv = rsrc(vg + static_cast<long>(c0) * v_stride, n * v_stride * SZ);
#pragma unroll
      for (int u = 0; u < NQ; ++u) {
        const int idx = u * kKT + tid;
        const int r = idx / (DK / VEC), cv = idx % (DK / VEC);
        rq[u] = bload16(rsq, static_cast<int>((r * qk_stride + cv * VEC) * SZ));
      }
#pragma unroll
      for (int u = 0; u < NV; ++u) {
        const int idx = u * kKT + tid;
        const int r = idx / (KNC / VEC), cv = idx % (KNC / VEC);
        rv[u] = bload16(rsv, static_cast<int>((r * v_stride + cv * VEC) * SZ));
      }
    }
    const long gs = static_cast<long>(args.h_v) * DK;
    const auto rsg = rsrc(args.gate + static_cast<long>(c0) * gs, n * gs * 4);
#pragma unroll
    for (int j = 0; j < TPT; ++j)
      rg[j] = bload4(rsg, static_cast<int>(((TPT * pt + j) * gs + h * DK + pc) * 4));
    const auto rsb = rsrc(args.beta + static_cast<long>(c0) * args.h_v, n * args.h_v * 4);
    rb = bload4(rsb, (lane * args.h_v + h) * 4);
  };
  if (lo < hi) prefetch(lo, (hi - lo < KC) ? hi - lo : KC);
  float ld_acc = 0.f;

  const int tid_in = tid;
  for (int c0 = lo; c0 < hi; c0 += KC) {
    // an opaque copy of the thread index keeps the compiler from hoisting the
    // loop-invariant LDS addresses out of the chunk loop (they would not all
    // fit in registers and were spilled to scratch); they are cheap to
    // recompute per chunk
    int tid_v = tid_in;
    asm volatile("" : "+v"(tid_v));
    const int tid = tid_v;
    const int lane = tid & 63;
    const int g = lane >> 4, ln = lane & 15;
    const int pc = tid % DK, pt = tid / DK;
    const int n = (hi - c0 < KC) ? hi - c0 : KC;
    lds_barrier();  // the previous chunk is done with every LDS buffer

    // ---- 1: publish S0; stage K (token-major) and V^T; gate prefix; beta ----
#pragma unroll
    for (int kl = 0; kl < NMH / 2; ++kl) {
      Frag<ST> f;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        f.set(i, st[2 * kl][i]);
        f.set(4 + i, st[2 * kl + 1][i]);
      }
      sm.s0f[cg][rgrp * (NMH / 2) + kl][lane] = f;
    }
#pragma unroll
    for (int u = 0; u < NQ; ++u) {
      const int idx = u * kKT + tid;
      const int r = idx / (DK / VEC), cv = idx % (DK / VEC);
#pragma unroll
      for (int e = 0; e < VEC; ++e)
        stv(sm.kk + r * LDK + cv * VEC + e, elem(rk[u], e, static_cast<const TIN*>(nullptr)));
    }
    if constexpr (!OP) {
#pragma unroll
      for (int u = 0; u < NV; ++u) {
        const int idx = u * kKT + tid;
        const int r = idx / (KNC / VEC), cv = idx % (KNC / VEC);
        if (r < KC) {
#pragma unroll
          for (int e = 0; e < VEC; ++e)
            stv(sm.vt + (cv * VEC + e) * LDV + r, elem(rv[u], e, static_cast<const TIN*>(nullptr)));
        }
      }
    }
    float pre[TPT];
    {
      float run = 0.f;
#pragma unroll
      for (int j = 0; j < TPT; ++j) {
        run += rg[j];
        pre[j] = run;
      }
      sm.part[pt * DK + pc] = run;  // a 16-token tile, or half of one (d_k = 64)
    }
    if (tid < KC) sm.beta[tid] = rb;
    lds_barrier();

    // ---- 2: thread (channel pc, part pt): tile-referred K, tile factors ----
    float hb[4], b_last = 0.f;  // Bbar of the four tiles of channel pc
    {
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        if constexpr (TPT == 16) {
          hb[p] = b_last;
          b_last += sm.part[p * DK + pc];
        } else {
          hb[p] = b_last;
          b_last += sm.part[(2 * p) * DK + pc] + sm.part[(2 * p + 1) * DK + pc];
        }
      }
      const int tile = (TPT == 16) ? pt : pt / 2;
      // within-tile prefix of this thread's first token's predecessors
      float base = 0.f;
      if constexpr (TPT == 8) base = (pt & 1) ? sm.part[(pt - 1) * DK + pc] : 0.f;
      const int t0 = TPT * pt;
      const float hbt = hb[tile];
#pragma unroll
      for (int j8 = 0; j8 < TPT; j8 += 8) {
        float kd[8];
#pragma unroll
        for (int jj = 0; jj < 8; ++jj) {
          const int j = j8 + jj, t = t0 + j;
          const float rel = base + pre[j];  // B_t - Bbar of the token's tile, <= 0
          const float kv = ldv(sm.kk + t * LDK + pc);
          const float qs = kv * __expf(rel), ks = kv * __expf(-rel);
          stv(sm.qk + t * LDK + pc, qs);
          stv(sm.kk + t * LDK + pc, ks);
          if constexpr (SPL) {
            stv(sm.qlo + t * LDK + pc, qs - bf16_round(qs));
            stv(sm.klo + t * LDK + pc, ks - bf16_round(ks));
          }
          if constexpr (PRE) kd[jj] = kv * __expf(b_last - hbt - rel);  // K exp(B_last - B_t)
        }
        if constexpr (PRE) st8(sm.kdt + pc * LDV + t0 + j8, kd);
      }
      if (TPT == 16 || (pt & 1) == 0) {
#pragma unroll
        for (int tk = 0; tk < 3; ++tk)
          if (tk < tile) sm.fx[pair_ix(tile, tk) * DK + pc] = __expf(hb[tile] - hb[tk]);
        sm.hx[tile * DK + pc] = __expf(hb[tile]);
        sm.gl[tile * DK + pc] = __expf(b_last - hb[tile]);
      }
      if (pt == 0) {
        sm.lx[pc] = __expf(b_last);
        float mx = b_last;
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off, 64));
        if (lane == 0) sm.bmax[wave] = mx;
      }
    }
    lds_barrier();

    // ---- 3: diag(beta) G (strict lower tiles) and diag(beta) R, R = V - Y,
    // Y = (K . exp(B)) S0 ----
    for (int tile = wave; tile < 10; tile += 8) {
      const int tq = (tile < 1) ? 0 : ((tile < 3) ? 1 : ((tile < 6) ? 2 : 3));
      const int tk = tile - tq * (tq + 1) / 2;
      const f32x4 acc = score_tile<ST, DK, OP, SPL>(sm.qk, sm.qlo, sm.kk, sm.klo, sm.fx, tq,
                                                    tk, g, ln);
      const int key = tk * 16 + ln;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int t = tq * 16 + 4 * g + i;
        sm.lt[t * LTD + key] = (key < t) ? acc[i] * sm.beta[t] : 0.f;
      }
    }
    {
      f32x4 r2[2];
#pragma unroll
      for (int mh = 0; mh < 2; ++mh) {
        const int mt = 2 * rgrp + mh;  // token tile
        f32x4 acc = zero4();
#pragma unroll
        for (int kt = 0; kt < DK / 32; ++kt)
          acc = mmk<OP>(frag_decayed<ST, SPL>(sm.qk, sm.qlo, LDK, mt * 16 + ln, 32 * kt, g,
                                              sm.hx + mt * DK),
                        sm.s0f[cg][kt][lane], acc);
        const float4 bt = *reinterpret_cast<const float4*>(sm.beta + mt * 16 + 4 * g);
        float vv[4] = {0.f, 0.f, 0.f, 0.f};
        if constexpr (!OP) {
#pragma unroll
          for (int i = 0; i < 4; ++i) vv[i] = ldv(sm.vt + (col16 + ln) * LDV + mt * 16 + 4 * g + i);
        }
        r2[mh][0] = bt.x * (vv[0] - acc[0]);
        r2[mh][1] = bt.y * (vv[1] - acc[1]);
        r2[mh][2] = bt.z * (vv[2] - acc[2]);
        r2[mh][3] = bt.w * (vv[3] - acc[3]);
      }
      Frag<ST> f;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        f.set(i, r2[0][i]);
        f.set(4 + i, r2[1][i]);
      }
      sm.rf[cg][rgrp][lane] = f;
    }
    lds_barrier();

    // ---- 4: inverses of the diagonal 16 x 16 blocks (wave 0, lane 16 b + j:
    // column j of block b); stage Q; prefetch the next chunk ----
    if (wave == 0) {
      const int b = lane >> 4, jc = lane & 15;
      const float* Lb = sm.lt + (16 * b) * LTD + 16 * b;
      float x[16];
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        float s = (i == jc) ? 1.f : 0.f;
#pragma unroll
        for (int k2 = 0; k2 < i; ++k2) s -= Lb[i * LTD + k2] * x[k2];
        x[i] = s;
      }
#pragma unroll
      for (int i = 0; i < 16; ++i) sm.lt[(16 * b + i) * LTD + 16 * b + jc] = x[i];
    }
    if constexpr (!OP) {
#pragma unroll
      for (int u = 0; u < NQ; ++u) {
        const int idx = u * kKT + tid;
        const int r = idx / (DK / VEC), cv = idx % (DK / VEC);
#pragma unroll
        for (int e = 0; e < VEC; ++e)
          stv(sm.qk + r * LDK + cv * VEC + e, elem(rq[u], e, static_cast<const TIN*>(nullptr)));
      }
    }
    prefetch(c0 + KC, (hi - c0 - KC < KC) ? hi - c0 - KC : KC);
    lds_barrier();

    // ---- 5: block rows of the inverse, T_ij = -X_i sum_{k=j}^{i-1} L_ik T_kj;
    // the query-side Q . exp(B - Bbar) meanwhile ----
    if constexpr (!OP) {
      float base = 0.f;
      if constexpr (TPT == 8) base = (pt & 1) ? sm.part[(pt - 1) * DK + pc] : 0.f;
#pragma unroll
      for (int j = 0; j < TPT; ++j) {
        const int t = TPT * pt + j;
        ST* qp = sm.qk + t * LDK + pc;
        const float qv = ldv(qp) * __expf(base + pre[j]);
        stv(qp, qv);
        if constexpr (SPL) stv(sm.qlo + t * LDK + pc, qv - bf16_round(qv));
      }
    }
#pragma unroll
    for (int bi = 1; bi < 4; ++bi) {
      f32x4 tij = zero4();
      if (wave < bi) {
        const int bj = wave;
        f32x4 m = zero4();
        for (int bk = bj; bk < bi; ++bk) {
          // T_kj: X_j on the diagonal of lt, else the block row bk written before
          const float* bp = sm.lt + (16 * bk) * LTD + 16 * bj;
          int ldb = LTD;
          if (TB && bk > bj) {
            bp = sm.tb + pair_ix(bk, bj) * 16 * TBS;
            ldb = TBS;
          }
          m = mm16p(sm.lt + (16 * bi) * LTD + 16 * bk, LTD, bp, ldb, m, g, ln);
        }
        const float4 a =
            *reinterpret_cast<const float4*>(sm.lt + (16 * bi + ln) * LTD + 16 * bi + 4 * g);
        const float av[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
        for (int j = 0; j < 4; ++j)
          tij = __builtin_amdgcn_mfma_f32_16x16x4f32(av[j], m[j], tij, 0, 0, 0);
      }
      if constexpr (TB) {
        if (wave < bi) {
          float* tp = sm.tb + pair_ix(bi, wave) * 16 * TBS;
#pragma unroll
          for (int i = 0; i < 4; ++i) tp[(4 * g + i) * TBS + ln] = -tij[i];
        }
        lds_barrier();
      } else {
        lds_barrier();  // L_ij is read by this block row until here
        if (wave < bi) {
#pragma unroll
          for (int i = 0; i < 4; ++i)
            sm.lt[(16 * bi + 4 * g + i) * LTD + 16 * wave + ln] = -tij[i];
        }
        lds_barrier();
      }
    }

    // ---- 6: N = T diag(beta) R (two token tiles of this wave's columns) ----
    f32x4 nt[2];
#pragma unroll
    for (int mh = 0; mh < 2; ++mh) {
      const int mt = 2 * rgrp + mh;
      f32x4 acc = zero4();
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
        if (32 * kt < 16 * (mt + 1)) {
          Frag<ST> ft;
          if constexpr (TB)
            ft = frag_T<ST, TBS>(sm.lt, sm.tb, mt, kt, g, ln);
          else
            ft = frag_f32<ST>(sm.lt, LTD, mt * 16 + ln, 32 * kt, g);
          acc = mmk<OP>(ft, sm.rf[cg][kt][lane], acc);
        }
      nt[mh] = acc;
    }
    if constexpr (!NS) lds_barrier();  // every wave is done reading diag(beta) R
    {
      Frag<ST> f;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        f.set(i, nt[0][i]);
        f.set(4 + i, nt[1][i]);
      }
      if constexpr (NS)
        sm.rf2[(cg * 2 + rgrp) * 64 + lane] = f;
      else
        sm.rf[cg][rgrp][lane] = f;
    }
    // ---- 7: A (lower tiles, inclusive) from the query-side Q (into la with
    // NS, else into lt, whose inverse is no longer read) ----
    if constexpr (!OP) {
      for (int tile = wave; tile < 10; tile += 8) {
        const int tq = (tile < 1) ? 0 : ((tile < 3) ? 1 : ((tile < 6) ? 2 : 3));
        const int tk = tile - tq * (tq + 1) / 2;
        const f32x4 acc = score_tile<ST, DK, OP, SPL>(sm.qk, sm.qlo, sm.kk, sm.klo, sm.fx, tq,
                                                      tk, g, ln);
        const int key = tk * 16 + ln;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int t = tq * 16 + 4 * g + i;
          const float x = (key <= t) ? acc[i] : 0.f;
          if constexpr (NS)
            stv(la + t * LDV + key, x);
          else
            sm.lt[t * LTD + key] = x;
        }
      }
      if constexpr (NS) {
        // the upper tiles (0, 1) and (2, 3) read with A's rows are zero (vt
        // held V^T there)
        const int t = tid >> 8, e = tid & 255;
        stv(la + (32 * t + (e >> 4)) * LDV + 32 * t + 16 + (e & 15), 0.f);
      }
    }
    lds_barrier();

    // ---- 8: outputs O = (Q . exp(B)) S0 + A N; state update ----
    if constexpr (!OP) {
      const long orow0 = (args.mode == 0) ? static_cast<long>(c0)
                                          : static_cast<long>(seg) * args.w + (c0 - lo);
      const auto rso = rsrc(args.o ? static_cast<const TIN*>(args.o) + orow0 * v_stride : nullptr,
                            args.o ? n * v_stride * static_cast<long>(sizeof(TIN)) : 0);
      const int ocol = static_cast<int>(h * DV + col + ln);
#pragma unroll
      for (int mh = 0; mh < 2; ++mh) {
        const int mt = 2 * rgrp + mh;
        f32x4 acc = zero4();
#pragma unroll
        for (int kt = 0; kt < DK / 32; ++kt)
          acc = mmk<OP>(frag_decayed<ST, SPL>(sm.qk, sm.qlo, LDK, mt * 16 + ln, 32 * kt, g,
                                              sm.hx + mt * DK),
                        sm.s0f[cg][kt][lane], acc);
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
          if (32 * kt < 16 * (mt + 1)) {
            if constexpr (NS)
              acc = mmk<OP>(frag_row(la, LDV, mt * 16 + ln, 32 * kt, g),
                            sm.rf2[(cg * 2 + kt) * 64 + lane], acc);
            else
              acc = mmk<OP>(frag_f32<ST>(sm.lt, LTD, mt * 16 + ln, 32 * kt, g),
                            sm.rf[cg][kt][lane], acc);
          }
#pragma unroll
        for (int i = 0; i < 4; ++i)
          bstore(rso, static_cast<int>(((mt * 16 + 4 * g + i) * v_stride + ocol) * sizeof(TIN)),
                 acc[i], static_cast<TIN*>(nullptr));
      }
    }
    float scale = 1.f;
    if constexpr (OP) {
      const float m = (DK > 64) ? fmaxf(sm.bmax[0], sm.bmax[1]) : sm.bmax[0];
      scale = __expf(-m);
      ld_acc += m;
    }
#pragma unroll
    for (int mt = 0; mt < NMH; ++mt) {
      const int r = row0 + mt * 16;
      const float4 lx = *reinterpret_cast<const float4*>(sm.lx + r + 4 * g);
      f32x4 acc = st[mt];
      acc[0] *= lx.x;
      acc[1] *= lx.y;
      acc[2] *= lx.z;
      acc[3] *= lx.w;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        Frag<ST> fa;
        if constexpr (PRE)
          fa = frag_row(sm.kdt, LDV, r + ln, 32 * kt, g);
        else
          fa = frag_kdec<ST, DK>(sm.kk, LDK, r + ln, 32 * kt, g, sm.gl);
        if constexpr (NS)
          acc = mmk<OP>(fa, sm.rf2[(cg * 2 + kt) * 64 + lane], acc);
        else
          acc = mmk<OP>(fa, sm.rf[cg][kt][lane], acc);
      }
      if constexpr (OP) acc *= scale;
      st[mt] = acc;
    }
  }

  // ---- the chain's results ----
  if constexpr (OP) {
    float* po = args.P_hat + sh * DK * DK + col + ln;
#pragma unroll
    for (int mt = 0; mt < NMH; ++mt)
#pragma unroll
      for (int i = 0; i < 4; ++i) po[(row0 + mt * 16 + 4 * g + i) * DK] = st[mt][i];
    if (args.log_decay != nullptr && cb == 0 && tid == 0) args.log_decay[sh] = ld_acc;
  } else if (args.S_out != nullptr) {
    float* so = args.S_out + sh * DK * DV + col + ln;
#pragma unroll
    for (int mt = 0; mt < NMH; ++mt)
#pragma unroll
      for (int i = 0; i < 4; ++i) so[(row0 + mt * 16 + 4 * g + i) * DV] = st[mt][i];
  }
}

template <typename TIN, typename ST, bool OP, int DK, int DV>
hipError_t launch_kda_t(const KdaArgs& a, int n_items, hipStream_t s) {
  constexpr int bytes = static_cast<int>(sizeof(KdaLds<ST, DK, OP>));
  static const hipError_t attr = hipFuncSetAttribute(
      reinterpret_cast<const void*>(&kda_scan_kernel<TIN, ST, OP, DK, DV>),
      hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL((kda_scan_kernel<TIN, ST, OP, DK, DV>), dim3(n_items), dim3(kKT), bytes, s,
                     a);
  return hipGetLastError();
}

template <typename TIN, int DK, int DV>
hipError_t launch_kda_dims(const KdaArgs& a, int n_chains, hipStream_t s) {
  const int64_t n_state = static_cast<int64_t>(n_chains) * a.h_v * (DV / KNC);
  if (n_state > 0x7fffffff) return hipErrorInvalidValue;
  hipError_t e = launch_kda_t<TIN, TIN, false, DK, DV>(a, static_cast<int>(n_state), s);
  if (e != hipSuccess || a.mode != 0 || a.P_hat == nullptr) return e;
  const int64_t n_op = static_cast<int64_t>(n_chains) * a.h_v * (DK / KNC);
  if (n_op > 0x7fffffff) return hipErrorInvalidValue;
  return launch_kda_t<TIN, float, true, DK, DV>(a, static_cast<int>(n_op), s);
}

template <typename TIN>
hipError_t launch_kda_in(const KdaArgs& a, int d_k, int d_v, int n_chains, hipStream_t s) {
  if (d_k == 64 && d_v == 64) return launch_kda_dims<TIN, 64, 64>(a, n_chains, s);
  if (d_k == 64 && d_v == 128) return launch_kda_dims<TIN, 64, 128>(a, n_chains, s);
  if (d_k == 128 && d_v == 64) return launch_kda_dims<TIN, 128, 64>(a, n_chains, s);
  return launch_kda_dims<TIN, 128, 128>(a, n_chains, s);
}

}  // namespace

hipError_t launch_kda_scan(const KdaArgs& a, int bf16, int d_k, int d_v, int n_chains,
                           hipStream_t s) {
  if (n_chains <= 0) return hipSuccess;
  return bf16 ? launch_kda_in<uint16_t>(a, d_k, d_v, n_chains, s)
              : launch_kda_in<float>(a, d_k, d_v, n_chains, s);
}

}  // namespace hypic
