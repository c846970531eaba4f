// Segment build, seam rescan and composition for the scalar and diagonal
// transition families of Tab. 1 on gfx950.
//
// Per head and token t (Tab. 1; these rows have no delta-rule correction):
//   scalar   (RetNet, Lightning-2, Mamba2):  S_t = exp(a_t) S_{t-1} + k_t v_t^T
//   diagonal (GLA):                          S_t = diag(exp(g_t)) S_{t-1} + k_t v_t^T
//   o_t = S_t^T q_t (the token reads the state after its own write, Eq. (2)).
// The segment operator of Tab. 3 is compressed to a scalar or a d_k vector;
// it is carried as its logarithm, log_decay = sum_t a_t (or sum_t g_t), which
// does not underflow on long segments.
//
// Chunked form (C = 64 tokens, incoming state S0, B_t = prefix sum of the
// gate inside the chunk, per channel for the diagonal family):
//   O = (Q . exp(B)) S0 + A V,   A_ti = sum_c q_tc k_ic exp(B_tc - B_ic)  (i <= t)
//   S <- exp(B_last) . S0 + (K . exp(B_last - B))^T V
// Scalar gates factor out of A: A = tril(Q K^T) . exp(b_t - b_i).  Per-channel
// gates do not; A is formed tile by tile over 16-token tiles with the gate
// referred to Bbar_T, the cumulative gate just before key tile T:
//   A_(tq, T) = (Q_tq . exp(B_tq - Bbar_T)) (K_T . exp(Bbar_T - B_T))^T,
// where the query factor never exceeds 1 and the key factor is bounded by the
// decay over at most 16 tokens.  The query factor is stored once as
// Q . exp(B - Bbar_tile(t)) and completed per tile pair by the channel vector
// exp(Bbar_tq - Bbar_T) <= 1; the inter-chunk query factor and the key decay of
// the state update are completed the same way from per-tile channel vectors.
// The diagonal path therefore needs every channel's gate sum over any 16
// consecutive tokens of a chunk to be above about -80 (float32 range); the
// scalar path has no such limit.
//
// Organisation: one workgroup of 8 waves runs one (segment or seam entry,
// v-head, column block) chain over its chunks in order; its barriers wait for
// LDS traffic only, so global loads and output stores stay in flight across
// them.  Two kernels:
//  * family_scan_kernel (diagonal family; float32 inputs of either family):
//    per chunk the whole workgroup stages Q, K and its V columns in LDS
//    (register prefetch of the next chunk runs meanwhile), forms the gate
//    prefix and the decayed operands, the 16 x 16 tiles of A on the matrix
//    cores, then the outputs and the state, which stays in registers (each
//    wave a 16-column group and a share of the d_k rows).
//  * family_pipe_kernel (scalar family, bf16 inputs): four waves hold the
//    state and make the outputs of chunk c while the other four stage and
//    form chunk c + 1, double-buffered.
// bf16 inputs use bf16 matrix-core products with float32 accumulation; the
// decayed operands of the state update and of the inter-chunk term are
// rounded to bf16 once, while the diagonal family's tile-referred Q and K of
// the intra-chunk scores A are kept as bf16 hi + lo pairs (three passes), so a
// score whose q . k terms cancel keeps its float32 accuracy.  float32 inputs
// use the float32 matrix cores.
//
// Composition (Eq. (6) with the compressed operators of Tab. 3) is
// elementwise: S <- exp(log_decay_i) . S + S_seg_i, streamed 16 bytes per
// lane with the running state in registers.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mfma.hpp"
#include "family.hpp"
#include "frag_common.hpp"

namespace hypic {

namespace {

constexpr int kFT = 512;  // threads of a scan workgroup (8 waves)
constexpr int FC = 64;    // tokens per chunk
// State columns per scan workgroup: 64, or 32 for float32 inputs at d_k = 128
// (whose operands would not fit in LDS with 64).  (32-column bf16 blocks would
// fit a scalar-family workgroup twice per compute unit, but the duplicated
// chunk-local work of four blocks per chain outweighs the overlap: 0.24 ms
// against 0.17 ms on 16 heads x 8 x 2048 tokens.)
template <int FAM, typename ST, int DK>
constexpr int fnc_of() {
  return (DK == 128 && sizeof(ST) == 4) ? 32 : 64;
}

template <int FAM, typename ST, int DK>
struct FamLds {
  static constexpr int FNC = fnc_of<FAM, ST, DK>();
  static constexpr bool DG = FAM == FAM_DIAGONAL;
  static constexpr int PAD = (sizeof(ST) == 2) ? 8 : 4;
  static constexpr int LDK = DK + PAD;  // Q, K rows (token-major)
  static constexpr int LDT = FC + PAD;  // rows of the token-minor operands and of A
  // diagonal family, bf16 operands: the tile-referred Q and K are also kept as
  // their bf16 remainders (lo), so the A tiles run on hi + lo operands
  static constexpr bool SPL = DG && sizeof(ST) == 2;
  alignas(16) ST q[FC * LDK];     // Q, then (diagonal) Q . exp(B - Bbar)
  alignas(16) ST k[FC * LDK];     // K, then (diagonal) K . exp(Bbar - B)
  alignas(16) ST qlo[SPL ? FC * LDK : 8];  // remainders of Q . exp(B - Bbar)
  alignas(16) ST klo[SPL ? FC * LDK : 8];  // remainders of K . exp(Bbar - B)
  ST kdt[DK * LDT];   // (K . exp(B_last - B))^T: channel-major
  ST vt[FNC * LDT];   // V^T of this workgroup's columns: column-major
  ST a[FC * LDT];     // A (lower 16 x 16 tiles; the upper tiles read stay 0)
  Frag<ST> s0f[FNC / 16][DK / 32][64];  // S0 as B fragments: column group, 32-row block, lane
  // scalar family: prefix b of the gate, exp(b)
  float bc[FC], gam[FC];
  // diagonal family, per channel: totals of the four 16-token tiles,
  // exp(Bbar_tq - Bbar_tk) for the six tile pairs tk < tq, exp(Bbar) per tile,
  // exp(B_last)
  float part[DG ? 4 * DK : 4];
  float fx[DG ? 6 * DK : 4];
  float hx[DG ? 4 * DK : 4];
  float lx[DG ? DK : 4];
};

__device__ __forceinline__ int fam_segment_of_rank(const FamArgs& a, int rank) {
  return a.n_inline > 0 ? static_cast<int>(a.order_inline[rank]) : a.order[rank];
}

template <int FAM, typename ST, int DK, int DV>
__global__ __launch_bounds__(kFT) void family_scan_kernel(FamArgs args) {
  using L = FamLds<FAM, ST, DK>;
  constexpr int LDK = L::LDK, LDT = L::LDT;
  constexpr int FNC = L::FNC;
  constexpr int NCG = FNC / 16;                            // column groups of 16
  constexpr int NRG = 8 / NCG;                             // row groups (waves per group)
  constexpr int VEC = 16 / static_cast<int>(sizeof(ST));  // elements per 16-byte load
  constexpr int NQ = FC * DK / (VEC * kFT);                // 16-byte loads of Q (and K)
  constexpr int NV = (FC * FNC + VEC * kFT - 1) / (VEC * kFT);  // 16-byte loads of V (rows
                                                                 // past the tile read zeros)
  constexpr int NMH = DK / (16 * NRG);                     // state row tiles per wave
  constexpr int NOT = 4 / NRG;                             // output token tiles per wave
  constexpr bool DIAG = FAM == FAM_DIAGONAL;
  static_assert(NQ >= 1 && NV >= 1, "tile split");
  static_assert(NMH % 2 == 0, "a wave's state rows must be whole 32-row blocks");
  static_assert(sizeof(L) <= 160 * 1024, "LDS budget");

  extern __shared__ __align__(16) unsigned char smem_raw[];
  L& sm = *reinterpret_cast<L*>(smem_raw);

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63;
  const int g = lane >> 4, ln = lane & 15;
  const int cg = wave % NCG, rgrp = wave / NCG;  // this wave's column group and row group

  // ---- work item: XCD-aware numbering of the column blocks of one chain ----
  constexpr int n_cb = DV / FNC;
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
    seg = fam_segment_of_rank(args, rank);
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
  const ST* qg = static_cast<const ST*>(args.q) + hk * DK;
  const ST* kg = static_cast<const ST*>(args.k) + hk * DK;
  const ST* vg = static_cast<const ST*>(args.v) + h * DV + cb * FNC;
  const long sh = static_cast<long>(seg) * args.h_v + h;
  const int col16 = 16 * cg;            // this wave's columns inside the block
  const int col = cb * FNC + col16;     // ... and in the state
  const int row0 = rgrp * (DK / NRG);     // this wave's first state row

  // ---- state: rows row0 .. row0 + DK/2 - 1, columns col .. col + 15 ----
  f32x4 st[NMH];
  if (args.mode == 1) {
    const float* s_in = args.S_in + sh * DK * DV + col + ln;
#pragma unroll
    for (int mt = 0; mt < NMH; ++mt)
#pragma unroll
      for (int i = 0; i < 4; ++i) st[mt][i] = s_in[(row0 + mt * 16 + 4 * g + i) * DV];
  } else {
#pragma unroll
    for (int mt = 0; mt < NMH; ++mt) st[mt] = zero4();
  }

  // the upper tiles of A read by the A V products, (0, 1) and (2, 3), stay zero
  {
    const int t = tid >> 8, e = tid & 255;
    stv(sm.a + (32 * t + (e >> 4)) * LDT + 32 * t + 16 + (e & 15), 0.f);
  }

  // ---- register prefetch of one chunk ----
  // Q, K, V: token-major 16-byte pieces.  Gates: scalar, lane = token (every
  // wave holds the chunk's 64 gates); diagonal, thread (channel pc, tile pt)
  // holds the 16 gates of its channel in its tile (threads below 4 d_k).
  uint4 rq[NQ], rk[NQ], rv[NV];
  float rg[DIAG ? 16 : 1];
  const int pc = tid % DK, pt = tid / DK;
  const bool gate_thread = !DIAG || tid < 4 * DK;
  // n tokens from c0 (n <= 0 past the end: nothing is read, zeros arrive)
  auto prefetch = [&](int c0, int n) __attribute__((always_inline)) {
    constexpr int SZ = static_cast<int>(sizeof(ST));
    const auto rsq = rsrc(qg + static_cast<long>(c0) * qk_stride, n * qk_stride * SZ);
    const auto rsk = rsrc(kg + static_cast<long>(c0) * qk_stride, n * qk_stride * SZ);
    const auto rsv = rsrc(vg + static_cast<long>(c0) * v_stride, n * v_stride * SZ);
#pragma unroll
    for (int u = 0; u < NQ; ++u) {
      const int idx = u * kFT + tid;
      const int r = idx / (DK / VEC), cv = idx % (DK / VEC);
      const int off = static_cast<int>((r * qk_stride + cv * VEC) * SZ);
      rq[u] = bload16(rsq, off);
      rk[u] = bload16(rsk, off);
    }
#pragma unroll
    for (int u = 0; u < NV; ++u) {
      const int idx = u * kFT + tid;
      const int r = idx / (FNC / VEC), cv = idx % (FNC / VEC);
      rv[u] = bload16(rsv, static_cast<int>((r * v_stride + cv * VEC) * SZ));
    }
    if constexpr (DIAG) {
      const long gs = static_cast<long>(args.h_v) * DK;  // gate elements per token
      const auto rsg = rsrc(args.gate + static_cast<long>(c0) * gs, n * gs * 4);
#pragma unroll
      for (int j = 0; j < 16; ++j)
        rg[j] = bload4(rsg, static_cast<int>(((16 * pt + j) * gs + h * DK + pc) * 4));
    } else {
      const auto rsg = rsrc(args.gate + static_cast<long>(c0) * args.h_v, n * args.h_v * 4);
      rg[0] = bload4(rsg, (lane * args.h_v + h) * 4);
    }
  };
  if (lo < hi) prefetch(lo, (hi - lo < FC) ? hi - lo : FC);
  {
    // As many (dropped) stores as a chunk's outputs: every path into the chunk
    // loop then has the same number of memory operations behind the prefetch,
    // so the waits for it do not extend to the previous chunk's output stores.
    const auto none = rsrc(nullptr, 0);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < 4 * NOT; ++i) bstore(none, 64 * i, 0.f, static_cast<ST*>(nullptr));
    __builtin_amdgcn_sched_barrier(0);
  }
  float ld_acc = 0.f;  // log_decay: every lane (scalar) or thread c < DK (diagonal)

  for (int c0 = lo; c0 < hi; c0 += FC) {
    const int n = (hi - c0 < FC) ? hi - c0 : FC;
    lds_barrier();  // the previous chunk is done with every LDS buffer

    // ---- P0: publish S0; stage Q, K (token-major) and V^T; gate prefix;
    // (scalar) the decayed keys, channel-major ----
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
    float dec_l = 0.f, b_l = 0.f;  // scalar: exp(b_last - b) and b of token `lane`
    if constexpr (!DIAG) {
      const float b = wave_inclusive_sum(rg[0]);
      const float b_last = __builtin_bit_cast(
          float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, b), 63));
      b_l = b;
      dec_l = __expf(b_last - b);
      ld_acc += b_last;
      if (wave == 0) {
        sm.bc[lane] = b;
        sm.gam[lane] = __expf(b);
      }
    }
#pragma unroll
    for (int u = 0; u < NQ; ++u) {
      const int idx = u * kFT + tid;
      const int r = idx / (DK / VEC), cv = idx % (DK / VEC);
      *reinterpret_cast<uint4*>(sm.q + r * LDK + cv * VEC) = rq[u];
      *reinterpret_cast<uint4*>(sm.k + r * LDK + cv * VEC) = rk[u];
      if constexpr (!DIAG) {
        const float d = __shfl(dec_l, r, 64);
#pragma unroll
        for (int e = 0; e < VEC; ++e)
          stv(sm.kdt + (cv * VEC + e) * LDT + r, elem(rk[u], e, static_cast<const ST*>(nullptr)) * d);
      }
    }
#pragma unroll
    for (int u = 0; u < NV; ++u) {
      const int idx = u * kFT + tid;
      const int r = idx / (FNC / VEC), cv = idx % (FNC / VEC);
      if (r < FC) {
#pragma unroll
        for (int e = 0; e < VEC; ++e) put_raw(sm.vt + (cv * VEC + e) * LDT + r, rv[u], e);
      }
    }
    float pre[DIAG ? 16 : 1];
    if constexpr (DIAG) {
      if (gate_thread) {
        float run = 0.f;
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          run += rg[j];
          pre[j] = run;
        }
        sm.part[pt * DK + pc] = run;
      }
    }
    prefetch(c0 + FC, (hi - c0 - FC < FC) ? hi - c0 - FC : FC);
    lds_barrier();

    if constexpr (DIAG) {
      // ---- P1: thread (channel pc, tile pt): the tile-referred Q and K, the
      // decayed keys (channel-major) and the per-channel tile factors ----
      if (gate_thread) {
        float hbv[4], b_last = 0.f;
#pragma unroll
        for (int p = 0; p < 4; ++p) {
          hbv[p] = b_last;  // Bbar of tile p: the gates of the tiles before it
          b_last += sm.part[p * DK + pc];
        }
        float off = hbv[0];
#pragma unroll
        for (int p = 1; p < 4; ++p)
          if (p == pt) off = hbv[p];
        const float gdec = __expf(b_last - off);
        const int t0 = 16 * pt;
#pragma unroll
        for (int j8 = 0; j8 < 16; j8 += 8) {
          float kd[8];
#pragma unroll
          for (int jj = 0; jj < 8; ++jj) {
            const int j = j8 + jj, t = t0 + j;
            ST* qp = sm.q + t * LDK + pc;
            ST* kp = sm.k + t * LDK + pc;
            const float kv = ldv(kp);
            const float e = __expf(pre[j]);      // exp(B_t - Bbar) <= 1
            const float ie = __expf(-pre[j]);    // >= 1, bounded by 16 tokens of decay
            const float qs = ldv(qp) * e, ks = kv * ie;
            stv(qp, qs);
            stv(kp, ks);
            if constexpr (L::SPL) {
              stv(sm.qlo + t * LDK + pc, qs - bf16_round(qs));
              stv(sm.klo + t * LDK + pc, ks - bf16_round(ks));
            }
            kd[jj] = kv * (gdec * ie);           // K exp(B_last - B_t)
          }
          st8(sm.kdt + pc * LDT + t0 + j8, kd);
        }
#pragma unroll
        for (int tk = 0; tk < 3; ++tk)
          if (tk < pt) sm.fx[pair_idx(pt, tk) * DK + pc] = __expf(off - hbv[tk]);
        sm.hx[pt * DK + pc] = __expf(off);
        if (pt == 0) {
          sm.lx[pc] = __expf(b_last);
          ld_acc += b_last;
        }
      }
      lds_barrier();
    }

    // ---- P3: the lower 16 x 16 tiles of A ----
    for (int tile = wave; tile < 10; tile += 8) {
      const int tq = (tile < 1) ? 0 : ((tile < 3) ? 1 : ((tile < 6) ? 2 : 3));
      const int tk = tile - tq * (tq + 1) / 2;
      f32x4 acc = zero4();
      if constexpr (L::SPL) {
        // q_t . k_i exp(B_t - B_i) can nearly cancel; one bf16 rounding of the
        // gate-scaled operands would then dominate the score, so both operands
        // run as hi + lo (three passes)
#pragma unroll
        for (int kb = 0; kb < DK; kb += 32) {
          const SplitFrag fa =
              (tk < tq) ? frag_row_split_scaled(sm.q, sm.qlo, LDK, tq * 16 + ln, kb, g,
                                                sm.fx + pair_idx(tq, tk) * DK)
                        : frag_row_split(sm.q, sm.qlo, LDK, tq * 16 + ln, kb, g);
          acc = mma3(fa, frag_row_split(sm.k, sm.klo, LDK, tk * 16 + ln, kb, g), acc);
        }
      } else {
#pragma unroll
        for (int kb = 0; kb < DK; kb += 32) {
          Frag<ST> fa;
          if (DIAG && tk < tq)
            fa = frag_row_scaled(sm.q, LDK, tq * 16 + ln, kb, g, sm.fx + pair_idx(tq, tk) * DK);
          else
            fa = frag_row(sm.q, LDK, tq * 16 + ln, kb, g);
          acc = mma(fa, frag_row(sm.k, LDK, tk * 16 + ln, kb, g), acc);
        }
      }
      const int key = tk * 16 + ln;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int t = tq * 16 + 4 * g + i;
        float x = acc[i];
        if constexpr (!DIAG) x *= __expf(fminf(sm.bc[t] - sm.bc[key], 0.f));
        stv(sm.a + t * LDT + key, (key <= t) ? x : 0.f);
      }
    }
    lds_barrier();

    // ---- P4: two output tiles and the state rows of this wave ----
    Frag<ST> bv[2];  // V as B operand over the chunk's tokens (A V and the update)
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) bv[kt] = frag_row(sm.vt, LDT, col16 + ln, 32 * kt, g);
    {
      // outputs: rows t < n of this chunk (none when o is NULL)
      const long orow0 = (args.mode == 0) ? static_cast<long>(c0)
                                          : static_cast<long>(seg) * args.w + (c0 - lo);
      const auto rso = rsrc(args.o ? static_cast<const ST*>(args.o) + orow0 * v_stride : nullptr,
                            args.o ? n * v_stride * static_cast<long>(sizeof(ST)) : 0);
      const int ocol = static_cast<int>(h * DV + col + ln);
#pragma unroll
      for (int mh = 0; mh < NOT; ++mh) {
        const int mt = NOT * rgrp + mh;  // token tile
        f32x4 acc = zero4();
#pragma unroll
        for (int kt = 0; kt < DK / 32; ++kt) {
          Frag<ST> fa;
          if constexpr (DIAG)
            fa = frag_row_scaled(sm.q, LDK, mt * 16 + ln, 32 * kt, g, sm.hx + mt * DK);
          else
            fa = frag_row(sm.q, LDK, mt * 16 + ln, 32 * kt, g);
          acc = mma(fa, sm.s0f[cg][kt][lane], acc);
        }
        if constexpr (!DIAG) {
          const float4 gm = *reinterpret_cast<const float4*>(sm.gam + mt * 16 + 4 * g);
          acc[0] *= gm.x;
          acc[1] *= gm.y;
          acc[2] *= gm.z;
          acc[3] *= gm.w;
        }
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
          if (32 * kt < 16 * (mt + 1))
            acc = mma(frag_row(sm.a, LDT, mt * 16 + ln, 32 * kt, g), bv[kt], acc);
#pragma unroll
        for (int i = 0; i < 4; ++i)
          bstore(rso, static_cast<int>(((mt * 16 + 4 * g + i) * v_stride + ocol) * sizeof(ST)),
                 acc[i], static_cast<ST*>(nullptr));
      }
    }
    // S <- exp(B_last) . S0 + (K . exp(B_last - B))^T V
    const float g_last = DIAG ? 0.f : __expf(__shfl(b_l, 63, 64));
#pragma unroll
    for (int mt = 0; mt < NMH; ++mt) {
      const int r = row0 + mt * 16;
      f32x4 acc = st[mt];
      if constexpr (DIAG) {
        const float4 lx = *reinterpret_cast<const float4*>(sm.lx + r + 4 * g);
        acc[0] *= lx.x;
        acc[1] *= lx.y;
        acc[2] *= lx.z;
        acc[3] *= lx.w;
      } else {
        acc *= g_last;
      }
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
        acc = mma(frag_row(sm.kdt, LDT, r + ln, 32 * kt, g), bv[kt], acc);
      st[mt] = acc;
    }
  }

  // ---- the chain's results ----
  if (args.S_out != nullptr) {
    float* so = args.S_out + sh * DK * DV + col + ln;
#pragma unroll
    for (int mt = 0; mt < NMH; ++mt)
#pragma unroll
      for (int i = 0; i < 4; ++i) so[(row0 + mt * 16 + 4 * g + i) * DV] = st[mt][i];
  }
  if (args.mode == 0 && args.log_decay != nullptr && cb == 0) {
    if constexpr (DIAG) {
      if (tid < DK) args.log_decay[sh * DK + tid] = ld_acc;
    } else {
      if (tid == 0) args.log_decay[sh] = ld_acc;
    }
  }
}

// ---------------------------------------------------------------------------
// Scalar family, bf16 inputs, software-pipelined: four state waves run chunk
// c's outputs and state update while four producer waves stage and form chunk
// c + 1 (its operands double-buffered in LDS).  Producers issue every global
// load and the state waves every output store, so neither waits on the other's
// memory operations.  Per iteration: stage A (state: outputs of c; producers:
// stage c + 1, its gate prefix and decayed keys, prefetch c + 2), stage C
// (state: update of c; producers: the A tiles of c + 1), each closed by an
// LDS-only barrier.  (The diagonal family keeps the 8-wave kernel above: its
// tile-referred operands make the producer side the longer one, 0.23 ms
// against 0.22 ms on 16 heads x 8 x 2048 tokens.)
// ---------------------------------------------------------------------------
template <int DK>
struct PipeLds {
  static constexpr int LDK = DK + 8;  // Q, K rows (token-major)
  static constexpr int LDT = FC + 8;  // rows of the token-minor operands and of A
  // The token-minor operands are written as 4-byte token pairs by lanes that
  // run over 8-column groups; their tokens are permuted per 16-row band (row
  // r keeps token t at t ^ (SW * (r >> 4)), SW = 16 for V^T and for the keys
  // at d_k = 64, 8 for the keys at d_k = 128) so those writes meet 64
  // distinct banks, while every 4-token group the matrix cores read stays whole.
  static constexpr int SWV = 16, SWK = (DK == 128) ? 8 : 16;
  u16 q[2][FC * LDK];    // Q, by chunk parity
  u16 kdt[2][DK * LDT];  // (K . exp(b_last - b))^T
  u16 vt[2][64 * LDT];   // V^T of the block's 64 columns
  u16 a[2][FC * LDT];    // A (lower 16 x 16 tiles; the upper tiles read stay 0)
  u16 k[FC * LDK];       // K; producers only
  float bc[2][FC], gam[2][FC];  // prefix b of the gate, exp(b)
};

template <int DK, int DV>
__global__ __launch_bounds__(512) void family_pipe_kernel(FamArgs args) {
  using L = PipeLds<DK>;
  constexpr int LDK = L::LDK, LDT = L::LDT, SWV = L::SWV, SWK = L::SWK;
  constexpr int PT = 256;                 // producer threads
  constexpr int NQ = FC * DK / (8 * PT);  // 16-byte loads of Q (and K) per producer thread
  constexpr int NV = FC * 64 / (8 * PT);  // 16-byte loads of V
  constexpr int NM = DK / 16;             // state row tiles
  static_assert(NQ >= 2 && NV == 2, "tile split");
  static_assert(sizeof(L) <= 160 * 1024, "LDS budget");

  extern __shared__ __align__(16) unsigned char smem_raw[];
  L& sm = *reinterpret_cast<L*>(smem_raw);

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63;
  const int g = lane >> 4, ln = lane & 15;
  const bool producer = wave >= 4;
  const int ptid = tid - PT;  // producer thread index

  // ---- work item: XCD-aware numbering of the column blocks of one chain ----
  constexpr int n_cb = DV / 64;
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
    seg = fam_segment_of_rank(args, rank);
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
  const int nc = (hi - lo + FC - 1) / FC;

  const long qk_stride = static_cast<long>(args.h_qk) * DK;
  const long v_stride = static_cast<long>(args.h_v) * DV;
  const long sh = static_cast<long>(seg) * args.h_v + h;

  // the upper tiles of A read by the A V products, (0, 1) and (2, 3), stay zero
  for (int idx = tid; idx < 2 * 2 * 256; idx += 512) {
    const int par = idx >> 9, t = (idx >> 8) & 1, e = idx & 255;
    sm.a[par][(32 * t + (e >> 4)) * LDT + 32 * t + 16 + (e & 15)] = 0;
  }

  if (!producer) {
    // ======================= state waves ===================================
    const int col16 = 16 * wave;           // columns inside the block
    const int col = cb * 64 + col16;        // ... and in the state
    f32x4 st[NM];
    if (args.mode == 1) {
      const float* s_in = args.S_in + sh * DK * DV + col + ln;
#pragma unroll
      for (int mt = 0; mt < NM; ++mt)
#pragma unroll
        for (int i = 0; i < 4; ++i) st[mt][i] = s_in[(mt * 16 + 4 * g + i) * DV];
    } else {
#pragma unroll
      for (int mt = 0; mt < NM; ++mt) st[mt] = zero4();
    }
    const int ocol = static_cast<int>(h * DV + col + ln);
    for (int c = -1; c < nc; ++c) {
      const int buf = c & 1;
      const int c0 = lo + c * FC;
      const int n = (hi - c0 < FC) ? hi - c0 : FC;
      Frag<u16> bv[2];
      if (c >= 0) {
        // ---- stage A: outputs of chunk c, (Q S0) . exp(b) + A V ----
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
          bv[kt] = frag_row_sw(sm.vt[buf], LDT, col16 + ln, 32 * kt, g, SWV * wave);
        Frag<u16> bs[NM / 2];
#pragma unroll
        for (int kt = 0; kt < NM / 2; ++kt)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            bs[kt].set(i, st[2 * kt][i]);
            bs[kt].set(4 + i, st[2 * kt + 1][i]);
          }
        const long orow0 = (args.mode == 0) ? static_cast<long>(c0)
                                            : static_cast<long>(seg) * args.w + (c0 - lo);
        const auto rso = rsrc(args.o ? static_cast<const u16*>(args.o) + orow0 * v_stride : nullptr,
                              args.o ? n * v_stride * 2 : 0);
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) {
          f32x4 acc = zero4();
#pragma unroll
          for (int kt = 0; kt < NM / 2; ++kt)
            acc = mma(frag_row(sm.q[buf], LDK, mt * 16 + ln, 32 * kt, g), bs[kt], acc);
          const float4 gm = *reinterpret_cast<const float4*>(sm.gam[buf] + mt * 16 + 4 * g);
          acc[0] *= gm.x;
          acc[1] *= gm.y;
          acc[2] *= gm.z;
          acc[3] *= gm.w;
#pragma unroll
          for (int kt = 0; kt < 2; ++kt)
            if (32 * kt < 16 * (mt + 1))
              acc = mma(frag_row(sm.a[buf], LDT, mt * 16 + ln, 32 * kt, g), bv[kt], acc);
#pragma unroll
          for (int i = 0; i < 4; ++i)
            bstore(rso, ((mt * 16 + 4 * g + i) * static_cast<int>(v_stride) + ocol) * 2, acc[i],
                   static_cast<u16*>(nullptr));
        }
      }
      lds_barrier();
      // ---- stage C: state update of chunk c ----
      if (c >= 0) {
        const float g_last = __expf(sm.bc[buf][FC - 1]);
#pragma unroll
        for (int mt = 0; mt < NM; ++mt) {
          f32x4 acc = st[mt] * g_last;
#pragma unroll
          for (int kt = 0; kt < 2; ++kt)
            acc = mma(frag_row_sw(sm.kdt[buf], LDT, mt * 16 + ln, 32 * kt, g, SWK * mt), bv[kt],
                      acc);
          st[mt] = acc;
        }
      }
      lds_barrier();
    }
    if (args.S_out != nullptr) {
      float* so = args.S_out + sh * DK * DV + col + ln;
#pragma unroll
      for (int mt = 0; mt < NM; ++mt)
#pragma unroll
        for (int i = 0; i < 4; ++i) so[(mt * 16 + 4 * g + i) * DV] = st[mt][i];
    }
  } else {
    // ======================= producer waves ================================
    const int pw = wave - 4;
    const u16* qg = static_cast<const u16*>(args.q) + hk * DK;
    const u16* kg = static_cast<const u16*>(args.k) + hk * DK;
    const u16* vg = static_cast<const u16*>(args.v) + h * DV + cb * 64;
    uint4 rq[NQ], rk[NQ], rv[NV];
    float rg;  // the gate of token `lane` (every producer wave holds the chunk's 64)
    // K and V go in token pairs: item i of this thread is tokens 2 rp and
    // 2 rp + 1 of one 8-column group, items running over the groups fastest
    // (whole rows per load), so the token-minor copies are written as pairs
    const int rpv = ptid / 8, cvv = ptid % 8;  // V: one item
    // the next chunk's loads, each issued as soon as its registers are free,
    // so that no single burst waits long at issue
    auto pf_q = [&](int c0, int n) __attribute__((always_inline)) {
      const auto rsq = rsrc(qg + static_cast<long>(c0) * qk_stride, n * qk_stride * 2);
#pragma unroll
      for (int u = 0; u < NQ; ++u) {
        const int idx = u * PT + ptid;
        const int r = idx / (DK / 8), cv = idx % (DK / 8);
        rq[u] = bload16(rsq, static_cast<int>((r * qk_stride + cv * 8) * 2));
      }
    };
    auto pf_k = [&](int c0, int n) __attribute__((always_inline)) {
      const auto rsk = rsrc(kg + static_cast<long>(c0) * qk_stride, n * qk_stride * 2);
#pragma unroll
      for (int u = 0; u < NQ; ++u) {
        const int idx = (u >> 1) * PT + ptid;
        const int r = 2 * (idx / (DK / 8)) + (u & 1), cv = idx % (DK / 8);
        rk[u] = bload16(rsk, static_cast<int>((r * qk_stride + cv * 8) * 2));
      }
    };
    auto pf_v = [&](int c0, int n) __attribute__((always_inline)) {
      const auto rsv = rsrc(vg + static_cast<long>(c0) * v_stride, n * v_stride * 2);
#pragma unroll
      for (int u = 0; u < NV; ++u)
        rv[u] = bload16(rsv, static_cast<int>(((2 * rpv + u) * v_stride + cvv * 8) * 2));
    };
    auto pf_g = [&](int c0, int n) __attribute__((always_inline)) {
      const auto rsg = rsrc(args.gate + static_cast<long>(c0) * args.h_v, n * args.h_v * 4);
      rg = bload4(rsg, (lane * args.h_v + h) * 4);
    };
    auto prefetch = [&](int c0, int n) __attribute__((always_inline)) {
      pf_q(c0, n);
      pf_k(c0, n);
      pf_v(c0, n);
      pf_g(c0, n);
    };
    if (nc > 0) prefetch(lo, (hi - lo < FC) ? hi - lo : FC);
    float ld_acc = 0.f;  // log_decay: sum of the chunk gate totals
    for (int p = 0; p <= nc; ++p) {  // the chunk this iteration forms
      const int buf = p & 1;
      const int c0 = lo + p * FC;
      const bool active = p < nc;
      // ---- stage A: stage chunk p, its gate prefix and decayed keys;
      // prefetch chunk p + 1, part by part ----
      if (active) {
        const int c1 = c0 + FC, n1 = (hi - c1 < FC) ? hi - c1 : FC;
#pragma unroll
        for (int u = 0; u < NQ; ++u) {
          const int idx = u * PT + ptid;
          const int r = idx / (DK / 8), cv = idx % (DK / 8);
          *reinterpret_cast<uint4*>(sm.q[buf] + r * LDK + cv * 8) = rq[u];
        }
        pf_q(c1, n1);
#pragma unroll
        for (int u = 0; u < NQ; ++u) {
          const int idx = (u >> 1) * PT + ptid;
          const int r = 2 * (idx / (DK / 8)) + (u & 1), cv = idx % (DK / 8);
          *reinterpret_cast<uint4*>(sm.k + r * LDK + cv * 8) = rk[u];
        }
#pragma unroll
        for (int e = 0; e < 8; ++e)
          *reinterpret_cast<uint32_t*>(sm.vt[buf] + (cvv * 8 + e) * LDT +
                                       ((2 * rpv) ^ (SWV * (cvv >> 1)))) =
              pair_raw(rv[0], rv[1], e);
        pf_v(c1, n1);
        const float b = wave_inclusive_sum(rg);
        pf_g(c1, n1);
        const float b_last = __builtin_bit_cast(
            float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, b), 63));
        const float dec = __expf(b_last - b);
        if (pw == 0) {
          sm.bc[buf][lane] = b;
          sm.gam[buf][lane] = __expf(b);
          ld_acc += b_last;
        }
#pragma unroll
        for (int j = 0; j < NQ / 2; ++j) {
          const int idx = j * PT + ptid;
          const int rp = idx / (DK / 8), cv = idx % (DK / 8);
          const float d0 = __shfl(dec, 2 * rp, 64), d1 = __shfl(dec, 2 * rp + 1, 64);
#pragma unroll
          for (int e = 0; e < 8; ++e)
            *reinterpret_cast<uint32_t*>(sm.kdt[buf] + (cv * 8 + e) * LDT +
                                         ((2 * rp) ^ (SWK * (cv >> 1)))) =
                pack_bf16(elem(rk[2 * j], e, static_cast<const u16*>(nullptr)) * d0,
                          elem(rk[2 * j + 1], e, static_cast<const u16*>(nullptr)) * d1);
        }
        pf_k(c1, n1);
      }
      lds_barrier();
      // ---- stage C: the lower 16 x 16 tiles of A for chunk p ----
      if (active) {
        for (int tile = pw; tile < 10; tile += 4) {
          const int tq = (tile < 1) ? 0 : ((tile < 3) ? 1 : ((tile < 6) ? 2 : 3));
          const int tk = tile - tq * (tq + 1) / 2;
          f32x4 acc = zero4();
#pragma unroll
          for (int kb = 0; kb < DK; kb += 32)
            acc = mma(frag_row(sm.q[buf], LDK, tq * 16 + ln, kb, g),
                      frag_row(sm.k, LDK, tk * 16 + ln, kb, g), acc);
          const int key = tk * 16 + ln;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int t = tq * 16 + 4 * g + i;
            const float x = acc[i] * __expf(fminf(sm.bc[buf][t] - sm.bc[buf][key], 0.f));
            stv(sm.a[buf] + t * LDT + key, (key <= t) ? x : 0.f);
          }
        }
      }
      lds_barrier();
    }
    if (args.mode == 0 && args.log_decay != nullptr && cb == 0 && ptid == 0)
      args.log_decay[sh] = ld_acc;
  }
}

// ---------------------------------------------------------------------------
// composition: S <- exp(log_decay_i) . S + S_seg_i, elementwise
// ---------------------------------------------------------------------------
constexpr int kCT = 256;          // threads
constexpr int kCPart = 4096;      // state elements per workgroup (16 per thread)

template <int FAM, int DK, int DV>
__global__ __launch_bounds__(kCT) void family_compose_kernel(FamComposeArgs a) {
  constexpr int NPART = DK * DV / kCPart;
  constexpr int NU = kCPart / (4 * kCT);  // float4 per thread
  constexpr bool DIAG = FAM == FAM_DIAGONAL;
  constexpr int LOOK = 2;
  const int tid = threadIdx.x;
  // head-major: the workgroups resident at one time share one head's slice of
  // the pool in the memory-side cache; incoming states stream past it
  // non-temporally
  const int chain = blockIdx.x / NPART, part = blockIdx.x % NPART;
  const int n_req = static_cast<int>(gridDim.x) / (NPART * a.h_v);
  const int req = chain % n_req, h = chain / n_req;
  const long state_sz = static_cast<long>(DK) * DV;
  const long hs = static_cast<long>(req) * a.h_v + h;
  int e[NU];
#pragma unroll
  for (int u = 0; u < NU; ++u) e[u] = part * kCPart + (u * kCT + tid) * 4;

  float4 s[NU];
  if (a.S_prefix != nullptr) {
#pragma unroll
    for (int u = 0; u < NU; ++u)
      s[u] = *reinterpret_cast<const float4*>(a.S_prefix + hs * state_sz + e[u]);
  } else {
#pragma unroll
    for (int u = 0; u < NU; ++u) s[u] = make_float4(0.f, 0.f, 0.f, 0.f);
  }
  struct Step {
    float4 s[NU];
    float g[DIAG ? NU : 1];
  };
  const int j0 = a.req_offsets[req], j1 = a.req_offsets[req + 1];
  auto load = [&](Step& t, int j) __attribute__((always_inline)) {
    const long ih = static_cast<long>(a.seg_ids[j]) * a.h_v + h;
#pragma unroll
    for (int u = 0; u < NU; ++u)
      t.s[u] = *reinterpret_cast<const float4*>(a.S_seg + ih * state_sz + e[u]);
    if constexpr (DIAG) {
#pragma unroll
      for (int u = 0; u < NU; ++u) t.g[u] = a.log_decay[ih * DK + e[u] / DV];
    } else {
      t.g[0] = a.log_decay[ih];
    }
  };
  Step buf[LOOK];
#pragma unroll
  for (int b = 0; b < LOOK; ++b)
    if (j0 + b < j1) load(buf[b], j0 + b);
  for (int j = j0; j < j1; j += LOOK) {
#pragma unroll
    for (int b = 0; b < LOOK; ++b) {
      const int jj = j + b;
      if (jj < j1) {
        Step cur = buf[b];
        if (jj + LOOK < j1) load(buf[b], jj + LOOK);
        if (a.S_incoming != nullptr) {
          float* dst = a.S_incoming + (static_cast<long>(jj) * a.h_v + h) * state_sz;
#pragma unroll
          for (int u = 0; u < NU; ++u)
            __builtin_nontemporal_store(f32x4{s[u].x, s[u].y, s[u].z, s[u].w},
                                        reinterpret_cast<f32x4*>(dst + e[u]));
        }
#pragma unroll
        for (int u = 0; u < NU; ++u) {
          const float f = __expf(cur.g[DIAG ? u : 0]);
          s[u].x = f * s[u].x + cur.s[u].x;
          s[u].y = f * s[u].y + cur.s[u].y;
          s[u].z = f * s[u].z + cur.s[u].z;
          s[u].w = f * s[u].w + cur.s[u].w;
        }
      }
    }
  }
#pragma unroll
  for (int u = 0; u < NU; ++u) *reinterpret_cast<float4*>(a.S_out + hs * state_sz + e[u]) = s[u];
}

template <int FAM, typename ST, int DK, int DV>
hipError_t launch_fscan_t(const FamArgs& a, int n_items, hipStream_t s) {
  constexpr int bytes = static_cast<int>(sizeof(FamLds<FAM, ST, DK>));
  static const hipError_t attr = hipFuncSetAttribute(
      reinterpret_cast<const void*>(&family_scan_kernel<FAM, ST, DK, DV>),
      hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL((family_scan_kernel<FAM, ST, DK, DV>), dim3(n_items), dim3(kFT), bytes, s,
                     a);
  return hipGetLastError();
}

template <int DK, int DV>
hipError_t launch_fpipe_t(const FamArgs& a, int n_items, hipStream_t s) {
  constexpr int bytes = static_cast<int>(sizeof(PipeLds<DK>));
  static const hipError_t attr = hipFuncSetAttribute(
      reinterpret_cast<const void*>(&family_pipe_kernel<DK, DV>),
      hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL((family_pipe_kernel<DK, DV>), dim3(n_items), dim3(512), bytes, s, a);
  return hipGetLastError();
}

hipError_t launch_fpipe_d(const FamArgs& a, int d_k, int d_v, int n_items, hipStream_t s) {
  if (d_k == 64 && d_v == 64) return launch_fpipe_t<64, 64>(a, n_items, s);
  if (d_k == 64 && d_v == 128) return launch_fpipe_t<64, 128>(a, n_items, s);
  if (d_k == 128 && d_v == 64) return launch_fpipe_t<128, 64>(a, n_items, s);
  return launch_fpipe_t<128, 128>(a, n_items, s);
}

template <int FAM, typename ST>
hipError_t launch_fscan_d(const FamArgs& a, int d_k, int d_v, int n_items, hipStream_t s) {
  if (d_k == 64 && d_v == 64) return launch_fscan_t<FAM, ST, 64, 64>(a, n_items, s);
  if (d_k == 64 && d_v == 128) return launch_fscan_t<FAM, ST, 64, 128>(a, n_items, s);
  if (d_k == 128 && d_v == 64) return launch_fscan_t<FAM, ST, 128, 64>(a, n_items, s);
  return launch_fscan_t<FAM, ST, 128, 128>(a, n_items, s);
}

template <int FAM, int DK, int DV>
hipError_t launch_fcompose_t(const FamComposeArgs& a, int n_req, hipStream_t s) {
  constexpr int NPART = DK * DV / kCPart;
  const long n_items = static_cast<long>(n_req) * a.h_v * NPART;
  if (n_items > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL((family_compose_kernel<FAM, DK, DV>), dim3(n_items), dim3(kCT), 0, s, a);
  return hipGetLastError();
}

template <int FAM>
hipError_t launch_fcompose_d(const FamComposeArgs& a, int d_k, int d_v, int n_req,
                             hipStream_t s) {
  if (d_k == 64 && d_v == 64) return launch_fcompose_t<FAM, 64, 64>(a, n_req, s);
  if (d_k == 64 && d_v == 128) return launch_fcompose_t<FAM, 64, 128>(a, n_req, s);
  if (d_k == 128 && d_v == 64) return launch_fcompose_t<FAM, 128, 64>(a, n_req, s);
  return launch_fcompose_t<FAM, 128, 128>(a, n_req, s);
}

}  // namespace

hipError_t launch_family_scan(const FamArgs& a, int family, int bf16, int d_k, int d_v,
                              int n_chains, hipStream_t s) {
  if (n_chains <= 0) return hipSuccess;
  int fnc = 64;
  if (d_k == 128) {
    if (family == FAM_DIAGONAL)
      fnc = bf16 ? fnc_of<FAM_DIAGONAL, uint16_t, 128>() : fnc_of<FAM_DIAGONAL, float, 128>();
    else
      fnc = bf16 ? fnc_of<FAM_SCALAR, uint16_t, 128>() : fnc_of<FAM_SCALAR, float, 128>();
  }
  const int64_t n_items = static_cast<int64_t>(n_chains) * a.h_v * (d_v / fnc);
  if (n_items > 0x7fffffff) return hipErrorInvalidValue;
  const int n = static_cast<int>(n_items);
  if (family == FAM_DIAGONAL && diag_pipe_supported(bf16, d_k, d_v, a.mode))
    return launch_diag_pipe(a, d_v, n_chains, s);
  if (family == FAM_SCALAR && diag_pipe_supported(bf16, d_k, d_v, a.mode))
    return launch_scalar_pipe(a, d_v, n_chains, s);
  // scalar family, bf16 inputs: the software-pipelined kernel (64-column blocks)
  if (family == FAM_DIAGONAL)
    return bf16 ? launch_fscan_d<FAM_DIAGONAL, uint16_t>(a, d_k, d_v, n, s)
                : launch_fscan_d<FAM_DIAGONAL, float>(a, d_k, d_v, n, s);
  return bf16 ? launch_fpipe_d(a, d_k, d_v, n, s)
              : launch_fscan_d<FAM_SCALAR, float>(a, d_k, d_v, n, s);
}

hipError_t launch_family_compose(const FamComposeArgs& a, int family, int d_k, int d_v,
                                 int n_req, hipStream_t s) {
  if (n_req <= 0) return hipSuccess;
  if (family == FAM_DIAGONAL) return launch_fcompose_d<FAM_DIAGONAL>(a, d_k, d_v, n_req, s);
  return launch_fcompose_d<FAM_SCALAR>(a, d_k, d_v, n_req, s);
}

}  // namespace hypic
