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
// Organisation: one workgroup of 4 waves runs one (segment or seam entry,
// v-head, 64-column block) chain over its chunks in order.  Each wave owns 16
// state columns with all d_k rows in registers.  Per chunk the workgroup
// stages Q, K and its V columns in LDS (register prefetch of the next chunk
// runs meanwhile), forms the gate prefix and the decayed operands, the
// 16 x 16 tiles of A on the matrix cores, then each wave its outputs and its
// state columns.  bf16 inputs use bf16 matrix-core products with float32
// accumulation (every decayed operand is rounded to bf16 once); float32
// inputs use the float32 matrix cores.
//
// Composition (Eq. (6) with the compressed operators of Tab. 3) is
// elementwise: S <- exp(log_decay_i) . S + S_seg_i, streamed 16 bytes per
// lane with the running state in registers.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mfma.hpp"
#include "scan.hpp"

namespace hypic {

namespace {

constexpr int kFT = 256;  // threads of a scan workgroup
constexpr int FC = 64;    // tokens per chunk
constexpr int FNC = 64;   // state columns per scan workgroup

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
  __device__ void set_raw(int j, u16 b) { x[j] = __builtin_bit_cast(__bf16, b); }
};
template <>
struct Frag<float> {
  float x[8];
  __device__ void set(int j, float v) { x[j] = v; }
  __device__ void set_raw(int j, float b) { x[j] = b; }
};

__device__ __forceinline__ f32x4 mma(const Frag<u16>& a, const Frag<u16>& b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a.x, b.x, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mma(const Frag<float>& a, const Frag<float>& b, f32x4 c) {
#pragma unroll
  for (int j = 0; j < 8; ++j) c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.x[j], b.x[j], c, 0, 0, 0);
  return c;
}

// slot j = M[row][kb + kap(g, j)] (contraction index contiguous in memory)
template <typename ST>
__device__ __forceinline__ Frag<ST> frag_row(const ST* M, int ld, int row, int kb, int g) {
  Frag<ST> f;
  const ST* p = M + row * ld + kb + 4 * g;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    f.set_raw(j, p[j]);
    f.set_raw(4 + j, p[16 + j]);
  }
  return f;
}
// slot j = M[row][kb + kap(g, j)] * s[kb + kap(g, j)]
template <typename ST>
__device__ __forceinline__ Frag<ST> frag_row_scaled(const ST* M, int ld, int row, int kb, int g,
                                                    const float* s) {
  Frag<ST> f;
  const ST* p = M + row * ld + kb + 4 * g;
  const float* q = s + kb + 4 * g;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    f.set(j, ldv(p + j) * q[j]);
    f.set(4 + j, ldv(p + 16 + j) * q[16 + j]);
  }
  return f;
}
// slot j = M[kb + kap(g, j)][col] (contraction index strided)
template <typename ST>
__device__ __forceinline__ Frag<ST> frag_col(const ST* M, int ld, int col, int kb, int g) {
  Frag<ST> f;
#pragma unroll
  for (int j = 0; j < 8; ++j) f.set_raw(j, M[(kb + kap(g, j)) * ld + col]);
  return f;
}

template <int FAM, typename ST, int DK>
struct FamLds {
  static constexpr int PAD = (sizeof(ST) == 2) ? 8 : 4;
  static constexpr int LDK = DK + PAD;   // Q, K rows
  static constexpr int LDV = FNC + PAD;  // V rows (this workgroup's columns)
  static constexpr int LDA = FC + PAD;   // A rows
  static constexpr int NPART = kFT / DK; // token parts of the per-channel prefix
  ST q[FC * LDK];   // Q, then (diagonal) Q . exp(B - Bbar)
  ST k[FC * LDK];   // K, then (diagonal) K . exp(Bbar - B)
  ST v[FC * LDV];
  ST a[FC * LDA];   // A (lower-triangular 16 x 16 tiles; the upper tiles read stay 0)
  // scalar family: b (prefix of the gate), exp(b), exp(b_last - b)
  float bc[FC], gam[FC], dec[FC];
  // diagonal family, per channel: part totals, Bbar of each 16-token tile,
  // exp(Bbar_tq - Bbar_tk) for the six tile pairs tk < tq, exp(Bbar), exp(B_last - Bbar),
  // exp(B_last), B_last
  float part[NPART * DK];
  float hb[4 * DK];
  float fx[6 * DK];
  float hx[4 * DK];
  float gx[4 * DK];
  float lx[DK];
  float bl[DK];
};

// index of the tile pair (tq, tk), tk < tq, in fx
__device__ __forceinline__ int pair_idx(int tq, int tk) { return tq * (tq - 1) / 2 + tk; }

__device__ __forceinline__ int fam_segment_of_rank(const FamArgs& a, int rank) {
  return a.n_inline > 0 ? static_cast<int>(a.order_inline[rank]) : a.order[rank];
}

template <int FAM, typename ST, int DK, int DV>
__global__ __launch_bounds__(kFT) void family_scan_kernel(FamArgs args) {
  using L = FamLds<FAM, ST, DK>;
  constexpr int LDK = L::LDK, LDV = L::LDV, LDA = L::LDA;
  constexpr int VEC = 16 / static_cast<int>(sizeof(ST));  // elements per 16-byte load
  constexpr int NQ = FC * DK / (VEC * kFT);                // 16-byte loads of Q (and K)
  constexpr int NV = FC * FNC / (VEC * kFT);               // 16-byte loads of V
  constexpr int NM = DK / 16;                              // state row tiles
  constexpr int NPART = L::NPART;
  constexpr int TPC = FC / NPART;                          // tokens per prefix part
  constexpr bool DIAG = FAM == FAM_DIAGONAL;
  static_assert(NQ >= 1 && NV >= 1, "tile split");
  static_assert(TPC % 16 == 0, "prefix parts must hold whole 16-token tiles");
  static_assert(sizeof(L) <= 160 * 1024, "LDS budget");

  extern __shared__ __align__(16) unsigned char smem_raw[];
  L& sm = *reinterpret_cast<L*>(smem_raw);

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63;
  const int g = lane >> 4, ln = lane & 15;

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
  const int col16 = 16 * wave;          // this wave's columns inside the block
  const int col = cb * FNC + col16;     // ... and in the state

  // ---- state columns col .. col + 15, all d_k rows ----
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

  // the upper tiles of A read by the A V products, (0, 1) and (2, 3), stay zero
  for (int idx = tid; idx < 2 * 256; idx += kFT) {
    const int t = idx >> 8, e = idx & 255;
    const int r = 32 * t + (e >> 4), c = 32 * t + 16 + (e & 15);
    stv(sm.a + r * LDA + c, 0.f);
  }

  // ---- register prefetch of one chunk ----
  uint4 rq[NQ], rk[NQ], rv[NV];
  float rg[DIAG ? TPC : 1];
  const int gc = tid % DK, gpart = tid / DK;  // diagonal prefix: channel, token part
  auto prefetch = [&](int c0, int n) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < NQ; ++u) {
      const int idx = u * kFT + tid;
      const int r = idx / (DK / VEC), cv = idx % (DK / VEC);
      const long off = static_cast<long>(c0 + r) * qk_stride + cv * VEC;
      rq[u] = (r < n) ? *reinterpret_cast<const uint4*>(qg + off) : make_uint4(0, 0, 0, 0);
      rk[u] = (r < n) ? *reinterpret_cast<const uint4*>(kg + off) : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int u = 0; u < NV; ++u) {
      const int idx = u * kFT + tid;
      const int r = idx / (FNC / VEC), cv = idx % (FNC / VEC);
      rv[u] = (r < n) ? *reinterpret_cast<const uint4*>(vg + static_cast<long>(c0 + r) * v_stride +
                                                         cv * VEC)
                      : make_uint4(0, 0, 0, 0);
    }
    if constexpr (DIAG) {
#pragma unroll
      for (int j = 0; j < TPC; ++j) {
        const int r = gpart * TPC + j;
        rg[j] = (r < n) ? args.gate[(static_cast<long>(c0 + r) * args.h_v + h) * DK + gc] : 0.f;
      }
    } else {
      rg[0] = (tid < n) ? args.gate[static_cast<long>(c0 + tid) * args.h_v + h] : 0.f;
    }
  };
  if (lo < hi) prefetch(lo, (hi - lo < FC) ? hi - lo : FC);
  float ld_acc = 0.f;  // log_decay: wave 0 (scalar) or thread c < DK (diagonal)

  for (int c0 = lo; c0 < hi; c0 += FC) {
    const int n = (hi - c0 < FC) ? hi - c0 : FC;
    __syncthreads();  // the previous chunk is done with every LDS buffer

    // ---- P0: stage the chunk; gate prefix ----
#pragma unroll
    for (int u = 0; u < NQ; ++u) {
      const int idx = u * kFT + tid;
      const int r = idx / (DK / VEC), cv = idx % (DK / VEC);
      *reinterpret_cast<uint4*>(sm.q + r * LDK + cv * VEC) = rq[u];
      *reinterpret_cast<uint4*>(sm.k + r * LDK + cv * VEC) = rk[u];
    }
#pragma unroll
    for (int u = 0; u < NV; ++u) {
      const int idx = u * kFT + tid;
      const int r = idx / (FNC / VEC), cv = idx % (FNC / VEC);
      *reinterpret_cast<uint4*>(sm.v + r * LDV + cv * VEC) = rv[u];
    }
    float pre[DIAG ? TPC : 1];
    if constexpr (DIAG) {
      float run = 0.f;
#pragma unroll
      for (int j = 0; j < TPC; ++j) {
        run += rg[j];
        pre[j] = run;
      }
      sm.part[gpart * DK + gc] = run;
    } else if (wave == 0) {
      float b = rg[0];
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const float u = __shfl_up(b, off, 64);
        if (lane >= off) b += u;
      }
      const float b_last = __shfl(b, 63, 64);
      sm.bc[lane] = b;
      sm.gam[lane] = __expf(b);
      sm.dec[lane] = __expf(b_last - b);
      ld_acc += b_last;
    }
    if (c0 + FC < hi) prefetch(c0 + FC, (hi - c0 - FC < FC) ? hi - c0 - FC : FC);
    __syncthreads();

    if constexpr (DIAG) {
      // ---- P1: per-channel prefix B, tile references Bbar, decayed Q and K ----
      float off = 0.f;
#pragma unroll
      for (int p = 0; p < NPART; ++p)
        if (p < gpart) off += sm.part[p * DK + gc];
      const int t0 = gpart * TPC;
#pragma unroll
      for (int tt = 0; tt < TPC / 16; ++tt) {
        const float bbar = (tt == 0) ? off : off + pre[16 * tt - 1];
        sm.hb[((t0 >> 4) + tt) * DK + gc] = bbar;
#pragma unroll
        for (int j = 16 * tt; j < 16 * tt + 16; ++j) {
          const float d = off + pre[j] - bbar;  // <= 0
          ST* qp = sm.q + (t0 + j) * LDK + gc;
          ST* kp = sm.k + (t0 + j) * LDK + gc;
          stv(qp, ldv(qp) * __expf(d));
          stv(kp, ldv(kp) * __expf(-d));
        }
      }
      if (gpart == NPART - 1) sm.bl[gc] = off + pre[TPC - 1];
      __syncthreads();
      // ---- P2: per-channel factors of the tile pairs and the state update ----
      for (int idx = tid; idx < 15 * DK; idx += kFT) {
        const int which = idx / DK, c = idx % DK;
        if (which < 6) {
          const int tq = (which < 1) ? 1 : ((which < 3) ? 2 : 3);
          const int tk = which - pair_idx(tq, 0);
          sm.fx[which * DK + c] = __expf(sm.hb[tq * DK + c] - sm.hb[tk * DK + c]);
        } else if (which < 10) {
          sm.hx[(which - 6) * DK + c] = __expf(sm.hb[(which - 6) * DK + c]);
        } else if (which < 14) {
          sm.gx[(which - 10) * DK + c] = __expf(sm.bl[c] - sm.hb[(which - 10) * DK + c]);
        } else {
          sm.lx[c] = __expf(sm.bl[c]);
        }
      }
      if (tid < DK) ld_acc += sm.bl[tid];
      __syncthreads();
    }

    // ---- P3: the lower 16 x 16 tiles of A ----
    for (int tile = wave; tile < 10; tile += 4) {
      const int tq = (tile < 1) ? 0 : ((tile < 3) ? 1 : ((tile < 6) ? 2 : 3));
      const int tk = tile - tq * (tq + 1) / 2;
      f32x4 acc = zero4();
#pragma unroll
      for (int kb = 0; kb < DK; kb += 32) {
        Frag<ST> fa;
        if (DIAG && tk < tq)
          fa = frag_row_scaled(sm.q, LDK, tq * 16 + ln, kb, g, sm.fx + pair_idx(tq, tk) * DK);
        else
          fa = frag_row(sm.q, LDK, tq * 16 + ln, kb, g);
        acc = mma(fa, frag_row(sm.k, LDK, tk * 16 + ln, kb, g), acc);
      }
      const int key = tk * 16 + ln;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int t = tq * 16 + 4 * g + i;
        float x = acc[i];
        if constexpr (!DIAG) x *= __expf(fminf(sm.bc[t] - sm.bc[key], 0.f));
        stv(sm.a + t * LDA + key, (key <= t) ? x : 0.f);
      }
    }
    __syncthreads();

    // ---- P4: outputs and state columns of this wave ----
    Frag<ST> bv[2];  // V as B operand over the chunk's tokens (shared by A V and the update)
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) bv[kt] = frag_col(sm.v, LDV, col16 + ln, 32 * kt, g);
    if (args.o != nullptr) {
      Frag<ST> bs[NM / 2];  // S0 as B operand over d_k
#pragma unroll
      for (int kt = 0; kt < NM / 2; ++kt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          bs[kt].set(i, st[2 * kt][i]);
          bs[kt].set(4 + i, st[2 * kt + 1][i]);
        }
      const long orow0 = (args.mode == 0) ? static_cast<long>(c0)
                                          : static_cast<long>(seg) * args.w + (c0 - lo);
      ST* og = static_cast<ST*>(args.o) + static_cast<long>(h) * DV + col + ln;
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) {
        f32x4 acc = zero4();
#pragma unroll
        for (int kt = 0; kt < NM / 2; ++kt) {
          Frag<ST> fa;
          if constexpr (DIAG)
            fa = frag_row_scaled(sm.q, LDK, mt * 16 + ln, 32 * kt, g, sm.hx + mt * DK);
          else
            fa = frag_row(sm.q, LDK, mt * 16 + ln, 32 * kt, g);
          acc = mma(fa, bs[kt], acc);
        }
        if constexpr (!DIAG) {
#pragma unroll
          for (int i = 0; i < 4; ++i) acc[i] *= sm.gam[mt * 16 + 4 * g + i];
        }
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
          if (32 * kt < 16 * (mt + 1))
            acc = mma(frag_row(sm.a, LDA, mt * 16 + ln, 32 * kt, g), bv[kt], acc);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int t = mt * 16 + 4 * g + i;
          if (t < n) stv(og + (orow0 + t) * v_stride, acc[i]);
        }
      }
    }
    // S <- exp(B_last) . S0 + (K . exp(B_last - B))^T V
    const float g_last = DIAG ? 0.f : __expf(sm.bc[FC - 1]);
#pragma unroll
    for (int mt = 0; mt < NM; ++mt) {
      f32x4 acc;
#pragma unroll
      for (int i = 0; i < 4; ++i)
        acc[i] = st[mt][i] * (DIAG ? sm.lx[mt * 16 + 4 * g + i] : g_last);
      const int ch = mt * 16 + ln;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        Frag<ST> fa;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int tok = 32 * kt + kap(g, j);
          const float s = DIAG ? sm.gx[(tok >> 4) * DK + ch] : sm.dec[tok];
          fa.set(j, ldv(sm.k + tok * LDK + ch) * s);
        }
        acc = mma(fa, bv[kt], acc);
      }
      st[mt] = acc;
    }
  }

  // ---- the chain's results ----
  if (args.S_out != nullptr) {
    float* so = args.S_out + sh * DK * DV + col + ln;
#pragma unroll
    for (int mt = 0; mt < NM; ++mt)
#pragma unroll
      for (int i = 0; i < 4; ++i) so[(mt * 16 + 4 * g + i) * DV] = st[mt][i];
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
  const int chain = blockIdx.x / NPART, part = blockIdx.x % NPART;
  const int req = chain / a.h_v, h = chain % a.h_v;
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
          for (int u = 0; u < NU; ++u) *reinterpret_cast<float4*>(dst + e[u]) = s[u];
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
  const int64_t n_items = static_cast<int64_t>(n_chains) * a.h_v * (d_v / FNC);
  if (n_items > 0x7fffffff) return hipErrorInvalidValue;
  const int n = static_cast<int>(n_items);
  if (family == FAM_DIAGONAL)
    return bf16 ? launch_fscan_d<FAM_DIAGONAL, uint16_t>(a, d_k, d_v, n, s)
                : launch_fscan_d<FAM_DIAGONAL, float>(a, d_k, d_v, n, s);
  return bf16 ? launch_fscan_d<FAM_SCALAR, uint16_t>(a, d_k, d_v, n, s)
              : launch_fscan_d<FAM_SCALAR, float>(a, d_k, d_v, n, s);
}

hipError_t launch_family_compose(const FamComposeArgs& a, int family, int d_k, int d_v,
                                 int n_req, hipStream_t s) {
  if (n_req <= 0) return hipSuccess;
  if (family == FAM_DIAGONAL) return launch_fcompose_d<FAM_DIAGONAL>(a, d_k, d_v, n_req, s);
  return launch_fcompose_d<FAM_SCALAR>(a, d_k, d_v, n_req, s);
}

}  // namespace hypic
