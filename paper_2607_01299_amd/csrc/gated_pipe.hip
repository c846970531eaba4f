// Software-pipelined segment build for per-channel (diagonal) gates on gfx950,
// bf16 inputs, d_k = 128, chunk 64: the diagonal transition family of Tab. 1
// (GLA),
//   S_t = diag(exp(g_t)) S_{t-1} + k_t v_t^T,   o_t = S_t^T q_t   (Eq. (2)).
//
// Chunked form (per chunk of 64 tokens, incoming state S0; B_t = per-channel
// inclusive prefix of the gate inside the chunk):
//   O = (Q . exp(B)) S0 + A V,   A_ti = sum_c q_tc k_ic exp(B_tc - B_ic) (i <= t)
//   S <- exp(B_last) . S0 + (K . exp(B_last - B))^T V.
// The segment operator of Tab. 3 is diagonal; its logarithm, the per-channel
// gate sum, is the cache's log_decay.
//
// Gates in the scores.  A is formed over 16-token tiles with the gate of query
// tile tq referred to s_tq, the cumulative gate before the tile: the query
// side is q_t exp(B_t - s_tq) (at most 1), the key side k_i exp(s_tq - B_i).
// Inside the diagonal tile the key factor is at least 1 and bounded by the
// tile's own decay; for an earlier key tile tk it is k_i exp(s_tk - B_i) times
// exp(s_tq - s_tk) <= 1.  So every channel's gate sum over 16 consecutive
// tokens must stay above about -87 (float32 range).  Every exponential of the
// chunk comes from two per element, exp(x) and exp(-x) of the in-tile prefix x:
// the tile factors are the last lane's exp(x), and exp(s_t), exp(B_last - s_t)
// are their products.  Both score operands are kept as bf16 hi + lo (three
// passes), so a score whose q . k terms cancel keeps its float32 accuracy; the
// decayed operands of the state update and of the inter-chunk term are rounded
// to bf16 once, as the inputs are.
//
// Organisation.  One workgroup of 8 waves runs one (segment, v-head,
// 64-column block) chain, software-pipelined two deep:
//   waves 0-1  state columns (32 each) of chunk c: outputs and the state update
//   waves 2-3  HBM loads, half a chunk each: the q, k and gate rows of chunk
//              c + 2, staged into LDS once the producers hold chunk c + 1's;
//              the gates are turned into their in-tile prefix on the way, and
//              the segment's log_decay summed
//   waves 4-7  chunk c + 1, one 32-channel slice of d_k each: the exponentials
//              of the staged gate prefix, the gate-scaled operands, their
//              share of the score tiles (one 32-deep contraction step each),
//              (Q . exp(B)) and (K . exp(B_last - B))^T of their channels, and
//              the row decays exp(B_last).  Each leaves its partial score
//              tiles in an LDS slab; after R1 each sums a quarter of the tiles.
// One barrier before the loop (chunk 0 staged), three LDS-only barriers per
// iteration: R0 (the producers hold chunk c + 1's staged rows in registers, so
// the staging area takes chunk c + 2's), R1 (partial scores written; the
// state waves are done with chunk c's operands), B2 (chunk c + 1's operands
// written), and one after the loop.  Every operand buffer is single: the
// state waves read chunk c's before R1, the producers write chunk c + 1's
// after it.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "family.hpp"
#include "frag32.hpp"

namespace hypic {

namespace {

using namespace f32frag;

constexpr int kThreads = 512;
constexpr int C = 64;      // tokens per chunk
constexpr int DK = 128;    // channels: four producer slices of 32
constexpr int NCOL = 64;   // state columns per workgroup
constexpr int NM = DK / 32;
constexpr int NU = DK / 16;
constexpr float kLog2e = 1.44269504088896341f;
constexpr float kLn2 = 0.693147180559945309f;
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

// ---- LDS plan (bytes) --------------------------------------------------------
struct Lds {
  static constexpr int FB = FR * 2;               // bytes of one fragment
  static constexpr int NW = 2 * NU;               // Q . exp(B): (32-token tile, 16-deep step)
  static constexpr int NKT = NM * 4;              // (K . exp(B_last - B))^T: (rho tile, token step)
  static constexpr int O_Q = 0;
  static constexpr int O_KT = O_Q + NW * FB;
  static constexpr int O_QK = O_KT + NKT * FB;    // A^T as B fragments, 6 fragments
  static constexpr int O_RD = O_QK + 6 * FB;      // exp(B_last) per true channel
  static constexpr int SLB = 10 * 64 * 16;        // one wave's 10 partial score tiles (float32)
  static constexpr int O_SL = O_RD + DK * 4;      // partial score tiles of waves 4-7
  static constexpr int O_TF = O_SL + 4 * SLB;     // tile factors of waves 4-7 (tile, row, 8 channels)
  // the next chunk's q, k (bf16) and gate (float32) rows, staged by the loader
  // waves; rows padded by 16 bytes so that 16 lanes reading 16 rows hit
  // distinct banks
  static constexpr int RQK = DK * 2 + 16;         // bytes per q / k row
  static constexpr int RG = DK * 4 + 16;          // bytes per gate row
  static constexpr int O_SK = O_TF + 4 * 4 * 4 * 8 * 4;  // (wave, row, tile, 8) floats above
  static constexpr int O_SQ = O_SK + C * RQK;
  static constexpr int O_SG = O_SQ + C * RQK;
  static constexpr int TOTAL = O_SG + C * RG;
  static_assert(TOTAL <= 160 * 1024, "LDS budget");
};

struct Chain {
  int seg, h, hk, lo, hi, nc, cb;
  long sh;         // seg * h_v + h
  long qk_stride;  // elements between token rows of q, k
  long v_stride;   // elements between token rows of v, o
};

__device__ __forceinline__ int chunk_len(const Chain& ch, int c) {
  const int r = ch.hi - (ch.lo + c * C);
  return (r < C) ? r : C;
}

// accumulator of score tile (query tile tq, key tile tk <= tq)
__device__ __forceinline__ constexpr int pair_idx(int tq, int tk) { return tq * (tq + 1) / 2 + tk; }

// =============================================================================
// waves 4-7: chunk c + 1, channels 32u .. 32u + 31
// =============================================================================
template <int DV>
__device__ __forceinline__ void producer_wave(const FamArgs& args, const Chain& ch,
                                              unsigned char* smem, int lane, int u) {
  using LP = Lds;
  const int g = lane >> 4, r = lane & 15;
  // this lane's part of the staged rows: channels 32u + 8g .. +7
  const unsigned char* sk = smem + LP::O_SK + (32 * u + 8 * g) * 2;
  const unsigned char* sq = smem + LP::O_SQ + (32 * u + 8 * g) * 2;
  const unsigned char* sgt = smem + LP::O_SG + (32 * u + 8 * g) * 4;
  u16* fQ = reinterpret_cast<u16*>(smem + LP::O_Q);
  u16* fKt = reinterpret_cast<u16*>(smem + LP::O_KT);
  u16* fQK = reinterpret_cast<u16*>(smem + LP::O_QK);
  float* rd = reinterpret_cast<float*>(smem + LP::O_RD);
  float* slab = reinterpret_cast<float*>(smem + LP::O_SL);
  // this lane row's tile factors (the same on the row's 16 lanes): 8 channels
  // of tile t at tf + 8 t
  float* tf = reinterpret_cast<float*>(smem + LP::O_TF) + (u * 4 + g) * 32;
  auto tfac = [&](int t, float (&f)[8]) __attribute__((always_inline)) {
    const float4 a = *reinterpret_cast<const float4*>(tf + 8 * t);
    const float4 b = *reinterpret_cast<const float4*>(tf + 8 * t + 4);
    f[0] = a.x; f[1] = a.y; f[2] = a.z; f[3] = a.w;
    f[4] = b.x; f[5] = b.y; f[6] = b.z; f[7] = b.w;
  };

  // The score tiles (query tile 0, key tile 1) and (2, 3) lie above the
  // diagonal inside fragments that are read; they stay zero.
  if (u == 0) {
    *reinterpret_cast<u16x4*>(fQK + scatter_off(tri_idx(0, 1), 0, lane)) = pack4(0.f, 0.f, 0.f, 0.f);
    *reinterpret_cast<u16x4*>(fQK + scatter_off(tri_idx(1, 3), 0, lane)) = pack4(0.f, 0.f, 0.f, 0.f);
  }

  lds_barrier();  // P0: chunk 0 is staged

  for (int it = -1; it < ch.nc; ++it) {
    const int p = it + 1;
    const bool active = p < ch.nc;
    // lane (g, r) of tile t: token 16t + r, channels 32u + 8g .. +7, from
    // the staged rows (rows past the chunk hold a repeated row: masked)
    uint4 kr[4], qr[4];
    float4 gr[4][2];
    if (active) {
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int tok = 16 * t + r;
        kr[t] = *reinterpret_cast<const uint4*>(sk + tok * LP::RQK);
        qr[t] = *reinterpret_cast<const uint4*>(sq + tok * LP::RQK);
        gr[t][0] = *reinterpret_cast<const float4*>(sgt + tok * LP::RG);
        gr[t][1] = *reinterpret_cast<const float4*>(sgt + tok * LP::RG + 16);
      }
    }
    lds_barrier();  // R0: the staged rows are in registers
    uint4 qe[4];        // Q . exp(B) of tile t, bf16
    u16x4 kd[4][2];     // (K . exp(B_last - B))^T tiles (token tile t, rho half h)
    float rdv[8];       // exp(B_last) of this lane row's channels
    if (active) {
      const int n = chunk_len(ch, p);
      bool keep[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) keep[t] = 16 * t + r < n;

      // Per tile, from the staged in-tile prefix x of the gate (log2 units):
      // exp(x) for the query side, the key side referred to the tile's start,
      // k_i exp(-x_i), and the tile factor F_t = exp(s_{t+1} - s_t), exp(x) of
      // the tile's last token
      float E[4][8], kk[4][8];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        float F[8];
        const float gv[8] = {gr[t][0].x, gr[t][0].y, gr[t][0].z, gr[t][0].w,
                             gr[t][1].x, gr[t][1].y, gr[t][1].z, gr[t][1].w};
        float kf[8];
        unpack8(mask4(kr[t], keep[t]), kf);
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          E[t][j] = __builtin_amdgcn_exp2f(gv[j]);
          kk[t][j] = kf[j] * __builtin_amdgcn_exp2f(-gv[j]);
          F[j] = row_last(E[t][j]);
        }
        if (r == 0) {
          *reinterpret_cast<float4*>(tf + 8 * t) = make_float4(F[0], F[1], F[2], F[3]);
          *reinterpret_cast<float4*>(tf + 8 * t + 4) = make_float4(F[4], F[5], F[6], F[7]);
        }
      }
      // this slice's share of the score tiles, query tile by query tile, each
      // left in this wave's slab as soon as it is formed
      float* sl = slab + (u * 10 * 64 + lane) * 4;
#pragma unroll
      for (int tq = 0; tq < 4; ++tq) {
        float qf[8], qq[8];
        unpack8(mask4(qr[tq], keep[tq]), qf);
#pragma unroll
        for (int j = 0; j < 8; ++j) qq[j] = qf[j] * E[tq][j];
        const Split8 Qs = split8(qq);
        *reinterpret_cast<f32x4*>(sl + pair_idx(tq, tq) * 256) =
            mma16_x3(split8(kk[tq]), Qs, f32x4{0.f, 0.f, 0.f, 0.f});
        // f = exp(s_tq - s_tk) for tk = tq - 1 down to 0
        float f[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) f[j] = 1.f;
#pragma unroll
        for (int tk = tq - 1; tk >= 0; --tk) {
          float ks[8], F[8];
          tfac(tk, F);
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            f[j] *= F[j];
            ks[j] = kk[tk][j] * f[j];
          }
          *reinterpret_cast<f32x4*>(sl + pair_idx(tq, tk) * 256) =
              mma16_x3(split8(ks), Qs, f32x4{0.f, 0.f, 0.f, 0.f});
        }
        // Q . exp(B) = (q exp(B - s_tq)) exp(s_tq); f = exp(s_tq) now
        bf16x8 qb;
#pragma unroll
        for (int j = 0; j < 8; ++j) qb[j] = static_cast<__bf16>(qq[j] * f[j]);
        qe[tq] = __builtin_bit_cast(uint4, qb);
      }
      // (K . exp(B_last - B))^T: k_i exp(s_t - B_i) exp(B_last - s_t), with
      // d = exp(B_last - s_t) = F_t F_{t+1} .. F_3
      // selectors of the transposes: B operand of 16x16x32, lane (g, n) slot j
      // is 1 where 8g + j == 16h + n with bits 2, 3 swapped (the columns come
      // out in rho order)
      bf16x8 esel[2];
      {
        const int pn = (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1);
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
          for (int j = 0; j < 8; ++j)
            esel[h][j] = static_cast<__bf16>((8 * g + j == 16 * h + pn) ? 1.f : 0.f);
      }
      float d[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) d[j] = 1.f;
#pragma unroll
      for (int t = 3; t >= 0; --t) {
        bf16x8 kb;
        float F[8];
        tfac(t, F);
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          d[j] *= F[j];
          kb[j] = static_cast<__bf16>(kk[t][j] * d[j]);
        }
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const f32x4 x4 = mma16(kb, esel[h], f32x4{0.f, 0.f, 0.f, 0.f});
          kd[t][h] = pack4(x4[0], x4[1], x4[2], x4[3]);
        }
      }
#pragma unroll
      for (int j = 0; j < 8; ++j) rdv[j] = d[j];  // exp(B_last)
    }
    lds_barrier();  // R1: the partial score tiles are written; the state
                    // waves are done with chunk c's operands
    if (active) {
      // Q . exp(B) fragments: the 16 bytes of lane (g, r) of tile (t, u) are
      // slot group g%2 of lane 16(t%2) + r of fragment (t/2, 2u + g/2)
#pragma unroll
      for (int t = 0; t < 4; ++t)
        *reinterpret_cast<uint4*>(fQ + ((t >> 1) * NU + 2 * u + (g >> 1)) * FR +
                                  (32 * (g & 1) + 16 * (t & 1) + r) * 8) = qe[t];
      // the four slices' partial tiles summed, wave u taking tiles 3u .. (tile
      // pairs (0,0) (1,0) (1,1) | (2,0) (2,1) (2,2) | (3,0) (3,1) | (3,2) (3,3));
      // A^T as B fragments (key step tk, query tile tq / 2): the tile holds
      // A[16tq + r][16tk + 4g + e]; kept where key <= query
#pragma unroll
      for (int tq = 0; tq < 4; ++tq)
#pragma unroll
        for (int tk = 0; tk <= tq; ++tk) {
          const int i = pair_idx(tq, tk);
          if (((i < 6) ? i / 3 : 2 + (i - 6) / 2) != u) continue;
          f32x4 a = *reinterpret_cast<const f32x4*>(slab + (i * 64 + lane) * 4);
#pragma unroll
          for (int w = 1; w < 4; ++w)
            a += *reinterpret_cast<const f32x4*>(slab + ((w * 10 + i) * 64 + lane) * 4);
          float v[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = (tk < tq || 4 * g + e <= r) ? a[e] : 0.f;
          *reinterpret_cast<u16x4*>(fQK + scatter_off(tri_idx(tq >> 1, tk), tq & 1, lane)) =
              pack4(v[0], v[1], v[2], v[3]);
        }
      // the transposed decayed keys: fragment (rho tile u, token step t)
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int h = 0; h < 2; ++h)
          *reinterpret_cast<u16x4*>(fKt + scatter_off(u * 4 + t, h, lane)) = kd[t][h];
      if (r == 0) {
        *reinterpret_cast<float4*>(rd + 32 * u + 8 * g) = make_float4(rdv[0], rdv[1], rdv[2], rdv[3]);
        *reinterpret_cast<float4*>(rd + 32 * u + 8 * g + 4) =
            make_float4(rdv[4], rdv[5], rdv[6], rdv[7]);
      }
    }
    lds_barrier();  // B2
  }
  lds_barrier();  // E0
}

// =============================================================================
// waves 0-1: the state update of chunk c
// =============================================================================
template <int DV>
__device__ __forceinline__ void state_wave(const FamArgs& args, const Chain& ch,
                                           unsigned char* smem, int lane, int col0) {
  using LP = Lds;
  const int g2 = lane >> 5, n32 = lane & 31;
  const u16* fQ = reinterpret_cast<const u16*>(smem + LP::O_Q);
  const u16* fKt = reinterpret_cast<const u16*>(smem + LP::O_KT);
  const u16* fQK = reinterpret_cast<const u16*>(smem + LP::O_QK);
  const float* rd = reinterpret_cast<const float*>(smem + LP::O_RD);
  const u16* vg = static_cast<const u16*>(args.v) + ch.h * DV + col0;
  u16* og = static_cast<u16*>(args.o);

  // state columns col0 .. col0 + 31, all d_k rows (order rho); a build starts
  // from zero
  f32x16 st[NM];
#pragma unroll
  for (int m = 0; m < NM; ++m) st[m] = zero16();
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
    const int c0 = ch.lo + c * C, n = chunk_len(ch, c);
    load_tile32<2>(vr[0], vg, ch.v_stride, c0, n, 0, lane);
    load_tile32<2>(vr[1], vg, ch.v_stride, c0, n, 1, lane);
  };
  if (ch.nc > 0) prefetch(0);
  lds_barrier();  // P0

  for (int it = -1; it < ch.nc; ++it) {
    const int c = it;
    const bool active = c >= 0;
    lds_barrier();  // R0
    bf16x8 vB[4];  // V (this wave's columns) as fragments over tokens
    if (active) {
      const int c0 = ch.lo + c * C, n = chunk_len(ch, c);
      // lane (g2, n) of fragment s holds V[slot token][col0 + n], by exact
      // products with the identity
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const bool keep = n == C || 32 * t + n32 < n;
        f32x16 acc = mma32(masked(vr[t][0], keep), isel[0], zero16());
        acc = mma32(masked(vr[t][1], keep), isel[1], acc);
        vB[2 * t] = frag_of(acc, 0);
        vB[2 * t + 1] = frag_of(acc, 1);
      }
      if (c + 1 < ch.nc) prefetch(c + 1);
      // S0 as bf16 operands (step u over rho)
      bf16x8 s0[NU];
#pragma unroll
      for (int u = 0; u < NU; ++u) s0[u] = frag_of(st[u >> 1], u & 1);
      // O^T = S0^T (Q . exp(B))^T + V^T A^T; lane (g2, n) holds
      // O[token 32tq + n][col0 + 8b + 4g2 + i]
#pragma unroll
      for (int tq = 0; tq < 2; ++tq) {
        f32x16 acc = zero16();
#pragma unroll
        for (int u = 0; u < NU; ++u) acc = mma32(s0[u], ldf(fQ, tq * NU + u, lane), acc);
#pragma unroll
        for (int s = 0; s < 2 * tq + 2; ++s)
          acc = mma32(vB[s], ldf(fQK, tri_idx(tq, s), lane), acc);
        const int row = 32 * tq + n32;
        if (og != nullptr && row < n) {
          u16* dst = og + (static_cast<long>(c0) + row) * ch.v_stride + ch.h * DV + col0 + 4 * g2;
#pragma unroll
          for (int b = 0; b < 4; ++b) {
            u16x4 o4;
#pragma unroll
            for (int i = 0; i < 4; ++i) o4[i] = bf16_bits(acc[4 * b + i]);
            *reinterpret_cast<u16x4*>(dst + 8 * b) = o4;
          }
        }
      }
    }
    if (active) {
      // S <- exp(B_last) . S0 + (K . exp(B_last - B))^T V
#pragma unroll
      for (int m = 0; m < NM; ++m) {
        f32x16 acc;
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          const float4 dv =
              *reinterpret_cast<const float4*>(rd + 32 * m + 16 * (b >> 1) + 8 * g2 + 4 * (b & 1));
          acc[4 * b] = st[m][4 * b] * dv.x;
          acc[4 * b + 1] = st[m][4 * b + 1] * dv.y;
          acc[4 * b + 2] = st[m][4 * b + 2] * dv.z;
          acc[4 * b + 3] = st[m][4 * b + 3] * dv.w;
        }
#pragma unroll
        for (int s = 0; s < 4; ++s) acc = mma32(ldf(fKt, m * 4 + s, lane), vB[s], acc);
        st[m] = acc;
      }
    }
    lds_barrier();  // R1
    lds_barrier();  // B2
  }
  lds_barrier();  // E0

  if (args.S_out != nullptr) {
    float* so = args.S_out + ch.sh * DK * DV + col0 + n32;
#pragma unroll
    for (int m = 0; m < NM; ++m)
#pragma unroll
      for (int e = 0; e < 16; ++e) so[true_row(m, e, g2) * DV] = st[m][e];
  }
}

// =============================================================================
// waves 2-3: HBM loads, staged into LDS
// =============================================================================
// Loader w takes tokens 32w .. 32w + 31 of a chunk: its q and k rows (4 rows
// of 256 bytes per instruction) and its gate rows, lanes 0-31 tile 2w and
// lanes 32-63 tile 2w + 1 (one token of each per instruction, 4 channels a
// lane), so that every load reads whole rows and each lane holds whole tiles
// of its channels.
__device__ __forceinline__ void loader_load(u32x4 (&buf)[32], const FamArgs& args,
                                            const Chain& ch, int c, int lane, int w) {
  const int c0 = ch.lo + c * C, n = chunk_len(ch, c);
  const u16* kb = static_cast<const u16*>(args.k) + ch.hk * DK + 8 * (lane & 15);
  const u16* qb = static_cast<const u16*>(args.q) + ch.hk * DK + 8 * (lane & 15);
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int tok = 32 * w + 4 * i + (lane >> 4);
    const long row = c0 + ((tok < n) ? tok : n - 1);
    buf[i] = *reinterpret_cast<const u32x4*>(kb + row * ch.qk_stride);
    buf[8 + i] = *reinterpret_cast<const u32x4*>(qb + row * ch.qk_stride);
  }
  const float* gb = args.gate + static_cast<long>(ch.h) * DK + 4 * (lane & 31);
  const long gs = static_cast<long>(args.h_v) * DK;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int tok = 32 * w + 16 * (lane >> 5) + i;
    const long row = c0 + ((tok < n) ? tok : n - 1);
    buf[16 + i] = *reinterpret_cast<const u32x4*>(gb + row * gs);
  }
}

// The gate rows in place as the in-tile inclusive prefix of the gate (log2
// units; tokens past the chunk carry none), and the tile's channel sums added
// to lsum.
__device__ __forceinline__ void gate_prefix(u32x4 (&buf)[32], float (&lsum)[4], int n, int lane,
                                            int w) {
  float run[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const bool keep = 32 * w + 16 * (lane >> 5) + i < n;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      run[e] += keep ? __uint_as_float(buf[16 + i][e]) * kLog2e : 0.f;
      buf[16 + i][e] = __float_as_uint(run[e]);
    }
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) lsum[e] += run[e];
}

__device__ __forceinline__ void loader_stage(const u32x4 (&buf)[32], unsigned char* smem,
                                             int lane, int w) {
  using LP = Lds;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int off = (32 * w + 4 * i + (lane >> 4)) * LP::RQK + 16 * (lane & 15);
    *reinterpret_cast<u32x4*>(smem + LP::O_SK + off) = buf[i];
    *reinterpret_cast<u32x4*>(smem + LP::O_SQ + off) = buf[8 + i];
  }
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int off = (32 * w + 16 * (lane >> 5) + i) * LP::RG + 16 * (lane & 31);
    *reinterpret_cast<u32x4*>(smem + LP::O_SG + off) = buf[16 + i];
  }
}

// A chunk's rows are loaded an iteration before they are staged (a load can
// wait at issue while the memory system is busy; this wave has nothing else to
// do) and their gate prefix formed between R1 and B2, when the producers'
// own arithmetic is done.  Chunk c + 2 is staged in iteration c once the
// producers have moved chunk c + 1's rows into registers (R0), and read by
// them after B2.
__device__ __forceinline__ void loader_wave(const FamArgs& args, const Chain& ch,
                                            unsigned char* smem, int lane, int w) {
  u32x4 buf[32];
  float lsum[4] = {0.f, 0.f, 0.f, 0.f};  // this lane's tile of its channels, summed (log2 units)
  if (ch.nc > 0) {
    loader_load(buf, args, ch, 0, lane, w);
    gate_prefix(buf, lsum, chunk_len(ch, 0), lane, w);
    loader_stage(buf, smem, lane, w);
    if (ch.nc > 1) loader_load(buf, args, ch, 1, lane, w);
  }
  lds_barrier();  // P0
  if (ch.nc > 1) gate_prefix(buf, lsum, chunk_len(ch, 1), lane, w);
  for (int it = -1; it < ch.nc; ++it) {
    lds_barrier();  // R0: the producers hold chunk it + 1's rows
    if (it + 2 < ch.nc) {
      loader_stage(buf, smem, lane, w);
      if (it + 3 < ch.nc) loader_load(buf, args, ch, it + 3, lane, w);
    }
    lds_barrier();  // R1
    // the gate prefix of the rows just loaded, while the producers store
    if (it + 3 < ch.nc) gate_prefix(buf, lsum, chunk_len(ch, it + 3), lane, w);
    lds_barrier();  // B2
  }
  // the segment's per-channel gate sums: lanes l and l + 32 of the two
  // loaders hold the four tiles of channels 4(l % 32) .. +3
  float* part = reinterpret_cast<float*>(smem + Lds::O_SL);
#pragma unroll
  for (int e = 0; e < 4; ++e) lsum[e] += __shfl_xor(lsum[e], 32, 64);
  if (w == 1 && lane < 32)
    *reinterpret_cast<float4*>(part + 4 * lane) = make_float4(lsum[0], lsum[1], lsum[2], lsum[3]);
  lds_barrier();  // E0
  if (w == 0 && lane < 32 && args.log_decay != nullptr && ch.cb == 0) {
    const float4 o = *reinterpret_cast<const float4*>(part + 4 * lane);
    float* ld = args.log_decay + ch.sh * DK + 4 * lane;
    *reinterpret_cast<float4*>(ld) = make_float4((lsum[0] + o.x) * kLn2, (lsum[1] + o.y) * kLn2,
                                                 (lsum[2] + o.z) * kLn2, (lsum[3] + o.w) * kLn2);
  }
}

__device__ __forceinline__ int segment_of(const FamArgs& a, int rank) {
  return a.n_inline > 0 ? static_cast<int>(a.order_inline[rank]) : a.order[rank];
}

// The chain of workgroup blockIdx.x, n_cb workgroups (64-column blocks) per
// (segment, v-head).  Workgroups are dealt to the 8 XCDs round-robin.  A unit
// is every workgroup that reads one q/k head's tokens (the column blocks of the
// group's v-head chains); a unit's workgroups are numbered to land on one XCD
// back to back, so they share its L2 for q and k; units past the last full
// group of 8 keep linear order.
template <int DV>
__device__ __forceinline__ Chain make_chain(const FamArgs& args) {
  constexpr int n_cb = DV / NCOL;
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
  Chain ch;
  ch.h = chain % args.h_v;
  ch.cb = cb;
  ch.seg = segment_of(args, chain / args.h_v);
  int lo = args.cu_seqlens[ch.seg], hi = args.cu_seqlens[ch.seg + 1];
  lo = (lo < 0) ? 0 : ((lo > args.n_tokens) ? args.n_tokens : lo);
  hi = (hi < lo) ? lo : ((hi > args.n_tokens) ? args.n_tokens : hi);
  ch.lo = lo;
  ch.hi = hi;
  ch.nc = (hi - lo + C - 1) / C;
  ch.hk = ch.h / args.group;
  ch.sh = static_cast<long>(ch.seg) * args.h_v + ch.h;
  ch.qk_stride = static_cast<long>(args.h_qk) * DK;
  ch.v_stride = static_cast<long>(args.h_v) * DV;
  return ch;
}

template <int DV>
__global__ __launch_bounds__(kThreads, 1) void diag_pipe_kernel(FamArgs args) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int lane = tid & 63;
  const Chain ch = make_chain<DV>(args);
  const int cb = ch.cb;

  if (wave < 2)
    state_wave<DV>(args, ch, smem, lane, cb * NCOL + 32 * wave);
  else if (wave < 4)
    loader_wave(args, ch, smem, lane, wave - 2);
  else
    producer_wave<DV>(args, ch, smem, lane, wave - 4);
}

template <int DV>
hipError_t launch_t(const FamArgs& a, int n_items, hipStream_t s) {
  constexpr int bytes = Lds::TOTAL;
  // one-time (thread-safe static initialisation) opt-in to more than 64 KiB of LDS
  static const hipError_t attr = hipFuncSetAttribute(
      reinterpret_cast<const void*>(&diag_pipe_kernel<DV>),
      hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL(diag_pipe_kernel<DV>, dim3(n_items), dim3(kThreads), bytes, s, a);
  return hipGetLastError();
}

// #############################################################################
// The scalar family (RetNet, Lightning-2, Mamba2 rows of Tab. 1):
//   S_t = exp(a_t) S_{t-1} + k_t v_t^T,   o_t = S_t^T q_t,
// per chunk (b = prefix of the gate inside the chunk, gamma = exp(b)):
//   O = diag(gamma) Q S0 + (tril(Q K^T) . Gamma) V,  Gamma_ti = exp(b_t - b_i)
//   S <- gamma_last S0 + K^T diag(exp(b_last - b)) V.
// A scalar gate factors out of the scores, so q and k enter the matrix cores
// exactly and every score tile is one bf16 pass over all of d_k: the producers
// split the ten tiles among them whole, with no partial sums.  The state waves
// apply gamma to Q S0 and exp(b_last - b) to V, as the GDN state update does.
// Same organisation as the diagonal kernel: waves 0-1 state columns of chunk
// c, waves 2-3 loaders (q and k rows of chunk c + 2, the gate prefix), waves
// 4-7 producers of chunk c + 1; barriers P0, then R0, R1, B2 per iteration.
// #############################################################################
struct SLds {
  static constexpr int FB = FR * 2;
  static constexpr int NW = 2 * NU;        // Q fragments: (32-token tile, 16-deep step)
  static constexpr int NKT = NM * 4;       // K^T fragments: (rho tile, token step)
  static constexpr int O_Q = 0;
  static constexpr int O_KT = O_Q + NW * FB;
  static constexpr int O_QK = O_KT + NKT * FB;  // (tril(Q K^T) . Gamma)^T as B fragments
  // gate ring, one entry per chunk mod 3 (a chunk's gates are read by the
  // producers one iteration and by the state waves the next): b (log2 units),
  // gamma = exp(b), dec = exp(b_last - b)
  static constexpr int GE = 3 * C * 4;     // bytes of one entry
  static constexpr int O_GR = O_QK + 6 * FB;
  static constexpr int RQK = DK * 2 + 16;  // bytes per staged q / k row
  static constexpr int O_SK = O_GR + 3 * GE;
  static constexpr int O_SQ = O_SK + C * RQK;
  static constexpr int TOTAL = O_SQ + C * RQK;
  static_assert(TOTAL <= 160 * 1024, "LDS budget");
};

// ---- waves 2-3: q and k rows of tokens 32w .. 32w + 31; wave 2 also the gates
__device__ __forceinline__ void sloader_load(u32x4 (&buf)[16], float& ga, const FamArgs& args,
                                             const Chain& ch, int c, int lane, int w) {
  const int c0 = ch.lo + c * C, n = chunk_len(ch, c);
  const u16* kb = static_cast<const u16*>(args.k) + ch.hk * DK + 8 * (lane & 15);
  const u16* qb = static_cast<const u16*>(args.q) + ch.hk * DK + 8 * (lane & 15);
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int tok = 32 * w + 4 * i + (lane >> 4);
    const long row = c0 + ((tok < n) ? tok : n - 1);
    buf[i] = *reinterpret_cast<const u32x4*>(kb + row * ch.qk_stride);
    buf[8 + i] = *reinterpret_cast<const u32x4*>(qb + row * ch.qk_stride);
  }
  if (w == 0) {
    const long row = c0 + ((lane < n) ? lane : n - 1);
    ga = (lane < n) ? args.gate[row * args.h_v + ch.h] : 0.f;
  }
}

// stage the rows; wave 2 writes the chunk's gate entry and returns its gate
// sum (natural log)
__device__ __forceinline__ float sloader_stage(const u32x4 (&buf)[16], float ga,
                                               unsigned char* smem, int c, int lane, int w) {
  using LP = SLds;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int off = (32 * w + 4 * i + (lane >> 4)) * LP::RQK + 16 * (lane & 15);
    *reinterpret_cast<u32x4*>(smem + LP::O_SK + off) = buf[i];
    *reinterpret_cast<u32x4*>(smem + LP::O_SQ + off) = buf[8 + i];
  }
  if (w != 0) return 0.f;
  float b = ga * kLog2e;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const float x = __shfl_up(b, off, 64);
    if (lane >= off) b += x;
  }
  const float b_last = __shfl(b, 63, 64);
  float* ge = reinterpret_cast<float*>(smem + LP::O_GR + (c % 3) * LP::GE);
  ge[lane] = b;
  ge[C + lane] = __builtin_amdgcn_exp2f(b);
  ge[2 * C + lane] = __builtin_amdgcn_exp2f(b_last - b);
  return b_last * kLn2;
}

__device__ __forceinline__ void sloader_wave(const FamArgs& args, const Chain& ch,
                                             unsigned char* smem, int lane, int w) {
  u32x4 buf[16];
  float ga = 0.f, ld = 0.f;
  if (ch.nc > 0) {
    sloader_load(buf, ga, args, ch, 0, lane, w);
    ld += sloader_stage(buf, ga, smem, 0, lane, w);
    if (ch.nc > 1) sloader_load(buf, ga, args, ch, 1, lane, w);
  }
  lds_barrier();  // P0
  for (int it = -1; it < ch.nc; ++it) {
    lds_barrier();  // R0: the producers hold chunk it + 1's rows
    if (it + 2 < ch.nc) {
      ld += sloader_stage(buf, ga, smem, it + 2, lane, w);
      if (it + 3 < ch.nc) sloader_load(buf, ga, args, ch, it + 3, lane, w);
    }
    lds_barrier();  // R1
    lds_barrier();  // B2
  }
  if (w == 0 && lane == 0 && args.log_decay != nullptr && ch.cb == 0) args.log_decay[ch.sh] = ld;
}

// ---- waves 4-7: chunk c + 1.  Producer U: the K^T fragments and the Q
// fragments of channels 32U .. 32U + 31, and whole score tiles (query tile
// tq, key tile tk): U = 0: (0,0) (1,0) (1,1); 1: (2,0) (2,1) (2,2); 2: (3,0)
// (3,1); 3: (3,2) (3,3).
template <int U>
struct STiles {
  static constexpr int N = (U < 2) ? 3 : 2;
  static constexpr int first = (U < 2) ? 3 * U : 6 + 2 * (U - 2);  // pair index of the first
  static constexpr int TQ0 = (U == 0) ? 0 : ((U == 1) ? 2 : 3);    // lowest query tile
  static constexpr int NQT = (U == 0) ? 2 : 1;                      // query tiles
  static constexpr int TK0 = (U == 3) ? 2 : 0;                      // lowest key tile
  static constexpr int NKT = (U == 0) ? 2 : ((U == 1) ? 3 : 2);     // key tiles
};
__device__ __forceinline__ constexpr int pair_tq(int i) {
  return (i < 1) ? 0 : ((i < 3) ? 1 : ((i < 6) ? 2 : 3));
}

template <int DV, int U>
__device__ __forceinline__ void sproducer_wave(const FamArgs& args, const Chain& ch,
                                               unsigned char* smem, int lane) {
  using LP = SLds;
  using TL = STiles<U>;
  const int g = lane >> 4, r = lane & 15;
  u16* fQ = reinterpret_cast<u16*>(smem + LP::O_Q);
  u16* fKt = reinterpret_cast<u16*>(smem + LP::O_KT);
  u16* fQK = reinterpret_cast<u16*>(smem + LP::O_QK);
  const unsigned char* sk = smem + LP::O_SK;
  const unsigned char* sq = smem + LP::O_SQ;
  if (U == 0) {
    // the score tiles (query tile 0, key tile 1) and (2, 3) lie above the
    // diagonal inside fragments that are read; they stay zero
    *reinterpret_cast<u16x4*>(fQK + scatter_off(tri_idx(0, 1), 0, lane)) = pack4(0.f, 0.f, 0.f, 0.f);
    *reinterpret_cast<u16x4*>(fQK + scatter_off(tri_idx(1, 3), 0, lane)) = pack4(0.f, 0.f, 0.f, 0.f);
  }
  // selectors of the K^T transposes (rho order, as in the diagonal kernel)
  bf16x8 esel[2];
  {
    const int pn = (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1);
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int j = 0; j < 8; ++j)
        esel[h][j] = static_cast<__bf16>((8 * g + j == 16 * h + pn) ? 1.f : 0.f);
  }
  lds_barrier();  // P0
  for (int it = -1; it < ch.nc; ++it) {
    const int p = it + 1;
    const bool active = p < ch.nc;
    // lane (g, r) of a 16-token tile t and 32-channel step kk: token 16t + r,
    // channels 32kk + 8g .. +7 of the staged rows
    uint4 ks[4], qs[4];                       // this wave's channel slice, tiles 0-3
    uint4 qt[TL::NQT][4], kt[TL::NKT][4];     // the score tiles' rows, all d_k
    if (active) {
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        ks[t] = *reinterpret_cast<const uint4*>(sk + (16 * t + r) * LP::RQK + (32 * U + 8 * g) * 2);
        qs[t] = *reinterpret_cast<const uint4*>(sq + (16 * t + r) * LP::RQK + (32 * U + 8 * g) * 2);
      }
#pragma unroll
      for (int i = 0; i < TL::NQT; ++i)
#pragma unroll
        for (int kk = 0; kk < 4; ++kk)
          qt[i][kk] = *reinterpret_cast<const uint4*>(sq + (16 * (TL::TQ0 + i) + r) * LP::RQK +
                                                      (32 * kk + 8 * g) * 2);
#pragma unroll
      for (int i = 0; i < TL::NKT; ++i)
#pragma unroll
        for (int kk = 0; kk < 4; ++kk)
          kt[i][kk] = *reinterpret_cast<const uint4*>(sk + (16 * (TL::TK0 + i) + r) * LP::RQK +
                                                      (32 * kk + 8 * g) * 2);
    }
    lds_barrier();  // R0: the staged rows are in registers
    u16x4 kd[4][2];    // K^T tiles (token tile t, rho half h)
    u16x4 sc[TL::N];   // the score tiles, masked and packed
    if (active) {
      const int n = chunk_len(ch, p);
      const float* gb = reinterpret_cast<const float*>(smem + LP::O_GR + (p % 3) * LP::GE);
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const bool keep = 16 * t + r < n;
        ks[t] = mask4(ks[t], keep);
        qs[t] = mask4(qs[t], keep);
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const f32x4 x4 = mma16(as_bf(ks[t]), esel[h], f32x4{0.f, 0.f, 0.f, 0.f});
          kd[t][h] = pack4(x4[0], x4[1], x4[2], x4[3]);
        }
      }
#pragma unroll
      for (int j = 0; j < TL::N; ++j) {
        const int i = TL::first + j;
        const int tq = pair_tq(i), tk = i - tq * (tq + 1) / 2;
        const bool kq = 16 * tq + r < n;
        // A = key rows, B = query rows: lane (g, r) holds (Q K^T)[16tq + r][16tk + 4g + e]
        f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < 4; ++kk)
          acc = mma16(as_bf(kt[tk - TL::TK0][kk]), masked(qt[tq - TL::TQ0][kk], kq), acc);
        const float bq = gb[16 * tq + r];
        const float4 bk = *reinterpret_cast<const float4*>(gb + 16 * tk + 4 * g);
        const float bkv[4] = {bk.x, bk.y, bk.z, bk.w};
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          // keys past the chunk have zero rows... unless repeated: masked by position
          const bool ok = (tk < tq || 4 * g + e <= r) && (16 * tk + 4 * g + e < n);
          const float x = acc[e] * __builtin_amdgcn_exp2f(bq - bkv[e]);
          v[e] = ok ? x : 0.f;
        }
        sc[j] = pack4(v[0], v[1], v[2], v[3]);
      }
    }
    lds_barrier();  // R1: the state waves are done with chunk c's operands
    if (active) {
      // Q fragments (the diagonal kernel's layout, unscaled)
#pragma unroll
      for (int t = 0; t < 4; ++t)
        *reinterpret_cast<uint4*>(fQ + ((t >> 1) * NU + 2 * U + (g >> 1)) * FR +
                                  (32 * (g & 1) + 16 * (t & 1) + r) * 8) = qs[t];
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int h = 0; h < 2; ++h)
          *reinterpret_cast<u16x4*>(fKt + scatter_off(U * 4 + t, h, lane)) = kd[t][h];
#pragma unroll
      for (int j = 0; j < TL::N; ++j) {
        const int i = TL::first + j;
        const int tq = pair_tq(i), tk = i - tq * (tq + 1) / 2;
        *reinterpret_cast<u16x4*>(fQK + scatter_off(tri_idx(tq >> 1, tk), tq & 1, lane)) = sc[j];
      }
    }
    lds_barrier();  // B2
  }
}

// ---- waves 0-1: the state update of chunk c -----------------------------------
template <int DV>
__device__ __forceinline__ void sstate_wave(const FamArgs& args, const Chain& ch,
                                            unsigned char* smem, int lane, int col0) {
  using LP = SLds;
  const int g2 = lane >> 5, n32 = lane & 31;
  const u16* fQ = reinterpret_cast<const u16*>(smem + LP::O_Q);
  const u16* fKt = reinterpret_cast<const u16*>(smem + LP::O_KT);
  const u16* fQK = reinterpret_cast<const u16*>(smem + LP::O_QK);
  const u16* vg = static_cast<const u16*>(args.v) + ch.h * DV + col0;
  u16* og = static_cast<u16*>(args.o);

  f32x16 st[NM];
#pragma unroll
  for (int m = 0; m < NM; ++m) st[m] = zero16();
  bf16x8 isel[2];
#pragma unroll
  for (int u = 0; u < 2; ++u)
#pragma unroll
    for (int j = 0; j < 8; ++j)
      isel[u][j] = static_cast<__bf16>((16 * u + 8 * g2 + j == n32) ? 1.f : 0.f);
  uint4 vr[2][2];
  auto prefetch = [&](int c) __attribute__((always_inline)) {
    const int c0 = ch.lo + c * C, n = chunk_len(ch, c);
    load_tile32<2>(vr[0], vg, ch.v_stride, c0, n, 0, lane);
    load_tile32<2>(vr[1], vg, ch.v_stride, c0, n, 1, lane);
  };
  if (ch.nc > 0) prefetch(0);
  lds_barrier();  // P0

  // V^T of the chunk as fragments over tokens (lane (g2, n) holds
  // V[slot][col0 + n], exact products with the identity) and S0 as bf16
  // operands: prepared between R1 and B2 of the previous iteration, while the
  // producers store
  bf16x8 vB[4], s0[NU];
  auto prepare = [&](int c) __attribute__((always_inline)) {
    const int n = chunk_len(ch, c);
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const bool keep = n == C || 32 * t + n32 < n;
      f32x16 acc = mma32(masked(vr[t][0], keep), isel[0], zero16());
      acc = mma32(masked(vr[t][1], keep), isel[1], acc);
      vB[2 * t] = frag_of(acc, 0);
      vB[2 * t + 1] = frag_of(acc, 1);
    }
    if (c + 1 < ch.nc) prefetch(c + 1);
#pragma unroll
    for (int u = 0; u < NU; ++u) s0[u] = frag_of(st[u >> 1], u & 1);
  };
  // O^T = (S0^T Q^T) diag(gamma) + V^T A^T for query tile tq; lane (g2, n)
  // holds O[token 32tq + n][col0 + 8b + 4g2 + i]
  auto outputs = [&](int c, int tq) __attribute__((always_inline)) {
    const int c0 = ch.lo + c * C, n = chunk_len(ch, c);
    const float* ggam = reinterpret_cast<const float*>(smem + LP::O_GR + (c % 3) * LP::GE) + C;
    f32x16 acc = zero16();
#pragma unroll
    for (int u = 0; u < NU; ++u) acc = mma32(s0[u], ldf(fQ, tq * NU + u, lane), acc);
    acc *= ggam[32 * tq + n32];
#pragma unroll
    for (int s = 0; s < 2 * tq + 2; ++s) acc = mma32(vB[s], ldf(fQK, tri_idx(tq, s), lane), acc);
    const int row = 32 * tq + n32;
    if (og != nullptr && row < n) {
      u16* dst = og + (static_cast<long>(c0) + row) * ch.v_stride + ch.h * DV + col0 + 4 * g2;
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        u16x4 o4;
#pragma unroll
        for (int i = 0; i < 4; ++i) o4[i] = bf16_bits(acc[4 * b + i]);
        *reinterpret_cast<u16x4*>(dst + 8 * b) = o4;
      }
    }
  };

  for (int it = -1; it < ch.nc; ++it) {
    const int c = it;
    const bool active = c >= 0;
    // the first output tile while the producers move their staged rows
    if (active) outputs(c, 0);
    lds_barrier();  // R0
    if (active) {
      outputs(c, 1);
      // S <- gamma_last S0 + K^T diag(exp(b_last - b)) V
      const float* gb = reinterpret_cast<const float*>(smem + LP::O_GR + (c % 3) * LP::GE);
      const float* gdec = gb + 2 * C;
      bf16x8 dv[4];
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        const float4 d0 = *reinterpret_cast<const float4*>(gdec + 16 * s + 4 * g2);
        const float4 d1 = *reinterpret_cast<const float4*>(gdec + 16 * s + 8 + 4 * g2);
        const float dd[8] = {d0.x, d0.y, d0.z, d0.w, d1.x, d1.y, d1.z, d1.w};
#pragma unroll
        for (int j = 0; j < 8; ++j)
          dv[s][j] = static_cast<__bf16>(static_cast<float>(vB[s][j]) * dd[j]);
      }
      const float g_last = gb[C + C - 1];
#pragma unroll
      for (int m = 0; m < NM; ++m) {
        f32x16 acc = st[m] * g_last;
#pragma unroll
        for (int s = 0; s < 4; ++s) acc = mma32(ldf(fKt, m * 4 + s, lane), dv[s], acc);
        st[m] = acc;
      }
    }
    lds_barrier();  // R1
    if (c + 1 < ch.nc) prepare(c + 1);
    lds_barrier();  // B2
  }

  if (args.S_out != nullptr) {
    float* so = args.S_out + ch.sh * DK * DV + col0 + n32;
#pragma unroll
    for (int m = 0; m < NM; ++m)
#pragma unroll
      for (int e = 0; e < 16; ++e) so[true_row(m, e, g2) * DV] = st[m][e];
  }
}

template <int DV>
__global__ __launch_bounds__(kThreads, 1) void scalar_pipe_kernel(FamArgs args) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int lane = tid & 63;
  const Chain ch = make_chain<DV>(args);
  if (wave < 2)
    sstate_wave<DV>(args, ch, smem, lane, ch.cb * NCOL + 32 * wave);
  else if (wave < 4)
    sloader_wave(args, ch, smem, lane, wave - 2);
  else if (wave == 4)
    sproducer_wave<DV, 0>(args, ch, smem, lane);
  else if (wave == 5)
    sproducer_wave<DV, 1>(args, ch, smem, lane);
  else if (wave == 6)
    sproducer_wave<DV, 2>(args, ch, smem, lane);
  else
    sproducer_wave<DV, 3>(args, ch, smem, lane);
}

template <int DV>
hipError_t launch_s(const FamArgs& a, int n_items, hipStream_t s) {
  constexpr int bytes = SLds::TOTAL;
  static const hipError_t attr = hipFuncSetAttribute(
      reinterpret_cast<const void*>(&scalar_pipe_kernel<DV>),
      hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL(scalar_pipe_kernel<DV>, dim3(n_items), dim3(kThreads), bytes, s, a);
  return hipGetLastError();
}

}  // namespace

bool diag_pipe_supported(int bf16, int d_k, int d_v, int mode) {
  return bf16 && mode == 0 && d_k == DK && (d_v == 64 || d_v == 128);
}

hipError_t launch_scalar_pipe(const FamArgs& a, int d_v, int n_chains, hipStream_t s) {
  const int64_t n_items = static_cast<int64_t>(n_chains) * a.h_v * (d_v / NCOL);
  if (n_items <= 0) return hipSuccess;
  if (n_items > 0x7fffffff || a.mode != 0) return hipErrorInvalidValue;
  const int n = static_cast<int>(n_items);
  if (d_v == 64) return launch_s<64>(a, n, s);
  return launch_s<128>(a, n, s);
}

hipError_t launch_diag_pipe(const FamArgs& a, int d_v, int n_chains, hipStream_t s) {
  const int64_t n_items = static_cast<int64_t>(n_chains) * a.h_v * (d_v / NCOL);
  if (n_items <= 0) return hipSuccess;
  if (n_items > 0x7fffffff || a.mode != 0) return hipErrorInvalidValue;
  const int n = static_cast<int>(n_items);
  if (d_v == 64) return launch_t<64>(a, n, s);
  return launch_t<128>(a, n, s);
}

}  // namespace hypic
