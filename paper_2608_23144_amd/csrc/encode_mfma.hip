// Encoder seed search with the projection on the matrix cores (C = 64, P <= 8).
//
// For a tile t and seed s the projection b = B_s^T (d .* r) (Eq. (3)) is a dot
// product of u_t = d_t .* r_t with +-1/sqrt(C) basis columns.  Stacking the
// P columns of two seeds as 16 rows and 64 tiles of one column block as
// columns turns one step into a dense [16 x 64] * [64 x 64] product:
//
//   * u is split exactly into three bf16 parts (u = hi + mid + lo, each part
//     truncated from the remainder of the previous one, which loses nothing
//     for an fp32 u), and the +-1 basis entries are exact in bf16, so three
//     v_mfma_f32_16x16x32_bf16 per (tile group, K step) give b with fp32
//     accumulation;
//   * the u fragments stay in registers for the whole seed loop; the +-1
//     fragments of each seed pair are read, already laid out per lane, from a
//     table built once per launch;
//   * the 16 x 64 result is transposed through LDS so that each lane holds
//     the P coefficients of its own tile, with the seed uniform across the
//     wavefront: per-column Cholesky factors are then scalar loads, and the
//     solve, quantization, score and top-k bookkeeping run on the vector ALUs
//     exactly as in the VALU screen.
//
// MFMA operand layout for 16x16x32 bf16 on gfx950: lane l supplies row
// (A) / column (B) l % 16 and the K slice 8*(l/16) .. 8*(l/16)+7; the 16x16
// fp32 result leaves rows 4*(l/16) .. 4*(l/16)+3 of column l % 16 in lane l.
// Both operands use the same coordinate for (lane group, element), so the
// sum over K is the same whichever order the hardware visits K in.
#include <math.h>

#include "awsrc_internal.h"
#include "mfma_bf16.h"
#include "rescore64.h"

namespace awsrc {

// ----------------------------------------------------------------------------
// +-1 basis fragments: frag[pair][ks][lane] = 8 bf16 (4 dwords) of row
// m = lane % 16 (seed 2*pair + m/8, column m % 8) at coordinates
// 32*ks + 8*(lane/16) + e.  Rows of absent seeds or columns are zero.
__global__ void k_mfma_frags(BasisTables bt, int C, int P, int S, u32x4* __restrict__ frag) {
  const int nks = C / 32;
  const int64_t n = (int64_t)((S + 1) / 2 + 2) * nks * 64;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int lane = (int)(i % 64);
  const int ks = (int)((i / 64) % nks);
  const int pair = (int)(i / (64 * nks));
  const int m = lane & 15;
  const int s = 2 * pair + (m >> 3);
  const int p = m & 7;
  u32x4 v = {0u, 0u, 0u, 0u};
  if (s < S && p < P) {
    const int j0 = 32 * ks + 8 * (lane >> 4);
    const uint64_t mk = bt.mask[((size_t)s * P + p) * 2 + (j0 >> 6)] >> (j0 & 63);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint32_t lo = ((mk >> (2 * q)) & 1ull) ? 0xBF80u : 0x3F80u;
      const uint32_t hi = ((mk >> (2 * q + 1)) & 1ull) ? 0xBF80u : 0x3F80u;
      v[q] = lo | (hi << 16);
    }
  }
  frag[i] = v;
}

// ----------------------------------------------------------------------------
// C = 64 screens.  One wavefront (one workgroup) = 64 consecutive rows of one
// column block and one range of seed pairs.  Seed ranges are used only when a
// module has too few row groups to fill the machine (each range costs its own
// tile loads and top lists).
struct ScreenTask {
  int blk, split, pair0, pair1;
  int64_t row0;
};

__device__ __forceinline__ ScreenTask screen_task(const EncodeArgs& a, int rows_per_wave) {
  // Workgroups are dealt to the 8 XCDs round-robin by index.  Give each XCD a
  // contiguous run of work items in column-block-major order, so that the
  // row groups of a column block share one L2 for their factor reads.
  const int64_t nwg = gridDim.x;
  const int64_t xcd = blockIdx.x % 8, q = nwg / 8, rem = nwg % 8;
  const int64_t w = xcd * q + (xcd < rem ? xcd : rem) + blockIdx.x / 8;
  const int nrg = (int)((a.rows + rows_per_wave - 1) / rows_per_wave);
  ScreenTask t;
  t.split = (int)(w % a.nsplit);
  const int64_t rest = w / a.nsplit;
  t.blk = (int)(rest / nrg);
  t.row0 = (rest % nrg) * rows_per_wave;
  const int n_pairs_all = (a.S + 1) / 2;
  const int pp = (n_pairs_all + a.nsplit - 1) / a.nsplit;
  t.pair0 = t.split * pp;
  t.pair1 = t.pair0 + pp < n_pairs_all ? t.pair0 + pp : n_pairs_all;
  return t;
}

// u = d .* r fragments of the 4 groups of 16 tiles (rows row0 + 16 nb + n),
// split in three bf16 parts; rows past the end give zeros.  en[nb] returns
// each tile's weighted energy sum_j d_j r_j^2 (summed over the four lanes
// n, n + 16, n + 32, n + 48 that share the tile's row).
// The u fragments of NB x 16 tiles (rows row0 + 16 nb + n) over the C = 32
// NKS coordinates of column block blk, per-column weights: lane (n, g) holds
// coordinates 32 ks + 8 g .. + 7 of each of its NB rows, split exactly in
// three bf16 parts; en[nb] gets the tile's weighted energy sum_j d_j r_j^2
// (over the four lanes n, n + 16, n + 32, n + 48 that share a row).  Every
// load is issued before any is used: the residual as 2 NB NKS chunks of four
// weights, the column weights as 2 NKS chunks (the same for every row).
template <int C, int NB>
__device__ __forceinline__ void load_u_col(const EncodeArgs& a, int64_t row0, int blk, int n, int g,
                                           u32x4 (&uh)[NB][C / 32], u32x4 (&um)[NB][C / 32],
                                           u32x4 (&ul)[NB][C / 32], float (&en)[NB]) {
  constexpr int NKS = C / 32;
  constexpr int NCH = 2 * NB * NKS;
  int64_t o[NCH];
  bool valid[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int64_t row = row0 + 16 * nb + n;
    valid[nb] = row < a.rows;
    const int64_t rr = valid[nb] ? row : a.rows - 1;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      const int64_t base = rr * a.cols + (int64_t)blk * C + 32 * ks + 8 * g;
      o[2 * (nb * NKS + ks)] = base;
      o[2 * (nb * NKS + ks) + 1] = base + 4;
    }
  }
  gf32x4 dv[2 * NKS];
#pragma unroll
  for (int ks = 0; ks < NKS; ++ks) {
    dv[2 * ks] = gload4f(a.d + (int64_t)blk * C + 32 * ks + 8 * g);
    dv[2 * ks + 1] = gload4f(a.d + (int64_t)blk * C + 32 * ks + 8 * g + 4);
  }
  float rv[NCH][4];
  load_residual4<NCH>(a.W, a.w_dtype, a.W0, o, rv);
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    float e = 0.0f;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      float u[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const float r = rv[2 * (nb * NKS + ks) + (k >> 2)][k & 3];
        const float dj = dv[2 * ks + (k >> 2)][k & 3];
        u[k] = valid[nb] ? dj * r : 0.0f;
        e = fmaf(dj * r, r, e);
      }
      split3(u, uh[nb][ks], um[nb][ks], ul[nb][ks]);
    }
    e += __shfl_xor(e, 16, 64);
    en[nb] = e + __shfl_xor(e, 32, 64);
  }
}

// b of one seed pair for the 64 tiles: rows 4g..4g+3 of each 16 x 16 result
// (seed g/2 of the pair, coefficients 4(g&1)..+3) for the tiles 16 nb + n.
__device__ __forceinline__ void project64(const u32x4& F0, const u32x4& F1, const u32x4 (&uh)[4][2],
                                          const u32x4 (&um)[4][2], const u32x4 (&ul)[4][2], f32x4 (&acc)[4]) {
  const bf16x8 A0 = as_bf16x8(F0), A1 = as_bf16x8(F1);
#pragma unroll
  for (int nb = 0; nb < 4; ++nb) {
    f32x4 c = {0.f, 0.f, 0.f, 0.f};
    c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A0, as_bf16x8(uh[nb][0]), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A0, as_bf16x8(um[nb][0]), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A0, as_bf16x8(ul[nb][0]), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A1, as_bf16x8(uh[nb][1]), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A1, as_bf16x8(um[nb][1]), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A1, as_bf16x8(ul[nb][1]), c, 0, 0, 0);
    acc[nb] = c;
  }
}

// Per-column weights.  The factor of G + eps I is one table entry per seed,
// shared by every tile of the wavefront, and the projections are used where
// the matrix cores leave them: lane (n, g) holds 4 coefficients of seed g/2
// for the tiles 16 nb + n.  One v_permlane16_swap per pair of registers
// trades halves between lane rows g and g^1, after which lane (n, g) holds
// all P coefficients of seed g/2 of the pair for two tiles, 16 nb0 + n and
// 16 (nb0 + 1) + n with nb0 = 2 (g & 1).  A lane thus scores one seed for two
// tiles (one factor read serves both), each tile's even and odd seeds live in
// lanes g and g^2, and the two lanes' lists are merged at the end.
//
// Every candidate gets the forward solve and its bound (screen_fwd); only
// those whose bound reaches the re-score's window below the tile's current
// best are scored in full.  Those few would leave most lanes idle, so each
// lane queues its survivors (w, the seed and which of its tiles) in its own
// LDS ring, and a scoring round takes the oldest entry of every lane that
// has one.  The threshold comes from the tile's best over both of its
// lanes' lists (below).  A lane's entries are scored in seed order, and
// thresholds only rise, so the merged lists agree with those of scoring
// every candidate in the best and in the second wherever the second lies
// inside the re-score's window.  The threshold is lowered by a relative
// 2^-9 (slack_thr) for the fp32 rounding of the bound and the score.
//
// Factor entries reach the wavefront through an LDS ring of the last NR
// pairs (both seeds' whole entries per slot): while pair k is bounded, every
// lane loads one 16-byte piece of pair k+1's entries (lane l takes piece
// l % 22, so the loads and stores need no branch; lanes with the same piece
// store the same value).  The bound reads its seed's entry from the slot of
// pair k, a scoring round reads each entry's from the slot of its pair, and
// rounds run before an entry's slot is reused.  Vector loads and LDS reads
// complete in order, so the waits for them are exact.
//
// With RPB > 0 (a wavefront screens every seed, generator version 1) the
// kernel also runs the fp64 re-score of its 64 tiles (rescore_block64 at PB =
// RPB), in LDS the screen no longer needs, so that the re-score's latency
// overlaps other wavefronts' screening and the lists never leave the chip.
template <bool POW2, int RPB>
__global__ __launch_bounds__(64, 2) void k_screen_col64(EncodeArgs a, const u32x4* __restrict__ frag,
                                                        int stride) {
  constexpr int C = 64;
  constexpr int PB = 8;
  constexpr int NB = PB * (PB - 1) / 2 + PB;      // L and 1/e: what the bound reads
  constexpr int NF = PB * (PB - 1) / 2 + 2 * PB;  // the whole entry (the full score also reads e)
  constexpr int QD = 4;                           // queue slots per lane (a power of two), plus a spare
  constexpr int QW = PB + 1;                      // words per entry: w, then seed + (tile << 16)
  constexpr int NR = 16;                          // factor ring slots (pairs; a power of two)
  static_assert(NF % 4 == 0, "factor pieces are 16 bytes");
  // one LDS buffer: the factor ring and the queues while screening, the
  // re-score's rows after (when fused)
  constexpr int kScreenLds = NR * 2 * NF + (QD + 1) * QW * 64;
  constexpr int kLds = RPB > 0 && kRescoreLds > kScreenLds ? kRescoreLds : kScreenLds;
  __shared__ __attribute__((aligned(16))) float lds[kLds];
  float* fr = lds;                  // [NR][2][NF]
  float* qb = lds + NR * 2 * NF;    // [QD + 1][QW][64]
  const int lane = threadIdx.x;
  const int nbk_cols = (int)(a.cols / C);
  const ScreenTask tk = screen_task(a, 64);
  const int blk = tk.blk, pair0 = tk.pair0, pair1 = tk.pair1;
  const int n = lane & 15, g = lane >> 4;
  const int sh = g >> 1;        // the seed of each pair this lane scores
  const int nb0 = 2 * (g & 1);  // its tiles: 16 nb0 + n and 16 (nb0 + 1) + n
  u32x4 uh[4][2], um[4][2], ul[4][2];
  float en[4];
  load_u_col<64, 4>(a, tk.row0, blk, n, g, uh, um, ul, en);
  const int64_t trow0 = tk.row0 + 16 * nb0 + n;
  const bool tv[2] = {trow0 < a.rows, trow0 + 16 < a.rows};
  const float qmax = (float)((1 << (a.b - 1)) - 1);
  const float inv_qmax = 1.0f / qmax;

  // top two per tile; a lane's seeds increase, so strict comparisons keep the
  // earlier seed first among equal scores
  float tg[2][2] = {{-INFINITY, -INFINITY}, {-INFINITY, -INFINITY}};
  uint32_t ts[2][2] = {{0, 0}, {0, 0}};  // seed words: seed | kEdge flag
  auto insert = [&](int t, float gsc, uint32_t s) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const bool c0 = t == j && gsc > tg[j][0], c1 = t == j && gsc > tg[j][1];
      tg[j][1] = c0 ? tg[j][0] : (c1 ? gsc : tg[j][1]);
      ts[j][1] = c0 ? ts[j][0] : (c1 ? s : ts[j][1]);
      tg[j][0] = c0 ? gsc : tg[j][0];
      ts[j][0] = c0 ? s : ts[j][0];
    }
  };
  // queue: qhead, qlen, and the pair of the head entry (INT_MAX when empty)
  int qhead = 0, qtail = 0, qlen = 0, hp = INT_MAX;
  int nscored = 0;  // candidates this lane scored in full
  auto score_round = [&]() {
    if (qlen > 0) {
      const float* e = &qb[qhead * (QW * 64) + lane];
      float wv[PB];
#pragma unroll
      for (int i = 0; i < PB; ++i) wv[i] = e[i * 64];
      const int code = __float_as_int(e[PB * 64]);
      const int s = code & 0xFFFF;
      const float* fe = &fr[((s >> 1) & (NR - 1)) * (2 * NF) + (s & 1) * NF];
      float f[NF];
#pragma unroll
      for (int i = 0; i < NF / 4; ++i) {
        const f32x4 v = *reinterpret_cast<const f32x4*>(&fe[4 * i]);
        f[4 * i] = v[0]; f[4 * i + 1] = v[1]; f[4 * i + 2] = v[2]; f[4 * i + 3] = v[3];
      }
      bool edge;
      const float gsc = screen_gain_w<PB, POW2, 3>(wv, f, qmax, inv_qmax, &edge);
      insert(code >> 16, gsc, (uint32_t)s | (edge ? kEdge : 0u));
      qhead = (qhead + 1) & (QD - 1);
      --qlen;
      ++nscored;
      // the next entry's seed (any word when the queue is now empty)
      const int nx = __float_as_int(qb[qhead * (QW * 64) + PB * 64 + lane]);
      hp = qlen > 0 ? (nx & 0xFFFF) >> 1 : INT_MAX;
    }
  };

  constexpr int NPC = 2 * NF / 4;  // 16-byte pieces per pair
  const int pc = lane % NPC;
  // the piece's seed within its pair and its byte offset in the seed's entry;
  // the block's rows of the table from a wavefront-uniform base
  const int psel = pc / (NF / 4);
  const uint32_t pofs = 16u * (uint32_t)(pc % (NF / 4)), strideB = 4u * (uint32_t)stride;
  const char* fac_blk = reinterpret_cast<const char*>(a.colfac + (size_t)blk * a.S * stride);
  auto fac_piece = [&](int pr) -> f32x4 {
    const int s = min(2 * pr + psel, a.S - 1);
    return *reinterpret_cast<const f32x4*>(fac_blk + __umul24((uint32_t)s, strideB) + pofs);
  };
  auto fac_store = [&](int pr, const f32x4& v) {
    *reinterpret_cast<f32x4*>(&fr[(pr & (NR - 1)) * (2 * NF) + 4 * pc]) = v;
  };

  // Pruning threshold of each tile: the re-score takes a second seed only
  // when its screened score lies within rescore_window of the best, so a
  // candidate below that window of the tile's current best (over both lanes'
  // lists; lane ^ 32 holds the other seed parity) is never needed, and the
  // window's lower edge only rises.  The threshold takes the window one
  // percent wider, far above the fp32 rounding of either, and the wide
  // window when the best is flagged as a knife edge; in raw units the energy
  // term is 64 times larger.  Lists change only in scoring rounds.
  const float e_raw[2] = {64.0f * en[nb0], 64.0f * en[nb0 + 1]};
  float thr[2] = {-INFINITY, -INFINITY};
  auto update_thr = [&]() {
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const auto r0 = __builtin_amdgcn_permlane32_swap(__float_as_uint(tg[t][0]), __float_as_uint(tg[t][0]), false,
                                                       false);
      const auto r1 = __builtin_amdgcn_permlane32_swap(ts[t][0], ts[t][0], false, false);
      const float og = __uint_as_float(sh ? r0[0] : r0[1]);
      const uint32_t ow = sh ? r1[0] : r1[1];
      const float best = fmaxf(tg[t][0], og);
      const bool edge = ((tg[t][0] >= og ? ts[t][0] : ow) & kEdge) != 0;
      thr[t] = slack_thr(best - 1.01f * rescore_window(best, e_raw[t], edge));
    }
  };

  // Raw units and the software pipeline as in k_screen_pe64: b is left
  // unscaled by 1/sqrt(C) = 1/8 (bound, scale and gain 8, 8 and 64 times
  // larger, rescaled at the end), and the matrix cores project pair k+1
  // while the vector ALUs post-process pair k.
  const u32x4* fp = frag + (size_t)pair0 * 128 + lane;
  // two register sets for the projections and the fragments, swapping roles
  // every pair (the loop runs two pairs per trip, so no copies are needed)
  f32x4 accA[4], accB[4];
  u32x4 FA0 = fp[128], FA1 = fp[192], FB0, FB1;
  project64(fp[0], fp[64], uh, um, ul, accA);
  fac_store(pair0, fac_piece(pair0));
  f32x4 fnext = fac_piece(pair0 + 1);
  auto step = [&](int pair, const f32x4 (&acc)[4], f32x4 (&accN)[4], const u32x4& F0, const u32x4& F1,
                  u32x4& F0n, u32x4& F1n) {
    // orders the last pair's ring accesses before this one's
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    // next pair's factors into its slot (the oldest pair's, whose entries the
    // last pair's rounds have scored), then this pair's global loads (factors
    // and +-1 fragments two pairs ahead) and factor reads, kept ahead of the
    // matrix-core work by the scheduling barrier so that they have the whole
    // pair's work to arrive
    fac_store(pair + 1, fnext);
    fnext = fac_piece(pair + 2);
    F0n = fp[(size_t)(pair - pair0 + 2) * 128];
    F1n = fp[(size_t)(pair - pair0 + 2) * 128 + 64];
    const int s = 2 * pair + sh;
    float f[NB];
    {
      const float* frow = &fr[(pair & (NR - 1)) * (2 * NF) + sh * NF];
#pragma unroll
      for (int i = 0; i < NB / 4; ++i) {
        const f32x4 v = *reinterpret_cast<const f32x4*>(&frow[4 * i]);
        f[4 * i] = v[0]; f[4 * i + 1] = v[1]; f[4 * i + 2] = v[2]; f[4 * i + 3] = v[3];
      }
    }
    __builtin_amdgcn_sched_barrier(0);
    project64(F0, F1, uh, um, ul, accN);
    // this lane's coefficients: tile t = [lower half, upper half]
    float bt[2][PB];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(acc[t][i]), __float_as_uint(acc[t + 2][i]),
                                                        false, false);
        bt[t][i] = __uint_as_float(r[0]);
        bt[t][4 + i] = __uint_as_float(r[1]);
      }
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      float wv[PB];
      const float bnd = screen_fwd<PB>(bt[t], f, wv);
      // a candidate that is not kept goes to the spare slot QD, so the stores
      // need no branch (one basic block keeps the matrix-core instructions
      // interleaved with this work); bitwise: a short-circuit would put the
      // bound under a branch
      const bool keep = (int)(bnd > thr[t]) & (int)tv[t] & (int)(s < a.S);
      float* e = &qb[(keep ? qtail : QD) * (QW * 64) + lane];
#pragma unroll
      for (int i = 0; i < PB; ++i) e[i * 64] = wv[i];
      e[PB * 64] = __int_as_float(s | (t << 16));
      hp = (keep && qlen == 0) ? pair : hp;
      qlen += keep ? 1 : 0;
      qtail = keep ? ((qtail + 1) & (QD - 1)) : qtail;
    }
#pragma unroll
    for (int i = 0; i < 24; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);
    }
    // room for the next pair's two entries, and no entry of the pair whose
    // slot the next pair refills
    if (__ballot(qlen > QD - 2 || hp <= pair + 2 - NR) != 0) {
      do {
        score_round();
      } while (__ballot(qlen > QD - 2 || hp <= pair + 2 - NR) != 0);
      update_thr();
    }
  };
  int pair = pair0;
  for (; pair + 1 < pair1; pair += 2) {
    step(pair, accA, accB, FA0, FA1, FB0, FB1);
    step(pair + 1, accB, accA, FB0, FB1, FA0, FA1);
  }
  if (pair < pair1) step(pair, accA, accB, FA0, FA1, FB0, FB1);
  while (__ballot(qlen > 0) != 0) score_round();
  // the wavefront's count of full scores, added once
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) nscored += __shfl_xor(nscored, m, 64);
  if (lane == 0) atomicAdd(a.scored, (unsigned long long)nscored);

  // merge each tile's lists from lanes g (this seed parity) and g ^ 2 (the
  // other): (gain desc, seed asc)
  auto better = [](float ga, uint32_t sa, float gb, uint32_t sb) {
    return ga > gb || (ga == gb && list_seed(sa) < list_seed(sb));
  };
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const float og0 = __shfl_xor(tg[t][0], 32, 64), og1 = __shfl_xor(tg[t][1], 32, 64);
    const uint32_t os0 = (uint32_t)__shfl_xor((int)ts[t][0], 32, 64), os1 = (uint32_t)__shfl_xor((int)ts[t][1], 32, 64);
    if (sh == 0 && tv[t]) {
      float r0, r1;
      uint32_t q0, q1;
      if (better(tg[t][0], ts[t][0], og0, os0)) {
        r0 = tg[t][0]; q0 = ts[t][0];
        const bool m = better(tg[t][1], ts[t][1], og0, os0);
        r1 = m ? tg[t][1] : og0; q1 = m ? ts[t][1] : os0;
      } else {
        r0 = og0; q0 = os0;
        const bool m = better(tg[t][0], ts[t][0], og1, os1);
        r1 = m ? tg[t][0] : og1; q1 = m ? ts[t][0] : os1;
      }
      if constexpr (RPB > 0) {
        // for the lane of the tile's row (below); the queues are drained
        float* st = &lds[4 * (16 * (nb0 + t) + n)];
        st[0] = r0 * (1.0f / 64.0f);  // back to gain units
        st[1] = r1 * (1.0f / 64.0f);
        st[2] = __uint_as_float(q0);
        st[3] = __uint_as_float(q1);
      } else {
        const int64_t at = (((trow0 + 16 * t) * nbk_cols + blk) * a.nsplit + tk.split) * kTop;
        a.top_gain[at + 0] = r0 * (1.0f / 64.0f);  // back to gain units
        a.top_gain[at + 1] = r1 * (1.0f / 64.0f);
        a.top_seed[at + 0] = q0;
        a.top_seed[at + 1] = q1;
      }
    }
  }
  if constexpr (RPB > 0) {
    static_assert(kTop == 2, "two kept seeds per tile");
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    // lane = the tile's row in the group (rows past the end read values
    // they never use)
    const f32x4 v = *reinterpret_cast<const f32x4*>(&lds[4 * lane]);
    const float mg[kTop] = {v[0], v[1]};
    const uint32_t ms[kTop] = {__float_as_uint(v[2]), __float_as_uint(v[3])};
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    rescore_block64<RPB>(a, blk, tk.row0, mg, ms, lds);
  }
}

// ----------------------------------------------------------------------------
// C = 128, per-column weights.  The u fragments of a 128-coordinate tile take
// twice the registers, so a wavefront holds 32 consecutive rows of one column
// block (2 groups of 16 tiles x 4 K steps x 3 bf16 parts) and gives the two
// seeds of a pair to its two lane halves: lane = (seed of the pair, tile).
// The seed is then uniform per half only, so each lane reads its seed's
// per-column factors with vector loads (two addresses per wavefront).  The
// bound works on raw b (without the 1/sqrt(128) of the basis), so it comes
// out C times larger and the threshold is scaled by C instead; a scoring
// round scales b by 1/sqrt(128) and solves again (not a power of two, so
// raw units would round the fp16 scale differently).
//
// Every candidate gets the forward solve with its seed's factor and the bound
// b^T (G + eps I)^-1 b on every rounding of its fit (screen_fwd); those whose
// bound reaches the re-score window below the tile's current best (over both
// halves) wait in one queue per wavefront, appended in step order, and a
// scoring round takes the 64 oldest, one per lane (each reading its entry's
// factor again), after which each owner lane inserts its results in queue
// order (seed order), as in the per-element screen.  Each half keeps its own
// top two, merged at the end.
template <int C, bool POW2>
__global__ __launch_bounds__(64, 2) void k_screen_mfma_halves(EncodeArgs a, const u32x4* __restrict__ frag,
                                                              int stride) {
  constexpr int PB = 8;
  constexpr int NKS = C / 32;
  constexpr int TS = 12;  // LDS stride (floats) of one lane's coefficients
  constexpr int LS = PB * (PB - 1) / 2;
  constexpr int NF = LS + 2 * PB;   // the whole factor entry (the full score also reads e)
  constexpr int NBD = LS + PB;      // L and 1/e: what the bound reads
  constexpr int QC = 128;           // queue slots
  constexpr int QW = PB + 1;        // words per entry: raw b, then seed | owner lane << 24
  static_assert(NBD % 4 == 0 && NF % 4 == 0, "factor pieces are 16 bytes");
  constexpr int NR = 4;              // factor ring slots (pairs)
  constexpr int NPC = 2 * NBD / 4;   // 16-byte pieces of a pair's two bound entries
  __shared__ __attribute__((aligned(16))) float tb[64 * TS];
  __shared__ float qb[QW * QC];
  __shared__ __attribute__((aligned(16))) float fr[NR * 2 * NBD];  // [slot][seed of the pair][L, 1/e]
  const int lane = threadIdx.x;
  const int nbk_cols = (int)(a.cols / C);
  const int nsplit = a.nsplit;
  const int64_t nwg = gridDim.x;
  const int64_t xcd = blockIdx.x % 8, q = nwg / 8, rem = nwg % 8;
  const int64_t w = xcd * q + (xcd < rem ? xcd : rem) + blockIdx.x / 8;
  const int nrg = (int)((a.rows + 31) / 32);
  const int split = (int)(w % nsplit);
  const int64_t rest = w / nsplit;
  const int blk = (int)(rest / nrg);
  const int64_t row0 = (rest % nrg) * 32;
  const int n_pairs_all = (a.S + 1) / 2;
  const int pp = (n_pairs_all + nsplit - 1) / nsplit;
  const int pair0 = split * pp;
  const int pair1 = pair0 + pp < n_pairs_all ? pair0 + pp : n_pairs_all;
  const int n = lane & 15, g = lane >> 4;

  // u fragments, and each tile's weighted energy sum_j d_j r_j^2 (over the
  // four lanes n, n + 16, n + 32, n + 48 that share a row)
  u32x4 uh[2][NKS], um[2][NKS], ul[2][NKS];
  float en[2];
  load_u_col<C, 2>(a, row0, blk, n, g, uh, um, ul, en);
  const int half = lane >> 5;
  const int64_t my_row = row0 + (lane & 31);
  const bool my_valid = my_row < a.rows;
  const float energy = en[(lane >> 4) & 1];  // this lane's tile, 16 nb + n
  const float qmax = (float)((1 << (a.b - 1)) - 1);
  const float inv_qmax = 1.0f / qmax;
  constexpr float isq = C == 64 ? 0.125f : 0.08838834764831845f;  // 1/sqrt(C)
  float tg0 = -INFINITY, tg1 = -INFINITY;
  uint32_t ts0 = 0, ts1 = 0;  // seed words: seed | kEdge flag
  float thr = -INFINITY;
  // the pruning threshold of this lane's tile: the re-score window below the
  // best over both halves (lane ^ 32), one percent wider, the wide one when
  // that best is a knife edge; in units of the raw bound (C times the bound
  // of the scaled b)
  auto update_thr = [&]() {
    const auto r0 = __builtin_amdgcn_permlane32_swap(__float_as_uint(tg0), __float_as_uint(tg0), false, false);
    const auto r1 = __builtin_amdgcn_permlane32_swap(ts0, ts0, false, false);
    const float og = __uint_as_float(half ? r0[0] : r0[1]);
    const uint32_t ow = half ? r1[0] : r1[1];
    const float best = fmaxf(tg0, og);
    const bool edge = ((tg0 >= og ? ts0 : ow) & kEdge) != 0;
    thr = slack_thr(best - 1.01f * rescore_window(best, energy, edge)) * (float)C;
  };
  int qhead = 0, qtail = 0;  // wavefront-uniform queue counters
  int nscored = 0;
  const uint64_t lt = lane ? (~0ull >> (64 - lane)) : 0ull;
  auto load_factor = [&](int s_, float (&f)[NF], int pieces) {
    const f32x4* fv = reinterpret_cast<const f32x4*>(a.colfac + ((size_t)blk * a.S + s_) * stride);
#pragma unroll
    for (int i = 0; i < NF / 4; ++i) {
      if (i < pieces) {
        const f32x4 v = fv[i];
        f[4 * i] = v[0]; f[4 * i + 1] = v[1]; f[4 * i + 2] = v[2]; f[4 * i + 3] = v[3];
      }
    }
  };
  // The bound's factor entries reach the wavefront through an LDS ring: at
  // the step of pair k every lane loads one 16-byte piece of pair k + 2's two
  // entries (lanes with the same piece load the same one) and stores the
  // piece it loaded at the step before (pair k + 1's); the bound of pair k
  // reads its seed's entry from slot k.  The wavefront barriers of every step
  // order the stores before the reads.
  const int pc = lane % NPC;
  // the piece's seed within its pair and its byte offset in the seed's entry;
  // the block's rows of the table from a wavefront-uniform base
  const int psel = pc / (NBD / 4);
  const uint32_t pofs = 16u * (uint32_t)(pc % (NBD / 4)), strideB = 4u * (uint32_t)stride;
  const char* fac_blk = reinterpret_cast<const char*>(a.colfac + (size_t)blk * a.S * stride);
  auto fac_piece = [&](int pr) -> f32x4 {
    const int s_ = min(2 * pr + psel, a.S - 1);
    return *reinterpret_cast<const f32x4*>(fac_blk + __umul24((uint32_t)s_, strideB) + pofs);
  };
  auto fac_store = [&](int pr, const f32x4& v) {
    *reinterpret_cast<f32x4*>(&fr[(pr & (NR - 1)) * (2 * NBD) + 4 * pc]) = v;
  };
  auto score_round = [&](int cnt) {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    const bool mine = lane < cnt;
    const int slot = (qhead + lane) & (QC - 1);
    int ol = 0;
    if (mine) {
      float bs[PB];
#pragma unroll
      for (int i = 0; i < PB; ++i) bs[i] = qb[i * QC + slot] * isq;
      const uint32_t word = __float_as_uint(qb[PB * QC + slot]);
      const int es = (int)(word & 0xFFFFu);
      ol = (int)(word >> 24);
      float f[NF];
      load_factor(es, f, NF / 4);
      bool edge;
      const float gsc = screen_score_ldl<PB, POW2, 0>(bs, f, qmax, inv_qmax, &edge);
      qb[slot] = gsc;
      qb[QC + slot] = __uint_as_float((uint32_t)es | (edge ? kEdge : 0u));
    }
    uint64_t mm = __ballot(mine);
#pragma unroll
    for (int b = 0; b < 6; ++b) {
      const uint64_t bal = __ballot((ol >> b) & 1);
      mm &= ((lane >> b) & 1) ? bal : ~bal;
    }
    nscored += __popcll(mm);
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    while (__ballot(mm != 0) != 0) {
      if (mm != 0) {
        const int r = (qhead + __builtin_ctzll(mm)) & (QC - 1);
        const float gsc = qb[r];
        const uint32_t sw = __float_as_uint(qb[QC + r]);
        const bool c0 = gsc > tg0, c1 = gsc > tg1;
        tg1 = c0 ? tg0 : (c1 ? gsc : tg1);
        ts1 = c0 ? ts0 : (c1 ? sw : ts1);
        tg0 = c0 ? gsc : tg0;
        ts0 = c0 ? sw : ts0;
        mm &= mm - 1;
      }
    }
    qhead += cnt;
    update_thr();
  };

  const u32x4* fp = frag + (size_t)pair0 * (NKS * 64) + lane;
  auto project = [&](const u32x4 (&F)[NKS], f32x4 (&acc)[2]) {
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
      f32x4 c = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) {
        const bf16x8 A = as_bf16x8(F[ks]);
        c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A, as_bf16x8(uh[nb][ks]), c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A, as_bf16x8(um[nb][ks]), c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A, as_bf16x8(ul[nb][ks]), c, 0, 0, 0);
      }
      acc[nb] = c;
    }
  };
  // rows 4g..4g+3 of the product = (seed g/2 of the pair, columns 4(g&1)..+3)
  // of tiles 16nb + n; lane (seed half, tile) reads them back
  auto stash = [&](const f32x4 (&acc)[2]) {
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
      *reinterpret_cast<f32x4*>(&tb[((g >> 1) * 32 + 16 * nb + n) * TS + 4 * (g & 1)]) = acc[nb];
  };
  u32x4 F[NKS];
  {
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) F[ks] = fp[ks * 64];
    f32x4 acc[2];
    project(F, acc);
    stash(acc);
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) F[ks] = fp[NKS * 64 + ks * 64];
  }
  fac_store(pair0, fac_piece(pair0));
  f32x4 fnext = fac_piece(pair0 + 1);
  for (int pair = pair0; pair < pair1; ++pair) {
    const int s = 2 * pair + half;
    // pair + 1's pieces (loaded a step ago) into the ring, pair + 2's in flight
    fac_store(pair + 1, fnext);
    fnext = fac_piece(pair + 2);
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    float f[NF];
    {
      const float* fe = &fr[(pair & (NR - 1)) * (2 * NBD) + half * NBD];
#pragma unroll
      for (int i = 0; i < NBD / 4; ++i) {
        const f32x4 v = *reinterpret_cast<const f32x4*>(&fe[4 * i]);
        f[4 * i] = v[0]; f[4 * i + 1] = v[1]; f[4 * i + 2] = v[2]; f[4 * i + 3] = v[3];
      }
    }
    float bv[PB];
    {
      const f32x4 b0 = *reinterpret_cast<const f32x4*>(&tb[lane * TS]);
      const f32x4 b1 = *reinterpret_cast<const f32x4*>(&tb[lane * TS + 4]);
      bv[0] = b0[0]; bv[1] = b0[1]; bv[2] = b0[2]; bv[3] = b0[3];
      bv[4] = b1[0]; bv[5] = b1[1]; bv[6] = b1[2]; bv[7] = b1[3];
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    f32x4 accN[2];
    project(F, accN);
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) F[ks] = fp[(size_t)(pair - pair0 + 2) * (NKS * 64) + ks * 64];
    float wv[PB];
    const float bnd = screen_fwd<PB>(bv, f, wv);
    const bool keep = (int)(bnd > thr) & (int)my_valid & (int)(s < a.S);
    // every lane stores its candidate (raw b), the kept ones first from the
    // tail on, the dropped ones after them (at most 63 wait before a step, so
    // the 64 slots written are free); the tail takes in the kept ones only
    const uint64_t kb = __ballot(keep);
    const int nk = __popcll(kb);
    const int pos = keep ? __popcll(kb & lt) : nk + __popcll(~kb & lt);
    const int qslot = (qtail + pos) & (QC - 1);
#pragma unroll
    for (int i = 0; i < PB; ++i) qb[i * QC + qslot] = bv[i];
    qb[PB * QC + qslot] = __uint_as_float((uint32_t)s | ((uint32_t)lane << 24));
    qtail += nk;
#pragma unroll
    for (int i = 0; i < 24; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x002, 3, 0);
    }
    if (qtail - qhead >= 64) score_round(64);
    stash(accN);
  }
  if (qtail > qhead) score_round(qtail - qhead);
#pragma unroll
  for (int k = 32; k >= 1; k >>= 1) nscored += __shfl_xor(nscored, k, 64);
  if (lane == 0) atomicAdd(a.scored, (unsigned long long)nscored);
  // merge the two halves' lists of each tile: (gain desc, seed asc)
  const float og0 = __shfl(tg0, lane + 32, 64), og1 = __shfl(tg1, lane + 32, 64);
  const uint32_t os0 = (uint32_t)__shfl((int)ts0, lane + 32, 64), os1 = (uint32_t)__shfl((int)ts1, lane + 32, 64);
  if (half == 0 && my_valid) {
    auto better = [](float ga, uint32_t sa, float gb, uint32_t sb) {
      return ga > gb || (ga == gb && list_seed(sa) < list_seed(sb));
    };
    float r0, r1;
    uint32_t q0, q1;
    if (better(tg0, ts0, og0, os0)) {
      r0 = tg0; q0 = ts0;
      const bool m = better(tg1, ts1, og0, os0);
      r1 = m ? tg1 : og0; q1 = m ? ts1 : os0;
    } else {
      r0 = og0; q0 = os0;
      const bool m = better(tg0, ts0, og1, os1);
      r1 = m ? tg0 : og1; q1 = m ? ts0 : os1;
    }
    const int64_t at = ((my_row * nbk_cols + blk) * nsplit + split) * kTop;
    a.top_gain[at + 0] = r0;
    a.top_gain[at + 1] = r1;
    a.top_seed[at + 0] = q0;
    a.top_seed[at + 1] = q1;
  }
}

bool screen_mfma_supported(int C, int P, int d_mode, int gen_version) {
  if (P < 1 || P > 8) return false;
  if (d_mode == AWSRC_D_PER_ELEM && gen_version != 1) return false;
  return C == 64 || (C == 128 && d_mode == AWSRC_D_PER_COL);
}

// Seed ranges per tile: split only while the module's row groups would leave
// the machine (about 2048 resident wavefronts at two per SIMD) under-filled,
// keeping at least 16 seed pairs per range.
int screen_nsplit(int C, int P, int S, int64_t rows, int64_t cols, int d_mode, int gen_version) {
  if (!screen_mfma_supported(C, P, d_mode, gen_version)) return 1;
  const int tpw = C == 128 ? 32 : 64;  // rows per wavefront
  const int64_t waves = (cols / C) * ((rows + tpw - 1) / tpw);
  const int pairs = (S + 1) / 2;
  int ns = 1;
  while (ns < 8 && waves * ns < 2048 && pairs / (2 * ns) >= 16) ns *= 2;
  return ns;
}

bool screen_pruned(int C, int P, int d_mode, int gen_version) {
  return (C == 64 || C == 128) && screen_mfma_supported(C, P, d_mode, gen_version) && d_mode == AWSRC_D_PER_COL;
}

bool screen_fuses_rescore(int C, int P, int d_mode, int gen_version, int nsplit) {
  return C == 64 && screen_pruned(C, P, d_mode, gen_version) && gen_version == 1 && nsplit == 1;
}

__global__ void k_scored_init(unsigned long long* p, unsigned long long v, int add) {
  if (threadIdx.x == 0) *p = (add ? *p : 0ull) + v;
}

hipError_t launch_scored_zero(unsigned long long* p, hipStream_t st) {
  hipLaunchKernelGGL(k_scored_init, dim3(1), dim3(64), 0, st, p, 0ull, 0);
  return hipGetLastError();
}

hipError_t launch_scored_init(const EncodeArgs& a, hipStream_t st, bool add) {
  const unsigned long long all = (unsigned long long)(a.rows * (a.cols / a.C)) * (unsigned long long)a.S;
  hipLaunchKernelGGL(k_scored_init, dim3(1), dim3(64), 0, st, a.scored,
                     screen_pruned(a.C, a.P, a.d_mode, a.gen_version) ? 0ull : all, add ? 1 : 0);
  return hipGetLastError();
}

// the table carries two zero pairs past the last seed (see the pipeline above)
size_t mfma_frag_bytes(int C, int S) { return (size_t)((S + 1) / 2 + 2) * (C / 32) * 64 * 16; }

template <bool POW2>
static hipError_t screen_mfma_fmt(const EncodeArgs& a, void* frag, hipStream_t st) {
  const u32x4* fr = static_cast<const u32x4*>(frag);
  if (a.C == 128) {
    const int64_t wgs = (a.cols / a.C) * ((a.rows + 31) / 32) * a.nsplit;
    hipLaunchKernelGGL((k_screen_mfma_halves<128, POW2>), dim3((unsigned)wgs), dim3(64), 0, st, a, fr,
                       colfac_stride(8));
    return hipGetLastError();
  }
  const int64_t wgs = (a.cols / a.C) * ((a.rows + 63) / 64) * a.nsplit;
  if (!a.fused_rescore)
    hipLaunchKernelGGL((k_screen_col64<POW2, 0>), dim3((unsigned)wgs), dim3(64), 0, st, a, fr, colfac_stride(8));
  else if (a.P <= 4)
    hipLaunchKernelGGL((k_screen_col64<POW2, 4>), dim3((unsigned)wgs), dim3(64), 0, st, a, fr, colfac_stride(8));
  else
    hipLaunchKernelGGL((k_screen_col64<POW2, 8>), dim3((unsigned)wgs), dim3(64), 0, st, a, fr, colfac_stride(8));
  return hipGetLastError();
}

hipError_t launch_mfma_frags(const BasisTables& bt, int C, int P, int S, void* frag, hipStream_t st) {
  const int64_t n = (int64_t)((S + 1) / 2 + 2) * (C / 32) * 64;
  hipLaunchKernelGGL(k_mfma_frags, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, bt, C, P, S,
                     static_cast<u32x4*>(frag));
  return hipGetLastError();
}

hipError_t launch_encode_screen_mfma(const EncodeArgs& a, void* frag, hipStream_t st) {
  const hipError_t e = launch_mfma_frags(a.basis, a.C, a.P, a.S, frag, st);
  if (e != hipSuccess) return e;
  if (a.scale_fmt == AWSRC_SCALE_POW2) return screen_mfma_fmt<true>(a, frag, st);
  return screen_mfma_fmt<false>(a, frag, st);
}

}  // namespace awsrc
