// Encoder seed search with per-element weights (the Fisher/activation blend of
// Sec. 3.3: d_t differs per row), C = 64, P <= 8, generator version 1, for
// any number of modules in one launch.
//
// Per (tile, seed) the screen needs b = B_s^T (d .* r) (Eq. (3)), the
// factor of the tile's own G + eps I and the score of the rounded fit
// (Sec. 3.2).  Work layout:
//
//   * one wavefront = 32 consecutive rows of one column block (32 tiles) of
//     one module; a module table maps the launch's work items onto modules,
//     so one launch covers a whole model and no module leaves the machine
//     half idle;
//   * the projections of a seed pair for the 32 tiles are a [16 x 64] x
//     [64 x 32] product on the matrix cores (u split exactly into three bf16
//     parts, +-1 basis fragments, fp32 accumulation), twelve
//     v_mfma_f32_16x16x32_bf16; one v_permlane16_swap per register pair
//     then leaves lane l with all P coefficients of one candidate: tile
//     l % 32, seed 2 pair + l / 32;
//   * G_pq = WHT(d_t)[c_p xor c_q] / C (the Sylvester XOR identity) is
//     gathered from a per-tile transform in LDS, laid out [coordinate][tile]
//     so that a lane's gather address is the XOR of c_p << 7, c_q << 7 (a
//     per-seed table of shifted columns) and 4 tile, and the 32 lanes of
//     each seed read 32 distinct banks;
//   * every candidate gets the LDL^T factor and the forward solve, whose
//     sum_k w_k^2 / e_k = b^T (G + eps I)^-1 b bounds the score of every
//     rounding of the fit (the score is a concave quadratic in the
//     coefficients with that maximum); only candidates whose bound reaches
//     the re-score's window below the tile's current best are scored in
//     full (the re-score looks at a second seed only inside that window, and
//     its lower edge only rises).  Those are few (a few percent), so each
//     lane queues them (w and the seed) in its own LDS ring, and a scoring
//     round refactors and scores the oldest entry of every lane that has
//     one, whenever some lane's ring is full;
//   * each tile's even and odd seeds live in lanes l and l ^ 32: their lists
//     share the pruning threshold (from the best over both, by a
//     v_permlane32_swap after each round) and are merged at the end.  A
//     lane's entries are scored in seed order and thresholds only rise, so
//     the merged top two agree with those of scoring every candidate in the
//     best and in the second wherever the second is inside the window.
//
// The kept lists go to the fp64 re-score (k_finalize_pe_modules, rescore_pe.hip).
#include <math.h>

#include "awsrc_internal.h"
#include "mfma_bf16.h"
#include "rescore64.h"

namespace awsrc {

namespace {

constexpr int kC = 64;
constexpr int kPB = 8;
constexpr int kNT = kPeRows;  // tiles per wavefront

// u = d .* r fragments of the two groups of 16 tiles (rows row0 + 16 nb + n,
// coordinates 32 ks + 8 g .. + 7), split in three bf16 parts; rows past the
// end give zeros.
__device__ __forceinline__ void load_u32rows(const ModEntry& md, int w_dtype, int64_t row0, int blk, int n, int g,
                                             u32x4 (&uh)[2][2], u32x4 (&um)[2][2], u32x4 (&ul)[2][2]) {
  // the four (nb, ks) segments of 8 weights as eight chunks of four; every
  // load is issued before any is used
  int64_t o[8];
  bool valid[2];
#pragma unroll
  for (int nb = 0; nb < 2; ++nb) {
    const int64_t row = row0 + 16 * nb + n;
    valid[nb] = row < md.rows;
    const int64_t rr = valid[nb] ? row : md.rows - 1;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const int64_t base = rr * md.cols + (int64_t)blk * kC + 32 * ks + 8 * g;
      o[4 * nb + 2 * ks] = base;
      o[4 * nb + 2 * ks + 1] = base + 4;
    }
  }
  gf32x4 dv[8];
#pragma unroll
  for (int c = 0; c < 8; ++c) dv[c] = gload4f(md.d + o[c]);
  float rv[8][4];
  load_residual4<8>(md.W, w_dtype, md.W0, o, rv);
#pragma unroll
  for (int nb = 0; nb < 2; ++nb)
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      float u[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int c = 4 * nb + 2 * ks + (e >> 2);
        u[e] = valid[nb] ? dv[c][e & 3] * rv[c][e & 3] : 0.0f;
      }
      split3(u, uh[nb][ks], um[nb][ks], ul[nb][ks]);
    }
}

// b of one seed pair for the 32 tiles: acc[nb] holds rows 4g..4g+3 (seed g/2
// of the pair, coefficients 4(g&1)..+3) of tile 16 nb + n.
__device__ __forceinline__ void project32(const u32x4& F0, const u32x4& F1, const u32x4 (&uh)[2][2],
                                          const u32x4 (&um)[2][2], const u32x4 (&ul)[2][2], f32x4 (&acc)[2]) {
  const bf16x8 A0 = as_bf16x8(F0), A1 = as_bf16x8(F1);
#pragma unroll
  for (int nb = 0; nb < 2; ++nb) {
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

// The Gram gathers of one candidate: G_pq (q < p) = wdl at byte offset
// cs[p] ^ cs[q] ^ tl4 (cs[p] = c_p << 7), packed like the strict lower factor.
template <int PB>
__device__ __forceinline__ void gather_pe(const float* wdl, const uint32_t (&cs)[PB], uint32_t tl4,
                                          float (&gq)[PB * (PB - 1) / 2]) {
  const char* wb = reinterpret_cast<const char*>(wdl);
#pragma unroll
  for (int p = 1; p < PB; ++p)
#pragma unroll
    for (int q = 0; q < p; ++q) gq[ltri(p, q)] = *reinterpret_cast<const float*>(wb + (cs[p] ^ cs[q] ^ tl4));
}

// G + eps I = L diag(e) L^T of one candidate, in the layout of the
// per-column factor table (strict lower L by rows, then 1/e, then e), from
// its gathers gq and the diagonal d0 = mean_j d_j.  Padded columns (p >= P)
// get L = 0, e = 1; FULLP: P == PB, so that no column is padding (the P = 8
// workloads).
template <int PB, bool FULLP>
__device__ __forceinline__ void factor_pe(const float (&gq)[PB * (PB - 1) / 2], float d0, float eps, int P,
                                          float (&f)[PB * (PB - 1) / 2 + 2 * PB]) {
  constexpr int LS = PB * (PB - 1) / 2;
  const float diag = d0 + eps;
#pragma unroll
  for (int p = 0; p < PB; ++p) {
    const bool real = FULLP || p < P;
    float E[PB];
#pragma unroll
    for (int q = 0; q < p; ++q) {
      float t = real ? gq[ltri(p, q)] : 0.0f;
#pragma unroll
      for (int kk = 0; kk < q; ++kk) t = fmaf(-E[kk], f[ltri(q, kk)], t);
      E[q] = t;
      f[ltri(p, q)] = t * f[LS + q];
    }
    float t = real ? diag : 1.0f;
#pragma unroll
    for (int kk = 0; kk < p; ++kk) t = fmaf(-E[kk], f[ltri(p, kk)], t);
    t = fmaxf(t, 1e-30f);
    f[LS + PB + p] = t;
    f[LS + p] = __builtin_amdgcn_rcpf(t);
  }
}

template <int PB>
__device__ __forceinline__ void unpack_cols(const u32x4& c0, const u32x4& c1, uint32_t (&cs)[PB]) {
#pragma unroll
  for (int p = 0; p < PB; ++p) cs[p] = p < 4 ? c0[p] : c1[p - 4];
}

}  // namespace

// Per-seed table of the selected columns shifted to LDS byte offsets of the
// [coordinate][32 tiles] transform: colsh[s][p] = c_p << 7 (0 for p >= P and
// for the padding seeds s >= S that the prefetch of the next pair may touch).
__global__ void k_pe_colsh(BasisTables bt, int P, int S, int n_rows, uint32_t* __restrict__ colsh) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n_rows * kPB) return;
  const int s = i / kPB, p = i % kPB;
  colsh[i] = (s < S && p < P) ? ((uint32_t)bt.col[(size_t)s * kMaxP + p] << 7) : 0u;
}

// three wavefronts per SIMD (at most 168 VGPRs; the LDS allows twelve per CU)
template <bool POW2, bool FULLP>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(3))) void k_screen_pe32(EncodeArgs a, const ModEntry* __restrict__ mods, int n_mods,
                                                       const u32x4* __restrict__ frag,
                                                       const u32x4* __restrict__ colsh) {
  constexpr int C = kC, PB = kPB, NT = kNT;
  constexpr int NF = PB * (PB - 1) / 2 + 2 * PB;
  constexpr int NL = PB * (PB - 1) / 2;
  constexpr int QC = 128;     // slots of the wavefront's queue: 12.8 KB of LDS in all, three wavefronts per SIMD
  constexpr int QW = PB + 1;  // words per entry: w, then the seed | owner lane << 24
  __shared__ float wdl[C * NT];            // WHT(d_t) / C, [coordinate][tile]
  __shared__ float qb[QW * QC];            // the queue, [word][slot]
  const int lane = threadIdx.x;
  const int64_t item = blockIdx.x;
  const int m = find_module(mods, n_mods, item);
  const ModEntry md = mods[m];
  const int nbk = (int)(md.cols / C);
  const int64_t local = item - md.item_off;
  const int blk = (int)(local % nbk);
  const int64_t row0 = (local / nbk) * NT;
  const int n = lane & 15, g = lane >> 4;
  const int tl = lane & 31;  // this lane's tile while screening
  const int sh = lane >> 5;  // and its seed parity
  const uint32_t tl4 = 4u * (uint32_t)tl;
  const int64_t my_row = row0 + tl;
  const bool valid = my_row < md.rows;
  float energy;
  {
    // WHT of the tile's weights; lanes tl and tl + 32 both transform it and
    // each stores one half
    const int64_t off = (valid ? my_row : md.rows - 1) * md.cols + (int64_t)blk * C;
    float wd[C];
#pragma unroll
    for (int j0 = 0; j0 < C; j0 += 8) {
      float v[8];
      load8_f(md.d + off + j0, v);
#pragma unroll
      for (int k = 0; k < 8; ++k) wd[j0 + k] = v[k];
    }
    // this lane's half of the tile's weighted energy sum_j d_j r_j^2 (for
    // the pruning window below)
    float eh = 0.0f;
    {
      int64_t o[C / 8];  // this lane's half in chunks of four, all loads issued first
#pragma unroll
      for (int k = 0; k < C / 8; ++k) o[k] = off + 32 * sh + 4 * k;
      float rv[C / 8][4];
      load_residual4<C / 8>(md.W, a.w_dtype, md.W0, o, rv);
#pragma unroll
      for (int j = 0; j < C / 2; ++j) {
        const float r = rv[j >> 2][j & 3];
        eh = fmaf((sh ? wd[32 + j] : wd[j]) * r, r, eh);
      }
    }
    const auto re = __builtin_amdgcn_permlane32_swap(__float_as_uint(eh), __float_as_uint(eh), false, false);
    energy = eh + __uint_as_float(sh ? re[0] : re[1]);
    fwht<C>(wd);
#pragma unroll
    for (int j = 0; j < C / 2; ++j) wdl[(j + 32 * sh) * NT + tl] = (sh ? wd[j + 32] : wd[j]) * (1.0f / C);
  }
  u32x4 uh[2][2], um[2][2], ul[2][2];
  load_u32rows(md, a.w_dtype, row0, blk, n, g, uh, um, ul);
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  const int P = a.P;
  const float qmax = (float)((1 << (a.b - 1)) - 1);
  const float inv_qmax = 1.0f / qmax;
  const float d0 = wdl[tl];  // G_pp = mean_j d_j
  const float eps = (float)a.lambda * d0;

  // this lane's top two (its seeds increase, so strict comparisons keep the
  // earlier seed first among equal scores) and the tile's pruning threshold
  float tg0 = -INFINITY, tg1 = -INFINITY;
  int ts0 = 0, ts1 = 0;
  float thr = -INFINITY;
  // The re-score takes a tile's second seed only when its screened score lies
  // within rescore_window of the best, so a candidate below that window of
  // the tile's current best (over both lanes' lists) can never be needed: the
  // window's lower edge only rises with the best.  The threshold takes the
  // window one percent wider, far above the fp32 rounding of either, and the
  // wide window when the best is flagged as a knife edge (its score may be
  // off by more than the narrow one); in raw units the energy term is 64
  // times larger.
  const float e_raw = 64.0f * energy;
  auto update_thr = [&]() {
    const auto r0 = __builtin_amdgcn_permlane32_swap(__float_as_uint(tg0), __float_as_uint(tg0), false, false);
    const auto r1 = __builtin_amdgcn_permlane32_swap(ts0, ts0, false, false);
    const float og = __uint_as_float(sh ? r0[0] : r0[1]);
    const uint32_t ow = sh ? r1[0] : r1[1];
    const float best = fmaxf(tg0, og);
    const bool edge = ((tg0 >= og ? ts0 : ow) & kEdge) != 0;
    thr = slack_thr(best - 1.01f * rescore_window(best, e_raw, edge));
  };
  // The survivors of the bound wait in one queue for the whole wavefront,
  // appended in step order (so each lane's own entries are in seed order);
  // a scoring round takes the 64 oldest (or, at the end, all that are left),
  // one per lane, and each owner lane then inserts its results into its
  // lists in queue order.  qhead and qtail are wavefront-uniform counters.
  int qhead = 0, qtail = 0;
  int nscored = 0;
  const uint64_t lt = lane ? (~0ull >> (64 - lane)) : 0ull;  // lanes below this one
  const float lam = (float)a.lambda;
  auto score_round = [&](int cnt) {
    const bool mine = lane < cnt;
    const int slot = (qhead + lane) & (QC - 1);
    int ol = 0;
    if (mine) {
      float wv[PB];
#pragma unroll
      for (int i = 0; i < PB; ++i) wv[i] = qb[i * QC + slot];
      const uint32_t word = __float_as_uint(qb[PB * QC + slot]);
      const int es = (int)(word & 0xFFFFu);
      ol = (int)(word >> 24);
      const int et = ol & 31;  // the entry's tile
      const float ed0 = wdl[et];
      uint32_t cs[PB];
      unpack_cols<PB>(colsh[2 * (size_t)es], colsh[2 * (size_t)es + 1], cs);
      float gr[NL], f[NF];
      gather_pe<PB>(wdl, cs, 4u * (uint32_t)et, gr);
      factor_pe<PB, FULLP>(gr, ed0, lam * ed0, P, f);
      bool edge;
      const float gsc = screen_gain_w<PB, POW2, 3>(wv, f, qmax, inv_qmax, &edge);
      qb[slot] = gsc;
      qb[QC + slot] = __uint_as_float((uint32_t)es | (edge ? kEdge : 0u));
    }
    // the round's lanes whose entry this lane owns, found by matching the
    // owner's six bits across the wavefront
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

  // Raw units: b is left unscaled by 1/sqrt(C) = 1/8, so the bound, alpha,
  // the scale and the score come out 64, 8, 8 and 64 times larger; codes and
  // the seed order are unchanged (a power-of-two factor commutes with the
  // roundings), and the kept scores are rescaled at the end.
  //
  // Software pipeline: the matrix cores project pair k+1 while the vector
  // ALUs work on pair k (the fragment and column tables carry padding pairs,
  // so the loads two pairs ahead need no bounds).
  const int n_pairs = (a.S + 1) / 2;
  const u32x4* fp = frag + lane;
  // two register sets for the projections, fragments and columns, swapping
  // roles every pair (the loop runs two pairs per trip, so no copies)
  f32x4 accA[2], accB[2];
  project32(fp[0], fp[64], uh, um, ul, accA);
  u32x4 FA0 = fp[128], FA1 = fp[192], FB0, FB1;
  u32x4 CA0 = colsh[2 * (size_t)sh], CA1 = colsh[2 * (size_t)sh + 1], CB0, CB1;
  auto step = [&](int pair, const f32x4 (&acc)[2], f32x4 (&accN)[2], const u32x4& F0, const u32x4& F1, u32x4& F0n,
                  u32x4& F1n, const u32x4& C0, const u32x4& C1, u32x4& C0n, u32x4& C1n) {
    const int s = 2 * pair + sh;
    // this lane's candidate: tile tl, seed s; its Gram gathers are issued
    // first, so that their latency overlaps the rest
    uint32_t cs[PB];
    unpack_cols<PB>(C0, C1, cs);
    float gq[NL];
    gather_pe<PB>(wdl, cs, tl4, gq);
    float bt[PB];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(acc[0][i]), __float_as_uint(acc[1][i]), false,
                                                      false);
      bt[i] = __uint_as_float(r[0]);
      bt[4 + i] = __uint_as_float(r[1]);
    }
    // next pair's projections and columns, and the fragments two pairs ahead
    project32(F0, F1, uh, um, ul, accN);
    F0n = fp[(size_t)(pair + 2) * 128];
    F1n = fp[(size_t)(pair + 2) * 128 + 64];
    C0n = colsh[2 * (size_t)(s + 2)];
    C1n = colsh[2 * (size_t)(s + 2) + 1];
    float f[NF];
    factor_pe<PB, FULLP>(gq, d0, eps, P, f);
    float wv[PB];
    const float bnd = screen_fwd<PB>(bt, f, wv);
    const bool keep = (int)(bnd > thr) & (int)valid & (int)(s < a.S);
    // Every lane stores its candidate, the kept ones first (in lane order)
    // from the tail on, the dropped ones after them; only the kept ones are
    // taken in by advancing the tail.  At most 63 entries wait before a
    // step, so the 64 slots written are free.
    const uint64_t kb = __ballot(keep);
    const int nk = __popcll(kb);
    const int pos = keep ? __popcll(kb & lt) : nk + __popcll(~kb & lt);
    const int slot = (qtail + pos) & (QC - 1);
#pragma unroll
    for (int i = 0; i < PB; ++i) qb[i * QC + slot] = wv[i];
    qb[PB * QC + slot] = __uint_as_float((uint32_t)s | ((uint32_t)lane << 24));
    qtail += nk;
#pragma unroll
    for (int i = 0; i < 12; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x002, 16, 0);
    }
    // a full round's worth waiting: score the 64 oldest
    if (qtail - qhead >= 64) score_round(64);
  };
  int pair = 0;
  for (; pair + 1 < n_pairs; pair += 2) {
    step(pair, accA, accB, FA0, FA1, FB0, FB1, CA0, CA1, CB0, CB1);
    step(pair + 1, accB, accA, FB0, FB1, FA0, FA1, CB0, CB1, CA0, CA1);
  }
  if (pair < n_pairs) step(pair, accA, accB, FA0, FA1, FB0, FB1, CA0, CA1, CB0, CB1);
  if (qtail > qhead) score_round(qtail - qhead);
#pragma unroll
  for (int k = 32; k >= 1; k >>= 1) nscored += __shfl_xor(nscored, k, 64);
  if (lane == 0) atomicAdd(a.scored, (unsigned long long)nscored);

  // merge the tile's even-seed (this lane) and odd-seed (lane + 32) lists
  // into (gain desc, seed asc) and store them for the re-score
  const float og0 = __shfl_xor(tg0, 32, 64), og1 = __shfl_xor(tg1, 32, 64);
  const uint32_t os0 = (uint32_t)__shfl_xor((int)ts0, 32, 64), os1 = (uint32_t)__shfl_xor((int)ts1, 32, 64);
  // (every lane's slot is written: rows past the module's end keep -inf and
  // seed 0, so the re-score never reads a stale entry)
  if (sh == 0) {
    auto better = [](float ga, uint32_t sa, float gb, uint32_t sb) {
      return ga > gb || (ga == gb && list_seed(sa) < list_seed(sb));
    };
    float r0, r1;
    uint32_t q0, q1;
    if (better(tg0, ts0, og0, os0)) {
      r0 = tg0; q0 = ts0;
      const bool mm = better(tg1, ts1, og0, os0);
      r1 = mm ? tg1 : og0; q1 = mm ? ts1 : os0;
    } else {
      r0 = og0; q0 = os0;
      const bool mm = better(tg0, ts0, og1, os1);
      r1 = mm ? tg0 : og1; q1 = mm ? ts0 : os1;
    }
    // work-item-major lists, [item][kTop][32 tiles], so that the stores and
    // the re-score's loads are whole lines
    const int64_t at = item * (kTop * NT) + tl;
    a.top_gain[at] = r0 * (1.0f / 64.0f);  // back to gain units
    a.top_gain[at + NT] = r1 * (1.0f / 64.0f);
    a.top_seed[at] = q0;
    a.top_seed[at + NT] = q1;
  }
}

__global__ void k_mod_table(ModChunk ch, int n, ModEntry* __restrict__ dst) {
  if (threadIdx.x == 0)
    for (int i = 0; i < n; ++i) dst[i] = ch.e[i];
}

hipError_t launch_mod_table(const ModEntry* host, int n, ModEntry* dev, hipStream_t st) {
  for (int i0 = 0; i0 < n; i0 += kModChunk) {
    ModChunk ch;
    const int k = n - i0 < kModChunk ? n - i0 : kModChunk;
    for (int i = 0; i < k; ++i) ch.e[i] = host[i0 + i];
    hipLaunchKernelGGL(k_mod_table, dim3(1), dim3(64), 0, st, ch, k, dev + i0);
  }
  return hipGetLastError();
}

bool pe_batched_supported(int C, int P, int d_mode, int gen_version) {
  return C == kC && P <= kPB && d_mode == AWSRC_D_PER_ELEM && gen_version == 1;
}

// rows of the shifted-column table: every seed, the odd seed of a last
// half-filled pair, and two pairs of padding for the prefetch
size_t pe_colsh_bytes(int S) { return (size_t)(2 * ((S + 1) / 2) + 4) * kPB * 4; }

hipError_t launch_pe_screen(const EncodeArgs& a, const ModEntry* mods, int n_mods, int64_t items, const void* frag,
                            uint32_t* colsh, hipStream_t st) {
  const int rows = 2 * ((a.S + 1) / 2) + 4;
  const hipError_t e = launch_mfma_frags(a.basis, a.C, a.P, a.S, const_cast<void*>(frag), st);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_pe_colsh, dim3((unsigned)((rows * kPB + 255) / 256)), dim3(256), 0, st, a.basis, a.P, a.S,
                     rows, colsh);
  if (items == 0) return hipGetLastError();
  const u32x4* fr = static_cast<const u32x4*>(frag);
  const u32x4* cw = reinterpret_cast<const u32x4*>(colsh);
  const dim3 grid((unsigned)items), blk(64);
  if (a.scale_fmt == AWSRC_SCALE_POW2) {
    if (a.P == kPB) hipLaunchKernelGGL((k_screen_pe32<true, true>), grid, blk, 0, st, a, mods, n_mods, fr, cw);
    else hipLaunchKernelGGL((k_screen_pe32<true, false>), grid, blk, 0, st, a, mods, n_mods, fr, cw);
  } else {
    if (a.P == kPB) hipLaunchKernelGGL((k_screen_pe32<false, true>), grid, blk, 0, st, a, mods, n_mods, fr, cw);
    else hipLaunchKernelGGL((k_screen_pe32<false, false>), grid, blk, 0, st, a, mods, n_mods, fr, cw);
  }
  return hipGetLastError();
}

}  // namespace awsrc
