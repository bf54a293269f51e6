// fp64 re-score of the batched per-element encoder (C = 64, P <= 8,
// generator version 1): the kept seeds of every tile of every module are
// re-scored with the complete chain of Sec. 3.2 in fp64 (projection through
// the Walsh-Hadamard transform of sigma .* d .* r, Gram entries through the
// transform of the tile's own d, Cholesky solve of Eq. (3), quantization,
// and the gain of the quantized fit); writes the encoder outputs.
//
// One wavefront per (module, 32-row group, column block), the screen's work
// items; two lanes per tile: lane l (tile l % 32) holds coordinates
// 32 (l / 32) .. + 31.  Each lane transforms its half with the first five
// butterfly stages of the length-64 transform in registers and stores the
// result in its tile's LDS row; the sixth stage, T[k] = X[k % 32] +- Y[k % 32]
// (X, Y the two halves' partial transforms, minus for k >= 32), is folded
// into the gathers, which read only the entries the fit needs.  This is the
// operation order of the full transform, so the values are the same; both
// lanes of a tile then run the same solve and the lower one writes.  Per lane
// this holds 32 doubles of a transform at a time, and the 32 gather rows
// (16.6 KB) are written once per transform, with no turn-taking.
#include <math.h>

#include "awsrc_internal.h"
#include "rescore64.h"

namespace awsrc {

namespace {

constexpr int kC = 64;
constexpr int kH = 32;                       // coordinates per lane
constexpr int kRowD = kC + 1;                // doubles per LDS gather row
constexpr int kLdsFloats = 2 * kPeRows * kRowD;  // the gather rows (fp64), or the r and d staging blocks (fp32)

__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Transform entry k of a tile from its LDS row: X[k % 32] + Y[k % 32] for
// k < 32, X[k % 32] - Y[k % 32] otherwise (the last butterfly stage).
__device__ __forceinline__ double tentry(const double* row, int k) {
  const double x = row[k & (kH - 1)], y = row[kH + (k & (kH - 1))];
  return (k & kH) ? x - y : x + y;
}

}  // namespace

template <int PB>
__global__ __launch_bounds__(64, 2) void k_finalize_pe_modules(EncodeArgs a, const ModEntry* __restrict__ mods,
                                                               int n_mods) {
  constexpr int NG = PB * (PB + 1) / 2;
  __shared__ __attribute__((aligned(16))) float lds[kLdsFloats];
  const int lane = threadIdx.x;
  const int tl = lane & 31, h = lane >> 5;
  const int64_t item = xcd_item(blockIdx.x, gridDim.x);
  const int m = find_module(mods, n_mods, item);
  const ModEntry md = mods[m];
  const int nb = (int)(md.cols / kC);
  const int64_t local = item - md.item_off;
  const int blk = (int)(local % nb);
  const int64_t row0 = (local / nb) * kPeRows;
  const int64_t c0 = (int64_t)blk * kC;

  // the tile's kept seeds (work-item-major lists; both lanes read them)
  float tg[kTop];
  uint32_t ts[kTop];
#pragma unroll
  for (int k = 0; k < kTop; ++k) {
    tg[k] = a.top_gain[item * (kTop * kPeRows) + k * kPeRows + tl];
    ts[k] = a.top_seed[item * (kTop * kPeRows) + k * kPeRows + tl];
  }

  int bs[2];
  uint2 bcol[2];
  uint32_t bsgn[2];
  // Stage the 32 x 64 residual and weight blocks in LDS (rows of 65 floats;
  // 16 lanes per row segment, 4 rows per pass: each instruction reads whole
  // cache lines); rows past the end repeat the last row.
  float* rsh = lds;
  float* dsh = lds + kPeRows * kRowD;
  {
    const int pc = lane & 15;
    constexpr int NP = kPeRows / 4;
    int64_t o[NP];
#pragma unroll
    for (int pass = 0; pass < NP; ++pass) {
      const int rl = 4 * pass + (lane >> 4);
      const int64_t rg = row0 + rl < md.rows ? row0 + rl : md.rows - 1;
      o[pass] = rg * md.cols + c0 + 4 * pc;
    }
    // the weights' loads go out with the residual's, before any wait
    gf32x4 z[NP];
#pragma unroll
    for (int pass = 0; pass < NP; ++pass) z[pass] = gload4f(md.d + o[pass]);
    float rv[NP][4];
    load_residual4<NP>(md.W, a.w_dtype, md.W0, o, rv);
    // the basis entries of both kept seeds (columns, this lane's sign word)
    // go out while the block is in flight; seeds outside [0, S) (none comes
    // from the screen) are replaced by 0 before use
    {
      const int s0r = list_seed(ts[0]), s1r = list_seed(ts[1]);
      bs[0] = s0r < a.S ? s0r : 0;
      bs[1] = s1r < a.S ? s1r : 0;
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        bcol[k] = *reinterpret_cast<const uint2*>(a.basis.col + (size_t)bs[k] * kMaxP);
        bsgn[k] = (uint32_t)(a.basis.sign[(size_t)bs[k] * 2] >> (kH * h));
      }
    }
#pragma unroll
    for (int pass = 0; pass < NP; ++pass) {
      const int rl = 4 * pass + (lane >> 4);
      float* rp = rsh + rl * kRowD + 4 * pc;
      float* dp = dsh + rl * kRowD + 4 * pc;
      rp[0] = rv[pass][0]; rp[1] = rv[pass][1]; rp[2] = rv[pass][2]; rp[3] = rv[pass][3];
      dp[0] = z[pass][0]; dp[1] = z[pass][1]; dp[2] = z[pass][2]; dp[3] = z[pass][3];
    }
  }
  wave_sync();
  float rr[kH], dd[kH];
#pragma unroll
  for (int j = 0; j < kH; ++j) {
    rr[j] = rsh[tl * kRowD + kH * h + j];
    dd[j] = dsh[tl * kRowD + kH * h + j];
  }
  const int64_t row = row0 + tl;
  const bool valid = row < md.rows;
  // the tile's weighted energy in the screen's order (each half, then the
  // two halves added), for the re-score window; the sum of d (exact in fp64)
  // for the ridge eps = lambda mean_j d_j
  float e32;
  double sumd;
  {
    float eh = 0.0f;
    double sh = 0.0;
#pragma unroll
    for (int j = 0; j < kH; ++j) {
      eh = fmaf(dd[j] * rr[j], rr[j], eh);
      sh += (double)dd[j];
    }
    const auto re = __builtin_amdgcn_permlane32_swap(__float_as_uint(eh), __float_as_uint(eh), false, false);
    e32 = eh + __uint_as_float(h ? re[0] : re[1]);
    const uint64_t sb = (uint64_t)__double_as_longlong(sh);
    const auto rl = __builtin_amdgcn_permlane32_swap((uint32_t)sb, (uint32_t)sb, false, false);
    const auto rh = __builtin_amdgcn_permlane32_swap((uint32_t)(sb >> 32), (uint32_t)(sb >> 32), false, false);
    const uint64_t ob = (uint64_t)(h ? rl[0] : rl[1]) | ((uint64_t)(h ? rh[0] : rh[1]) << 32);
    const double so = __longlong_as_double((long long)ob);
    sumd = h ? so + sh : sh + so;  // lower half first
  }
  const double eps = a.lambda * (sumd / kC);
  const int P = a.P;
  const double isq = 1.0 / sqrt((double)kC);
  const int qmax = (1 << (a.b - 1)) - 1;
  double* grow = reinterpret_cast<double*>(lds) + tl * kRowD;

  // The second kept seed is re-scored only when its screened gain lies
  // within the re-score's window of the best (the wide one if either is a
  // knife edge).  The lower lane of a tile scores the best seed, the upper
  // lane the second one where needed (else the best again).
  const float thr = tg[0] - rescore_window(tg[0], e32, ((ts[0] | ts[1]) & kEdge) != 0);
  const bool need = valid && tg[1] >= thr && tg[1] > -INFINITY;
  const bool two = __ballot(need) != 0;
  const bool mine2 = h == 1 && need;
  // seeds index the basis tables: any value outside [0, S) (none comes from
  // the screen) is replaced by 0 before use
  const int s0 = bs[0], s1 = bs[1];
  const int s_me = mine2 ? s1 : s0;
  int c[PB];
  {
    const uint2 cw = mine2 ? bcol[1] : bcol[0];
#pragma unroll
    for (int p = 0; p < PB; ++p) c[p] = (p < P) ? (int)(((p < 4 ? cw.x : cw.y) >> (8 * (p & 3))) & 0xFFu) : 0;
  }

  // projections through the transform of sigma .* d .* r: the best seed's
  // signs, then (when some tile of the wavefront needs it) the second's
  double bv[PB];
#pragma unroll
  for (int pass = 0; pass < 2; ++pass) {
    if (pass == 1 && !two) break;
    const uint32_t sw = pass ? bsgn[1] : bsgn[0];
    double v[kH];
#pragma unroll
    for (int j = 0; j < kH; ++j) {
      const double u = (double)dd[j] * (double)rr[j];
      v[j] = ((sw >> j) & 1u) ? -u : u;
    }
    fwht<kH>(v);
    wave_sync();
#pragma unroll
    for (int j = 0; j < kH; ++j) grow[kH * h + j] = v[j];
    wave_sync();
    if (mine2 == (pass == 1)) {
#pragma unroll
      for (int p = 0; p < PB; ++p) bv[p] = (p < P) ? tentry(grow, c[p]) * isq : 0.0;
    }
  }
  // Gram entries of this lane's seed through the transform of d
  double g[NG];
  {
    double v[kH];
#pragma unroll
    for (int j = 0; j < kH; ++j) v[j] = (double)dd[j];
    fwht<kH>(v);
    wave_sync();
#pragma unroll
    for (int j = 0; j < kH; ++j) grow[kH * h + j] = v[j];
    wave_sync();
#pragma unroll
    for (int p = 0; p < PB; ++p)
#pragma unroll
      for (int r = 0; r <= p; ++r) g[p * (p + 1) / 2 + r] = tentry(grow, c[p] ^ c[r]);
  }
  double L[PB * (PB - 1) / 2], e[PB], inv[PB];
  ldl64<kC, PB>(P, g, eps, L, e, inv);
  int q[PB];
  double al[PB];
  uint16_t bits;
  const double gk = solve_score_ldl<PB>(a, bv, L, e, inv, eps, qmax, q, al, &bits);

  // the better of the tile's two results (ties: the lower seed) is written
  // by the lane that holds it
  const uint64_t gb = (uint64_t)__double_as_longlong(gk);
  const auto xl = __builtin_amdgcn_permlane32_swap((uint32_t)gb, (uint32_t)gb, false, false);
  const auto xh = __builtin_amdgcn_permlane32_swap((uint32_t)(gb >> 32), (uint32_t)(gb >> 32), false, false);
  const double go = __longlong_as_double(
      (long long)((uint64_t)(h ? xl[0] : xl[1]) | ((uint64_t)(h ? xh[0] : xh[1]) << 32)));
  const bool second_wins = need && (h ? (gk > go || (gk == go && s1 < s0)) : (go > gk || (go == gk && s1 < s0)));
  if (valid && (h == 1) == second_wins) {
    const int64_t t = md.tile_off + row * nb + blk;
    a.seed_out[t] = (uint16_t)s_me;
    a.scale_out[t] = bits;
    a.gain_out[t] = gk;
    // the codes in one store when they fill an aligned word (P = 8 or 4)
    int8_t* cp = a.code_out + t * P;
    if (P == PB && (PB == 8 || PB == 4) && (reinterpret_cast<uintptr_t>(cp) & (PB - 1)) == 0) {
      uint64_t w = 0;
#pragma unroll
      for (int p = 0; p < PB; ++p) w |= (uint64_t)(uint8_t)q[p] << (8 * p);
      if (PB == 8) *reinterpret_cast<uint64_t*>(cp) = w;
      else *reinterpret_cast<uint32_t*>(cp) = (uint32_t)w;
    } else {
#pragma unroll
      for (int p = 0; p < PB; ++p)
        if (p < P) cp[p] = (int8_t)q[p];
    }
    if (a.alpha_out) {
#pragma unroll
      for (int p = 0; p < PB; ++p)
        if (p < P) a.alpha_out[t * P + p] = (float)al[p];
    }
  }
}

hipError_t launch_finalize_pe_modules(const EncodeArgs& a, const ModEntry* mods, int n_mods, int64_t items,
                                      hipStream_t st) {
  if (items == 0) return hipSuccess;
  if (a.P <= 4)
    hipLaunchKernelGGL((k_finalize_pe_modules<4>), dim3((unsigned)items), dim3(64), 0, st, a, mods, n_mods);
  else
    hipLaunchKernelGGL((k_finalize_pe_modules<8>), dim3((unsigned)items), dim3(64), 0, st, a, mods, n_mods);
  return hipGetLastError();
}

__global__ void k_pe_lists_tile_order(const float* __restrict__ tg, const uint32_t* __restrict__ ts,
                                      const ModEntry* __restrict__ mods, int n_mods, float* __restrict__ gout,
                                      uint32_t* __restrict__ sout) {
  const int64_t item = blockIdx.x;
  const int tl = threadIdx.x;
  const int m = find_module(mods, n_mods, item);
  const ModEntry md = mods[m];
  const int nb = (int)(md.cols / kC);
  const int64_t local = item - md.item_off;
  const int64_t row = (local / nb) * kPeRows + tl;
  if (row >= md.rows) return;
  const int64_t t = md.tile_off + row * nb + local % nb;
#pragma unroll
  for (int k = 0; k < kTop; ++k) {
    gout[t * kTop + k] = tg[item * (kTop * kPeRows) + k * kPeRows + tl];
    sout[t * kTop + k] = ts[item * (kTop * kPeRows) + k * kPeRows + tl];
  }
}

hipError_t launch_pe_lists_tile_order(const float* tg, const uint32_t* ts, const ModEntry* mods, int n_mods,
                                      int64_t items, float* gain_out, uint32_t* seed_out, hipStream_t st) {
  if (items == 0) return hipSuccess;
  hipLaunchKernelGGL(k_pe_lists_tile_order, dim3((unsigned)items), dim3(kPeRows), 0, st, tg, ts, mods, n_mods,
                     gain_out, seed_out);
  return hipGetLastError();
}

}  // namespace awsrc
