// fp64 re-score helpers shared by the encoder kernels (device code only).
#pragma once

#include <math.h>

#include "awsrc_internal.h"

namespace awsrc {

// fp16 scale of Sec. 3.2: f16(f32(v)) with saturation at 65504; returns bits.
__device__ __forceinline__ uint16_t scale_bits_from_f32(float v) {
  uint16_t hb = __half_as_ushort(__float2half_rn(v));
  if ((hb & 0x7FFFu) == 0x7C00u) hb = 0x7BFFu;
  return hb;
}

// The same from an fp64 quotient: round to fp32 first, then to fp16.  The
// empty asm keeps the fp32 value opaque; without it the compiler folds the two
// conversions into one fp64 -> fp16 rounding, which differs from the two-step
// rounding in about 7e-5 of cases (values near an fp16 rounding midpoint).
__device__ __forceinline__ uint16_t scale_bits_from_f64(double v) {
  float f = __double2float_rn(v);
  __asm__ volatile("" : "+v"(f));
  return scale_bits_from_f32(f);
}

// In-register fast Walsh-Hadamard transform, natural (Sylvester) order.
template <int C, typename T>
__device__ __forceinline__ void fwht(T (&v)[C]) {
#pragma unroll
  for (int h = 1; h < C; h <<= 1)
#pragma unroll
    for (int i = 0; i < C; i += 2 * h)
#pragma unroll
      for (int k = i; k < i + h; ++k) {
        const T x = v[k], y = v[k + h];
        v[k] = x + y;
        v[k + h] = x - y;
      }
}

// fp64 Cholesky factor of G + eps I for one seed: G_pq = wd[c_p ^ c_q] / C
// (wd = WHT of the weights, read through any pointer type), G + eps I =
// L L^T, inv_p = 1 / L_pp.  Padding columns p >= P get an identity row.
template <int C, int PB, typename WD>
__device__ __forceinline__ void chol64(int P, const WD& wd, const int (&c)[PB], double eps, double (&L)[PB][PB],
                                       double (&inv)[PB]) {
#pragma unroll
  for (int p = 0; p < PB; ++p)
#pragma unroll
    for (int r = 0; r <= p; ++r) {
      double acc;
      if (p < P && r < P) acc = wd[c[p] ^ c[r]] / C + (p == r ? eps : 0.0);
      else acc = (p == r) ? 1.0 : 0.0;
#pragma unroll
      for (int kk = 0; kk < r; ++kk) acc -= L[p][kk] * L[r][kk];
      if (p == r) {
        L[p][p] = sqrt(fmax(acc, 1e-300));
        inv[p] = 1.0 / L[p][p];
      } else {
        L[p][r] = acc * inv[r];
      }
    }
}

// fp64 re-score of one candidate from its projections bv = B^T u and the
// factor of its G + eps I: the solve for the unquantized fit al, the stored
// scale (bits) and codes q, and the gain 2 a.b - a^T G0 a of the quantized
// fit a = scale q (a^T G0 a = |L^T a|^2 - eps |a|^2).
template <int PB>
__device__ __forceinline__ double solve_score64(const EncodeArgs& a, const double (&bv)[PB], const double (&L)[PB][PB],
                                                const double (&inv)[PB], double eps, int qmax, int (&q)[PB],
                                                double (&al)[PB], uint16_t* bits_out) {
  double z[PB];
#pragma unroll
  for (int p = 0; p < PB; ++p) {
    double acc = bv[p];
#pragma unroll
    for (int kk = 0; kk < p; ++kk) acc -= L[p][kk] * z[kk];
    z[p] = acc * inv[p];
  }
#pragma unroll
  for (int p = PB - 1; p >= 0; --p) {
    double acc = z[p];
#pragma unroll
    for (int kk = p + 1; kk < PB; ++kk) acc -= L[kk][p] * al[kk];
    al[p] = acc * inv[p];
  }
  double m = 0.0;
#pragma unroll
  for (int p = 0; p < PB; ++p) m = fmax(m, fabs(al[p]));
  uint16_t bits = 0;
  double sc = 0.0;
  if (m > 0.0) {
    if (a.scale_fmt == AWSRC_SCALE_POW2) {
      // smallest e with m <= qmax 2^e, by exact comparisons; field e + 128
      int e;
      frexp(m / (double)qmax, &e);
      while (m > (double)qmax * ldexp(1.0, e)) ++e;
      while (m <= (double)qmax * ldexp(1.0, e - 1)) --e;
      e = e < -128 ? -128 : (e > 127 ? 127 : e);
      bits = (uint16_t)(e + 128);
      sc = ldexp(1.0, e);
    } else {
      // fp16 scale: f16(f32(m / qmax)), both round-to-nearest-even
      bits = scale_bits_from_f64(m / (double)qmax);
      sc = (double)__half2float(__ushort_as_half(bits));
      if (!(sc > 0.0)) { bits = 0; sc = 0.0; }
    }
  }
  double ah[PB];
#pragma unroll
  for (int p = 0; p < PB; ++p) {
    double qv = 0.0;
    if (sc > 0.0) qv = fmin(fmax(rint(al[p] / sc), (double)-qmax), (double)qmax);
    q[p] = (int)qv;
    ah[p] = sc * qv;
  }
  // gain = 2 a^T b - a^T G0 a, with a^T G0 a = |L^T a|^2 - eps |a|^2
  double t1 = 0.0, aa = 0.0, quad = 0.0;
#pragma unroll
  for (int p = 0; p < PB; ++p) { t1 += ah[p] * bv[p]; aa += ah[p] * ah[p]; }
#pragma unroll
  for (int kk = 0; kk < PB; ++kk) {
    double y = 0.0;
#pragma unroll
    for (int i = kk; i < PB; ++i) y += L[i][kk] * ah[i];
    quad += y * y;
  }
  *bits_out = bits;
  return 2.0 * t1 - (quad - eps * aa);
}


// 1 / x in fp64: the hardware reciprocal refined by two Newton steps (the
// error of the estimate squares at each step; well inside the solve's own
// rounding).
__device__ __forceinline__ double recip64(double x) {
  double r = __builtin_amdgcn_rcp(x);
  r = fma(r, fma(-x, r, 1.0), r);
  return fma(r, fma(-x, r, 1.0), r);
}

// G + eps I = L diag(e) L^T (L unit lower triangular, strict part packed by
// rows) in fp64 from the gathered transform values g (packed lower triangle
// with the diagonal; G_pr = g / C); inv = 1 / e.  Padding columns p >= P get
// L = 0, e = 1.  No square roots, one reciprocal per pivot.
template <int C, int PB>
__device__ __forceinline__ void ldl64(int P, const double (&g)[PB * (PB + 1) / 2], double eps,
                                      double (&L)[PB * (PB - 1) / 2], double (&e)[PB], double (&inv)[PB]) {
#pragma unroll
  for (int p = 0; p < PB; ++p) {
    double E[PB];  // row p of L diag(e)
#pragma unroll
    for (int r = 0; r < p; ++r) {
      double acc = (p < P && r < P) ? g[p * (p + 1) / 2 + r] * (1.0 / C) : 0.0;
#pragma unroll
      for (int k = 0; k < r; ++k) acc = fma(-E[k], L[ltri(r, k)], acc);
      E[r] = acc;
      L[ltri(p, r)] = acc * inv[r];
    }
    double acc = p < P ? fma(g[p * (p + 1) / 2 + p], 1.0 / C, eps) : 1.0;
#pragma unroll
    for (int k = 0; k < p; ++k) acc = fma(-E[k], L[ltri(p, k)], acc);
    e[p] = fmax(acc, 1e-300);
    inv[p] = recip64(e[p]);
  }
}

// The fp64 re-score of one candidate from its projections bv = B^T u and the
// factor of its G + eps I: the solve of Eq. (3) for the unquantized fit al,
// the stored scale (bits) and codes q (Sec. 3.2), and the gain
// 2 a.b - a^T G0 a of the quantized fit a = scale q, with
// a^T G0 a = sum_k e_k ((L^T a)_k)^2 - eps |a|^2.
template <int PB>
__device__ __forceinline__ double solve_score_ldl(const EncodeArgs& a, const double (&bv)[PB],
                                                  const double (&L)[PB * (PB - 1) / 2], const double (&e)[PB],
                                                  const double (&inv)[PB], double eps, int qmax, int (&q)[PB],
                                                  double (&al)[PB], uint16_t* bits_out) {
  double z[PB];
#pragma unroll
  for (int p = 0; p < PB; ++p) {
    double acc = bv[p];
#pragma unroll
    for (int k = 0; k < p; ++k) acc = fma(-L[ltri(p, k)], z[k], acc);
    z[p] = acc;
  }
#pragma unroll
  for (int p = PB - 1; p >= 0; --p) {
    double acc = z[p] * inv[p];
#pragma unroll
    for (int k = p + 1; k < PB; ++k) acc = fma(-L[ltri(k, p)], al[k], acc);
    al[p] = acc;
  }
  double m = 0.0;
#pragma unroll
  for (int p = 0; p < PB; ++p) m = fmax(m, fabs(al[p]));
  uint16_t bits = 0;
  double sc = 0.0;
  if (m > 0.0) {
    if (a.scale_fmt == AWSRC_SCALE_POW2) {
      // smallest e with m <= qmax 2^e, by exact comparisons; field e + 128
      int ex;
      frexp(m / (double)qmax, &ex);
      while (m > (double)qmax * ldexp(1.0, ex)) ++ex;
      while (m <= (double)qmax * ldexp(1.0, ex - 1)) --ex;
      ex = ex < -128 ? -128 : (ex > 127 ? 127 : ex);
      bits = (uint16_t)(ex + 128);
      sc = ldexp(1.0, ex);
    } else {
      // fp16 scale: f16(f32(m / qmax)), both round-to-nearest-even
      bits = scale_bits_from_f64(m / (double)qmax);
      sc = (double)__half2float(__ushort_as_half(bits));
      if (!(sc > 0.0)) { bits = 0; sc = 0.0; }
    }
  }
  const double isc = sc > 0.0 ? 1.0 / sc : 0.0;
  double ah[PB];
#pragma unroll
  for (int p = 0; p < PB; ++p) {
    const double qv = fmin(fmax(rint(al[p] * isc), (double)-qmax), (double)qmax);
    q[p] = (int)qv;
    ah[p] = sc * qv;
  }
  double t1 = 0.0, aa = 0.0, quad = 0.0;
#pragma unroll
  for (int p = 0; p < PB; ++p) {
    t1 = fma(ah[p], bv[p], t1);
    aa = fma(ah[p], ah[p], aa);
  }
#pragma unroll
  for (int k = 0; k < PB; ++k) {
    double y = ah[k];
#pragma unroll
    for (int i = k + 1; i < PB; ++i) y = fma(L[ltri(i, k)], ah[i], y);
    quad = fma(e[k] * y, y, quad);
  }
  *bits_out = bits;
  return 2.0 * t1 - (quad - eps * aa);
}

// Loads through a global-address-space view: global (not flat) loads, which
// count on the vector-memory counter only, so that a wait for them does not
// also wait for LDS work.
typedef float gf32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t gu32x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ gf32x4 gload4f(const float* p) {
  return *(const __attribute__((address_space(1))) gf32x4*)(p);
}
__device__ __forceinline__ gu32x2 gload2u(const uint16_t* p) {
  return *(const __attribute__((address_space(1))) gu32x2*)(p);
}

// Four consecutive weights of W (fp32 or bf16) and of W0 at each of NP
// element offsets: every load is issued before any is used (one wait for
// all of them; the dtype branch is taken once, outside the loads), and
// r = f32(W - W0).
template <int NP>
__device__ __forceinline__ void load_residual4(const void* W, int w_dtype, const float* W0, const int64_t (&o)[NP],
                                               float (&r)[NP][4]) {
  gf32x4 y[NP];
  if (w_dtype == AWSRC_DTYPE_F32) {
    gf32x4 x[NP];
#pragma unroll
    for (int p = 0; p < NP; ++p) x[p] = gload4f(static_cast<const float*>(W) + o[p]);
#pragma unroll
    for (int p = 0; p < NP; ++p) y[p] = gload4f(W0 + o[p]);
#pragma unroll
    for (int p = 0; p < NP; ++p)
#pragma unroll
      for (int k = 0; k < 4; ++k) r[p][k] = x[p][k] - y[p][k];
  } else {
    gu32x2 x[NP];
#pragma unroll
    for (int p = 0; p < NP; ++p) x[p] = gload2u(static_cast<const uint16_t*>(W) + o[p]);
#pragma unroll
    for (int p = 0; p < NP; ++p) y[p] = gload4f(W0 + o[p]);
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      r[p][0] = __uint_as_float(x[p][0] << 16) - y[p][0];
      r[p][1] = __uint_as_float(x[p][0] & 0xFFFF0000u) - y[p][1];
      r[p][2] = __uint_as_float(x[p][1] << 16) - y[p][2];
      r[p][3] = __uint_as_float(x[p][1] & 0xFFFF0000u) - y[p][3];
    }
  }
}

// Loads 8 consecutive weights of W (fp32 or bf16) starting at element i.
__device__ __forceinline__ void load8_w(const void* W, int dt, int64_t i, float (&w)[8]) {
  if (dt == AWSRC_DTYPE_F32) {
    const float4* p = reinterpret_cast<const float4*>(static_cast<const float*>(W) + i);
    const float4 x = p[0], y = p[1];
    w[0] = x.x; w[1] = x.y; w[2] = x.z; w[3] = x.w; w[4] = y.x; w[5] = y.y; w[6] = y.z; w[7] = y.w;
  } else {
    const uint4 x = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(W) + i);
    const uint32_t v[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      w[2 * k] = __uint_as_float(v[k] << 16);
      w[2 * k + 1] = __uint_as_float(v[k] & 0xFFFF0000u);
    }
  }
}

__device__ __forceinline__ void load8_f(const float* p, float (&w)[8]) {
  const float4 x = reinterpret_cast<const float4*>(p)[0], y = reinterpret_cast<const float4*>(p)[1];
  w[0] = x.x; w[1] = x.y; w[2] = x.z; w[3] = x.w; w[4] = y.x; w[5] = y.y; w[6] = y.z; w[7] = y.w;
}

// LDS floats that rescore_block64 needs: the 64 x 65 residual rows (later
// the 32 x 65 fp64 gather rows), the block's d and its WHT (64 doubles).
constexpr int kRescoreLds = 64 * 65 + 64 + 2 * 64;

// fp64 re-score of the 64 tiles (rows row0 .. row0 + 63) of column block blk,
// per-column weights, generator version 1, C = 64, one tile per lane, from
// each tile's kept seeds (tg: screened gains in decreasing order, -inf for
// none; ts: their seeds); writes the encoder outputs.  Called by a whole
// wavefront (every lane), with `lds` kRescoreLds floats of its own.
//
// Each lane keeps its tile in registers (fp64) and transforms it in place;
// the residual block comes in through LDS, loaded with 16 lanes per row
// segment (4 rows per pass) so that each cache line is read whole by one
// instruction (row-per-lane loads of 16 bytes left each line to 8 or 16
// instructions, and with two wavefronts per SIMD the lines in flight
// outgrew the L2 and were fetched again), and only the gather of the P
// projections out of the transform goes through LDS again, half a
// wavefront at a time.  A second kept seed (a near tie, rare) reloads the
// tile's row directly.
template <int PB>
__device__ __forceinline__ void rescore_block64(const EncodeArgs& a, int blk, int64_t row0, const float (&tg)[kTop],
                                                const uint32_t (&ts)[kTop], float* lds) {
  constexpr int C = 64;
  const int lane = threadIdx.x & 63;
  const int nb = (int)(a.cols / C);
  float* rsh = lds;                                          // [64][C + 1] fp32 rows
  double* gb = reinterpret_cast<double*>(lds);               // [32][C + 1] fp64 gather rows (later)
  float* dsh = lds + 64 * (C + 1);                           // the block's d
  double* wdsh = reinterpret_cast<double*>(dsh + C);         // its WHT, for the Gram entries
  const int64_t row = row0 + lane;
  dsh[lane] = a.d[(int64_t)blk * C + lane];
  wdsh[lane] = a.wd64[(int64_t)blk * C + lane];
  {
    const int pc = lane & 15;
    int64_t o[16];
#pragma unroll
    for (int pass = 0; pass < 16; ++pass) {
      const int rl = 4 * pass + (lane >> 4);
      const int64_t rg = row0 + rl < a.rows ? row0 + rl : a.rows - 1;
      o[pass] = rg * a.cols + (int64_t)blk * C + 4 * pc;
    }
    float rv[16][4];
    load_residual4<16>(a.W, a.w_dtype, a.W0, o, rv);  // every load issued before any is used
#pragma unroll
    for (int pass = 0; pass < 16; ++pass) {
      const int rl = 4 * pass + (lane >> 4);
#pragma unroll
      for (int k = 0; k < 4; ++k) rsh[rl * (C + 1) + 4 * pc + k] = rv[pass][k];
    }
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  if (row >= a.rows) return;  // no cross-lane exchange below but the gather's (per row pair)
  const int64_t off = row * a.cols + (int64_t)blk * C;
  const int64_t t = row * nb + blk;
  const int P = a.P;
  const double isq = 1.0 / sqrt((double)C);
  const int qmax = (1 << (a.b - 1)) - 1;
  double* grow = &gb[(lane & 31) * (C + 1)];

  // Score seed s: u = d .* r in fp64 (also the tile's weighted energy e32 and
  // sum of d), sigma .* u transformed in place, the P projections gathered
  // through this lane's LDS row (lanes l and l + 32 share a row, so the two
  // halves take turns, ordered by the wavefront barriers), then the solve
  // with the Cholesky factor of the seed's G + eps I.
  auto score = [&](int s, bool first, float* e32, int (&q)[PB], double (&al)[PB], uint16_t* bits) -> double {
    // r: the first seed's from the LDS rows, a second seed's (after the
    // gather has reused the buffer) loaded directly; then u with the
    // block's d from LDS
    float rr[C];
    if (first) {
#pragma unroll
      for (int j = 0; j < C; ++j) rr[j] = rsh[lane * (C + 1) + j];
    } else {
#pragma unroll
      for (int j0 = 0; j0 < C; j0 += 8) {
        float wv[8], w0[8];
        load8_w(a.W, a.w_dtype, off + j0, wv);
        load8_f(a.W0 + off + j0, w0);
#pragma unroll
        for (int k = 0; k < 8; ++k) rr[j0 + k] = wv[k] - w0[k];
      }
    }
    double u[C];
    float e = 0.0f;
    double sumd = 0.0;
#pragma unroll
    for (int j = 0; j < C; ++j) {
      const float dj = dsh[j];
      e += dj * rr[j] * rr[j];
      sumd += (double)dj;
      u[j] = (double)dj * (double)rr[j];
    }
    // pin e and sumd here: left to the compiler, their sums sink to their
    // uses after the transform and keep r and d live (and spilled) across it
    asm volatile("" ::"v"(e), "v"(sumd));
    *e32 = e;
    const double eps = a.lambda * (sumd / C);
    const uint64_t s0 = a.basis.sign[(size_t)s * 2];
    int c[PB];
#pragma unroll
    for (int p = 0; p < PB; ++p) c[p] = (p < P) ? a.basis.col[(size_t)s * kMaxP + p] : 0;
#pragma unroll
    for (int i = 0; i < C; ++i) u[i] = ((s0 >> i) & 1ull) ? -u[i] : u[i];
    fwht<C>(u);
    double bv[PB];
#pragma unroll
    for (int ph = 0; ph < 2; ++ph) {
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      if ((lane >> 5) == ph) {
#pragma unroll
        for (int j = 0; j < C; ++j) grow[j] = u[j];
#pragma unroll
        for (int p = 0; p < PB; ++p) bv[p] = (p < P) ? grow[c[p]] * isq : 0.0;
      }
    }
    // the transform is dead from here
    __builtin_amdgcn_sched_barrier(0);
    double L[PB][PB], inv[PB];
    chol64<C, PB>(P, wdsh, c, eps, L, inv);
    return solve_score64<PB>(a, bv, L, inv, eps, qmax, q, al, bits);
  };

  int best_q[PB];
  double best_al[PB];
  uint16_t best_bits;
  float e32;
  int best_s = list_seed(ts[0]);
  double best_g = score(best_s, true, &e32, best_q, best_al, &best_bits);
  // the second kept seed only when its screened gain lies within the
  // re-score's window of the best (the wide one if either is a knife edge)
  const float thr = tg[0] - rescore_window(tg[0], e32, ((ts[0] | ts[1]) & kEdge) != 0);
#pragma unroll
  for (int k = 1; k < kTop; ++k) {
    if (tg[k] >= thr && tg[k] > -INFINITY) {
      int q[PB];
      double al[PB];
      uint16_t bits;
      float e_;
      const int sk = list_seed(ts[k]);
      const double g = score(sk, false, &e_, q, al, &bits);
      if (g > best_g || (g == best_g && sk < best_s)) {
        best_g = g;
        best_s = sk;
        best_bits = bits;
#pragma unroll
        for (int p = 0; p < PB; ++p) { best_q[p] = q[p]; best_al[p] = al[p]; }
      }
    }
  }
  a.seed_out[t] = (uint16_t)best_s;
  a.scale_out[t] = best_bits;
  a.gain_out[t] = best_g;
#pragma unroll
  for (int p = 0; p < PB; ++p) {
    if (p < P) {
      a.code_out[t * P + p] = (int8_t)best_q[p];
      if (a.alpha_out) a.alpha_out[t * P + p] = (float)best_al[p];
    }
  }
}

// fp64 Cholesky factor of G + eps I for one seed from its gathered Gram
// entries g (packed lower triangle with the diagonal, (p, r) at
// p (p + 1) / 2 + r, unscaled transform values: G_pr = g / C), G + eps I =
// L L^T, inv_p = 1 / L_pp.  Padding columns p >= P get an identity row.
template <int C, int PB>
__device__ __forceinline__ void chol64_vals(int P, const double (&g)[PB * (PB + 1) / 2], double eps,
                                            double (&L)[PB][PB], double (&inv)[PB]) {
#pragma unroll
  for (int p = 0; p < PB; ++p)
#pragma unroll
    for (int r = 0; r <= p; ++r) {
      double acc;
      if (p < P && r < P) acc = g[p * (p + 1) / 2 + r] / C + (p == r ? eps : 0.0);
      else acc = (p == r) ? 1.0 : 0.0;
#pragma unroll
      for (int kk = 0; kk < r; ++kk) acc -= L[p][kk] * L[r][kk];
      if (p == r) {
        L[p][p] = sqrt(fmax(acc, 1e-300));
        inv[p] = 1.0 / L[p][p];
      } else {
        L[p][r] = acc * inv[r];
      }
    }
}

}  // namespace awsrc
