// Encoder seed search (Sec. 3.2): for every tile r_t and every seed s, fit the
// activation-weighted ridge least squares of Eq. (3) in the basis B_s of
// Eq. (2), quantize the coefficients with one fp16 scale, and score the
// weighted error reduction of the quantized reconstruction (numerator of
// Eq. (4)); keep the seed with the largest reduction.
//
// Two passes share one set of tables:
//  * screen   - every (tile, seed) in fp32, one lane per tile; the seed loop
//               is uniform across the wavefront, so basis patterns and the
//               per-column factors are scalar loads.  The four best screened
//               seeds of each tile are kept.
//  * finalize - the screened seeds whose fp32 gain lies within a small margin
//               of the best are re-scored in fp64 with the complete chain
//               (projection, Gram matrix, Cholesky solve, quantization,
//               gain in its definition form); outputs come from that pass.
//
// Identities used (they follow from B_s having orthonormal +-1/sqrt(C)
// columns of a Sylvester Hadamard matrix):
//  * G = B^T D B has entries (1/C) sum_j d_j (-1)^popcount(j & (c_p xor c_q)),
//    independent of the sign pattern, so for per-column weights G and its
//    Cholesky factor depend only on (column block, seed);
//  * for per-element weights G_pq = WHT(d_t)[c_p xor c_q] / C, one fast
//    Walsh-Hadamard transform of d_t per tile;
//  * sum_j d_j (r_j^2 - (r_j - [B a]_j)^2) = 2 a^T b - a^T G0 a with
//    b = B^T D r and G0 = B^T D B (screening only).
#include <math.h>

#include "awsrc_internal.h"

namespace awsrc {

namespace {

template <int C>
struct InvSqrtC;
template <> struct InvSqrtC<16> { static constexpr float v = 0.25f; };
template <> struct InvSqrtC<32> { static constexpr float v = 0.17677669529663688f; };
template <> struct InvSqrtC<64> { static constexpr float v = 0.125f; };
template <> struct InvSqrtC<128> { static constexpr float v = 0.08838834764831845f; };

__device__ __forceinline__ float load_w_any(const void* W, int dt, int64_t i) {
  if (dt == AWSRC_DTYPE_F32) return static_cast<const float*>(W)[i];
  return __uint_as_float((uint32_t)static_cast<const uint16_t*>(W)[i] << 16);
}


// fp16 scale of Sec. 3.2: f16(f32(v)) with saturation at 65504; returns bits.
__device__ __forceinline__ uint16_t scale_bits_from_f32(float v) {
  uint16_t hb = __half_as_ushort(__float2half_rn(v));
  if ((hb & 0x7FFFu) == 0x7C00u) hb = 0x7BFFu;
  return hb;
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

}  // namespace

// ----------------------------------------------------------------------------
// fp64 Walsh-Hadamard transform of each column block's weights (per-column
// mode): the Gram entries of every seed are gathers from it.
template <int C>
__global__ __launch_bounds__(64) void k_block_wht64(const float* __restrict__ d, int nb, double* __restrict__ out) {
  // one wavefront per block; lane l holds coordinates l + 64 k.  Stage h of
  // the butterfly pairs coordinates j and j ^ h: the one without bit h gets
  // x + y, the other x - y (x the lower, y the upper), the same additions as
  // the in-register transform, so the results are identical.
  constexpr int V = C > 64 ? C / 64 : 1;
  const int blk = blockIdx.x;
  const int lane = threadIdx.x;
  double v[V];
#pragma unroll
  for (int k = 0; k < V; ++k) {
    const int j = lane + 64 * k;
    v[k] = j < C ? (double)d[(int64_t)blk * C + j] : 0.0;
  }
#pragma unroll
  for (int h = 1; h < C && h < 64; h <<= 1) {
#pragma unroll
    for (int k = 0; k < V; ++k) {
      const double o = __shfl_xor(v[k], h, 64);
      v[k] = (lane & h) ? o - v[k] : v[k] + o;
    }
  }
  if constexpr (V == 2) {
    const double x = v[0], y = v[1];
    v[0] = x + y;
    v[1] = x - y;
  }
#pragma unroll
  for (int k = 0; k < V; ++k) {
    const int j = lane + 64 * k;
    if (j < C) out[(int64_t)blk * C + j] = v[k];
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

// ----------------------------------------------------------------------------
// Per-column factor table: for each (column block, seed), G = B^T D B + eps I
// in fp64, its Cholesky factor stored in fp32 for the screen:
//   [packed lower L (PB(PB+1)/2)] [1/L_pp (PB)] [eps]
// Padding columns p >= P get an identity row so that the padded system solves
// to alpha_p = 0.
// Generator version 2 permutes the coordinates, so the XOR identity no longer
// applies: G_pq = (sum_j d_j - 2 sum of d_j where B_s[j, p] and B_s[j, q]
// differ in sign) / C, from the negative-entry patterns and the block's d
// staged in LDS.  Grid: (seed groups of 64, column blocks).
template <int C, int PB>
__global__ __launch_bounds__(64) void k_col_factors(EncodeArgs a, int nb, int stride) {
  __shared__ double sd[C];
  const int blk = blockIdx.y;
  const int s = blockIdx.x * 64 + threadIdx.x;
  if (a.gen_version != 1) {
    for (int j = threadIdx.x; j < C; j += 64) sd[j] = (double)a.d[(int64_t)blk * C + j];
    __syncthreads();
  }
  if (s >= a.S) return;
  const int64_t idx = (int64_t)blk * a.S + s;
  const uint8_t* cs = a.basis.col + (size_t)s * kMaxP;
  double G[PB][PB];
  if (a.gen_version == 1) {
    const double* wd = a.wd64 + (int64_t)blk * C;  // WHT(d) of this block: G_pq = wd[c_p ^ c_q] / C
    const double eps = a.lambda * (wd[0] / C);
#pragma unroll
    for (int p = 0; p < PB; ++p)
#pragma unroll
      for (int q = 0; q <= p; ++q) {
        double g;
        if (p < a.P && q < a.P) g = wd[cs[p] ^ cs[q]] / C + (p == q ? eps : 0.0);
        else g = (p == q) ? 1.0 : 0.0;
        G[p][q] = g;
      }
  } else {
    double sum = 0.0;
    for (int j = 0; j < C; ++j) sum += sd[j];
    const double eps = a.lambda * (sum / C);
    const uint64_t* mk = a.basis.mask + (size_t)s * a.P * 2;
#pragma unroll
    for (int p = 0; p < PB; ++p)
#pragma unroll
      for (int q = 0; q <= p; ++q) {
        double g;
        if (p < a.P && q < a.P) {
          double acc = sum;
          if (p != q) {
            double diff = 0.0;
#pragma unroll
            for (int w = 0; w < (C + 63) / 64; ++w) {
              const uint64_t x = mk[2 * p + w] ^ mk[2 * q + w];
              for (int j = 0; j < (C < 64 ? C : 64); ++j)
                if ((x >> j) & 1ull) diff += sd[64 * w + j];
            }
            acc -= 2.0 * diff;
          }
          g = acc / C + (p == q ? eps : 0.0);
        } else {
          g = (p == q) ? 1.0 : 0.0;
        }
        G[p][q] = g;
      }
  }
  // LDL^T (G is SPD: d > 0 and the columns are orthonormal)
  double L[PB][PB], e[PB];
#pragma unroll
  for (int p = 0; p < PB; ++p) {
#pragma unroll
    for (int q = 0; q < p; ++q) {
      double acc = G[p][q];
#pragma unroll
      for (int k = 0; k < q; ++k) acc -= L[p][k] * L[q][k] * e[k];
      L[p][q] = acc / e[q];
    }
    double acc = G[p][p];
#pragma unroll
    for (int k = 0; k < p; ++k) acc -= L[p][k] * L[p][k] * e[k];
    e[p] = fmax(acc, 1e-300);
  }
  float* out = a.colfac + (size_t)idx * stride;
#pragma unroll
  for (int p = 0; p < PB; ++p) {
#pragma unroll
    for (int q = 0; q < p; ++q) out[ltri(p, q)] = (float)L[p][q];
    out[PB * (PB - 1) / 2 + p] = (float)(1.0 / e[p]);
    out[PB * (PB - 1) / 2 + PB + p] = (float)e[p];
  }
}

// ----------------------------------------------------------------------------
// fp32 screen of all seeds.  Wavefront = 64 consecutive rows of one column
// block; lane = tile.  Keeps the kTop best (gain, seed) per tile, ties to the
// lower seed.
template <int C, int PB, bool PE, bool V2>
__global__ __launch_bounds__(64) void k_screen_valu(EncodeArgs a, int stride) {
  // generator version 2 with per-element weights: each seed's Gram comes
  // from the transform of its permuted d, gathered from the lane's raw d row
  __shared__ float s_draw[V2 ? 64 * (C + 1) : 1];
  const int nb = (int)(a.cols / C);
  const int blk = blockIdx.x % nb;
  const int64_t row = (int64_t)(blockIdx.x / nb) * 64 + threadIdx.x;
  const bool active = row < a.rows;
  const int64_t rr = active ? row : a.rows - 1;
  const int64_t off = rr * a.cols + (int64_t)blk * C;
  const int P = a.P;
  float u[C];
  float wd[PE ? C : 1];
#pragma unroll
  for (int j = 0; j < C; ++j) {
    const float r = load_w_any(a.W, a.w_dtype, off + j) - a.W0[off + j];
    const float dj = PE ? a.d[off + j] : a.d[(int64_t)blk * C + j];
    u[j] = dj * r;
    if constexpr (PE && V2) s_draw[threadIdx.x * (C + 1) + j] = dj;
    else if constexpr (PE) wd[j] = dj;
  }
  if constexpr (PE && !V2) fwht<C>(wd);
  const float qmax = (float)((1 << (a.b - 1)) - 1);
  const float inv_qmax = 1.0f / qmax;
  const bool pow2 = a.scale_fmt == AWSRC_SCALE_POW2;
  const float invC = 1.0f / C;
  float tg[kTop];
  int ts[kTop];
#pragma unroll
  for (int k = 0; k < kTop; ++k) { tg[k] = -INFINITY; ts[k] = 0; }

  for (int s = 0; s < a.S; ++s) {
    // projection b = B_s^T (d .* r)
    float bv[PB];
    const uint64_t* mk = a.basis.mask + (size_t)s * P * 2;
#pragma unroll
    for (int p = 0; p < PB; ++p) {
      float acc = 0.0f;
      if (p < P) {
        const uint64_t m0 = mk[2 * p], m1 = mk[2 * p + 1];
#pragma unroll
        for (int j = 0; j < C; ++j) {
          const uint64_t m = (j < 64) ? m0 : m1;
          acc += ((m >> (j & 63)) & 1ull) ? -u[j] : u[j];
        }
      }
      bv[p] = acc * InvSqrtC<C>::v;
    }
    float g;
    if constexpr (PE) {
      // Cholesky factor of G = B^T D B + eps I from the Gram gathers
      float L[PB][PB], inv[PB];
      const uint8_t* cs = a.basis.col + (size_t)s * kMaxP;
      int c[PB];
#pragma unroll
      for (int p = 0; p < PB; ++p) c[p] = (p < P) ? cs[p] : 0;
      if constexpr (V2) {
        // WHT(d o pi^-1): coordinate i of the permuted vector is d at pi^-1(i)
        const uint8_t* ip = a.basis.iperm + (size_t)s * kMaxC;
#pragma unroll
        for (int i = 0; i < C; ++i) wd[i] = s_draw[threadIdx.x * (C + 1) + ip[i]];
        fwht<C>(wd);
      }
      const float eps = (float)a.lambda * wd[0] * invC;
#pragma unroll
      for (int p = 0; p < PB; ++p)
#pragma unroll
        for (int q = 0; q <= p; ++q) {
          float acc;
          if (p < P && q < P) acc = wd[c[p] ^ c[q]] * invC + (p == q ? eps : 0.0f);
          else acc = (p == q) ? 1.0f : 0.0f;
#pragma unroll
          for (int k = 0; k < q; ++k) acc -= L[p][k] * L[q][k];
          if (p == q) {
            L[p][p] = sqrtf(fmaxf(acc, 1e-30f));
            inv[p] = 1.0f / L[p][p];
          } else {
            L[p][q] = acc * inv[q];
          }
        }
      // solve L L^T alpha = b
      float z[PB], al[PB];
#pragma unroll
      for (int p = 0; p < PB; ++p) {
        float acc = bv[p];
#pragma unroll
        for (int k = 0; k < p; ++k) acc -= L[p][k] * z[k];
        z[p] = acc * inv[p];
      }
#pragma unroll
      for (int p = PB - 1; p >= 0; --p) {
        float acc = z[p];
#pragma unroll
        for (int k = p + 1; k < PB; ++k) acc -= L[k][p] * al[k];
        al[p] = acc * inv[p];
      }
      // quantize with one fp16 scale and score
      float m = 0.0f;
#pragma unroll
      for (int p = 0; p < PB; ++p) m = fmaxf(m, fabsf(al[p]));
      float isc;
      const float sc = pow2 ? screen_scale<true>(m, inv_qmax, &isc) : screen_scale<false>(m, inv_qmax, &isc);
      g = 0.0f;
      if (sc > 0.0f) {
        float q[PB], t1 = 0.0f, qq = 0.0f;
#pragma unroll
        for (int p = 0; p < PB; ++p) {
          q[p] = fminf(fmaxf(rintf(al[p] * isc), -qmax), qmax);
          t1 += q[p] * bv[p];
          qq += q[p] * q[p];
        }
        float quad = 0.0f;
#pragma unroll
        for (int k = 0; k < PB; ++k) {
          float y = 0.0f;
#pragma unroll
          for (int i = k; i < PB; ++i) y += L[i][k] * q[i];
          quad += y * y;
        }
        quad -= eps * qq;
        g = sc * (2.0f * t1 - sc * quad);
      }
    } else {
      const float* fs = a.colfac + ((size_t)blk * a.S + s) * stride;
      g = pow2 ? screen_score_ldl<PB, true>(bv, fs, qmax, inv_qmax) : screen_score_ldl<PB, false>(bv, fs, qmax, inv_qmax);
    }
    // keep the best kTop, earlier (lower) seeds first among equals
    float cg = g;
    int cs_ = s;
#pragma unroll
    for (int k = 0; k < kTop; ++k) {
      if (cg > tg[k]) {
        const float tgk = tg[k];
        const int tsk = ts[k];
        tg[k] = cg; ts[k] = cs_;
        cg = tgk; cs_ = tsk;
      }
    }
  }
  if (active) {
    const int64_t t = row * nb + blk;
#pragma unroll
    for (int k = 0; k < kTop; ++k) {
      a.top_gain[t * kTop + k] = tg[k];
      a.top_seed[t * kTop + k] = (uint16_t)ts[k];
    }
  }
}

// ----------------------------------------------------------------------------
// fp64 re-score of the screened candidates; writes the encoder outputs.
// For one (tile, seed): b = WHT(sigma .* d .* r)[c] / sqrt(C) and
// G_pq = WHT(d)[c_p xor c_q] / C (+ eps on the diagonal), Cholesky solve,
// fp16-scale quantization, and the gain 2 a^T b - a^T G0 a of the quantized
// coefficients a (G0 = G without the ridge), all in fp64.  Each lane keeps
// its transformed vector in a private LDS row for the data-dependent gathers.
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

// u_j = d_j r_j in fp64 (exact: a product of two fp32 values) into the lane's LDS row.
template <int C, bool PE>
__device__ __forceinline__ void tile_u64(const EncodeArgs& a, int64_t off, int blk, double* my, float* e32,
                                          double* sumd) {
  float e = 0.0f;
  double sd = 0.0;
#pragma unroll 2
  for (int j0 = 0; j0 < C; j0 += 8) {
    float w[8], w0[8], dj[8];
    load8_w(a.W, a.w_dtype, off + j0, w);
    load8_f(a.W0 + off + j0, w0);
    load8_f(PE ? a.d + off + j0 : a.d + (int64_t)blk * C + j0, dj);
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const float r = w[k] - w0[k];
      e += dj[k] * r * r;
      sd += (double)dj[k];
      my[j0 + k] = (double)dj[k] * (double)r;
    }
  }
  *e32 = e;
  *sumd = sd;
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
      bits = scale_bits_from_f32(__double2float_rn(m / (double)qmax));
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

template <int C, int PB, bool PE>
__global__ __launch_bounds__(64) void k_finalize(EncodeArgs a, const double* __restrict__ wdb) {
  constexpr int NT = (C == 128) ? 32 : 64;  // rows per workgroup (keeps the LDS rows under 64 KiB)
  extern __shared__ double fsh[];
  double* my = fsh + threadIdx.x * (C + 1);
  const int nb = (int)(a.cols / C);
  // Workgroups are dealt to the 8 XCDs round-robin by index: give each XCD a
  // contiguous run of (row group, column block) items, so that neighbouring
  // column blocks (adjacent per-tile outputs) share one L2.
  const int64_t nwg = gridDim.x;
  const int64_t xcd = blockIdx.x % 8, q = nwg / 8, rem = nwg % 8;
  const int64_t w = xcd * q + (xcd < rem ? xcd : rem) + blockIdx.x / 8;
  const int blk = (int)(w % nb);
  const int64_t row = (w / nb) * NT + threadIdx.x;
  if (row >= a.rows) return;
  const int64_t off = row * a.cols + (int64_t)blk * C;
  const int64_t t = row * nb + blk;
  const int P = a.P;
  float e32;
  double sumd;
  tile_u64<C, PE>(a, off, blk, my, &e32, &sumd);
  bool row_is_u = true;  // my[] holds u (true) or a transformed vector (false)
  const double eps = a.lambda * (sumd / C);
  const double isq = 1.0 / sqrt((double)C);
  const int qmax = (1 << (a.b - 1)) - 1;

  // merge the seed ranges' lists into the best kTop: ranges come in seed order
  // and each list is ordered (gain desc, seed asc), so strict comparisons
  // keep the lower seed first among equal gains
  float tg[kTop];
  int ts[kTop];
#pragma unroll
  for (int k = 0; k < kTop; ++k) { tg[k] = -INFINITY; ts[k] = 0; }
  for (int sp = 0; sp < a.nsplit; ++sp) {
#pragma unroll
    for (int k = 0; k < kTop; ++k) {
      const int64_t at = (t * a.nsplit + sp) * kTop + k;
      float g = a.top_gain[at];
      int sd = a.top_seed[at];
#pragma unroll
      for (int m = 0; m < kTop; ++m) {
        if (g > tg[m]) {
          const float tgm = tg[m];
          const int tsm = ts[m];
          tg[m] = g; ts[m] = sd;
          g = tgm; sd = tsm;
        }
      }
    }
  }
  const float thr = tg[0] - (1e-4f * fabsf(tg[0]) + 1e-7f * e32);

  double best_g = -INFINITY;
  int best_s = 0x7FFFFFFF;
  int best_q[PB];
  uint16_t best_bits = 0;
  float best_al[PB];
#pragma unroll
  for (int p = 0; p < PB; ++p) { best_q[p] = 0; best_al[p] = 0.f; }

  for (int k = 0; k < kTop; ++k) {
    if (k > 0 && !(tg[k] >= thr && tg[k] > -INFINITY)) continue;
    const int s = ts[k];
    const uint64_t* sw = a.basis.sign + (size_t)s * 2;
    const uint8_t* cs = a.basis.col + (size_t)s * kMaxP;
    int c[PB];
#pragma unroll
    for (int p = 0; p < PB; ++p) c[p] = (p < P) ? cs[p] : 0;
    // projection through the fast transform of sigma .* u
    if (!row_is_u) {
      float e_, *ep = &e_;
      double sd_;
      tile_u64<C, PE>(a, off, blk, my, ep, &sd_);
    }
    const bool v2 = a.gen_version != 1;
    const uint8_t* ip = a.basis.iperm + (size_t)s * kMaxC;  // pi^-1 (generator version 2)
    {
      double v[C];
      const uint64_t s0 = sw[0], s1 = sw[1];
#pragma unroll
      for (int i = 0; i < C; ++i) {
        // version 2: coordinate i of the permuted vector is sigma_j u_j at j = pi^-1(i)
        const int j = v2 ? (int)ip[i] : i;
        const double u = my[j];
        const uint64_t sg = (j < 64) ? (s0 >> j) : (s1 >> (j - 64));
        v[i] = (sg & 1ull) ? -u : u;
      }
      fwht<C>(v);
#pragma unroll
      for (int j = 0; j < C; ++j) my[j] = v[j];
      row_is_u = false;
    }
    double bv[PB];
#pragma unroll
    for (int p = 0; p < PB; ++p) bv[p] = (p < P) ? my[c[p]] * isq : 0.0;
    // Gram entries
    const double* wd;
    if (v2) {
      // WHT(d o pi^-1) of this tile's (or column block's) weights
      const float* dsrc = PE ? a.d + off : a.d + (int64_t)blk * C;
      double v[C];
#pragma unroll
      for (int i = 0; i < C; ++i) v[i] = (double)dsrc[ip[i]];
      fwht<C>(v);
#pragma unroll
      for (int j = 0; j < C; ++j) my[j] = v[j];
      wd = my;
    } else if constexpr (PE) {
      double v[C];
#pragma unroll
      for (int j0 = 0; j0 < C; j0 += 8) {
        float dj[8];
        load8_f(a.d + off + j0, dj);
#pragma unroll
        for (int k = 0; k < 8; ++k) v[j0 + k] = (double)dj[k];
      }
      fwht<C>(v);
#pragma unroll
      for (int j = 0; j < C; ++j) my[j] = v[j];
      wd = my;
    } else {
      wd = wdb + (int64_t)blk * C;
    }
    int q[PB];
    double al[PB];
    uint16_t bits;
    double L[PB][PB], inv[PB];
    chol64<C, PB>(P, wd, c, eps, L, inv);
    const double gsum = solve_score64<PB>(a, bv, L, inv, eps, qmax, q, al, &bits);
    if (gsum > best_g || (gsum == best_g && s < best_s)) {
      best_g = gsum;
      best_s = s;
      best_bits = bits;
#pragma unroll
      for (int p = 0; p < PB; ++p) { best_q[p] = q[p]; best_al[p] = (float)al[p]; }
    }
  }
  a.seed_out[t] = (uint16_t)best_s;
  a.scale_out[t] = best_bits;
  a.gain_out[t] = best_g;
#pragma unroll
  for (int p = 0; p < PB; ++p) {
    if (p < P) {
      a.code_out[t * P + p] = (int8_t)best_q[p];
      if (a.alpha_out) a.alpha_out[t * P + p] = best_al[p];
    }
  }
}

// Per-column weights, generator version 1, C = 64 (the common case).  Each
// lane keeps its tile in registers (fp64) and transforms it in place; only
// the gather of the P projections out of the transform goes through LDS,
// half a wavefront at a time.  A workgroup thus needs half the LDS of
// k_finalize, and two wavefronts fit per SIMD.  The second kept seed (a
// near tie, rare) reloads the tile.
template <int PB>
__global__ __launch_bounds__(64, 2) void k_finalize_col64(EncodeArgs a) {
  constexpr int C = 64;
  __shared__ double gb[32 * (C + 1)];
  const int lane = threadIdx.x;
  const int nb = (int)(a.cols / C);
  // Workgroups are dealt to the 8 XCDs round-robin by index: give each XCD a
  // contiguous run of work items in column-block-major order (the block's d
  // and weight transform stay in its L2).
  const int64_t nwg = gridDim.x;
  const int64_t xcd = blockIdx.x % 8, qq = nwg / 8, rem = nwg % 8;
  const int64_t w = xcd * qq + (xcd < rem ? xcd : rem) + blockIdx.x / 8;
  const int64_t nrg = (a.rows + 63) / 64;
  const int blk = (int)(w / nrg);
  const int64_t row = (w % nrg) * 64 + lane;
  const float* dcol = a.d + (int64_t)blk * C;
  // the block's d, one coordinate per lane (C = wavefront size), staged by
  // every lane before the rows past the end leave
  __shared__ float dsh[C];
  __shared__ double wdsh[C];  // WHT(d) of the block, for the Gram entries
  dsh[lane] = dcol[lane];
  wdsh[lane] = a.wd64[(int64_t)blk * C + lane];
  // The work item's 64 x 64 residual block r = W - W0 (fp32) through LDS:
  // loaded with 16 lanes per row segment (4 rows per pass), so each cache
  // line is read whole by one instruction, then each lane reads its own row.
  // (Row-per-lane loads of 16 bytes leave each line to 8 or 16 separate
  // instructions, and with two wavefronts per SIMD the lines in flight
  // outgrow the L2 and are fetched again.)  The gather buffer holds the rows.
  float* rsh = reinterpret_cast<float*>(gb);  // [64][C + 1]
  {
    const int64_t row0 = (w % nrg) * 64;
    const int pc = lane & 15;
#pragma unroll
    for (int pass = 0; pass < 16; ++pass) {
      const int rl = 4 * pass + (lane >> 4);
      const int64_t rg = row0 + rl < a.rows ? row0 + rl : a.rows - 1;
      const int64_t o = rg * a.cols + (int64_t)blk * C + 4 * pc;
      float wv[4], w0[4];
      if (a.w_dtype == AWSRC_DTYPE_F32) {
        const float4 x = *reinterpret_cast<const float4*>(static_cast<const float*>(a.W) + o);
        wv[0] = x.x; wv[1] = x.y; wv[2] = x.z; wv[3] = x.w;
      } else {
        const uint2 x = *reinterpret_cast<const uint2*>(static_cast<const uint16_t*>(a.W) + o);
        wv[0] = __uint_as_float(x.x << 16); wv[1] = __uint_as_float(x.x & 0xFFFF0000u);
        wv[2] = __uint_as_float(x.y << 16); wv[3] = __uint_as_float(x.y & 0xFFFF0000u);
      }
      const float4 y = *reinterpret_cast<const float4*>(a.W0 + o);
      w0[0] = y.x; w0[1] = y.y; w0[2] = y.z; w0[3] = y.w;
#pragma unroll
      for (int k = 0; k < 4; ++k) rsh[rl * (C + 1) + 4 * pc + k] = wv[k] - w0[k];
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

  // merge the seed ranges' lists into the best kTop (as in k_finalize)
  float tg[kTop];
  int ts[kTop];
#pragma unroll
  for (int k = 0; k < kTop; ++k) { tg[k] = -INFINITY; ts[k] = 0; }
  for (int sp = 0; sp < a.nsplit; ++sp) {
#pragma unroll
    for (int k = 0; k < kTop; ++k) {
      const int64_t at = (t * a.nsplit + sp) * kTop + k;
      float g = a.top_gain[at];
      int sd = a.top_seed[at];
#pragma unroll
      for (int m = 0; m < kTop; ++m) {
        if (g > tg[m]) {
          const float tgm = tg[m];
          const int tsm = ts[m];
          tg[m] = g; ts[m] = sd;
          g = tgm; sd = tsm;
        }
      }
    }
  }

  // Score seed s: u = d .* r in fp64 (also the tile's weighted energy e32 and
  // sum of d), sigma .* u transformed in place, the P projections gathered
  // through this lane's LDS row (lanes l and l + 32 share a row, so the two
  // halves take turns, ordered by the wavefront barriers), then the solve
  // with the Cholesky factor of the seed's G + eps I.
  auto score = [&](int s, bool first, float* e32, int (&q)[PB], double (&al)[PB], uint16_t* bits) -> double {
    // r: the first seed's from the LDS rows, a second seed's (a rare near
    // tie, after the gather has reused the buffer) loaded directly; then u
    // with the block's d from LDS
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
  int best_s = ts[0];
  double best_g = score(best_s, true, &e32, best_q, best_al, &best_bits);
  // the second kept seed only when its screened gain is close to the best
  const float thr = tg[0] - (1e-4f * fabsf(tg[0]) + 1e-7f * e32);
#pragma unroll
  for (int k = 1; k < kTop; ++k) {
    if (tg[k] >= thr && tg[k] > -INFINITY) {
      int q[PB];
      double al[PB];
      uint16_t bits;
      float e_;
      const double g = score(ts[k], false, &e_, q, al, &bits);
      if (g > best_g || (g == best_g && ts[k] < best_s)) {
        best_g = g;
        best_s = ts[k];
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

// ----------------------------------------------------------------------------
static int pad_p(int P) { return P <= 4 ? 4 : (P <= 8 ? 8 : 16); }

bool encode_supported(int C, int P) {
  return (C == 16 || C == 32 || C == 64 || C == 128) && P >= 1 && P <= kMaxP && P <= C;
}

int factor_pb(int C, int P) { return screen_mfma_supported(C, P, AWSRC_D_PER_COL, 1) ? 8 : pad_p(P); }

template <int C, int PB>
static hipError_t run_factors(const EncodeArgs& a, hipStream_t st) {
  const int nb = (int)(a.cols / C);
  const int n = nb * a.S;
  (void)n;
  if (a.gen_version == 1)
    hipLaunchKernelGGL((k_block_wht64<C>), dim3(nb), dim3(64), 0, st, a.d, nb, a.wd64);
  hipLaunchKernelGGL((k_col_factors<C, PB>), dim3((unsigned)((a.S + 63) / 64), (unsigned)nb), dim3(64), 0, st,
                     a, nb, colfac_stride(PB));
  return hipGetLastError();
}

template <int C, int PB>
static hipError_t run_screen(const EncodeArgs& a, hipStream_t st) {
  const int nb = (int)(a.cols / C);
  const int64_t waves = nb * ((a.rows + 63) / 64);
  if (a.d_mode == AWSRC_D_PER_ELEM && a.gen_version != 1)
    hipLaunchKernelGGL((k_screen_valu<C, PB, true, true>), dim3((unsigned)waves), dim3(64), 0, st, a,
                       colfac_stride(PB));
  else if (a.d_mode == AWSRC_D_PER_ELEM)
    hipLaunchKernelGGL((k_screen_valu<C, PB, true, false>), dim3((unsigned)waves), dim3(64), 0, st, a,
                       colfac_stride(PB));
  else
    hipLaunchKernelGGL((k_screen_valu<C, PB, false, false>), dim3((unsigned)waves), dim3(64), 0, st, a,
                       colfac_stride(PB));
  return hipGetLastError();
}

template <int C, int PB>
static hipError_t run_finalize(const EncodeArgs& a, hipStream_t st) {
  constexpr int NT = (C == 128) ? 32 : 64;
  const int nb = (int)(a.cols / C);
  const int64_t groups = nb * ((a.rows + NT - 1) / NT);
  const size_t lds = (size_t)NT * (C + 1) * sizeof(double);
  if (a.d_mode == AWSRC_D_PER_ELEM) {
    hipLaunchKernelGGL((k_finalize<C, PB, true>), dim3((unsigned)groups), dim3(NT), lds, st, a,
                       (const double*)nullptr);
  } else if (C == 64 && PB <= 8 && a.gen_version == 1) {
    if constexpr (C == 64 && PB <= 8)
      hipLaunchKernelGGL((k_finalize_col64<PB>), dim3((unsigned)groups), dim3(64), 0, st, a);
  } else {
    hipLaunchKernelGGL((k_finalize<C, PB, false>), dim3((unsigned)groups), dim3(NT), lds, st, a,
                       (const double*)a.wd64);
  }
  return hipGetLastError();
}

#define AWSRC_DISPATCH(FN, a, st)                                       \
  do {                                                                  \
    const int pb_ = PBSEL((a).C, (a).P);                                \
    switch ((a).C) {                                                    \
      case 16:                                                          \
        if (pb_ == 4) return FN<16, 4>(a, st);                          \
        if (pb_ == 8) return FN<16, 8>(a, st);                          \
        return FN<16, 16>(a, st);                                       \
      case 32:                                                          \
        if (pb_ == 4) return FN<32, 4>(a, st);                          \
        if (pb_ == 8) return FN<32, 8>(a, st);                          \
        return FN<32, 16>(a, st);                                       \
      case 64:                                                          \
        if (pb_ == 4) return FN<64, 4>(a, st);                          \
        if (pb_ == 8) return FN<64, 8>(a, st);                          \
        return FN<64, 16>(a, st);                                       \
      case 128:                                                         \
        if (pb_ == 4) return FN<128, 4>(a, st);                         \
        if (pb_ == 8) return FN<128, 8>(a, st);                         \
        return FN<128, 16>(a, st);                                      \
      default: return hipErrorInvalidValue;                             \
    }                                                                   \
  } while (0)

#define PBSEL(C_, P_) factor_pb(C_, P_)
hipError_t launch_col_factors(const EncodeArgs& a, hipStream_t st) { AWSRC_DISPATCH(run_factors, a, st); }
hipError_t launch_encode_screen(const EncodeArgs& a, hipStream_t st) {
  if (screen_mfma_supported(a.C, a.P, a.d_mode, a.gen_version)) return launch_encode_screen_mfma(a, a.frag, st);
  AWSRC_DISPATCH(run_screen, a, st);
}
#undef PBSEL
#define PBSEL(C_, P_) pad_p(P_)
hipError_t launch_encode_finalize(const EncodeArgs& a, hipStream_t st) { AWSRC_DISPATCH(run_finalize, a, st); }
#undef PBSEL

}  // namespace awsrc
