// Encoder seed search (Sec. 3.2): for every tile r_t and every seed s, fit the
// activation-weighted ridge least squares of Eq. (3) in the basis B_s of
// Eq. (2), quantize the coefficients with one fp16 scale, and score the
// weighted error reduction of the quantized reconstruction (numerator of
// Eq. (4)); keep the seed with the largest reduction.
//
// Two passes share one set of tables:
//  * screen   - every (tile, seed) in fp32, one lane per tile; the seed loop
//               is uniform across the wavefront, so basis patterns and the
//               per-column factors are scalar loads.  The two best screened
//               seeds of each tile (kTop) are kept.
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
#include "rescore64.h"

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
  uint32_t ts[kTop];  // seed words: seed | kEdge flag
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
    bool edge = false;
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
      const float sc = pow2 ? screen_scale<true>(m, inv_qmax, &isc, &edge) : screen_scale<false>(m, inv_qmax, &isc, &edge);
      g = 0.0f;
      if (sc > 0.0f) {
        float q[PB], t1 = 0.0f, qq = 0.0f;
#pragma unroll
        for (int p = 0; p < PB; ++p) {
          const float x = al[p] * isc;
          q[p] = fminf(fmaxf(rintf(x), -qmax), qmax);
          edge = edge || code_edge(x, qmax);
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
      g = pow2 ? screen_score_ldl<PB, true, 0>(bv, fs, qmax, inv_qmax, &edge)
               : screen_score_ldl<PB, false, 0>(bv, fs, qmax, inv_qmax, &edge);
    }
    // keep the best kTop, earlier (lower) seeds first among equals
    float cg = g;
    uint32_t cs_ = (uint32_t)s | (edge ? kEdge : 0u);
#pragma unroll
    for (int k = 0; k < kTop; ++k) {
      if (cg > tg[k]) {
        const float tgk = tg[k];
        const uint32_t tsk = ts[k];
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
      a.top_seed[t * kTop + k] = ts[k];
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


// The re-score of one tile (row, column block) of the module `a` describes,
// with `my` a private LDS row of C + 1 doubles.
template <int C, int PB, bool PE>
__device__ __forceinline__ void finalize_tile(const EncodeArgs& a, const double* __restrict__ wdb, int64_t row,
                                              int blk, double* my) {
  const int nb = (int)(a.cols / C);
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
  uint32_t ts[kTop];  // seed words: seed | kEdge flag
#pragma unroll
  for (int k = 0; k < kTop; ++k) { tg[k] = -INFINITY; ts[k] = 0; }
  for (int sp = 0; sp < a.nsplit; ++sp) {
#pragma unroll
    for (int k = 0; k < kTop; ++k) {
      const int64_t at = (t * a.nsplit + sp) * kTop + k;
      float g = a.top_gain[at];
      uint32_t sd = a.top_seed[at];
#pragma unroll
      for (int m = 0; m < kTop; ++m) {
        if (g > tg[m]) {
          const float tgm = tg[m];
          const uint32_t tsm = ts[m];
          tg[m] = g; ts[m] = sd;
          g = tgm; sd = tsm;
        }
      }
    }
  }
  const float thr = tg[0] - rescore_window(tg[0], e32, ((ts[0] | ts[1]) & kEdge) != 0);

  double best_g = -INFINITY;
  int best_s = 0x7FFFFFFF;
  int best_q[PB];
  uint16_t best_bits = 0;
  float best_al[PB];
#pragma unroll
  for (int p = 0; p < PB; ++p) { best_q[p] = 0; best_al[p] = 0.f; }

  for (int k = 0; k < kTop; ++k) {
    if (k > 0 && !(tg[k] >= thr && tg[k] > -INFINITY)) continue;
    const int s = list_seed(ts[k]);
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
  finalize_tile<C, PB, PE>(a, wdb, row, blk, my);
}

// Per-column weights, generator version 1, C = 64 (the common case), when
// the screen leaves the re-score to a kernel of its own (seed ranges split
// over wavefronts): one wavefront per (row group of 64, column block) merges
// each tile's lists over the ranges and runs rescore_block64.  Two
// wavefronts fit per SIMD (the general k_finalize keeps a 65-double LDS row
// per lane: one per SIMD).
template <int PB>
__global__ __launch_bounds__(64, 2) void k_finalize_col64(EncodeArgs a) {
  constexpr int C = 64;
  __shared__ __attribute__((aligned(16))) float lds[kRescoreLds];
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
  const int64_t row0 = (w % nrg) * 64;
  const int64_t row = row0 + lane < a.rows ? row0 + lane : a.rows - 1;
  const int64_t t = row * nb + blk;
  // merge the seed ranges' lists into the best kTop: ranges come in seed order
  // and each list is ordered (gain desc, seed asc), so strict comparisons
  // keep the lower seed first among equal gains
  float tg[kTop];
  uint32_t ts[kTop];  // seed words: seed | kEdge flag
#pragma unroll
  for (int k = 0; k < kTop; ++k) { tg[k] = -INFINITY; ts[k] = 0; }
  for (int sp = 0; sp < a.nsplit; ++sp) {
#pragma unroll
    for (int k = 0; k < kTop; ++k) {
      const int64_t at = (t * a.nsplit + sp) * kTop + k;
      float g = a.top_gain[at];
      uint32_t sd = a.top_seed[at];
#pragma unroll
      for (int m = 0; m < kTop; ++m) {
        if (g > tg[m]) {
          const float tgm = tg[m];
          const uint32_t tsm = ts[m];
          tg[m] = g; ts[m] = sd;
          g = tgm; sd = tsm;
        }
      }
    }
  }
  rescore_block64<PB>(a, blk, row0, tg, ts, lds);
}

// Per-column weights, generator version 1, C = 128 (the C = 128 screen's
// lists): one wavefront per (16-row group, column block), four lanes per
// tile.  Lane l works on tile l % 16 and its coordinates 32 (l / 16) .. + 31:
// it forms sigma .* d .* r for them in fp64 and runs the first five butterfly
// stages of the length-128 transform on them in registers; the last two
// stages, which combine the four quarters, are folded into the gathers of
// the P projections (the same additions in the same order as the full
// transform, so the same values).  The Gram entries come from the column
// block's fp64 weight transform, eps from the sum of the block's d in
// coordinate order, and the solve is the per-element re-score's (LDL^T with
// refined reciprocals).  Work items go row group major (the next item is the next column
// block of the same rows, whose outputs share cache lines), in contiguous
// ranges per XCD.
constexpr int kQ128 = 33;                  // doubles per quarter in a gather row (padded)
constexpr int kRow128 = 4 * kQ128 + 1;     // doubles per gather row

__device__ __forceinline__ double tentry128(const double* row, int k) {
  const int kk = k & 31, q = k >> 5;
  const double x0 = row[kk], x1 = row[kQ128 + kk], x2 = row[2 * kQ128 + kk], x3 = row[3 * kQ128 + kk];
  // stage h = 32, then h = 64
  const double y0 = x0 + x1, y1 = x0 - x1, y2 = x2 + x3, y3 = x2 - x3;
  return q == 0 ? y0 + y2 : q == 1 ? y1 + y3 : q == 2 ? y0 - y2 : y1 - y3;
}

template <int PB>
__global__ __launch_bounds__(64, 2) void k_finalize_col128(EncodeArgs a) {
  constexpr int C = 128, NTL = 16, H = 32;
  __shared__ __attribute__((aligned(16))) double gsh[NTL * kRow128];  // r staging (fp32), then gather rows
  __shared__ float dsh[C];
  __shared__ double wdsh[C];
  const int lane = threadIdx.x;
  const int tl = lane & (NTL - 1), qd = lane >> 4;
  const int nb = (int)(a.cols / C);
  const int64_t w = xcd_item(blockIdx.x, gridDim.x);
  const int blk = (int)(w % nb);
  const int64_t row0 = (w / nb) * NTL;
  const int64_t row = row0 + tl;
  const bool valid = row < a.rows;
  for (int j = lane; j < C; j += 64) {
    dsh[j] = a.d[(int64_t)blk * C + j];
    wdsh[j] = a.wd64[(int64_t)blk * C + j];
  }
  // the 16 x 128 residual block, 32 lanes per row (4 coordinates each), two
  // rows per pass, every load issued before any is used; rows past the end
  // repeat the last row
  float* rsh = reinterpret_cast<float*>(gsh);
  {
    const int pc = lane & 31;
    constexpr int NP = NTL / 2;
    int64_t o[NP];
#pragma unroll
    for (int pass = 0; pass < NP; ++pass) {
      const int rl = 2 * pass + (lane >> 5);
      const int64_t rg = row0 + rl < a.rows ? row0 + rl : a.rows - 1;
      o[pass] = rg * a.cols + (int64_t)blk * C + 4 * pc;
    }
    float rv[NP][4];
    load_residual4<NP>(a.W, a.w_dtype, a.W0, o, rv);
#pragma unroll
    for (int pass = 0; pass < NP; ++pass) {
      float* rp = rsh + (2 * pass + (lane >> 5)) * (C + 1) + 4 * pc;
      rp[0] = rv[pass][0]; rp[1] = rv[pass][1]; rp[2] = rv[pass][2]; rp[3] = rv[pass][3];
    }
  }
  __syncthreads();
  float rr[H];
#pragma unroll
  for (int j = 0; j < H; ++j) rr[j] = rsh[tl * (C + 1) + H * qd + j];
  // the tile's weighted energy (each lane's quarter, then the quarters
  // added), for the re-score window; eps from the block's d summed in
  // coordinate order
  float e32;
  {
    float eq = 0.0f;
#pragma unroll
    for (int j = 0; j < H; ++j) {
      const float dj = dsh[H * qd + j];
      eq = fmaf(dj * rr[j], rr[j], eq);
    }
    eq += __shfl_xor(eq, 16, 64);
    e32 = eq + __shfl_xor(eq, 32, 64);
  }
  double sumd = 0.0;  // in order, one value at a time (left unrolled, all 128 are held in registers)
#pragma unroll 1
  for (int j = 0; j < C; ++j) sumd += (double)dsh[j];
  const double eps = a.lambda * (sumd / C);
  const int P = a.P;
  const double isq = 1.0 / sqrt((double)C);
  const int qmax = (1 << (a.b - 1)) - 1;
  const int64_t t = (valid ? row : a.rows - 1) * nb + blk;

  // merge the seed ranges' lists into the best kTop (as finalize_tile)
  float tg[kTop];
  uint32_t ts[kTop];
#pragma unroll
  for (int k = 0; k < kTop; ++k) { tg[k] = -INFINITY; ts[k] = 0; }
  for (int sp = 0; sp < a.nsplit; ++sp) {
#pragma unroll
    for (int k = 0; k < kTop; ++k) {
      const int64_t at = (t * a.nsplit + sp) * kTop + k;
      float g = a.top_gain[at];
      uint32_t sd = a.top_seed[at];
#pragma unroll
      for (int m = 0; m < kTop; ++m) {
        if (g > tg[m]) {
          const float tgm = tg[m];
          const uint32_t tsm = ts[m];
          tg[m] = g; ts[m] = sd;
          g = tgm; sd = tsm;
        }
      }
    }
  }
  // the second kept seed is re-scored when its screened gain lies within the
  // window of the best; lanes of quarter 0 score the best seed, lanes of
  // quarter 1 the second one where needed (else the best again)
  const float thr = tg[0] - rescore_window(tg[0], e32, ((ts[0] | ts[1]) & kEdge) != 0);
  const bool need = valid && tg[1] >= thr && tg[1] > -INFINITY;
  const bool two = __ballot(need) != 0;
  const int s0r = list_seed(ts[0]), s1r = list_seed(ts[1]);
  const int s0 = s0r < a.S ? s0r : 0, s1 = s1r < a.S ? s1r : 0;
  const bool mine2 = qd == 1 && need;
  const int s_me = mine2 ? s1 : s0;
  int c[PB];
#pragma unroll
  for (int p = 0; p < PB; ++p) c[p] = (p < P) ? a.basis.col[(size_t)s_me * kMaxP + p] : 0;
  double* grow = gsh + tl * kRow128;
  double bv[PB];
#pragma unroll
  for (int p = 0; p < PB; ++p) bv[p] = 0.0;
#pragma unroll
  for (int pass = 0; pass < 2; ++pass) {
    if (pass == 1 && !two) break;
    const int sp_ = pass ? s1 : s0;
    const uint32_t sw = (uint32_t)(a.basis.sign[(size_t)sp_ * 2 + (qd >> 1)] >> (H * (qd & 1)));
    double v[H];
#pragma unroll
    for (int j = 0; j < H; ++j) {
      const double u = (double)dsh[H * qd + j] * (double)rr[j];
      v[j] = ((sw >> j) & 1u) ? -u : u;
    }
    fwht<H>(v);
    __syncthreads();  // the staging rows (pass 0) or the previous gathers are done
#pragma unroll
    for (int j = 0; j < H; ++j) grow[kQ128 * qd + j] = v[j];
    __syncthreads();
    // quarter 0 gathers from the best seed's pass, quarter 1 from the second
    // seed's pass where its tile needs it, else from the best seed's
    if (qd < 2 && (pass == 1) == mine2) {
#pragma unroll
      for (int p = 0; p < PB; ++p) bv[p] = (p < P) ? tentry128(grow, c[p]) * isq : 0.0;
    }
  }
  // quarters 0 and 1 solve (the best seed, and the second or the best again)
  double gk = -INFINITY;
  int q[PB];
  double al[PB];
  uint16_t bits = 0;
  if (qd < 2) {
    double g[PB * (PB + 1) / 2];
#pragma unroll
    for (int p = 0; p < PB; ++p)
#pragma unroll
      for (int r = 0; r <= p; ++r) g[p * (p + 1) / 2 + r] = wdsh[c[p] ^ c[r]];
    double L[PB * (PB - 1) / 2], e[PB], inv[PB];
    ldl64<C, PB>(P, g, eps, L, e, inv);
    gk = solve_score_ldl<PB>(a, bv, L, e, inv, eps, qmax, q, al, &bits);
  }
  // the better of the two results (ties: the lower seed) is written by the
  // lane that holds it
  const double go = __shfl_xor(gk, 16, 64);
  const bool second_wins =
      need && (qd == 1 ? (gk > go || (gk == go && s1 < s0)) : (go > gk || (go == gk && s1 < s0)));
  if (valid && qd < 2 && (qd == 1) == second_wins) {
    a.seed_out[t] = (uint16_t)s_me;
    a.scale_out[t] = bits;
    a.gain_out[t] = gk;
#pragma unroll
    for (int p = 0; p < PB; ++p) {
      if (p < P) {
        a.code_out[t * P + p] = (int8_t)q[p];
        if (a.alpha_out) a.alpha_out[t * P + p] = (float)al[p];
      }
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
  } else if (C == 128 && PB == 8 && a.gen_version == 1) {
    if constexpr (C == 128 && PB == 8) {
      const int64_t items = nb * ((a.rows + 15) / 16);
      hipLaunchKernelGGL((k_finalize_col128<PB>), dim3((unsigned)items), dim3(64), 0, st, a);
    }
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
