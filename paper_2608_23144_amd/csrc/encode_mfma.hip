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

namespace awsrc {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

namespace {

__device__ __forceinline__ float load_w_any2(const void* W, int dt, int64_t i) {
  if (dt == AWSRC_DTYPE_F32) return static_cast<const float*>(W)[i];
  return __uint_as_float((uint32_t)static_cast<const uint16_t*>(W)[i] << 16);
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// Exact three-way bf16 split of eight fp32 values, packed two per dword.
__device__ __forceinline__ void split3(const float (&u)[8], u32x4& hi, u32x4& mid, u32x4& lo) {
  uint32_t h[8], m[8], l[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const uint32_t ub = __float_as_uint(u[e]);
    h[e] = ub & 0xFFFF0000u;
    const float r1 = u[e] - __uint_as_float(h[e]);
    m[e] = __float_as_uint(r1) & 0xFFFF0000u;
    const float r2 = r1 - __uint_as_float(m[e]);
    l[e] = __float_as_uint(r2) & 0xFFFF0000u;
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    hi[i] = (h[2 * i] >> 16) | h[2 * i + 1];
    mid[i] = (m[2 * i] >> 16) | m[2 * i + 1];
    lo[i] = (l[2 * i] >> 16) | l[2 * i + 1];
  }
}

}  // namespace

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
// Screen: one wavefront (one workgroup) = 64 consecutive rows of one column
// block and one range of seed pairs; lane = tile during the per-candidate
// stage.  Seed ranges are used only when a module has too few row groups to
// fill the machine (each range costs its own tile loads and top list).
template <bool PE, bool POW2>
__global__ __launch_bounds__(64, 2) void k_screen_mfma64(EncodeArgs a, const u32x4* __restrict__ frag,
                                                         int stride) {
  constexpr int C = 64;
  constexpr int PB = 8;
  constexpr int TS = 12;  // LDS stride (floats) of one tile's coefficients
  __shared__ __attribute__((aligned(16))) float tb[2 * 64 * TS];
  __shared__ float wdl[PE ? 64 * (C + 1) : 1];
  const int lane = threadIdx.x;
  const int nbk_cols = (int)(a.cols / C);
  const int nsplit = a.nsplit;
  // Workgroups are dealt to the 8 XCDs round-robin by index.  Give each XCD a
  // contiguous run of work items in column-block-major order, so that the
  // row groups of a column block share one L2 for their factor reads.
  const int64_t nwg = gridDim.x;
  const int64_t xcd = blockIdx.x % 8, q = nwg / 8, rem = nwg % 8;
  const int64_t w = xcd * q + (xcd < rem ? xcd : rem) + blockIdx.x / 8;
  const int nrg = (int)((a.rows + 63) / 64);
  const int split = (int)(w % nsplit);
  const int64_t rest = w / nsplit;
  const int blk = (int)(rest / nrg);
  const int64_t row0 = (rest % nrg) * 64;
  const int n_pairs_all = (a.S + 1) / 2;
  const int pp = (n_pairs_all + nsplit - 1) / nsplit;
  const int pair0 = split * pp;
  const int pair1 = pair0 + pp < n_pairs_all ? pair0 + pp : n_pairs_all;
  const int n = lane & 15, g = lane >> 4;

  // ---- u = d .* r fragments for the 4 groups of 16 tiles, split in three bf16 parts
  u32x4 uh[4][2], um[4][2], ul[4][2];
#pragma unroll
  for (int nb = 0; nb < 4; ++nb) {
    const int64_t row = row0 + 16 * nb + n;
    const bool valid = row < a.rows;
    const int64_t rr = valid ? row : a.rows - 1;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const int jc = 32 * ks + 8 * g;
      const int64_t base = rr * a.cols + (int64_t)blk * C + jc;
      float u[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float r = load_w_any2(a.W, a.w_dtype, base + e) - a.W0[base + e];
        const float dj = PE ? a.d[base + e] : a.d[(int64_t)blk * C + jc + e];
        u[e] = valid ? dj * r : 0.0f;
      }
      split3(u, uh[nb][ks], um[nb][ks], ul[nb][ks]);
    }
  }
  const int64_t my_row = row0 + lane;
  const bool my_valid = my_row < a.rows;
  const int64_t my_off = (my_valid ? my_row : a.rows - 1) * a.cols + (int64_t)blk * C;
  const int P = a.P;
  if constexpr (PE) {
    // WHT of this lane's tile weights, for the Gram gathers G_pq = WHT(d)[c_p ^ c_q] / C
    float wd[C];
#pragma unroll
    for (int j = 0; j < C; ++j) wd[j] = a.d[my_off + j];
#pragma unroll
    for (int h = 1; h < C; h <<= 1)
#pragma unroll
      for (int i = 0; i < C; i += 2 * h)
#pragma unroll
        for (int k = i; k < i + h; ++k) {
          const float x = wd[k], y = wd[k + h];
          wd[k] = x + y;
          wd[k + h] = x - y;
        }
    // stored divided by C, so the gathers are the Gram entries themselves
#pragma unroll
    for (int j = 0; j < C; ++j) wdl[lane * (C + 1) + j] = wd[j] * (1.0f / C);
  }
  const float qmax = (float)((1 << (a.b - 1)) - 1);
  const float inv_qmax = 1.0f / qmax;
  const float lam = (float)a.lambda;
  float tg0 = -INFINITY, tg1 = -INFINITY;
  int ts0 = 0, ts1 = 0;

  // Post-processing runs in "raw" units: b is left unscaled by 1/sqrt(C) = 1/8,
  // so alpha, the scale and the gain come out 8, 8 and 64 times larger; the
  // codes and the seed order are unchanged (scaling by a power of two commutes
  // with the roundings), and the kept gains are rescaled once at the end.
  //
  // Software pipeline: while the vector ALUs post-process seed pair k, the
  // matrix cores compute the projections of pair k+1 (the fragment table is
  // padded with zero pairs, so the last iterations need no special case).
  const u32x4* fp = frag + (size_t)pair0 * 128 + lane;
  auto project = [&](const u32x4& F0, const u32x4& F1, f32x4 (&acc)[4]) {
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
  };
  // rows 4g..4g+3 of the product = (seed g/2, columns 4(g&1)..+3) of tiles 16nb + n
  auto stash = [&](const f32x4 (&acc)[4]) {
#pragma unroll
    for (int nb = 0; nb < 4; ++nb)
      *reinterpret_cast<f32x4*>(&tb[((g >> 1) * 64 + 16 * nb + n) * TS + 4 * (g & 1)]) = acc[nb];
  };
  {
    f32x4 acc[4];
    project(fp[0], fp[64], acc);
    stash(acc);
  }
  u32x4 F0 = fp[128], F1 = fp[192];
  // per-column factors rotate through two register sets: the first seed's of
  // the next pair load while the second seed of this pair is scored, and the
  // second seed's load while the first is scored, hiding the load latency
  constexpr int NF = PB * (PB - 1) / 2 + 2 * PB;
  typedef const __attribute__((address_space(4))) float* cfp;
  auto fac_ptr = [&](int s) -> cfp {
    const int sc_ = s < a.S ? s : a.S - 1;
    return (cfp)(a.colfac + ((size_t)blk * a.S + sc_) * stride);
  };
  float fA[PE ? 1 : NF], fB[PE ? 1 : NF];
  if constexpr (!PE) {
    const cfp f0 = fac_ptr(2 * pair0);
#pragma unroll
    for (int i = 0; i < NF; ++i) fA[i] = f0[i];
  }
  for (int pair = pair0; pair < pair1; ++pair) {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    float bk[2][PB];
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const f32x4 b0 = *reinterpret_cast<const f32x4*>(&tb[(k * 64 + lane) * TS]);
      const f32x4 b1 = *reinterpret_cast<const f32x4*>(&tb[(k * 64 + lane) * TS + 4]);
      bk[k][0] = b0[0]; bk[k][1] = b0[1]; bk[k][2] = b0[2]; bk[k][3] = b0[3];
      bk[k][4] = b1[0]; bk[k][5] = b1[1]; bk[k][6] = b1[2]; bk[k][7] = b1[3];
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    // projections of the next pair (zero rows past the last seed) and the prefetch after it
    f32x4 accN[4];
    project(F0, F1, accN);
    F0 = fp[(size_t)(pair - pair0 + 2) * 128];
    F1 = fp[(size_t)(pair - pair0 + 2) * 128 + 64];
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const int s = 2 * pair + k;
      float gsc;
      if constexpr (PE) {
        // this tile's G + eps I = L diag(e) L^T from the Gram gathers, row by
        // row (E = L diag(e) kept for the current row only), in the layout of
        // the per-column table so the same score routine applies
        constexpr int NF = PB * (PB - 1) / 2 + 2 * PB;
        constexpr int LS = PB * (PB - 1) / 2;
        float f[NF];
        const int sc_ = s < a.S ? s : a.S - 1;
        // the seed's columns: two scalar dword loads (uniform across the wavefront)
        const __attribute__((address_space(4))) uint32_t* cw =
            (const __attribute__((address_space(4))) uint32_t*)(a.basis.col + (size_t)sc_ * kMaxP);
        const uint32_t cw0 = cw[0], cw1 = cw[1];
        int c[PB];
#pragma unroll
        for (int p = 0; p < PB; ++p) c[p] = (p < P) ? (int)(((p < 4 ? cw0 : cw1) >> (8 * (p & 3))) & 0xFFu) : 0;
        const float* wrow = &wdl[lane * (C + 1)];
        const float eps = lam * wrow[0];
#pragma unroll
        for (int p = 0; p < PB; ++p) {
          float E[PB];
#pragma unroll
          for (int q = 0; q < p; ++q) {
            float t = (p < P && q < P) ? wrow[c[p] ^ c[q]] : 0.0f;
#pragma unroll
            for (int kk = 0; kk < q; ++kk) t = fmaf(-E[kk], f[ltri(q, kk)], t);
            E[q] = t;
            f[ltri(p, q)] = t * f[LS + q];
          }
          float t = (p < P) ? wrow[0] + eps : 1.0f;
#pragma unroll
          for (int kk = 0; kk < p; ++kk) t = fmaf(-E[kk], f[ltri(p, kk)], t);
          t = fmaxf(t, 1e-30f);
          f[LS + PB + p] = t;
          f[LS + p] = __builtin_amdgcn_rcpf(t);
        }
        gsc = screen_score_ldl<PB, POW2>(bk[k], f, qmax, inv_qmax);
      } else {
        // uniform across the wavefront: scalar loads through the constant address space
        if (k == 0) {
          const cfp fb = fac_ptr(s + 1);
#pragma unroll
          for (int i = 0; i < NF; ++i) fB[i] = fb[i];
          gsc = screen_score_ldl<PB, POW2>(bk[0], fA, qmax, inv_qmax);
        } else {
          const cfp fa = fac_ptr(s + 1);
#pragma unroll
          for (int i = 0; i < NF; ++i) fA[i] = fa[i];
          gsc = screen_score_ldl<PB, POW2>(bk[1], fB, qmax, inv_qmax);
        }
      }
      gsc = s < a.S ? gsc : -INFINITY;
      // branch-free insertion into the top two (earlier seeds first among equals)
      const bool c0 = gsc > tg0, c1 = gsc > tg1;
      tg1 = c0 ? tg0 : (c1 ? gsc : tg1);
      ts1 = c0 ? ts0 : (c1 ? s : ts1);
      tg0 = c0 ? gsc : tg0;
      ts0 = c0 ? s : ts0;
    }
    // interleave the 24 matrix-core instructions with the vector work above
#pragma unroll
    for (int i = 0; i < 24; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x002, 12, 0);
    }
    stash(accN);
  }
  if (my_valid) {
    const int64_t at = ((my_row * nbk_cols + blk) * nsplit + split) * kTop;
    a.top_gain[at + 0] = tg0 * (1.0f / 64.0f);  // back to gain units
    a.top_gain[at + 1] = tg1 * (1.0f / 64.0f);
    a.top_seed[at + 0] = (uint16_t)ts0;
    a.top_seed[at + 1] = (uint16_t)ts1;
  }
}

// ----------------------------------------------------------------------------
// C = 128, per-column weights.  The u fragments of a 128-coordinate tile take
// twice the registers, so a wavefront holds 32 consecutive rows of one column
// block (2 groups of 16 tiles x 4 K steps x 3 bf16 parts) and gives the two
// seeds of a pair to its two lane halves: lane = (seed of the pair, tile).
// The seed is then uniform per half only, so each lane reads its seed's
// per-column factors with vector loads (two addresses per wavefront).  b is
// scaled by 1/sqrt(128) before scoring (not a power of two, so raw units
// would round the fp16 scale differently); each half keeps its own top two,
// merged at the end.  (Written for any C that is a multiple of 32; at C = 64
// it measured slower than k_screen_mfma64, which is used there.)
template <int C, bool POW2>
__global__ __launch_bounds__(64, 2) void k_screen_mfma_halves(EncodeArgs a, const u32x4* __restrict__ frag,
                                                              int stride) {
  constexpr int PB = 8;
  constexpr int NKS = C / 32;
  constexpr int TS = 12;  // LDS stride (floats) of one lane's coefficients
  constexpr int NF = PB * (PB - 1) / 2 + 2 * PB;
  __shared__ __attribute__((aligned(16))) float tb[64 * TS];
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

  u32x4 uh[2][NKS], um[2][NKS], ul[2][NKS];
#pragma unroll
  for (int nb = 0; nb < 2; ++nb) {
    const int64_t row = row0 + 16 * nb + n;
    const bool valid = row < a.rows;
    const int64_t rr = valid ? row : a.rows - 1;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      const int jc = 32 * ks + 8 * g;
      const int64_t base = rr * a.cols + (int64_t)blk * C + jc;
      float u[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float r = load_w_any2(a.W, a.w_dtype, base + e) - a.W0[base + e];
        u[e] = valid ? a.d[(int64_t)blk * C + jc + e] * r : 0.0f;
      }
      split3(u, uh[nb][ks], um[nb][ks], ul[nb][ks]);
    }
  }
  const int half = lane >> 5;
  const int64_t my_row = row0 + (lane & 31);
  const bool my_valid = my_row < a.rows;
  const float qmax = (float)((1 << (a.b - 1)) - 1);
  const float inv_qmax = 1.0f / qmax;
  constexpr float isq = C == 64 ? 0.125f : 0.08838834764831845f;  // 1/sqrt(C)
  float tg0 = -INFINITY, tg1 = -INFINITY;
  int ts0 = 0, ts1 = 0;

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
  for (int pair = pair0; pair < pair1; ++pair) {
    const int s = 2 * pair + half;
    const int sc_ = s < a.S ? s : a.S - 1;
    const f32x4* fv = reinterpret_cast<const f32x4*>(a.colfac + ((size_t)blk * a.S + sc_) * stride);
    float f[NF];
#pragma unroll
    for (int i = 0; i < NF / 4; ++i) {
      const f32x4 v = fv[i];
      f[4 * i] = v[0]; f[4 * i + 1] = v[1]; f[4 * i + 2] = v[2]; f[4 * i + 3] = v[3];
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    float bv[PB];
    {
      const f32x4 b0 = *reinterpret_cast<const f32x4*>(&tb[lane * TS]);
      const f32x4 b1 = *reinterpret_cast<const f32x4*>(&tb[lane * TS + 4]);
      bv[0] = b0[0] * isq; bv[1] = b0[1] * isq; bv[2] = b0[2] * isq; bv[3] = b0[3] * isq;
      bv[4] = b1[0] * isq; bv[5] = b1[1] * isq; bv[6] = b1[2] * isq; bv[7] = b1[3] * isq;
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    f32x4 accN[2];
    project(F, accN);
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) F[ks] = fp[(size_t)(pair - pair0 + 2) * (NKS * 64) + ks * 64];
    float gsc = screen_score_ldl<PB, POW2>(bv, f, qmax, inv_qmax);
    gsc = s < a.S ? gsc : -INFINITY;
    // this lane's seeds increase, so strict comparisons keep the lower seed among equals
    const bool c0 = gsc > tg0, c1 = gsc > tg1;
    tg1 = c0 ? tg0 : (c1 ? gsc : tg1);
    ts1 = c0 ? ts0 : (c1 ? s : ts1);
    tg0 = c0 ? gsc : tg0;
    ts0 = c0 ? s : ts0;
#pragma unroll
    for (int i = 0; i < 24; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x002, 6, 0);
    }
    stash(accN);
  }
  // merge the two halves' lists of each tile: (gain desc, seed asc)
  const float og0 = __shfl(tg0, lane + 32, 64), og1 = __shfl(tg1, lane + 32, 64);
  const int os0 = __shfl(ts0, lane + 32, 64), os1 = __shfl(ts1, lane + 32, 64);
  if (half == 0 && my_valid) {
    auto better = [](float ga, int sa, float gb, int sb) { return ga > gb || (ga == gb && sa < sb); };
    float r0, r1;
    int q0, q1;
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
    a.top_seed[at + 0] = (uint16_t)q0;
    a.top_seed[at + 1] = (uint16_t)q1;
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
  if (a.d_mode == AWSRC_D_PER_ELEM)
    hipLaunchKernelGGL((k_screen_mfma64<true, POW2>), dim3((unsigned)wgs), dim3(64), 0, st, a, fr, colfac_stride(8));
  else
    hipLaunchKernelGGL((k_screen_mfma64<false, POW2>), dim3((unsigned)wgs), dim3(64), 0, st, a, fr, colfac_stride(8));
  return hipGetLastError();
}

hipError_t launch_encode_screen_mfma(const EncodeArgs& a, void* frag, hipStream_t st) {
  const int64_t n = (int64_t)((a.S + 1) / 2 + 2) * (a.C / 32) * 64;
  hipLaunchKernelGGL(k_mfma_frags, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, a.basis, a.C, a.P, a.S,
                     static_cast<u32x4*>(frag));
  if (a.scale_fmt == AWSRC_SCALE_POW2) return screen_mfma_fmt<true>(a, frag, st);
  return screen_mfma_fmt<false>(a, frag, st);
}

}  // namespace awsrc
