// Decoder (Sec. 3.2): every record regenerates its basis B_s and adds
// B_s (scale * q) onto its tile of W0; tiles without a record are untouched.
//
// validate - one thread per record: field ranges, finite non-negative scale,
//            and a bitmap over tiles that catches a tile appearing twice
//            (records of a valid stream touch disjoint tiles, which is what
//            lets the apply pass run without atomics or ordering).
// validate also writes each record in a decoded form (tile within its
//            module, module, seed, scale, codes and their sum);
// apply    - C/8 lanes per record, eight consecutive weights per lane; each
//            weight gets rhat_j = (1/sqrt(C)) sum_p (+-1) scale*q_p with the
//            signs of row j of B_s read from the transposed sign table.
#include "awsrc_internal.h"

namespace awsrc {

constexpr int kLdsModules = 256;  // module tables up to this size are staged in LDS

struct Rec {
  uint64_t idx;
  uint32_t seed;
  int32_t q[kMaxP];
  uint32_t scale;
};

__device__ __forceinline__ uint64_t get_bits(const uint64_t (&w)[3], int& pos, int nbits) {
  if (nbits <= 0) return 0;
  const int o = pos & 63, k = pos >> 6;
  uint64_t v = w[k] >> o;
  if (o + nbits > 64) v |= w[k + 1] << (64 - o);
  pos += nbits;
  return nbits == 64 ? v : (v & ((1ull << nbits) - 1ull));
}

// Record i of the stream, read with aligned 4-byte loads.  The record area
// starts h = 40 + 8n bytes into an 8-byte aligned stream, so it is 4-byte
// aligned.  A record of at most 32 + 16 + 16*8 + 16 = 192 bits (24 bytes)
// spans at most 7 words from its first word; records whose 7 words all lie
// in the record area load them unconditionally (independent loads in flight
// together), the last few records take a guarded byte-wise path.
__device__ __forceinline__ Rec parse(const DecodeArgs& a, int64_t i) {
  const int64_t o = i * a.L_rec;
  const int64_t total = a.K * a.L_rec;
  const int64_t d0 = o >> 2;
  const int sh = (int)(o & 3) * 8;
  const uint32_t* r32 = reinterpret_cast<const uint32_t*>(a.recs);
  uint32_t wd[7];
  if (d0 + 7 <= (total >> 2)) {
#pragma unroll
    for (int k = 0; k < 7; ++k) wd[k] = r32[d0 + k];
  } else {
#pragma unroll
    for (int k = 0; k < 7; ++k) {
      uint32_t v = 0;
      for (int b = 0; b < 4; ++b) {
        const int64_t at = (d0 + k) * 4 + b;
        if (at < o + a.L_rec && at < total) v |= (uint32_t)a.recs[at] << (8 * b);
      }
      wd[k] = v;
    }
  }
  uint64_t w[3];
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    const uint64_t lo = (uint64_t)wd[2 * k] | ((uint64_t)wd[2 * k + 1] << 32);
    const uint64_t hi = (uint64_t)wd[2 * k + 2];
    w[k] = sh ? ((lo >> sh) | (hi << (64 - sh))) : lo;
  }
  // bits beyond the record are not used: every field lies within L_rec bytes
  Rec out;
  int pos = 0;
  out.idx = get_bits(w, pos, a.idx_bits);
  out.seed = (uint32_t)get_bits(w, pos, a.seed_bits);
  for (int p = 0; p < a.P; ++p) {
    int64_t c = (int64_t)get_bits(w, pos, a.b);
    if (c >> (a.b - 1)) c -= (int64_t)1 << a.b;
    out.q[p] = (int32_t)c;
  }
  out.scale = (uint32_t)get_bits(w, pos, a.scale_fmt == AWSRC_SCALE_POW2 ? 8 : 16);
  return out;
}

__global__ void k_fill_u32(uint32_t* p, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = 0u;
}

__global__ void k_decode_validate(DecodeArgs a) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= a.K) return;
  const Rec r = parse(a, i);
  const int qmax = (1 << (a.b - 1)) - 1;
  bool bad = r.idx >= a.T_total || r.seed >= (uint32_t)a.S;
  for (int p = 0; p < a.P; ++p) bad |= r.q[p] < -qmax || r.q[p] > qmax;
  // fp16 scale: negative, inf or NaN; every 8-bit exponent is valid
  if (a.scale_fmt != AWSRC_SCALE_POW2) bad |= (r.scale & 0x8000u) != 0 || (r.scale & 0x7C00u) == 0x7C00u;
  if (!bad) {
    const uint32_t bit = 1u << (r.idx & 31);
    const uint32_t old = atomicOr(&a.bitmap[r.idx >> 5], bit);
    bad = (old & bit) != 0;
    a.tmap[r.idx] = (uint32_t)i;
  }
  if (bad) atomicAdd(a.errors, 1ull);
  // decoded form for the apply pass (only used once the whole stream is valid)
  int lo = 0, hi = a.n_modules - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (a.mod_tile_off[mid] <= r.idx) lo = mid; else hi = mid - 1;
  }
  uint32_t qw[4] = {0u, 0u, 0u, 0u};
  int32_t tot = 0;
  for (int p = 0; p < a.P; ++p) {
    qw[p >> 2] |= ((uint32_t)r.q[p] & 0xFFu) << (8 * (p & 3));
    tot += r.q[p];
  }
  a.dec[2 * i] = make_uint4((uint32_t)(r.idx - a.mod_tile_off[lo]), (uint32_t)lo, r.seed | (r.scale << 16),
                            (uint32_t)tot);
  a.dec[2 * i + 1] = make_uint4(qw[0], qw[1], qw[2], qw[3]);
}

// C/8 lanes per record, eight consecutive weights per lane.  With integer
// codes, C * rhat_j / sqrt(C) = scale * sum_p sign_jp q_p is scale times an
// exact integer: sum_p q_p minus twice the codes at the negative entries of
// row j, the latter one int8 dot product per four codes against a 0/1 byte
// mask spread from the row's sign bits.  Blocks loop over record groups so
// that the table of W0 pointers is staged in LDS once per block.
template <int C, typename TW, int G>
__global__ __launch_bounds__(256) void k_decode_apply(DecodeArgs a) {
  constexpr int LPR = C / 8;           // lanes per record
  constexpr int RPB = 256 / LPR;       // records per block per iteration
  __shared__ void* s_ptr[kLdsModules];
  const bool lds_tab = a.n_modules <= kLdsModules;
  if (lds_tab)
    for (int m = threadIdx.x; m < a.n_modules; m += 256) s_ptr[m] = a.mod_ptr[m];
  __syncthreads();
  void* const* mptr = lds_tab ? s_ptr : a.mod_ptr;
  constexpr float isq = (C == 16) ? 0.25f : (C == 32) ? 0.17677669529663688f
                      : (C == 64) ? 0.125f : 0.08838834764831845f;
  const int sub = threadIdx.x % LPR;
  for (int64_t i = (int64_t)blockIdx.x * RPB + threadIdx.x / LPR; i < a.K; i += (int64_t)gridDim.x * RPB) {
    const uint4 e0 = a.dec[2 * i];
    const uint4 e1 = a.dec[2 * i + 1];
    const uint32_t q4[4] = {e1.x, e1.y, e1.z, e1.w};
    // signs of rows 8*sub .. 8*sub+7 of B_s, one u16 of P bits per row
    const uint4 tsv = *reinterpret_cast<const uint4*>(a.basis.tsign + (size_t)(e0.z & 0xFFFFu) * kMaxC + sub * 8);
    const uint32_t tw[4] = {tsv.x, tsv.y, tsv.z, tsv.w};
    const uint32_t sfield = e0.z >> 16;
    const float scl = a.scale_fmt == AWSRC_SCALE_POW2 ? ldexpf(isq, (int)sfield - 128)
                                                      : __half2float(__ushort_as_half((uint16_t)sfield)) * isq;
    const int32_t tot = (int32_t)e0.w;
    float add[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const uint32_t ts = (tw[e >> 1] >> (16 * (e & 1))) & 0xFFFFu;
      int32_t neg = 0;
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const uint32_t mask = (((ts >> (4 * g)) & 0xFu) * 0x204081u) & 0x01010101u;
        neg = __builtin_amdgcn_sdot4((int)mask, (int)q4[g], neg, false);
      }
      add[e] = (float)(tot - 2 * neg) * scl;
    }
    TW* W0 = static_cast<TW*>(mptr[e0.y]);
    const int64_t base = (int64_t)e0.x * C + sub * 8;
    if constexpr (sizeof(TW) == 4) {
      float4* q = reinterpret_cast<float4*>(W0 + base);
      float4 v0 = q[0], v1 = q[1];
      v0.x += add[0]; v0.y += add[1]; v0.z += add[2]; v0.w += add[3];
      v1.x += add[4]; v1.y += add[5]; v1.z += add[6]; v1.w += add[7];
      q[0] = v0;
      q[1] = v1;
    } else {
      uint4* q = reinterpret_cast<uint4*>(W0 + base);
      const uint4 v = *q;
      const uint32_t in[4] = {v.x, v.y, v.z, v.w};
      uint32_t o[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        uint32_t h2 = 0;
#pragma unroll
        for (int e = 0; e < 2; ++e) {
          const uint32_t bits = e ? (in[k] & 0xFFFF0000u) : (in[k] << 16);
          uint32_t u = __float_as_uint(__uint_as_float(bits) + add[2 * k + e]);
          u += 0x7FFFu + ((u >> 16) & 1u);  // round to nearest even (finite values)
          h2 |= (u >> 16) << (16 * e);
        }
        o[k] = h2;
      }
      *q = make_uint4(o[0], o[1], o[2], o[3]);
    }
  }
}

// ---------------------------------------------------------------- dense bf16 reconstruction
// One streaming pass over every weight of every module.  Lanes own 16
// consecutive weights: 8 bytes of codes in, 32 bytes of bf16 out, W0 =
// f32(q - z) * s recomputed from the backbone.  A lane whose tile has a record
// (bit set in the validation bitmap) finds it through the tile -> record map
// and adds its 16 corrections before the single rounding to bf16, so record
// tiles cost no extra pass over the backbone or the output.

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t bf16_pair(float lo, float hi) {
  const f32x2_t v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));  // nearest even
}

// Corrections of 16 consecutive coordinates (rows sub*16 .. sub*16+15 of
// B_s) of record i, added onto w.  With integer codes, sqrt(C) rhat_j is the
// scale times sum_p q_p minus twice the codes at the negative entries of row
// j, the latter one int8 dot product per four codes against a 0/1 byte mask
// spread from the row's sign bits.
template <int C, int G>
__device__ __forceinline__ void add_record16(const DecodeArgs& a, uint32_t i, int sub, float (&w)[16]) {
  constexpr float isq = (C == 16) ? 0.25f : (C == 32) ? 0.17677669529663688f
                      : (C == 64) ? 0.125f : 0.08838834764831845f;
  const uint4 e0 = a.dec[2 * (size_t)i];
  const uint4 e1 = a.dec[2 * (size_t)i + 1];
  const uint32_t q4[4] = {e1.x, e1.y, e1.z, e1.w};
  const uint4* tsp = reinterpret_cast<const uint4*>(a.basis.tsign + (size_t)(e0.z & 0xFFFFu) * kMaxC + sub * 16);
  const uint4 ta = tsp[0], tb = tsp[1];
  const uint32_t tw[8] = {ta.x, ta.y, ta.z, ta.w, tb.x, tb.y, tb.z, tb.w};
  const uint32_t sfield = e0.z >> 16;
  const float scl = a.scale_fmt == AWSRC_SCALE_POW2 ? ldexpf(isq, (int)sfield - 128)
                                                    : __half2float(__ushort_as_half((uint16_t)sfield)) * isq;
  const int32_t tot = (int32_t)e0.w;
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    const uint32_t ts = (tw[e >> 1] >> (16 * (e & 1))) & 0xFFFFu;
    int32_t neg = 0;
#pragma unroll
    for (int gg = 0; gg < G; ++gg) {
      const uint32_t mask = (((ts >> (4 * gg)) & 0xFu) * 0x204081u) & 0x01010101u;
      neg = __builtin_amdgcn_sdot4((int)mask, (int)q4[gg], neg, false);
    }
    w[e] += (float)(tot - 2 * neg) * scl;
  }
}

// global-address-space views: loads and stores through them are issued as
// global (not flat) memory instructions
#define AWSRC_GLOBAL __attribute__((address_space(1)))
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

template <int C, int G>
__global__ __launch_bounds__(256) void k_reconstruct(DecodeArgs a, BackboneTabs bb) {
  constexpr int UPT = C / 16;                            // lanes per tile
  constexpr int LOG_UPT = (C == 16) ? 0 : (C == 32) ? 1 : (C == 64) ? 2 : 3;
  constexpr int NU = 4;                                  // units per lane per block iteration
  constexpr int CHUNK = NU * 256;
  __shared__ uint64_t s_off[kLdsModules + 1];
  const bool lds_tab = a.n_modules <= kLdsModules;
  if (lds_tab)
    for (int m = threadIdx.x; m <= a.n_modules; m += 256) s_off[m] = a.mod_tile_off[m];
  __syncthreads();
  const uint64_t* off = lds_tab ? s_off : a.mod_tile_off;
  const uint64_t n_units = a.T_total << LOG_UPT;
  // per-lane module state, kept in registers; units only move forward, so
  // the module walk costs at most n_modules steps per lane over the launch
  int m = 0;
  uint64_t m_lo = 0, m_hi = off[1] << LOG_UPT;
  int64_t cols = a.mod_cols[0];
  uint32_t upr = (uint32_t)(cols >> 4), gpr = (uint32_t)(cols >> bb.gshift);
  const AWSRC_GLOBAL uint8_t* cp = (const AWSRC_GLOBAL uint8_t*)bb.codes[0];
  const AWSRC_GLOBAL uint16_t* sp = (const AWSRC_GLOBAL uint16_t*)bb.scale[0];
  const AWSRC_GLOBAL uint8_t* zp = (const AWSRC_GLOBAL uint8_t*)bb.zero[0];
  AWSRC_GLOBAL uint16_t* op = (AWSRC_GLOBAL uint16_t*)a.mod_ptr[0];
  for (uint64_t c0 = (uint64_t)blockIdx.x * CHUNK; c0 < n_units; c0 += (uint64_t)gridDim.x * CHUNK) {
    // addresses of this lane's NU units, then all their loads, then the math
    const AWSRC_GLOBAL u32x2_t* qa[NU];
    const AWSRC_GLOBAL uint16_t* sa[NU];
    const AWSRC_GLOBAL uint8_t* za[NU];
    AWSRC_GLOBAL u32x4_t* oa[NU];
    uint64_t tt[NU];
    int sub[NU];
    bool ok[NU];
#pragma unroll
    for (int k = 0; k < NU; ++k) {
      const uint64_t u = c0 + k * 256 + threadIdx.x;
      ok[k] = u < n_units;
      if (ok[k] && u >= m_hi) {
        do { ++m; } while ((off[m + 1] << LOG_UPT) <= u);
        m_lo = off[m] << LOG_UPT;
        m_hi = off[m + 1] << LOG_UPT;
        cols = a.mod_cols[m];
        upr = (uint32_t)(cols >> 4);
        gpr = (uint32_t)(cols >> bb.gshift);
        cp = (const AWSRC_GLOBAL uint8_t*)bb.codes[m];
        sp = (const AWSRC_GLOBAL uint16_t*)bb.scale[m];
        zp = (const AWSRC_GLOBAL uint8_t*)bb.zero[m];
        op = (AWSRC_GLOBAL uint16_t*)a.mod_ptr[m];
      }
      const uint32_t uw = (uint32_t)(u - m_lo);          // unit within the module
      const uint32_t row = uw / upr;
      const uint32_t col0 = (uw - row * upr) * 16;
      const int64_t el = (int64_t)row * cols + col0;
      const uint32_t g = row * gpr + (col0 >> bb.gshift);
      qa[k] = (const AWSRC_GLOBAL u32x2_t*)(cp + (el >> 1));
      sa[k] = sp + g;
      za[k] = zp + g;
      oa[k] = (AWSRC_GLOBAL u32x4_t*)(op + el);
      tt[k] = u >> LOG_UPT;
      sub[k] = (int)(uw & (UPT - 1));
    }
    u32x2_t q16[NU];
    uint32_t sraw[NU], zraw[NU], bits[NU];
#pragma unroll
    for (int k = 0; k < NU; ++k) {
      if (ok[k]) {
        q16[k] = *qa[k];
        sraw[k] = *sa[k];
        zraw[k] = *za[k];
        bits[k] = a.bitmap[tt[k] >> 5];
      }
    }
#pragma unroll
    for (int k = 0; k < NU; ++k) {
      if (!ok[k]) continue;
      const float s = __half2float(__ushort_as_half((uint16_t)sraw[k]));
      const float z = (float)zraw[k];
      float w[16];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        w[e] = ((float)((q16[k].x >> (4 * e)) & 0xFu) - z) * s;
        w[8 + e] = ((float)((q16[k].y >> (4 * e)) & 0xFu) - z) * s;
      }
      if ((bits[k] >> (tt[k] & 31)) & 1u) add_record16<C, G>(a, a.tmap[tt[k]], sub[k], w);
      const u32x4_t lo = {bf16_pair(w[0], w[1]), bf16_pair(w[2], w[3]), bf16_pair(w[4], w[5]),
                          bf16_pair(w[6], w[7])};
      const u32x4_t hi = {bf16_pair(w[8], w[9]), bf16_pair(w[10], w[11]), bf16_pair(w[12], w[13]),
                          bf16_pair(w[14], w[15])};
      oa[k][0] = lo;
      oa[k][1] = hi;
    }
  }
}

template <int C>
static void launch_rec_c(const DecodeArgs& a, const BackboneTabs& bb, unsigned nb, hipStream_t st) {
  switch ((a.P + 3) / 4) {
    case 1: hipLaunchKernelGGL((k_reconstruct<C, 1>), dim3(nb), dim3(256), 0, st, a, bb); break;
    case 2: hipLaunchKernelGGL((k_reconstruct<C, 2>), dim3(nb), dim3(256), 0, st, a, bb); break;
    case 3: hipLaunchKernelGGL((k_reconstruct<C, 3>), dim3(nb), dim3(256), 0, st, a, bb); break;
    default: hipLaunchKernelGGL((k_reconstruct<C, 4>), dim3(nb), dim3(256), 0, st, a, bb); break;
  }
}

hipError_t launch_reconstruct_bf16(const DecodeArgs& a, const BackboneTabs& bb, hipStream_t st) {
  const uint64_t n_units = a.T_total * (uint64_t)(a.C / 16);
  uint64_t nb = (n_units + 1023) / 1024;
  if (nb > 256 * 8) nb = 256 * 8;  // eight resident blocks per CU, grid-stride beyond
  switch (a.C) {
    case 16: launch_rec_c<16>(a, bb, (unsigned)nb, st); break;
    case 32: launch_rec_c<32>(a, bb, (unsigned)nb, st); break;
    case 64: launch_rec_c<64>(a, bb, (unsigned)nb, st); break;
    case 128: launch_rec_c<128>(a, bb, (unsigned)nb, st); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_decode_validate(const DecodeArgs& a, hipStream_t st) {
  const int64_t nwords = (int64_t)((a.T_total + 31) / 32);
  int64_t fb = (nwords + 255) / 256;
  if (fb > 4096) fb = 4096;
  if (fb < 1) fb = 1;
  hipLaunchKernelGGL(k_fill_u32, dim3((unsigned)fb), dim3(256), 0, st, a.bitmap, nwords);
  hipLaunchKernelGGL(k_fill_u32, dim3(1), dim3(64), 0, st, reinterpret_cast<uint32_t*>(a.errors), (int64_t)2);
  if (a.K > 0)
    hipLaunchKernelGGL(k_decode_validate, dim3((unsigned)((a.K + 255) / 256)), dim3(256), 0, st, a);
  return hipGetLastError();
}

template <int C, int G>
static hipError_t apply_cg(const DecodeArgs& a, hipStream_t st) {
  constexpr int RPB = 256 / (C / 8);
  // up to eight resident blocks per CU, each looping over record groups
  int64_t nb = (a.K + RPB - 1) / RPB;
  if (nb > 256 * 8) nb = 256 * 8;
  const unsigned blocks = (unsigned)nb;
  if (a.w0_dtype == AWSRC_DTYPE_F32)
    hipLaunchKernelGGL((k_decode_apply<C, float, G>), dim3(blocks), dim3(256), 0, st, a);
  else
    hipLaunchKernelGGL((k_decode_apply<C, uint16_t, G>), dim3(blocks), dim3(256), 0, st, a);
  return hipGetLastError();
}

template <int C>
static hipError_t apply_c(const DecodeArgs& a, hipStream_t st) {
  switch ((a.P + 3) / 4) {  // groups of four codes
    case 1: return apply_cg<C, 1>(a, st);
    case 2: return apply_cg<C, 2>(a, st);
    case 3: return apply_cg<C, 3>(a, st);
    default: return apply_cg<C, 4>(a, st);
  }
}

hipError_t launch_decode_apply(const DecodeArgs& a, hipStream_t st) {
  if (a.K <= 0) return hipSuccess;
  switch (a.C) {
    case 16: return apply_c<16>(a, st);
    case 32: return apply_c<32>(a, st);
    case 64: return apply_c<64>(a, st);
    case 128: return apply_c<128>(a, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace awsrc
