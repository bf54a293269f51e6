// Decoder (Sec. 3.2): every record regenerates its basis B_s and adds
// B_s (scale * q) onto its tile of W0; tiles without a record are untouched.
//
// validate - one thread per record: field ranges, finite non-negative scale,
//            and a bitmap over tiles that catches a tile appearing twice
//            (records of a valid stream touch disjoint tiles, which is what
//            lets the apply pass run without atomics or ordering).
// apply    - C/4 lanes per record, four consecutive weights per lane; each
//            weight gets rhat_j = (1/sqrt(C)) sum_p (+-1) scale*q_p with the
//            signs read from the precomputed negative-entry masks of B_s.
#include "awsrc_internal.h"

namespace awsrc {

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

__device__ __forceinline__ Rec parse(const uint8_t* r, const DecodeArgs& a) {
  uint64_t w[3] = {0, 0, 0};
  for (int k = 0; k < a.L_rec; ++k) w[k >> 3] |= (uint64_t)r[k] << (8 * (k & 7));
  Rec out;
  int pos = 0;
  out.idx = get_bits(w, pos, a.idx_bits);
  out.seed = (uint32_t)get_bits(w, pos, a.seed_bits);
  for (int p = 0; p < a.P; ++p) {
    int64_t c = (int64_t)get_bits(w, pos, a.b);
    if (c >> (a.b - 1)) c -= (int64_t)1 << a.b;
    out.q[p] = (int32_t)c;
  }
  out.scale = (uint32_t)get_bits(w, pos, 16);
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
  const Rec r = parse(a.recs + i * a.L_rec, a);
  const int qmax = (1 << (a.b - 1)) - 1;
  bool bad = r.idx >= a.T_total || r.seed >= (uint32_t)a.S;
  for (int p = 0; p < a.P; ++p) bad |= r.q[p] < -qmax || r.q[p] > qmax;
  bad |= (r.scale & 0x8000u) != 0 || (r.scale & 0x7C00u) == 0x7C00u;  // negative, inf or NaN
  if (!bad) {
    const uint32_t bit = 1u << (r.idx & 31);
    const uint32_t old = atomicOr(&a.bitmap[r.idx >> 5], bit);
    bad = (old & bit) != 0;
  }
  if (bad) atomicAdd(a.errors, 1ull);
}

template <int C, typename TW>
__global__ __launch_bounds__(256) void k_decode_apply(DecodeArgs a) {
  constexpr int LPR = C / 4;           // lanes per record
  constexpr int RPB = 256 / LPR;       // records per block
  const int sub = threadIdx.x % LPR;
  const int64_t i = (int64_t)blockIdx.x * RPB + threadIdx.x / LPR;
  if (i >= a.K) return;
  const Rec r = parse(a.recs + i * a.L_rec, a);
  // module of this global tile index
  int lo = 0, hi = a.n_modules - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (a.mod_tile_off[mid] <= r.idx) lo = mid; else hi = mid - 1;
  }
  const int64_t cols = a.mod_cols[lo];
  const int64_t local = (int64_t)(r.idx - a.mod_tile_off[lo]);
  const int64_t nb = cols / C;
  const int64_t row = local / nb;
  const int64_t blk = local - row * nb;
  const int64_t base = row * cols + blk * C + sub * 4;
  const float sc = __half2float(__ushort_as_half((uint16_t)r.scale));
  constexpr float isq = (C == 16) ? 0.25f : (C == 32) ? 0.17677669529663688f
                      : (C == 64) ? 0.125f : 0.08838834764831845f;
  const uint64_t* mk = a.basis.mask + (size_t)r.seed * a.P * 2;
  const int j0 = sub * 4;
  float add[4] = {0.f, 0.f, 0.f, 0.f};
  for (int p = 0; p < a.P; ++p) {
    const float ah = sc * (float)r.q[p];
    const uint64_t m = mk[2 * p + (j0 >> 6)] >> (j0 & 63);
#pragma unroll
    for (int e = 0; e < 4; ++e) add[e] += ((m >> e) & 1ull) ? -ah : ah;
  }
  TW* W0 = static_cast<TW*>(a.mod_ptr[lo]);
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    if constexpr (sizeof(TW) == 4) {
      W0[base + e] = W0[base + e] + add[e] * isq;
    } else {
      const float w = __uint_as_float((uint32_t)W0[base + e] << 16) + add[e] * isq;
      uint32_t u = __float_as_uint(w);
      u += 0x7FFFu + ((u >> 16) & 1u);  // round to nearest even (finite values)
      W0[base + e] = (TW)(u >> 16);
    }
  }
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

template <int C>
static hipError_t apply_c(const DecodeArgs& a, hipStream_t st) {
  constexpr int RPB = 256 / (C / 4);
  const unsigned blocks = (unsigned)((a.K + RPB - 1) / RPB);
  if (a.w0_dtype == AWSRC_DTYPE_F32)
    hipLaunchKernelGGL((k_decode_apply<C, float>), dim3(blocks), dim3(256), 0, st, a);
  else
    hipLaunchKernelGGL((k_decode_apply<C, uint16_t>), dim3(blocks), dim3(256), 0, st, a);
  return hipGetLastError();
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
