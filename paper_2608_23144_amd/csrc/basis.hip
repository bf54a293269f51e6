// Seeded basis tables, GenBasis(s, C, P) of Eq. (2).
//
// One thread per seed draws the sign words and the P distinct Hadamard
// columns from the splitmix64 counter stream and precomputes, for every
// selected column p, the C-bit pattern of negative entries of B_s[:, p]
// (sigma_j xor parity(j & c_p)), which the encoder and decoder kernels use
// instead of regenerating the basis per tile; a second kernel transposes the
// patterns into one u16 of P sign bits per coordinate for the decoder.
// Generator version 2 adds the seeded coordinate permutation
// B_s[j, p] = sigma_j H[pi(j), c_p] / sqrt(C): one wavefront per seed draws a
// sort key per coordinate (the words after the column words), ranks them
// (pi(j) = rank of (key_j, j)), and builds the negative-entry patterns
// sigma_j xor parity(pi(j) & c_p) by wavefront ballots.
#include "awsrc_internal.h"

namespace awsrc {

// Position of the m-th zero bit (0-based) among the low `width` bits of w.
__device__ __forceinline__ int nth_zero(uint64_t w, int m, int width) {
  uint64_t z = ~w;
  if (width < 64) z &= (1ull << width) - 1ull;
  int pos = 0;
#pragma unroll
  for (int half = 32; half >= 1; half >>= 1) {
    const uint64_t lowmask = (1ull << half) - 1ull;
    const int cnt = __popcll(z & lowmask);
    if (m >= cnt) { m -= cnt; z >>= half; pos += half; }
  }
  return pos;
}

// Bit j of the result is parity(j & c) for j = 64*w .. 64*w + 63: the XOR of
// the patterns "bit b of j" over the set bits b of c.
__device__ __forceinline__ uint64_t hadamard_neg_word(int c, int w) {
  const uint64_t pat[6] = {0xAAAAAAAAAAAAAAAAull, 0xCCCCCCCCCCCCCCCCull, 0xF0F0F0F0F0F0F0F0ull,
                           0xFF00FF00FF00FF00ull, 0xFFFF0000FFFF0000ull, 0xFFFFFFFF00000000ull};
  uint64_t x = 0ull;
#pragma unroll
  for (int b = 0; b < 6; ++b)
    if ((c >> b) & 1) x ^= pat[b];
  if (((c >> 6) & 1) && w == 1) x = ~x;
  return x;
}

__global__ void k_gen_basis(uint64_t key, int C, int P, int S, int gen_version, uint64_t* __restrict__ sign,
                            uint64_t* __restrict__ mask, uint8_t* __restrict__ col) {
  const int s = blockIdx.x * blockDim.x + threadIdx.x;
  if (s >= S) return;
  const int nw = (C + 63) / 64;
  const uint64_t base = (uint64_t)s << 32;
  uint64_t sw[2] = {0ull, 0ull};
  for (int i = 0; i < nw; ++i) sw[i] = splitmix64(key, base + (uint64_t)i);
  if (C < 64) sw[0] &= (1ull << C) - 1ull;
  sign[2 * (size_t)s] = sw[0];
  sign[2 * (size_t)s + 1] = sw[1];
  const uint64_t valid0 = C < 64 ? (1ull << C) - 1ull : ~0ull;
  uint64_t used[2] = {0ull, 0ull};
  for (int p = 0; p < P; ++p) {
    const uint64_t v = splitmix64(key, base + (uint64_t)(nw + p));
    int m = (int)(((v >> 32) * (uint64_t)(C - p)) >> 32);  // Lemire multiply-shift into [0, C-p)
    // the m-th smallest column not drawn yet
    const int w0 = C < 64 ? C : 64;
    const int z0 = w0 - __popcll(used[0] & valid0);
    int c;
    if (m < z0) c = nth_zero(used[0], m, w0);
    else c = 64 + nth_zero(used[1], m - z0, 64);
    used[c >> 6] |= 1ull << (c & 63);
    col[(size_t)s * kMaxP + p] = (uint8_t)c;
    if (gen_version != 1) continue;  // version 2: k_basis_perm builds the patterns
    for (int w = 0; w < 2; ++w) {
      uint64_t mk = 0ull;
      if (w < nw) mk = (hadamard_neg_word(c, w) ^ sw[w]) & (w == 0 ? valid0 : ~0ull);
      mask[((size_t)s * P + p) * 2 + w] = mk;
    }
  }
}

// Transposed signs, one thread per (seed, coordinate j): the P sign bits of
// row j of B_s packed into one u16.
__global__ void k_basis_tsign(int C, int P, int S, const uint64_t* __restrict__ mask,
                              uint16_t* __restrict__ tsign) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (int64_t)S * C) return;
  const int s = (int)(i / C), j = (int)(i % C);
  uint32_t t = 0;
  for (int p = 0; p < P; ++p)
    t |= (uint32_t)((mask[((size_t)s * P + p) * 2 + (j >> 6)] >> (j & 63)) & 1ull) << p;
  tsign[(size_t)s * kMaxC + j] = (uint16_t)t;
}

// Version 2: one wavefront per seed, lane j (and j + 64) owns coordinate j.
__global__ __launch_bounds__(64) void k_basis_perm(uint64_t key, int C, int P, BasisTables t) {
  __shared__ uint64_t s_key[kMaxC];
  const int s = blockIdx.x;
  const int nw = (C + 63) / 64;
  const uint64_t base = ((uint64_t)s << 32) + (uint64_t)(nw + P);
  for (int j = threadIdx.x; j < C; j += 64) s_key[j] = splitmix64(key, base + (uint64_t)j);
  __syncthreads();
  const uint64_t sw0 = t.sign[2 * (size_t)s], sw1 = t.sign[2 * (size_t)s + 1];
  for (int h = 0; h < nw; ++h) {
    const int j = threadIdx.x + 64 * h;
    const bool on = j < C;
    int rank = 0;
    if (on) {
      const uint64_t kj = s_key[j];
      for (int i = 0; i < C; ++i) {
        const uint64_t ki = s_key[i];
        rank += (ki < kj) || (ki == kj && i < j);
      }
      t.perm[(size_t)s * kMaxC + j] = (uint8_t)rank;
      t.iperm[(size_t)s * kMaxC + rank] = (uint8_t)j;
    }
    const uint64_t sg = ((h == 0 ? sw0 : sw1) >> (j & 63)) & 1ull;
    for (int p = 0; p < P; ++p) {
      const int c = t.col[(size_t)s * kMaxP + p];
      const bool neg = on && ((sg ^ (uint64_t)(__popc((unsigned)(rank & c)) & 1)) != 0);
      const uint64_t word = __ballot(neg);
      if (threadIdx.x == 0) t.mask[((size_t)s * P + p) * 2 + h] = word;
    }
  }
  if (nw == 1 && threadIdx.x == 0)
    for (int p = 0; p < P; ++p) t.mask[((size_t)s * P + p) * 2 + 1] = 0ull;
}

hipError_t launch_gen_basis(uint64_t key, int C, int P, int S, int gen_version, BasisTables t, hipStream_t st) {
  const int threads = 64;
  const int blocks = (S + threads - 1) / threads;
  hipLaunchKernelGGL(k_gen_basis, dim3(blocks), dim3(threads), 0, st, key, C, P, S, gen_version, t.sign,
                     t.mask, t.col);
  if (gen_version == 2) hipLaunchKernelGGL(k_basis_perm, dim3((unsigned)S), dim3(64), 0, st, key, C, P, t);
  const int64_t n = (int64_t)S * C;
  hipLaunchKernelGGL(k_basis_tsign, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, C, P, S,
                     t.mask, t.tsign);
  return hipGetLastError();
}

}  // namespace awsrc
