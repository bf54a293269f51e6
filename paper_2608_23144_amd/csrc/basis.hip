// Seeded basis tables, GenBasis(s, C, P) of Eq. (2), generator version 1.
//
// One thread per seed draws the sign words and the P distinct Hadamard
// columns from the splitmix64 counter stream and precomputes, for every
// selected column p, the C-bit pattern of negative entries of B_s[:, p]
// (sigma_j xor parity(j & c_p)), which the encoder and decoder kernels use
// instead of regenerating the basis per tile.
#include "awsrc_internal.h"

namespace awsrc {

__global__ void k_gen_basis(uint64_t key, int C, int P, int S, uint64_t* __restrict__ sign,
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

  uint64_t used[2] = {0ull, 0ull};
  for (int p = 0; p < P; ++p) {
    const uint64_t v = splitmix64(key, base + (uint64_t)(nw + p));
    const uint32_t m = (uint32_t)(((v >> 32) * (uint64_t)(C - p)) >> 32);  // Lemire, [0, C-p)
    int c = 0;
    uint32_t seen = 0;
    for (int j = 0; j < C; ++j) {  // the m-th smallest column not drawn yet
      if ((used[j >> 6] >> (j & 63)) & 1ull) continue;
      if (seen == m) { c = j; break; }
      ++seen;
    }
    used[c >> 6] |= 1ull << (c & 63);
    col[(size_t)s * kMaxP + p] = (uint8_t)c;
    for (int w = 0; w < 2; ++w) {
      uint64_t mk = 0ull;
      for (int jj = 0; jj < 64; ++jj) {
        const int j = 64 * w + jj;
        if (j >= C) break;
        const uint64_t neg = ((uint64_t)__popc((unsigned)(j & c)) & 1ull) ^ ((sw[w] >> jj) & 1ull);
        mk |= neg << jj;
      }
      mask[((size_t)s * P + p) * 2 + w] = mk;
    }
  }
}

hipError_t launch_gen_basis(uint64_t key, int C, int P, int S, BasisTables t, hipStream_t st) {
  const int threads = 64;
  const int blocks = (S + threads - 1) / threads;
  hipLaunchKernelGGL(k_gen_basis, dim3(blocks), dim3(threads), 0, st, key, C, P, S, t.sign, t.mask,
                     t.col);
  return hipGetLastError();
}

}  // namespace awsrc
