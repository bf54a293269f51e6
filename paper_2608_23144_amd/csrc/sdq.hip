// Scale double quantization (SDQ) of the RTN backbone's group scales
// (Sec. 3.3 names it, after QLoRA's double quantization of quantization
// constants; Sec. 4 gives its size for RTN g128), and the backbone W0 with
// the dequantized scales.
//
// Format (the paper specifies only the rate): blocks of kSdqBlock = 256
// consecutive group scales (row-major order); per block
//   mu    = f32(sum_g s_g / n)   (sum in fp64, in group order; one division)
//   dlt_g = f32(s_g - mu)
//   a     = max_g |dlt_g|
//   c_g   = rint(dlt_g * 127 / a) in [-127, 127] (fp64: the product is exact,
//           one division, ties to even); all 0 when a = 0
//   step  = f32(a / 127)         (fp64 division, one rounding)
// and s_hat_g = f32(mu + c_g * step), evaluated in fp64 where both terms and
// their sum are exact (|mu| / step < 2^19 and c_g * step has 31 bits), so
// one rounding.
#include <math.h>

#include "awsrc_internal.h"

namespace awsrc {

namespace {

// One wavefront per block: the scales go through LDS so that lane 0 can sum
// them in order (the order fixes the rounding when the fp64 sum is inexact).
__global__ __launch_bounds__(64) void k_sdq_encode(const uint16_t* __restrict__ s16, int64_t n, int8_t* __restrict__ code,
                                                   float* __restrict__ mean, float* __restrict__ step) {
  __shared__ float sv[kSdqBlock];
  __shared__ float mu_sh;
  const int lane = threadIdx.x;
  const int64_t b = blockIdx.x;
  const int64_t g0 = b * kSdqBlock;
  const int nb = (int)(n - g0 < kSdqBlock ? n - g0 : kSdqBlock);
#pragma unroll
  for (int k = 0; k < kSdqBlock / 64; ++k) {
    const int i = k * 64 + lane;
    sv[i] = i < nb ? __half2float(__ushort_as_half(s16[g0 + i])) : 0.0f;
  }
  __syncthreads();
  if (lane == 0) {
    double tot = 0.0;
    for (int i = 0; i < nb; ++i) tot += (double)sv[i];
    mu_sh = (float)(tot / (double)nb);
  }
  __syncthreads();
  const float mu = mu_sh;
  float dl[kSdqBlock / 64];
  float am = 0.0f;
#pragma unroll
  for (int k = 0; k < kSdqBlock / 64; ++k) {
    const int i = k * 64 + lane;
    dl[k] = sv[i] - mu;  // one fp32 rounding
    if (i < nb) am = fmaxf(am, fabsf(dl[k]));
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) am = fmaxf(am, __shfl_xor(am, m, 64));
  const double a = (double)am;
#pragma unroll
  for (int k = 0; k < kSdqBlock / 64; ++k) {
    const int i = k * 64 + lane;
    if (i < nb) {
      double c = a > 0.0 ? rint((double)dl[k] * 127.0 / a) : 0.0;
      c = fmin(fmax(c, -127.0), 127.0);
      code[g0 + i] = (int8_t)(int)c;
    }
  }
  if (lane == 0) {
    mean[b] = mu;
    step[b] = (float)(a / 127.0);
  }
}

// W0 = f32(q - z) * s_hat per group; each thread writes 4 consecutive weights
// (2 code bytes in, one 16-byte store out), so that a wavefront's stores are
// adjacent (8 weights per thread, as two stores 32 bytes apart, ran 14%
// slower).
__global__ __launch_bounds__(256) void k_sdq_dequant(const uint8_t* __restrict__ codes, const uint8_t* __restrict__ zero,
                                                     const int8_t* __restrict__ sc, const float* __restrict__ mean,
                                                     const float* __restrict__ step, int64_t n4, int group,
                                                     float* __restrict__ W0) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t w0 = 4 * i;        // first weight (row-major; groups never straddle rows)
    const int64_t g = w0 / group;    // global group index
    const int64_t blk = g / kSdqBlock;
    const float sh = (float)((double)mean[blk] + (double)sc[g] * (double)step[blk]);
    const float z = (float)zero[g];
    const uint32_t q2 = *reinterpret_cast<const uint16_t*>(codes + 2 * i);
    float o[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) o[k] = ((float)((q2 >> (4 * k)) & 0xFu) - z) * sh;
    *reinterpret_cast<float4*>(W0 + w0) = make_float4(o[0], o[1], o[2], o[3]);
  }
}

}  // namespace

int64_t sdq_blocks(int64_t n_groups) { return (n_groups + kSdqBlock - 1) / kSdqBlock; }

hipError_t launch_sdq_encode(const uint16_t* s16, int64_t n_groups, int8_t* code, float* mean, float* step,
                             hipStream_t st) {
  const int64_t nb = sdq_blocks(n_groups);
  if (nb > 0) hipLaunchKernelGGL(k_sdq_encode, dim3((unsigned)nb), dim3(64), 0, st, s16, n_groups, code, mean, step);
  return hipGetLastError();
}

hipError_t launch_sdq_dequant(const uint8_t* codes, const uint8_t* zero, const int8_t* sc, const float* mean,
                              const float* step, int64_t rows, int64_t cols, int group, float* W0, hipStream_t st) {
  const int64_t n4 = rows * cols / 4;
  if (n4 <= 0) return hipSuccess;
  int64_t nb = (n4 + 255) / 256;
  if (nb > 256 * 32) nb = 256 * 32;
  hipLaunchKernelGGL(k_sdq_dequant, dim3((unsigned)nb), dim3(256), 0, st, codes, zero, sc, mean, step, n4, group, W0);
  return hipGetLastError();
}

}  // namespace awsrc
