// Backbone quantizer W0 = Q(W) of Eq. (1): asymmetric RTN-INT4 per group of
// consecutive input columns (Sec. 4 uses RTN with group size 128).
//
// One 64-lane wavefront owns one group per iteration (E = group/64 elements
// per lane, contiguous, so each load and store of the wavefront is one
// coalesced segment); min/max come from a wavefront butterfly reduction.
// Arithmetic is fp32 with correctly rounded division (this file is built
// without FMA contraction), so codes, scales and zero points are bit-exact
// with the fp32 recipe documented in awsrc.h.
#include "awsrc_internal.h"

namespace awsrc {

__device__ __forceinline__ float load_w(const float* W, int64_t i) { return W[i]; }
__device__ __forceinline__ float load_w(const uint16_t* W, int64_t i) {
  return __uint_as_float((uint32_t)W[i] << 16);
}

template <int E, typename TW>
__global__ __launch_bounds__(256) void k_backbone_rtn(const TW* __restrict__ W, int64_t rows,
                                                      int64_t cols, uint8_t* __restrict__ codes,
                                                      uint16_t* __restrict__ scale,
                                                      uint8_t* __restrict__ zero,
                                                      float* __restrict__ W0) {
  constexpr int G = 64 * E;
  const int lane = threadIdx.x & 63;
  const int64_t gpr = cols / G;  // groups per row
  const int64_t n_groups = rows * gpr;
  const int64_t wave0 = (int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
  const int64_t wstride = (int64_t)gridDim.x * (blockDim.x >> 6);
  for (int64_t g = wave0; g < n_groups; g += wstride) {
    const int64_t row = g / gpr;
    const int64_t gi = g - row * gpr;
    const int64_t base = row * cols + gi * G + (int64_t)lane * E;
    float w[E];
#pragma unroll
    for (int e = 0; e < E; ++e) w[e] = load_w(W, base + e);
    float mn = w[0], mx = w[0];
#pragma unroll
    for (int e = 1; e < E; ++e) { mn = fminf(mn, w[e]); mx = fmaxf(mx, w[e]); }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      mn = fminf(mn, __shfl_xor(mn, off, 64));
      mx = fmaxf(mx, __shfl_xor(mx, off, 64));
    }
    const float s32 = (mx - mn) / 15.0f;
    __half h = __float2half_rn(s32);
    uint16_t hb = __half_as_ushort(h);
    if ((hb & 0x7FFFu) == 0x7C00u) hb = 0x7BFFu;  // saturate +inf at 65504
    const bool degenerate = (hb & 0x7FFFu) == 0u;
    if (degenerate) hb = 0x3C00u;
    const float s = __half2float(__ushort_as_half(hb));
    float z = degenerate ? 0.0f : fminf(fmaxf(rintf(-mn / s), 0.0f), 15.0f);
    uint32_t q[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const float qf = degenerate ? 0.0f : fminf(fmaxf(rintf(w[e] / s) + z, 0.0f), 15.0f);
      q[e] = (uint32_t)qf;
      if (W0) W0[base + e] = (qf - z) * s;
    }
    // pack two 4-bit codes per byte, even column in the low nibble
    if constexpr (E == 1) {
      const uint32_t other = (uint32_t)__shfl_down((int)q[0], 1, 64);
      if ((lane & 1) == 0) codes[base >> 1] = (uint8_t)(q[0] | (other << 4));
    } else {
#pragma unroll
      for (int e = 0; e < E; e += 2) codes[(base + e) >> 1] = (uint8_t)(q[e] | (q[e + 1] << 4));
    }
    if (lane == 0) {
      scale[g] = hb;
      zero[g] = (uint8_t)z;
    }
  }
}

template <int E>
static hipError_t launch_e(const void* W, int w_dtype, int64_t rows, int64_t cols, uint8_t* codes,
                           uint16_t* scale, uint8_t* zero, float* W0, hipStream_t st) {
  const int64_t n_groups = rows * (cols / (64 * E));
  int64_t blocks = (n_groups + 3) / 4;
  if (blocks > 256 * 64) blocks = 256 * 64;
  if (blocks < 1) blocks = 1;
  if (w_dtype == AWSRC_DTYPE_F32)
    hipLaunchKernelGGL((k_backbone_rtn<E, float>), dim3((unsigned)blocks), dim3(256), 0, st,
                       static_cast<const float*>(W), rows, cols, codes, scale, zero, W0);
  else
    hipLaunchKernelGGL((k_backbone_rtn<E, uint16_t>), dim3((unsigned)blocks), dim3(256), 0, st,
                       static_cast<const uint16_t*>(W), rows, cols, codes, scale, zero, W0);
  return hipGetLastError();
}

hipError_t launch_backbone(const void* W, int w_dtype, int64_t rows, int64_t cols, int group,
                           uint8_t* codes, uint16_t* scale, uint8_t* zero, float* W0,
                           hipStream_t st) {
  switch (group) {
    case 64: return launch_e<1>(W, w_dtype, rows, cols, codes, scale, zero, W0, st);
    case 128: return launch_e<2>(W, w_dtype, rows, cols, codes, scale, zero, W0, st);
    case 256: return launch_e<4>(W, w_dtype, rows, cols, codes, scale, zero, W0, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace awsrc
