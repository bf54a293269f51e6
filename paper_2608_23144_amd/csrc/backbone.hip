// Backbone quantizer W0 = Q(W) of Eq. (1): asymmetric RTN-INT4 per group of
// consecutive input columns (Sec. 4 uses RTN with group size 128).
//
// Lanes own 8 weights of one group; the lanes of a group reduce min/max with
// butterfly shuffles, and every load and store is a wide coalesced access.
// Arithmetic is fp32 with correctly rounded division (this file is built
// without FMA contraction), so codes, scales and zero points are bit-exact
// with the fp32 recipe documented in awsrc.h.
#include "awsrc_internal.h"

namespace awsrc {

// LPG = group/8 lanes share one group, and lane sub of a group owns elements
// 4 sub .. 4 sub + 3 of each half of it, so that the group's lanes cover each
// half with adjacent accesses: per half, an 8-byte load of bf16 W (16-byte for
// fp32), a 16-byte W0 store and a 2-byte store of 4 codes, and every W0
// store instruction writes whole 64-byte pieces.  (With 8 consecutive weights
// per lane, its two 16-byte W0 stores 32 bytes apart reached memory as
// partial lines, 1.07 times the bytes, and the kernel ran 9% slower.)  A
// wavefront covers 64/LPG groups per iteration.
template <int LPG, typename TW>
__global__ __launch_bounds__(256) void k_backbone_rtn(const TW* __restrict__ W, int64_t rows,
                                                      int64_t cols, uint8_t* __restrict__ codes,
                                                      uint16_t* __restrict__ scale,
                                                      uint8_t* __restrict__ zero,
                                                      float* __restrict__ W0) {
  constexpr int G = 8 * LPG;            // group size
  constexpr int GPW = 64 / LPG;         // groups per wavefront per iteration
  const int lane = threadIdx.x & 63;
  const int sub = lane % LPG;           // position within the group
  const int64_t gpr = cols / G;         // groups per row
  const int64_t n_groups = rows * gpr;
  const int64_t wave0 = (int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
  const int64_t wstride = (int64_t)gridDim.x * (blockDim.x >> 6);
  for (int64_t g0 = wave0 * GPW; g0 < n_groups; g0 += wstride * GPW) {
    const int64_t g = g0 + lane / LPG;
    const bool valid = g < n_groups;
    const int64_t gg = valid ? g : n_groups - 1;
    const int64_t row = gg / gpr;
    // this lane's run in the first half of the group; the second is G/2 on
    const int64_t base = row * cols + (gg - row * gpr) * G + (int64_t)sub * 4;
    float w[8];  // w[0..3]: first half, w[4..7]: second half
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int64_t b = base + h * (G / 2);
      if constexpr (sizeof(TW) == 4) {
        const float4 x = *reinterpret_cast<const float4*>(W + b);
        w[4 * h] = x.x; w[4 * h + 1] = x.y; w[4 * h + 2] = x.z; w[4 * h + 3] = x.w;
      } else {
        const uint2 x = *reinterpret_cast<const uint2*>(W + b);
        w[4 * h] = __uint_as_float(x.x << 16);
        w[4 * h + 1] = __uint_as_float(x.x & 0xFFFF0000u);
        w[4 * h + 2] = __uint_as_float(x.y << 16);
        w[4 * h + 3] = __uint_as_float(x.y & 0xFFFF0000u);
      }
    }
    float mn = w[0], mx = w[0];
#pragma unroll
    for (int e = 1; e < 8; ++e) { mn = fminf(mn, w[e]); mx = fmaxf(mx, w[e]); }
#pragma unroll
    for (int off = LPG / 2; off >= 1; off >>= 1) {
      mn = fminf(mn, __shfl_xor(mn, off, 64));
      mx = fmaxf(mx, __shfl_xor(mx, off, 64));
    }
    const float s32 = (mx - mn) / 15.0f;
    uint16_t hb = __half_as_ushort(__float2half_rn(s32));
    if ((hb & 0x7FFFu) == 0x7C00u) hb = 0x7BFFu;  // saturate +inf at 65504
    const bool degenerate = (hb & 0x7FFFu) == 0u;
    if (degenerate) hb = 0x3C00u;
    const float s = __half2float(__ushort_as_half(hb));
    const float z = degenerate ? 0.0f : fminf(fmaxf(rintf(-mn / s), 0.0f), 15.0f);
    uint32_t packed = 0;
    float o[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float qf = degenerate ? 0.0f : fminf(fmaxf(rintf(w[e] / s) + z, 0.0f), 15.0f);
      packed |= (uint32_t)qf << (4 * e);  // even column in the low nibble of each byte (per half)
      o[e] = (qf - z) * s;
    }
    if (valid) {
      if (W0) {
        // streaming stores: W0 is written once and read by later launches
        typedef float f32x4_nt __attribute__((ext_vector_type(4)));
        __builtin_nontemporal_store(f32x4_nt{o[0], o[1], o[2], o[3]}, reinterpret_cast<f32x4_nt*>(W0 + base));
        __builtin_nontemporal_store(f32x4_nt{o[4], o[5], o[6], o[7]},
                                    reinterpret_cast<f32x4_nt*>(W0 + base + G / 2));
      }
      *reinterpret_cast<uint16_t*>(codes + (base >> 1)) = (uint16_t)packed;
      *reinterpret_cast<uint16_t*>(codes + ((base + G / 2) >> 1)) = (uint16_t)(packed >> 16);
      if (sub == 0) {
        scale[g] = hb;
        zero[g] = (uint8_t)z;
      }
    }
  }
}

template <int LPG>
static hipError_t launch_e(const void* W, int w_dtype, int64_t rows, int64_t cols, uint8_t* codes,
                           uint16_t* scale, uint8_t* zero, float* W0, hipStream_t st) {
  const int64_t n_groups = rows * (cols / (8 * LPG));
  const int64_t per_block = 4 * (64 / LPG);
  int64_t blocks = (n_groups + per_block - 1) / per_block;
  if (blocks > 256 * 32) blocks = 256 * 32;
  if (blocks < 1) blocks = 1;
  if (w_dtype == AWSRC_DTYPE_F32)
    hipLaunchKernelGGL((k_backbone_rtn<LPG, float>), dim3((unsigned)blocks), dim3(256), 0, st,
                       static_cast<const float*>(W), rows, cols, codes, scale, zero, W0);
  else
    hipLaunchKernelGGL((k_backbone_rtn<LPG, uint16_t>), dim3((unsigned)blocks), dim3(256), 0, st,
                       static_cast<const uint16_t*>(W), rows, cols, codes, scale, zero, W0);
  return hipGetLastError();
}

hipError_t launch_backbone(const void* W, int w_dtype, int64_t rows, int64_t cols, int group,
                           uint8_t* codes, uint16_t* scale, uint8_t* zero, float* W0,
                           hipStream_t st) {
  switch (group) {
    case 64: return launch_e<8>(W, w_dtype, rows, cols, codes, scale, zero, W0, st);
    case 128: return launch_e<16>(W, w_dtype, rows, cols, codes, scale, zero, W0, st);
    case 256: return launch_e<32>(W, w_dtype, rows, cols, codes, scale, zero, W0, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace awsrc
