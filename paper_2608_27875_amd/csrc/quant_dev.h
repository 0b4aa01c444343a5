// Device helpers of per-block symmetric quantization (Algorithm 2, Stage 2),
// shared by the prefill quantizer and the decode cache's block merges.
#pragma once

#include "hyq_internal.h"

namespace hyq {

constexpr int kQuantThreads = 256;

// Maximum over the kQuantThreads threads of a workgroup (every thread gets it).
__device__ __forceinline__ float block_max(float v, float* sh) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) sh[w] = v;
  __syncthreads();
  float r = sh[0];
  for (int i = 1; i < kQuantThreads / 64; ++i) r = fmaxf(r, sh[i]);
  __syncthreads();
  return r;
}

// 32 bf16 values (64 bytes) as float.
__device__ __forceinline__ void load32(const uint16_t* p, float* x) {
  const uint4* q = reinterpret_cast<const uint4*>(p);
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const uint4 w = q[u];
    const uint32_t ww[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      x[u * 8 + 2 * e] = bf16_lo(ww[e]);
      x[u * 8 + 2 * e + 1] = bf16_hi(ww[e]);
    }
  }
}

__device__ __forceinline__ int quant1(float x, float s, float c) {
  // s > 0 here; x / s is the correctly rounded IEEE quotient
  const float q = __builtin_rintf(x / s);
  return (int)fminf(fmaxf(q, -c), c);
}

// E4M3 bit pattern of x / s (s > 0); the clamp keeps -0 and bounds the
// quotient by the largest finite value.
__device__ __forceinline__ int quant1_fp8(float x, float s) {
  const float y = fminf(fmaxf(x / s, -448.0f), 448.0f);
  return __builtin_amdgcn_cvt_pk_fp8_f32(y, 0.0f, 0, false) & 0xff;
}

// E2M1 code (0..15) of x / s (s > 0): the nearest of the magnitudes 0, 0.5,
// 1, 1.5, 2, 3, 4, 6 (codes 0..7), a tie going to the even code, beyond 5
// the largest; bit 3 is the sign of the quotient (so -0 gives 8).
__device__ __forceinline__ int quant1_fp4(float x, float s) {
  const float y = x / s;
  const float a = fabsf(y);
  const int c = (a > 0.25f) + (a >= 0.75f) + (a > 1.25f) + (a >= 1.75f) + (a > 2.5f) +
                (a >= 3.5f) + (a > 5.0f);
  return c | (int)((__float_as_uint(y) >> 31) << 3);
}

// E2M3 code (0..63) of x / s (s > 0): the nearest of the 32 magnitudes
// (eighths below 2, quarters up to 4, halves up to 7.5), a tie going to the
// even code, beyond 7.5 the largest; bit 5 is the sign of the quotient.
// Within each binade [0,1), [1,2), [2,4), [4,8) the magnitudes are evenly
// spaced and start at an even code, so the nearest one is the binade's
// first code plus rint((a - base) / step), computed exactly.
__device__ __forceinline__ int quant1_fp6(float x, float s) {
  const float y = x / s;
  const float a = fabsf(y);
  const float base = a < 1.0f ? 0.0f : a < 2.0f ? 1.0f : a < 4.0f ? 2.0f : 4.0f;
  const float inv = a < 2.0f ? 8.0f : a < 4.0f ? 4.0f : 2.0f;
  const int c0 = a < 1.0f ? 0 : a < 2.0f ? 8 : a < 4.0f ? 16 : 24;
  const int c = min(31, c0 + (int)__builtin_rintf(fminf(a - base, 8.0f) * inv));
  return c | (int)((__float_as_uint(y) >> 31) << 5);
}

template <int FMT>
__device__ __forceinline__ int quant_code(float x, float s, float c) {
  if (FMT == HYQ_FMT_FP8) return quant1_fp8(x, s);
  if (FMT == HYQ_FMT_FP4) return quant1_fp4(x, s);
  if (FMT == HYQ_FMT_FP4Q6) return quant1_fp6(x, s);
  return quant1(x, s, c);
}

// c_B of a code format and bit-width (Algorithm 2, Stage 2).
template <int BITS, int FMT>
constexpr float code_bound() {
  return FMT == HYQ_FMT_FP8 ? 448.0f : FMT == HYQ_FMT_FP4 ? 6.0f : (BITS == 8 ? 127.0f : 7.0f);
}

}  // namespace hyq
