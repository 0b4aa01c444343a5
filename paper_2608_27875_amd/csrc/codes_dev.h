// Device conversions of quantized codes (int8, packed int4, FP8 E4M3, packed
// FP4 E2M1) to f16
// MFMA operands, shared by the prefill and decode attention kernels.  Every
// conversion is exact: codes are small integers or E4M3 values, both exact in
// f16, and the only scaling applied is by a power of two.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "hyq.h"

namespace hyq {

typedef _Float16 v2h __attribute__((ext_vector_type(2)));

// Power-of-two factor applied to the V codes of one tile while they are
// converted to f16 (vmul = 2^e; nbias = -1152 * 2^e for the int8 route).
struct VScale {
  v2h vmul, nbias;
  float f32;
};

__device__ __forceinline__ VScale make_vscale(float p2) {
  VScale v;
  v.vmul = v2h{(_Float16)p2, (_Float16)p2};
  v.nbias = v2h{(_Float16)(-1152.0f * p2), (_Float16)(-1152.0f * p2)};
  v.f32 = p2;
  return v;
}

// int8 codes (4 per dword) -> f16 pairs of code * 2^e, exact: bytes biased to
// unsigned, placed as the low mantissa byte of 1024 (f16 0x64xx), then one
// fused (x * 2^e - 1152 * 2^e) per pair.
__device__ __forceinline__ void i8x4_to_h(uint32_t w, uint32_t& h01, uint32_t& h23,
                                          const VScale& vs) {
  const uint32_t u = w ^ 0x80808080u;
  const uint32_t a = __builtin_amdgcn_perm(0x64646464u, u, 0x04010400u);
  const uint32_t b = __builtin_amdgcn_perm(0x64646464u, u, 0x04030402u);
  const v2h ha = __builtin_elementwise_fma(__builtin_bit_cast(v2h, a), vs.vmul, vs.nbias);
  const v2h hb = __builtin_elementwise_fma(__builtin_bit_cast(v2h, b), vs.vmul, vs.nbias);
  h01 = __builtin_bit_cast(uint32_t, ha);
  h23 = __builtin_bit_cast(uint32_t, hb);
}

// Four E4M3 codes (one per byte) -> f16 pairs of value * 2^e, exact unless
// the result is below the f16 range (the conversion applies power-of-two
// scales exactly).
__device__ __forceinline__ void e4m3x4_to_h(uint32_t w, uint32_t& h01, uint32_t& h23,
                                            const VScale& vs) {
  h01 = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(w, vs.f32, false));
  h23 = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(w, vs.f32, true));
}

template <int FMT>
__device__ __forceinline__ void codes4_to_h(uint32_t w, uint32_t& h01, uint32_t& h23,
                                            const VScale& vs) {
  if constexpr (FMT == HYQ_FMT_FP8) e4m3x4_to_h(w, h01, h23, vs);
  else i8x4_to_h(w, h01, h23, vs);
}

// Eight packed E2M1 codes (element 2i in the low nibble of byte i) -> f16
// pairs (elements 2i, 2i+1 in h[i]) of value * p2, p2 a power of two: exact
// unless the result is below the f16 range.
__device__ __forceinline__ void e2m1x8_to_h(uint32_t w, uint32_t (&h)[4], float p2) {
  h[0] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, p2, 0));
  h[1] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, p2, 1));
  h[2] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, p2, 2));
  h[3] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, p2, 3));
}

// Packed int4 (8 nibbles, element 2i low / 2i+1 high in byte i) -> 8 int8 of
// value 16*code, in element order.
__device__ __forceinline__ void i4x8_to_i8(uint32_t w, uint32_t& o0, uint32_t& o1) {
  const uint32_t lo = (w << 4) & 0xF0F0F0F0u;   // elements 0,2,4,6 (x16)
  const uint32_t hi = w & 0xF0F0F0F0u;          // elements 1,3,5,7 (x16)
  o0 = __builtin_amdgcn_perm(hi, lo, 0x05010400u);
  o1 = __builtin_amdgcn_perm(hi, lo, 0x07030602u);
}

}  // namespace hyq
