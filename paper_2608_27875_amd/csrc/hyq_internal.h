// Internal declarations shared by the libhyq translation units (host launch
// wrappers and small device helpers).  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "hyq.h"

namespace hyq {

// ---- host-side launch wrappers (each returns a hipError_t) ----------------

hipError_t launch_select(const hyq_shape& s, const hyq_sizes& z, const uint16_t* Q,
                         const uint16_t* K, int32_t* idx, float* scores, float* qsum,
                         hipStream_t st);

hipError_t launch_quantize(const hyq_shape& s, const hyq_sizes& z, const uint16_t* Q,
                           const uint16_t* K, const uint16_t* V, const int32_t* idx,
                           int8_t* q_codes, float* q_scale, uint8_t* k_codes, float* k_scale,
                           uint8_t* v_codes, float* v_scale, int32_t* kq_pos, hipStream_t st);

hipError_t launch_attn_prefill(const hyq_shape& s, const hyq_sizes& z, const uint16_t* Q,
                               const uint16_t* K, const uint16_t* V, const int32_t* idx,
                               const int8_t* q_codes, const float* q_scale,
                               const uint8_t* k_codes, const float* k_scale,
                               const uint8_t* v_codes, const float* v_scale,
                               const int32_t* kq_pos, float softmax_scale, void* out,
                               int out_dtype, hipStream_t st);

// ---- device helpers -------------------------------------------------------

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t b) {
  return __uint_as_float(b << 16);
}

// Low / high bf16 of a packed pair, widened exactly.
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

constexpr int kHeadDim = 128;
constexpr int kBlock = 64;

}  // namespace hyq
