// Internal declarations shared by the libhyq translation units (host launch
// wrappers and small device helpers).  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "hyq.h"

namespace hyq {

// ---- host-side launch wrappers (each returns a hipError_t) ----------------

// Selection (Algorithm 1, or the column mass) into idx.  Scratch: scores
// ([B][Hkv][P], may be the caller's output), qsum (the per-head tail sums,
// [B][Hq][D]), hist ([B][Hkv][kSelHistBins] key counts), tws
// (select_topk_ws_bytes of top-k candidates and bitmaps), cm_ws (the column
// mass's scratch).
size_t select_topk_ws_bytes(int BH, int P);
hipError_t launch_select(const hyq_shape& s, const hyq_sizes& z, const uint16_t* Q,
                         const uint16_t* K, int32_t* idx, float* scores, float* qsum,
                         uint32_t* hist, uint32_t* tws, float* cm_ws, hipStream_t st);

// Column-mass scores (eq. vl_score) into scores[B][Hkv][P]; cm_ws holds
// colmass_ws_bytes(s) bytes of scratch.
size_t colmass_ws_bytes(const hyq_shape& s);
hipError_t launch_colmass_scores(const hyq_shape& s, const hyq_sizes& z, const uint16_t* Q,
                                 const uint16_t* K, float* scores, float* cm_ws, hipStream_t st);

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

// Building blocks of hyq_quantize, reused by the decode cache's Freeze:
// compaction of the non-vertical prefix into kq_pos (nslots slots per (b, j))
// and the K/V block quantization of n_blocks blocks, each (b, j) owning
// blk_stride blocks of the outputs.
void launch_compact(const int32_t* idx, int32_t* kq_pos, int k, int P, int nQ, int nslots,
                    int BHkv, hipStream_t st);
void launch_quant_kv(int bits, int fmt, const uint16_t* K, const uint16_t* V,
                     const int32_t* kq_pos, uint8_t* k_codes, float* k_scale, uint8_t* v_codes,
                     float* v_scale, int L, int nQ, int n_blocks, int blk_stride, int BHkv,
                     hipStream_t st);

// Decode: split of the sequence axis (quantized splits S_q, full-precision
// splits S_f, per KV head), workspace size, and the launches.
struct DecodeSplit {
  int nbq, S_q, S_f;   // quantized blocks; quantized and full-precision workgroups per KV head
};
constexpr int kDecodePartFloats = 132;   // one partial: acc[128], m, l, padding
DecodeSplit decode_split(const hyq_dcache& c);
size_t decode_ws_bytes(const hyq_dcache& c);
// Partials (bytes) that one decode attention launch writes for the cache's
// current state.
size_t decode_part_bytes(const hyq_dcache& c);
// Device address of the allocation-free call's scratch on the current device.
hipError_t noalloc_scratch(float** out);
hipError_t launch_freeze_gather(const hyq_dcache& c, int N, const uint16_t* K, const uint16_t* V,
                                hipStream_t st);
hipError_t launch_decode_append(const hyq_dcache& c, const uint16_t* k_new, const uint16_t* v_new,
                                bool merge, int slot, hipStream_t st);
hipError_t launch_decode_attn(const hyq_dcache& c, const uint16_t* q, float softmax_scale,
                              void* out, int out_dtype, float* part, hipStream_t st);

// ---- device helpers -------------------------------------------------------

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t b) {
  return __uint_as_float(b << 16);
}

// Low / high bf16 of a packed pair, widened exactly.
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

constexpr int kHeadDim = 128;
constexpr int kBlock = 64;
// Top-k key histogram: bins of the top kSelHistBits bits of the score order key.
constexpr int kSelHistBits = 12;
constexpr int kSelHistBins = 1 << kSelHistBits;

}  // namespace hyq
