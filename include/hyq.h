/*
 * hyq.h - C ABI of libhyq, the MI355X (gfx950) implementation of HyQuant's
 * hybrid-precision prefill attention (HyQuant, arxiv 2608.27875).
 *
 * The prefill operator is three calls, composed as Algorithm 2 (App. A.2):
 *
 *   hyq_select_vertical  Algorithm 1 (App. A.1): vertical-line key positions
 *                        of the non-window prefix, per KV head;
 *   hyq_quantize         Algorithm 2, Stages 1-2: partition of the keys and
 *                        per-block symmetric quantization of Q and of the
 *                        keys/values that are neither vertical lines nor in
 *                        the window;
 *   hyq_attn_prefill     Algorithm 2, Stage 3 / eq. (prefill_hybrid) of
 *                        Section 4.2: one causal online softmax over the
 *                        quantized keys and the full-precision vertical-line
 *                        and window keys.
 *
 * Conventions for every call:
 *  - Tensor pointers are DEVICE pointers owned by the caller.  Nothing is
 *    allocated, nothing is kept between calls, and nothing is read back to
 *    the host: every call only validates its arguments on the host and then
 *    enqueues kernels on `stream` (a hipStream_t; NULL = the null stream).
 *  - Q is [B][Hq][L][D], K and V are [B][Hkv][L][D], all bf16, contiguous.
 *    Query head h uses KV head h / (Hq/Hkv) (consecutive grouping).
 *  - The window is the last `window` keys [L-W, L); the prefix is [0, P) with
 *    P = max(0, L-W).  The vertical budget is k = 0 if budget_ppm = 0 or
 *    P = 0, else min(P, max(1, ceil(P * budget_ppm / 1e6))) (Algorithm 1).
 *  - Arguments are validated before anything is enqueued; on error nothing
 *    is enqueued, the call returns a negative code and hyq_last_error()
 *    describes the problem (thread-local).
 *  - Inputs must be finite.
 */
#ifndef HYQ_H
#define HYQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#if defined(__GNUC__)
#define HYQ_API __attribute__((visibility("default")))
#else
#define HYQ_API
#endif

/* Return codes. */
#define HYQ_OK            0
#define HYQ_EINVAL       -1   /* bad shape, pointer or argument combination          */
#define HYQ_EUNSUPPORTED -2   /* valid for the method but not built here (D != 128,
                                 block != 64, Hq/Hkv > 8, bits not in {16, 8, 4})   */
#define HYQ_EHIP         -3   /* a HIP launch or runtime error                      */

#define HYQ_KQ_POS_PAD 0x7fffffff   /* kq_pos value of padding slots */

/* Code formats of the quantized path (Algorithm 2 takes B in {INT8, FP8}). */
#define HYQ_FMT_INT 0   /* symmetric integer codes: int8 (c = 127) or int4 (c = 7) */
#define HYQ_FMT_FP8 1   /* OCP FP8 E4M3 codes (c = 448) for Q, K and V; needs
                           bits_kv = 8.  Each code byte is the E4M3 bit pattern of
                           the value nearest to x / s (ties to even, saturating at
                           +-448, zero keeps the sign of x), s = max|x| / 448.     */

typedef struct hyq_shape {
  int32_t B, Hq, Hkv, L, D;  /* batch, query heads, KV heads, sequence, head dim      */
  int32_t window;            /* W >= 0: full-precision window = last W keys          */
  int32_t budget_ppm;        /* vertical ratio r in parts per million, 0..1000000    */
  int32_t bits_kv;           /* 16 (no quantization), 8 (int8) or 4 (packed int4)   */
  int32_t block;             /* quantization block in tokens (64)                   */
  int32_t kv_format;         /* HYQ_FMT_INT or HYQ_FMT_FP8 (ignored when bits = 16) */
} hyq_shape;

typedef struct hyq_sizes {
  int32_t P;               /* non-window prefix length                               */
  int32_t k;               /* vertical lines per KV head                             */
  int32_t nQ;              /* quantized keys per KV head: P - k                      */
  int32_t n_qblk;          /* Q blocks per query head: ceil(L / block)               */
  int32_t n_kvblk;         /* K/V blocks per KV head: ceil(nQ / block)               */
  int32_t kv_row_bytes;    /* bytes per K code row: D (8-bit), D/2 (4-bit), 0 (16)   */
  size_t idx_bytes;        /* int32 idx[B][Hkv][k]                                   */
  size_t kq_pos_bytes;     /* int32 kq_pos[B][Hkv][n_kvblk*block]                    */
  size_t q_codes_bytes;    /* q_codes[B][Hq][L][D], one byte per code (int8 or E4M3) */
  size_t q_scale_bytes;    /* float q_scale[B][Hq][n_qblk]                           */
  size_t k_codes_bytes;    /* k_codes[B][Hkv][n_kvblk*block][kv_row_bytes]           */
  size_t v_codes_bytes;    /* v_codes[B][Hkv][n_kvblk][D][block*bits/8]              */
  size_t kv_scale_bytes;   /* float k_scale (and v_scale) [B][Hkv][n_kvblk]          */
  size_t scores_bytes;     /* float scores[B][Hkv][P]                                */
  size_t select_ws_bytes;  /* workspace needed by hyq_select_vertical                */
} hyq_sizes;

/* Pure host arithmetic: the derived sizes of a shape (same formulas as the
 * budget rule of Algorithm 1).  Validates the shape like the calls below.   */
HYQ_API int hyq_sizes_for(const hyq_shape* shape, hyq_sizes* out);

/*
 * Algorithm 1 (Vertical Token Identification), GQA-native, per KV head:
 *   qsum[b][j] = sum over the g query heads of group j and the last
 *                t = min(W, L) rows of Q (float32; per head, rows ascending
 *                from +0, then heads in order);
 *   S[b][j][p] = qsum . K[b][j][p] for p < P (float32 products, then the
 *                upper half of the 128 products folded onto the lower half
 *                repeatedly: 64, 32, ..., 1);
 *   idx[b][j]  = the k positions with the largest S, ties to the lowest
 *                position (-0 == +0), written in ascending order.
 * Q, K:    bf16 device tensors as above.
 * idx:     int32 [B][Hkv][k] (output).  Untouched when k = 0.
 * scores:  optional float [B][Hkv][P] output of S (NULL: not written).
 * ws:      device workspace of at least sizes.select_ws_bytes bytes (may be
 *          NULL when that is 0); its contents are scratch.
 * Errors:  HYQ_EINVAL also when W = 0 and k > 0 (no tail queries).
 */
HYQ_API int hyq_select_vertical(const hyq_shape* shape, const void* Q, const void* K,
                        int32_t* idx, float* scores, void* ws, size_t ws_bytes,
                        void* stream);

/*
 * Algorithm 2, Stages 1-2.  No-op (returns HYQ_OK) when bits_kv = 16.
 *   kq_pos[b][j][n]  the n-th quantized key position ([0, P) minus idx,
 *                    ascending); slots n >= nQ hold HYQ_KQ_POS_PAD.
 *   Q blocks:        rows [i*64, i*64+64) of each query head (ragged last);
 *   K/V blocks:      compacted rows [c*64, c*64+64) (K and V at kq_pos),
 *                    ragged last block; padding rows get code 0.
 *   scale s = fl32(max|x| / c), code = clamp(rint(fl32(x / s)), -c, c),
 *   c = 127 for Q and 8-bit K/V, c = 7 for 4-bit K/V; s = 0 gives codes 0.
 * Layouts (all outputs written in full, padding included):
 *   q_codes int8 [B][Hq][L][D];           q_scale float [B][Hq][n_qblk]
 *   k_codes [B][Hkv][n_kvblk*64][row]:    8-bit: int8 per channel;
 *            4-bit: byte i = channel 2i (low nibble) | channel 2i+1 (high
 *            nibble), two's-complement nibbles;
 *   v_codes [B][Hkv][n_kvblk][D][64*bits/8]: each block stored channel-major
 *            (transposed): row d lists the block's 64 keys; 4-bit: byte i =
 *            key 2i (low nibble) | key 2i+1 (high nibble);
 *   k_scale, v_scale float [B][Hkv][n_kvblk].
 * idx: the output of hyq_select_vertical (ignored when k = 0).
 */
HYQ_API int hyq_quantize(const hyq_shape* shape, const void* Q, const void* K, const void* V,
                 const int32_t* idx, int8_t* q_codes, float* q_scale,
                 void* k_codes, float* k_scale, void* v_codes, float* v_scale,
                 int32_t* kq_pos, void* stream);

/*
 * Algorithm 2, Stage 3 and eq. (prefill_hybrid), causal by original key
 * position:
 *   out[b][h][t] = sum_k w_k value_k / sum_k w_k over keys k <= t, with
 *   w_k = exp(z_k - max z), and
 *   - quantized key (position kq_pos[n], block c = n/64):
 *       z = alpha * q_scale[t/64] * k_scale[c] * <q_code[t], k_code[n]>,
 *       value = v_scale[c] * v_code[n];
 *   - vertical-line key (idx) or window key ([P, L)), and every key when
 *     bits_kv = 16:  z = alpha * <Q[t], K[k]>, value = V[k] (bf16 inputs).
 * alpha = softmax_scale (1/sqrt(D) for the paper's operator).
 * out: [B][Hq][L][D], float32 (out_dtype 0) or bf16 (out_dtype 1).
 * The quantization buffers (q_codes ... kq_pos) are the outputs of
 * hyq_quantize for the same shape; they are not read when bits_kv = 16.
 * Precision: quantized logits are exact int32 dot products scaled in
 * float32; full-precision logits are bf16 x bf16 products accumulated in
 * float32; softmax weights enter the P.V products as f16 (quantized keys,
 * against exact f16 codes) or as a high + low pair of bf16 (full-precision
 * keys, against bf16 V); all accumulation is float32.
 */
HYQ_API int hyq_attn_prefill(const hyq_shape* shape, const void* Q, const void* K, const void* V,
                     const int32_t* idx, const int8_t* q_codes, const float* q_scale,
                     const void* k_codes, const float* k_scale,
                     const void* v_codes, const float* v_scale,
                     const int32_t* kq_pos, float softmax_scale,
                     void* out, int32_t out_dtype, void* stream);

/* Static description of a return code. */
HYQ_API const char* hyq_strerror(int code);

/* Message of the last failing call on this thread ("" if none). */
HYQ_API const char* hyq_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* HYQ_H */
