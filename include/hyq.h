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
 *                        and window keys;
 *   hyq_prefill          the three in order, as one call.
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

/* Code formats of the quantized path (Algorithm 2 takes B in {INT8, FP8};
   Section 4.2 names INT4/FP4 for the low-precision bulk path as well). */
#define HYQ_FMT_INT 0   /* symmetric integer codes: int8 (c = 127) or int4 (c = 7) */
#define HYQ_FMT_FP8 1   /* OCP FP8 E4M3 codes (c = 448) for Q, K and V; needs
                           bits_kv = 8.  Each code byte is the E4M3 bit pattern of
                           the value nearest to x / s (ties to even, saturating at
                           +-448, zero keeps the sign of x), s = max|x| / 448.     */
#define HYQ_FMT_FP4 2   /* OCP FP4 E2M1 codes (c = 6) for K and V, needs bits_kv =
                           4: the code of x is the E2M1 value nearest to x / s
                           (ties to the even code, saturating at +-6, zero keeps
                           the sign of x), s = max|x| / 6; codes are packed two
                           per byte like int4 (element 2i in the low nibble).  Q
                           keeps 8 bits as E4M3 codes exactly as with
                           HYQ_FMT_FP8.                                          */
#define HYQ_FMT_FP4Q6 3 /* K and V exactly as HYQ_FMT_FP4 (bits_kv = 4); Q as OCP
                           FP6 E2M3 codes (c = 7.5), one per byte (bit 5 sign,
                           bits 4..3 exponent, bits 2..0 mantissa): the E2M3
                           value nearest to x / s, ties to the even code,
                           saturating at +-7.5, zero keeps the sign of x,
                           s = max|x| / 7.5 per 64-row block.  Both operands of
                           the quantized Q.K product are then at most 6 bits
                           wide.  Prefill calls only (decode queries stay bf16;
                           the decode cache rejects this format).             */

/* Readings of the full-precision window (eq. win_def of Section 4.1). */
#define HYQ_WIN_FIXED 0   /* the last W keys [L-W, L), as Algorithms 1, 2 and 4 use it */
#define HYQ_WIN_BAND  1   /* per query row t: keys [t+1-W, t] (eq. win_def with t0 = t+1);
                             quantizable keys older than the band are seen quantized.
                             Affects hyq_attn_prefill only (selection, quantization and
                             the decode cache use the fixed window).                  */

/* Vertical-line scores (Section 4.1). */
#define HYQ_SEL_PROXY   0   /* Algorithm 1: qsum . K, qsum the summed tail queries  */
#define HYQ_SEL_COLMASS 1   /* eq. vl_score: the attention mass the tail queries put
                               on each key (causal softmax, alpha = 1/sqrt(D), summed
                               over the tail rows and the g heads); same budget, top-k
                               and tie rule                                          */

typedef struct hyq_shape {
  int32_t B, Hq, Hkv, L, D;  /* batch, query heads, KV heads, sequence, head dim      */
  int32_t window;            /* W >= 0: full-precision window = last W keys          */
  int32_t budget_ppm;        /* vertical ratio r in parts per million, 0..1000000    */
  int32_t bits_kv;           /* 16 (no quantization), 8 (int8 / E4M3) or 4 (packed
                                int4 / E2M1), see kv_format                          */
  int32_t block;             /* quantization block in tokens (64)                   */
  int32_t kv_format;         /* HYQ_FMT_INT, HYQ_FMT_FP8 (bits 8), HYQ_FMT_FP4 or
                                HYQ_FMT_FP4Q6 (bits 4); ignored when bits = 16      */
  int32_t window_mode;       /* HYQ_WIN_FIXED or HYQ_WIN_BAND                       */
  int32_t selector;          /* HYQ_SEL_PROXY or HYQ_SEL_COLMASS                    */
  int32_t staging;           /* decode only: staging capacity W_s in tokens, 0 for
                                HYQ_DECODE_WS, else a multiple of 64 <= window      */
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
 * With selector = HYQ_SEL_COLMASS, S[b][j][p] is instead the column mass of
 * eq. vl_score: the sum over the tail rows i in [L-t, L) and the g heads of
 * group j of softmax_{k <= i}(alpha <Q[i], K[k]>)[p], computed with bf16
 * MFMA products and float32 exponentials and sums (not bit-reproducible
 * against another summation order; the top-k is the same kernel).
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
 *   c = 127 for Q and 8-bit K/V, c = 7 for 4-bit K/V; s = 0 gives codes 0
 *   (HYQ_FMT_INT; the floating-point formats round as described at
 *   HYQ_FMT_FP8 and HYQ_FMT_FP4, Q then in E4M3 with c = 448).
 * Layouts (all outputs written in full, padding included):
 *   q_codes int8 [B][Hq][L][D];           q_scale float [B][Hq][n_qblk]
 *   k_codes [B][Hkv][n_kvblk*64][row]:    8-bit: one code byte per channel;
 *            4-bit: byte i = channel 2i (low nibble) | channel 2i+1 (high
 *            nibble), two's-complement int4 or E2M1 nibbles;
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
 * With window_mode = HYQ_WIN_BAND the window of row t is [t+1-W, t]: a
 * quantizable key k is taken in full precision (as above) when t+1-W <= k
 * and quantized when k <= t - W; vertical lines and keys >= P as above.
 * alpha = softmax_scale (1/sqrt(D) for the paper's operator).
 * out: [B][Hq][L][D], float32 (out_dtype 0) or bf16 (out_dtype 1).
 * The quantization buffers (q_codes ... kq_pos) are the outputs of
 * hyq_quantize for the same shape; they are not read when bits_kv = 16.
 * Precision: quantized logits are exact int32 dot products scaled in
 * float32 (int codes) or the float32 results of the E4M3 / E2M1 x E4M3
 * MFMA; full-precision logits are bf16 x bf16 products accumulated in
 * float32; softmax weights enter the P.V products as f16, against exact
 * f16 codes (quantized keys) or against V / sVref in f16 (full-precision
 * keys: exact for bf16 V within 2^16 of the reference sVref, a power of two
 * the kernel raises when a tile's V exceeds that range); all accumulation is
 * float32.
 */
HYQ_API int hyq_attn_prefill(const hyq_shape* shape, const void* Q, const void* K, const void* V,
                     const int32_t* idx, const int8_t* q_codes, const float* q_scale,
                     const void* k_codes, const float* k_scale,
                     const void* v_codes, const float* v_scale,
                     const int32_t* kq_pos, float softmax_scale,
                     void* out, int32_t out_dtype, void* stream);

/* hyq_prefill - Algorithm 2 as one call: hyq_select_vertical (with no
 * scores output), hyq_quantize and hyq_attn_prefill on `stream`, in that
 * order.  Arguments, layouts, ownership and sizes are those of the three
 * calls (ws / ws_bytes: the selection workspace); the arguments of all
 * three are validated before the first launch, so an invalid argument
 * returns HYQ_EINVAL with nothing launched.  Allocates nothing and keeps no
 * state, so the call can be captured in a HIP graph.
 */
HYQ_API int hyq_prefill(const hyq_shape* shape, const void* Q, const void* K, const void* V,
                        int32_t* idx, int8_t* q_codes, float* q_scale, void* k_codes,
                        float* k_scale, void* v_codes, float* v_scale, int32_t* kq_pos,
                        float softmax_scale, void* out, int32_t out_dtype, void* ws,
                        size_t ws_bytes, void* stream);

/* ======================================================================
 * Decode: Algorithm 4 (Freeze, App. A.4) and Algorithm 3 (HyQuant Decode,
 * App. A.3).
 *
 * Freeze turns a prefill of N tokens into the hybrid KV cache of decode:
 *   - vertical-line tokens (Algorithm 1 on the prefill's tail queries, held
 *     fixed from then on): K and V kept in bf16;
 *   - the other non-window tokens [0, N-W) minus the vertical lines:
 *     per-block quantized exactly as hyq_quantize quantizes K_Q and V_Q;
 *   - the last W tokens (the window): kept in bf16;
 *   - an empty staging buffer of W_s tokens (shape.staging, default
 *     HYQ_DECODE_WS), kept in bf16.
 * Each decode step appends one token.  When it arrives with the staging
 * buffer full, the W_s oldest window tokens are first quantized into W_s/64
 * new blocks of the quantized prefix (same formula, c_B and format, 64
 * tokens per block, oldest first) and the staged tokens join the window,
 * which stays W tokens long.
 * Decode attention of one query row per (b, h) is one softmax over every
 * cached key (no mask): quantized keys enter as scale * code, all other
 * keys as their bf16 values; the query is used in full precision.
 *
 * Memory: the window and the staging buffer share one ring of
 * ring_rows = roundup(W, 64) + W_s bf16 rows per KV head (window = the W
 * oldest valid rows from ring_head on, staging = the rest), so a merge
 * moves no full-precision data.  Vertical-line rows and the ring are stored
 * together: fp_k row i < vl_rows is vertical line i (rows >= n_vl are zero
 * padding), row vl_rows + s is ring slot s.  fp_v holds the same rows
 * transposed (channel-major), the layout the P.V matrix product reads.
 * The caller owns every buffer; state lives in the struct, which
 * hyq_decode_append advances on the host.
 * ==================================================================== */

#define HYQ_DECODE_WS 64   /* default staging buffer capacity W_s (tokens)    */

typedef struct hyq_dcache {
  /* geometry, set by hyq_dcache_init */
  int32_t B, Hq, Hkv, D;
  int32_t window;        /* W, 64 <= W <= N                                      */
  int32_t bits_kv;       /* 8 or 4                                               */
  int32_t kv_format;     /* HYQ_FMT_INT, HYQ_FMT_FP8 (bits 8) or HYQ_FMT_FP4 (bits 4)*/
  int32_t n_vl;          /* k: vertical-line tokens per KV head                  */
  int32_t vl_rows;       /* k rounded up to a multiple of 64                     */
  int32_t ring_rows;     /* roundup(W, 64) + staging                             */
  int32_t n_frozen;      /* quantized tokens written by Freeze (nQ of the prefill)*/
  int32_t cap_blocks;    /* quantized blocks the buffers hold (Freeze + merges)  */
  /* state, set by hyq_freeze and advanced by hyq_decode_append */
  int32_t n_merged;      /* merged blocks, stored after the ceil(nQ/64) frozen ones */
  int32_t ring_head;     /* ring slot of the oldest window token                 */
  int32_t n_staged;      /* tokens in the staging buffer, 0..staging             */
  int32_t staging;       /* W_s: staging capacity, a multiple of 64, <= window   */
  int64_t t;             /* tokens cached: N + appended tokens                   */
  /* caller-owned device buffers (byte sizes from hyq_dcache_init) */
  void* k_codes;         /* [B][Hkv][cap_blocks*64][row] row-major, as hyq_quantize */
  void* v_codes;         /* [B][Hkv][cap_blocks][D][64*bits/8] channel-major blocks */
  float* k_scale;        /* [B][Hkv][cap_blocks]                                 */
  float* v_scale;        /* [B][Hkv][cap_blocks]                                 */
  int32_t* q_pos;        /* [B][Hkv][cap_blocks*64]: original position of each
                            quantized token; HYQ_KQ_POS_PAD in padding slots     */
  void* fp_k;            /* bf16 [B][Hkv][vl_rows + ring_rows][D]                */
  void* fp_v;            /* bf16 [B][Hkv][D][vl_rows + ring_rows]                */
  int32_t* vl_pos;       /* [B][Hkv][n_vl]: vertical-line positions, ascending   */
} hyq_dcache;

typedef struct hyq_dcache_sizes {
  size_t k_codes_bytes, v_codes_bytes, k_scale_bytes, v_scale_bytes, q_pos_bytes;
  size_t fp_k_bytes, fp_v_bytes, vl_pos_bytes;
  size_t freeze_ws_bytes;   /* workspace of hyq_freeze                              */
  size_t attn_ws_bytes;     /* workspace of hyq_decode_attn (any state of the cache)*/
} hyq_dcache_sizes;

/*
 * Pure host arithmetic: fills the geometry of a decode cache for a prefill
 * of shape `prefill` (L = N tokens; window, budget, bits and format as for
 * the prefill calls; bits_kv must be 8 or 4) that will hold up to
 * max_tokens tokens (>= N), zeroes its state and buffer pointers, and
 * returns the byte size of every buffer.
 * Errors: HYQ_EINVAL if W < W_s, N < W or max_tokens < N, or if
 * prefill->staging is neither 0 nor a multiple of 64.
 */
HYQ_API int hyq_dcache_init(const hyq_shape* prefill, int64_t max_tokens, hyq_dcache* cache,
                            hyq_dcache_sizes* sizes);

/*
 * Algorithm 4 (Freeze).  Q, K, V: the prefill's bf16 tensors (shape as for
 * the prefill calls); only the last min(W, N) query rows are read.  Fills
 * every buffer of `cache` (whose pointers the caller has set) and sets its
 * state: no merged blocks, ring_head 0, nothing staged, t = N.
 * ws: device workspace of at least freeze_ws_bytes (scratch).
 */
HYQ_API int hyq_freeze(const hyq_shape* prefill, const void* Q, const void* K, const void* V,
                       hyq_dcache* cache, void* ws, size_t ws_bytes, void* stream);

/*
 * One decode step's key and value rows, k_new and v_new bf16 [B][Hkv][D],
 * enter the staging buffer; when the staging buffer is full they are
 * preceded by the merge of the W_s oldest window tokens into quantized
 * blocks ceil(n_frozen/64) + n_merged, ... (W_s/64 of them).  Advances the state in
 * `cache` (host memory).
 * Errors: HYQ_EINVAL when a merge is due and all cap_blocks blocks are in
 * use (nothing is enqueued and the state is unchanged).
 */
HYQ_API int hyq_decode_append(hyq_dcache* cache, const void* k_new, const void* v_new,
                              void* stream);

/*
 * Algorithm 3: attention of one query row per (b, h) over every token of
 * the cache, split over the sequence axis and merged as in its
 * ReduceSoftmax step:
 *   out[b][h] = sum_k w_k value_k / sum_k w_k,  w_k = exp(z_k - max z),
 *   z_k = alpha * <q[b][h], key_k>, with key/value = scale * code for
 *   quantized tokens and the bf16 rows for vertical-line, window and staged
 *   tokens.  alpha = softmax_scale.
 * q: bf16 [B][Hq][D]; out: [B][Hq][D], float32 (out_dtype 0) or bf16 (1).
 * ws: device workspace of at least attn_ws_bytes (scratch).
 * Precision: the query enters the products with quantized keys as f16
 * after an exact power-of-two scaling per head (exact unless an entry is
 * below 2^-29 of the head's largest), codes as exact f16; full-precision
 * keys as bf16 x bf16; float32 accumulation; weights as f16 against
 * quantized values and as a high + low bf16 pair against bf16 values.
 */
HYQ_API int hyq_decode_attn(const hyq_dcache* cache, const void* q, float softmax_scale,
                            void* out, int32_t out_dtype, void* ws, size_t ws_bytes,
                            void* stream);

/*
 * hyq_decode_attn without a workspace, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, runtimes
 * that forbid hipMalloc): the same kernels and result, bit for bit, with
 * the split partials in a scratch array of HYQ_NOALLOC_SCRATCH_BYTES that
 * the library holds on each GPU (from its first use there until the process
 * ends).  Nothing is allocated by this call or by the library for it.
 * The scratch is shared by every call on a GPU: calls that overlap on one
 * GPU (different streams, or host threads without ordering) race and give
 * wrong results; calls ordered on one stream are fine.  The first call on
 * a device looks up the scratch's address (once per device, with that
 * device current), so make it outside graph capture.
 * Errors: as hyq_decode_attn; HYQ_EUNSUPPORTED when this launch's partials
 * (B * Hkv * splits * (Hq/Hkv) * 132 floats; about 9 MB for batch 16 at a
 * 32k-token cache) exceed the scratch.  Nothing is enqueued on error.
 */
#define HYQ_NOALLOC_SCRATCH_BYTES ((size_t)16 << 20)
HYQ_API int hyq_decode_attn_noalloc(const hyq_dcache* cache, const void* q, float softmax_scale,
                                    void* out, int32_t out_dtype, void* stream);

/* Static description of a return code. */
HYQ_API const char* hyq_strerror(int code);

/* Message of the last failing call on this thread ("" if none). */
HYQ_API const char* hyq_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* HYQ_H */
