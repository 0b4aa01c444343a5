// C ABI of libhyq: argument validation, derived sizes, error reporting, and
// the launches of the selection, quantization and attention kernels.
// Nothing here allocates device memory or reads device memory back.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include "hyq_internal.h"

namespace {

thread_local char g_err[512] = "";

int fail(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return code;
}

int ok() {
  g_err[0] = '\0';
  return HYQ_OK;
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Shape checks shared by every entry point, then the derived sizes
// (Algorithm 1: P = max(0, L - W); k = min(P, max(1, ceil(P r))), 0 if r = 0
// or P = 0).
int check_shape(const hyq_shape* s, hyq_sizes* z) {
  if (!s) return fail(HYQ_EINVAL, "shape is NULL");
  if (s->B < 1 || s->Hq < 1 || s->Hkv < 1 || s->L < 1 || s->D < 1)
    return fail(HYQ_EINVAL, "B, Hq, Hkv, L, D must be >= 1 (got %d, %d, %d, %d, %d)", s->B,
                s->Hq, s->Hkv, s->L, s->D);
  if (s->Hq % s->Hkv) return fail(HYQ_EINVAL, "Hq (%d) must be a multiple of Hkv (%d)", s->Hq, s->Hkv);
  if (s->window < 0) return fail(HYQ_EINVAL, "window must be >= 0 (got %d)", s->window);
  if (s->budget_ppm < 0 || s->budget_ppm > 1000000)
    return fail(HYQ_EINVAL, "budget_ppm must be in [0, 1000000] (got %d)", s->budget_ppm);
  if (s->block < 1) return fail(HYQ_EINVAL, "block must be >= 1 (got %d)", s->block);
  if (s->bits_kv != 16 && s->bits_kv != 8 && s->bits_kv != 4)
    return fail(HYQ_EUNSUPPORTED, "bits_kv must be 16, 8 or 4 (got %d)", s->bits_kv);
  if (s->kv_format != HYQ_FMT_INT && s->kv_format != HYQ_FMT_FP8 && s->kv_format != HYQ_FMT_FP4 &&
      s->kv_format != HYQ_FMT_FP4Q6)
    return fail(HYQ_EINVAL,
                "kv_format must be HYQ_FMT_INT, HYQ_FMT_FP8, HYQ_FMT_FP4 or HYQ_FMT_FP4Q6 (got %d)",
                s->kv_format);
  if (s->kv_format == HYQ_FMT_FP8 && s->bits_kv == 4)
    return fail(HYQ_EINVAL, "FP8 codes need bits_kv = 8 (got 4)");
  if ((s->kv_format == HYQ_FMT_FP4 || s->kv_format == HYQ_FMT_FP4Q6) && s->bits_kv == 8)
    return fail(HYQ_EINVAL, "FP4 codes need bits_kv = 4 (got 8)");
  if (s->selector != HYQ_SEL_PROXY && s->selector != HYQ_SEL_COLMASS)
    return fail(HYQ_EINVAL, "selector must be HYQ_SEL_PROXY or HYQ_SEL_COLMASS (got %d)",
                s->selector);
  if (s->staging != 0 && (s->staging < 64 || s->staging % 64))
    return fail(HYQ_EINVAL, "staging must be 0 or a positive multiple of 64 (got %d)", s->staging);
  if (s->window_mode != HYQ_WIN_FIXED && s->window_mode != HYQ_WIN_BAND)
    return fail(HYQ_EINVAL, "window_mode must be HYQ_WIN_FIXED or HYQ_WIN_BAND (got %d)",
                s->window_mode);
  if (s->D != hyq::kHeadDim)
    return fail(HYQ_EUNSUPPORTED, "head dim %d not supported (only %d)", s->D, hyq::kHeadDim);
  if (s->block != hyq::kBlock)
    return fail(HYQ_EUNSUPPORTED, "block %d not supported (only %d)", s->block, hyq::kBlock);
  if (s->Hq / s->Hkv > 8)
    return fail(HYQ_EUNSUPPORTED, "GQA group size %d not supported (at most 8)", s->Hq / s->Hkv);
  // 32-bit element offsets inside one head; whole tensors use 64-bit offsets
  if ((int64_t)s->L * s->D > (int64_t)1 << 30)
    return fail(HYQ_EUNSUPPORTED, "sequence length %d too long", s->L);

  const int64_t L = s->L, W = s->window;
  const int64_t P = L > W ? L - W : 0;
  int64_t k = 0;
  if (s->budget_ppm > 0 && P > 0) {
    k = (P * s->budget_ppm + 999999) / 1000000;
    if (k < 1) k = 1;
    if (k > P) k = P;
  }
  if (k > 0 && (W < L ? W : L) < 1)
    return fail(HYQ_EINVAL, "a vertical budget needs window >= 1 (the tail-query proxy averages "
                            "the last min(W, L) queries)");
  const int64_t nQ = P - k;
  const int64_t bs = s->block;
  memset(z, 0, sizeof *z);
  z->P = (int32_t)P;
  z->k = (int32_t)k;
  z->nQ = (int32_t)nQ;
  z->n_qblk = (int32_t)((L + bs - 1) / bs);
  z->n_kvblk = (int32_t)((nQ + bs - 1) / bs);
  const size_t B = s->B, Hq = s->Hq, Hkv = s->Hkv, D = s->D;
  const size_t slots = (size_t)z->n_kvblk * bs;
  const bool quant = s->bits_kv != 16;
  z->kv_row_bytes = !quant ? 0 : (s->bits_kv == 8 ? (int32_t)D : (int32_t)D / 2);
  z->idx_bytes = B * Hkv * (size_t)k * 4;
  z->scores_bytes = B * Hkv * (size_t)P * 4;
  if (quant) {
    z->kq_pos_bytes = B * Hkv * slots * 4;
    z->q_codes_bytes = B * Hq * (size_t)L * D;
    z->q_scale_bytes = B * Hq * (size_t)z->n_qblk * 4;
    z->k_codes_bytes = B * Hkv * slots * z->kv_row_bytes;
    z->v_codes_bytes = B * Hkv * (size_t)z->n_kvblk * D * (size_t)(bs * s->bits_kv / 8);
    z->kv_scale_bytes = B * Hkv * (size_t)z->n_kvblk * 4;
  }
  z->select_ws_bytes = k > 0 ? align256(B * Hq * D * 4) + align256(z->scores_bytes) +
                                   align256(B * Hkv * hyq::kSelHistBins * 4) +
                                   align256(hyq::select_topk_ws_bytes((int)(B * Hkv), (int)P)) +
                                   (s->selector == HYQ_SEL_COLMASS
                                        ? align256(hyq::colmass_ws_bytes(*s)) : 0)
                             : 0;
  return HYQ_OK;
}

// The selection workspace: per-head tail sums [B][Hq][D], the scores
// [B][Hkv][P] (unused when the caller passes its own), the top-k key
// histogram, the top-k candidates and bitmaps, the column mass's scratch.
struct SelectWs {
  float* qsum;
  float* scores;
  uint32_t* hist;
  uint32_t* tws;
  float* cm;
};
SelectWs select_ws(const hyq_shape& s, const hyq_sizes& z, void* ws, float* scores_out) {
  char* p = static_cast<char*>(ws);
  SelectWs r;
  r.qsum = reinterpret_cast<float*>(p);
  p += align256((size_t)s.B * s.Hq * s.D * 4);
  r.scores = scores_out ? scores_out : reinterpret_cast<float*>(p);
  p += align256(z.scores_bytes);
  r.hist = reinterpret_cast<uint32_t*>(p);
  p += align256((size_t)s.B * s.Hkv * hyq::kSelHistBins * 4);
  r.tws = reinterpret_cast<uint32_t*>(p);
  p += align256(hyq::select_topk_ws_bytes(s.B * s.Hkv, z.P));
  r.cm = reinterpret_cast<float*>(p);
  return r;
}

int64_t round_up64(int64_t x) { return (x + 63) / 64 * 64; }

// Geometry of the decode cache of a prefill shape (Algorithm 4's buffers);
// state zeroed, pointers NULL.
int dcache_geometry(const hyq_shape* s, int64_t max_tokens, hyq_dcache* c, hyq_dcache_sizes* out) {
  hyq_sizes z;
  int rc = check_shape(s, &z);
  if (rc) return rc;
  if (s->bits_kv == 16)
    return fail(HYQ_EINVAL, "the decode cache needs a quantized format (bits_kv 8 or 4)");
  if (s->kv_format == HYQ_FMT_FP4Q6)
    return fail(HYQ_EINVAL, "decode keeps its queries in bf16: use HYQ_FMT_FP4 for the cache "
                            "(HYQ_FMT_FP4Q6 sets the prefill's query codes)");
  const int32_t ws = s->staging ? s->staging : HYQ_DECODE_WS;
  if (s->window < ws)
    return fail(HYQ_EINVAL, "decode needs window >= the staging capacity %d (a merge moves that "
                "many window tokens), got %d", ws, s->window);
  if (s->L < s->window)
    return fail(HYQ_EINVAL, "decode needs a prefill of at least window tokens (L = %d < W = %d)",
                s->L, s->window);
  if (max_tokens < s->L || max_tokens > (int64_t)0x7fffffff)
    return fail(HYQ_EINVAL, "max_tokens must be in [L, 2^31 - 1] (got %lld)",
                (long long)max_tokens);
  memset(c, 0, sizeof *c);
  c->B = s->B;
  c->Hq = s->Hq;
  c->Hkv = s->Hkv;
  c->D = s->D;
  c->window = s->window;
  c->bits_kv = s->bits_kv;
  c->kv_format = s->kv_format;
  c->n_vl = z.k;
  c->vl_rows = (int32_t)round_up64(z.k);
  c->ring_rows = (int32_t)(round_up64(s->window) + ws);
  c->staging = ws;
  c->n_frozen = z.nQ;
  const int64_t nbf = (z.nQ + 63) / 64;
  const int64_t merges = (max_tokens - s->L + HYQ_DECODE_WS - 1) / HYQ_DECODE_WS;
  if (nbf + merges > (int64_t)1 << 24) return fail(HYQ_EUNSUPPORTED, "cache too long");
  c->cap_blocks = (int32_t)(nbf + merges);
  c->t = s->L;
  if (out) {
    const size_t BH = (size_t)s->B * s->Hkv, D = s->D, cap = c->cap_blocks;
    const size_t row = s->bits_kv == 8 ? D : D / 2;
    const size_t nfp = (size_t)c->vl_rows + c->ring_rows;
    memset(out, 0, sizeof *out);
    out->k_codes_bytes = BH * cap * 64 * row;
    out->v_codes_bytes = BH * cap * D * (64 * s->bits_kv / 8);
    out->k_scale_bytes = out->v_scale_bytes = BH * cap * 4;
    out->q_pos_bytes = BH * cap * 64 * 4;
    out->fp_k_bytes = out->fp_v_bytes = BH * nfp * D * 2;
    out->vl_pos_bytes = BH * (size_t)z.k * 4;
    out->freeze_ws_bytes = z.select_ws_bytes;
    out->attn_ws_bytes = hyq::decode_ws_bytes(*c);
  }
  return HYQ_OK;
}

// Consistency of a cache struct (geometry as dcache_geometry makes it, state
// in range, buffers present).
int check_dcache(const hyq_dcache* c) {
  if (!c) return fail(HYQ_EINVAL, "cache is NULL");
  if (c->B < 1 || c->Hq < 1 || c->Hkv < 1 || c->Hq % c->Hkv || c->Hq / c->Hkv > 8 ||
      c->D != hyq::kHeadDim)
    return fail(HYQ_EINVAL, "cache geometry is invalid (B, Hq, Hkv, D)");
  if ((c->bits_kv != 8 && c->bits_kv != 4) ||
      (c->kv_format != HYQ_FMT_INT && c->kv_format != HYQ_FMT_FP8 && c->kv_format != HYQ_FMT_FP4) ||
      (c->kv_format == HYQ_FMT_FP8 && c->bits_kv != 8) ||
      (c->kv_format == HYQ_FMT_FP4 && c->bits_kv != 4))
    return fail(HYQ_EINVAL, "cache format is invalid (bits_kv %d, kv_format %d)", c->bits_kv,
                c->kv_format);
  if (c->staging < 64 || c->staging % 64 || c->window < c->staging || c->n_vl < 0 ||
      c->vl_rows != round_up64(c->n_vl) || c->ring_rows != round_up64(c->window) + c->staging ||
      c->n_frozen < 0)
    return fail(HYQ_EINVAL, "cache geometry is invalid (window, staging, n_vl, vl_rows, ring_rows)");
  const int64_t nbf = (c->n_frozen + 63) / 64;
  if (c->n_merged < 0 || nbf + c->n_merged > c->cap_blocks || c->n_staged < 0 ||
      c->n_staged > c->staging || c->ring_head < 0 || c->ring_head >= c->ring_rows ||
      c->ring_head % 64 != 0 || c->t < (int64_t)c->window)
    return fail(HYQ_EINVAL, "cache state is invalid (n_merged %d, n_staged %d, ring_head %d)",
                c->n_merged, c->n_staged, c->ring_head);
  if (!c->fp_k || !c->fp_v) return fail(HYQ_EINVAL, "fp_k and fp_v must be non-NULL");
  if (c->cap_blocks > 0 &&
      (!c->k_codes || !c->v_codes || !c->k_scale || !c->v_scale || !c->q_pos))
    return fail(HYQ_EINVAL, "k_codes, v_codes, k_scale, v_scale and q_pos must be non-NULL");
  if (c->n_vl > 0 && !c->vl_pos) return fail(HYQ_EINVAL, "vl_pos must be non-NULL when n_vl > 0");
  return HYQ_OK;
}

// Arguments shared by the two decode attention calls.
int check_decode_attn(const hyq_dcache* cache, const void* q, float softmax_scale, void* out,
                      int32_t out_dtype) {
  const int rc = check_dcache(cache);
  if (rc) return rc;
  if (!q || !out) return fail(HYQ_EINVAL, "q and out must be non-NULL");
  if (out_dtype != 0 && out_dtype != 1)
    return fail(HYQ_EINVAL, "out_dtype must be 0 (float32) or 1 (bf16), got %d", out_dtype);
  if (!(softmax_scale > 0.0f) || softmax_scale == INFINITY)
    return fail(HYQ_EINVAL, "softmax_scale must be positive and finite");
  return HYQ_OK;
}

int hip_status(hipError_t e, const char* what) {
  if (e != hipSuccess) return fail(HYQ_EHIP, "%s: %s", what, hipGetErrorString(e));
  return ok();
}

}  // namespace

extern "C" {

HYQ_API const char* hyq_strerror(int code) {
  switch (code) {
    case HYQ_OK: return "success";
    case HYQ_EINVAL: return "invalid argument";
    case HYQ_EUNSUPPORTED: return "unsupported configuration";
    case HYQ_EHIP: return "HIP runtime error";
    default: return "unknown error";
  }
}

HYQ_API const char* hyq_last_error(void) { return g_err; }

HYQ_API int hyq_sizes_for(const hyq_shape* shape, hyq_sizes* out) {
  if (!out) return fail(HYQ_EINVAL, "sizes output is NULL");
  hyq_sizes z;
  const int rc = check_shape(shape, &z);
  if (rc) return rc;
  *out = z;
  return ok();
}

// Argument checks of the three prefill calls (after check_shape), shared by
// the calls themselves and by hyq_prefill, which runs all three before it
// launches anything.
static int check_select_args(const hyq_sizes& z, const void* Q, const void* K, const int32_t* idx,
                             const void* ws, size_t ws_bytes) {
  if (z.k == 0) return ok();
  if (!Q || !K || !idx) return fail(HYQ_EINVAL, "Q, K and idx must be non-NULL");
  if (!ws || ws_bytes < z.select_ws_bytes)
    return fail(HYQ_EINVAL, "workspace too small: %zu bytes given, %zu needed", ws_bytes,
                z.select_ws_bytes);
  return ok();
}

static int check_quantize_args(const hyq_shape* shape, const hyq_sizes& z, const void* Q,
                               const void* K, const void* V, const int32_t* idx,
                               const void* q_codes, const void* q_scale, const void* k_codes,
                               const void* k_scale, const void* v_codes, const void* v_scale,
                               const void* kq_pos) {
  if (shape->bits_kv == 16) return ok();
  if (!Q || !K || !V || !q_codes || !q_scale)
    return fail(HYQ_EINVAL, "Q, K, V, q_codes and q_scale must be non-NULL");
  if (z.k > 0 && !idx) return fail(HYQ_EINVAL, "idx must be non-NULL when k > 0");
  if (z.n_kvblk > 0 && (!k_codes || !k_scale || !v_codes || !v_scale || !kq_pos))
    return fail(HYQ_EINVAL,
                "k_codes, k_scale, v_codes, v_scale and kq_pos must be non-NULL when nQ > 0");
  return ok();
}

static int check_attn_args(const hyq_shape* shape, const hyq_sizes& z, const void* Q,
                           const void* K, const void* V, const int32_t* idx, const void* q_codes,
                           const void* q_scale, const void* k_codes, const void* k_scale,
                           const void* v_codes, const void* v_scale, const void* kq_pos,
                           float softmax_scale, const void* out, int32_t out_dtype) {
  if (!Q || !K || !V || !out) return fail(HYQ_EINVAL, "Q, K, V and out must be non-NULL");
  if (out_dtype != 0 && out_dtype != 1)
    return fail(HYQ_EINVAL, "out_dtype must be 0 (float32) or 1 (bf16), got %d", out_dtype);
  if (!(softmax_scale > 0.0f) || softmax_scale == INFINITY)
    return fail(HYQ_EINVAL, "softmax_scale must be positive and finite");
  if (shape->bits_kv != 16) {
    if (z.k > 0 && !idx) return fail(HYQ_EINVAL, "idx must be non-NULL when k > 0");
    if (!q_codes || !q_scale) return fail(HYQ_EINVAL, "q_codes and q_scale must be non-NULL");
    if (z.n_kvblk > 0 && (!k_codes || !k_scale || !v_codes || !v_scale || !kq_pos))
      return fail(HYQ_EINVAL,
                  "k_codes, k_scale, v_codes, v_scale and kq_pos must be non-NULL when nQ > 0");
  }
  return ok();
}

HYQ_API int hyq_select_vertical(const hyq_shape* shape, const void* Q, const void* K, int32_t* idx,
                        float* scores, void* ws, size_t ws_bytes, void* stream) {
  hyq_sizes z;
  int rc = check_shape(shape, &z);
  if (rc) return rc;
  if (z.k == 0) return ok();
  if ((rc = check_select_args(z, Q, K, idx, ws, ws_bytes))) return rc;
  const SelectWs w = select_ws(*shape, z, ws, scores);
  return hip_status(hyq::launch_select(*shape, z, static_cast<const uint16_t*>(Q),
                                       static_cast<const uint16_t*>(K), idx, w.scores, w.qsum,
                                       w.hist, w.tws, w.cm, static_cast<hipStream_t>(stream)),
                    "hyq_select_vertical launch");
}

HYQ_API int hyq_quantize(const hyq_shape* shape, const void* Q, const void* K, const void* V,
                 const int32_t* idx, int8_t* q_codes, float* q_scale, void* k_codes,
                 float* k_scale, void* v_codes, float* v_scale, int32_t* kq_pos, void* stream) {
  hyq_sizes z;
  int rc = check_shape(shape, &z);
  if (rc) return rc;
  if (shape->bits_kv == 16) return ok();
  if ((rc = check_quantize_args(shape, z, Q, K, V, idx, q_codes, q_scale, k_codes, k_scale,
                                v_codes, v_scale, kq_pos)))
    return rc;
  return hip_status(
      hyq::launch_quantize(*shape, z, static_cast<const uint16_t*>(Q),
                           static_cast<const uint16_t*>(K), static_cast<const uint16_t*>(V), idx,
                           q_codes, q_scale, static_cast<uint8_t*>(k_codes), k_scale,
                           static_cast<uint8_t*>(v_codes), v_scale, kq_pos,
                           static_cast<hipStream_t>(stream)),
      "hyq_quantize launch");
}

HYQ_API int hyq_attn_prefill(const hyq_shape* shape, const void* Q, const void* K, const void* V,
                     const int32_t* idx, const int8_t* q_codes, const float* q_scale,
                     const void* k_codes, const float* k_scale, const void* v_codes,
                     const float* v_scale, const int32_t* kq_pos, float softmax_scale,
                     void* out, int32_t out_dtype, void* stream) {
  hyq_sizes z;
  int rc = check_shape(shape, &z);
  if (rc) return rc;
  if ((rc = check_attn_args(shape, z, Q, K, V, idx, q_codes, q_scale, k_codes, k_scale, v_codes,
                            v_scale, kq_pos, softmax_scale, out, out_dtype)))
    return rc;
  return hip_status(
      hyq::launch_attn_prefill(
          *shape, z, static_cast<const uint16_t*>(Q), static_cast<const uint16_t*>(K),
          static_cast<const uint16_t*>(V), idx, q_codes, q_scale,
          static_cast<const uint8_t*>(k_codes), k_scale, static_cast<const uint8_t*>(v_codes),
          v_scale, kq_pos, softmax_scale, out, out_dtype, static_cast<hipStream_t>(stream)),
      "hyq_attn_prefill launch");
}

HYQ_API int hyq_prefill(const hyq_shape* shape, const void* Q, const void* K, const void* V,
                        int32_t* idx, int8_t* q_codes, float* q_scale, void* k_codes,
                        float* k_scale, void* v_codes, float* v_scale, int32_t* kq_pos,
                        float softmax_scale, void* out, int32_t out_dtype, void* ws,
                        size_t ws_bytes, void* stream) {
  hyq_sizes z;
  int rc = check_shape(shape, &z);
  if (rc) return rc;
  if ((rc = check_select_args(z, Q, K, idx, ws, ws_bytes))) return rc;
  if ((rc = check_quantize_args(shape, z, Q, K, V, idx, q_codes, q_scale, k_codes, k_scale,
                                v_codes, v_scale, kq_pos)))
    return rc;
  if ((rc = check_attn_args(shape, z, Q, K, V, idx, q_codes, q_scale, k_codes, k_scale, v_codes,
                            v_scale, kq_pos, softmax_scale, out, out_dtype)))
    return rc;
  if ((rc = hyq_select_vertical(shape, Q, K, idx, nullptr, ws, ws_bytes, stream))) return rc;
  if ((rc = hyq_quantize(shape, Q, K, V, idx, q_codes, q_scale, k_codes, k_scale, v_codes,
                         v_scale, kq_pos, stream)))
    return rc;
  return hyq_attn_prefill(shape, Q, K, V, idx, q_codes, q_scale, k_codes, k_scale, v_codes,
                          v_scale, kq_pos, softmax_scale, out, out_dtype, stream);
}

HYQ_API int hyq_dcache_init(const hyq_shape* prefill, int64_t max_tokens, hyq_dcache* cache,
                            hyq_dcache_sizes* sizes) {
  if (!cache) return fail(HYQ_EINVAL, "cache is NULL");
  hyq_dcache c;
  hyq_dcache_sizes z;
  const int rc = dcache_geometry(prefill, max_tokens, &c, &z);
  if (rc) return rc;
  *cache = c;
  if (sizes) *sizes = z;
  return ok();
}

HYQ_API int hyq_freeze(const hyq_shape* prefill, const void* Q, const void* K, const void* V,
                       hyq_dcache* cache, void* ws, size_t ws_bytes, void* stream) {
  hyq_sizes z;
  int rc = check_shape(prefill, &z);
  if (rc) return rc;
  rc = check_dcache(cache);
  if (rc) return rc;
  if (!Q || !K || !V) return fail(HYQ_EINVAL, "Q, K and V must be non-NULL");
  hyq_dcache ref;
  hyq_dcache_sizes rz;
  rc = dcache_geometry(prefill, prefill->L, &ref, &rz);
  if (rc) return rc;
  if (ref.B != cache->B || ref.Hq != cache->Hq || ref.Hkv != cache->Hkv ||
      ref.window != cache->window || ref.bits_kv != cache->bits_kv ||
      ref.kv_format != cache->kv_format || ref.n_vl != cache->n_vl ||
      ref.staging != cache->staging ||
      ref.n_frozen != cache->n_frozen || cache->cap_blocks < (ref.n_frozen + 63) / 64)
    return fail(HYQ_EINVAL, "cache geometry does not match the prefill shape");
  if (rz.freeze_ws_bytes > 0 && (!ws || ws_bytes < rz.freeze_ws_bytes))
    return fail(HYQ_EINVAL, "workspace too small: %zu bytes given, %zu needed", ws_bytes,
                rz.freeze_ws_bytes);
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int BHkv = prefill->B * prefill->Hkv;
  if (z.k > 0) {
    const SelectWs w = select_ws(*prefill, z, ws, nullptr);
    hipError_t e = hyq::launch_select(*prefill, z, static_cast<const uint16_t*>(Q),
                                      static_cast<const uint16_t*>(K), cache->vl_pos, w.scores,
                                      w.qsum, w.hist, w.tws, w.cm, st);
    if (e != hipSuccess) return hip_status(e, "hyq_freeze selection launch");
  }
  if (cache->cap_blocks > 0) {
    hyq::launch_compact(cache->vl_pos, cache->q_pos, z.k, z.P, z.nQ, cache->cap_blocks * 64,
                        BHkv, st);
    hyq::launch_quant_kv(prefill->bits_kv, prefill->kv_format, static_cast<const uint16_t*>(K),
                         static_cast<const uint16_t*>(V), cache->q_pos,
                         static_cast<uint8_t*>(cache->k_codes), cache->k_scale,
                         static_cast<uint8_t*>(cache->v_codes), cache->v_scale, prefill->L, z.nQ,
                         z.n_kvblk, cache->cap_blocks, BHkv, st);
  }
  const hipError_t e = hyq::launch_freeze_gather(*cache, prefill->L,
                                                 static_cast<const uint16_t*>(K),
                                                 static_cast<const uint16_t*>(V), st);
  if (e != hipSuccess) return hip_status(e, "hyq_freeze launch");
  cache->n_merged = 0;
  cache->ring_head = 0;
  cache->n_staged = 0;
  cache->t = prefill->L;
  return ok();
}

HYQ_API int hyq_decode_append(hyq_dcache* cache, const void* k_new, const void* v_new,
                              void* stream) {
  const int rc = check_dcache(cache);
  if (rc) return rc;
  if (!k_new || !v_new) return fail(HYQ_EINVAL, "k_new and v_new must be non-NULL");
  const bool merge = cache->n_staged == cache->staging;
  const int nbf = (cache->n_frozen + 63) / 64, nb_merge = cache->staging / 64;
  if (merge && nbf + cache->n_merged + nb_merge > cache->cap_blocks)
    return fail(HYQ_EINVAL, "decode cache full: all %d quantized blocks are in use",
                cache->cap_blocks);
  if (cache->t >= (int64_t)0x7fffffff) return fail(HYQ_EINVAL, "decode cache full (positions)");
  const int head = merge ? (cache->ring_head + cache->staging) % cache->ring_rows : cache->ring_head;
  const int staged = merge ? 0 : cache->n_staged;
  const int slot = (head + cache->window + staged) % cache->ring_rows;
  const hipError_t e = hyq::launch_decode_append(*cache, static_cast<const uint16_t*>(k_new),
                                                 static_cast<const uint16_t*>(v_new), merge, slot,
                                                 static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_status(e, "hyq_decode_append launch");
  if (merge) cache->n_merged += nb_merge;
  cache->ring_head = head;
  cache->n_staged = staged + 1;
  cache->t += 1;
  return ok();
}

HYQ_API int hyq_decode_attn(const hyq_dcache* cache, const void* q, float softmax_scale,
                            void* out, int32_t out_dtype, void* ws, size_t ws_bytes,
                            void* stream) {
  int rc = check_decode_attn(cache, q, softmax_scale, out, out_dtype);
  if (rc) return rc;
  const size_t need = hyq::decode_ws_bytes(*cache);
  if (!ws || ws_bytes < need)
    return fail(HYQ_EINVAL, "workspace too small: %zu bytes given, %zu needed", ws_bytes, need);
  // the partials this launch writes (never more than `need`; checked so that
  // a launch can never write past the workspace)
  const size_t used = hyq::decode_part_bytes(*cache);
  if (used > ws_bytes)
    return fail(HYQ_EINVAL, "workspace too small for this launch: %zu bytes given, %zu used",
                ws_bytes, used);
  return hip_status(hyq::launch_decode_attn(*cache, static_cast<const uint16_t*>(q), softmax_scale,
                                            out, out_dtype, static_cast<float*>(ws),
                                            static_cast<hipStream_t>(stream)),
                    "hyq_decode_attn launch");
}

HYQ_API int hyq_decode_attn_noalloc(const hyq_dcache* cache, const void* q, float softmax_scale,
                                    void* out, int32_t out_dtype, void* stream) {
  int rc = check_decode_attn(cache, q, softmax_scale, out, out_dtype);
  if (rc) return rc;
  const size_t used = hyq::decode_part_bytes(*cache);
  if (used > HYQ_NOALLOC_SCRATCH_BYTES)
    return fail(HYQ_EUNSUPPORTED,
                "this decode launch needs %zu bytes of scratch, more than the %zu bytes the "
                "allocation-free call holds; use hyq_decode_attn with a workspace",
                used, (size_t)HYQ_NOALLOC_SCRATCH_BYTES);
  float* part = nullptr;
  const hipError_t e = hyq::noalloc_scratch(&part);
  if (e != hipSuccess) return hip_status(e, "hyq_decode_attn_noalloc scratch lookup");
  return hip_status(hyq::launch_decode_attn(*cache, static_cast<const uint16_t*>(q), softmax_scale,
                                            out, out_dtype, part, static_cast<hipStream_t>(stream)),
                    "hyq_decode_attn_noalloc launch");
}

}  // extern "C"
