// Decode path of HyQuant (Section 4.3): Freeze (Algorithm 4, App. A.4), the
// staging buffer and its merges into the quantized prefix, and the decode
// attention of Algorithm 3 (App. A.3): the quantized prefix split along the
// sequence axis, every split an online softmax, the splits and the
// full-precision segments merged by ReduceSoftmax.
//
// Decode attention is bound by HBM bandwidth: every cached byte is read once
// per step and each key meets only g = Hq/Hkv query rows.  The kernel is laid
// out so that each byte goes from HBM straight into an MFMA operand register
// with no LDS round trip:
//   - one wave owns whole 64-token units (a quantization block, or a tile of
//     64 full-precision rows) and keeps its own online-softmax state;
//   - S^T = K q^T with the 16x16x32 MFMA (keys as rows, the g heads of the
//     KV group as columns, padded to 16): the A operand is read directly from
//     the row-major K codes (one 16-byte load per lane and 16 keys);
//   - the accumulator layout of S^T (lane l: head l%16, keys
//     (l/16)*16 + 4t + r of the unit for tile t, register r) is exactly the
//     B operand layout of O^T = V^T P^T, and the channel-major V codes of a
//     block are exactly its A operand, so P never leaves registers and V is
//     never transposed on chip;
//   - quantized codes become exact f16 MFMA operands (codes_dev.h); the
//     query enters as f16 after an exact power-of-two scaling per head;
//     full-precision tiles use the bf16 MFMA with P as a high + low bf16
//     pair.
// A workgroup (4 waves) merges its waves' states in LDS and writes one
// partial (m, l, acc) per query head; a second kernel reduces the partials.
#include "codes_dev.h"
#include "decode_split.h"

#include <mutex>
#include "hyq_internal.h"
#include "quant_dev.h"

#include <algorithm>
#include <atomic>
#include <type_traits>

namespace hyq {
namespace {

typedef _Float16 v8h __attribute__((ext_vector_type(8)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef unsigned v4u __attribute__((ext_vector_type(4)));
typedef unsigned v2u __attribute__((ext_vector_type(2)));

constexpr int kDecWaves = kDecodeWaves;
static_assert(kBlock == 64 && kHeadDim == 128, "decode_shape_for assumes 64-token blocks, D = 128");
constexpr int kDecThreads = kDecWaves * 64;
constexpr int kPartStride = kDecodePartFloats;
constexpr float kLazyD = 8.0f;             // rescale only when the max grows by > 2^8
constexpr float kMinusBigD = -1.0e30f;
constexpr int kMaxGroup = 8;

// ---------------------------------------------------------------------------
// Freeze: gather the vertical-line rows and the window into the bf16 rows of
// the cache (K row-major, V channel-major); every other row is zeroed.
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(256)
freeze_gather_kernel(const uint16_t* __restrict__ K, const uint16_t* __restrict__ V,
                     const int32_t* __restrict__ idx, uint16_t* __restrict__ fk,
                     uint16_t* __restrict__ fv, int N, int W, int k, int vl_rows, int nfp) {
  __shared__ uint16_t tile[kBlock][kHeadDim + 2];
  const int bj = blockIdx.y;
  const int row = threadIdx.x >> 2, c0 = (threadIdx.x & 3) * 32;
  const int i = blockIdx.x * kBlock + row;
  int src = -1;
  if (i < k) src = idx[(size_t)bj * k + i];
  else if (i >= vl_rows && i - vl_rows < W) src = N - W + (i - vl_rows);
  v4u kw[4], vw[4];
  if (src >= 0) {
    const v4u* kp = reinterpret_cast<const v4u*>(K + ((size_t)bj * N + src) * kHeadDim + c0);
    const v4u* vp = reinterpret_cast<const v4u*>(V + ((size_t)bj * N + src) * kHeadDim + c0);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      kw[u] = kp[u];
      vw[u] = vp[u];
    }
  } else {
#pragma unroll
    for (int u = 0; u < 4; ++u) kw[u] = vw[u] = v4u{0u, 0u, 0u, 0u};
  }
  v4u* kd = reinterpret_cast<v4u*>(fk + ((size_t)bj * nfp + i) * kHeadDim + c0);
#pragma unroll
  for (int u = 0; u < 4; ++u) kd[u] = kw[u];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      tile[row][c0 + u * 8 + 2 * e] = (uint16_t)(vw[u][e] & 0xffffu);
      tile[row][c0 + u * 8 + 2 * e + 1] = (uint16_t)(vw[u][e] >> 16);
    }
  }
  __syncthreads();
  // transposed write: thread -> (channel d, 32 rows)
  const int d = threadIdx.x >> 1, r0 = (threadIdx.x & 1) * 32;
  v4u o[4];
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int e = 0; e < 4; ++e)
      o[u][e] = (uint32_t)tile[r0 + u * 8 + 2 * e][d] |
                ((uint32_t)tile[r0 + u * 8 + 2 * e + 1][d] << 16);
  v4u* vd = reinterpret_cast<v4u*>(fv + ((size_t)bj * kHeadDim + d) * nfp +
                                   (size_t)blockIdx.x * kBlock + r0);
#pragma unroll
  for (int u = 0; u < 4; ++u) vd[u] = o[u];
}

// ---------------------------------------------------------------------------
// Append one token (and, first, merge the W_s oldest window tokens into W_s/64
// new quantized blocks when the staging buffer is full).  blockIdx.y = 0: K,
// 1: V; blockIdx.z: the merged block; one workgroup per (b, j, K/V, block).
// Only block 0 writes the new token: with W a multiple of 64 it takes the
// first slot that block has just quantized.
// ---------------------------------------------------------------------------
struct AppendArgs {
  const uint16_t* k_new;
  const uint16_t* v_new;
  uint16_t* fk;
  uint16_t* fv;
  uint8_t* kc;
  uint8_t* vc;
  float* ks;
  float* vs;
  int32_t* q_pos;
  int nfp, vl_rows, ring_rows, W;
  int merge;          // 1: quantize ring slots [head + 64z, +64) into block blk + z
  int head;           // ring head before the merge
  int blk;            // block index of the first merged block
  int cap_blocks;
  int pos0;           // original position of the oldest window token
  int slot;           // ring slot the new token goes to
};

template <int BITS, int FMT>
__global__ void __launch_bounds__(kQuantThreads)
append_kernel(AppendArgs a) {
  constexpr float C = code_bound<BITS, FMT>();
  constexpr int kRow = BITS == 8 ? kHeadDim : kHeadDim / 2;
  constexpr int vRow = BITS == 8 ? kBlock : kBlock / 2;
  __shared__ float red[kQuantThreads / 64];
  const int bj = blockIdx.x;
  const bool is_v = blockIdx.y == 1;
  const int z = blockIdx.z;
  const int head = a.head + z * kBlock, blk = a.blk + z;
  if (a.merge) {
    float x[32];
    if (!is_v) {
      const int row = threadIdx.x >> 2, c0 = (threadIdx.x & 3) * 32;
      const int slot = (head + row) % a.ring_rows;
      load32(a.fk + ((size_t)bj * a.nfp + a.vl_rows + slot) * kHeadDim + c0, x);
      float m = 0.0f;
#pragma unroll
      for (int e = 0; e < 32; ++e) m = fmaxf(m, fabsf(x[e]));
      const float s = block_max(m, red) / C;
      uint8_t* dst = a.kc + ((size_t)bj * a.cap_blocks * kBlock + (size_t)blk * kBlock + row) * kRow;
      if (BITS == 8) {
        v4u w[2];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          uint32_t v = 0;
#pragma unroll
          for (int q = 0; q < 4; ++q)
            v |= (uint32_t)((s > 0.0f ? quant_code<FMT>(x[4 * e + q], s, C) : 0) & 0xff) << (8 * q);
          w[e >> 2][e & 3] = v;
        }
        v4u* d4 = reinterpret_cast<v4u*>(dst + c0);
        d4[0] = w[0];
        d4[1] = w[1];
      } else {
        v4u w;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          uint32_t v = 0;
#pragma unroll
          for (int q = 0; q < 8; ++q)
            v |= (uint32_t)((s > 0.0f ? quant_code<FMT>(x[8 * e + q], s, C) : 0) & 0xf) << (4 * q);
          w[e] = v;
        }
        *reinterpret_cast<v4u*>(dst + c0 / 2) = w;
      }
      if (threadIdx.x == 0) a.ks[(size_t)bj * a.cap_blocks + blk] = s;
      if ((threadIdx.x & 3) == 0)
        a.q_pos[(size_t)bj * a.cap_blocks * kBlock + (size_t)blk * kBlock + row] = a.pos0 + z * kBlock + row;
    } else {
      // V rows are stored channel-major: thread -> (channel d, 32 tokens)
      const int d = threadIdx.x >> 1, r0 = (threadIdx.x & 1) * 32;
      const uint16_t* src = a.fv + ((size_t)bj * kHeadDim + d) * a.nfp + a.vl_rows;
#pragma unroll
      for (int e = 0; e < 32; ++e) x[e] = bf16_bits_to_f32(src[(head + r0 + e) % a.ring_rows]);
      float m = 0.0f;
#pragma unroll
      for (int e = 0; e < 32; ++e) m = fmaxf(m, fabsf(x[e]));
      const float s = block_max(m, red) / C;
      uint8_t* dst = a.vc + (((size_t)bj * a.cap_blocks + blk) * kHeadDim + d) * vRow;
      if (BITS == 8) {
        v4u w[2];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          uint32_t v = 0;
#pragma unroll
          for (int q = 0; q < 4; ++q)
            v |= (uint32_t)((s > 0.0f ? quant_code<FMT>(x[4 * e + q], s, C) : 0) & 0xff) << (8 * q);
          w[e >> 2][e & 3] = v;
        }
        v4u* d4 = reinterpret_cast<v4u*>(dst + r0);
        d4[0] = w[0];
        d4[1] = w[1];
      } else {
        v4u w;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          uint32_t v = 0;
#pragma unroll
          for (int q = 0; q < 8; ++q)
            v |= (uint32_t)((s > 0.0f ? quant_code<FMT>(x[8 * e + q], s, C) : 0) & 0xf) << (4 * q);
          w[e] = v;
        }
        *reinterpret_cast<v4u*>(dst + r0 / 2) = w;
      }
      if (threadIdx.x == 0) a.vs[(size_t)bj * a.cap_blocks + blk] = s;
    }
    __syncthreads();   // the new token may take a slot the merge has just read
  }
  if (z != 0) return;
  if (!is_v) {
    if (threadIdx.x < 16) {
      const v4u* s = reinterpret_cast<const v4u*>(a.k_new + (size_t)bj * kHeadDim);
      v4u* d = reinterpret_cast<v4u*>(a.fk + ((size_t)bj * a.nfp + a.vl_rows + a.slot) * kHeadDim);
      d[threadIdx.x] = s[threadIdx.x];
    }
  } else if (threadIdx.x < kHeadDim) {
    a.fv[((size_t)bj * kHeadDim + threadIdx.x) * a.nfp + a.vl_rows + a.slot] =
        a.v_new[(size_t)bj * kHeadDim + threadIdx.x];
  }
}

// ---------------------------------------------------------------------------
// Decode attention.
// ---------------------------------------------------------------------------
struct DecodeArgs {
  const uint8_t* kc;
  const uint8_t* vc;
  const uint16_t* fk;
  const uint16_t* fv;
  const uint16_t* q;
  float* part;
  int Hq, Hkv, g;
  int cap_blocks;
  int nbq;          // quantized blocks in use (frozen + merged)
  int nbf;          // frozen blocks; block nbf-1 holds n_last tokens
  int n_last;
  int n_vl, vl_rows, nfp, ring_head, ring_rows, ring_valid;
  int S_q, S_f;     // quantized splits, full-precision splits
  float c_log2;     // softmax_scale * log2(e)
};

// Packed int4 codes (nibble n = element n, two's complement) -> f16 values
// code * 2^e in the element order [0, 4, 1, 5, 2, 6, 3, 7]: each nibble,
// biased by 8, is placed in the low mantissa bits of 1024 (f16 0x6400),
// either at bit 0 (value 1024 + u) or at bit 4 (1024 + 16 u), and one fused
// multiply-add per pair removes the offset and applies 2^e.  Exact.  The
// bias is folded into the constants: ((w ^ 0x88888888) & M) | 0x6400_6400 =
// (w & M) ^ D with D = (0x88888888 & M) | 0x64006400, one 3-input logic op.
struct I4Scale {
  v2h m1, b1, m16, b16;
};
__device__ __forceinline__ I4Scale make_i4scale(float p2) {
  I4Scale s;
  const _Float16 a = (_Float16)p2, b = (_Float16)(-1032.0f * p2);
  const _Float16 c = (_Float16)(p2 * 0.0625f), d = (_Float16)(-72.0f * p2);
  s.m1 = v2h{a, a};
  s.b1 = v2h{b, b};
  s.m16 = v2h{c, c};
  s.b16 = v2h{d, d};
  return s;
}
__device__ __forceinline__ v8h i4x8_to_h_perm(uint32_t w, const I4Scale& s) {
  constexpr uint32_t M0 = 0x000F000Fu, D0 = 0x64086408u;   // nibbles 0, 4 (after >> 8: 2, 6)
  constexpr uint32_t M1 = 0x00F000F0u, D1 = 0x64806480u;   // nibbles 1, 5 (after >> 8: 3, 7)
  const uint32_t w8 = w >> 8;
  const v2h a = __builtin_bit_cast(v2h, (w & M0) ^ D0);
  const v2h b = __builtin_bit_cast(v2h, (w & M1) ^ D1);
  const v2h c = __builtin_bit_cast(v2h, (w8 & M0) ^ D0);
  const v2h d = __builtin_bit_cast(v2h, (w8 & M1) ^ D1);
  const v2h ha = __builtin_elementwise_fma(a, s.m1, s.b1);    // elements 0, 4
  const v2h hb = __builtin_elementwise_fma(b, s.m16, s.b16);  // elements 1, 5
  const v2h hc = __builtin_elementwise_fma(c, s.m1, s.b1);    // elements 2, 6
  const v2h hd = __builtin_elementwise_fma(d, s.m16, s.b16);  // elements 3, 7
  return v8h{ha[0], ha[1], hb[0], hb[1], hc[0], hc[1], hd[0], hd[1]};
}

// 8 packed E2M1 codes (one dword) -> their f16 values, element order.
__device__ __forceinline__ v8h e2m1x8_to_h8(uint32_t w) {
  uint32_t h[4];
  e2m1x8_to_h(w, h, 1.0f);
  return __builtin_bit_cast(v8h, v4u{h[0], h[1], h[2], h[3]});
}

// 8 one-byte codes (two dwords) -> f16 values code * 2^e, element order.
template <int FMT>
__device__ __forceinline__ v8h b8x8_to_h(uint32_t w0, uint32_t w1, const VScale& vs) {
  uint32_t h[4];
  codes4_to_h<FMT>(w0, h[0], h[1], vs);
  codes4_to_h<FMT>(w1, h[2], h[3], vs);
  return __builtin_bit_cast(v8h, v4u{h[0], h[1], h[2], h[3]});
}

// Per-block registers of one wave: K rows of the 4 MFMA tiles, V^T rows of
// the 8 channel tiles, and the block's two scales.
template <int BITS>
struct QRegs {
  static constexpr int kK = BITS == 8 ? 2 : 1;   // 16-byte loads per K tile
  v4u k[4][kK];
  typename std::conditional<BITS == 8, v4u, v2u>::type v[8];
  float sk, sv;
};

// Row of a quantized block read by MFMA tile t, A-operand row m:
// (m/4)*16 + 4t + m%4, so that accumulator register r of lane l holds key
// (l/16)*16 + 4t + r, which is the B-operand order of the P V product.
__device__ __forceinline__ int unit_row(int t, int m) { return ((m >> 2) << 4) + (t << 2) + (m & 3); }

// Channels of K-step s held by lane group G (8 per step; the k-slice of an
// MFMA operand may be any set as long as both operands use the same one).
// Each map makes the 4 lane groups of one load instruction read one
// contiguous 64-byte run of a row:
//   kMapI4:   int4 / E2M1 K rows (64 B): channels 32G + 8s .. (one 16-byte
//             load);
//   kMapB8:   int8 / E4M3 K rows (128 B): load u = s/2 holds channels
//             64u + 16G .. +16, step s the half s%2 of it;
//   kMapBF16: bf16 rows (256 B): channels 32s + 8G .. (one load per step).
constexpr int kMapI4 = 0, kMapB8 = 1, kMapBF16 = 2;
template <int MAP>
__device__ __forceinline__ int step_chan(int s, int G) {
  if constexpr (MAP == kMapI4) return G * 32 + s * 8;
  else if constexpr (MAP == kMapB8) return (s >> 1) * 64 + G * 16 + (s & 1) * 8;
  else return s * 32 + G * 8;
}

// The 4 x 8 query channels of lane (head hl, group G) in the order of a map.
template <int MAP>
__device__ __forceinline__ void load_q(v4u (&qw)[4], const uint16_t* qrow, bool ok, int G) {
#pragma unroll
  for (int s = 0; s < 4; ++s)
    qw[s] = ok ? *reinterpret_cast<const v4u*>(qrow + step_chan<MAP>(s, G)) : v4u{0u, 0u, 0u, 0u};
}

// Rows of a full-precision tile read by MFMA tile t, A-operand row m:
// (t/2)*32 + (m/4)*8 + (t%2)*4 + m%4, so that lane group G holds keys
// 32s + 8G .. 32s + 8G + 7 for P V step s (tiles 2s, 2s+1), which makes the
// channel-major V^T loads contiguous too.
__device__ __forceinline__ int fp_row(int t, int m) {
  return ((t >> 1) << 5) + ((m >> 2) << 3) + ((t & 1) << 2) + (m & 3);
}

// blk is wave-uniform, so the two scale loads are scalar loads, which complete
// independently of the vector loads of the codes.
template <int BITS>
__device__ __forceinline__ void load_block(QRegs<BITS>& r, const DecodeArgs& a,
                                           const float* __restrict__ ks,
                                           const float* __restrict__ vs, int bj, int blk,
                                           int hl, int G) {
  constexpr int kRow = BITS == 8 ? kHeadDim : kHeadDim / 2;
  constexpr int vRow = BITS == 8 ? kBlock : kBlock / 2;
  const size_t cb = (size_t)bj * a.cap_blocks + blk;
  r.sk = ks[cb];
  r.sv = vs[cb];
  const uint8_t* kb = a.kc + cb * kBlock * kRow;
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const uint8_t* row = kb + unit_row(t, hl) * kRow;
#pragma unroll
    for (int u = 0; u < QRegs<BITS>::kK; ++u)   // channels step_chan(2u, G) .. +16 (8-bit), 32G .. (4-bit)
      r.k[t][u] = __builtin_nontemporal_load(
          reinterpret_cast<const v4u*>(row + (BITS == 8 ? u * 64 + G * 16 : G * 16)));
  }
  const uint8_t* vb = a.vc + cb * kHeadDim * vRow;
#pragma unroll
  for (int ct = 0; ct < 8; ++ct) {
    const uint8_t* p = vb + (ct * 16 + hl) * vRow + G * (vRow / 4);
    if constexpr (BITS == 8) r.v[ct] = __builtin_nontemporal_load(reinterpret_cast<const v4u*>(p));
    else r.v[ct] = __builtin_nontemporal_load(reinterpret_cast<const v2u*>(p));
  }
}

__device__ __forceinline__ float xgroup_max(float x) {
  x = fmaxf(x, __shfl_xor(x, 16, 64));
  return fmaxf(x, __shfl_xor(x, 32, 64));
}

// Online state of one wave.  The accumulator holds sum p * value / 2^eref,
// eref the largest V-scale exponent met so far (blocks with smaller scales
// enter through smaller weights), so that every f16 weight stays <= 2^8.
struct WaveState {
  v4f acc[8];     // O^T tiles: lane l holds head l%16, channels 16ct + 4(l/16) + r
  float m;        // running max (log2 domain), the same on the 4 lanes of a head
  float l;        // this lane's share of the weight sum
  int eref;       // wave-uniform
};

// Raise the running max (lazily) and the V-scale exponent to cover a new
// unit with logits y * cs (cs > 0) and exponent e; rescales the state when
// either moves.
__device__ __forceinline__ void advance(WaveState& st, const float (&y)[16], float cs, int e) {
  float bm = fmaxf(fmaxf(y[0], y[1]), y[2]);
#pragma unroll
  for (int i = 3; i < 16; i += 2) bm = fmaxf(fmaxf(bm, y[i]), y[i + 1 < 16 ? i + 1 : i]);
  bm = xgroup_max(bm) * cs;
  const float mnew = bm > st.m + kLazyD ? bm : st.m;
  const int enew = e > st.eref ? e : st.eref;
  if (__ballot(mnew != st.m) || enew != st.eref) {
    const float cl = __builtin_amdgcn_exp2f(st.m - mnew);
    const float ca = __builtin_ldexpf(cl, st.eref - enew);
#pragma unroll
    for (int ct = 0; ct < 8; ++ct) st.acc[ct] *= ca;
    st.l *= cl;
    st.m = mnew;
    st.eref = enew;
  }
}

template <int BITS, int FMT>
__device__ __forceinline__ void process_block(WaveState& st, const QRegs<BITS>& r,
                                              const v8h (&qh)[4], float c_q, int n_valid,
                                              int G) {
  // S^T = K q^T: 4 tiles of 16 keys, 4 steps of 32 channels
  v4f sc[4];
  const I4Scale one4 = make_i4scale(1.0f);
  const VScale one8 = make_vscale(1.0f);
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    sc[t] = v4f{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      v8h ka;
      if constexpr (FMT == HYQ_FMT_FP4) ka = e2m1x8_to_h8(r.k[t][0][s]);
      else if constexpr (BITS == 4) ka = i4x8_to_h_perm(r.k[t][0][s], one4);
      else ka = b8x8_to_h<FMT>(r.k[t][s >> 1][(s & 1) * 2], r.k[t][s >> 1][(s & 1) * 2 + 1], one8);
      sc[t] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ka, qh[s], sc[t], 0, 0, 0);
    }
  }
  // logits in the log2 domain are sc * cs (cs > 0: a zero K block only has
  // zero raw scores, so flooring cs changes nothing that matters)
  const float cs = fmaxf(c_q * r.sk, 1e-30f);
  if (n_valid < kBlock) {
    // the ragged last block of the Freeze: padding keys take no weight (a
    // real branch, not if-converted, since only one block per head has it)
    asm volatile("" ::: "memory");
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (G * 16 + t * 4 + q >= n_valid) sc[t][q] = -INFINITY;
  }
  float y[16];
#pragma unroll
  for (int t = 0; t < 4; ++t)
#pragma unroll
    for (int q = 0; q < 4; ++q) y[t * 4 + q] = sc[t][q];
  // V scale sV = fm * 2^e, fm in [1/2, 1); an all-zero block (sV = 0) adds nothing
  int e = st.eref;
  float fm = 1.0f;
  if (r.sv > 0.0f) fm = __builtin_frexpf(r.sv, &e);
  advance(st, y, cs, e);
  // weights p * fm * 2^(e - eref) in f16 (below 2^-60 they are zero in f16 anyway)
  const int d = max(e - st.eref, -60);
  const float nbias = __builtin_amdgcn_logf(fm) + (float)d - st.m;
  _Float16 p[16];
  float ps = 0.0f;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const float pw = __builtin_amdgcn_exp2f(__builtin_fmaf(y[i], cs, nbias));
    p[i] = (_Float16)pw;
    ps += pw;
  }
  st.l += ps * __builtin_ldexpf(__builtin_amdgcn_rcpf(fm), -d);
  // O^T += V^T P^T: 8 channel tiles x 2 steps of 32 keys
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    v8h pb;
    if constexpr (BITS == 4 && FMT == HYQ_FMT_INT) {   // the int4 conversion's key order
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        pb[2 * q] = p[(2 * s) * 4 + q];
        pb[2 * q + 1] = p[(2 * s + 1) * 4 + q];
      }
    } else {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        pb[q] = p[(2 * s) * 4 + q];
        pb[4 + q] = p[(2 * s + 1) * 4 + q];
      }
    }
#pragma unroll
    for (int ct = 0; ct < 8; ++ct) {
      v8h va;
      if constexpr (FMT == HYQ_FMT_FP4) va = e2m1x8_to_h8(r.v[ct][s]);
      else if constexpr (BITS == 4) va = i4x8_to_h_perm(r.v[ct][s], one4);
      else va = b8x8_to_h<FMT>(r.v[ct][2 * s], r.v[ct][2 * s + 1], one8);
      st.acc[ct] = __builtin_amdgcn_mfma_f32_16x16x32_f16(va, pb, st.acc[ct], 0, 0, 0);
    }
  }
}

// One tile of 64 full-precision rows (vertical lines or ring slots); their
// values are exact bf16, a "scale" of 2^0.
__device__ __forceinline__ void process_fp_tile(WaveState& st, const DecodeArgs& a, int bj,
                                                int tile, const v8bf (&qb)[4], int hl, int G) {
  const int base = tile * kBlock;
  v4u kr[4][4];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const uint16_t* row = a.fk + ((size_t)bj * a.nfp + base + fp_row(t, hl)) * kHeadDim;
#pragma unroll
    for (int s = 0; s < 4; ++s)
      kr[t][s] = __builtin_nontemporal_load(
          reinterpret_cast<const v4u*>(row + step_chan<kMapBF16>(s, G)));
  }
  v4u vr[8][2];
#pragma unroll
  for (int ct = 0; ct < 8; ++ct) {
    const uint16_t* vrow = a.fv + ((size_t)bj * kHeadDim + ct * 16 + hl) * a.nfp + base + G * 8;
    vr[ct][0] = __builtin_nontemporal_load(reinterpret_cast<const v4u*>(vrow));        // keys 8G ..
    vr[ct][1] = __builtin_nontemporal_load(reinterpret_cast<const v4u*>(vrow + 32));   // keys 32 + 8G ..
  }
  v4f sc[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    sc[t] = v4f{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int s = 0; s < 4; ++s)
      sc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(v8bf, kr[t][s]), qb[s],
                                                      sc[t], 0, 0, 0);
  }
  float y[16];
#pragma unroll
  for (int t = 0; t < 4; ++t)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int i = base + fp_row(t, G * 4 + q);
      const int r0 = i - a.vl_rows - a.ring_head;
      const int rs = r0 + (r0 < 0 ? a.ring_rows : 0);
      const bool valid = (i < a.n_vl) | ((i >= a.vl_rows) & (rs < a.ring_valid));
      y[t * 4 + q] = valid ? sc[t][q] : -INFINITY;
    }
  advance(st, y, a.c_log2, 0);
  const int d = max(-st.eref, -60);
  const float nbias = (float)d - st.m;
  uint32_t hi[16], lo[16];
  float ps = 0.0f;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const float pv = __builtin_amdgcn_exp2f(__builtin_fmaf(y[i], a.c_log2, nbias));
    const uint32_t hb = __float_as_uint(pv) & 0xffff0000u;
    const float rem = pv - __uint_as_float(hb);
    const uint32_t lb = __float_as_uint(rem);
    const uint32_t lr = (lb + 0x7fffu + ((lb >> 16) & 1u)) & 0xffff0000u;   // round to nearest even
    hi[i] = hb >> 16;
    lo[i] = lr >> 16;
    ps += pv;
  }
  st.l += __builtin_ldexpf(ps, -d);
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    v4u ph, pl;
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      ph[q] = hi[(2 * s) * 4 + 2 * q] | (hi[(2 * s) * 4 + 2 * q + 1] << 16);
      ph[2 + q] = hi[(2 * s + 1) * 4 + 2 * q] | (hi[(2 * s + 1) * 4 + 2 * q + 1] << 16);
      pl[q] = lo[(2 * s) * 4 + 2 * q] | (lo[(2 * s) * 4 + 2 * q + 1] << 16);
      pl[2 + q] = lo[(2 * s + 1) * 4 + 2 * q] | (lo[(2 * s + 1) * 4 + 2 * q + 1] << 16);
    }
    const v8bf bh = __builtin_bit_cast(v8bf, ph), bl = __builtin_bit_cast(v8bf, pl);
#pragma unroll
    for (int ct = 0; ct < 8; ++ct) {
      const v8bf va = __builtin_bit_cast(v8bf, vr[ct][s]);
      st.acc[ct] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, bh, st.acc[ct], 0, 0, 0);
      st.acc[ct] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, bl, st.acc[ct], 0, 0, 0);
    }
  }
}

// Grid (S_q + S_f, B*Hkv): in workgroups x < S_q each of the 4 S_q waves of
// KV head (b, j) takes an even share of consecutive quantized blocks; in the
// others wave t takes the full-precision tiles t, t + 4 S_f, ...  Each
// workgroup writes one partial (acc[128], m, l) per query head of the group.
template <int BITS, int FMT>
__global__ void __launch_bounds__(kDecThreads, 2)
decode_attn_kernel(DecodeArgs a, const float* __restrict__ ks, const float* __restrict__ vs) {
  __shared__ float r_acc[kDecWaves][kMaxGroup][kHeadDim];
  __shared__ float r_m[kDecWaves][kMaxGroup], r_l[kDecWaves][kMaxGroup];
  const int bj = blockIdx.y, split = blockIdx.x;
  const int b = bj / a.Hkv, j = bj - b * a.Hkv;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int hl = lane & 15, G = lane >> 4;

  // query row of lane (head hl, group G); heads hl >= g are zero columns
  const bool qok = hl < a.g;
  const uint16_t* qrow = a.q + ((size_t)b * a.Hq + (size_t)j * a.g + (qok ? hl : 0)) * kHeadDim;
  v4u qw[4];

  WaveState st;
#pragma unroll
  for (int ct = 0; ct < 8; ++ct) st.acc[ct] = v4f{0.0f, 0.0f, 0.0f, 0.0f};
  st.m = kMinusBigD;
  st.l = 0.0f;
  st.eref = -1000;

  if (split < a.S_q) {
    // an even share of the quantized blocks: wave gw of the nw = S_q * 4
    // takes the consecutive blocks [gw * nbq / nw, (gw + 1) * nbq / nw)
    const int nw = a.S_q * kDecWaves, gw = split * kDecWaves + w;
    const int first = (int)((int64_t)gw * a.nbq / nw);
    const int n_my = (int)((int64_t)(gw + 1) * a.nbq / nw) - first;
    QRegs<BITS> r0, r1;
    load_q<BITS == 4 ? kMapI4 : kMapB8>(qw, qrow, qok, G);   // first: waits for it never wait for codes
    if (n_my > 0) load_block<BITS>(r0, a, ks, vs, bj, first, hl, G);
    // f16 query: q * 2^eq with max |q * 2^eq| in [2^14, 2^15) per head
    uint32_t mx = 0;
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        mx = max(mx, qw[s][e] & 0x7fffu);
        mx = max(mx, (qw[s][e] >> 16) & 0x7fffu);
      }
    float qmax = bf16_bits_to_f32(mx);
    qmax = xgroup_max(qmax);
    int E = 0;
    if (qmax > 0.0f) frexpf(qmax, &E);
    const int eq = qmax > 0.0f ? 15 - E : 0;
    const float qmul = __builtin_ldexpf(1.0f, eq);
    v8h qh[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      float f[8];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        f[2 * e] = bf16_lo(qw[s][e]) * qmul;
        f[2 * e + 1] = bf16_hi(qw[s][e]) * qmul;
      }
      if constexpr (BITS == 4 && FMT == HYQ_FMT_INT) {   // the int4 conversion's order
        const int ord[8] = {0, 4, 1, 5, 2, 6, 3, 7};
#pragma unroll
        for (int e = 0; e < 8; ++e) qh[s][e] = (_Float16)f[ord[e]];
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) qh[s][e] = (_Float16)f[e];
      }
    }
    const float c_q = a.c_log2 * __builtin_ldexpf(1.0f, -eq);

    // two register sets alternate so that the next block's loads are always
    // in flight while one block is computed; inside the loop every load is
    // unconditional, which keeps each wait for a block's codes from also
    // waiting for the prefetched block
    auto proc = [&](const QRegs<BITS>& r, int i) {
      const int blk = first + i;
      const int n_valid = blk == a.nbf - 1 ? a.n_last : kBlock;
      // keep the scheduler from starting the next block's conversions (and
      // so waiting for its loads) inside this one
      __builtin_amdgcn_sched_barrier(0);
      process_block<BITS, FMT>(st, r, qh, c_q, n_valid, G);
      __builtin_amdgcn_sched_barrier(0);
    };
    int i = 0;
    for (; i + 2 < n_my; i += 2) {
      load_block<BITS>(r1, a, ks, vs, bj, first + i + 1, hl, G);
      proc(r0, i);
      load_block<BITS>(r0, a, ks, vs, bj, first + i + 2, hl, G);
      proc(r1, i + 1);
    }
    if (i + 1 < n_my) {
      load_block<BITS>(r1, a, ks, vs, bj, first + i + 1, hl, G);
      proc(r0, i);
      proc(r1, i + 1);
    } else if (i < n_my) {
      proc(r0, i);
    }
  } else {
    // full-precision tiles tile, tile + 4 S_f, ...
    const int nft = a.nfp / kBlock;
    int tile = (split - a.S_q) * kDecWaves + w;
    if (tile < nft) {
      load_q<kMapBF16>(qw, qrow, qok, G);
      v8bf qb[4];
#pragma unroll
      for (int s = 0; s < 4; ++s) qb[s] = __builtin_bit_cast(v8bf, qw[s]);
      for (; tile < nft; tile += a.S_f * kDecWaves) process_fp_tile(st, a, bj, tile, qb, hl, G);
    }
  }

  // wave totals -> LDS (the accumulator back in value units)
  float l = st.l;
  l += __shfl_xor(l, 16, 64);
  l += __shfl_xor(l, 32, 64);
  if (hl < a.g) {
    if (G == 0) {
      r_m[w][hl] = st.m;
      r_l[w][hl] = l;
    }
#pragma unroll
    for (int ct = 0; ct < 8; ++ct)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        r_acc[w][hl][ct * 16 + G * 4 + q] = __builtin_ldexpf(st.acc[ct][q], st.eref);
  }
  __syncthreads();
  // merge the 4 waves: one partial per query head of the group
  const int S = a.S_q + a.S_f;
  for (int e = threadIdx.x; e < a.g * kHeadDim; e += kDecThreads) {
    const int h = e >> 7, c = e & (kHeadDim - 1);
    float M = r_m[0][h];
#pragma unroll
    for (int v = 1; v < kDecWaves; ++v) M = fmaxf(M, r_m[v][h]);
    float acc = 0.0f, lsum = 0.0f;
#pragma unroll
    for (int v = 0; v < kDecWaves; ++v) {
      const float f = __builtin_amdgcn_exp2f(r_m[v][h] - M);
      acc += r_acc[v][h][c] * f;
      lsum += r_l[v][h] * f;
    }
    float* dst = a.part + (((size_t)bj * S + split) * a.g + h) * kPartStride;
    dst[c] = acc;
    if (c == 0) {
      dst[kHeadDim] = M;
      dst[kHeadDim + 1] = lsum;
    }
  }
}

// ReduceSoftmax over the S partials of each (b, h): one workgroup of two waves
// per query row.  Thread -> (share ph of the partials, 4 channels): an online
// max over its share (loads issued 8 deep), then the 4 shares of each channel
// quad merged through LDS.  The kernel is bound by latency, not bytes: fewer,
// longer shares beat more threads.
constexpr int kCombThreads = 128;
constexpr int kCombShares = kCombThreads / (kHeadDim / 4);
__global__ void __launch_bounds__(kCombThreads)
decode_combine_kernel(const float* __restrict__ part, void* __restrict__ out, int Hq, int Hkv,
                      int g, int S, int out_bf16) {
  __shared__ float x_acc[kCombShares][kHeadDim / 4][4];
  __shared__ float x_m[kCombShares][kHeadDim / 4], x_l[kCombShares][kHeadDim / 4];
  const int bh = blockIdx.x;
  const int b = bh / Hq, h = bh - b * Hq;
  const int j = h / g, r = h - j * g;
  const size_t bj = (size_t)b * Hkv + j;
  const int c4 = threadIdx.x & 31, ph = threadIdx.x >> 5;
  const float* base = part + (bj * S * g + r) * kPartStride;
  const size_t stride = (size_t)g * kPartStride;
  float M = kMinusBigD, L = 0.0f;
  v4f acc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll 8
  for (int s = ph; s < S; s += kCombShares) {
    const float* p = base + s * stride;
    const v2u ml = *reinterpret_cast<const v2u*>(p + kHeadDim);
    const v4f v = *reinterpret_cast<const v4f*>(p + c4 * 4);
    const float m = __uint_as_float(ml[0]), l = __uint_as_float(ml[1]);
    const float Mn = fmaxf(M, m);
    const float a1 = __builtin_amdgcn_exp2f(M - Mn), f = __builtin_amdgcn_exp2f(m - Mn);
    acc = acc * a1 + v * f;
    L = L * a1 + l * f;
    M = Mn;
  }
  x_m[ph][c4] = M;
  x_l[ph][c4] = L;
#pragma unroll
  for (int e = 0; e < 4; ++e) x_acc[ph][c4][e] = acc[e];
  __syncthreads();
  if (ph != 0) return;
  for (int q = 1; q < kCombShares; ++q) {
    const float Mn = fmaxf(M, x_m[q][c4]);
    const float a1 = __builtin_amdgcn_exp2f(M - Mn), f = __builtin_amdgcn_exp2f(x_m[q][c4] - Mn);
#pragma unroll
    for (int e = 0; e < 4; ++e) acc[e] = acc[e] * a1 + x_acc[q][c4][e] * f;
    L = L * a1 + x_l[q][c4] * f;
    M = Mn;
  }
  const float inv = 1.0f / L;
  const size_t off = (size_t)bh * kHeadDim + c4 * 4;
  if (out_bf16) {
    uint32_t w[2];
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      uint32_t u0 = __float_as_uint(acc[2 * e] * inv), u1 = __float_as_uint(acc[2 * e + 1] * inv);
      u0 = (u0 + 0x7fffu + ((u0 >> 16) & 1u)) >> 16;
      u1 = (u1 + 0x7fffu + ((u1 >> 16) & 1u)) >> 16;
      w[e] = u0 | (u1 << 16);
    }
    *reinterpret_cast<v2u*>(reinterpret_cast<uint16_t*>(out) + off) = v2u{w[0], w[1]};
  } else {
    *reinterpret_cast<v4f*>(reinterpret_cast<float*>(out) + off) = acc * inv;
  }
}

}  // namespace

// ---- host launchers -------------------------------------------------------

// Compute units of the current device (cached per device).
// Scratch of hyq_decode_attn_noalloc: the split partials of one launch, in
// a file-scope device array (each GPU holds its own copy at its own address,
// from the first use of the library on it until the process ends).  Host
// code must not pass the array's name to a kernel: its device address comes
// from hipGetSymbolAddress, looked up once per device with that device
// current.
constexpr size_t kNoAllocFloats = HYQ_NOALLOC_SCRATCH_BYTES / sizeof(float);
__device__ __align__(256) float scratch[kNoAllocFloats];

hipError_t noalloc_scratch(float** out) {
  constexpr int kMaxDev = 64;
  static std::mutex mu;
  static float* addr[kMaxDev];
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDev) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    addr[dev] = static_cast<float*>(p);
  }
  *out = addr[dev];
  return hipSuccess;
}

static int device_cus() {
  constexpr int kMaxDev = 64;
  static std::atomic<int> cus[kMaxDev];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDev) return 256;
  int n = cus[dev].load(std::memory_order_relaxed);
  if (n <= 0) {
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        n <= 0)
      n = 256;
    cus[dev].store(n, std::memory_order_relaxed);
  }
  return n;
}

DecodeSplit decode_split(const hyq_dcache& c) {
  DecodeSplit d;
  const int nbf = (c.n_frozen + kBlock - 1) / kBlock;
  d.nbq = nbf + c.n_merged;
  const int nft = (c.vl_rows + c.ring_rows) / kBlock;
  const DecodeShape sh = decode_shape_for(d.nbq, nft, (int64_t)c.B * c.Hkv, device_cus(), c.bits_kv);
  d.S_q = sh.S_q;
  d.S_f = sh.S_f;
  return d;
}

size_t decode_part_bytes(const hyq_dcache& c) {
  const DecodeSplit d = decode_split(c);
  return (size_t)c.B * c.Hkv * (size_t)(d.S_q + d.S_f) * (c.Hq / c.Hkv) * kPartStride *
         sizeof(float);
}

size_t decode_ws_bytes(const hyq_dcache& c) {
  const int nft = (c.vl_rows + c.ring_rows) / kBlock;
  const int64_t S = (c.cap_blocks + 2 * kDecWaves - 1) / (2 * kDecWaves) +
                    (nft + kDecWaves - 1) / kDecWaves;
  return (size_t)c.B * c.Hkv * S * (c.Hq / c.Hkv) * kPartStride * sizeof(float);
}

hipError_t launch_freeze_gather(const hyq_dcache& c, int N, const uint16_t* K, const uint16_t* V,
                                hipStream_t st) {
  const int nfp = c.vl_rows + c.ring_rows;
  dim3 grid(nfp / kBlock, c.B * c.Hkv);
  freeze_gather_kernel<<<grid, 256, 0, st>>>(K, V, c.vl_pos, static_cast<uint16_t*>(c.fp_k),
                                             static_cast<uint16_t*>(c.fp_v), N, c.window, c.n_vl,
                                             c.vl_rows, nfp);
  return hipGetLastError();
}

hipError_t launch_decode_append(const hyq_dcache& c, const uint16_t* k_new, const uint16_t* v_new,
                                bool merge, int slot, hipStream_t st) {
  AppendArgs a;
  a.k_new = k_new;
  a.v_new = v_new;
  a.fk = static_cast<uint16_t*>(c.fp_k);
  a.fv = static_cast<uint16_t*>(c.fp_v);
  a.kc = static_cast<uint8_t*>(c.k_codes);
  a.vc = static_cast<uint8_t*>(c.v_codes);
  a.ks = c.k_scale;
  a.vs = c.v_scale;
  a.q_pos = c.q_pos;
  a.nfp = c.vl_rows + c.ring_rows;
  a.vl_rows = c.vl_rows;
  a.ring_rows = c.ring_rows;
  a.W = c.window;
  a.merge = merge ? 1 : 0;
  a.head = c.ring_head;
  a.blk = (c.n_frozen + kBlock - 1) / kBlock + c.n_merged;
  a.cap_blocks = c.cap_blocks;
  a.pos0 = (int)(c.t - c.n_staged - c.window);
  a.slot = slot;
  dim3 grid(c.B * c.Hkv, 2, merge ? c.staging / kBlock : 1);
  if (c.kv_format == HYQ_FMT_FP4) append_kernel<4, HYQ_FMT_FP4><<<grid, kQuantThreads, 0, st>>>(a);
  else if (c.kv_format == HYQ_FMT_FP8) append_kernel<8, HYQ_FMT_FP8><<<grid, kQuantThreads, 0, st>>>(a);
  else if (c.bits_kv == 8) append_kernel<8, HYQ_FMT_INT><<<grid, kQuantThreads, 0, st>>>(a);
  else append_kernel<4, HYQ_FMT_INT><<<grid, kQuantThreads, 0, st>>>(a);
  return hipGetLastError();
}

hipError_t launch_decode_attn(const hyq_dcache& c, const uint16_t* q, float softmax_scale,
                              void* out, int out_dtype, float* part, hipStream_t st) {
  const DecodeSplit d = decode_split(c);
  DecodeArgs a;
  a.kc = static_cast<const uint8_t*>(c.k_codes);
  a.vc = static_cast<const uint8_t*>(c.v_codes);
  a.fk = static_cast<const uint16_t*>(c.fp_k);
  a.fv = static_cast<const uint16_t*>(c.fp_v);
  a.q = q;
  a.part = part;
  a.Hq = c.Hq;
  a.Hkv = c.Hkv;
  a.g = c.Hq / c.Hkv;
  a.cap_blocks = c.cap_blocks;
  a.nbq = d.nbq;
  a.nbf = (c.n_frozen + kBlock - 1) / kBlock;
  a.n_last = c.n_frozen - (a.nbf - 1) * kBlock;
  a.n_vl = c.n_vl;
  a.vl_rows = c.vl_rows;
  a.nfp = c.vl_rows + c.ring_rows;
  a.ring_head = c.ring_head;
  a.ring_rows = c.ring_rows;
  a.ring_valid = c.window + c.n_staged;
  a.S_q = d.S_q;
  a.S_f = d.S_f;
  a.c_log2 = softmax_scale * 1.4426950408889634f;
  const int S = d.S_q + d.S_f;
  dim3 grid(S, c.B * c.Hkv);
  if (c.kv_format == HYQ_FMT_FP4)
    decode_attn_kernel<4, HYQ_FMT_FP4><<<grid, kDecThreads, 0, st>>>(a, c.k_scale, c.v_scale);
  else if (c.kv_format == HYQ_FMT_FP8)
    decode_attn_kernel<8, HYQ_FMT_FP8><<<grid, kDecThreads, 0, st>>>(a, c.k_scale, c.v_scale);
  else if (c.bits_kv == 8)
    decode_attn_kernel<8, HYQ_FMT_INT><<<grid, kDecThreads, 0, st>>>(a, c.k_scale, c.v_scale);
  else
    decode_attn_kernel<4, HYQ_FMT_INT><<<grid, kDecThreads, 0, st>>>(a, c.k_scale, c.v_scale);
  decode_combine_kernel<<<c.B * c.Hq, kCombThreads, 0, st>>>(part, out, c.Hq, c.Hkv, a.g, S,
                                                             out_dtype);
  return hipGetLastError();
}

}  // namespace hyq
