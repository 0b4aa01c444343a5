// Partition and per-block symmetric quantization: Algorithm 2, Stages 1-2
// (App. A.2) of HyQuant.
//
//   kq_pos  = [0, P) minus the vertical positions, ascending (the K_Q set of
//             the partition of Section 4.1);
//   Q       : blocks of 64 query rows per head;
//   K, V    : blocks of 64 consecutive entries of the compacted K_Q sequence
//             (rows gathered through kq_pos);
//   s = fl32(max|x| / c), code = clamp(rint(fl32(x / s)), -c, c), s = 0 ->
//   codes 0 (c = 127 for 8-bit, 7 for 4-bit);
//   FP8 codes (c = 448): the OCP E4M3 value nearest to fl32(x / s), ties to
//   even, saturating at +-448, zero keeping the sign (the hardware
//   float32 -> E4M3 conversion, which rounds to nearest even).
//
// The division is the IEEE correctly rounded float32 division (no
// reciprocal shortcut) and rint rounds half to even, so codes match the
// definition bit for bit.  HBM-bound: each input row is read once and each
// code written once, with 16-byte accesses.
#include "hyq_internal.h"
#include "quant_dev.h"

#pragma clang fp contract(off)

namespace hyq {
namespace {

constexpr int kMaxLdsIdx = 8192;

// slots n < nQ: the n-th non-vertical prefix position; slots [nQ, nslots):
// padding marker.  Position p (not vertical) goes to slot p - #{idx < p}.
__global__ void __launch_bounds__(256)
compact_kernel(const int32_t* __restrict__ idx, int32_t* __restrict__ kq_pos, int k, int P,
               int nQ, int nslots) {
  __shared__ int32_t sidx[kMaxLdsIdx];
  const int bj = blockIdx.y;
  const int32_t* id = idx + (size_t)bj * k;
  const bool in_lds = k <= kMaxLdsIdx;
  if (in_lds)
    for (int i = threadIdx.x; i < k; i += blockDim.x) sidx[i] = id[i];
  __syncthreads();
  const int32_t* src = in_lds ? sidx : id;
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  int32_t* out = kq_pos + (size_t)bj * nslots;
  if (i < P) {
    int lo = 0, hi = k;  // lower_bound of i in the ascending idx list
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (src[mid] < i) lo = mid + 1; else hi = mid;
    }
    const bool vertical = lo < k && src[lo] == i;
    const int slot = i - lo;
    if (!vertical && slot >= 0 && slot < nQ) out[slot] = i;
  }
  if (i >= nQ && i < nslots) out[i] = HYQ_KQ_POS_PAD;
}

// Thread layout of one 64 x 128 block: row = tid / 4, channels (tid % 4) * 32 .. +32.
template <int FMT>
__global__ void __launch_bounds__(kQuantThreads)
quant_q_kernel(const uint16_t* __restrict__ Q, int8_t* __restrict__ qc, float* __restrict__ qs,
               int L, int n_qblk) {
  constexpr float C = FMT == HYQ_FMT_FP8 ? 448.0f : FMT == HYQ_FMT_FP4Q6 ? 7.5f : 127.0f;
  __shared__ float red[kQuantThreads / 64];
  const int bh = blockIdx.y, blk = blockIdx.x;
  const int row = threadIdx.x >> 2, c0 = (threadIdx.x & 3) * 32;
  const int t = blk * kBlock + row;
  float x[32];
  if (t < L) {
    load32(Q + ((size_t)bh * L + t) * kHeadDim + c0, x);
  } else {
#pragma unroll
    for (int e = 0; e < 32; ++e) x[e] = 0.0f;
  }
  float m = 0.0f;
#pragma unroll
  for (int e = 0; e < 32; ++e) m = fmaxf(m, fabsf(x[e]));
  const float amax = block_max(m, red);
  const float s = amax / C;
  if (threadIdx.x == 0) qs[(size_t)bh * n_qblk + blk] = s;
  if (t >= L) return;
  uint32_t packed[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    uint32_t w = 0;
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const int code = s > 0.0f ? quant_code<FMT>(x[4 * e + b], s, C) : 0;
      w |= (uint32_t)(code & 0xff) << (8 * b);
    }
    packed[e] = w;
  }
  uint4* dst = reinterpret_cast<uint4*>(qc + ((size_t)bh * L + t) * kHeadDim + c0);
  dst[0] = make_uint4(packed[0], packed[1], packed[2], packed[3]);
  dst[1] = make_uint4(packed[4], packed[5], packed[6], packed[7]);
}

// One workgroup per (b, j, compacted block).  K codes are written row-major,
// V codes channel-major (the block transposed) through an LDS tile.
// n_kvblk is the number of blocks each (b, j) owns in the outputs (kq_pos
// slots n_kvblk * 64); the grid may cover fewer.
template <int BITS, int FMT>
__global__ void __launch_bounds__(kQuantThreads)
quant_kv_kernel(const uint16_t* __restrict__ K, const uint16_t* __restrict__ V,
                const int32_t* __restrict__ kq_pos, uint8_t* __restrict__ kc,
                float* __restrict__ ks, uint8_t* __restrict__ vc, float* __restrict__ vs,
                int L, int nQ, int n_kvblk) {
  static_assert((FMT != HYQ_FMT_FP8 || BITS == 8) && (FMT != HYQ_FMT_FP4 || BITS == 4),
                "FP8 codes are 8-bit, FP4 codes 4-bit");
  constexpr float C = code_bound<BITS, FMT>();
  constexpr int kRow = BITS == 8 ? kHeadDim : kHeadDim / 2;   // bytes per K code row
  constexpr int vRow = BITS == 8 ? kBlock : kBlock / 2;        // bytes per V code row (one channel)
  __shared__ float red[kQuantThreads / 64];
  __shared__ int8_t vt[kBlock][kHeadDim + 4];                   // V codes, [key][channel]
  const int bj = blockIdx.y, blk = blockIdx.x;
  const int row = threadIdx.x >> 2, c0 = (threadIdx.x & 3) * 32;
  const int n = blk * kBlock + row;
  const size_t slots = (size_t)n_kvblk * kBlock;
  float xk[32], xv[32];
  const int pos = n < nQ ? kq_pos[(size_t)bj * slots + n] : -1;
  if ((unsigned)pos < (unsigned)L) {
    load32(K + ((size_t)bj * L + pos) * kHeadDim + c0, xk);
    load32(V + ((size_t)bj * L + pos) * kHeadDim + c0, xv);
  } else {
#pragma unroll
    for (int e = 0; e < 32; ++e) xk[e] = xv[e] = 0.0f;
  }
  float mk = 0.0f, mv = 0.0f;
#pragma unroll
  for (int e = 0; e < 32; ++e) {
    mk = fmaxf(mk, fabsf(xk[e]));
    mv = fmaxf(mv, fabsf(xv[e]));
  }
  const float sk = block_max(mk, red) / C;
  const float sv = block_max(mv, red) / C;
  if (threadIdx.x == 0) {
    ks[(size_t)bj * n_kvblk + blk] = sk;
    vs[(size_t)bj * n_kvblk + blk] = sv;
  }
  int ck[32], cv[32];
#pragma unroll
  for (int e = 0; e < 32; ++e) {
    ck[e] = sk > 0.0f ? quant_code<FMT>(xk[e], sk, C) : 0;
    cv[e] = sv > 0.0f ? quant_code<FMT>(xv[e], sv, C) : 0;
  }
  // K: row-major codes
  uint8_t* kdst = kc + ((size_t)bj * slots + n) * kRow;
  if (BITS == 8) {
    uint32_t w[8];
#pragma unroll
    for (int e = 0; e < 8; ++e)
      w[e] = (uint32_t)(ck[4 * e] & 0xff) | ((uint32_t)(ck[4 * e + 1] & 0xff) << 8) |
             ((uint32_t)(ck[4 * e + 2] & 0xff) << 16) | ((uint32_t)(ck[4 * e + 3] & 0xff) << 24);
    uint4* d4 = reinterpret_cast<uint4*>(kdst + c0);
    d4[0] = make_uint4(w[0], w[1], w[2], w[3]);
    d4[1] = make_uint4(w[4], w[5], w[6], w[7]);
  } else {
    uint32_t w[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      uint32_t a = 0;
#pragma unroll
      for (int b = 0; b < 8; ++b) a |= (uint32_t)(ck[8 * e + b] & 0xf) << (4 * b);
      w[e] = a;
    }
    *reinterpret_cast<uint4*>(kdst + c0 / 2) = make_uint4(w[0], w[1], w[2], w[3]);
  }
  // V: stage codes, then write channel-major
#pragma unroll
  for (int e = 0; e < 32; ++e) vt[row][c0 + e] = (int8_t)cv[e];
  __syncthreads();
  {
    const int d = threadIdx.x >> 1, k0 = (threadIdx.x & 1) * 32;
    uint8_t* vdst = vc + (((size_t)bj * n_kvblk + blk) * kHeadDim + d) * vRow;
    if (BITS == 8) {
      uint32_t w[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        uint32_t a = 0;
#pragma unroll
        for (int b = 0; b < 4; ++b) a |= (uint32_t)(uint8_t)vt[k0 + 4 * e + b][d] << (8 * b);
        w[e] = a;
      }
      uint4* d4 = reinterpret_cast<uint4*>(vdst + k0);
      d4[0] = make_uint4(w[0], w[1], w[2], w[3]);
      d4[1] = make_uint4(w[4], w[5], w[6], w[7]);
    } else {
      uint32_t w[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        uint32_t a = 0;
#pragma unroll
        for (int b = 0; b < 8; ++b) a |= (uint32_t)(vt[k0 + 8 * e + b][d] & 0xf) << (4 * b);
        w[e] = a;
      }
      *reinterpret_cast<uint4*>(vdst + k0 / 2) = make_uint4(w[0], w[1], w[2], w[3]);
    }
  }
}

}  // namespace

void launch_compact(const int32_t* idx, int32_t* kq_pos, int k, int P, int nQ, int nslots,
                    int BHkv, hipStream_t st) {
  const int span = P > nslots ? P : nslots;
  if (nslots <= 0) return;
  dim3 cg((span + 255) / 256, BHkv);
  compact_kernel<<<cg, 256, 0, st>>>(idx, kq_pos, k, P, nQ, nslots);
}

void launch_quant_kv(int bits, int fmt, const uint16_t* K, const uint16_t* V,
                     const int32_t* kq_pos, uint8_t* k_codes, float* k_scale, uint8_t* v_codes,
                     float* v_scale, int L, int nQ, int n_blocks, int blk_stride, int BHkv,
                     hipStream_t st) {
  if (n_blocks <= 0) return;
  dim3 kg(n_blocks, BHkv);
  if (fmt == HYQ_FMT_FP4 || fmt == HYQ_FMT_FP4Q6)   // the same E2M1 key/value codes
    quant_kv_kernel<4, HYQ_FMT_FP4><<<kg, kQuantThreads, 0, st>>>(
        K, V, kq_pos, k_codes, k_scale, v_codes, v_scale, L, nQ, blk_stride);
  else if (fmt == HYQ_FMT_FP8)
    quant_kv_kernel<8, HYQ_FMT_FP8><<<kg, kQuantThreads, 0, st>>>(
        K, V, kq_pos, k_codes, k_scale, v_codes, v_scale, L, nQ, blk_stride);
  else if (bits == 8)
    quant_kv_kernel<8, HYQ_FMT_INT><<<kg, kQuantThreads, 0, st>>>(
        K, V, kq_pos, k_codes, k_scale, v_codes, v_scale, L, nQ, blk_stride);
  else
    quant_kv_kernel<4, HYQ_FMT_INT><<<kg, kQuantThreads, 0, st>>>(
        K, V, kq_pos, k_codes, k_scale, v_codes, v_scale, L, nQ, blk_stride);
}

hipError_t launch_quantize(const hyq_shape& s, const hyq_sizes& z, const uint16_t* Q,
                           const uint16_t* K, const uint16_t* V, const int32_t* idx,
                           int8_t* q_codes, float* q_scale, uint8_t* k_codes, float* k_scale,
                           uint8_t* v_codes, float* v_scale, int32_t* kq_pos, hipStream_t st) {
  if (s.bits_kv == 16) return hipSuccess;
  const int BHkv = s.B * s.Hkv;
  launch_compact(idx, kq_pos, z.k, z.P, z.nQ, z.n_kvblk * kBlock, BHkv, st);
  dim3 qg(z.n_qblk, s.B * s.Hq);
  if (s.kv_format == HYQ_FMT_FP4Q6)   // E2M3 queries
    quant_q_kernel<HYQ_FMT_FP4Q6><<<qg, kQuantThreads, 0, st>>>(Q, q_codes, q_scale, s.L,
                                                                z.n_qblk);
  else if (s.kv_format != HYQ_FMT_INT)   // E4M3 queries for FP8 and FP4
    quant_q_kernel<HYQ_FMT_FP8><<<qg, kQuantThreads, 0, st>>>(Q, q_codes, q_scale, s.L, z.n_qblk);
  else
    quant_q_kernel<HYQ_FMT_INT><<<qg, kQuantThreads, 0, st>>>(Q, q_codes, q_scale, s.L, z.n_qblk);
  launch_quant_kv(s.bits_kv, s.kv_format, K, V, kq_pos, k_codes, k_scale, v_codes, v_scale, s.L,
                  z.nQ, z.n_kvblk, z.n_kvblk, BHkv, st);
  return hipGetLastError();
}

}  // namespace hyq
