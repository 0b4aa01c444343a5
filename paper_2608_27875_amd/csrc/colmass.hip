// Exact column-mass score of the vertical-line selection: eq. (vl_score) and
// eq. (vl_topk) of Section 4.1 of HyQuant.
//
//   S[b][j][k] = sum over the considered queries of their attention
//                probability on key k, k < P,
//
// the considered queries being the tail rows [L - t, L), t = min(W, L), of
// the g query heads of KV head j (the rows Algorithm 1 summarizes), each
// probability the causal softmax of alpha * <q, k> over keys <= the row.
// Two passes over the keys (the normalizer of a row is needed before any of
// its probabilities):
//   colmass_lse_kernel   per query row, log2-sum-exp over its keys, split
//                        over the key axis into partials;
//   colmass_merge_kernel the partials of each row merged;
//   colmass_sum_kernel   per prefix key, the probabilities of every
//                        considered row summed (prefix keys precede every
//                        tail row, so no mask).
// Both passes are bf16 MFMA products with keys as rows (S^T = K Q^T), the
// exponentials in float32.  The operand that every wave of a workgroup needs
// (key tiles in pass 1, query tiles in pass 2) is staged once per workgroup
// in LDS, double-buffered through registers, so the L2 traffic is that of
// one workgroup per 8 query tiles (pass 1) or per 512 keys (pass 2).  The
// top-k then follows with the selection's own kernel (same budget and tie
// rule).
#include "hyq_internal.h"

namespace hyq {
namespace {

typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef unsigned v4u __attribute__((ext_vector_type(4)));

constexpr int kCmWaves = 8;
constexpr int kCmThreads = kCmWaves * 64;
constexpr int kCmSplits = 8;              // key-axis splits of pass 1
constexpr float kLog2e = 1.4426950408889634f;
constexpr int kRowPitch = kHeadDim * 2 + 16;   // bytes per staged bf16 row (+16: bank shift)
constexpr int kStageRows = 64;                 // rows per LDS stage (keys or query rows)
constexpr int kStageBytes = kStageRows * kRowPitch;

// Query q of KV head bj (q < g * ntr * 32): head r = q / (ntr * 32), tail row
// i = q % (ntr * 32) (valid when i < t), sequence row L - t + i.
struct CmGeom {
  int Hq, Hkv, g, L, t, ntr, P, ks;
  float c;   // alpha * log2(e)
};

// 32 x 16 bf16 A/B fragment of a row-major [rows][128] bf16 matrix: lane l
// takes row l%32, k-elements 16*step + 8*(l/32) .. +8.
__device__ __forceinline__ v8bf frag_bf16(const uint16_t* row, int step, int lh) {
  return *reinterpret_cast<const v8bf*>(row + step * 16 + lh * 8);
}
__device__ __forceinline__ v8bf frag_lds(const uint8_t* buf, int row, int step, int lh) {
  return *reinterpret_cast<const v8bf*>(buf + row * kRowPitch + (step * 16 + lh * 8) * 2);
}

// 64 rows of 256 bytes (rows clamped to [0, nrows)), 32 bytes per thread:
// thread t takes row t / 8, bytes 32 * (t % 8) .. +32.
__device__ __forceinline__ void stage_rows_load(v4u (&r)[2], const uint16_t* base, int row0,
                                                int nrows) {
  const int t = threadIdx.x, row = min(row0 + (t >> 3), nrows - 1);
  const v4u* p = reinterpret_cast<const v4u*>(base + (size_t)row * kHeadDim) + (t & 7) * 2;
  r[0] = p[0];
  r[1] = p[1];
}
__device__ __forceinline__ void stage_rows_store(uint8_t* buf, const v4u (&r)[2]) {
  const int t = threadIdx.x;
  v4u* d = reinterpret_cast<v4u*>(buf + (t >> 3) * kRowPitch + (t & 7) * 32);
  d[0] = r[0];
  d[1] = r[1];
}

// Pass 1: one workgroup per (8 query tiles of 32 rows, key split); wave w
// owns query tile 8*blockIdx.x/ks + w and scans every key of the split, 64
// at a time from LDS.  Writes the partial (max, sum) of every row in the
// log2 domain.
__global__ void __launch_bounds__(kCmThreads)
colmass_lse_kernel(const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
                   float* __restrict__ part, CmGeom gm) {
  __shared__ __attribute__((aligned(16))) uint8_t kbuf[2][kStageBytes];
  const int bj = blockIdx.y;
  const int grp = blockIdx.x / gm.ks, split = blockIdx.x % gm.ks;
  const int b = bj / gm.Hkv, j = bj % gm.Hkv;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63, col = lane & 31, lh = lane >> 5;
  const int nqt = gm.g * gm.ntr;
  const int qt = grp * kCmWaves + w;
  const bool wave_ok = qt < nqt;
  const int qtc = wave_ok ? qt : nqt - 1;
  const int r = qtc / gm.ntr, i0 = (qtc % gm.ntr) * 32;
  const int row0 = gm.L - gm.t + i0;                 // first sequence row of the wave's tile
  const int qi = i0 + col;                           // this lane's tail row
  const int qrow = gm.L - gm.t + min(qi, gm.t - 1);
  const uint16_t* qp = Q + (((size_t)b * gm.Hq + (size_t)j * gm.g + r) * gm.L + qrow) * kHeadDim;
  const uint16_t* Kh = K + (size_t)bj * gm.L * kHeadDim;
  v8bf qb[8];
#pragma unroll
  for (int st = 0; st < 8; ++st) qb[st] = frag_bf16(qp, st, lh);

  // every key [0, L) in 64-key stages (the tail rows end at L - 1; keys past
  // a row are masked in the stages that reach beyond the wave's first row)
  const int nst = (gm.L - 1) / kStageRows + 1;
  const int chunk = (nst + gm.ks - 1) / gm.ks;
  const int s0 = split * chunk, s1 = min(nst, s0 + chunk);
  float m = -INFINITY, l = 0.0f;
  if (s0 < s1) {
    v4u rg[2];
    stage_rows_load(rg, Kh, s0 * kStageRows, gm.L);
    stage_rows_store(kbuf[0], rg);
    __syncthreads();
    for (int sg = s0; sg < s1; ++sg) {
      const uint8_t* cur = kbuf[(sg - s0) & 1];
      if (sg + 1 < s1) stage_rows_load(rg, Kh, (sg + 1) * kStageRows, gm.L);
      const int key0 = sg * kStageRows;
      const bool diag = key0 + kStageRows - 1 > row0;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        v16f s = {};
#pragma unroll
        for (int st = 0; st < 8; ++st)
          s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(frag_lds(cur, h * 32 + col, st, lh), qb[st],
                                                      s, 0, 0, 0);
        if (diag) {   // only the stages that reach past the wave's first row
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const int key = key0 + h * 32 + (e >> 2) * 8 + lh * 4 + (e & 3);
            if (!(key <= qrow && key < gm.L)) s[e] = -INFINITY;
          }
        }
        // the logits are s * c (c > 0): the running max moves with the raw
        // maximum, and each weight is one fused multiply-add and exp2
        float sm = fmaxf(fmaxf(s[0], s[1]), s[2]);
#pragma unroll
        for (int e = 3; e < 15; e += 2) sm = fmaxf(fmaxf(sm, s[e]), s[e + 1]);
        sm = fmaxf(sm, s[15]);
        const float mn = fmaxf(m, sm * gm.c);
        if (mn > -INFINITY) {
          float ps = 0.0f;
#pragma unroll
          for (int e = 0; e < 16; ++e) ps += __builtin_amdgcn_exp2f(__builtin_fmaf(s[e], gm.c, -mn));
          l = l * __builtin_amdgcn_exp2f(m - mn) + ps;
          m = mn;
        }
      }
      if (sg + 1 < s1) stage_rows_store(kbuf[(sg - s0 + 1) & 1], rg);
      __syncthreads();
    }
  }
  // the two lane halves hold the same row, different keys
  const float mo = __shfl_xor(m, 32, 64), lo = __shfl_xor(l, 32, 64);
  const float M = fmaxf(m, mo);
  const float Lsum = M > -INFINITY ? l * __builtin_amdgcn_exp2f(m - M) + lo * __builtin_amdgcn_exp2f(mo - M) : 0.0f;
  if (wave_ok && lh == 0) {
    const int nq = nqt * 32;
    float* dst = part + (((size_t)bj * gm.ks + split) * nq + qt * 32 + col) * 2;
    dst[0] = M;
    dst[1] = Lsum;
  }
}

// The partials of each query row merged into log2(sum of 2^y) (+inf for
// padding rows, so that their probabilities are 0 in pass 2).
__global__ void __launch_bounds__(256)
colmass_merge_kernel(const float* __restrict__ part, float* __restrict__ lse, CmGeom gm) {
  const int bj = blockIdx.y;
  const int nq = gm.g * gm.ntr * 32;
  const int q = blockIdx.x * 256 + threadIdx.x;
  if (q >= nq) return;
  const bool ok = (q % (gm.ntr * 32)) < gm.t;
  float M = -INFINITY;
  for (int s = 0; s < gm.ks; ++s) M = fmaxf(M, part[(((size_t)bj * gm.ks + s) * nq + q) * 2]);
  float L = 0.0f;
  for (int s = 0; s < gm.ks; ++s) {
    const float* p = part + (((size_t)bj * gm.ks + s) * nq + q) * 2;
    if (p[0] > -INFINITY) L += p[1] * __builtin_amdgcn_exp2f(p[0] - M);
  }
  lse[(size_t)bj * nq + q] = ok && L > 0.0f ? M + __builtin_amdgcn_logf(L) : INFINITY;
}

// Pass 2: one workgroup per 512 prefix keys, wave w owning keys 64w .. +64
// (two 32-key halves, fragments in registers); every query tile streams
// through LDS, two at a time, with the normalizers of its rows.  Each lane
// accumulates the probabilities of its 16 keys of each half over its
// queries; the 32 query lanes are summed at the end.
__global__ void __launch_bounds__(kCmThreads)
colmass_sum_kernel(const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
                   const float* __restrict__ lse, float* __restrict__ S, CmGeom gm) {
  __shared__ __attribute__((aligned(16))) uint8_t qbuf[2][kStageBytes];
  __shared__ float lbuf[2][kStageRows];
  const int bj = blockIdx.y;
  const int b = bj / gm.Hkv, j = bj % gm.Hkv;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63, col = lane & 31, lh = lane >> 5;
  const int nqt = gm.g * gm.ntr, nq = nqt * 32;
  const int key0 = blockIdx.x * (kCmWaves * 64) + w * 64;
  const uint16_t* Kh = K + (size_t)bj * gm.L * kHeadDim;
  v8bf ka[2][8];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int krow = min(key0 + h * 32 + col, gm.P - 1);
#pragma unroll
    for (int st = 0; st < 8; ++st) ka[h][st] = frag_bf16(Kh + (size_t)krow * kHeadDim, st, lh);
  }
  float acc[2][16];
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[h][e] = 0.0f;

  // stage u holds query rows 64u .. 64u + 63 of the bj's nq rows (2 tiles):
  // row q is (head q / (ntr*32), tail row q % (ntr*32)), clamped to the tail
  const int nsg = (nq + kStageRows - 1) / kStageRows;
  auto load = [&](v4u (&rg)[2], float& lv, int u) {
    const int t = threadIdx.x, q = min(u * kStageRows + (t >> 3), nq - 1);
    const int r = q / (gm.ntr * 32), i = min(q % (gm.ntr * 32), gm.t - 1);
    const v4u* p = reinterpret_cast<const v4u*>(
        Q + (((size_t)b * gm.Hq + (size_t)j * gm.g + r) * gm.L + gm.L - gm.t + i) * kHeadDim) +
        (t & 7) * 2;
    rg[0] = p[0];
    rg[1] = p[1];
    lv = lse[(size_t)bj * nq + min(u * kStageRows + (t & 63), nq - 1)];
  };
  auto store = [&](int buf, const v4u (&rg)[2], float lv) {
    stage_rows_store(qbuf[buf], rg);
    if (threadIdx.x < kStageRows) lbuf[buf][threadIdx.x] = lv;
  };
  v4u rg[2];
  float lv;
  load(rg, lv, 0);
  store(0, rg, lv);
  __syncthreads();
  for (int u = 0; u < nsg; ++u) {
    const int cb = u & 1;
    if (u + 1 < nsg) load(rg, lv, u + 1);
#pragma unroll
    for (int half = 0; half < 2; ++half) {   // the two query tiles of the stage
      const int qrow = half * 32 + col;
      // padding rows (beyond nq, or tail rows >= t) carry lse = +inf: weight 0
      const float nl = u * kStageRows + qrow < nq ? -lbuf[cb][qrow] : -INFINITY;
      v8bf qf[8];
#pragma unroll
      for (int st = 0; st < 8; ++st) qf[st] = frag_lds(qbuf[cb], qrow, st, lh);
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        v16f s = {};
#pragma unroll
        for (int st = 0; st < 8; ++st)
          s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[h][st], qf[st], s, 0, 0, 0);
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[h][e] += __builtin_amdgcn_exp2f(__builtin_fmaf(s[e], gm.c, nl));
      }
    }
    if (u + 1 < nsg) store(cb ^ 1, rg, lv);
    __syncthreads();
  }
  // sum over the 32 query lanes of each half (same keys); each of the 64 keys
  // of the wave belongs to one (h, e, lh): key h*32 + (e/4)*8 + lh*4 + e%4
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      float v = acc[h][e];
#pragma unroll
      for (int o = 16; o >= 1; o >>= 1) v += __shfl_xor(v, o, 32);
      const int key = key0 + h * 32 + (e >> 2) * 8 + lh * 4 + (e & 3);
      if (col == 0 && key < gm.P) S[(size_t)bj * gm.P + key] = v;
    }
}

}  // namespace

size_t colmass_ws_bytes(const hyq_shape& s) {
  const int t = s.window < s.L ? s.window : s.L;
  const size_t nq = (size_t)(s.Hq / s.Hkv) * ((t + 31) / 32) * 32;
  const size_t BH = (size_t)s.B * s.Hkv;
  return BH * nq * (2 * kCmSplits + 1) * sizeof(float);
}

hipError_t launch_colmass_scores(const hyq_shape& s, const hyq_sizes& z, const uint16_t* Q,
                                 const uint16_t* K, float* scores, float* ws, hipStream_t st) {
  CmGeom gm;
  gm.Hq = s.Hq;
  gm.Hkv = s.Hkv;
  gm.g = s.Hq / s.Hkv;
  gm.L = s.L;
  gm.t = s.window < s.L ? s.window : s.L;
  gm.ntr = (gm.t + 31) / 32;
  gm.P = z.P;
  gm.ks = kCmSplits;
  gm.c = kLog2e / sqrtf((float)kHeadDim);
  const int BH = s.B * s.Hkv;
  const int nq = gm.g * gm.ntr * 32;
  float* part = ws;
  float* lse = ws + (size_t)BH * nq * 2 * kCmSplits;
  const int ngrp = (gm.g * gm.ntr + kCmWaves - 1) / kCmWaves;
  colmass_lse_kernel<<<dim3(ngrp * gm.ks, BH), kCmThreads, 0, st>>>(Q, K, part, gm);
  colmass_merge_kernel<<<dim3((nq + 255) / 256, BH), 256, 0, st>>>(part, lse, gm);
  colmass_sum_kernel<<<dim3((z.P + kCmWaves * 64 - 1) / (kCmWaves * 64), BH), kCmThreads, 0, st>>>(
      Q, K, lse, scores, gm);
  return hipGetLastError();
}

}  // namespace hyq
