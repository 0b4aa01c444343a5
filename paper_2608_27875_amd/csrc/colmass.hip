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
//   colmass_sum_kernel   per 64 prefix keys, the probabilities of every
//                        considered row summed (prefix keys precede every
//                        tail row, so no mask).
// Both passes are bf16 MFMA products with keys as rows (S^T = K Q^T), the
// exponentials in float32.  The top-k then follows with the selection's own
// kernel (same budget and tie rule).
#include "hyq_internal.h"

namespace hyq {
namespace {

typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));

constexpr int kCmWaves = 4;
constexpr int kCmThreads = kCmWaves * 64;
constexpr float kLog2e = 1.4426950408889634f;

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

// Pass 1: one workgroup per (query tile of 32 rows of one head, key split);
// wave w takes the split's key tiles w, w + 4, ...  Writes the partial
// (max, sum) of every row in the log2 domain.
__global__ void __launch_bounds__(kCmThreads)
colmass_lse_kernel(const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
                   float* __restrict__ part, CmGeom gm) {
  __shared__ float sm_m[kCmWaves][32], sm_l[kCmWaves][32];
  const int bj = blockIdx.y;
  const int qt = blockIdx.x / gm.ks, split = blockIdx.x % gm.ks;
  const int b = bj / gm.Hkv, j = bj % gm.Hkv;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63, col = lane & 31, lh = lane >> 5;
  const int r = qt / gm.ntr, i0 = (qt % gm.ntr) * 32;
  const int row0 = gm.L - gm.t + i0;                 // first sequence row of the tile
  const int qi = i0 + col;                           // this lane's tail row
  const bool qok = qi < gm.t;
  const int qrow = gm.L - gm.t + (qok ? qi : 0);
  const uint16_t* qp = Q + (((size_t)b * gm.Hq + (size_t)j * gm.g + r) * gm.L + qrow) * kHeadDim;
  const uint16_t* Kh = K + (size_t)bj * gm.L * kHeadDim;
  v8bf qb[8];
#pragma unroll
  for (int s = 0; s < 8; ++s) qb[s] = frag_bf16(qp, s, lh);

  // keys [0, last_key] are seen by some row of the tile
  const int last_key = min(gm.L - 1, row0 + 31);
  const int nkt = last_key / 32 + 1;
  float m = -INFINITY, l = 0.0f;
  const int kstep = gm.ks * kCmWaves;
  // K fragments of tile kt (loaded at a clamped index past the last tile)
  auto load_k = [&](v8bf (&f)[8], int kt) {
    const int krow = min(min(kt, nkt - 1) * 32 + col, gm.L - 1);
    const uint16_t* kp = Kh + (size_t)krow * kHeadDim;
#pragma unroll
    for (int st = 0; st < 8; ++st) f[st] = frag_bf16(kp, st, lh);
  };
  auto tile = [&](const v8bf (&kf)[8], int kt) {
    __builtin_amdgcn_sched_barrier(0);
    const int key0 = kt * 32;
    v16f s = {};
#pragma unroll
    for (int st = 0; st < 8; ++st)
      s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[st], qb[st], s, 0, 0, 0);
    float y[16];
    const bool diag = key0 + 31 > row0;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int key = key0 + (e >> 2) * 8 + lh * 4 + (e & 3);
      const bool vis = !diag || (key <= qrow && key < gm.L);
      y[e] = vis ? s[e] * gm.c : -INFINITY;
    }
    float mt = y[0];
#pragma unroll
    for (int e = 1; e < 16; ++e) mt = fmaxf(mt, y[e]);
    const float mn = fmaxf(m, mt);
    if (mn > -INFINITY) {
      float ps = 0.0f;
#pragma unroll
      for (int e = 0; e < 16; ++e) ps += __builtin_amdgcn_exp2f(y[e] - mn);
      l = l * __builtin_amdgcn_exp2f(m - mn) + ps;
      m = mn;
    }
    __builtin_amdgcn_sched_barrier(0);
  };
  // two register sets alternate: the next tile's fragments load while one
  // tile is computed, with no register copy between tiles
  v8bf k0[8], k1[8];
  int kt = split * kCmWaves + w;
  load_k(k0, kt);
  for (; kt + kstep < nkt; kt += 2 * kstep) {
    load_k(k1, kt + kstep);
    tile(k0, kt);
    load_k(k0, kt + 2 * kstep);
    tile(k1, kt + kstep);
  }
  if (kt < nkt) tile(k0, kt);
  // the two lane halves hold the same row, different keys
  const float mo = __shfl_xor(m, 32, 64), lo = __shfl_xor(l, 32, 64);
  const float M = fmaxf(m, mo);
  const float Lsum = M > -INFINITY ? l * __builtin_amdgcn_exp2f(m - M) + lo * __builtin_amdgcn_exp2f(mo - M) : 0.0f;
  if (lh == 0) {
    sm_m[w][col] = M;
    sm_l[w][col] = Lsum;
  }
  __syncthreads();
  if (threadIdx.x < 32) {
    float Mw = sm_m[0][col];
#pragma unroll
    for (int v = 1; v < kCmWaves; ++v) Mw = fmaxf(Mw, sm_m[v][col]);
    float Lw = 0.0f;
    if (Mw > -INFINITY) {
#pragma unroll
      for (int v = 0; v < kCmWaves; ++v) Lw += sm_l[v][col] * __builtin_amdgcn_exp2f(sm_m[v][col] - Mw);
    }
    const int nq = gm.g * gm.ntr * 32;
    float* dst = part + (((size_t)bj * gm.ks + split) * nq + qt * 32 + col) * 2;
    dst[0] = Mw;
    dst[1] = Lw;
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

// Pass 2: one workgroup per 64 prefix keys; wave w takes the query tiles
// w, w + 4, ...  Each lane accumulates the probabilities of its 16 keys of
// each 32-key half over its queries; lanes and waves are summed at the end.
__global__ void __launch_bounds__(kCmThreads)
colmass_sum_kernel(const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
                   const float* __restrict__ lse, float* __restrict__ S, CmGeom gm) {
  extern __shared__ float sh[];                  // lse of every query, then the reduction
  const int bj = blockIdx.y;
  const int b = bj / gm.Hkv, j = bj % gm.Hkv;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63, col = lane & 31, lh = lane >> 5;
  const int nq = gm.g * gm.ntr * 32;
  for (int q = threadIdx.x; q < nq; q += kCmThreads) sh[q] = lse[(size_t)bj * nq + q];
  const int key0 = blockIdx.x * 64;
  const uint16_t* Kh = K + (size_t)bj * gm.L * kHeadDim;
  v8bf ka[2][8];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int krow = min(key0 + h * 32 + col, gm.P - 1);
#pragma unroll
    for (int s = 0; s < 8; ++s) ka[h][s] = frag_bf16(Kh + (size_t)krow * kHeadDim, s, lh);
  }
  __syncthreads();
  float acc[2][16];
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[h][e] = 0.0f;
  const int nqt = gm.g * gm.ntr;
  auto load_q = [&](v8bf (&f)[8], int qt) {
    qt = min(qt, nqt - 1);
    const int r = qt / gm.ntr, i = (qt % gm.ntr) * 32 + col;
    const int qrow = gm.L - gm.t + min(i, gm.t - 1);
    const uint16_t* qp = Q + (((size_t)b * gm.Hq + (size_t)j * gm.g + r) * gm.L + qrow) * kHeadDim;
#pragma unroll
    for (int st = 0; st < 8; ++st) f[st] = frag_bf16(qp, st, lh);
  };
  auto qtile = [&](const v8bf (&qf)[8], int qt) {
    __builtin_amdgcn_sched_barrier(0);
    const float nl = -sh[qt * 32 + col];        // -inf for padding rows
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      v16f s = {};
#pragma unroll
      for (int st = 0; st < 8; ++st)
        s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[h][st], qf[st], s, 0, 0, 0);
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[h][e] += __builtin_amdgcn_exp2f(__builtin_fmaf(s[e], gm.c, nl));
    }
    __builtin_amdgcn_sched_barrier(0);
  };
  v8bf q0[8], q1[8];
  int qt = w;
  load_q(q0, qt);
  for (; qt + kCmWaves < nqt; qt += 2 * kCmWaves) {
    load_q(q1, qt + kCmWaves);
    qtile(q0, qt);
    load_q(q0, qt + 2 * kCmWaves);
    qtile(q1, qt + kCmWaves);
  }
  if (qt < nqt) qtile(q0, qt);
  // sum over the 32 query lanes of each half (same keys), then over waves
  __syncthreads();
  // each of the 64 keys belongs to one lane half: (h, e, lh) -> key
  // h*32 + (e/4)*8 + lh*4 + e%4, every key exactly once
  float* red = sh;                               // [kCmWaves][64 keys]
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      float v = acc[h][e];
#pragma unroll
      for (int o = 16; o >= 1; o >>= 1) v += __shfl_xor(v, o, 32);
      if (col == 0) red[w * 64 + h * 32 + (e >> 2) * 8 + lh * 4 + (e & 3)] = v;
    }
  __syncthreads();
  if (threadIdx.x < 64) {
    const int key = key0 + threadIdx.x;
    float v = 0.0f;
#pragma unroll
    for (int ww = 0; ww < kCmWaves; ++ww) v += red[ww * 64 + threadIdx.x];
    if (key < gm.P) S[(size_t)bj * gm.P + key] = v;
  }
}

}  // namespace

size_t colmass_ws_bytes(const hyq_shape& s) {
  const int t = s.window < s.L ? s.window : s.L;
  const size_t nq = (size_t)(s.Hq / s.Hkv) * ((t + 31) / 32) * 32;
  const size_t BH = (size_t)s.B * s.Hkv;
  return BH * nq * (2 * kColmassSplits + 1) * sizeof(float);
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
  gm.ks = kColmassSplits;
  gm.c = kLog2e / sqrtf((float)kHeadDim);
  const int BH = s.B * s.Hkv;
  const int nq = gm.g * gm.ntr * 32;
  float* part = ws;
  float* lse = ws + (size_t)BH * nq * 2 * kColmassSplits;
  colmass_lse_kernel<<<dim3(gm.g * gm.ntr * gm.ks, BH), kCmThreads, 0, st>>>(Q, K, part, gm);
  colmass_merge_kernel<<<dim3((nq + 255) / 256, BH), 256, 0, st>>>(part, lse, gm);
  const size_t shbytes = (size_t)(nq > kCmWaves * 64 ? nq : kCmWaves * 64) * sizeof(float);
  colmass_sum_kernel<<<dim3((z.P + 63) / 64, BH), kCmThreads, shbytes, st>>>(Q, K, lse, scores, gm);
  return hipGetLastError();
}

}  // namespace hyq
