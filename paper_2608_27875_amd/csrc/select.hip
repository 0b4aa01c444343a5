// Vertical-line selection: Algorithm 1 (App. A.1, Vertical Token
// Identification) of HyQuant, GQA-native, one vertical set per KV head.
// (The exact column-mass score of eq. vl_score, HYQ_SEL_COLMASS, is computed
// in colmass.hip; the top-k below serves both.)
//
//   1. tail proxy   qsum[b][j] = sum over the g heads of the group and the
//                   last t = min(W, L) query rows (float32, pinned order);
//   2. scores       S[b][j][p] = qsum . K[b][j][p], p < P (pinned tree);
//   3. top-k        k largest S, ties to the lowest position, ascending.
//
// Every floating-point operation here is a separately rounded float32
// add or multiply in a fixed order, so the result is reproducible bit for
// bit; contraction into fused multiply-adds is disabled for this file.
#include "hyq_internal.h"

#pragma clang fp contract(off)

namespace hyq {
namespace {

constexpr int kTailBatch = 32;

// One workgroup per (b, j); thread (r, d) owns query head j*g + r and
// channel d.  Each thread adds its t tail values in ascending row order
// from +0 (loads are issued a batch at a time to hide latency); then the
// g per-head sums are added in head order.
__global__ void __launch_bounds__(1024)
tail_proxy_kernel(const uint16_t* __restrict__ Q, float* __restrict__ qsum,
                  int Hq, int Hkv, int L, int t) {
  extern __shared__ float part[];  // [g][D]
  const int g = Hq / Hkv;
  const int bj = blockIdx.x;
  const int b = bj / Hkv, j = bj % Hkv;
  const int r = threadIdx.x / kHeadDim, d = threadIdx.x % kHeadDim;
  const uint16_t* q = Q + ((size_t)(b * Hq + j * g + r) * L + (L - t)) * kHeadDim + d;
  float a = 0.0f;
  int i = 0;
  for (; i + kTailBatch <= t; i += kTailBatch) {
    uint32_t v[kTailBatch];
#pragma unroll
    for (int u = 0; u < kTailBatch; ++u) v[u] = q[(size_t)(i + u) * kHeadDim];
#pragma unroll
    for (int u = 0; u < kTailBatch; ++u) a = a + bf16_bits_to_f32(v[u]);
  }
  for (; i < t; ++i) a = a + bf16_bits_to_f32(q[(size_t)i * kHeadDim]);
  part[r * kHeadDim + d] = a;
  __syncthreads();
  if (r == 0) {
    float s = part[d];
    for (int rr = 1; rr < g; ++rr) s = s + part[rr * kHeadDim + d];
    qsum[(size_t)bj * kHeadDim + d] = s;
  }
}

// One thread per prefix key: products qsum[d] * K[p][d] rounded separately,
// then v[l] = prod[l] + prod[l + 64] and repeated halving 32 .. 1.
__global__ void __launch_bounds__(256)
score_kernel(const uint16_t* __restrict__ K, const float* __restrict__ qsum,
             float* __restrict__ S, int L, int P) {
  __shared__ float qs[kHeadDim];
  const int bj = blockIdx.y;
  if (threadIdx.x < kHeadDim) qs[threadIdx.x] = qsum[(size_t)bj * kHeadDim + threadIdx.x];
  __syncthreads();
  const int p = blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= P) return;
  const uint4* row = reinterpret_cast<const uint4*>(K + ((size_t)bj * L + p) * kHeadDim);
  uint4 lo[8], hi[8];
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    lo[u] = row[u];       // channels 0..63
    hi[u] = row[u + 8];   // channels 64..127
  }
  float v[64];
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    const uint32_t wl[4] = {lo[u].x, lo[u].y, lo[u].z, lo[u].w};
    const uint32_t wh[4] = {hi[u].x, hi[u].y, hi[u].z, hi[u].w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int l0 = u * 8 + e * 2;
      const float p0 = qs[l0] * bf16_lo(wl[e]);
      const float p1 = qs[l0 + 1] * bf16_hi(wl[e]);
      const float h0 = qs[l0 + 64] * bf16_lo(wh[e]);
      const float h1 = qs[l0 + 65] * bf16_hi(wh[e]);
      v[l0] = p0 + h0;
      v[l0 + 1] = p1 + h1;
    }
  }
#pragma unroll
  for (int h = 32; h >= 1; h >>= 1) {
#pragma unroll
    for (int l = 0; l < h; ++l) v[l] = v[l] + v[l + h];
  }
  S[(size_t)bj * P + p] = v[0];
}

// Order-preserving map float -> uint32 (larger float, larger key); -0 -> +0.
__device__ __forceinline__ uint32_t order_key(float f) {
  uint32_t u = __float_as_uint(f + 0.0f);   // -0 + 0 = +0
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

constexpr int kTopkThreads = 1024;
constexpr int kTopkWaves = kTopkThreads / 64;

// One workgroup per (b, j).  Radix select over the 32-bit order keys, 8 bits
// per pass (per-wave LDS histograms), finds the k-th largest key T and how
// many keys equal to T are taken (the lowest positions).  Then an ordered
// compaction writes the chosen positions ascending (below).
__global__ void __launch_bounds__(kTopkThreads)
topk_kernel(const float* __restrict__ S, int32_t* __restrict__ idx, int P, int k) {
  __shared__ uint32_t hist[kTopkWaves][256];
  __shared__ int w_gt[kTopkWaves], w_eq[kTopkWaves];
  __shared__ uint32_t sh_digit;
  __shared__ int sh_remaining;
  const int bj = blockIdx.x;
  const float* s = S + (size_t)bj * P;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;

  uint32_t prefix = 0, mask = 0;
  int remaining = k;  // how many of the keys matching `prefix` are still to take
  for (int shift = 24; shift >= 0; shift -= 8) {
    for (int i = threadIdx.x; i < kTopkWaves * 256; i += kTopkThreads) (&hist[0][0])[i] = 0;
    __syncthreads();
    for (int p = threadIdx.x; p < P; p += kTopkThreads) {
      const uint32_t u = order_key(s[p]);
      if ((u & mask) == prefix) atomicAdd(&hist[w][(u >> shift) & 255u], 1u);
    }
    __syncthreads();
    if (w == 0) {
      // lane owns bins 4*lane .. 4*lane+3; suffix sums from the top bin down
      uint32_t c[4];
      uint32_t mine = 0;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        uint32_t t = 0;
        for (int ww = 0; ww < kTopkWaves; ++ww) t += hist[ww][4 * lane + e];
        c[e] = t;
        mine += t;
      }
      // inclusive suffix sum over lanes: above[lane] = sum of bins >= 4*lane
      uint32_t suf = mine;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const uint32_t y = __shfl_down(suf, o, 64);
        if (lane + o < 64) suf += y;
      }
      const uint32_t above_lane = suf - mine;   // count in bins > 4*lane+3
      // the digit is in this lane's bins if above_lane < remaining <= suf
      if (above_lane < (uint32_t)remaining && (uint32_t)remaining <= suf) {
        uint32_t acc = above_lane;
        for (int e = 3; e >= 0; --e) {
          if (acc + c[e] >= (uint32_t)remaining) {
            sh_digit = 4 * lane + e;
            sh_remaining = remaining - (int)acc;
            break;
          }
          acc += c[e];
        }
      }
    }
    __syncthreads();
    prefix |= sh_digit << shift;
    mask |= 255u << shift;
    remaining = sh_remaining;
    __syncthreads();
  }
  const uint32_t T = prefix;
  const int need_eq = remaining;  // keys equal to T to take, lowest positions first

  // Ordered compaction: wave w owns positions [w*R, (w+1)*R) and reads them
  // 64 at a time (coalesced); a first sweep counts its keys above and equal to
  // T, the wave totals give each wave its output offset and its share of the
  // keys equal to T, a second sweep writes the positions in order.
  const int R = ((P + kTopkWaves - 1) / kTopkWaves + 63) & ~63;
  const int q0 = min(P, w * R), q1 = min(P, q0 + R);
  int gtc = 0, eqc = 0;   // wave-uniform
  for (int b = q0; b < q1; b += 64) {
    const int p = b + lane;
    const uint32_t u = p < q1 ? order_key(s[p]) : 0u;
    gtc += (int)__popcll(__ballot(p < q1 && u > T));
    eqc += (int)__popcll(__ballot(p < q1 && u == T));
  }
  if (lane == 0) {
    w_gt[w] = gtc;
    w_eq[w] = eqc;
  }
  __syncthreads();
  int o = 0, eq_before = 0;
  for (int v = 0; v < w; ++v) {
    o += w_gt[v] + max(0, min(w_eq[v], need_eq - eq_before));
    eq_before += w_eq[v];
  }
  const int take_eq = max(0, min(eqc, need_eq - eq_before));
  int32_t* out = idx + (size_t)bj * k;
  int eq_seen = 0;
  for (int b = q0; b < q1; b += 64) {
    const int p = b + lane;
    const bool in = p < q1;
    const uint32_t u = in ? order_key(s[p]) : 0u;
    const bool is_eq = in && u == T;
    const uint64_t meq = __ballot(is_eq);
    const int eq_rank = eq_seen + (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(meq >> 32),
                                      __builtin_amdgcn_mbcnt_lo((uint32_t)meq, 0u));
    const bool sel = in && (u > T || (is_eq && eq_rank < take_eq));
    const uint64_t msel = __ballot(sel);
    if (sel) {
      const int pos = o + (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(msel >> 32),
                                                         __builtin_amdgcn_mbcnt_lo((uint32_t)msel, 0u));
      if (pos < k) out[pos] = p;   // never more than k (guards a malformed threshold)
    }
    o += (int)__popcll(msel);
    eq_seen += (int)__popcll(meq);
  }
}

}  // namespace

hipError_t launch_select(const hyq_shape& s, const hyq_sizes& z, const uint16_t* Q,
                         const uint16_t* K, int32_t* idx, float* scores, float* qsum,
                         float* cm_ws, hipStream_t st) {
  if (z.k == 0) return hipSuccess;
  const int g = s.Hq / s.Hkv;
  const int t = s.window < s.L ? s.window : s.L;
  const int BH = s.B * s.Hkv;
  if (s.selector == HYQ_SEL_COLMASS) {
    const hipError_t e = launch_colmass_scores(s, z, Q, K, scores, cm_ws, st);
    if (e != hipSuccess) return e;
  } else {
    tail_proxy_kernel<<<BH, g * kHeadDim, g * kHeadDim * sizeof(float), st>>>(Q, qsum, s.Hq,
                                                                                s.Hkv, s.L, t);
    dim3 sg((z.P + 255) / 256, BH);
    score_kernel<<<sg, 256, 0, st>>>(K, qsum, scores, s.L, z.P);
  }
  topk_kernel<<<BH, kTopkThreads, 0, st>>>(scores, idx, z.P, z.k);
  return hipGetLastError();
}

}  // namespace hyq
