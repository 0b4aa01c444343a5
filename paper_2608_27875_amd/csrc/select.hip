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
//
// The top-k works on order keys (an order-preserving map of the float
// scores to uint32):
//   - while the scores are produced, every workgroup counts its keys by
//     their top 12 bits in LDS and adds the non-empty bins to a histogram of
//     its KV head in the workspace;
//   - the classification kernel (1024 keys per workgroup) finds the bin
//     holding the k-th largest key from that histogram, writes a bitmap of
//     the positions in higher bins and appends the keys of that bin (about
//     1% of them) to a candidate list;
//   - one workgroup per KV head resolves the remaining 20 bits of the
//     threshold with two 10-bit radix passes over the candidates, then
//     writes the chosen positions in ascending order (ordered compaction of
//     the bitmaps; keys equal to the threshold lowest position first).
// The per-key work runs on many workgroups; the one workgroup per head
// touches only the candidates and one bitmap word per 32 positions.
#include "hyq_internal.h"

#pragma clang fp contract(off)

namespace hyq {
namespace {

constexpr int kHistShift = 32 - kSelHistBits;   // the histogram bin is key >> kHistShift

// Order-preserving map float -> uint32 (larger float, larger key); -0 -> +0.
__device__ __forceinline__ uint32_t order_key(float f) {
  uint32_t u = __float_as_uint(f + 0.0f);   // -0 + 0 = +0
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Per-head top-k scratch in the workspace: a 4-word header (the candidate
// count, then the bin of the k-th largest key and the keys still to take in
// it, as the classification finds them), the candidate list ((key, position) of the keys in the
// threshold's bin, at most P of them) and the bitmap of positions in higher
// bins (an even number of words).
__host__ __device__ __forceinline__ size_t topk_ws_words(int P) {
  return 4 + 2 * (size_t)P + (size_t)(P + 63) / 64 * 2;
}
struct TopkWs {
  uint32_t* ncand;   // header: [0] candidates, [1] bin, [2] keys of the bin to take
  uint2* cand;
  uint32_t* gt;
};
__device__ __forceinline__ TopkWs topk_ws(uint32_t* base, int bj, int P) {
  uint32_t* h = base + (size_t)bj * topk_ws_words(P);
  TopkWs w;
  w.ncand = h;
  w.cand = reinterpret_cast<uint2*>(h + 4);
  w.gt = h + 4 + 2 * (size_t)P;
  return w;
}

// One workgroup per (b, h, group of 16 channels), so that the short kernel
// spreads over the chip.  The head's t tail rows are staged through LDS
// kTailRows at a time (thread r loads the 32 bytes of row r); then lane d of
// the first wave adds the staged values of channel d in ascending row order,
// continuing from +0 over all t rows, which gives qpart[b][h][d].  The score
// kernel adds the g heads of a group in head order.  The first workgroup of
// each group also clears the key histogram and the top-k candidate count of
// its (b, j), which the next kernels fill.
constexpr int kTailRows = 256;
constexpr int kTailThreads = kTailRows;
constexpr int kTailCh = 16;   // channels per workgroup
__global__ void __launch_bounds__(kTailThreads)
tail_proxy_kernel(const uint16_t* __restrict__ Q, float* __restrict__ qpart,
                  uint32_t* __restrict__ hist, uint32_t* __restrict__ tws, int Hq, int Hkv, int L,
                  int t, int P) {
  __shared__ uint4 rows[kTailRows][kTailCh / 8];
  const int g = Hq / Hkv;
  const int bh = blockIdx.x, c0 = blockIdx.y * kTailCh;
  if (bh % g == 0 && blockIdx.y == 0) {
    uint32_t* hj = hist + (size_t)(bh / g) * kSelHistBins;
    for (int i = threadIdx.x; i < kSelHistBins; i += kTailThreads) hj[i] = 0u;
    if (threadIdx.x < 4) tws[(size_t)(bh / g) * topk_ws_words(P) + threadIdx.x] = 0u;
  }
  const uint16_t* q = Q + ((size_t)bh * L + (L - t)) * kHeadDim + c0;
  const int d = threadIdx.x;   // channel c0 + d for the adding lanes
  float a = 0.0f;
  for (int r0 = 0; r0 < t; r0 += kTailRows) {
    const int n = min(kTailRows, t - r0);
    // rows past the tail re-read its last row (never added)
    const uint4* src = reinterpret_cast<const uint4*>(
        q + (size_t)min(r0 + (int)threadIdx.x, t - 1) * kHeadDim);
    const uint4 v0 = src[0], v1 = src[1];
    rows[threadIdx.x][0] = v0;
    rows[threadIdx.x][1] = v1;
    __syncthreads();
    if (d < kTailCh) {
      const uint16_t* col = reinterpret_cast<const uint16_t*>(&rows[0][0]) + d;
      for (int i0 = 0; i0 < n; i0 += 32) {   // 32 LDS reads in flight, then the adds in order
        uint16_t x[32];
#pragma unroll
        for (int i = 0; i < 32; ++i) x[i] = col[(size_t)min(i0 + i, kTailRows - 1) * kTailCh];
#pragma unroll
        for (int i = 0; i < 32; ++i)
          if (i0 + i < n) a = a + bf16_bits_to_f32(x[i]);
      }
    }
    __syncthreads();
  }
  if (d < kTailCh) qpart[(size_t)bh * kHeadDim + c0 + d] = a;
}

// Workgroup-local key histogram (top kSelHistBits bits of the order key),
// flushed into the KV head's histogram in global memory.
constexpr int kHistThreads = 1024;         // hist_kernel: one key per thread
constexpr int kScoreThreads = 512;         // score_kernel: 64 keys per wave
constexpr int kScoreRows = kScoreThreads;  // keys per score workgroup

__device__ __forceinline__ void hist_clear(uint32_t* lh) {
  for (int i = threadIdx.x; i < kSelHistBins; i += blockDim.x) lh[i] = 0u;
}
__device__ __forceinline__ void hist_flush(const uint32_t* lh, uint32_t* __restrict__ gh) {
  for (int i = threadIdx.x; i < kSelHistBins; i += blockDim.x) {
    const uint32_t c = lh[i];
    if (c) atomicAdd(gh + i, c);
  }
}

// Lane exchange within groups of four lanes (DPP quad permutations).
__device__ __forceinline__ float xor1(float x) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0xB1, 0xF, 0xF, true));
}
__device__ __forceinline__ float xor2(float x) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0x4E, 0xF, 0xF, true));
}

// Scores of 512 prefix keys per workgroup (two workgroups per CU, so that one
// computes while the other loads), 64 per wave.  A key row is read
// by 4 lanes: lane c (0..3) of the row's group loads the 16-byte chunks c,
// c+4, c+8, c+12 (channels 8c.., 32+8c.., 64+8c.., 96+8c.., eight each), so
// one load instruction covers 16 rows, 64 contiguous bytes each.  The pinned
// fold then runs as a butterfly: the halving steps l + 64 and l + 32 are
// in-lane, steps 16 and 8 pair lane c with lane c^2 and c^1 (the lower lane
// of a pair holds v[l], its partner v[l + h]; float addition is
// commutative, so both lanes get the bits of v[l] + v[l + h]), and steps
// 4, 2, 1 are in-lane again.
__global__ void __launch_bounds__(kScoreThreads, 2)
score_kernel(const uint16_t* __restrict__ K, const float* __restrict__ qpart,
             float* __restrict__ S, uint32_t* __restrict__ hist, int g, int L, int P) {
  __shared__ uint32_t lh[kSelHistBins];
  __shared__ float4 qs[kHeadDim / 4];
  const int bj = blockIdx.x;   // consecutive workgroups take consecutive heads (see the launch)
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int c = lane & 3, rsub = lane >> 2;
  const int base = blockIdx.y * kScoreRows + w * 64;
  const uint4* Kb = reinterpret_cast<const uint4*>(K + (size_t)bj * L * kHeadDim);
  uint4 kr[4][4];   // [iteration][quarter q]: chunk c + 4q of row base + 16*it + rsub
#pragma unroll
  for (int it = 0; it < 4; ++it) {
    // rows past P load row P-1 (unconditional loads stay in flight together);
    // their scores are never stored
    const uint4* rp = Kb + (size_t)min(base + it * 16 + rsub, P - 1) * (kHeadDim / 8);
#pragma unroll
    for (int q = 0; q < 4; ++q) kr[it][q] = rp[c + 4 * q];
  }
  hist_clear(lh);
  if (threadIdx.x < kHeadDim) {   // qsum = the g head partials added in head order
    const float* pp = qpart + (size_t)bj * g * kHeadDim + threadIdx.x;
    float part[8];   // g <= 8; unconditional loads, all in flight
#pragma unroll
    for (int r = 0; r < 8; ++r) part[r] = pp[(size_t)min(r, g - 1) * kHeadDim];
    float a = part[0];
#pragma unroll
    for (int r = 1; r < 8; ++r)
      if (r < g) a = a + part[r];
    reinterpret_cast<float*>(qs)[threadIdx.x] = a;
  }
  __syncthreads();
  // qv[q][e] = qsum[32q + 8c + e]
  float qv[4][8];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const float4 a = qs[8 * q + 2 * c], b = qs[8 * q + 2 * c + 1];
    qv[q][0] = a.x; qv[q][1] = a.y; qv[q][2] = a.z; qv[q][3] = a.w;
    qv[q][4] = b.x; qv[q][5] = b.y; qv[q][6] = b.z; qv[q][7] = b.w;
  }

  float sv[4];
#pragma unroll
  for (int it = 0; it < 4; ++it) {
    float pr[4][8];   // products of channel 32q + 8c + e
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint32_t wq[4] = {kr[it][q].x, kr[it][q].y, kr[it][q].z, kr[it][q].w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        pr[q][2 * e] = qv[q][2 * e] * bf16_lo(wq[e]);
        pr[q][2 * e + 1] = qv[q][2 * e + 1] * bf16_hi(wq[e]);
      }
    }
    float v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float a = pr[0][e] + pr[2][e];   // step 64: l = 8c+e,    l + 64
      const float b = pr[1][e] + pr[3][e];   //          l = 32+8c+e, l + 64
      v[e] = a + b;                          // step 32: l = 8c+e,    l + 32
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = v[e] + xor2(v[e]);   // step 16
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = v[e] + xor1(v[e]);   // step 8
#pragma unroll
    for (int h = 4; h >= 1; h >>= 1)
#pragma unroll
      for (int e = 0; e < h; ++e) v[e] = v[e] + v[e + h];
    sv[it] = v[0];
  }
  // lane l takes the score of row base + l: iteration l/16, row group l%16
  float s = 0.0f;
#pragma unroll
  for (int it = 0; it < 4; ++it) {
    const float x = __shfl(sv[it], 4 * (lane & 15), 64);
    if ((lane >> 4) == it) s = x;
  }
  const int p = base + lane;
  if (p < P) {
    S[(size_t)bj * P + p] = s;
    atomicAdd(&lh[order_key(s) >> kHistShift], 1u);
  }
  __syncthreads();
  hist_flush(lh, hist + (size_t)bj * kSelHistBins);
}

// Clears the key histogram and the top-k candidate count of each head (one
// workgroup per head; the tail-proxy kernel does this on the other path).
__global__ void hist_zero_kernel(uint32_t* __restrict__ hist, uint32_t* __restrict__ tws, int P) {
  const int bj = blockIdx.x;
  for (int i = threadIdx.x; i < kSelHistBins; i += blockDim.x)
    hist[(size_t)bj * kSelHistBins + i] = 0u;
  if (threadIdx.x == 0) tws[(size_t)bj * topk_ws_words(P)] = 0u;
}

// Key histogram of scores computed elsewhere (the column-mass selector).
__global__ void __launch_bounds__(kHistThreads)
hist_kernel(const float* __restrict__ S, uint32_t* __restrict__ hist, int P) {
  __shared__ uint32_t lh[kSelHistBins];
  const int bj = blockIdx.x;
  hist_clear(lh);
  __syncthreads();
  const int p = blockIdx.y * kHistThreads + threadIdx.x;
  if (p < P) atomicAdd(&lh[order_key(S[(size_t)bj * P + p]) >> kHistShift], 1u);
  __syncthreads();
  hist_flush(lh, hist + (size_t)bj * kSelHistBins);
}

constexpr int kTopkThreads = 1024;
constexpr int kTopkWaves = kTopkThreads / 64;
constexpr int kDigitBits = 10;
constexpr int kDigitBins = 1 << kDigitBits;
static_assert(kSelHistBits + 2 * kDigitBits == 32, "bin + two digits cover the key");
static_assert(kSelHistBins == 4 * kTopkThreads, "four histogram bins per thread");
static_assert(kDigitBins == kTopkThreads, "one digit bin per thread");

struct TopkShared {
  uint32_t dig[kDigitBins];
  uint32_t wtot[kTopkWaves];
  uint32_t sel_bin;
  int sel_rem;
};

// Inclusive suffix sum over the workgroup's threads in thread order: the
// sum of x over this thread and every later one.
__device__ __forceinline__ uint32_t block_suffix(uint32_t x, TopkShared& sh) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  uint32_t s = x;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t y = __shfl_down(s, o, 64);
    if (lane + o < 64) s += y;
  }
  if (lane == 0) sh.wtot[w] = s;
  __syncthreads();
  uint32_t later = 0;
  for (int v = w + 1; v < kTopkWaves; ++v) later += sh.wtot[v];
  __syncthreads();
  return s + later;
}

// Exclusive prefix sum over the workgroup's threads in thread order; the
// sum over all threads goes to `total`.
__device__ __forceinline__ uint32_t block_prefix_excl(uint32_t x, TopkShared& sh,
                                                      uint32_t& total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  uint32_t s = x;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t y = __shfl_up(s, o, 64);
    if (lane >= o) s += y;
  }
  if (lane == 63) sh.wtot[w] = s;
  __syncthreads();
  uint32_t before = 0, all = 0;
  for (int v = 0; v < kTopkWaves; ++v) {
    const uint32_t t = sh.wtot[v];
    before += v < w ? t : 0u;
    all += t;
  }
  __syncthreads();
  total = all;
  return before + s - x;
}

// Thread t owns the n bins c[0..n) = bins n*t .. n*t+n-1 of an ascending
// histogram.  Finds the bin holding the need-th largest key and how many
// keys of that bin are still to take; the owning thread publishes both.
template <int N>
__device__ __forceinline__ void find_bin(const uint32_t (&c)[N], int need, TopkShared& sh) {
  uint32_t mine = 0;
#pragma unroll
  for (int e = 0; e < N; ++e) mine += c[e];
  const uint32_t suf = block_suffix(mine, sh);
  const uint32_t above = suf - mine;   // keys in the bins of later threads
  if (above < (uint32_t)need && (uint32_t)need <= suf) {
    uint32_t acc = above;
#pragma unroll
    for (int e = N - 1; e >= 0; --e) {
      if (acc + c[e] >= (uint32_t)need) {
        sh.sel_bin = (uint32_t)(N * threadIdx.x + e);
        sh.sel_rem = need - (int)acc;
        break;
      }
      acc += c[e];
    }
  }
  __syncthreads();
}

// The bin of the k-th largest key of head bj from its histogram.
__device__ __forceinline__ void hist_bin(const uint32_t* __restrict__ hist, int bj, int k,
                                         TopkShared& sh) {
  const uint4 h4 = reinterpret_cast<const uint4*>(hist + (size_t)bj * kSelHistBins)[threadIdx.x];
  const uint32_t hc[4] = {h4.x, h4.y, h4.z, h4.w};
  find_bin<4>(hc, k, sh);
}

// Classification, 1024 keys per workgroup (grid: head fastest, then key
// chunk; one key per thread, coalesced): every workgroup finds the bin of
// the k-th largest key from the histogram; a ballot per wave gives the 64
// positions' bits "in a higher bin" as two bitmap words; the keys of that
// bin are appended to the head's candidate list (one atomic reservation per
// wave).
__global__ void __launch_bounds__(kTopkThreads)
topk_classify_kernel(const float* __restrict__ S, const uint32_t* __restrict__ hist,
                     uint32_t* __restrict__ tws, int P, int k) {
  __shared__ TopkShared sh;
  const int bj = blockIdx.x;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int p = blockIdx.y * kTopkThreads + (int)threadIdx.x;
  const bool in = p < P;
  const uint32_t u = order_key(S[(size_t)bj * P + min(p, P - 1)]);   // in flight meanwhile
  hist_bin(hist, bj, k, sh);
  const uint32_t bin = sh.sel_bin;
  const TopkWs f = topk_ws(tws, bj, P);
  if (blockIdx.y == 0 && threadIdx.x == 0) {
    f.ncand[1] = bin;
    f.ncand[2] = (uint32_t)sh.sel_rem;
  }
  const uint32_t b = u >> kHistShift;
  const uint64_t mg = __ballot(in && b > bin);
  const uint64_t mc = __ballot(in && b == bin);
  const int x = (blockIdx.y * kTopkThreads + w * 64) / 32;   // word of this wave's first position
  if (lane == 0 && x * 32 < P)
    *reinterpret_cast<uint2*>(&f.gt[x]) = make_uint2((uint32_t)mg, (uint32_t)(mg >> 32));
  if (mc) {
    uint32_t base = 0;
    if (lane == 0) base = atomicAdd(f.ncand, (uint32_t)__popcll(mc));
    base = __shfl(base, 0, 64);
    const uint32_t r = __builtin_amdgcn_mbcnt_hi((uint32_t)(mc >> 32),
                                                 __builtin_amdgcn_mbcnt_lo((uint32_t)mc, 0u));
    if (in && b == bin && base + r < (uint32_t)P) f.cand[base + r] = make_uint2(u, (uint32_t)p);
  }
}

// Radix pass over the candidates whose bits above `shift + kDigitBits`
// equal `prefix`: histogram of the next 10-bit digit, then the digit holding
// the need-th largest of them.
__device__ __forceinline__ void cand_digit_pass(const uint2* cand, int nc, uint32_t prefix,
                                                int shift, int need, TopkShared& sh) {
  sh.dig[threadIdx.x] = 0u;
  __syncthreads();
  const int top = shift + kDigitBits;
  for (int c = threadIdx.x; c < nc; c += kTopkThreads) {
    const uint32_t key = cand[c].x;
    if ((key >> top) == prefix) atomicAdd(&sh.dig[(key >> shift) & (kDigitBins - 1)], 1u);
  }
  __syncthreads();
  const uint32_t c1[1] = {sh.dig[threadIdx.x]};
  __syncthreads();
  find_bin<1>(c1, need, sh);
}

// Final top-k, one workgroup per (b, j):
//  1. the bin of the k-th largest key (from the classification) and the
//     candidates into LDS: the first kCandLds list entries are loaded
//     together with the count (more candidates, in crowded or tied bins, are
//     read from the workspace instead);
//  2. two digit passes over the candidates give T and how many keys equal
//     to T to take;
//  3. per window of kMapWords bitmap words: candidates above T and equal to
//     T are marked in two LDS bitmaps; then, one word (32 positions) per
//     thread and round, the positions in higher bins plus the marked ones
//     above T plus the lowest positions equal to T are written in ascending
//     order.
constexpr int kCandLds = 2048;
constexpr int kMapWords = 4096;   // bitmap words per window (131072 positions)
__global__ void __launch_bounds__(kTopkThreads)
topk_final_kernel(uint32_t* __restrict__ tws, int32_t* __restrict__ idx, int P, int k) {
  __shared__ TopkShared sh;
  __shared__ uint2 lcand[kCandLds];
  __shared__ uint32_t xgt[kMapWords], xeq[kMapWords];
  const int bj = blockIdx.x;
  const TopkWs f = topk_ws(tws, bj, P);
  const uint4 hdr = *reinterpret_cast<const uint4*>(f.ncand);
  constexpr int kPre = kCandLds / kTopkThreads;
  uint2 pre[kPre];   // list entries loaded before the count is known (in bounds: P entries)
#pragma unroll
  for (int i = 0; i < kPre; ++i) pre[i] = f.cand[min((int)threadIdx.x + i * kTopkThreads, P - 1)];
  const int nc = (int)min(hdr.x, (uint32_t)P);
  const uint32_t bin = hdr.y;
  const int need = (int)hdr.z;
  const uint2* cand = f.cand;
  if (nc <= kCandLds) {
#pragma unroll
    for (int i = 0; i < kPre; ++i) lcand[threadIdx.x + i * kTopkThreads] = pre[i];
    cand = lcand;
    __syncthreads();
  }
  cand_digit_pass(cand, nc, bin, kDigitBits, need, sh);
  const uint32_t d1 = sh.sel_bin;
  cand_digit_pass(cand, nc, (bin << kDigitBits) | d1, 0, sh.sel_rem, sh);
  const uint32_t T = (bin << (2 * kDigitBits)) | (d1 << kDigitBits) | sh.sel_bin;
  const int need_eq = sh.sel_rem;   // keys equal to T to take, lowest positions first

  int32_t* out = idx + (size_t)bj * k;
  uint32_t o_base = 0, eq_base = 0;
  const int W = (P + 31) / 32;
  for (int m0 = 0; m0 < W; m0 += kMapWords) {
    const int m1 = min(W, m0 + kMapWords);
    for (int x = threadIdx.x; x < kMapWords; x += kTopkThreads) xgt[x] = xeq[x] = 0u;
    __syncthreads();
    for (int c = threadIdx.x; c < nc; c += kTopkThreads) {
      const uint2 e = cand[c];
      const int x = (int)(e.y >> 5);
      if (x < m0 || x >= m1) continue;
      const uint32_t bit = 1u << (e.y & 31);
      if (e.x > T) atomicOr(&xgt[x - m0], bit);
      else if (e.x == T) atomicOr(&xeq[x - m0], bit);
    }
    __syncthreads();
    for (int x0 = m0; x0 < m1; x0 += kTopkThreads) {
      const int x = x0 + (int)threadIdx.x;
      const bool ok = x < m1;
      uint32_t e = ok ? xeq[x - m0] : 0u;
      const uint32_t g = ok ? f.gt[x] | xgt[x - m0] : 0u;
      const int ne = __popc(e);
      uint32_t eq_tot;
      const int eq_before = (int)(eq_base + block_prefix_excl((uint32_t)ne, sh, eq_tot));
      int keep = max(0, min(ne, need_eq - eq_before));
      uint32_t kept = 0;
      for (; keep > 0; --keep) {   // the lowest `keep` positions equal to T
        const uint32_t low = e & (0u - e);
        kept |= low;
        e ^= low;
      }
      uint32_t sel = g | kept;
      uint32_t sel_tot;
      uint32_t o = o_base + block_prefix_excl((uint32_t)__popc(sel), sh, sel_tot);
      while (sel) {
        const int b = __builtin_ctz(sel);
        if (o < (uint32_t)k) out[o] = x * 32 + b;   // never more than k
        ++o;
        sel &= sel - 1u;
      }
      o_base += sel_tot;
      eq_base += eq_tot;
    }
    __syncthreads();   // the window's bitmaps are read before the next window clears them
  }
}

}  // namespace

size_t select_topk_ws_bytes(int BH, int P) { return (size_t)BH * topk_ws_words(P) * 4; }

hipError_t launch_select(const hyq_shape& s, const hyq_sizes& z, const uint16_t* Q,
                         const uint16_t* K, int32_t* idx, float* scores, float* qsum,
                         uint32_t* hist, uint32_t* tws, float* cm_ws, hipStream_t st) {
  if (z.k == 0) return hipSuccess;
  const int g = s.Hq / s.Hkv;
  const int t = s.window < s.L ? s.window : s.L;
  const int BH = s.B * s.Hkv;
  // (KV head, key chunk) with the head index fastest: workgroups are spread
  // over the XCDs round-robin, so with B*Hkv a multiple of 8 every chunk of a
  // head (and its final top-k workgroup) runs on one XCD and shares that
  // XCD's L2.
  if (s.selector == HYQ_SEL_COLMASS) {
    hist_zero_kernel<<<BH, 256, 0, st>>>(hist, tws, z.P);
    const hipError_t e = launch_colmass_scores(s, z, Q, K, scores, cm_ws, st);
    if (e != hipSuccess) return e;
    hist_kernel<<<dim3(BH, (z.P + kHistThreads - 1) / kHistThreads), kHistThreads, 0, st>>>(
        scores, hist, z.P);
  } else {
    tail_proxy_kernel<<<dim3(s.B * s.Hq, kHeadDim / kTailCh), kTailThreads, 0, st>>>(
        Q, qsum, hist, tws, s.Hq, s.Hkv, s.L, t, z.P);
    score_kernel<<<dim3(BH, (z.P + kScoreRows - 1) / kScoreRows), kScoreThreads, 0, st>>>(
        K, qsum, scores, hist, g, s.L, z.P);
  }
  const dim3 cg(BH, (z.P + kTopkThreads - 1) / kTopkThreads);
  topk_classify_kernel<<<cg, kTopkThreads, 0, st>>>(scores, hist, tws, z.P, z.k);
  topk_final_kernel<<<BH, kTopkThreads, 0, st>>>(tws, idx, z.P, z.k);
  return hipGetLastError();
}

}  // namespace hyq
