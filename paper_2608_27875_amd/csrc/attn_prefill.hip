// Hybrid-precision causal prefill attention: Algorithm 2, Stage 3 (App. A.2)
// and eq. (prefill_hybrid) of Section 4.2 of HyQuant.
//
// One workgroup = one KV head (b, j) x one tile of 32 query rows; wave w of
// the workgroup owns query head j*g + w (the g heads of a GQA group share
// every K/V tile staged in LDS).  Each wave keeps one online-softmax state
// per query row and scans
//   segment A: the quantized keys (compacted K_Q order) in tiles of 64 =
//              one quantization block: S^T = K_codes * Qcodes^T with the int8
//              MFMA (exact int32), logits scaled by alpha*log2(e)*sQ*sK;
//              P V with the f16 MFMA on the V codes (exact in f16);
//   segments B and C: the full-precision keys (vertical lines, then the
//              window), 64 at a time gathered into LDS: S^T with the bf16
//              MFMA; P V with the bf16 MFMA on bf16 V, P split into a high
//              and a low bf16 part so that P keeps ~16 bits.
// Causality is by original key position in every segment.
//
// Register layout (32x32 MFMA, wave64): lane l, accumulator register r holds
// row (r/4)*8 + (l/32)*4 + r%4 and column l%32.  With keys as rows (S^T),
// each lane owns one query (column) and 16 keys per 32-key half; those 16
// values are reused directly as the B operand of the P V product, and the
// V^T tile in LDS stores each 16-key group in the matching order
// [0-3, 8-11, 4-7, 12-15].
//
// V scales are folded into the exponent: P' = 2^(y - m + log2(sV/sVref))
// with sVref a power of two >= every sV of the head, so P' <= 1 fits f16 and
// the accumulator holds O * l / sVref.  The row sum l adds P' * (sVref/sV)
// per tile (from the same f16 values that enter the MFMA).  Tiles whose
// sV/sVref is below 2^-14 (including all-zero V blocks) take a slow path
// that sums the unscaled weights instead.
#include "hyq_internal.h"

namespace hyq {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef _Float16 v8h __attribute__((ext_vector_type(8)));
typedef _Float16 v2h __attribute__((ext_vector_type(2)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));

#ifndef HYQ_ATTN_NB
#define HYQ_ATTN_NB 1
#endif
constexpr int kNB = HYQ_ATTN_NB;          // 32-query MFMA column blocks per wave
constexpr int kTile = 64;
constexpr int kWaves = 4;                 // waves per workgroup (one per SIMD)
constexpr int kThreads = kWaves * 64;
constexpr int kStageThreads = kThreads;
constexpr int kNBuf = 3;                  // quantized tiles c-1, c, c+1 resident
constexpr float kLazy = 8.0f;             // rescale only when the max grows by > 2^8
// instruction classes of __builtin_amdgcn_sched_group_barrier
constexpr int kSchedMfma = 0x008;
constexpr int kSchedDsRead = 0x100;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kMinusBig = -1.0e30f;

// LDS row pitches (bytes).  +16 keeps the 16-byte reads of 8 consecutive
// rows on distinct banks.
// int8 K tile: 64 rows of 128 B with no padding; the 16-byte chunk j of row r
// is stored at slot j ^ (r % 8), which keeps 16-byte reads of 8 consecutive
// rows on distinct banks and lets a wave fill 8 rows with one 1 KB direct
// global-to-LDS load.
constexpr int kKRowI8 = kHeadDim;
constexpr int kKPitchBf = kHeadDim * 2 + 16;    // bf16 K row
constexpr int kVPitch = kTile * 2 + 16;          // one channel of 64 f16/bf16 keys
constexpr int kVBytes = kHeadDim * kVPitch;

struct QBuf {                       // one quantized tile
  alignas(16) uint8_t k[kTile * kKRowI8];
  alignas(16) uint8_t v[kVBytes];
  int32_t pos[kTile];
};
struct FBuf {                       // one full-precision tile
  alignas(16) uint8_t k[kTile * kKPitchBf];
  alignas(16) uint8_t v[kVBytes];
  int32_t pos[kTile];
};
union Smem {
  QBuf q[kNBuf];
  FBuf f;
};

__device__ __forceinline__ float xhalf_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float xhalf_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Number of entries <= x in the ascending array a[0, n) (wave-cooperative
// 64-ary search; every lane returns the same value).
__device__ int count_le(const int32_t* __restrict__ a, int n, int x) {
  const int lane = threadIdx.x & 63;
  int lo = 0, hi = n;  // answer in [lo, hi]
  while (hi > lo) {
    const int step = (hi - lo + 63) / 64;
    const int i = lo + (lane + 1) * step - 1;
    const bool pred = i < hi && a[i] <= x;
    const int cnt = __popcll(__ballot(pred));
    lo = lo + cnt * step;
    const int nhi = lo + step - 1;
    hi = nhi < hi ? nhi : hi;
    if (step == 1) break;
  }
  return lo;
}

// int8 codes (4 per dword) -> f16 pairs, exact: bytes biased to unsigned,
// placed as the low mantissa byte of 1024 (f16 0x64xx), minus 1152.
__device__ __forceinline__ void i8x4_to_h(uint32_t w, uint32_t& h01, uint32_t& h23) {
  const uint32_t u = w ^ 0x80808080u;
  const uint32_t a = __builtin_amdgcn_perm(0x64646464u, u, 0x04010400u);
  const uint32_t b = __builtin_amdgcn_perm(0x64646464u, u, 0x04030402u);
  const v2h bias = {(_Float16)1152.0f, (_Float16)1152.0f};
  const v2h ha = __builtin_bit_cast(v2h, a) - bias;
  const v2h hb = __builtin_bit_cast(v2h, b) - bias;
  h01 = __builtin_bit_cast(uint32_t, ha);
  h23 = __builtin_bit_cast(uint32_t, hb);
}

// Packed int4 (8 nibbles, element 2i low / 2i+1 high in byte i) -> 8 int8 of
// value 16*code, in element order.
__device__ __forceinline__ void i4x8_to_i8(uint32_t w, uint32_t& o0, uint32_t& o1) {
  const uint32_t lo = (w << 4) & 0xF0F0F0F0u;   // elements 0,2,4,6 (x16)
  const uint32_t hi = w & 0xF0F0F0F0u;          // elements 1,3,5,7 (x16)
  o0 = __builtin_amdgcn_perm(hi, lo, 0x05010400u);
  o1 = __builtin_amdgcn_perm(hi, lo, 0x07030602u);
}

// Slot of key e (0..63) in the permuted V^T row.
__device__ __forceinline__ int vslot(int e) {
  const int r = e & 15, c4 = r >> 2;
  const int sc = (c4 == 1) ? 2 : (c4 == 2) ? 1 : c4;
  return (e & ~15) + sc * 4 + (r & 3);
}

// ---------------------------------------------------------------------------
// Quantized tiles: each thread prefetches its share of tile c+1 from global
// memory into registers while tile c is computed, then converts and writes it
// into the other LDS buffer (one barrier per tile).
// ---------------------------------------------------------------------------
__device__ __forceinline__ int kswz(int row, int chunk) {
  return row * kKRowI8 + ((chunk ^ (row & 7)) << 4);
}

typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) void glob_void_t;

// Group 0, 8-bit K: direct global -> LDS loads, two 1 KB instructions per
// wave (LDS slots P = row*8 + slot, lane i of an instruction fills slot
// base + i and reads the global chunk that belongs there).  Asynchronous:
// the issuing waves wait (vmcnt) before the barrier that publishes the tile.
__device__ __forceinline__ void k_direct_issue(uint8_t* kdst, const uint8_t* __restrict__ kc,
                                               int wave_in_group, int lane) {
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int base = (wave_in_group * 2 + i) * 64;
    const int P = base + lane;
    const int row = P >> 3, slot = P & 7;
    const int chunk = slot ^ (row & 7);
    __builtin_amdgcn_global_load_lds((glob_void_t*)(kc + row * kKRowI8 + chunk * 16),
                                     (lds_void_t*)(kdst + base * 16), 16, 0, 0);
  }
}

// Group 0, 4-bit K: one 16-byte packed chunk per thread (32 channels of one
// row), expanded to int8 (16*code) and stored as two swizzled chunks.
__device__ __forceinline__ uint4 k4_load(const uint8_t* __restrict__ kc, int tid) {
  return reinterpret_cast<const uint4*>(kc)[tid];
}
__device__ __forceinline__ void k4_store(uint8_t* kdst, uint4 w, int tid) {
  const int row = tid >> 2, j4 = tid & 3;
  uint32_t o[8];
  i4x8_to_i8(w.x, o[0], o[1]);
  i4x8_to_i8(w.y, o[2], o[3]);
  i4x8_to_i8(w.z, o[4], o[5]);
  i4x8_to_i8(w.w, o[6], o[7]);
  *reinterpret_cast<uint4*>(kdst + kswz(row, 2 * j4)) = make_uint4(o[0], o[1], o[2], o[3]);
  *reinterpret_cast<uint4*>(kdst + kswz(row, 2 * j4 + 1)) = make_uint4(o[4], o[5], o[6], o[7]);
}

// Group 1: V codes (channel-major in global) and kq_pos of a tile, loaded
// into registers during the MFMA step and converted/stored during the VALU
// step.  V -> f16 [128][kVPitch] in the permuted key order.
template <int BITS>
struct VTileRegs {
  uint4 v[BITS == 8 ? 2 : 1];
  int32_t pos;
};

template <int BITS>
__device__ __forceinline__ void v_load(VTileRegs<BITS>& r, const uint8_t* __restrict__ vc,
                                       const int32_t* __restrict__ kq, int tid) {
  constexpr int n = BITS == 8 ? 2 : 1;
#pragma unroll
  for (int i = 0; i < n; ++i) r.v[i] = reinterpret_cast<const uint4*>(vc)[tid + i * kStageThreads];
  r.pos = tid < kTile ? kq[tid] : 0;
}

template <int BITS>
__device__ __forceinline__ void v_store(QBuf& b, const VTileRegs<BITS>& r, int tid) {
  if (BITS == 8) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int q = tid + i * kStageThreads;
      const int d = q >> 2, kg = q & 3;   // channel d, keys kg*16 .. +16
      const uint4 w = r.v[i];
      uint32_t h[8];
      i8x4_to_h(w.x, h[0], h[1]);   // keys 0..3
      i8x4_to_h(w.y, h[2], h[3]);   // keys 4..7
      i8x4_to_h(w.z, h[4], h[5]);   // keys 8..11
      i8x4_to_h(w.w, h[6], h[7]);   // keys 12..15
      uint8_t* dst = b.v + d * kVPitch + kg * 32;
      *reinterpret_cast<uint4*>(dst) = make_uint4(h[0], h[1], h[4], h[5]);
      *reinterpret_cast<uint4*>(dst + 16) = make_uint4(h[2], h[3], h[6], h[7]);
    }
  } else {
    const int d = tid >> 1, kh = tid & 1;   // channel d, keys kh*32 .. +32 (16 B packed)
    const uint4 w = r.v[0];
    const uint32_t ww[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int g16 = 0; g16 < 2; ++g16) {
      uint32_t bb[4];
      i4x8_to_i8(ww[2 * g16], bb[0], bb[1]);
      i4x8_to_i8(ww[2 * g16 + 1], bb[2], bb[3]);
      uint32_t h[8];
      i8x4_to_h(bb[0], h[0], h[1]);
      i8x4_to_h(bb[1], h[2], h[3]);
      i8x4_to_h(bb[2], h[4], h[5]);
      i8x4_to_h(bb[3], h[6], h[7]);
      uint8_t* dst = b.v + d * kVPitch + (kh * 2 + g16) * 32;
      *reinterpret_cast<uint4*>(dst) = make_uint4(h[0], h[1], h[4], h[5]);
      *reinterpret_cast<uint4*>(dst + 16) = make_uint4(h[2], h[3], h[6], h[7]);
    }
  }
  if (tid < kTile) b.pos[tid] = r.pos;
}

// Stage full-precision tile: entries e0 .. e0+63 of the list
// [vertical positions (nvl of them), then base, base+1, ...]; entries at or
// beyond `count` are padding (position HYQ_KQ_POS_PAD, zero rows).
__device__ __forceinline__ void stage_fp(FBuf& b, const uint16_t* __restrict__ Kh,
                                         const uint16_t* __restrict__ Vh,
                                         const int32_t* __restrict__ vl, int nvl, int base,
                                         int e0, int count, int L) {
  const int tid = threadIdx.x;
  if (tid < kTile) {
    const int e = e0 + tid;
    b.pos[tid] = e >= count ? HYQ_KQ_POS_PAD : (e < nvl ? vl[e] : base + (e - nvl));
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < (kTile * 16) / kThreads; ++i) {
    const int q = tid + i * kThreads;
    const int e = q >> 4, col = q & 15;
    const int p = b.pos[e];
    uint4 kw = make_uint4(0, 0, 0, 0), vw = make_uint4(0, 0, 0, 0);
    if ((unsigned)p < (unsigned)L) {
      kw = reinterpret_cast<const uint4*>(Kh + (size_t)p * kHeadDim)[col];
      vw = reinterpret_cast<const uint4*>(Vh + (size_t)p * kHeadDim)[col];
    }
    *reinterpret_cast<uint4*>(b.k + e * kKPitchBf + col * 16) = kw;
    const int slot = vslot(e);
    const uint32_t vv[4] = {vw.x, vw.y, vw.z, vw.w};
#pragma unroll
    for (int i2 = 0; i2 < 4; ++i2) {
      const int d = col * 8 + 2 * i2;
      *reinterpret_cast<uint16_t*>(b.v + d * kVPitch + slot * 2) = (uint16_t)(vv[i2] & 0xffff);
      *reinterpret_cast<uint16_t*>(b.v + (d + 1) * kVPitch + slot * 2) = (uint16_t)(vv[i2] >> 16);
    }
  }
}

// Online-softmax state of one 32-query block of a wave (each lane owns one
// query and the keys of its half of every 32-key group).
struct NState {
  float m;        // reference max (log2 domain); the true max is <= m + kLazy
  float l;        // this lane's part of the row sum, relative to m
  float corr;     // rescale of acc still to apply: 2^(m_before - m)
  v16f acc[4];    // O^T accumulator, 4 groups of 32 channels
};

__device__ __forceinline__ int xhalf_max_i(int x) {
  const auto r = __builtin_amdgcn_permlane32_swap((unsigned)x, (unsigned)x, false, false);
  return max((int)r[0], (int)r[1]);
}

// Key index (0..63) of accumulator register r of half-tile kh for this lane.
__device__ __forceinline__ int key_of(int kh, int r, int half) {
  return kh * 32 + (r >> 2) * 8 + half * 4 + (r & 3);
}

// Raise the reference max of every lane of the wave when some lane's tile
// max exceeds it by more than kLazy (2^kLazy bounds the unnormalized
// weights).  Branch-free: the row sum is rescaled now, the accumulator before
// the next P V product that adds to it.
__device__ __forceinline__ void lazy_max(NState& ns, float mt) {
  const bool any = __ballot(mt > ns.m + kLazy) != 0;
  const float mn = any ? fmaxf(ns.m, mt) : ns.m;
  const float c = __builtin_amdgcn_exp2f(ns.m - mn);   // 1 when unchanged
  ns.l *= c;
  ns.corr = c;
  ns.m = mn;
}

__device__ __forceinline__ void apply_corr(NState& ns) {
  if (__ballot(ns.corr != 1.0f)) {
#pragma unroll
    for (int dg = 0; dg < 4; ++dg)
#pragma unroll
      for (int r = 0; r < 16; ++r) ns.acc[dg][r] *= ns.corr;
  }
  ns.corr = 1.0f;
}

// Softmax of one 32-query block on one quantized tile: int32 logits s[2]
// (two 32-key halves) -> f16 weights p[4] (the B operands of the four 16-key
// P V steps), updating m and l.
__device__ __forceinline__ void softmax_q(NState& ns, const v16i (&s)[2], v8h (&p)[4], float cqk,
                                          float f, bool diag, const int32_t* pos, int tq,
                                          int half) {
  if (!diag && f >= 6.103515625e-05f) {
    // fast path: every key visible; the f16 weights carry the V scale
    int mi = s[0][0];
#pragma unroll
    for (int kh = 0; kh < 2; ++kh)
#pragma unroll
      for (int r = (kh == 0 ? 1 : 0); r < 16; r += 2) {
        if (r + 1 < 16) mi = max(mi, max(s[kh][r], s[kh][r + 1]));
        else mi = max(mi, s[kh][r]);
      }
    mi = xhalf_max_i(mi);
    lazy_max(ns, (float)mi * cqk);
    const float bias = __builtin_amdgcn_logf(f) - ns.m;   // log2
    float ps = 0.0f;
    const v2h one2 = {(_Float16)1.0f, (_Float16)1.0f};
#pragma unroll
    for (int kh = 0; kh < 2; ++kh)
#pragma unroll
      for (int r = 0; r < 16; r += 2) {
        const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf((float)s[kh][r], cqk, bias));
        const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf((float)s[kh][r + 1], cqk, bias));
        v2h pk;
        pk[0] = (_Float16)p0;
        pk[1] = (_Float16)p1;
        ps = __builtin_amdgcn_fdot2(pk, one2, ps, false);
        p[kh * 2 + (r >> 3)][r & 7] = pk[0];
        p[kh * 2 + (r >> 3)][(r & 7) + 1] = pk[1];
      }
    ns.l = __builtin_fmaf(ps, __builtin_amdgcn_rcpf(f), ns.l);   // 1-ulp reciprocal
  } else {
    // general path: causal mask by original position, tiny V scales.  No
    // per-lane branches, so the cross-lane swap sees every lane's operand;
    // the visibility test is evaluated twice rather than kept in registers.
    int mi = INT_MIN;
#pragma unroll
    for (int kh = 0; kh < 2; ++kh)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const bool vis = (!diag) | (pos[key_of(kh, r, half)] <= tq);
        mi = max(mi, vis ? s[kh][r] : INT_MIN);
      }
    mi = xhalf_max_i(mi);
    lazy_max(ns, mi == INT_MIN ? -INFINITY : (float)mi * cqk);
    // The row sum adds the same f16 weights the MFMA uses (divided by f),
    // unless f is so small that they lose precision; then the float32 ones.
    const bool f_ok = f >= 6.103515625e-05f;
    float ps = 0.0f;
#pragma unroll
    for (int kh = 0; kh < 2; ++kh)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const bool vis = (!diag) | (pos[key_of(kh, r, half)] <= tq);
        const float ex = __builtin_amdgcn_exp2f((float)s[kh][r] * cqk - ns.m);
        const float e = vis ? ex : 0.0f;
        const _Float16 hp = (_Float16)(e * f);
        ps += f_ok ? (float)hp : e;
        p[kh * 2 + (r >> 3)][r & 7] = hp;
      }
    ns.l += f_ok ? ps * __builtin_amdgcn_rcpf(f) : ps;
  }
}

// Everything one wave needs for the quantized segment.
struct SegA {
  const uint8_t* kc0;
  const uint8_t* vc0;
  const int32_t* kq0;
  const float* ks0;
  const float* vs0;
  int n;              // quantized tiles to scan
  int t0;             // first query row of the wave
  float cq;           // alpha * log2(e) * s_Q
  float inv_vref;
  int lane, half, col, w;
};

// One tile of the quantized segment: stage tile c+1, S^T of tile c, P V of
// tile c-1 (weights pprev; zeros when c = 0), softmax of tile c -> pcur.
template <int BITS, int NB>
__device__ __forceinline__ void segA_tile(Smem& sm, const SegA& a, int c, const v4i (&qf)[NB][4],
                                          NState (&st)[NB], const v8h (&pprev)[NB][4],
                                          v8h (&pcur)[NB][4], VTileRegs<BITS>& vr, uint4& k4r) {
  constexpr int kRow = BITS == 8 ? kHeadDim : kHeadDim / 2;
  constexpr int vRow = BITS == 8 ? kTile : kTile / 2;
  constexpr float kSub = BITS == 8 ? 1.0f : 0.0625f;   // 4-bit codes are staged as 16*code
  const int tid = threadIdx.x;
  const bool more = c + 1 < a.n;
  // stage tile c+1 into the ring (its previous tile, c-2, is no longer read)
  if (more) {
    const uint8_t* kn = a.kc0 + (size_t)(c + 1) * kTile * kRow;
    if (BITS == 8) k_direct_issue(sm.q[(c + 1) % kNBuf].k, kn, a.w, a.lane);
    else k4r = k4_load(kn, tid);
    v_load<BITS>(vr, a.vc0 + (size_t)(c + 1) * kHeadDim * vRow, a.kq0 + (size_t)(c + 1) * kTile,
                 tid);
  }
  const float sk = a.ks0[c] * kSub;
  const float sv = a.vs0[c] * kSub;
  const QBuf& cur = sm.q[c % kNBuf];
  const QBuf& prv = sm.q[c >= 1 ? (c - 1) % kNBuf : 0];

  // pending accumulator rescales (from the softmax of tile c-1)
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) apply_corr(st[nb]);

  // S^T of tile c: each K fragment serves every query block
  v4i ka[2][4];
#pragma unroll
  for (int kh = 0; kh < 2; ++kh)
#pragma unroll
    for (int k4 = 0; k4 < 4; ++k4)
      ka[kh][k4] = *reinterpret_cast<const v4i*>(cur.k + kswz(kh * 32 + a.col, k4 * 2 + a.half));
  v16i s[NB][2];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int kh = 0; kh < 2; ++kh) {
      s[nb][kh] = v16i{0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
      for (int k4 = 0; k4 < 4; ++k4)
        s[nb][kh] = __builtin_amdgcn_mfma_i32_32x32x32_i8(ka[kh][k4], qf[nb][k4], s[nb][kh], 0, 0, 0);
    }
  // P V of tile c-1: each V fragment serves every query block
#pragma unroll
  for (int dg = 0; dg < 4; ++dg)
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const v8h va = *reinterpret_cast<const v8h*>(prv.v + (dg * 32 + a.col) * kVPitch + ks * 32 +
                                                   a.half * 16);
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
        st[nb].acc[dg] = __builtin_amdgcn_mfma_f32_32x32x16_f16(va, pprev[nb][ks], st[nb].acc[dg], 0, 0, 0);
    }
  // softmax of tile c (independent of the P V products above)
  const float cqk = a.cq * sk;
  const float f = sv * a.inv_vref;
  const int last = __builtin_amdgcn_readfirstlane(cur.pos[kTile - 1]);
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int tq = a.t0 + nb * 32 + a.col;
    softmax_q(st[nb], s[nb], pcur[nb], cqk, f, last > a.t0 + nb * 32, cur.pos, tq, a.half);
  }
  if (more) {
    // after the math, so that the wait for memory comes last
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("" ::: "memory");
    if (BITS == 4) k4_store(sm.q[(c + 1) % kNBuf].k, k4r, tid);
    v_store<BITS>(sm.q[(c + 1) % kNBuf], vr, tid);
    __builtin_amdgcn_s_waitcnt(0);   // direct K loads complete
  }
  __syncthreads();
}

template <int BITS, int OUT_BF16, int NB>
__global__ void __launch_bounds__(kThreads, NB == 1 ? 2 : 1)
attn_prefill_kernel(const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
                    const uint16_t* __restrict__ V, const int32_t* __restrict__ idx,
                    const int8_t* __restrict__ q_codes, const float* __restrict__ q_scale,
                    const uint8_t* __restrict__ k_codes, const float* __restrict__ k_scale,
                    const uint8_t* __restrict__ v_codes, const float* __restrict__ v_scale,
                    const int32_t* __restrict__ kq_pos, void* __restrict__ out, int Hq, int Hkv,
                    int nbj, int L, int P, int k, int nQ, int n_qblk, int n_kvblk,
                    float alpha_log2e) {
  __shared__ Smem sm;
  const int g = Hq / Hkv;
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int half = lane >> 5, col = lane & 31;

  // Work units of one KV head: (block rb of 32*NB rows, query head hh of the
  // group), ordered by rb; a workgroup takes 4 consecutive units, longest first.
  constexpr int kRows = 32 * NB;
  const int nrb = (L + kRows - 1) / kRows;
  const int units = g * nrb;
  const int wg_per_bj = (units + kWaves - 1) / kWaves;
  const int wgi = wg_per_bj - 1 - (int)blockIdx.x / nbj;
  const int bj = (int)blockIdx.x % nbj;
  const int u = wgi * kWaves + w;
  const bool active = u < units;
  const int uu = active ? u : units - 1;   // an idle wave mirrors the last unit, stores nothing
  const int rb = uu / g, hh = uu % g;
  const int u_last = min(wgi * kWaves + kWaves - 1, units - 1);
  const int t_last = min(L - 1, (u_last / g) * kRows + kRows - 1);   // workgroup
  const int b = bj / Hkv, j = bj % Hkv, h = j * g + hh;
  const size_t bh = (size_t)b * Hq + h;
  const int t0 = rb * kRows;

  const uint16_t* Kh = K + (size_t)bj * L * kHeadDim;
  const uint16_t* Vh = V + (size_t)bj * L * kHeadDim;
  const int32_t* vl = idx + (size_t)bj * k;

  NState st[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    st[nb].m = kMinusBig;
    st[nb].l = 0.0f;
    st[nb].corr = 1.0f;
#pragma unroll
    for (int dg = 0; dg < 4; ++dg)
#pragma unroll
      for (int r = 0; r < 16; ++r) st[nb].acc[dg][r] = 0.0f;
  }

  // Which keys are visible to rows up to t_last.
  int nvl, nq_tiles, fp_count, fp_base;
  float vref = 1.0f;
  if (BITS == 16) {
    nvl = 0;
    nq_tiles = 0;
    fp_base = 0;
    fp_count = t_last + 1;
  } else {
    nvl = count_le(vl, k, t_last);
    const int nq_vis = t_last < P ? (t_last + 1) - nvl : nQ;
    nq_tiles = min((nq_vis + kTile - 1) / kTile, n_kvblk);
    fp_base = P;
    fp_count = nvl + max(0, t_last + 1 - P);
    // sVref: smallest power of two >= every V scale of this head
    float mx = 0.0f;
    for (int i = lane; i < n_kvblk; i += 64) mx = fmaxf(mx, v_scale[(size_t)bj * n_kvblk + i]);
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 64));
    if (BITS == 4) mx *= 0.0625f;
    if (mx > 0.0f) {
      int e;
      frexpf(mx, &e);
      e = max(-100, min(100, e));
      vref = ldexpf(1.0f, e);
    }
  }
  const float inv_vref = 1.0f / vref;

  // ---------------- segment A: quantized keys ----------------
  if (nq_tiles > 0) {
    constexpr int kRow = BITS == 8 ? kHeadDim : kHeadDim / 2;
    constexpr int vRow = BITS == 8 ? kTile : kTile / 2;
    const size_t slots = (size_t)n_kvblk * kTile;
    SegA a;
    a.kc0 = k_codes + (size_t)bj * slots * kRow;
    a.vc0 = v_codes + (size_t)bj * n_kvblk * kHeadDim * vRow;
    a.kq0 = kq_pos + (size_t)bj * slots;
    a.ks0 = k_scale + (size_t)bj * n_kvblk;
    a.vs0 = v_scale + (size_t)bj * n_kvblk;
    a.n = nq_tiles;
    a.t0 = t0;
    a.cq = alpha_log2e * q_scale[bh * n_qblk + t0 / kBlock];
    a.inv_vref = inv_vref;
    a.lane = lane;
    a.half = half;
    a.col = col;
    a.w = w;

    v4i qf[NB][4];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const int tq = t0 + nb * 32 + col;
      const bool ok = active && tq < L;
      const int8_t* qrow = q_codes + (bh * L + (ok ? tq : 0)) * kHeadDim;
#pragma unroll
      for (int k4 = 0; k4 < 4; ++k4)
        qf[nb][k4] = ok ? *reinterpret_cast<const v4i*>(qrow + k4 * 32 + half * 16) : v4i{0, 0, 0, 0};
    }

    // prologue: tile 0
    VTileRegs<BITS> vr;
    uint4 k4r = make_uint4(0, 0, 0, 0);
    if (BITS == 8) {
      k_direct_issue(sm.q[0].k, a.kc0, w, lane);
    } else {
      k4r = k4_load(a.kc0, threadIdx.x);
      k4_store(sm.q[0].k, k4r, threadIdx.x);
    }
    v_load<BITS>(vr, a.vc0, a.kq0, threadIdx.x);
    v_store<BITS>(sm.q[0], vr, threadIdx.x);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();

    // the P V of tile c runs in iteration c+1, next to the softmax of c+1;
    // the weights alternate between two register sets
    v8h pa[NB][4], pb[NB][4];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int e = 0; e < 8; ++e) pa[nb][i][e] = pb[nb][i][e] = (_Float16)0.0f;
    int c = 0;
    for (; c + 1 < nq_tiles; c += 2) {
      segA_tile<BITS, NB>(sm, a, c, qf, st, pa, pb, vr, k4r);
      segA_tile<BITS, NB>(sm, a, c + 1, qf, st, pb, pa, vr, k4r);
    }
    if (c < nq_tiles) {
      segA_tile<BITS, NB>(sm, a, c, qf, st, pa, pb, vr, k4r);
      ++c;
    }
    // P V of the last tile
    const v8h (&plast)[NB][4] = (nq_tiles & 1) ? pb : pa;
    const QBuf& lb = sm.q[(nq_tiles - 1) % kNBuf];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) apply_corr(st[nb]);
#pragma unroll
    for (int dg = 0; dg < 4; ++dg)
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const v8h va = *reinterpret_cast<const v8h*>(lb.v + (dg * 32 + col) * kVPitch + ks * 32 +
                                                     half * 16);
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
          st[nb].acc[dg] = __builtin_amdgcn_mfma_f32_32x32x16_f16(va, plast[nb][ks], st[nb].acc[dg], 0, 0, 0);
      }
    __syncthreads();   // the FP segment reuses the LDS
  }

  // ---------------- segments B and C: full-precision keys ----------------
  if (fp_count > 0) {
    v8bf qb[NB][8];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const int tq = t0 + nb * 32 + col;
      const uint16_t* qrow = Q + (bh * L + ((active && tq < L) ? tq : 0)) * kHeadDim;
#pragma unroll
      for (int ks = 0; ks < 8; ++ks) qb[nb][ks] = *reinterpret_cast<const v8bf*>(qrow + ks * 16 + half * 8);
    }
    const int nft = (fp_count + kTile - 1) / kTile;
    FBuf& fb = sm.f;
    for (int ft = 0; ft < nft; ++ft) {
      __syncthreads();
      stage_fp(fb, Kh, Vh, vl, nvl, fp_base, ft * kTile, fp_count, L);
      __syncthreads();
      v8bf ka[2][8];
#pragma unroll
      for (int kh = 0; kh < 2; ++kh)
#pragma unroll
        for (int ks = 0; ks < 8; ++ks)
          ka[kh][ks] = *reinterpret_cast<const v8bf*>(fb.k + (kh * 32 + col) * kKPitchBf + ks * 32 +
                                                      half * 16);
      v8bf phi[NB][4], plo[NB][4];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const int tq = t0 + nb * 32 + col;
        v16f sf[2];
#pragma unroll
        for (int kh = 0; kh < 2; ++kh) {
#pragma unroll
          for (int r = 0; r < 16; ++r) sf[kh][r] = 0.0f;
#pragma unroll
          for (int ks = 0; ks < 8; ++ks)
            sf[kh] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[kh][ks], qb[nb][ks], sf[kh], 0, 0, 0);
        }
        float mt = -INFINITY;
#pragma unroll
        for (int kh = 0; kh < 2; ++kh)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const bool vis = fb.pos[key_of(kh, r, half)] <= tq;
            mt = fmaxf(mt, vis ? sf[kh][r] * alpha_log2e : -INFINITY);
          }
        lazy_max(st[nb], xhalf_max(mt));
        apply_corr(st[nb]);
        float ps = 0.0f;
#pragma unroll
        for (int kh = 0; kh < 2; ++kh)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const bool vis = fb.pos[key_of(kh, r, half)] <= tq;
            const float ex = __builtin_amdgcn_exp2f(sf[kh][r] * alpha_log2e - st[nb].m);
            const float pv = vis ? ex : 0.0f;
            ps += pv;
            const float pp = pv * inv_vref;
            const __bf16 hi = (__bf16)pp;
            const __bf16 lo = (__bf16)(pp - (float)hi);
            phi[nb][kh * 2 + (r >> 3)][r & 7] = hi;
            plo[nb][kh * 2 + (r >> 3)][r & 7] = lo;
          }
        st[nb].l += ps;
      }
#pragma unroll
      for (int dg = 0; dg < 4; ++dg)
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
          const v8bf va = *reinterpret_cast<const v8bf*>(fb.v + (dg * 32 + col) * kVPitch + ks * 32 +
                                                         half * 16);
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) {
            st[nb].acc[dg] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, phi[nb][ks], st[nb].acc[dg], 0, 0, 0);
            st[nb].acc[dg] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, plo[nb][ks], st[nb].acc[dg], 0, 0, 0);
          }
        }
    }
  }

  // ---------------- finalize: O = acc * sVref / l ----------------
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const float ltot = xhalf_sum(st[nb].l);
    const float sc = vref / ltot;
    const int tq = t0 + nb * 32 + col;
    if (!(active && tq < L)) continue;
    const size_t obase = (bh * L + tq) * kHeadDim;
#pragma unroll
    for (int dg = 0; dg < 4; ++dg)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const int d = dg * 32 + r4 * 8 + half * 4;
        const float o0 = st[nb].acc[dg][r4 * 4 + 0] * sc, o1 = st[nb].acc[dg][r4 * 4 + 1] * sc;
        const float o2 = st[nb].acc[dg][r4 * 4 + 2] * sc, o3 = st[nb].acc[dg][r4 * 4 + 3] * sc;
        if (OUT_BF16) {
          uint16_t* o = reinterpret_cast<uint16_t*>(out) + obase + d;
          const __bf16 b0 = (__bf16)o0, b1 = (__bf16)o1, b2 = (__bf16)o2, b3 = (__bf16)o3;
          const uint32_t w0 = (uint32_t)__builtin_bit_cast(uint16_t, b0) |
                              ((uint32_t)__builtin_bit_cast(uint16_t, b1) << 16);
          const uint32_t w1 = (uint32_t)__builtin_bit_cast(uint16_t, b2) |
                              ((uint32_t)__builtin_bit_cast(uint16_t, b3) << 16);
          *reinterpret_cast<uint2*>(o) = make_uint2(w0, w1);
        } else {
          float* o = reinterpret_cast<float*>(out) + obase + d;
          *reinterpret_cast<float4*>(o) = make_float4(o0, o1, o2, o3);
        }
      }
  }
}

template <int BITS, int OB>
hipError_t launch_t(const hyq_shape& s, const hyq_sizes& z, const uint16_t* Q,
                    const uint16_t* K, const uint16_t* V, const int32_t* idx,
                    const int8_t* q_codes, const float* q_scale, const uint8_t* k_codes,
                    const float* k_scale, const uint8_t* v_codes, const float* v_scale,
                    const int32_t* kq_pos, float softmax_scale, void* out, hipStream_t st) {
  const int g = s.Hq / s.Hkv;
  const int nrb = (s.L + 32 * kNB - 1) / (32 * kNB);
  const int wg_per_bj = (g * nrb + kWaves - 1) / kWaves;
  const int nbj = s.B * s.Hkv;
  const dim3 grid(wg_per_bj * nbj);
  attn_prefill_kernel<BITS, OB, kNB><<<grid, kThreads, 0, st>>>(
      Q, K, V, idx, q_codes, q_scale, k_codes, k_scale, v_codes, v_scale, kq_pos, out, s.Hq,
      s.Hkv, nbj, s.L, z.P, z.k, z.nQ, z.n_qblk, z.n_kvblk, softmax_scale * kLog2e);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attn_prefill(const hyq_shape& s, const hyq_sizes& z, const uint16_t* Q,
                               const uint16_t* K, const uint16_t* V, const int32_t* idx,
                               const int8_t* q_codes, const float* q_scale,
                               const uint8_t* k_codes, const float* k_scale,
                               const uint8_t* v_codes, const float* v_scale,
                               const int32_t* kq_pos, float softmax_scale, void* out,
                               int out_dtype, hipStream_t st) {
#define HYQ_LAUNCH(BITS, OB)                                                                  \
  return launch_t<BITS, OB>(s, z, Q, K, V, idx, q_codes, q_scale, k_codes, k_scale, v_codes, \
                            v_scale, kq_pos, softmax_scale, out, st)
  if (s.bits_kv == 16) {
    if (out_dtype) HYQ_LAUNCH(16, 1);
    HYQ_LAUNCH(16, 0);
  } else if (s.bits_kv == 8) {
    if (out_dtype) HYQ_LAUNCH(8, 1);
    HYQ_LAUNCH(8, 0);
  } else {
    if (out_dtype) HYQ_LAUNCH(4, 1);
    HYQ_LAUNCH(4, 0);
  }
#undef HYQ_LAUNCH
}

}  // namespace hyq
