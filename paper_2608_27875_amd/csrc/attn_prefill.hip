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

constexpr int kRowsPerWave = 32;
constexpr int kTile = 64;
constexpr int kWaves = 4;                 // waves per workgroup
constexpr int kThreads = kWaves * 64;
constexpr float kLazy = 8.0f;             // rescale only when the max grows by > 2^8
// instruction classes of __builtin_amdgcn_sched_group_barrier
constexpr int kSchedMfma = 0x008;
constexpr int kSchedDsRead = 0x100;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kMinusBig = -1.0e30f;

// LDS row pitches (bytes).  +16 keeps the 16-byte reads of 8 consecutive
// rows on distinct banks.
constexpr int kKPitchI8 = kHeadDim + 16;        // int8 K codes row
constexpr int kKPitchBf = kHeadDim * 2 + 16;    // bf16 K row
constexpr int kVPitch = kTile * 2 + 16;          // one channel of 64 f16/bf16 keys
constexpr int kKBytes = kTile * kKPitchBf;
constexpr int kVBytes = kHeadDim * kVPitch;

struct Buf {
  alignas(16) uint8_t k[kKBytes];
  alignas(16) uint8_t v[kVBytes];
  int32_t pos[kTile];
};
struct Smem {
  Buf buf[2];   // double buffer: tile c is computed while tile c+1 is written
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
template <int BITS>
struct QTileRegs {
  uint4 k[BITS == 8 ? 2 : 1];
  uint4 v[BITS == 8 ? 2 : 1];
  int32_t pos;
};

// An empty asm that "modifies" the value: a global load stored unchanged to
// LDS is otherwise turned into a memcpy, which is lowered (with its wait for
// the load) where the load was issued instead of where the store is.
__device__ __forceinline__ void opaque(uint4& w) {
  asm volatile("" : "+v"(w.x), "+v"(w.y), "+v"(w.z), "+v"(w.w));
}

template <int BITS>
__device__ __forceinline__ void load_qtile(QTileRegs<BITS>& r, const uint8_t* __restrict__ kc,
                                           const uint8_t* __restrict__ vc,
                                           const int32_t* __restrict__ kq) {
  const int tid = threadIdx.x;
  constexpr int n = BITS == 8 ? 2 : 1;
#pragma unroll
  for (int i = 0; i < n; ++i) {
    r.k[i] = reinterpret_cast<const uint4*>(kc)[tid + i * kThreads];
    r.v[i] = reinterpret_cast<const uint4*>(vc)[tid + i * kThreads];
  }
  r.pos = tid < kTile ? kq[tid] : 0;
}

// K codes -> int8 [64][kKPitchI8] (4-bit: 16*code); V codes (channel-major in
// global) -> f16 [128][kVPitch] in the permuted key order; kq_pos -> pos.
template <int BITS>
__device__ __forceinline__ void store_qtile(Buf& b, const QTileRegs<BITS>& r) {
  const int tid = threadIdx.x;
  if (BITS == 8) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int q = tid + i * kThreads;   // K: 512 chunks of 16 B, 8 per row
      uint4 kw = r.k[i];
      opaque(kw);
      *reinterpret_cast<uint4*>(b.k + (q >> 3) * kKPitchI8 + (q & 7) * 16) = kw;
      const int d = q >> 2, kg = q & 3;   // V: channel d, keys kg*16 .. +16
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
    {
      const int q = tid;   // K: 256 chunks of 16 B packed = 32 channels
      const uint4 w = r.k[0];
      uint32_t o[8];
      i4x8_to_i8(w.x, o[0], o[1]);
      i4x8_to_i8(w.y, o[2], o[3]);
      i4x8_to_i8(w.z, o[4], o[5]);
      i4x8_to_i8(w.w, o[6], o[7]);
      uint8_t* dst = b.k + (q >> 2) * kKPitchI8 + (q & 3) * 32;
      *reinterpret_cast<uint4*>(dst) = make_uint4(o[0], o[1], o[2], o[3]);
      *reinterpret_cast<uint4*>(dst + 16) = make_uint4(o[4], o[5], o[6], o[7]);
    }
    {
      const int q = tid;   // V: channel q/2, keys (q&1)*32 .. +32 (16 B packed)
      const int d = q >> 1, kh = q & 1;
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
  }
  if (tid < kTile) b.pos[tid] = r.pos;
}

// Stage full-precision tile: entries e0 .. e0+63 of the list
// [vertical positions (nvl of them), then base, base+1, ...]; entries at or
// beyond `count` are padding (position HYQ_KQ_POS_PAD, zero rows).
__device__ __forceinline__ void stage_fp(Buf& b, const uint16_t* __restrict__ Kh,
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

struct SoftmaxState {
  float m;        // reference max of the log2-domain logits (lazy: true max <= m + kLazy)
  float l;        // this lane's part of the row sum (keys of its half)
  v16f acc[4];    // O^T accumulator, 4 groups of 32 channels
};

// Raise the reference max of the lanes whose tile max exceeds it by more than
// kLazy (2^kLazy bounds the unnormalized weights), rescaling their state.
__device__ __forceinline__ void raise_max(SoftmaxState& st, float mt) {
  if (__ballot(mt > st.m + kLazy)) {
    const float mn = fmaxf(st.m, mt);
    const float corr = __builtin_amdgcn_exp2f(st.m - mn);
    st.l *= corr;
#pragma unroll
    for (int dg = 0; dg < 4; ++dg)
#pragma unroll
      for (int r = 0; r < 16; ++r) st.acc[dg][r] *= corr;
    st.m = mn;
  }
}

__device__ __forceinline__ int xhalf_max_i(int x) {
  const auto r = __builtin_amdgcn_permlane32_swap((unsigned)x, (unsigned)x, false, false);
  return max((int)r[0], (int)r[1]);
}

// Key index (0..63) of accumulator register r of half-tile kh for this lane.
__device__ __forceinline__ int key_of(int kh, int r, int half) {
  return kh * 32 + (r >> 2) * 8 + half * 4 + (r & 3);
}

template <int BITS, int OUT_BF16>
__global__ void __launch_bounds__(kThreads, 2)
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
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int half = lane >> 5, col = lane & 31;

  // Work units of one KV head: (32-row block rb, query head hh of the group),
  // ordered by rb; a workgroup takes 4 consecutive units, longest first.
  const int nrb = (L + kRowsPerWave - 1) / kRowsPerWave;
  const int units = g * nrb;
  const int wg_per_bj = (units + kWaves - 1) / kWaves;
  const int wgi = wg_per_bj - 1 - (int)blockIdx.x / nbj;
  const int bj = (int)blockIdx.x % nbj;
  const int u = wgi * kWaves + w;
  const bool active = u < units;
  const int uu = active ? u : units - 1;   // an idle wave mirrors the last unit, stores nothing
  const int rb = uu / g, hh = uu % g;
  const int u_last = min(wgi * kWaves + kWaves - 1, units - 1);
  const int t_last = min(L - 1, (u_last / g) * kRowsPerWave + kRowsPerWave - 1);   // workgroup
  const int b = bj / Hkv, j = bj % Hkv, h = j * g + hh;
  const size_t bh = (size_t)b * Hq + h;
  const int t0 = rb * kRowsPerWave;
  const int tq = t0 + col;
  const bool valid_q = active && tq < L;

  const uint16_t* Kh = K + (size_t)bj * L * kHeadDim;
  const uint16_t* Vh = V + (size_t)bj * L * kHeadDim;
  const int32_t* vl = idx + (size_t)bj * k;

  SoftmaxState st;
  st.m = kMinusBig;
  st.l = 0.0f;
#pragma unroll
  for (int dg = 0; dg < 4; ++dg)
#pragma unroll
    for (int r = 0; r < 16; ++r) st.acc[dg][r] = 0.0f;

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
    v4i qf[4];
    const int8_t* qrow = q_codes + (bh * L + (valid_q ? tq : 0)) * kHeadDim;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      qf[s] = valid_q ? *reinterpret_cast<const v4i*>(qrow + s * 32 + half * 16) : v4i{0, 0, 0, 0};
    }
    const float cq = alpha_log2e * q_scale[bh * n_qblk + t0 / kBlock];
    const size_t slots = (size_t)n_kvblk * kTile;
    constexpr int kRow = BITS == 8 ? kHeadDim : kHeadDim / 2;
    constexpr int vRow = BITS == 8 ? kTile : kTile / 2;
    constexpr float kSub = BITS == 8 ? 1.0f : 0.0625f;   // 4-bit codes are staged as 16*code
    const uint8_t* kc0 = k_codes + (size_t)bj * slots * kRow;
    const uint8_t* vc0 = v_codes + (size_t)bj * n_kvblk * kHeadDim * vRow;
    const int32_t* kq0 = kq_pos + (size_t)bj * slots;
    const float* ks0 = k_scale + (size_t)bj * n_kvblk;
    const float* vs0 = v_scale + (size_t)bj * n_kvblk;

    QTileRegs<BITS> pf;
    load_qtile<BITS>(pf, kc0, vc0, kq0);
    store_qtile<BITS>(sm.buf[0], pf);
    __syncthreads();
    for (int c = 0; c < nq_tiles; ++c) {
      const Buf& cur = sm.buf[c & 1];
      const bool more = c + 1 < nq_tiles;
      if (more)
        load_qtile<BITS>(pf, kc0 + (size_t)(c + 1) * kTile * kRow,
                         vc0 + (size_t)(c + 1) * kHeadDim * vRow, kq0 + (size_t)(c + 1) * kTile);
      const float sk = ks0[c] * kSub;
      const float sv = vs0[c] * kSub;

      // all 8 K fragments are read before the first MFMA (hides LDS latency)
      v4i ka[2][4];
#pragma unroll
      for (int kh = 0; kh < 2; ++kh)
#pragma unroll
        for (int st4 = 0; st4 < 4; ++st4)
          ka[kh][st4] = *reinterpret_cast<const v4i*>(cur.k + (kh * 32 + col) * kKPitchI8 +
                                                      st4 * 32 + half * 16);
      v16i s[2];
#pragma unroll
      for (int kh = 0; kh < 2; ++kh) {
        s[kh] = v16i{0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
        for (int st4 = 0; st4 < 4; ++st4)
          s[kh] = __builtin_amdgcn_mfma_i32_32x32x32_i8(ka[kh][st4], qf[st4], s[kh], 0, 0, 0);
      }
      // scheduling: the 8 LDS reads first, then the 8 MFMAs
      __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 8, 0);
      __builtin_amdgcn_sched_group_barrier(kSchedMfma, 8, 0);
      const float cqk = cq * sk;
      const float f = sv * inv_vref;
      // wave-uniform: some key of this tile lies after the wave's first row
      const bool diag = __builtin_amdgcn_readfirstlane(cur.pos[kTile - 1]) > t0;
      v8h pf16[4];
      if (!diag && f >= 6.103515625e-05f) {
        // fast path: every key visible, f16 weights carry the V scale
        int mi = s[0][0];
#pragma unroll
        for (int kh = 0; kh < 2; ++kh)
#pragma unroll
          for (int r = (kh == 0 ? 1 : 0); r < 16; r += 2) {
            if (r + 1 < 16) mi = max(mi, max(s[kh][r], s[kh][r + 1]));
            else mi = max(mi, s[kh][r]);
          }
        mi = xhalf_max_i(mi);
        raise_max(st, (float)mi * cqk);
        const float bias = __builtin_amdgcn_logf(f) - st.m;   // log2
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
            pf16[kh * 2 + (r >> 3)][r & 7] = pk[0];
            pf16[kh * 2 + (r >> 3)][(r & 7) + 1] = pk[1];
          }
        st.l = __builtin_fmaf(ps, __builtin_amdgcn_rcpf(f), st.l);   // 1-ulp reciprocal
      } else {
        // general path: causal mask by original position, tiny V scales.
        // Written without per-lane branches so that the cross-lane swap in
        // xhalf_max_i always runs with every lane's operand up to date.
        bool vis[2][16];
        int mi = INT_MIN;
#pragma unroll
        for (int kh = 0; kh < 2; ++kh)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            vis[kh][r] = (!diag) | (cur.pos[key_of(kh, r, half)] <= tq);
            mi = max(mi, vis[kh][r] ? s[kh][r] : INT_MIN);
          }
        mi = xhalf_max_i(mi);
        raise_max(st, mi == INT_MIN ? -INFINITY : (float)mi * cqk);
        // The row sum adds the same f16 weights the MFMA uses (divided by f),
        // unless f is so small that they lose precision; then the float32 ones.
        const bool f_ok = f >= 6.103515625e-05f;
        float ps = 0.0f;
#pragma unroll
        for (int kh = 0; kh < 2; ++kh)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const float ex = __builtin_amdgcn_exp2f((float)s[kh][r] * cqk - st.m);
            const float e = vis[kh][r] ? ex : 0.0f;
            const _Float16 hp = (_Float16)(e * f);
            ps += f_ok ? (float)hp : e;
            pf16[kh * 2 + (r >> 3)][r & 7] = hp;
          }
        st.l += f_ok ? ps * __builtin_amdgcn_rcpf(f) : ps;
      }
      // V fragments are read 8 at a time (two channel groups) ahead of their MFMAs
#pragma unroll
      for (int dp = 0; dp < 2; ++dp) {
        v8h va[2][4];
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int ks = 0; ks < 4; ++ks)
            va[i][ks] = *reinterpret_cast<const v8h*>(cur.v + ((dp * 2 + i) * 32 + col) * kVPitch +
                                                      ks * 32 + half * 16);
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int ks = 0; ks < 4; ++ks)
            st.acc[dp * 2 + i] =
                __builtin_amdgcn_mfma_f32_32x32x16_f16(va[i][ks], pf16[ks], st.acc[dp * 2 + i], 0, 0, 0);
      }
      // scheduling: keep four V reads ahead of the MFMA stream
      __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 4, 1);
#pragma unroll
      for (int i = 0; i < 12; ++i) {
        __builtin_amdgcn_sched_group_barrier(kSchedMfma, 1, 1);
        __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 1, 1);
      }
      __builtin_amdgcn_sched_group_barrier(kSchedMfma, 4, 1);
      // Keep the LDS stores of tile c+1 after this tile's math: hoisted next
      // to their loads they would make every iteration wait for memory.
      __builtin_amdgcn_sched_barrier(0);
      asm volatile("" ::: "memory");
      if (more) store_qtile<BITS>(sm.buf[(c + 1) & 1], pf);
      __syncthreads();
    }
  }

  // ---------------- segments B and C: full-precision keys ----------------
  if (fp_count > 0) {
    v8bf qb[8];
    const uint16_t* qrow = Q + (bh * L + (valid_q ? tq : 0)) * kHeadDim;
#pragma unroll
    for (int s = 0; s < 8; ++s) qb[s] = *reinterpret_cast<const v8bf*>(qrow + s * 16 + half * 8);
    const int nft = (fp_count + kTile - 1) / kTile;
    Buf& fb = sm.buf[0];
    for (int ft = 0; ft < nft; ++ft) {
      __syncthreads();
      stage_fp(fb, Kh, Vh, vl, nvl, fp_base, ft * kTile, fp_count, L);
      __syncthreads();
      v16f s[2];
#pragma unroll
      for (int kh = 0; kh < 2; ++kh) {
#pragma unroll
        for (int r = 0; r < 16; ++r) s[kh][r] = 0.0f;
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) {
          const v8bf a = *reinterpret_cast<const v8bf*>(fb.k + (kh * 32 + col) * kKPitchBf +
                                                       ks * 32 + half * 16);
          s[kh] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qb[ks], s[kh], 0, 0, 0);
        }
      }
      bool vis[2][16];
      float mt = -INFINITY;
#pragma unroll
      for (int kh = 0; kh < 2; ++kh)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          vis[kh][r] = fb.pos[key_of(kh, r, half)] <= tq;
          mt = fmaxf(mt, vis[kh][r] ? s[kh][r] * alpha_log2e : -INFINITY);
        }
      raise_max(st, xhalf_max(mt));
      v8bf phi[4], plo[4];
      float ps = 0.0f;
#pragma unroll
      for (int kh = 0; kh < 2; ++kh)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float ex = __builtin_amdgcn_exp2f(s[kh][r] * alpha_log2e - st.m);
          const float p = vis[kh][r] ? ex : 0.0f;
          ps += p;
          const float pp = p * inv_vref;
          const __bf16 hi = (__bf16)pp;
          const __bf16 lo = (__bf16)(pp - (float)hi);
          phi[kh * 2 + (r >> 3)][r & 7] = hi;
          plo[kh * 2 + (r >> 3)][r & 7] = lo;
        }
      st.l += ps;
#pragma unroll
      for (int dg = 0; dg < 4; ++dg)
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
          const v8bf a = *reinterpret_cast<const v8bf*>(fb.v + (dg * 32 + col) * kVPitch +
                                                       ks * 32 + half * 16);
          st.acc[dg] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, phi[ks], st.acc[dg], 0, 0, 0);
          st.acc[dg] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, plo[ks], st.acc[dg], 0, 0, 0);
        }
    }
  }

  // ---------------- finalize: O = acc * sVref / l ----------------
  const float ltot = xhalf_sum(st.l);
  const float sc = vref / ltot;
  if (!valid_q) return;
  const size_t obase = (bh * L + tq) * kHeadDim;
#pragma unroll
  for (int dg = 0; dg < 4; ++dg)
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4) {
      const int d = dg * 32 + r4 * 8 + half * 4;
      const float o0 = st.acc[dg][r4 * 4 + 0] * sc, o1 = st.acc[dg][r4 * 4 + 1] * sc;
      const float o2 = st.acc[dg][r4 * 4 + 2] * sc, o3 = st.acc[dg][r4 * 4 + 3] * sc;
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

template <int BITS, int OB>
hipError_t launch_t(const hyq_shape& s, const hyq_sizes& z, const uint16_t* Q,
                    const uint16_t* K, const uint16_t* V, const int32_t* idx,
                    const int8_t* q_codes, const float* q_scale, const uint8_t* k_codes,
                    const float* k_scale, const uint8_t* v_codes, const float* v_scale,
                    const int32_t* kq_pos, float softmax_scale, void* out, hipStream_t st) {
  const int g = s.Hq / s.Hkv;
  const int nrb = (s.L + kRowsPerWave - 1) / kRowsPerWave;
  const int wg_per_bj = (g * nrb + kWaves - 1) / kWaves;
  const int nbj = s.B * s.Hkv;
  const dim3 grid(wg_per_bj * nbj);
  attn_prefill_kernel<BITS, OB><<<grid, kThreads, 0, st>>>(
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
