// Hybrid-precision causal prefill attention: Algorithm 2, Stage 3 (App. A.2)
// and eq. (prefill_hybrid) of Section 4.2 of HyQuant.
//
// One workgroup = one KV head (b, j) x 8 work units, a unit being (32 query
// rows, one query head of the group); with g = 4 that is two 32-row tiles of
// the 4 heads.  The 8 waves (two per SIMD) share every K/V tile staged in
// LDS.  Each wave keeps one online-softmax state per query row and scans
//   segment A: the quantized keys (compacted K_Q order) in tiles of 64 =
//              one quantization block: S^T = K_codes * Qcodes^T with the int8
//              MFMA (exact int32) or, for FP8 codes, the E4M3 MFMA (float32),
//              or, for FP4 codes, the scaled MFMA with E2M1 keys against
//              E4M3 queries; logits scaled by alpha*log2(e)*sQ*sK; P V with
//              the f16 MFMA on the V codes (int8, E4M3 and E2M1 values are
//              exact in f16);
//   segments B and C: the full-precision keys (vertical lines, then the
//              window), 64 at a time gathered into two alternating LDS
//              buffers a tile ahead through registers: S^T with the bf16
//              MFMA; P V with the f16 MFMA on V / sVref converted to f16
//              (exact for bf16 values of that range); a tile whose V / sVref
//              leaves the f16 range raises sVref (the accumulator rescaled
//              exactly) and is staged again.
// Causality is by original key position in every segment.  With the
// per-query window (HYQ_WIN_BAND) row t sees keys t+1-W .. t in full
// precision and a quantized key only once it is older than that: segment A
// compares positions with t - W, and the full-precision list also carries the
// quantizable keys of the workgroup's band, each seen by W rows.
//
// Register layout (32x32 MFMA, wave64): lane l, accumulator register r holds
// row (r/4)*8 + (l/32)*4 + r%4 and column l%32.  With keys as rows (S^T),
// each lane owns one query (column) and 16 keys per 32-key half; those 16
// values are reused directly as the B operand of the P V product, and the
// V^T tile in LDS stores each 16-key group in the matching order
// [0-3, 8-11, 4-7, 12-15].
//
// Quantized tiles run through LDS rings fed from registers (K four
// buffers, V two): while tile c is computed, K(c+2) and V(c) (loaded into
// registers during tile c-1) are converted and written to LDS and K(c+3),
// V(c+1) are loaded, so global latency is covered by a whole tile and each
// barrier waits only for LDS writes.  The P V product of tile c-1 is issued
// interleaved with the softmax of tile c (one MFMA per weight pair) so that
// the matrix cores and the vector ALUs overlap within each wave.
//
// V scales: with sVref a power of two >= every sV of the head, the ratio
// sV/sVref = fm * 2^e is split into its mantissa fm in [1/2, 1) and its
// power of two.  2^e is applied exactly to the V codes when they are
// staged as f16 (a block with a small scale only ever gives small V values,
// whose rounding stays small against the output); fm is folded into the
// exponent, P' = 2^(y - m + log2 fm), so the f16 weights never lose range.
// The accumulator holds O * l / sVref; the row sum l adds P' / fm per tile
// (from the same f16 values that enter the MFMA).  An all-zero V block
// (sV = 0) folds nothing.
#include "codes_dev.h"
#include "hyq_internal.h"

#include <type_traits>

namespace hyq {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v8i __attribute__((ext_vector_type(8)));
typedef unsigned v4u __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef _Float16 v8h __attribute__((ext_vector_type(8)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef float v2f __attribute__((ext_vector_type(2)));

constexpr int kTile = 64;
#ifndef HYQ_ATTN_WAVES
#define HYQ_ATTN_WAVES 8
#endif
constexpr int kWaves = HYQ_ATTN_WAVES;    // waves per workgroup (kWaves / 4 per SIMD)
constexpr int kThreads = kWaves * 64;
constexpr int kWgPerCu = 8 / kWaves;      // workgroups per CU (two waves per SIMD)
// 16-byte chunks of one staged tile: 8-bit K and V tiles are 512 chunks, 4-bit 256
constexpr int kChunks8 = kTile * kHeadDim / 16;
constexpr int kChunks4 = kChunks8 / 2;
static_assert(kChunks8 % kThreads == 0, "8-bit tile chunks must split evenly");
constexpr float kLazy = 8.0f;             // general path: rescale only when the max grows by > 2^8
constexpr float kFastMax = 32768.0f;      // fast path: largest accepted weight sum of a lane
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kMinusBig = -1.0e30f;

// Key/value codes of the two FP4 formats are the same E2M1 nibbles; they
// differ only in the query codes (E4M3, or E2M3 for HYQ_FMT_FP4Q6).
constexpr bool kv_fp4(int fmt) { return fmt == HYQ_FMT_FP4 || fmt == HYQ_FMT_FP4Q6; }

// LDS row pitches (bytes).  +16 keeps the 16-byte reads of 8 consecutive
// rows on distinct banks.
// int8 K tile: 64 rows of 128 B with no padding; the 16-byte chunk j of row r
// is stored at slot j ^ ((r / 2) % 8): a 256-byte bank row holds two K rows,
// so the 16 lanes of one 16-byte read phase (16 consecutive rows, one chunk)
// land on distinct banks.
constexpr int kKRowI8 = kHeadDim;
constexpr int kKPitchBf = kHeadDim * 2 + 16;    // bf16 K row
constexpr int kVPitch = kTile * 2 + 16;          // one channel of 64 f16/bf16 keys
constexpr int kVBytes = kHeadDim * kVPitch;

// Tile metadata: kq_pos of the 64 slots, the bits of sK and sV (read from
// LDS rather than with scalar loads, whose counter would also wait for every
// pending LDS read), and one slot that absorbs the stores of the other
// staging threads so that staging needs no branch.
constexpr int kMetaSK = kTile, kMetaSV = kTile + 1, kMetaSink = kTile + 2;
struct KBuf {                       // K codes and metadata of one quantized tile
  alignas(16) uint8_t k[kTile * kKRowI8];
  int32_t pos[kTile + 4];
};
struct VBuf {                       // V of one quantized tile as f16 V^T
  alignas(16) uint8_t v[kVBytes];
};
// Quantized segment: tile c multiplies K(c) (fragments read from kb[c%4] at
// the end of tile c-1) and V(c-1) from vb[(c-1)%2]; it writes K(c+2) to
// kb[(c+2)%4] and V(c) to vb[c%2], and reads the fragments of K(c+1) from
// kb[(c+1)%4] (published one barrier earlier) before its closing barrier.
constexpr int kKRing = 4;
struct QRing {
  KBuf kb[kKRing];
  VBuf vb[2];
};
struct FBuf {                       // one full-precision tile
  alignas(16) uint8_t k[kTile * kKPitchBf];   // bf16 K rows
  alignas(16) uint8_t v[kVBytes];             // V^T as f16 V / sVref
  alignas(16) int32_t pos[kTile];             // rows t >= pos see the key ...
  alignas(16) int32_t hi[kTile];              // ... up to row hi
  int32_t ovf;     // (f << 8) | E: tile f staged here had a V / sVref outside the f16
                   // range, E the largest biased float exponent of its V values
};
// Full-precision tiles alternate between two buffers: tile f+1 is written
// while tile f is computed.
union Smem {
  QRing q;
  FBuf f[2];
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

// Slot of key e (0..63) in the permuted V^T row.
__device__ __forceinline__ int vslot(int e) {
  const int r = e & 15, c4 = r >> 2;
  const int sc = (c4 == 1) ? 2 : (c4 == 2) ? 1 : c4;
  return (e & ~15) + sc * 4 + (r & 3);
}

// ---------------------------------------------------------------------------
// Quantized tiles, staged through registers: K codes (compacted order), V
// codes (channel-major), kq_pos and the two block scales of one tile.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int kswz(int row, int chunk) {
  return row * kKRowI8 + ((chunk ^ ((row >> 1) & 7)) << 4);
}
// E2M1 K tile: 64 rows of 64 B (four 16-byte chunks); a 256-byte bank row
// holds four K rows, so chunk j of row r sits at slot j ^ ((r / 4) % 4) and
// the 16 rows of one read phase land on distinct banks.
__device__ __forceinline__ int kswz4(int row, int chunk) {
  return row * (kHeadDim / 2) + ((chunk ^ ((row >> 2) & 3)) << 4);
}

// (native vectors: aggregate copies of HIP's uint4 would go through memory)
// Chunks per thread: 8-bit tiles split evenly; a 4-bit tile has one chunk for
// each of its first 256 threads, and the other threads (if any) repeat them
// (same data to the same LDS bytes), which keeps staging branch-free.
template <int BITS>
constexpr int chunks_per_thread() {
  return BITS == 8 ? kChunks8 / kThreads : (kChunks4 >= kThreads ? kChunks4 / kThreads : 1);
}
template <int BITS>
__device__ __forceinline__ int chunk_id(int tid, int i) {
  return BITS == 8 ? tid + i * kThreads : ((tid + i * kThreads) & (kChunks4 - 1));
}

template <int BITS>
struct StageRegs {
  v4u k[chunks_per_thread<BITS>()];   // 16-byte chunks chunk_id(tid, i) of a K tile
  v4u v[chunks_per_thread<BITS>()];   // same for a V tile
  int32_t meta;                 // threads 0..63: kq_pos; 64, 65: sK, sV bits (K's tile)
};

// K fragments of one tile for the S^T product (A operands of the two 32-key
// halves).  int8: 4 steps of v_mfma_i32_32x32x32_i8, lane half h holding
// channels 32*step + 16h .. +16; E4M3: 2 steps of
// v_mfma_scale_f32_32x32x64_f8f6f4, lane half h holding channels
// 64*step + 32h .. +32.  Q fragments (the B operands) split the channels the
// same way, which is all the dot product needs.
// E2M1 keys against E4M3 queries (2 steps of the same scaled MFMA): the
// 4-bit A operand of lane half h takes the products 16h .. +16 and
// 32 + 16h .. +16 of the step's 64, the 8-bit B operand of half h the
// products 32h .. +32; channels are assigned so that the K fragment is the
// 16 contiguous bytes of channels 64*step + 32h .. +32, and the Q fragment
// the two 16-byte runs at channels 64*step + 16h and 64*step + 32 + 16h.
// E2M1 keys against E2M3 queries (HYQ_FMT_FP4Q6): the 6-bit B operand of
// lane half h pairs element n with element n of the 4-bit A operand's half
// h (measured with one-hot operands), its 32 codes packed 6 bits apart in
// six registers; so the Q fragment is channels 64*step + 32h .. +32, the
// same channels as the K fragment, packed from one code byte each.
template <int FMT>
struct KFrag {
  v4i f[2][4];
};
template <>
struct KFrag<HYQ_FMT_FP8> {
  v8i f[2][2];
};
template <>
struct KFrag<HYQ_FMT_FP4> {
  v4i f[2][2];
};
template <>
struct KFrag<HYQ_FMT_FP4Q6> {
  v4i f[2][2];
};
template <int FMT>
struct QFrag {
  v4i f[4];
};
template <>
struct QFrag<HYQ_FMT_FP8> {
  v8i f[2];
};
template <>
struct QFrag<HYQ_FMT_FP4> {
  v8i f[2];
};
template <>
struct QFrag<HYQ_FMT_FP4Q6> {   // six registers of packed E2M3 codes per step
  v8i f[2];
};

template <int FMT>
__device__ __forceinline__ void read_kfrag(KFrag<FMT>& kf, const KBuf& b, int col, int half) {
#pragma unroll
  for (int kh = 0; kh < 2; ++kh) {
    if constexpr (FMT == HYQ_FMT_FP8) {
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        const v4i lo = *reinterpret_cast<const v4i*>(b.k + kswz(kh * 32 + col, kk * 4 + half * 2));
        const v4i hi = *reinterpret_cast<const v4i*>(b.k + kswz(kh * 32 + col, kk * 4 + half * 2 + 1));
        kf.f[kh][kk] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
      }
    } else if constexpr (kv_fp4(FMT)) {
#pragma unroll
      for (int kk = 0; kk < 2; ++kk)
        kf.f[kh][kk] = *reinterpret_cast<const v4i*>(b.k + kswz4(kh * 32 + col, kk * 2 + half));
    } else {
#pragma unroll
      for (int k4 = 0; k4 < 4; ++k4)
        kf.f[kh][k4] = *reinterpret_cast<const v4i*>(b.k + kswz(kh * 32 + col, k4 * 2 + half));
    }
  }
}

template <int FMT>
__device__ __forceinline__ void read_qfrag(QFrag<FMT>& qf, const int8_t* qrow, bool ok, int half) {
  if constexpr (FMT == HYQ_FMT_FP8) {
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
      qf.f[kk] = ok ? *reinterpret_cast<const v8i*>(qrow + kk * 64 + half * 32) : v8i{};
  } else if constexpr (FMT == HYQ_FMT_FP4) {
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const v4i lo = ok ? *reinterpret_cast<const v4i*>(qrow + kk * 64 + half * 16) : v4i{};
      const v4i hi = ok ? *reinterpret_cast<const v4i*>(qrow + kk * 64 + 32 + half * 16) : v4i{};
      qf.f[kk] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
    }
  } else if constexpr (FMT == HYQ_FMT_FP4Q6) {
    // 32 code bytes (channels 64*kk + 32*half ..) -> 6-bit slots 0..31 of six
    // registers (slot n at bits 6n .. 6n+5); done once per wave
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const v4u lo = ok ? *reinterpret_cast<const v4u*>(qrow + kk * 64 + half * 32) : v4u{};
      const v4u hi = ok ? *reinterpret_cast<const v4u*>(qrow + kk * 64 + half * 32 + 16) : v4u{};
      const uint32_t w[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
      uint32_t r[6] = {0u, 0u, 0u, 0u, 0u, 0u};
#pragma unroll
      for (int n = 0; n < 32; ++n) {
        const uint32_t code = (w[n >> 2] >> (8 * (n & 3))) & 0x3Fu;
        const int bit = 6 * n;
        r[bit >> 5] |= code << (bit & 31);
        if ((bit & 31) > 26) r[(bit >> 5) + 1] |= code >> (32 - (bit & 31));
      }
      qf.f[kk] = v8i{(int)r[0], (int)r[1], (int)r[2], (int)r[3], (int)r[4], (int)r[5], 0, 0};
    }
  } else {
#pragma unroll
    for (int k4 = 0; k4 < 4; ++k4)
      qf.f[k4] = ok ? *reinterpret_cast<const v4i*>(qrow + k4 * 32 + half * 16) : v4i{};
  }
}

// S^T of one tile: int32 (int8 codes) or float32 (E4M3, E2M1 codes) logits.
template <int FMT>
using SVec = std::conditional_t<FMT == HYQ_FMT_INT, v16i, v16f>;

template <int FMT>
__device__ __forceinline__ void qk_tile(SVec<FMT> (&s)[2], const KFrag<FMT>& kf,
                                        const QFrag<FMT>& qf) {
#pragma unroll
  for (int kh = 0; kh < 2; ++kh) {
    s[kh] = SVec<FMT>{};
    if constexpr (FMT == HYQ_FMT_FP8) {
#pragma unroll
      for (int kk = 0; kk < 2; ++kk)   // format 0 = E4M3 for both operands, unit scales
        s[kh] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(kf.f[kh][kk], qf.f[kk], s[kh], 0,
                                                                0, 0, 127, 0, 127);
    } else if constexpr (FMT == HYQ_FMT_FP4) {
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {   // A format 4 = E2M1 (4 registers), B format 0 = E4M3
        const v8i ka = __builtin_shufflevector(kf.f[kh][kk], v4i{}, 0, 1, 2, 3, 4, 5, 6, 7);
        s[kh] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(ka, qf.f[kk], s[kh], 4, 0, 0, 127,
                                                                0, 127);
      }
    } else if constexpr (FMT == HYQ_FMT_FP4Q6) {
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {   // A format 4 = E2M1, B format 2 = E2M3 (6 registers)
        const v8i ka = __builtin_shufflevector(kf.f[kh][kk], v4i{}, 0, 1, 2, 3, 4, 5, 6, 7);
        s[kh] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(ka, qf.f[kk], s[kh], 4, 2, 0, 127,
                                                                0, 127);
      }
    } else {
#pragma unroll
      for (int k4 = 0; k4 < 4; ++k4)
        s[kh] = __builtin_amdgcn_mfma_i32_32x32x32_i8(kf.f[kh][k4], qf.f[k4], s[kh], 0, 0, 0);
    }
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
  int lane, half, col;
};

// K codes and metadata of tile tk, V codes of tile tv.
template <int BITS>
__device__ __forceinline__ void stage_load(StageRegs<BITS>& r, const SegA& a, int tk, int tv,
                                           int tid) {
  constexpr int kRow = BITS == 8 ? kHeadDim : kHeadDim / 2;
  constexpr int vRow = BITS == 8 ? kTile : kTile / 2;
  constexpr int n = chunks_per_thread<BITS>();
  const int t = tk;
  const v4u* kc = reinterpret_cast<const v4u*>(a.kc0 + (size_t)tk * kTile * kRow);
  const v4u* vc = reinterpret_cast<const v4u*>(a.vc0 + (size_t)tv * kHeadDim * vRow);
#pragma unroll
  for (int i = 0; i < n; ++i) r.k[i] = kc[chunk_id<BITS>(tid, i)];
#pragma unroll
  for (int i = 0; i < n; ++i) r.v[i] = vc[chunk_id<BITS>(tid, i)];
  // wave 0: kq_pos; wave 1: lane 0 sK, lane 1 sV; the rest reload sV
  // (choices uniform per wave or between two uniform addresses: no branch)
  const int w = tid >> 6, lane = tid & 63;
  const int32_t* pk = a.kq0 + (size_t)t * kTile + lane;
  const int32_t* psk = reinterpret_cast<const int32_t*>(a.ks0 + t);
  const int32_t* psv = reinterpret_cast<const int32_t*>(a.vs0 + t);
  const int32_t* ps = (w == 1 && lane == 0) ? psk : psv;
  r.meta = *(w == 0 ? pk : ps);
}

// int8 K: chunk q = row*8 + j goes to the swizzled slot of (row, j).  4-bit
// K: chunk tid holds 32 channels of row tid/4, expanded to int8 (16*code)
// and stored as two chunks.  V: f16 [128][kVPitch] in the permuted key order.
template <int BITS, int FMT>
__device__ __forceinline__ void stage_store(KBuf& kb, VBuf& vb, const StageRegs<BITS>& r, int tid,
                                            const VScale& vs) {
  if (BITS == 8) {
#pragma unroll
    for (int i = 0; i < chunks_per_thread<BITS>(); ++i) {
      const int q = chunk_id<BITS>(tid, i);
      *reinterpret_cast<v4u*>(kb.k + kswz(q >> 3, q & 7)) = r.k[i];
    }
#pragma unroll
    for (int i = 0; i < chunks_per_thread<BITS>(); ++i) {
      const int q = chunk_id<BITS>(tid, i);
      const int d = q >> 2, kg = q & 3;   // channel d, keys kg*16 .. +16
      const v4u w = r.v[i];
      uint32_t h[8];
      codes4_to_h<FMT>(w.x, h[0], h[1], vs);   // keys 0..3
      codes4_to_h<FMT>(w.y, h[2], h[3], vs);   // keys 4..7
      codes4_to_h<FMT>(w.z, h[4], h[5], vs);   // keys 8..11
      codes4_to_h<FMT>(w.w, h[6], h[7], vs);   // keys 12..15
      uint8_t* dst = vb.v + d * kVPitch + kg * 32;
      *reinterpret_cast<v4u*>(dst) = v4u{h[0], h[1], h[4], h[5]};
      *reinterpret_cast<v4u*>(dst + 16) = v4u{h[2], h[3], h[6], h[7]};
    }
  } else if constexpr (kv_fp4(FMT)) {
    // E2M1 K: the 16-byte chunk as it is (the MFMA reads 4-bit operands);
    // V: E2M1 -> f16 times 2^e, two codes per conversion, exact
    const int q4 = chunk_id<BITS>(tid, 0);
    *reinterpret_cast<v4u*>(kb.k + kswz4(q4 >> 2, q4 & 3)) = r.k[0];
    const int d = q4 >> 1, kh = q4 & 1;   // channel d, keys kh*32 .. +32 (16 B packed)
    const v4u w = r.v[0];
    const uint32_t ww[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int g16 = 0; g16 < 2; ++g16) {
      uint32_t h[8];   // h[e]: keys 2e, 2e + 1 of the 16
      e2m1x8_to_h(ww[2 * g16], *reinterpret_cast<uint32_t(*)[4]>(&h[0]), vs.f32);
      e2m1x8_to_h(ww[2 * g16 + 1], *reinterpret_cast<uint32_t(*)[4]>(&h[4]), vs.f32);
      uint8_t* dst = vb.v + d * kVPitch + (kh * 2 + g16) * 32;
      *reinterpret_cast<v4u*>(dst) = v4u{h[0], h[1], h[4], h[5]};
      *reinterpret_cast<v4u*>(dst + 16) = v4u{h[2], h[3], h[6], h[7]};
    }
  } else {
    const int q4 = chunk_id<BITS>(tid, 0);
    {
      const int row = q4 >> 2, j4 = q4 & 3;
      const v4u w = r.k[0];
      uint32_t o[8];
      i4x8_to_i8(w.x, o[0], o[1]);
      i4x8_to_i8(w.y, o[2], o[3]);
      i4x8_to_i8(w.z, o[4], o[5]);
      i4x8_to_i8(w.w, o[6], o[7]);
      *reinterpret_cast<v4u*>(kb.k + kswz(row, 2 * j4)) = v4u{o[0], o[1], o[2], o[3]};
      *reinterpret_cast<v4u*>(kb.k + kswz(row, 2 * j4 + 1)) = v4u{o[4], o[5], o[6], o[7]};
    }
    const int d = q4 >> 1, kh = q4 & 1;   // channel d, keys kh*32 .. +32 (16 B packed)
    const v4u w = r.v[0];
    const uint32_t ww[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int g16 = 0; g16 < 2; ++g16) {
      uint32_t bb[4];
      i4x8_to_i8(ww[2 * g16], bb[0], bb[1]);
      i4x8_to_i8(ww[2 * g16 + 1], bb[2], bb[3]);
      uint32_t h[8];
      i8x4_to_h(bb[0], h[0], h[1], vs);
      i8x4_to_h(bb[1], h[2], h[3], vs);
      i8x4_to_h(bb[2], h[4], h[5], vs);
      i8x4_to_h(bb[3], h[6], h[7], vs);
      uint8_t* dst = vb.v + d * kVPitch + (kh * 2 + g16) * 32;
      *reinterpret_cast<v4u*>(dst) = v4u{h[0], h[1], h[4], h[5]};
      *reinterpret_cast<v4u*>(dst + 16) = v4u{h[2], h[3], h[6], h[7]};
    }
  }
  const int w = tid >> 6, lane = tid & 63;
  kb.pos[w == 0 ? lane : (w == 1 ? min(kMetaSK + lane, kMetaSink) : kMetaSink)] = r.meta;
}

// The full-precision key list of a workgroup: nvl vertical lines (idx, seen
// from their position on), then nqb quantizable keys of the per-query band
// (kq[nq0 ..], each seen by the W rows from its position on), then the
// window positions base .. (seen from their position on; in band mode by W
// rows, which is every later row).  Entries at or beyond `count` are padding
// (position HYQ_KQ_POS_PAD, seen by no row, zero rows).
struct FpList {
  const int32_t* vl;
  const int32_t* kq;
  const int32_t* dummy;   // any readable word (entries whose position is computed)
  int nvl, nq0, nqb, base, count, band_w;
};
// Entry e's position comes from a load (vertical lines, band keys) or is
// computed (window); fp_src gives the word to load, always readable, and
// fp_resolve turns the loaded word into (position, last row).
__device__ __forceinline__ const int32_t* fp_src(const FpList& f, int e) {
  return e < f.nvl ? f.vl + e : (e < f.nvl + f.nqb ? f.kq + (f.nq0 + (e - f.nvl)) : f.dummy);
}
__device__ __forceinline__ void fp_resolve(const FpList& f, int e, int32_t w, int& p, int& hi) {
  if (e >= f.count) {
    p = HYQ_KQ_POS_PAD;
    hi = -1;
  } else if (e < f.nvl) {
    p = w;
    hi = INT32_MAX;
  } else if (e < f.nvl + f.nqb) {
    p = w;
    hi = w + f.band_w - 1;
  } else {
    p = f.base + (e - f.nvl - f.nqb);
    hi = f.band_w > 0 ? p + f.band_w - 1 : INT32_MAX;
  }
}

// A full-precision tile in registers.  K: thread tid holds the 16-byte
// chunks q = tid + i * kThreads (key q / 16, channels 8 * (q % 16) ..), with
// the key's position and last row.  V: item q = tid + i * kThreads is the
// chunk q / 32 of the key pair (2 * (q % 32), +1), so that one LDS store
// writes both keys of a channel (adjacent V^T slots) and the 64 lanes of a
// wave (32 pairs, two chunks) hit distinct banks.  Also the position words of
// the same keys of the following tile.
constexpr int kFpPairs = kTile * 16 / kThreads;
constexpr int kFpVItems = (kTile / 2) * 16 / kThreads;
static_assert((kTile * 16) % kThreads == 0 && ((kTile / 2) * 16) % kThreads == 0,
              "full-precision chunks must split evenly");
struct FpRegs {
  v4u k[kFpPairs], v[2 * kFpVItems];
  int32_t pos[kFpPairs], hi[kFpPairs], vpos[2 * kFpVItems];
  int32_t wnext[kFpPairs], vwnext[2 * kFpVItems];
};
__device__ __forceinline__ int fp_kkey(int i) { return ((int)threadIdx.x + i * kThreads) >> 4; }
__device__ __forceinline__ int fp_vkey(int i, int s) {
  return 2 * (((int)threadIdx.x + i * kThreads) & 31) + s;
}
__device__ __forceinline__ int fp_vchunk(int i) { return ((int)threadIdx.x + i * kThreads) >> 5; }

// Position words of tile ft (before its first fp_load).
__device__ __forceinline__ void fp_load_words(FpRegs& r, const FpList& f, int ft) {
#pragma unroll
  for (int i = 0; i < kFpPairs; ++i) r.wnext[i] = *fp_src(f, ft * kTile + fp_kkey(i));
#pragma unroll
  for (int i = 0; i < kFpVItems; ++i)
#pragma unroll
    for (int s = 0; s < 2; ++s) r.vwnext[2 * i + s] = *fp_src(f, ft * kTile + fp_vkey(i, s));
}

// Load the rows of tile ft (padding rows read row 0, zeroed at the store)
// from the position words loaded earlier, then the words of tile ft+1.
// Tiles past the end are all padding.
__device__ __forceinline__ void fp_load(FpRegs& r, const FpList& f, const uint16_t* __restrict__ Kh,
                                        const uint16_t* __restrict__ Vh, int ft, int L) {
#pragma unroll
  for (int i = 0; i < kFpPairs; ++i) {
    int p, hi;
    fp_resolve(f, ft * kTile + fp_kkey(i), r.wnext[i], p, hi);
    r.pos[i] = p;
    r.hi[i] = hi;
    const size_t row = (unsigned)p < (unsigned)L ? (size_t)p : 0;
    r.k[i] = reinterpret_cast<const v4u*>(Kh + row * kHeadDim)[((int)threadIdx.x + i * kThreads) & 15];
  }
#pragma unroll
  for (int i = 0; i < kFpVItems; ++i)
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      int p, hi;
      fp_resolve(f, ft * kTile + fp_vkey(i, s), r.vwnext[2 * i + s], p, hi);
      r.vpos[2 * i + s] = p;
      const size_t row = (unsigned)p < (unsigned)L ? (size_t)p : 0;
      r.v[2 * i + s] = reinterpret_cast<const v4u*>(Vh + row * kHeadDim)[fp_vchunk(i)];
    }
  fp_load_words(r, f, ft + 1);
}

// V^T stores of one key pair (adjacent slots from the even key's) and one
// 16-byte chunk: channel d gets the 32-bit word (f16 of key 2m, of key 2m+1)
// of V / sVref (sVref a power of two: exact for bf16 values of that range,
// down to the f16 subnormals).  Returns the largest |V| of the pair's chunk.
__device__ __forceinline__ float fp_store_vpair(FBuf& b, v4u v0, v4u v1, int key0, int chunk,
                                                float inv_vref) {
  const int slot = vslot(key0);
  float mx = 0.0f;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int d = chunk * 8 + 2 * j;
    const float a0 = __uint_as_float(v0[j] << 16), a1 = __uint_as_float(v1[j] << 16);
    const float b0 = __uint_as_float(v0[j] & 0xffff0000u), b1 = __uint_as_float(v1[j] & 0xffff0000u);
    mx = fmaxf(mx, fmaxf(fabsf(a0), fabsf(a1)));
    mx = fmaxf(mx, fmaxf(fabsf(b0), fabsf(b1)));
    const v2f lo = {a0 * inv_vref, a1 * inv_vref}, hi = {b0 * inv_vref, b1 * inv_vref};
    *reinterpret_cast<v2h*>(b.v + d * kVPitch + slot * 2) = __builtin_convertvector(lo, v2h);
    *reinterpret_cast<v2h*>(b.v + (d + 1) * kVPitch + slot * 2) = __builtin_convertvector(hi, v2h);
  }
  return mx;
}

// Write a loaded tile to LDS: K rows as bf16, V^T as f16 V / sVref,
// positions and last rows.  A V ratio outside the f16 range records
// (tile << 8) | (largest biased exponent of |V|) in ovf (a NaN is not
// recorded: it stays a NaN in f16).
__device__ __forceinline__ void fp_store(FBuf& b, const FpRegs& r, float inv_vref, int tag, int L) {
#pragma unroll
  for (int i = 0; i < kFpPairs; ++i) {
    const int e = fp_kkey(i), col = ((int)threadIdx.x + i * kThreads) & 15;
    const unsigned keep = (unsigned)r.pos[i] < (unsigned)L ? 0xffffffffu : 0u;
    *reinterpret_cast<v4u*>(b.k + e * kKPitchBf + col * 16) = r.k[i] & keep;
    if (col == 0) {
      b.pos[e] = r.pos[i];
      b.hi[e] = r.hi[i];
    }
  }
  float mx = 0.0f;
#pragma unroll
  for (int i = 0; i < kFpVItems; ++i) {
    const unsigned k0 = (unsigned)r.vpos[2 * i] < (unsigned)L ? 0xffffffffu : 0u;
    const unsigned k1 = (unsigned)r.vpos[2 * i + 1] < (unsigned)L ? 0xffffffffu : 0u;
    mx = fmaxf(mx, fp_store_vpair(b, r.v[2 * i] & k0, r.v[2 * i + 1] & k1, fp_vkey(i, 0),
                                  fp_vchunk(i), inv_vref));
  }
  if (!(mx * inv_vref <= 65504.0f)) atomicMax(&b.ovf, (tag << 8) | (int)(__float_as_uint(mx) >> 23));
}

// Rewrite the V^T of a published tile with a new sVref (positions from LDS).
__device__ __forceinline__ void fp_restage_v(FBuf& b, const uint16_t* __restrict__ Vh, int L,
                                             float inv_vref) {
#pragma unroll
  for (int i = 0; i < kFpVItems; ++i) {
    v4u vw[2];
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const int p = b.pos[fp_vkey(i, s)];
      vw[s] = v4u{0u, 0u, 0u, 0u};
      if ((unsigned)p < (unsigned)L)
        vw[s] = reinterpret_cast<const v4u*>(Vh + (size_t)p * kHeadDim)[fp_vchunk(i)];
    }
    fp_store_vpair(b, vw[0], vw[1], fp_vkey(i, 0), fp_vchunk(i), inv_vref);
  }
}

// Visibility of this lane's 32 keys of a full-precision tile to row tq, bit
// kh * 16 + r for accumulator register r of half-tile kh.  Without the band
// every listed key is seen from its position on (padding has a position
// past every row), so only the positions are read.
__device__ __forceinline__ uint32_t fp_vis_mask(const FBuf& b, int tq, int half, bool band) {
  uint32_t m = 0;
#pragma unroll
  for (int kh = 0; kh < 2; ++kh)
#pragma unroll
    for (int rg = 0; rg < 4; ++rg) {
      const int e = kh * 32 + rg * 8 + half * 4;
      const v4i p4 = *reinterpret_cast<const v4i*>(&b.pos[e]);
#pragma unroll
      for (int j = 0; j < 4; ++j) m |= (uint32_t)(p4[j] <= tq) << (kh * 16 + rg * 4 + j);
    }
  if (band) {
    uint32_t mh = 0;
#pragma unroll
    for (int kh = 0; kh < 2; ++kh)
#pragma unroll
      for (int rg = 0; rg < 4; ++rg) {
        const int e = kh * 32 + rg * 8 + half * 4;
        const v4i h4 = *reinterpret_cast<const v4i*>(&b.hi[e]);
#pragma unroll
        for (int j = 0; j < 4; ++j) mh |= (uint32_t)(tq <= h4[j]) << (kh * 16 + rg * 4 + j);
      }
    m &= mh;
  }
  return m;
}

// Online-softmax state of one 32-query block of a wave (each lane owns one
// query and the keys of its half of every 32-key group).
struct NState {
  float m;        // reference max (log2 domain); the true max is <= m + kLazy
  float l;        // this lane's part of the row sum, relative to m
  float corr;     // rescale of acc still to apply: 2^(m_before - m)
  v16f acc[4];    // O^T accumulator, 4 groups of 32 channels
};

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

// General path: causal mask by original position, or a tile whose maximum
// outgrew the reference max.  Raises m to the masked tile
// maximum when needed and rescales l and the accumulator at once (the
// accumulator already holds every P V product of earlier tiles).  No
// per-lane branches, so the cross-lane swap sees every lane's operand; the
// visibility test is evaluated twice rather than kept in registers.
template <typename SV>
__device__ __forceinline__ void softmax_general(NState& ns, const SV (&s)[2], v8h (&p)[4],
                                             float cqk, float fm, bool diag, const int32_t* pos,
                                             int tq, int half) {
  float mx = -INFINITY;
#pragma unroll
  for (int kh = 0; kh < 2; ++kh)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const bool vis = (!diag) | (pos[key_of(kh, r, half)] <= tq);
      mx = fmaxf(mx, vis ? (float)s[kh][r] : -INFINITY);
    }
  mx = xhalf_max(mx);
  lazy_max(ns, mx == -INFINITY ? -INFINITY : mx * cqk);
  apply_corr(ns);
  // the row sum adds the same f16 weights the MFMA uses, divided by fm
  float ps = 0.0f;
#pragma unroll
  for (int kh = 0; kh < 2; ++kh)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const bool vis = (!diag) | (pos[key_of(kh, r, half)] <= tq);
      const float ex = __builtin_amdgcn_exp2f((float)s[kh][r] * cqk - ns.m);
      const _Float16 hp = (_Float16)((vis ? ex : 0.0f) * fm);
      ps += (float)hp;
      p[kh * 2 + (r >> 3)][r & 7] = hp;
    }
  ns.l += ps * __builtin_amdgcn_rcpf(fm);
}

// Softmax of one full-precision tile (logits of hidden keys already -inf):
// raise the reference max when the tile's exceeds it by more than kLazy,
// weights 2^(s * alpha * log2(e) - m) as f16 into p (the B operands of P V),
// and their f16 sum into the row sum.  alpha > 0, so the tile max of the
// scaled logits is the scaled max of the raw ones.
__device__ __forceinline__ void fp_softmax(NState& st, const v16f (&sf)[2], float alpha_log2e,
                                           v8h (&p)[4]) {
  float mx = -INFINITY;
#pragma unroll
  for (int kh = 0; kh < 2; ++kh)
#pragma unroll
    for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sf[kh][r]);
  lazy_max(st, xhalf_max(mx) * alpha_log2e);
  apply_corr(st);
  const v2h one2 = {(_Float16)1.0f, (_Float16)1.0f};
  float ps = 0.0f;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int kh = i >> 3, r = (i & 7) * 2;
    v2f e;
    e[0] = __builtin_amdgcn_exp2f(__builtin_fmaf(sf[kh][r], alpha_log2e, -st.m));
    e[1] = __builtin_amdgcn_exp2f(__builtin_fmaf(sf[kh][r + 1], alpha_log2e, -st.m));
    const v2h pk = __builtin_convertvector(e, v2h);
    ps = __builtin_amdgcn_fdot2(pk, one2, ps, false);
    p[kh * 2 + (r >> 3)][r & 7] = pk[0];
    p[kh * 2 + (r >> 3)][(r & 7) + 1] = pk[1];
  }
  st.l += ps;
}

// One tile of the quantized segment:
//   publish tile c+1 (registers -> LDS) and load tile c+2 into registers;
//   S^T of tile c (int8 MFMA);
//   P V of tile c-1 (weights pprev; zeros when c = 0) interleaved with the
//   fast-path softmax of tile c -> pcur;
//   the general path instead when the tile touches the diagonal, its V
//   scale ratio is tiny, or some weight overflowed the fast-path bound.
// The accumulator never carries a pending rescale between tiles: only the
// general path moves the reference max, and it rescales on the spot.
// PH = c % 4 is a template argument so that every LDS address is a per-lane
// constant plus an immediate offset.
template <int BITS, int FMT, int PH>
__device__ __forceinline__ void segA_tile(Smem& sm, const SegA& a, int c, const QFrag<FMT>& qf,
                                          NState& st, const v8h (&pprev)[4], v8h (&pcur)[4],
                                          StageRegs<BITS>& sr, KFrag<FMT>& kf) {
  // 4-bit integer codes are staged as 16*code
  constexpr float kSub = (BITS == 8 || kv_fp4(FMT)) ? 1.0f : 0.0625f;
  const int tid = threadIdx.x;
  const KBuf& cur = sm.q.kb[PH];
  const VBuf& prv = sm.q.vb[(PH + 1) & 1];
  const float sk = __int_as_float(cur.pos[kMetaSK]) * kSub;
  const float sv = __int_as_float(cur.pos[kMetaSV]) * kSub;
  const int last = __builtin_amdgcn_readfirstlane(cur.pos[kTile - 1]);
  // sV / sVref = fm * 2^ev (sVref a power of two: the product is exact)
  int ev;
  float fm = __builtin_frexpf(sv * a.inv_vref, &ev);
  if (!(sv > 0.0f)) {   // all-zero V block: its V codes are 0, fold nothing
    fm = 1.0f;
    ev = 0;
  }
  const VScale vs = make_vscale(__builtin_ldexpf(1.0f, ev));

  // S^T of tile c (its K fragments arrived during the previous tile)
  SVec<FMT> s[2];
  qk_tile<FMT>(s, kf, qf);
  // publish K(c+2) and V(c) (registers loaded during tile c-1) and load K(c+3)
  // and V(c+1); the conversion runs in the shadow of the MFMAs above.  Past
  // the end the last tile is staged again into the free buffers (no branch).
  stage_store<BITS, FMT>(sm.q.kb[(PH + 2) % kKRing], sm.q.vb[PH & 1], sr, tid, vs);
  stage_load<BITS>(sr, a, min(c + 3, a.n - 1), min(c + 1, a.n - 1), tid);

  // Fast path: weights against the current reference max, without the tile
  // max; accepted unless some lane's weights sum above kFastMax (then some
  // weight may have left the f16 range).  Step i issues the MFMA of
  // (channel group i%4, key group i/4) of P V(c-1) and the weight pair i.
  const float cqk = a.cq * sk;
  const float bias = __builtin_amdgcn_logf(fm) - st.m;   // log2
  const v2h one2 = {(_Float16)1.0f, (_Float16)1.0f};
  // The wave in this loop issues ahead of its SIMD partner while that one
  // stages and runs its S^T MFMAs (measured: 1-2% faster than equal
  // priorities; raising the S^T part instead is slower).
  __builtin_amdgcn_s_setprio(1);
  float ps = 0.0f;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int dg = i & 3, ks = i >> 2;
    const v8h va = *reinterpret_cast<const v8h*>(prv.v + (dg * 32 + a.col) * kVPitch + ks * 32 +
                                                 a.half * 16);
    st.acc[dg] = __builtin_amdgcn_mfma_f32_32x32x16_f16(va, pprev[ks], st.acc[dg], 0, 0, 0);
    const int kh = i >> 3, r = (i & 7) * 2;
    const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf((float)s[kh][r], cqk, bias));
    const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf((float)s[kh][r + 1], cqk, bias));
    v2h pk;
    pk[0] = (_Float16)p0;
    pk[1] = (_Float16)p1;
    ps = __builtin_amdgcn_fdot2(pk, one2, ps, false);
    pcur[kh * 2 + (r >> 3)][r & 7] = pk[0];
    pcur[kh * 2 + (r >> 3)][(r & 7) + 1] = pk[1];
  }
  // keep the fast-path weights computed here, next to the MFMAs, rather
  // than sunk into the branch below that consumes them
  asm volatile("" : "+v"(pcur[0]), "+v"(pcur[1]), "+v"(pcur[2]), "+v"(pcur[3]), "+v"(ps));
  __builtin_amdgcn_s_setprio(0);
  const bool diag = last > a.t0;
  const bool redo = diag || __ballot(!(ps <= kFastMax)) != 0;
  if (redo) {
    softmax_general(st, s, pcur, cqk, fm, diag, cur.pos, a.t0 + a.col, a.half);
  } else {
    st.l = __builtin_fmaf(ps, __builtin_amdgcn_rcpf(fm), st.l);   // 1-ulp reciprocal
  }
  // K fragments of tile c+1 (published by the previous barrier); past the
  // end they read a staged copy and are not used
  read_kfrag<FMT>(kf, sm.q.kb[(PH + 1) % kKRing], a.col, a.half);
  __syncthreads();
}

template <int BITS, int OUT_BF16, int FMT>
__global__ void __launch_bounds__(kThreads, kWgPerCu)
attn_prefill_kernel(const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
                    const uint16_t* __restrict__ V, const int32_t* __restrict__ idx,
                    const int8_t* __restrict__ q_codes, const float* __restrict__ q_scale,
                    const uint8_t* __restrict__ k_codes, const float* __restrict__ k_scale,
                    const uint8_t* __restrict__ v_codes, const float* __restrict__ v_scale,
                    const int32_t* __restrict__ kq_pos, void* __restrict__ out, int Hq, int Hkv,
                    int nbj, int L, int P, int k, int nQ, int n_qblk, int n_kvblk,
                    float alpha_log2e, int band_w) {
  __shared__ Smem sm;
  const int g = Hq / Hkv;
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int half = lane >> 5, col = lane & 31;

  // Work units of one KV head: (block rb of 32 rows, query head hh of the
  // group), ordered by rb; a workgroup takes kWaves consecutive units, longest first.
  constexpr int kRows = 32;
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
  const int tq = t0 + col;                 // this lane's query row
  const bool row_ok = active && tq < L;

  const uint16_t* Kh = K + (size_t)bj * L * kHeadDim;
  const uint16_t* Vh = V + (size_t)bj * L * kHeadDim;
  const int32_t* vl = idx + (size_t)bj * k;

  NState st;
  st.m = kMinusBig;
  st.l = 0.0f;
  st.corr = 1.0f;
#pragma unroll
  for (int dg = 0; dg < 4; ++dg)
#pragma unroll
    for (int r = 0; r < 16; ++r) st.acc[dg][r] = 0.0f;

  // Which keys are visible to rows up to t_last.  A quantized key at
  // position p is seen by rows t >= p + shift: shift = 0 for the fixed window,
  // W for the per-query band (whose rows see p in full precision instead).
  const int shift = BITS == 16 ? 0 : band_w;
  int nvl, nq_tiles, fp_count, fp_base, nq0 = 0, nqb = 0;
  float vref = 1.0f;
  if (BITS == 16) {
    nvl = 0;
    nq_tiles = 0;
    fp_base = 0;
    fp_count = t_last + 1;
  } else {
    nvl = count_le(vl, k, t_last);
    const int tq_last = t_last - shift;        // last quantized position any row sees
    // (for the fixed window tq_last = t_last: the count is nvl, no second search)
    const int nq_vis = tq_last < 0 ? 0 : (tq_last < P ? (tq_last + 1) -
                                          (shift == 0 ? nvl : count_le(vl, k, tq_last)) : nQ);
    nq_tiles = min((nq_vis + kTile - 1) / kTile, n_kvblk);
    fp_base = P;
    if (band_w > 0) {
      // band keys of the workgroup's rows: positions [lo, t_last], lo from its first row
      const int t0_wg = ((wgi * kWaves) / g) * kRows;
      const int lo = max(0, t0_wg + 1 - band_w);
      const int hi_q = min(t_last, P - 1);    // quantizable band keys: non-vertical in [lo, hi_q]
      if (lo <= hi_q) {
        nq0 = lo - count_le(vl, k, lo - 1);    // non-vertical positions below lo
        nqb = (hi_q + 1) - count_le(vl, k, hi_q) - nq0;
      }
      fp_base = max(P, lo);
    }
    fp_count = nvl + nqb + max(0, t_last + 1 - fp_base);
    // sVref: smallest power of two >= every V scale of this head
    float mx = 0.0f;
    for (int i = lane; i < n_kvblk; i += 64) mx = fmaxf(mx, v_scale[(size_t)bj * n_kvblk + i]);
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 64));
    if (BITS == 4 && FMT == HYQ_FMT_INT) mx *= 0.0625f;
    if (mx > 0.0f) {
      int e;
      frexpf(mx, &e);
      e = max(-100, min(100, e));
      vref = ldexpf(1.0f, e);
    }
  }
  float inv_vref = 1.0f / vref;

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
    a.t0 = t0 - shift;   // rows t see quantized positions <= t - shift
    a.cq = alpha_log2e * q_scale[bh * n_qblk + t0 / kBlock];
    a.inv_vref = inv_vref;
    a.lane = lane;
    a.half = half;
    a.col = col;

    QFrag<FMT> qf;
    read_qfrag<FMT>(qf, q_codes + (bh * L + (row_ok ? tq : 0)) * kHeadDim, row_ok, half);

    // prologue: K(0), K(1) into LDS, K(2) and V(0) into registers, the
    // fragments of K(0) read; the V buffer that tile 0 multiplies by zero
    // weights is cleared (no stale NaNs)
    StageRegs<BITS> sr;
    stage_load<BITS>(sr, a, 0, 0, threadIdx.x);
    const VScale unit = make_vscale(1.0f);   // the V written here is cleared below
    stage_store<BITS, FMT>(sm.q.kb[0], sm.q.vb[1], sr, threadIdx.x, unit);
    stage_load<BITS>(sr, a, min(1, nq_tiles - 1), 0, threadIdx.x);
    stage_store<BITS, FMT>(sm.q.kb[1], sm.q.vb[1], sr, threadIdx.x, unit);
    stage_load<BITS>(sr, a, min(2, nq_tiles - 1), 0, threadIdx.x);
    __syncthreads();
    for (int i = threadIdx.x; i < kVBytes / 16; i += kThreads)
      reinterpret_cast<v4u*>(sm.q.vb[1].v)[i] = v4u{0u, 0u, 0u, 0u};
    KFrag<FMT> kf;
    read_kfrag<FMT>(kf, sm.q.kb[0], col, half);
    __syncthreads();

    // the P V of tile c runs in iteration c+1, next to the softmax of c+1;
    // the weights alternate between two register sets
    v8h pa[4], pb[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int e = 0; e < 8; ++e) pa[i][e] = pb[i][e] = (_Float16)0.0f;
    int c = 0;
    for (; c + 3 < nq_tiles; c += 4) {
      segA_tile<BITS, FMT, 0>(sm, a, c, qf, st, pa, pb, sr, kf);
      segA_tile<BITS, FMT, 1>(sm, a, c + 1, qf, st, pb, pa, sr, kf);
      segA_tile<BITS, FMT, 2>(sm, a, c + 2, qf, st, pa, pb, sr, kf);
      segA_tile<BITS, FMT, 3>(sm, a, c + 3, qf, st, pb, pa, sr, kf);
    }
    if (c < nq_tiles) segA_tile<BITS, FMT, 0>(sm, a, c, qf, st, pa, pb, sr, kf);
    if (c + 1 < nq_tiles) segA_tile<BITS, FMT, 1>(sm, a, c + 1, qf, st, pb, pa, sr, kf);
    if (c + 2 < nq_tiles) segA_tile<BITS, FMT, 2>(sm, a, c + 2, qf, st, pa, pb, sr, kf);
    // P V of the last tile
    const v8h (&plast)[4] = (nq_tiles & 1) ? pb : pa;
    const VBuf& lb = sm.q.vb[(nq_tiles - 1) & 1];
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
#pragma unroll
      for (int dg = 0; dg < 4; ++dg) {
        const v8h va = *reinterpret_cast<const v8h*>(lb.v + (dg * 32 + col) * kVPitch + ks * 32 +
                                                     half * 16);
        st.acc[dg] = __builtin_amdgcn_mfma_f32_32x32x16_f16(va, plast[ks], st.acc[dg], 0, 0, 0);
      }
    __syncthreads();   // the FP segment reuses the LDS
  }

  // ---------------- segments B and C: full-precision keys ----------------
  if (fp_count > 0) {
    v8bf qb[8];
    {
      const uint16_t* qrow = Q + (bh * L + (row_ok ? tq : 0)) * kHeadDim;
#pragma unroll
      for (int ks = 0; ks < 8; ++ks) qb[ks] = *reinterpret_cast<const v8bf*>(qrow + ks * 16 + half * 8);
    }
    const int nft = (fp_count + kTile - 1) / kTile;
    FpList fl;
    fl.vl = vl;
    fl.kq = kq_pos + (size_t)bj * n_kvblk * kTile;
    fl.dummy = reinterpret_cast<const int32_t*>(Kh);
    fl.nvl = nvl;
    fl.nq0 = nq0;
    fl.nqb = nqb;
    fl.base = fp_base;
    fl.count = fp_count;
    fl.band_w = shift;
    // prologue: tile 0 published, tile 1 in registers.  Tile f is computed
    // from sm.f[f % 2] while tile f+1 (loaded during tile f-1) is written to
    // the other buffer and the rows of tile f+2 (and the position words of
    // tile f+3) are loaded; one barrier per tile.  Tiles past the end are
    // staged as padding into the free buffer (no branch).
    if (threadIdx.x == 0) sm.f[0].ovf = sm.f[1].ovf = -1;
    FpRegs fr;
    fp_load_words(fr, fl, 0);
    fp_load(fr, fl, Kh, Vh, 0, L);
    __syncthreads();
    fp_store(sm.f[0], fr, inv_vref, 0, L);
    fp_load(fr, fl, Kh, Vh, 1, L);
    __syncthreads();
    for (int ft = 0; ft < nft; ++ft) {
      FBuf& cur = sm.f[ft & 1];
      // without the band the list is ascending: a tile whose last position
      // is at or before the wave's first row is seen whole by every row
      const bool full = shift == 0 && cur.pos[kTile - 1] <= t0;
      uint32_t vis = ~0u;
      if (!full) vis = fp_vis_mask(cur, tq, half, shift > 0);
      {
        // V of this tile outside the f16 range at the current sVref: raise
        // sVref to 2^(E - 134) (every |V| / sVref of the tile below 2^8),
        // rescale the accumulator (exact), restage the tile's V
        const int ov = cur.ovf;
        if ((ov >> 8) == ft) {
          const int ex = max(-100, (ov & 0xff) - 134);
          const float nv = fmaxf(vref, __builtin_ldexpf(1.0f, ex));
          const float c = vref / nv;
#pragma unroll
          for (int dg = 0; dg < 4; ++dg)
#pragma unroll
            for (int r = 0; r < 16; ++r) st.acc[dg][r] *= c;
          vref = nv;
          inv_vref = 1.0f / nv;
          fp_restage_v(cur, Vh, L, inv_vref);
          __syncthreads();
        }
      }
      v16f sf[2];
#pragma unroll
      for (int kh = 0; kh < 2; ++kh) {
#pragma unroll
        for (int r = 0; r < 16; ++r) sf[kh][r] = 0.0f;
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) {
          const v8bf ka = *reinterpret_cast<const v8bf*>(cur.k + (kh * 32 + col) * kKPitchBf +
                                                         ks * 32 + half * 16);
          sf[kh] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qb[ks], sf[kh], 0, 0, 0);
        }
      }
      fp_store(sm.f[(ft + 1) & 1], fr, inv_vref, ft + 1, L);
      fp_load(fr, fl, Kh, Vh, ft + 2, L);
      if (!full) {
#pragma unroll
        for (int kh = 0; kh < 2; ++kh)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            sf[kh][r] = (vis >> (kh * 16 + r)) & 1 ? sf[kh][r] : -INFINITY;
      }
      // f16 weights against f16 V / sVref
      v8h p[4];
      fp_softmax(st, sf, alpha_log2e, p);
#pragma unroll
      for (int ks = 0; ks < 4; ++ks)
#pragma unroll
        for (int dg = 0; dg < 4; ++dg) {
          const v8h va = *reinterpret_cast<const v8h*>(cur.v + (dg * 32 + col) * kVPitch +
                                                       ks * 32 + half * 16);
          st.acc[dg] = __builtin_amdgcn_mfma_f32_32x32x16_f16(va, p[ks], st.acc[dg], 0, 0, 0);
        }
      __syncthreads();
    }
  }

  // ---------------- finalize: O = acc * sVref / l ----------------
  const float ltot = xhalf_sum(st.l);
  const float sc = vref / ltot;
  if (!row_ok) return;
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

template <int BITS, int OB, int FMT>
hipError_t launch_t(const hyq_shape& s, const hyq_sizes& z, const uint16_t* Q,
                    const uint16_t* K, const uint16_t* V, const int32_t* idx,
                    const int8_t* q_codes, const float* q_scale, const uint8_t* k_codes,
                    const float* k_scale, const uint8_t* v_codes, const float* v_scale,
                    const int32_t* kq_pos, float softmax_scale, void* out, hipStream_t st) {
  const int g = s.Hq / s.Hkv;
  const int nrb = (s.L + 31) / 32;
  const int wg_per_bj = (g * nrb + kWaves - 1) / kWaves;
  const int nbj = s.B * s.Hkv;
  const dim3 grid(wg_per_bj * nbj);
  attn_prefill_kernel<BITS, OB, FMT><<<grid, kThreads, 0, st>>>(
      Q, K, V, idx, q_codes, q_scale, k_codes, k_scale, v_codes, v_scale, kq_pos, out, s.Hq,
      s.Hkv, nbj, s.L, z.P, z.k, z.nQ, z.n_qblk, z.n_kvblk, softmax_scale * kLog2e,
      s.window_mode == HYQ_WIN_BAND ? s.window : 0);
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
#define HYQ_LAUNCH(BITS, OB, FMT)                                                              \
  return launch_t<BITS, OB, FMT>(s, z, Q, K, V, idx, q_codes, q_scale, k_codes, k_scale,       \
                                 v_codes, v_scale, kq_pos, softmax_scale, out, st)
  if (s.bits_kv == 16) {
    if (out_dtype) HYQ_LAUNCH(16, 1, HYQ_FMT_INT);
    HYQ_LAUNCH(16, 0, HYQ_FMT_INT);
  } else if (s.bits_kv == 4 && s.kv_format == HYQ_FMT_FP4) {
    if (out_dtype) HYQ_LAUNCH(4, 1, HYQ_FMT_FP4);
    HYQ_LAUNCH(4, 0, HYQ_FMT_FP4);
  } else if (s.bits_kv == 4 && s.kv_format == HYQ_FMT_FP4Q6) {
    if (out_dtype) HYQ_LAUNCH(4, 1, HYQ_FMT_FP4Q6);
    HYQ_LAUNCH(4, 0, HYQ_FMT_FP4Q6);
  } else if (s.bits_kv == 8 && s.kv_format == HYQ_FMT_FP8) {
    if (out_dtype) HYQ_LAUNCH(8, 1, HYQ_FMT_FP8);
    HYQ_LAUNCH(8, 0, HYQ_FMT_FP8);
  } else if (s.bits_kv == 8) {
    if (out_dtype) HYQ_LAUNCH(8, 1, HYQ_FMT_INT);
    HYQ_LAUNCH(8, 0, HYQ_FMT_INT);
  } else {
    if (out_dtype) HYQ_LAUNCH(4, 1, HYQ_FMT_INT);
    HYQ_LAUNCH(4, 0, HYQ_FMT_INT);
  }
#undef HYQ_LAUNCH
}

}  // namespace hyq
