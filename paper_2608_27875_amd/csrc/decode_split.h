// Host-side choice of the decode attention launch shape: how many workgroups
// per KV head take quantized blocks (S_q) and how many take full-precision
// tiles (S_f).  Plain C++ (no HIP), so that the policy can be checked on any
// host.
//
// By default a quantized wave takes about 32 KB of codes (u blocks: 4 int4 or
// 2 8-bit) and a full-precision wave one tile.  The decode loop is bound by
// each SIMD's vector ALU, so a launch takes about as long as its busiest SIMD:
// (workgroups on the busiest CU) x (bytes of the busiest wave).  When the
// default leaves the CUs unevenly loaded (312 workgroups on 256 CUs: some CUs
// run two), the launch is reshaped to k workgroups per CU with fewer, longer
// splits, and the full-precision tiles per wave chosen so that no wave reads
// many more bytes than the others; the shape with the smallest busiest-SIMD
// bytes wins.  Splits never exceed the default, which bounds the workspace.
#pragma once

#include <algorithm>
#include <cstdint>

namespace hyq {

struct DecodeShape {
  int S_q;   // workgroups per KV head over the quantized blocks
  int S_f;   // workgroups per KV head over the full-precision tiles
};

// nbq quantized blocks and nft full-precision tiles per KV head; `heads` KV
// heads in the launch; `waves` waves per workgroup; u blocks per wave by
// default; blk_bytes / tile_bytes per block / tile; n_cu compute units.
inline DecodeShape choose_decode_split(int64_t nbq, int64_t nft, int64_t heads, int64_t n_cu,
                                       int waves, int u, int64_t blk_bytes, int64_t tile_bytes) {
  DecodeShape d;
  d.S_q = (int)((nbq + (int64_t)waves * u - 1) / ((int64_t)waves * u));
  d.S_f = (int)((nft + waves - 1) / waves);
  if (d.S_q == 0 || heads <= 0 || n_cu <= 0) return d;
  auto wave_bytes = [&](int64_t s_q, int64_t s_f) {
    const int64_t blks = (nbq + waves * s_q - 1) / (waves * s_q);
    const int64_t tiles = s_f ? (nft + waves * s_f - 1) / (waves * s_f) : 0;
    return std::max(blks * blk_bytes, tiles * tile_bytes);
  };
  const int sq_def = d.S_q, sf_def = d.S_f;   // the bounds of every candidate
  const int64_t rounds = ((int64_t)(sq_def + sf_def) * heads + n_cu - 1) / n_cu;
  int64_t best = rounds * wave_bytes(sq_def, sf_def);
  for (int64_t k = 1; k < rounds && k <= 32; ++k) {
    const int64_t fit = k * n_cu / heads;   // workgroups per KV head
    for (int f = 1; f <= 4; ++f) {          // full-precision tiles per wave
      const int64_t s_f = (nft + (int64_t)waves * f - 1) / ((int64_t)waves * f);
      const int64_t s_q = std::min<int64_t>(sq_def, fit - s_f);
      if (s_q < 1 || s_f > sf_def) continue;
      const int64_t cost = k * wave_bytes(s_q, s_f);
      if (cost < best) {
        best = cost;
        d.S_q = (int)s_q;
        d.S_f = (int)s_f;
      }
    }
  }
  return d;
}

// Waves per workgroup of the decode attention kernel.
constexpr int kDecodeWaves = 4;

// The launch shape the decode kernel uses for nbq quantized blocks and nft
// full-precision tiles per KV head at `bits` (8 or 4): the defaults above
// filled in from the kernel's geometry (64-token blocks and tiles of 128
// channels; u = 4 int4 or 2 8-bit blocks per wave).
inline DecodeShape decode_shape_for(int64_t nbq, int64_t nft, int64_t heads, int64_t n_cu,
                                    int bits) {
  return choose_decode_split(nbq, nft, heads, n_cu, kDecodeWaves, bits == 4 ? 4 : 2,
                             2LL * 64 * 128 * bits / 8,   // K and V codes of a block
                             2LL * 64 * 128 * 2);         // K and V bf16 rows of a tile
}

}  // namespace hyq
