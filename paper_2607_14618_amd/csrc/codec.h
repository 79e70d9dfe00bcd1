// Arrangement of one 64-row x 32-channel chunk and of the group metadata in
// the packed buffer (the layout declared in include/polyq.h).  pack/unpack use
// these helpers; the GEMV and GEMM kernels read the same arrangement.
//
// Chunk: 64 lane slices of 4*b bytes.  Lane l's slice holds the 8 consecutive
// channels 8*(l/16) .. 8*(l/16)+7 of the 4 rows 16*r + (l % 16), r = 0..3 --
// the A-operand fragment of a 16x16x32 MFMA for each of the 4 row sub-tiles.
// Inside the slice the 32 codes form 16 pairs P = 4*r + j (codes 2j and 2j+1 of
// row sub-tile r, i.e. slice code 2P and 2P+1), laid out per bit-width so that
// one pair unpacks with one instruction (see encode_slice).
//
// Group metadata (b <= 8), 256 bytes per (tile, group):
//   [0, 128)   z of row 16*r + i at half (i*4 + r)        (read by lane i, i+16, ...)
//   [128, 256) s of row 16*r + 4*q + e at half (q*16 + r*4 + e)
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace polyq {

// Field position (bit offset in a half-word) of pair p (0..4) of a 3-bit word.
__host__ __device__ constexpr int f3(int p) { return p == 0 ? 0 : p == 1 ? 3 : p == 2 ? 6 : p == 3 ? 10 : 13; }

// Slice code index i (0..31) of row sub-tile r (0..3) and in-fragment channel t (0..7).
__host__ __device__ constexpr int slice_index(int r, int t) { return 8 * r + t; }

// 32 codes of one lane slice -> B words.
//   b = 2, 4, 8, 16: word d holds slice codes [d*P, (d+1)*P), P = 32/b; even
//       codes fill the low half and odd codes the high half, in order: code
//       2p+h of the word sits at bits [16h + b*p, 16h + b*p + b).
//   b = 3: word d (0..2) holds codes 10d .. 10d+9 as five pairs; pair p sits at
//       bits f3(p) .. f3(p)+2 (even code) and 16+f3(p) .. (odd code); codes 30
//       and 31 keep bit j in bit 9 (code 30) and bit 25 (code 31) of word j.
template <int B>
__device__ __forceinline__ void encode_slice(const uint16_t* q, uint32_t* w) {
#pragma unroll
  for (int d = 0; d < B; ++d) w[d] = 0u;
  if constexpr (B == 3) {
#pragma unroll
    for (int i = 0; i < 30; ++i) {
      const int d = i / 10, j = i % 10, p = j >> 1, h = j & 1;
      w[d] |= (static_cast<uint32_t>(q[i]) & 7u) << (16 * h + f3(p));
    }
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const uint32_t c = q[30 + h] & 7u;
#pragma unroll
      for (int j = 0; j < 3; ++j) w[j] |= ((c >> j) & 1u) << (9 + 16 * h);
    }
  } else {
    constexpr int P = 32 / B;
    constexpr uint32_t mask = B == 16 ? 0xFFFFu : ((1u << B) - 1u);
#pragma unroll
    for (int i = 0; i < 32; ++i) {
      const int d = i / P, j = i % P, p = j >> 1, h = j & 1;
      w[d] |= (static_cast<uint32_t>(q[i]) & mask) << (16 * h + B * p);
    }
  }
}

// Code i (0..31) of a lane slice.
template <int B>
__device__ __forceinline__ uint32_t slice_code(const uint32_t* w, int i) {
  if constexpr (B == 3) {
    if (i < 30) {
      const int d = i / 10, j = i % 10, p = j >> 1, h = j & 1;
      return (w[d] >> (16 * h + f3(p))) & 7u;
    }
    const int h = i - 30;
    return ((w[0] >> (9 + 16 * h)) & 1u) | (((w[1] >> (9 + 16 * h)) & 1u) << 1) |
           (((w[2] >> (9 + 16 * h)) & 1u) << 2);
  } else {
    constexpr int P = 32 / B;
    constexpr uint32_t mask = B == 16 ? 0xFFFFu : ((1u << B) - 1u);
    const int d = i / P, j = i % P, p = j >> 1, h = j & 1;
    return (w[d] >> (16 * h + B * p)) & mask;
  }
}

// Byte offset, inside a block region, of lane slice `lane` of block-local chunk c of tile t.
__device__ __forceinline__ int64_t slice_offset(int64_t tile_bytes, int64_t record_bytes,
                                                int meta_bytes, int b, int t, int c, int lane) {
  const int g = c / 4, cc = c % 4;
  return static_cast<int64_t>(t) * tile_bytes + static_cast<int64_t>(g) * record_bytes +
         meta_bytes + static_cast<int64_t>(cc) * 64 * 4 * b + static_cast<int64_t>(lane) * 4 * b;
}

// Half index of z and s of tile row R (0..63) inside a group's 256-byte metadata.
__host__ __device__ constexpr int meta_z_half(int R) { return (R % 16) * 4 + R / 16; }
__host__ __device__ constexpr int meta_s_half(int R) {
  return 64 + ((R % 16) / 4) * 16 + (R / 16) * 4 + (R % 4);
}

}  // namespace polyq
