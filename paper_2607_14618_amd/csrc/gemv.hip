// Decode / small-batch GEMV over the mixed-bit clustered weight (Sec. 4.1-4.2),
// 1 <= M <= 16 tokens, on the matrix cores.
//
// Mapping on gfx950: a wave owns one 64-row tile and a contiguous,
// group-aligned range of one bit block's 32-channel chunks.  For each chunk,
// lane l loads its 4b-byte slice (rows 16r + l%16, r = 0..3, channels
// 8(l/16) .. +7: one contiguous 512 B .. 4 KB run per wave), unpacks the 32
// codes into exact fp16 integers q -- the A fragments of four
// v_mfma_f32_16x16x32_f16, one per 16-row sub-tile -- and the B fragment is the
// 8 activations x'[token l%16][8(l/16) .. +7] from LDS.  The 16 columns of the
// MFMA are the tokens, so M = 1 and M = 16 cost the same.
//
// Unpacking: a code field placed at mantissa bits [f, f+b) of an fp16 half is
// turned into the exact fp16 value (2^(10-f) + q) by OR-ing in the exponent
// field 25-f (one v_and_or_b32 for two codes); adding -(2^(10-f) + z) gives
// q - z exactly for an integer zero point |z| <= 1023 (any other z enters as
// its nearest such integer zi, and the group's fold subtracts
// (z - zi) * sum x' in fp32).  Each 128-channel group
// accumulates into its own fp32 tile, scaled once by the row's fp16 scale:
// y += s * sum_group (q - z) x'.  All products are exact; only fp32
// accumulation rounds.  16-bit channels enter the MFMA as their fp16 weights.
//
// Each wave stages its own channel range of the permuted activations
// x'[k'] = x[perm[k']] (Eq. 9) and of the group metadata into LDS (one token
// gathers through the permutation in-kernel; for several, the host launch
// shuffles x once beforehand and the kernel reads x' as given); the waves of
// a work-group (tile, split) reduce through LDS, and the splits of a tile
// across work-groups are combined by the last-arriving work-group (fixed
// order).
#include <hip/hip_runtime.h>
#include <string.h>

#include <algorithm>
#include <type_traits>

#include "codec.h"
#include "internal.h"

namespace polyq {
namespace {

typedef _Float16 h2 __attribute__((ext_vector_type(2)));
typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int kWaves = 4;  // waves per work-group (the host plan uses the same)

constexpr int kMaxItems = POLYQ_MAX_BATCH;

// One linear of a launch: exactly 64 dwords, so that one vector load (a dword
// per lane) fetches it.
struct GemvItem {
  const uint8_t* packed;
  const int32_t* perm;
  const uint16_t* x;
  float* y;
  float* partial;     // [S][m][n_tiles * 64], only when S > 1
  uint32_t* counter;  // [n_tiles], only when S > 1
  const uint16_t* xscale;  // fp16 [k] factors on x' (one token only), or NULL
  int32_t n, k, m, nblocks, S;
  int32_t wave_lds;       // LDS bytes of one wave's staging region
  int32_t n_tiles, n_chunks;
  uint32_t tiles_magic;   // div_magic(n_tiles)
  int32_t zero_offset;    // LDS offset of the work-group's zero row
  int32_t bits[POLYQ_MAX_BLOCKS];
  int32_t chunk_begin[POLYQ_MAX_BLOCKS];
  int32_t wave_begin[POLYQ_MAX_BLOCKS];  // first wave (per tile) of each block
  int32_t waves[POLYQ_MAX_BLOCKS];       // waves per tile given to each block
  uint32_t magic[POLYQ_MAX_BLOCKS];      // div_magic(waves)
  int32_t tile_bytes[POLYQ_MAX_BLOCKS];
  int64_t block_offset[POLYQ_MAX_BLOCKS];
};

// The launch: work-group (x, y) runs linear y; x = s * n_tiles + tile.
struct GemvBatchArgs {
  GemvItem item[kMaxItems];
};

__device__ __forceinline__ h2 as_h2(uint32_t u) { return __builtin_bit_cast(h2, u); }
__device__ __forceinline__ uint32_t as_u32(h2 v) { return __builtin_bit_cast(uint32_t, v); }
// (a & mask) | c in one v_and_or_b32.  gfx950 VOP3 encodings take no literal,
// so the mask is passed in an SGPR and the exponent field in a VGPR (both are
// loop-invariant and materialized once by the compiler).
__device__ __forceinline__ uint32_t and_or(uint32_t a, uint32_t mask, uint32_t c) {
  uint32_t r;
  asm("v_and_or_b32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "s"(mask), "v"(c));
  return r;
}
// fp16 with exponent field e and zero mantissa, in both halves: value 2^(e-15)
__host__ __device__ constexpr uint32_t magic(int e) {
  return (static_cast<uint32_t>(e) << 10) * 0x00010001u;
}
__device__ __forceinline__ h2 splat(float v) {
  const _Float16 h = static_cast<_Float16>(v);
  return h2{h, h};
}
__device__ __forceinline__ h8 splat8(float v) {
  const _Float16 h = static_cast<_Float16>(v);
  return h8{h, h, h, h, h, h, h, h};
}

// Raw pair values (2^(10-f) + q_even, 2^(10-f) + q_odd) of the 16 pairs of one
// lane slice (pair P = slice codes 2P, 2P+1), and the index of each pair's
// offset in the block's offset list.
template <int B> struct Unpack;

template <> struct Unpack<2> {
  static constexpr int kOffsets = 5;
  static constexpr float offset[kOffsets] = {1024.f, 256.f, 64.f, 16.f, 4.f};
  static constexpr int which[16] = {0, 1, 2, 3, 4, 0, 1, 2, 0, 1, 2, 3, 4, 0, 1, 2};
  __device__ static __forceinline__ void run(const uint32_t* w, uint32_t* v) {
#pragma unroll
    for (int d = 0; d < 2; ++d) {
      const uint32_t u = w[d], t = u >> 10;
      v[8 * d + 0] = and_or(u, 0x00030003u, magic(25));
      v[8 * d + 1] = and_or(u, 0x000C000Cu, magic(23));
      v[8 * d + 2] = and_or(u, 0x00300030u, magic(21));
      v[8 * d + 3] = and_or(u, 0x00C000C0u, magic(19));
      v[8 * d + 4] = and_or(u, 0x03000300u, magic(17));
      v[8 * d + 5] = and_or(t, 0x00030003u, magic(25));
      v[8 * d + 6] = and_or(t, 0x000C000Cu, magic(23));
      v[8 * d + 7] = and_or(t, 0x00300030u, magic(21));
    }
  }
};

template <> struct Unpack<3> {
  static constexpr int kOffsets = 3;
  static constexpr float offset[kOffsets] = {1024.f, 128.f, 16.f};
  static constexpr int which[16] = {0, 1, 2, 0, 1, 0, 1, 2, 0, 1, 0, 1, 2, 0, 1, 0};
  __device__ static __forceinline__ void run(const uint32_t* w, uint32_t* v) {
#pragma unroll
    for (int d = 0; d < 3; ++d) {
      const uint32_t u = w[d], t = u >> 10;
      v[5 * d + 0] = and_or(u, 0x00070007u, magic(25));
      v[5 * d + 1] = and_or(u, 0x00380038u, magic(22));
      v[5 * d + 2] = and_or(u, 0x01C001C0u, magic(19));
      v[5 * d + 3] = and_or(t, 0x00070007u, magic(25));
      v[5 * d + 4] = and_or(t, 0x00380038u, magic(22));
    }
    v[15] = ((w[0] >> 9) & 0x00010001u) | ((w[1] >> 8) & 0x00020002u) |
            ((w[2] >> 7) & 0x00040004u) | magic(25);
  }
};

template <> struct Unpack<4> {
  static constexpr int kOffsets = 2;
  static constexpr float offset[kOffsets] = {1024.f, 64.f};
  static constexpr int which[16] = {0, 1, 0, 1, 0, 1, 0, 1, 0, 1, 0, 1, 0, 1, 0, 1};
  __device__ static __forceinline__ void run(const uint32_t* w, uint32_t* v) {
#pragma unroll
    for (int d = 0; d < 4; ++d) {
      const uint32_t u = w[d], t = u >> 8;
      v[4 * d + 0] = and_or(u, 0x000F000Fu, magic(25));
      v[4 * d + 1] = and_or(u, 0x00F000F0u, magic(21));
      v[4 * d + 2] = and_or(t, 0x000F000Fu, magic(25));
      v[4 * d + 3] = and_or(t, 0x00F000F0u, magic(21));
    }
  }
};

template <> struct Unpack<8> {
  static constexpr int kOffsets = 1;
  static constexpr float offset[kOffsets] = {1024.f};
  static constexpr int which[16] = {0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0};
  __device__ static __forceinline__ void run(const uint32_t* w, uint32_t* v) {
    // bytes of word d: [q(4d), q(4d+2), q(4d+1), q(4d+3)]; v_perm_b32 selects
    // source bytes 4..7 from the word and byte 0 (0x64) from the exponent word.
#pragma unroll
    for (int d = 0; d < 8; ++d) {
      v[2 * d + 0] = __builtin_amdgcn_perm(w[d], 0x64646464u, 0x00060004u);
      v[2 * d + 1] = __builtin_amdgcn_perm(w[d], 0x64646464u, 0x00070005u);
    }
  }
};

typedef unsigned int u2v __attribute__((ext_vector_type(2)));
typedef unsigned int u3v __attribute__((ext_vector_type(3)));
typedef unsigned int u4v __attribute__((ext_vector_type(4)));

// Buffer resource over one tile of one block region (raw, byte-addressed): reads
// past `bytes` return zero.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t tile_rsrc(const uint8_t* base, int64_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(base), static_cast<short>(0),
                                           static_cast<int>(bytes), 0x00020000);
}

// Load one lane slice (4*B bytes) at byte offset voff (per lane) + soff (uniform).
template <int B>
__device__ __forceinline__ void load_slice(__amdgpu_buffer_rsrc_t r, int voff, int soff, uint32_t* w) {
  if constexpr (B == 2) {
    const u2v u = __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, 0);
    w[0] = u.x; w[1] = u.y;
  } else if constexpr (B == 3) {
    const u3v u = __builtin_amdgcn_raw_buffer_load_b96(r, voff, soff, 0);
    w[0] = u.x; w[1] = u.y; w[2] = u.z;
  } else {
#pragma unroll
    for (int i = 0; i < B / 4; ++i) {
      const u4v u = __builtin_amdgcn_raw_buffer_load_b128(r, voff + 16 * i, soff, 0);
      w[4 * i + 0] = u.x; w[4 * i + 1] = u.y; w[4 * i + 2] = u.z; w[4 * i + 3] = u.w;
    }
  }
}

// Ring geometry per bit-width: a slot holds the lane slices of up to NS chunks
// (at most 16 dwords per lane); slots end on multiples of NS chunks of the
// block's group grid, so every slot but a segment's first starts aligned.
template <int B>
struct Geo {
  static constexpr int NS = B == 2 ? 8 : (B <= 4 ? 4 : (B == 8 ? 2 : 1));  // chunks per slot
  static constexpr int CB = 4 * B;                                          // bytes per lane slice
  // dwords between consecutive slices in a slot (3-bit slices start 4-aligned:
  // a 96-bit register tuple must start on an even register)
  static constexpr int SW = B == 3 ? 4 : B;
  static constexpr int META = B <= 8 ? kMetaBytes : 0;
};

struct Slot {
  uint32_t w[16];
};

// Issue the loads of the slot of NS chunks starting at block-local chunk c of
// one tile; positions at or past l1 re-read chunk l1 - 1, so every slot issues
// the same number of loads.  voff = lane * 4B (the lane's slice offset).
template <int B>
__device__ __forceinline__ void issue(Slot& sl, __amdgpu_buffer_rsrc_t r, int record_bytes, int c,
                                      int l1, int voff) {
  using G = Geo<B>;
#pragma unroll
  for (int j = 0; j < G::NS; ++j) {
    const int cj = min(c + j, l1 - 1);
    load_slice<B>(r, voff, (cj >> 2) * record_bytes + G::META + (cj & 3) * (64 * G::CB),
                  &sl.w[j * G::SW]);
  }
}

// State of the group being accumulated: the per-pair constants subtracted
// from the unpacked raw values, c[P] = -(2^(10-f) + z_row) with z_row an
// integer of magnitude <= 1023 (one exact add leaves q - z_row), and the
// group's own accumulators (one f4 per 16-row sub-tile).  In a wave whose zero
// points are not all such integers (`fixed`), the unpack subtracts the nearest
// one, zi = rint(z) clamped to [-1023, 1023], and the fold adds the remainder:
// s (sum (q - zi) x' - (z - zi) sum x').
struct Group {
  h2 c[16];
  f4 part[4];
};

__device__ __forceinline__ h8 frag(const uint32_t* w4) {
  const uint4 u{w4[0], w4[1], w4[2], w4[3]};
  return __builtin_bit_cast(h8, u);
}

// Zero for a pair of fp16 zero points (one dword) that are both integers of
// magnitude <= 1023, else nonzero.  With a = |z| (sign bit cleared), a + 1024
// is exact and lies in [1024, 2048), where the fp16 spacing is 1, exactly when
// a is such an integer: otherwise the sum rounds (then (a + 1024) - 1024 != a)
// or reaches 2048 or beyond (exponent field above 25; NaN and inf included).
// Both halves at once with packed fp16 adds (round to nearest even).
__device__ __forceinline__ uint32_t z_pair_bad(uint32_t w) {
  const uint32_t a = w & 0x7FFF7FFFu;
  const uint32_t k1024 = 0x64006400u;  // fp16 1024 in both halves
  uint32_t u, t;
  asm("v_pk_add_f16 %0, %1, %2" : "=v"(u) : "v"(a), "v"(k1024));
  asm("v_pk_add_f16 %0, %1, %2 neg_lo:[0,1] neg_hi:[0,1]" : "=v"(t) : "v"(u), "v"(k1024));
  return (t ^ a) | ((u & 0x7C007C00u) ^ 0x64006400u);
}

// Zero point used by the unpack in a `fixed` wave: rint(z) clamped to
// [-1023, 1023] (an integer, exact in fp16).
__device__ __forceinline__ float z_int(float z) { return fminf(fmaxf(rintf(z), -1023.f), 1023.f); }

// Group start: this lane's zero points (A-fragment rows 16r + l%16, r = 0..3,
// one 8-byte LDS read) -> the pair constants.
template <int B, bool Fixed>
__device__ __forceinline__ void start_group(const uint8_t* gm, int lane, Group& gs) {
  using U = Unpack<B>;
  const uint2 zz = *reinterpret_cast<const uint2*>(gm + (lane & 15) * 8);
  h2 z01 = as_h2(zz.x), z23 = as_h2(zz.y);
  if constexpr (Fixed) {
    z01 = h2{static_cast<_Float16>(z_int(static_cast<float>(z01[0]))),
             static_cast<_Float16>(z_int(static_cast<float>(z01[1])))};
    z23 = h2{static_cast<_Float16>(z_int(static_cast<float>(z23[0]))),
             static_cast<_Float16>(z_int(static_cast<float>(z23[1])))};
  }
  const h2 zs[4] = {h2{z01[0], z01[0]}, h2{z01[1], z01[1]}, h2{z23[0], z23[0]}, h2{z23[1], z23[1]}};
#pragma unroll
  for (int P = 0; P < 16; ++P) {
    const h2 off = splat(U::offset[U::which[P]]);
    gs.c[P] = -(zs[P >> 2] + off);
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) gs.part[r] = f4{0.f, 0.f, 0.f, 0.f};
}

// Unpack one lane slice of a b <= 8 block into fp16 (q - z) fragments and run
// the four MFMAs of its 16-row sub-tiles.
template <int B>
__device__ __forceinline__ void quant_slice(const uint32_t* w, h8 xb, Group& gs) {
  using U = Unpack<B>;
  uint32_t v[16];
  U::run(w, v);
  uint32_t d[16];
#pragma unroll
  for (int P = 0; P < 16; ++P) {
    d[P] = as_u32(as_h2(v[P]) + gs.c[P]);
  }
#pragma unroll
  for (int r = 0; r < 4; ++r)
    gs.part[r] = __builtin_amdgcn_mfma_f32_16x16x32_f16(frag(&d[4 * r]), xb, gs.part[r], 0, 0, 0);
}

// Group end: acc += s * part.  Lane l holds rows 16r + 4(l/16) + e of token
// l%16; their scales are 16 consecutive halves.  With Fixed (the wave's zero
// points are not all small integers), part first takes the zero-point remainders: part -= (z - zi) * sum x'.  The
// token's sum runs over the group's staged chunks [g0, g1] (block-local): each
// lane adds its quarter (8 channels per chunk, the B fragment it read) and the
// lanes l ^ 16, l ^ 32 hold the other quarters of the same token.  The
// remainders come from the zero points: rows 16r + 4(l/16) + e are halves
// 16(l/16) + 4e + r of the group's zero-point array.
template <bool Fixed>
__device__ __forceinline__ void fold_group(const uint8_t* gm, const uint32_t* xlane, int g0, int g1,
                                           int lane, Group& gs, f4 (&acc)[4]) {
  if constexpr (Fixed) {
    float xsum = 0.f;
    for (int q = g0; q <= g1; ++q) {
      const h8 v = __builtin_bit_cast(h8, *reinterpret_cast<const uint4*>(xlane + q * 16));
#pragma unroll
      for (int e = 0; e < 8; ++e) xsum += static_cast<float>(v[e]);
    }
    xsum += __shfl_xor(xsum, 16);
    xsum += __shfl_xor(xsum, 32);
    const uint4* zp = reinterpret_cast<const uint4*>(gm + 32 * (lane >> 4));
    const uint4 za = zp[0], zb = zp[1];
    const uint32_t zw[8] = {za.x, za.y, za.z, za.w, zb.x, zb.y, zb.z, zb.w};
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int i = 4 * e + r;
        const float z = static_cast<float>(
            __builtin_bit_cast(_Float16, static_cast<uint16_t>(zw[i >> 1] >> (16 * (i & 1)))));
        gs.part[r][e] = fmaf(-(z - z_int(z)), xsum, gs.part[r][e]);
      }
  }
  const uint4* sp = reinterpret_cast<const uint4*>(gm + 128 + (lane >> 4) * 32);
  const uint4 s0 = sp[0], s1 = sp[1];
  const uint32_t sw[8] = {s0.x, s0.y, s0.z, s0.w, s1.x, s1.y, s1.z, s1.w};
#pragma unroll
  for (int r = 0; r < 4; ++r)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int i = 4 * r + e;
      const float sc = static_cast<float>(
          __builtin_bit_cast(_Float16, static_cast<uint16_t>(sw[i >> 1] >> (16 * (i & 1)))));
      acc[r][e] = fmaf(sc, gs.part[r][e], acc[r][e]);
    }
}

// Unpack and accumulate the slot starting at block-local chunk c (chunks
// c .. min(c + NS, l1) - 1).  Wave ranges start on group boundaries, so for
// b <= 4 a slot holds whole groups and slot position j starts a group when
// j % 4 == 0; an 8-bit group spans two slots.  `xlane` is this lane's
// activation fragment of block-local chunk 0 (LDS); `meta` is the LDS copy of
// the metadata of block-local group 0.  Fixed: the wave's zero points are not
// all integers of magnitude <= 1023 (a separate copy of the loop).
template <int B, bool Fixed>
__device__ __forceinline__ void compute(const Slot& sl, int c, int l1, const uint32_t* xlane,
                                        const uint8_t* meta, int lane, Group& gs, f4 (&acc)[4]) {
  using G = Geo<B>;
#pragma unroll
  for (int j = 0; j < G::NS; ++j) {
    const int pos = c + j;
    if (pos >= l1) break;
    const h8 xb = __builtin_bit_cast(h8, *reinterpret_cast<const uint4*>(xlane + pos * 16));
    if constexpr (B == 16) {
#pragma unroll
      for (int r = 0; r < 4; ++r)
        acc[r] = __builtin_amdgcn_mfma_f32_16x16x32_f16(frag(&sl.w[j * G::SW + 4 * r]), xb, acc[r], 0, 0, 0);
    } else {
      const uint8_t* gm = meta + (pos >> 2) * kMetaBytes;
      const bool start = B <= 4 ? (j & 3) == 0 : (j == 0 && (c & 3) == 0);
      if (start) start_group<B, Fixed>(gm, lane, gs);
      quant_slice<B>(&sl.w[j * G::SW], xb, gs);
      const bool end = (B <= 4 && (j & 3) == 3) || (B == 8 && (pos & 3) == 3) || pos == l1 - 1;
      if (end) fold_group<Fixed>(gm, xlane, pos & ~3, pos, lane, gs, acc);
    }
  }
}

// Block-local chunks [l0, l1) of one tile through a three-slot ring: while a
// slot is unpacked the next two are in flight.  A slot is always issued (past
// the segment end it re-reads the last chunk, an L1/L2 hit), so the number of
// loads between a slot's issue and its use is fixed and each wait leaves the
// two younger slots outstanding.  `sa`/`sb` already hold the first two slots.
template <int B, bool Fixed>
__device__ __forceinline__ void run_segment(__amdgpu_buffer_rsrc_t rs, int record_bytes, int l0,
                                            int l1, const uint32_t* xlane, const uint8_t* meta,
                                            int lane, Slot& sa, Slot& sb, f4 (&acc)[4]) {
  constexpr int NS = Geo<B>::NS;
  const int voff = lane * Geo<B>::CB;
  Slot sc;
  Group gs;
  for (int c = l0;;) {
    issue<B>(sc, rs, record_bytes, c + 2 * NS, l1, voff);
    compute<B, Fixed>(sa, c, l1, xlane, meta, lane, gs, acc);
    c += NS;
    if (c >= l1) break;
    issue<B>(sa, rs, record_bytes, c + 2 * NS, l1, voff);
    compute<B, Fixed>(sb, c, l1, xlane, meta, lane, gs, acc);
    c += NS;
    if (c >= l1) break;
    issue<B>(sb, rs, record_bytes, c + 2 * NS, l1, voff);
    compute<B, Fixed>(sc, c, l1, xlane, meta, lane, gs, acc);
    c += NS;
    if (c >= l1) break;
  }
}

template <int B>
__device__ __forceinline__ void preload(__amdgpu_buffer_rsrc_t rs, int rb, int l0, int l1,
                                        int voff, Slot& sa, Slot& sb) {
  issue<B>(sa, rs, rb, l0, l1, voff);
  issue<B>(sb, rs, rb, l0 + Geo<B>::NS, l1, voff);
}

// Dword `dw` of a 64-dword argument record held one dword per lane, as a
// scalar (v_readlane; dw must be wave-uniform).
template <class T>
__device__ __forceinline__ T kfield(uint32_t kv, int dw) {
  if constexpr (sizeof(T) == 8) {
    const uint64_t lo = static_cast<uint32_t>(__builtin_amdgcn_readlane(kv, dw));
    const uint64_t hi = static_cast<uint32_t>(__builtin_amdgcn_readlane(kv, dw + 1));
    return __builtin_bit_cast(T, lo | (hi << 32));
  } else {
    return __builtin_bit_cast(T, static_cast<uint32_t>(__builtin_amdgcn_readlane(kv, dw)));
  }
}
#define ITEM(T, field) kfield<T>(kv, offsetof(GemvItem, field) / 4)

// Block descriptors of the work-group's linear, read from the per-lane copy of
// its argument record with v_readlane at a uniform (possibly run-time) index:
// no dependent loads, and no indexed private array for the compiler to spill
// to scratch memory.
struct Blocks {
  uint32_t kv;
  int nblocks, n_chunks;
  __device__ int bits(int i) const { return kfield<int32_t>(kv, offsetof(GemvItem, bits) / 4 + i); }
  __device__ int cb(int i) const { return kfield<int32_t>(kv, offsetof(GemvItem, chunk_begin) / 4 + i); }
  // a block ends where the next one begins (i + 1 must be a compile-time index
  // or uniform; reads past the last block fall back to the layer end)
  __device__ int ce(int i) const {
    return i + 1 < nblocks ? kfield<int32_t>(kv, offsetof(GemvItem, chunk_begin) / 4 + i + 1) : n_chunks;
  }
  __device__ int64_t off(int i) const {
    return kfield<int64_t>(kv, offsetof(GemvItem, block_offset) / 4 + 2 * i);
  }
  __device__ int tb(int i) const { return kfield<int32_t>(kv, offsetof(GemvItem, tile_bytes) / 4 + i); }
  // record of a group: 256 bytes of metadata (b <= 8) + 4 chunk slices of 256 b bytes
  __device__ int rb(int i) const {
    const int b = bits(i);
    return (b <= 8 ? kMetaBytes : 0) + kChunksPerGroup * 64 * 4 * b;
  }
  __device__ int w0(int i) const { return kfield<int32_t>(kv, offsetof(GemvItem, wave_begin) / 4 + i); }
  __device__ int nw(int i) const { return kfield<int32_t>(kv, offsetof(GemvItem, waves) / 4 + i); }
  __device__ uint32_t magic(int i) const { return kfield<uint32_t>(kv, offsetof(GemvItem, magic) / 4 + i); }
};

__device__ __forceinline__ size_t align16(size_t v) { return (v + 15) & ~static_cast<size_t>(15); }

// Global-address-space view of a device pointer.  Pointers rebuilt from the
// argument block are generic to the compiler; generic (flat) loads also count
// against the LDS counter and may alias LDS, which forces full waits between
// the staging loads and the LDS stores.
template <class T>
__device__ __forceinline__ const __attribute__((address_space(1))) T* gl(const T* p) {
  return (const __attribute__((address_space(1))) T*)(p);
}
// 16 bytes per lane from global memory straight into LDS (no registers): lane
// i writes lds + 16 i; `lds` must be wave-uniform.  Completion is counted like
// any other vector load.
__device__ __forceinline__ void ldg16_to_lds(const void* p, void* lds) {
  __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)(p),
                                   (__attribute__((address_space(3))) void*)(lds), 16, 0, 0);
}
__device__ __forceinline__ uint4 ldg16(const void* p) {
  const u4v v = *gl(reinterpret_cast<const u4v*>(p));
  return uint4{v.x, v.y, v.z, v.w};
}

// One work-group = (linear, 64-row tile, split); its four waves each take one
// block's range of the split (wave_range) and stage their own x'.
__global__ __launch_bounds__(kWaves * 64) void gemv_kernel(const GemvBatchArgs a) {
  extern __shared__ uint32_t smem[];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  // The work-group's linear (blockIdx.y) is read with one vector load (a dword
  // per lane) and broadcast with v_readlane; scalar loads of it would miss the
  // scalar cache line by line.
  const uint32_t* kargs = (const uint32_t*)(__builtin_amdgcn_kernarg_segment_ptr());
  static_assert(sizeof(GemvItem) == 256 && offsetof(GemvBatchArgs, item) == 0, "argument layout");
  const uint32_t kv = kargs[blockIdx.y * 64 + lane];
  const int n_tiles = ITEM(int32_t, n_tiles), S = ITEM(int32_t, S);
  const int local = blockIdx.x;
  const int s = static_cast<int>(
      div_by_magic(static_cast<uint32_t>(local), ITEM(uint32_t, tiles_magic), static_cast<uint32_t>(n_tiles)));
  if (s >= S) return;  // this linear has fewer work-groups than the launch's widest
  const int tile = local - s * n_tiles;
  const int m = ITEM(int32_t, m), nblocks = ITEM(int32_t, nblocks), n_chunks = ITEM(int32_t, n_chunks);
  const Blocks bd{kv, nblocks, n_chunks};
  // this wave's chunks [c0, c1): one block's share (wave_range)
  int c0, c1, first;
  wave_range(__builtin_amdgcn_readfirstlane(s * kWaves + wave), nblocks, n_chunks, bd, &c0, &c1, &first);
  c0 = __builtin_amdgcn_readfirstlane(c0);
  c1 = __builtin_amdgcn_readfirstlane(c1);
  first = __builtin_amdgcn_readfirstlane(first);
  const uint8_t* packed = ITEM(const uint8_t*, packed);
  const int32_t* perm = ITEM(const int32_t*, perm);
  const uint16_t* xg = ITEM(const uint16_t*, x);
  const int kdim = ITEM(int32_t, k);
  // ---- Prologue.  Vector loads complete in issue order, so the order of
  // issue below is the order in which the wave can use them: permutation ->
  // activation gathers and group metadata -> the first two weight slots.  The
  // gathers are waited for (x' into LDS) while the weight slots are still in
  // flight.  Each wave stages only its own channels: the waves of a
  // work-group share no x', so no work-group barrier is needed before the
  // main loop.
  const bool has_work = c0 < c1 && first >= 0;
  const int fb = has_work ? bd.bits(first) : 16, fcb = has_work ? bd.cb(first) : 0;
  const int fl0 = c0 - fcb, fl1 = has_work ? c1 - fcb : 0;
  const int frb = has_work ? bd.rb(first) : 0;
  const int ftb = has_work ? bd.tb(first) : 0;
  const uint8_t* ftile = has_work ? packed + bd.off(first) + static_cast<int64_t>(tile) * ftb : packed;
  // The block's slice offset, formed before any staging load is issued (an
  // opaque value the compiler keeps live: rematerialized later, it would land
  // in a register with a pending load and cost a full wait).
  int fvoff;
  asm volatile("v_mul_u32_u24 %0, %1, %2" : "=v"(fvoff) : "v"(lane), "s"(4 * fb));

  // LDS of this wave: x' rows 0..m-1 for its channels, then its group
  // metadata.  The MFMA columns of absent tokens read the work-group's zero
  // row, which every wave fills for the length of its own range (the same
  // zeros: no barrier needed before its reads).
  const int range = has_work ? (c1 - c0) * kChunk : 0;
  // first channel of the range (0 for a wave without work, whose index loads
  // must still stay inside the permutation array)
  const int kbase = has_work ? c0 * kChunk : 0;
  uint16_t* xs16 = reinterpret_cast<uint16_t*>(reinterpret_cast<uint8_t*>(smem) +
                                               static_cast<size_t>(wave) * ITEM(int32_t, wave_lds));
  uint8_t* wmeta = reinterpret_cast<uint8_t*>(xs16) + align16(m * range * 2);
  uint16_t* zs16 = reinterpret_cast<uint16_t*>(reinterpret_cast<uint8_t*>(smem) + ITEM(int32_t, zero_offset));

  // Steps (1)-(5) run for exactly the number of 512-channel rounds the range
  // needs (one code copy per count and per form of x), so that every load of
  // a step is issued before the first of them is used.
  constexpr int kRound = 64 * 8;
  constexpr int kFastRounds = 4;
  constexpr int kTokBatch = 8;  // tokens staged per memory round trip (m > 1)
  const int fast_end = min(range, kFastRounds * kRound);
  const int rounds = max((fast_end + kRound - 1) / kRound, 1);
  const bool use_perm = perm != nullptr;
  const uint16_t* xsc = ITEM(const uint16_t*, xscale);
  const bool use_scale = xsc != nullptr;  // one token only (the host makes sure)
  // Token 0's activations as a raw buffer of k halves: a byte offset at or
  // past 2k (an index outside [0, k)) reads 0.
  const __amdgpu_buffer_rsrc_t xrs =
      tile_rsrc(reinterpret_cast<const uint8_t*>(xg), 2 * static_cast<int64_t>(kdim));
  const int fg0 = fl0 >> 2, fpieces = (fb <= 8 && fl0 < fl1) ? ((((fl1 - 1) >> 2) + 1 - fg0) * 16) : 0;
  uint4 mv[kFastRounds];
  Slot sa, sb;
  // (3) Metadata of the wave's first groups, 16-byte pieces, one per lane per
  // round (a range of R rounds has at most 64 R pieces within its first four
  // rounds), then (4) the first two weight slots.
  auto issue_meta_and_weights = [&](auto rounds_tag) {
    constexpr int R = decltype(rounds_tag)::value;
#pragma unroll
    for (int u = 0; u < R; ++u) {
      const int j = min(u * 64 + lane, max(fpieces - 1, 0));
      mv[u] = ldg16(ftile + static_cast<int64_t>(fg0 + (j >> 4)) * frb + (j & 15) * 16);
    }
    const __amdgpu_buffer_rsrc_t rs = tile_rsrc(ftile, ftb);
    switch (fb) {
      case 2: preload<2>(rs, frb, fl0, fl1, fvoff, sa, sb); break;
      case 3: preload<3>(rs, frb, fl0, fl1, fvoff, sa, sb); break;
      case 4: preload<4>(rs, frb, fl0, fl1, fvoff, sa, sb); break;
      case 8: preload<8>(rs, frb, fl0, fl1, fvoff, sa, sb); break;
      default: preload<16>(rs, frb, fl0, fl1, fvoff, sa, sb); break;
    }
  };
  // (3') The wave's metadata pieces into LDS, the zero points checked on the
  // way (the unpack subtracts integers with |z| <= 1023 exactly), right after
  // the x' stores of each staging form.
  uint32_t z_bad = 0;  // nonzero once a zero point is not such an integer
  auto meta_store = [&](int j, uint4 v) {
    reinterpret_cast<uint4*>(wmeta)[j] = v;
    if ((j & 15) < kMetaBytes / 32) {  // a piece of zero points
      const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int h = 0; h < 4; ++h) z_bad |= z_pair_bad(w[h]);
    }
  };
  auto store_meta = [&](auto rounds_tag) {
    constexpr int R = decltype(rounds_tag)::value;
#pragma unroll
    for (int u = 0; u < R; ++u)
      if (u * 64 + lane < fpieces) meta_store(u * 64 + lane, mv[u]);
  };
  // (5) x' of token 0 (8 channels per lane and round) and the zero row into LDS.
  auto store_x = [&](int u, uint4 q) {
    const int kk = u * kRound + lane * 8;
    if (kk < fast_end) {
      *reinterpret_cast<uint4*>(xs16 + kk) = q;
      *reinterpret_cast<uint4*>(zs16 + kk) = uint4{0u, 0u, 0u, 0u};
    }
  };
  // x' times the channel factors (Eq. 8's 1/s_j; packed fp16 products, exact
  // for powers of two)
  auto scale8 = [&](uint4 q, uint4 f) {
    return uint4{as_u32(as_h2(q.x) * as_h2(f.x)), as_u32(as_h2(q.y) * as_h2(f.y)),
                 as_u32(as_h2(q.z) * as_h2(f.z)), as_u32(as_h2(q.w) * as_h2(f.w))};
  };
  auto stage_fast = [&](auto rounds_tag, auto perm_tag, auto scale_tag, auto multi_tag) {
    constexpr int R = decltype(rounds_tag)::value;
    constexpr bool SC = decltype(scale_tag)::value;
    constexpr bool MT = decltype(multi_tag)::value;  // several tokens (clustered x, no factors)
    // lanes past the range load the range's first channels again; their
    // values are never stored
    int kp[R];
#pragma unroll
    for (int u = 0; u < R; ++u) {
      const int kk = u * kRound + lane * 8;
      kp[u] = kbase + (kk < fast_end ? kk : 0);
    }
    if constexpr (!decltype(perm_tag)::value) {
      // x already clustered: 8 consecutive channels per lane and round.
      uint4 xv[R], fv[R];
#pragma unroll
      for (int u = 0; u < R; ++u) xv[u] = ldg16(xg + kp[u]);
      if constexpr (SC) {
#pragma unroll
        for (int u = 0; u < R; ++u) fv[u] = ldg16(xsc + kp[u]);
      }
      // the other tokens' x' goes straight into LDS, in the same round trip
      // as token 0's (several tokens come without factors: the host's
      // shuffle applied them)
      if constexpr (MT) {
        for (int t = 1; t < m; ++t) {
#pragma unroll
          for (int u = 0; u < R; ++u)
            if (u * kRound + lane * 8 < fast_end)
              ldg16_to_lds(xg + static_cast<int64_t>(t) * kdim + kbase + u * kRound + lane * 8,
                           xs16 + t * range + u * kRound);
        }
      }
      issue_meta_and_weights(rounds_tag);
#pragma unroll
      for (int u = 0; u < R; ++u) store_x(u, SC ? scale8(xv[u], fv[u]) : xv[u]);
      store_meta(rounds_tag);
      // every load of this form done before the common code: no LDS write of
      // the copies above is left in flight past this point
      if constexpr (MT) __builtin_amdgcn_s_waitcnt(0);
    } else {
      // (1) The permutation of the lane's 8 channels per round, then (2) one
      // 2-byte gather per channel (one memory round trip each).
      uint4 pv[R][2], fv[R];
#pragma unroll
      for (int u = 0; u < R; ++u) {
        pv[u][0] = ldg16(perm + kp[u]);
        pv[u][1] = ldg16(perm + kp[u] + 4);
      }
      if constexpr (SC) {
#pragma unroll
        for (int u = 0; u < R; ++u) fv[u] = ldg16(xsc + kp[u]);
      }
      uint32_t h[R][8];
#pragma unroll
      for (int u = 0; u < R; ++u) {
        const uint32_t p8[8] = {pv[u][0].x, pv[u][0].y, pv[u][0].z, pv[u][0].w,
                                pv[u][1].x, pv[u][1].y, pv[u][1].z, pv[u][1].w};
#pragma unroll
        for (int e = 0; e < 8; ++e)
          h[u][e] = __builtin_amdgcn_raw_buffer_load_b16(xrs, min(p8[e], static_cast<uint32_t>(kdim)) << 1, 0, 0);
      }
      issue_meta_and_weights(rounds_tag);
#pragma unroll
      for (int u = 0; u < R; ++u) {
        const uint4 q{h[u][0] | (h[u][1] << 16), h[u][2] | (h[u][3] << 16), h[u][4] | (h[u][5] << 16),
                      h[u][6] | (h[u][7] << 16)};
        store_x(u, SC ? scale8(q, fv[u]) : q);
      }
      store_meta(rounds_tag);
    }
  };
  using I1 = std::integral_constant<int, 1>;
  using I2 = std::integral_constant<int, 2>;
  using I3 = std::integral_constant<int, 3>;
  using I4 = std::integral_constant<int, 4>;
  using Gather = std::true_type;
  using Clustered = std::false_type;
  // A wave without work stages nothing (and waits for nothing).
  bool exact = true;
  if (has_work) {
    // one copy of the staging per count of rounds, form of x and scaling, so
    // that the unscaled forms issue exactly the loads they did without it
    auto stage = [&](auto perm_tag, auto scale_tag, auto multi_tag) {
      switch (rounds) {
        case 4: stage_fast(I4{}, perm_tag, scale_tag, multi_tag); break;
        case 3: stage_fast(I3{}, perm_tag, scale_tag, multi_tag); break;
        case 2: stage_fast(I2{}, perm_tag, scale_tag, multi_tag); break;
        default: stage_fast(I1{}, perm_tag, scale_tag, multi_tag); break;
      }
    };
    using One = std::false_type;
    using Several = std::true_type;
    if (use_perm) {
      if (use_scale)
        stage(Gather{}, std::true_type{}, One{});
      else
        stage(Gather{}, std::false_type{}, One{});
    } else if (m > 1) {
      stage(Clustered{}, std::false_type{}, Several{});
    } else {
      if (use_scale)
        stage(Clustered{}, std::true_type{}, One{});
      else
        stage(Clustered{}, std::false_type{}, One{});
    }
    // (6) More tokens, or channels past the fast rounds (these loads wait behind
    // the weight slots).  Clustered x: tokens go in batches of kTokBatch, every
    // load of a batch issued before the first of them is used (one memory
    // round trip per batch), a 16-byte load per token.  With a permutation
    // (one token): one 2-byte gather per channel through token 0's bounded
    // buffer (indices outside [0, k) read 0).
    auto stage_slow = [&](int k_lo, int k_hi, int t_lo, bool zero_row) {
      for (int kk = k_lo + lane * 8; kk < k_hi; kk += kRound) {
        // channel factors (one token only: several come scaled by the host's shuffle)
        const uint4 f = use_scale ? ldg16(xsc + kbase + kk) : uint4{0u, 0u, 0u, 0u};
        if (!use_perm) {
          for (int t0 = t_lo; t0 < m; t0 += kTokBatch) {
            uint4 v[kTokBatch];
#pragma unroll
            for (int j = 0; j < kTokBatch; ++j)
              v[j] = ldg16(xg + static_cast<int64_t>(min(t0 + j, m - 1)) * kdim + kbase + kk);
#pragma unroll
            for (int j = 0; j < kTokBatch; ++j)
              if (t0 + j < m)
                *reinterpret_cast<uint4*>(xs16 + (t0 + j) * range + kk) = use_scale ? scale8(v[j], f) : v[j];
          }
        } else {
          // a permutation comes with one token (several take the explicit
          // shuffle first): one 2-byte gather per channel
          const uint4 p0 = ldg16(perm + kbase + kk), p1 = ldg16(perm + kbase + kk + 4);
          const uint32_t p8[8] = {p0.x, p0.y, p0.z, p0.w, p1.x, p1.y, p1.z, p1.w};
          uint32_t h[8];
#pragma unroll
          for (int e = 0; e < 8; ++e)
            h[e] = __builtin_amdgcn_raw_buffer_load_b16(xrs, min(p8[e], static_cast<uint32_t>(kdim)) << 1, 0, 0);
          const uint4 q{h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16)};
          *reinterpret_cast<uint4*>(xs16 + kk) = use_scale ? scale8(q, f) : q;
        }
        if (zero_row) *reinterpret_cast<uint4*>(zs16 + kk) = uint4{0u, 0u, 0u, 0u};
      }
    };
    if (range > fast_end) stage_slow(fast_end, range, 0, true);

      // (7) Metadata pieces past the first four rounds (groups beyond the first
    // 16), stored and checked as in (3').
    for (int j = 4 * 64 + lane; j < fpieces; j += 64)
      meta_store(j, ldg16(ftile + static_cast<int64_t>(fg0 + (j >> 4)) * frb + (j & 15) * 16));
    exact = __all(z_bad == 0);
  }

  // Zero points that are not all integers of magnitude <= 1023 (rare): the
  // group start and fold of this wave take the `fixed` path.
  const bool fixed = !exact;

  // ---- Main loop over the wave's block range.
  f4 acc[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) acc[r] = f4{0.f, 0.f, 0.f, 0.f};
  const int tok = lane & 15;
  if (has_work) {
    const __amdgpu_buffer_rsrc_t rs = tile_rsrc(ftile, ftb);
    // this lane's activation fragment of block-local chunk 0 (token lane%16,
    // or the zero row; channel quarter lane/16), relative to the staged range
    const uint32_t* xlane = reinterpret_cast<const uint32_t*>(tok < m ? xs16 + tok * range : zs16) +
                            4 * (lane >> 4) + (fcb - c0) * 16;
    // metadata of block-local group 0 (only groups >= fl0 / 4 are read)
    const uint8_t* meta = wmeta - fg0 * kMetaBytes;
    auto run = [&](auto fixed_tag) {
      constexpr bool F = decltype(fixed_tag)::value;
      switch (fb) {
        case 2: run_segment<2, F>(rs, frb, fl0, fl1, xlane, meta, lane, sa, sb, acc); break;
        case 3: run_segment<3, F>(rs, frb, fl0, fl1, xlane, meta, lane, sa, sb, acc); break;
        case 4: run_segment<4, F>(rs, frb, fl0, fl1, xlane, meta, lane, sa, sb, acc); break;
        case 8: run_segment<8, F>(rs, frb, fl0, fl1, xlane, meta, lane, sa, sb, acc); break;
        default: run_segment<16, false>(rs, frb, fl0, fl1, xlane, meta, lane, sa, sb, acc); break;
      }
    };
    if (fixed)
      run(std::true_type{});
    else
      run(std::false_type{});
  }

  // Reduce the waves' partial sums (fixed order).  MFMA result layout: lane l
  // holds rows 16r + 4(l/16) + e of token l%16.
  __syncthreads();
  float* red = reinterpret_cast<float*>(smem);
  if (tok < m) {
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
      for (int e = 0; e < 4; ++e) red[(wave * m + tok) * 64 + 16 * r + 4 * (lane >> 4) + e] = acc[r][e];
  }
  __syncthreads();
  // The waves share the output tokens: wave w takes tokens w, w + 4, ... (mw
  // of them; none for w >= m).
  const int mw = m > wave ? (m - wave + kWaves - 1) / kWaves : 0;
  const int n = ITEM(int32_t, n);
  float* y = ITEM(float*, y);
  const int row = tile * 64 + lane;
  auto wg_sum = [&](int mi) {
    float v = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) v += red[(w * m + mi) * 64 + lane];
    return v;
  };
  if (S == 1) {
    for (int j = 0; j < mw; ++j) {
      const int mi = wave + kWaves * j;
      if (row < n) y[static_cast<int64_t>(mi) * n + row] = wg_sum(mi);
    }
    return;
  }
  // Split-K fix-up.  Each partial is written, and later read back and zeroed,
  // with a returning device-scope atomic swap, and a work-group takes its ticket
  // only after the swaps of all its waves have returned (each wave waits for
  // its own, then the work-group barrier): swaps and the ticket add on one
  // address are ordered at that address's device-wide point of coherence, so
  // the work-group whose ticket closes the round (ticket mod S == S-1, whatever
  // the counter held before) reads every partial of the round.  Its waves sum
  // them in split order (deterministic), leave them zero, and one lane resets
  // the counter.  (A release/acquire-fence version is both slower -- every
  // fence writes back or invalidates the XCD's whole L2 -- and was measured to
  // read stale partials.)
  float* partial = ITEM(float*, partial);
  uint32_t* counter = ITEM(uint32_t*, counter);
  const int rows_pad = n_tiles * kTileRows;
  // the wave's j-th token; indices past its last are clamped to it: a repeated
  // swap writes the same value again, and in the finisher a repeated
  // read-and-zero (issued after the real one, from the same lane) returns 0
  auto tok_of = [&](int j) { return wave + kWaves * min(j, mw - 1); };
  // A wave's tokens go in batches of TB (1, 2 or 4: no more than it has,
  // except 3 -> 4), all swaps of a batch in flight at once.  Swaps past the real
  // tokens or splits repeat one address, and the device serializes those.
  auto write_partials = [&](auto tb_tag) {
    constexpr int TB = decltype(tb_tag)::value;
    for (int j0 = 0; j0 < mw; j0 += TB) {
      float old[TB];
#pragma unroll
      for (int j = 0; j < TB; ++j) {
        const int mi = tok_of(j0 + j);
        old[j] = __hip_atomic_exchange(&partial[(static_cast<int64_t>(s) * m + mi) * rows_pad + row],
                                       wg_sum(mi), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
#pragma unroll
      for (int j = 0; j < TB; ++j) asm volatile("" ::"v"(old[j]));  // keep the returning form
    }
  };
  // SB splits of TB tokens in flight at a time (SB: 4, 8, 12 or 16, the
  // smallest that covers S, else 16)
  auto finish = [&](auto tb_tag, auto sb_tag) {
    constexpr int TB = decltype(tb_tag)::value, SB = decltype(sb_tag)::value;
    for (int j0 = 0; j0 < mw; j0 += TB) {
      float v[TB];
#pragma unroll
      for (int j = 0; j < TB; ++j) v[j] = 0.f;
      for (int s0 = 0; s0 < S; s0 += SB) {
        float t[TB][SB];
#pragma unroll
        for (int j = 0; j < TB; ++j)
#pragma unroll
          for (int u = 0; u < SB; ++u)
            t[j][u] = __hip_atomic_exchange(
                &partial[(static_cast<int64_t>(min(s0 + u, S - 1)) * m + tok_of(j0 + j)) * rows_pad + row],
                0.f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
#pragma unroll
        for (int j = 0; j < TB; ++j)
#pragma unroll
          for (int u = 0; u < SB; ++u) v[j] += t[j][u];
      }
#pragma unroll
      for (int j = 0; j < TB; ++j)
        if (j0 + j < mw && row < n) y[static_cast<int64_t>(tok_of(j0 + j)) * n + row] = v[j];
    }
  };
  auto finish_sb = [&](auto tb_tag) {
    if (S <= 4)
      finish(tb_tag, std::integral_constant<int, 4>{});
    else if (S <= 8)
      finish(tb_tag, std::integral_constant<int, 8>{});
    else if (S <= 12)
      finish(tb_tag, std::integral_constant<int, 12>{});
    else
      finish(tb_tag, std::integral_constant<int, 16>{});
  };
  using One = std::integral_constant<int, 1>;
  using Two = std::integral_constant<int, 2>;
  using Four = std::integral_constant<int, 4>;
  if (mw == 1)
    write_partials(One{});
  else if (mw == 2)
    write_partials(Two{});
  else if (mw > 2)
    write_partials(Four{});
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_waitcnt(0);  // this wave's swaps have returned
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __syncthreads();  // ... and every other wave's (the partial sums in LDS are dead)
  uint32_t* tk = reinterpret_cast<uint32_t*>(smem);
  if (wave == 0 && lane == 0)
    *tk = __hip_atomic_fetch_add(&counter[tile], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __syncthreads();
  const uint32_t ticket = __builtin_amdgcn_readfirstlane(*tk);
  if (ticket % static_cast<uint32_t>(S) != static_cast<uint32_t>(S - 1)) return;
  if (mw == 1)
    finish_sb(One{});
  else if (mw == 2)
    finish_sb(Two{});
  else if (mw > 2)
    finish_sb(Four{});
  if (wave == 0 && lane == 0) __hip_atomic_store(&counter[tile], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

}  // namespace
}  // namespace polyq

using namespace polyq;

namespace {

// Plans of a batch: every linear's splits are sized for the whole launch.
// Workspace: per item its split-K region (counters, partials; the part that
// must be zero on entry and is zero again on return), then one clustered copy
// x' = x[:, perm] (times the channel factors of Eq. 8, if any) per distinct
// (x, perm, factors) of the items that take Eq. 9's explicit shuffle (several
// tokens with a permutation or factors: each wave then stages its tokens'
// activations with 16-byte loads instead of one 2-byte gather per channel and
// token).
struct BatchPlan {
  GemvPlan plans[POLYQ_MAX_BATCH];
  size_t split_off[POLYQ_MAX_BATCH];
  int64_t xp_off[POLYQ_MAX_BATCH];  // -1: the item reads x as given
  bool xp_first[POLYQ_MAX_BATCH];   // this item's copy is made here (not shared with an earlier item)
  size_t zero, total, lds;
};

polyq_status plan_batch(const polyq_gemv_item* items, int32_t count, int32_t m, BatchPlan* bp) {
  if (items == nullptr || count < 1) return POLYQ_ERR_ARG;
  if (count > POLYQ_MAX_BATCH) return POLYQ_ERR_CAPACITY;
  if (m < 1) return POLYQ_ERR_ARG;
  if (m > POLYQ_MAX_M_GEMV) return POLYQ_ERR_CAPACITY;
  int tiles = 0;
  for (int i = 0; i < count; ++i) {
    if (!layout_is_valid(items[i].layout)) return POLYQ_ERR_ARG;
    tiles += items[i].layout->n_tiles;
  }
  size_t off = 0, l = 0;
  for (int i = 0; i < count; ++i) {
    const polyq_layout& L = *items[i].layout;
    if (plan_gemv(L, m, tiles, &bp->plans[i]) != 0 || bp->plans[i].W != kWaves) return POLYQ_ERR_CAPACITY;
    bp->split_off[i] = off;
    off += static_cast<size_t>(align_up(static_cast<int64_t>(gemv_workspace_for(L, m, bp->plans[i])), 256));
    l = std::max(l, gemv_lds_bytes(bp->plans[i], m));
  }
  bp->zero = off;
  for (int i = 0; i < count; ++i) {
    bp->xp_off[i] = -1;
    bp->xp_first[i] = false;
    if (m == 1 || (items[i].perm == nullptr && items[i].xscale == nullptr)) continue;
    for (int j = 0; j < i; ++j)
      if (bp->xp_off[j] >= 0 && items[j].perm == items[i].perm && items[j].x == items[i].x &&
          items[j].xscale == items[i].xscale && items[j].layout->k == items[i].layout->k) {
        bp->xp_off[i] = bp->xp_off[j];
        break;
      }
    if (bp->xp_off[i] < 0) {
      bp->xp_off[i] = static_cast<int64_t>(off);
      bp->xp_first[i] = true;
      off += static_cast<size_t>(align_up(static_cast<int64_t>(m) * items[i].layout->k * 2, 256));
    }
  }
  bp->total = off;
  bp->lds = l;
  return POLYQ_OK;
}

// Pointer and alignment checks of every item (the planner reads only the
// layouts, permutations and activation pointers).
polyq_status check_items(const polyq_gemv_item* items, int32_t count) {
  for (int i = 0; i < count; ++i) {
    const polyq_gemv_item& t = items[i];
    if (t.packed == nullptr || t.x == nullptr || t.y == nullptr) return POLYQ_ERR_ARG;
    if (reinterpret_cast<uintptr_t>(t.packed) % 256 != 0) return POLYQ_ERR_ARG;
    if (reinterpret_cast<uintptr_t>(t.x) % 16 != 0 || reinterpret_cast<uintptr_t>(t.y) % 4 != 0 ||
        reinterpret_cast<uintptr_t>(t.perm) % 16 != 0 || reinterpret_cast<uintptr_t>(t.xscale) % 16 != 0)
      return POLYQ_ERR_ARG;  // activations, permutation and factors are read as 16-byte vectors
    for (int b = 0; b < t.layout->nblocks; ++b)
      if (t.layout->tile_bytes[b] > INT32_MAX) return POLYQ_ERR_UNSUPPORTED;
  }
  return POLYQ_OK;
}

}  // namespace

namespace polyq {

polyq_status gemv_batch_workspace_status(const polyq_gemv_item* items, int32_t count, int32_t m,
                                         size_t* need, size_t* zero) {
  BatchPlan bp;
  const polyq_status st = plan_batch(items, count, m, &bp);
  if (st != POLYQ_OK) return st;
  const polyq_status ct = check_items(items, count);
  if (ct != POLYQ_OK) return ct;
  *need = bp.total;
  *zero = bp.zero;
  return POLYQ_OK;
}

}  // namespace polyq

extern "C" size_t polyq_gemv_batch_workspace_bytes(const polyq_gemv_item* items, int32_t count,
                                                   int32_t m) {
  BatchPlan bp;
  if (plan_batch(items, count, m, &bp) != POLYQ_OK) return 0;
  return bp.total;
}

extern "C" size_t polyq_gemv_batch_workspace_zero_bytes(const polyq_gemv_item* items, int32_t count,
                                                        int32_t m) {
  BatchPlan bp;
  if (plan_batch(items, count, m, &bp) != POLYQ_OK) return 0;
  return bp.zero;
}

extern "C" polyq_status polyq_gemv_batch(const polyq_gemv_item* items, int32_t count, int32_t m,
                                         void* workspace, size_t workspace_bytes, void* stream) {
  BatchPlan bp;
  const polyq_status st = plan_batch(items, count, m, &bp);
  if (st != POLYQ_OK) return st;
  const polyq_status ct = check_items(items, count);
  if (ct != POLYQ_OK) return ct;
  if (bp.total > 0 && (workspace == nullptr || workspace_bytes < bp.total)) return POLYQ_ERR_CAPACITY;
  if (bp.total > 0 && reinterpret_cast<uintptr_t>(workspace) % 256 != 0) return POLYQ_ERR_ARG;

  uint8_t* ws = static_cast<uint8_t*>(workspace);
  GemvBatchArgs a;
  memset(&a, 0, sizeof(a));
  int wgs = 0;
  for (int i = 0; i < count; ++i) {
    const polyq_gemv_item& t = items[i];
    const polyq_layout& L = *t.layout;
    const GemvPlan& p = bp.plans[i];
    GemvItem& g = a.item[i];
    const bool shuffled = bp.xp_off[i] >= 0;
    g.packed = static_cast<const uint8_t*>(t.packed);
    g.perm = shuffled ? nullptr : t.perm;
    g.xscale = shuffled ? nullptr : t.xscale;
    g.x = shuffled ? reinterpret_cast<const uint16_t*>(ws + bp.xp_off[i]) : t.x;
    g.y = t.y;
    g.partial = nullptr;
    g.counter = nullptr;
    if (p.S > 1) {  // [counters: n_tiles x u32, 256-aligned][partials: S x m x n_tiles*64 fp32]
      uint8_t* w = ws + bp.split_off[i];
      g.counter = reinterpret_cast<uint32_t*>(w);
      g.partial = reinterpret_cast<float*>(w + align_up(static_cast<int64_t>(L.n_tiles) * 4, 256));
    }
    g.n = L.n;
    g.k = L.k;
    g.m = m;
    g.nblocks = L.nblocks;
    g.S = p.S;
    g.wave_lds = static_cast<int32_t>(gemv_wave_lds_bytes(p, m));
    g.zero_offset = static_cast<int32_t>(gemv_zero_offset(p, m));
    g.n_tiles = L.n_tiles;
    g.n_chunks = L.n_chunks;
    g.tiles_magic = div_magic(static_cast<uint32_t>(L.n_tiles));
    int w0 = 0;
    for (int b = 0; b < POLYQ_MAX_BLOCKS; ++b) {
      const bool used = b < L.nblocks;
      g.bits[b] = used ? L.block[b].bits : 0;
      g.chunk_begin[b] = used ? L.k_begin[b] / kChunk : L.n_chunks;
      g.wave_begin[b] = w0;
      g.waves[b] = used ? p.waves[b] : 0;
      g.magic[b] = div_magic(static_cast<uint32_t>(g.waves[b]));
      w0 += g.waves[b];
      g.block_offset[b] = used ? L.block_offset[b] : 0;
      g.tile_bytes[b] = used ? static_cast<int32_t>(L.tile_bytes[b]) : 0;
    }
    wgs = std::max(wgs, L.n_tiles * p.S);
  }
  hipStream_t hs = static_cast<hipStream_t>(stream);
  // Eq. 9's explicit shuffle first (with Eq. 8's factors folded in), once per
  // distinct (x, perm, factors) of several tokens
  ShuffleJob jobs[kMaxItems];
  int njobs = 0;
  for (int i = 0; i < count; ++i)
    if (bp.xp_first[i])
      jobs[njobs++] = ShuffleJob{items[i].perm, items[i].xscale, items[i].x,
                                 reinterpret_cast<uint16_t*>(ws + bp.xp_off[i]), items[i].layout->k, 0};
  launch_shuffle(jobs, njobs, m, false, hs);
  hipLaunchKernelGGL(gemv_kernel, dim3(wgs, count), dim3(kWaves * 64), bp.lds, hs, a);
  return hipGetLastError() == hipSuccess ? POLYQ_OK : POLYQ_ERR_DEVICE;
}

extern "C" polyq_status polyq_gemv(const polyq_layout* layout, const void* packed,
                                   const int32_t* perm, const uint16_t* x, int32_t m, float* y,
                                   void* workspace, size_t workspace_bytes, void* stream) {
  const polyq_gemv_item item{layout, packed, perm, x, y, nullptr};
  return polyq_gemv_batch(&item, 1, m, workspace, workspace_bytes, stream);
}
