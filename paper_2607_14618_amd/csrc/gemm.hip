// Prefill GEMM over the mixed-bit clustered weight (Sec. 4.1-4.2), M tokens:
//   y[m][n] = sum_k' w_hat[n][k'] x'[m][k'],  x' = x[:, perm] (Eq. 9)
//
// Prefill is a dense contraction, so it runs on the bf16 matrix cores
// (v_mfma_f32_16x16x32_bf16, fp32 accumulation).  A work-group of 8 waves owns
// 256 tokens x 128 weight rows (two packed tiles) and walks K one 32-channel
// chunk at a time through a two-stage LDS ring:
//   * every thread prefetches, three chunks ahead of their multiply (two
//     register slots), 32 bytes of activations and
//     its share of the packed chunk (8 codes of one row: one row sub-tile of
//     one lane slice) plus that row's zero point and scale;
//   * the packed share is dequantized once per work-group into a bf16 tile in
//     LDS that all waves multiply (weights are the MFMA A operand, activations
//     the B operand);
//   * wave (tq, rt) multiplies rows 64 rt.. by tokens 64 tq..: 16 MFMAs per
//     chunk; one barrier per chunk.
// The loop is specialized per bit-width: a block's chunks run through the
// copy of the loop compiled for its bit-width, one 128-channel group per
// iteration, so the unpack, the group start and the group fold are fixed at
// compile time and a step's common path has no branch.  The blocks (whose
// bit-widths ascend) are visited by straight-line code, one copy per
// bit-width, so that no loop carries the accumulators through every copy.
// Each block starts in LDS stage 0, so chunk i of a group always sits in
// stage i & 1 (compile-time addresses).  In the steady part of a block a
// thread fetches exactly the packed words it unpacks (4, 8, 12 or 16 bytes)
// and each step's instructions are issued in a fixed interleaving: fragment
// reads, then every MFMA followed by part of the next chunk's dequantization.
//
// Numerics.  The dequantized operand is (q - z), an integer of magnitude
// <= 255 that bf16 holds exactly when z is an integer in [0, 255]; each
// 128-channel group accumulates into its own fp32 tile, which is then scaled
// by the row's fp16 scale s (fp32 FMA) into the output accumulator.  A code
// field at bit f of a half-word, OR-ed with the fp16 exponent field 25 - f,
// reads as the fp16 value 2^(10-f) + q (exact), and one packed fp16 add of
// -(2^(10-f) + z) leaves q - z exactly for such z; the bf16 value is the upper
// half of its fp32 conversion.  A 16-bit channel, or a group whose zero point
// is not such an integer, enters as the pair hi + lo of bf16 values (two
// MFMAs): for fp16 weights the pair is exact; for any other z, q is recovered
// exactly in fp32 and q - z rounds once before the split.
#include <hip/hip_runtime.h>

#include <string.h>

#include <algorithm>
#include <type_traits>

#include "codec.h"
#include "internal.h"

namespace polyq {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef _Float16 h2 __attribute__((ext_vector_type(2)));
typedef uint32_t u4v __attribute__((ext_vector_type(4)));
typedef uint32_t u3v __attribute__((ext_vector_type(3)));
typedef uint32_t u2v __attribute__((ext_vector_type(2)));

constexpr int kTokWG = 256;                 // tokens per work-group
constexpr int kRowsWG = 2 * kTileRows;      // weight rows per work-group (two packed tiles)
constexpr int kThreads = 512;               // 8 waves
constexpr int kLdsRow = 48;                 // bf16 per LDS row: 32 channels + 16 pad (96-byte rows: fewest bank conflicts measured among 16-byte-aligned strides)
constexpr int kStageA = kTokWG * kLdsRow;   // bf16 of one activation stage
constexpr int kStageB = kRowsWG * kLdsRow;  // bf16 of one weight tile (hi or lo) of a stage

// One linear of a launch.
struct GemmItem {
  const uint8_t* packed;
  const uint16_t* x;  // bf16 [m][k], clustered order
  float* y;           // fp32 [m][n]
  int32_t n, k, nblocks, n_tiles, n_chunks;
  int32_t y_vec;  // rows of y can take 16-byte stores (n % 4 == 0, y 16-byte aligned)
  int32_t bits[POLYQ_MAX_BLOCKS];
  int32_t cb[POLYQ_MAX_BLOCKS];  // first chunk of each block
  int32_t ce[POLYQ_MAX_BLOCKS];  // end chunk of each block
  int32_t pad;
  int64_t off[POLYQ_MAX_BLOCKS];
  int64_t tb[POLYQ_MAX_BLOCKS];  // bytes of one packed tile of the block
  int64_t rb[POLYQ_MAX_BLOCKS];  // bytes of one group record (meta + 4 chunks)
};

// A launch: the linears' work-groups one after another (item i owns
// work-groups wg_begin[i] .. wg_begin[i + 1] - 1), all with the same m.
// K is split (count == 1 only) into `splits` chunk ranges starting at group
// boundaries (split_chunk, unused when splits == 1); split s writes its sums
// to partial[s][m][n] and a second kernel adds the splits in order.
constexpr int kMaxSplits = 8;

struct GemmBatchArgs {
  GemmItem item[POLYQ_MAX_BATCH];
  int32_t count, m, m_tiles, splits;
  int32_t wg_begin[POLYQ_MAX_BATCH + 1];
  int32_t split_chunk[kMaxSplits + 1];
  float* partial;
};

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), static_cast<short>(0),
                                           static_cast<int>(bytes), 0x00020000);
}

// Prefetched data of one chunk for one thread.
struct Pre {
  u4v av[2];     // two 16-byte activation pieces
  u4v w;         // 16 bytes at this thread's row sub-tile of its lane slice (b bytes used, 12 for 3 bits)
  uint32_t z, s; // fp16 zero point and scale of the thread's row (loaded at a group's first chunk)
};

__host__ __device__ constexpr uint32_t exp_field(int e) { return (static_cast<uint32_t>(e) << 10) * 0x00010001u; }

// The fields at bits f and 16 + f of w (mask m2 covers both, already shifted
// to f) as the fp16 pair (2^(10-f) + q_even, 2^(10-f) + q_odd).
__device__ __forceinline__ uint32_t field_pair(uint32_t w, uint32_t m2, int f) {
  return (w & m2) | exp_field(25 - f);
}

// The 4 code pairs (channels 2j, 2j+1) of row sub-tile r of a lane slice, in
// the arrangement of codec.h, as fp16 pairs (off[j] + q) with off[j] =
// 2^(10 - f) for the field position f each pair is read at.  `w` holds the
// 16 bytes loaded at the sub-tile's offset (sub_offset); r is wave-uniform.
template <int B>
__device__ __forceinline__ void unpack_sub_tile(const u4v w, int r, uint32_t* hp) {
  if constexpr (B == 2) {  // word r/2 holds sub-tiles r & ~1 (bits 0..7) and r | 1 (8..15)
    const uint32_t u = w.x >> (8 * (r & 1));
    hp[0] = field_pair(u, 0x00030003u, 0);
    hp[1] = field_pair(u, 0x000C000Cu, 2);
    hp[2] = field_pair(u, 0x00300030u, 4);
    hp[3] = field_pair(u, 0x00C000C0u, 6);
  } else if constexpr (B == 4) {  // word r, pairs at 0, 4, 8, 12
    const uint32_t t = w.x >> 8;
    hp[0] = field_pair(w.x, 0x000F000Fu, 0);
    hp[1] = field_pair(w.x, 0x00F000F0u, 4);
    hp[2] = field_pair(t, 0x000F000Fu, 0);
    hp[3] = field_pair(t, 0x00F000F0u, 4);
  } else if constexpr (B == 8) {  // words 2r, 2r+1, pairs at bytes (0, 2) and (1, 3); 0x64 = exponent 25
    hp[0] = __builtin_amdgcn_perm(w.x, 0x64646464u, 0x00060004u);
    hp[1] = __builtin_amdgcn_perm(w.x, 0x64646464u, 0x00070005u);
    hp[2] = __builtin_amdgcn_perm(w.y, 0x64646464u, 0x00060004u);
    hp[3] = __builtin_amdgcn_perm(w.y, 0x64646464u, 0x00070005u);
  } else {  // B == 3: pair P = 4r + j in word P/5 at f3(P%5); fields at 10, 13 read after >> 10
    const uint32_t t0 = w.x >> 10, t1 = w.y >> 10, t2 = w.z >> 10;
    switch (r) {
      case 0:
        hp[0] = field_pair(w.x, 0x00070007u, 0);
        hp[1] = field_pair(w.x, 0x00380038u, 3);
        hp[2] = field_pair(w.x, 0x01C001C0u, 6);
        hp[3] = field_pair(t0, 0x00070007u, 0);
        break;
      case 1:
        hp[0] = field_pair(t0, 0x00380038u, 3);
        hp[1] = field_pair(w.y, 0x00070007u, 0);
        hp[2] = field_pair(w.y, 0x00380038u, 3);
        hp[3] = field_pair(w.y, 0x01C001C0u, 6);
        break;
      case 2:
        hp[0] = field_pair(t1, 0x00070007u, 0);
        hp[1] = field_pair(t1, 0x00380038u, 3);
        hp[2] = field_pair(w.z, 0x00070007u, 0);
        hp[3] = field_pair(w.z, 0x00380038u, 3);
        break;
      default:  // codes 30, 31: bit d of each in bits 9 and 25 of word d
        hp[0] = field_pair(w.z, 0x01C001C0u, 6);
        hp[1] = field_pair(t2, 0x00070007u, 0);
        hp[2] = field_pair(t2, 0x00380038u, 3);
        hp[3] = ((w.x >> 9) & 0x00010001u) | ((w.y >> 8) & 0x00020002u) | ((w.z >> 7) & 0x00040004u) |
                exp_field(25);
        break;
    }
  }
}

// off[j] of unpack_sub_tile for sub-tile r.
template <int B>
__device__ __forceinline__ void pair_offsets(int r, float* off) {
  if constexpr (B == 2) {
    off[0] = 1024.f; off[1] = 256.f; off[2] = 64.f; off[3] = 16.f;
  } else if constexpr (B == 4) {
    off[0] = 1024.f; off[1] = 64.f; off[2] = 1024.f; off[3] = 64.f;
  } else if constexpr (B == 8) {
    off[0] = off[1] = off[2] = off[3] = 1024.f;
  } else {
    const float t[4][4] = {{1024.f, 128.f, 16.f, 1024.f}, {128.f, 1024.f, 128.f, 16.f},
                           {1024.f, 128.f, 1024.f, 128.f}, {16.f, 1024.f, 128.f, 1024.f}};
    switch (r) {
      case 0: for (int j = 0; j < 4; ++j) off[j] = t[0][j]; break;
      case 1: for (int j = 0; j < 4; ++j) off[j] = t[1][j]; break;
      case 2: for (int j = 0; j < 4; ++j) off[j] = t[2][j]; break;
      default: for (int j = 0; j < 4; ++j) off[j] = t[3][j]; break;
    }
  }
}

__device__ __forceinline__ uint32_t hi_half_pair(float lo, float hi) {
  return __builtin_amdgcn_perm(__builtin_bit_cast(uint32_t, hi), __builtin_bit_cast(uint32_t, lo),
                               0x07060302u);
}

// fp32 -> bf16 bits, round to nearest even (finite inputs).
__device__ __forceinline__ uint32_t bf16_rne(float f) {
  const uint32_t u = __builtin_bit_cast(uint32_t, f);
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

// Eight values of one row as the bf16 pair hi (nearest) + lo (nearest to the
// remainder).
__device__ __forceinline__ void store_pair(const float* v, uint16_t* hi_dst, uint16_t* lo_dst) {
  uint32_t hb[8], lb[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    hb[i] = bf16_rne(v[i]);
    lb[i] = bf16_rne(v[i] - __builtin_bit_cast(float, hb[i] << 16));
  }
  *reinterpret_cast<uint4*>(hi_dst) =
      uint4{hb[0] | (hb[1] << 16), hb[2] | (hb[3] << 16), hb[4] | (hb[5] << 16), hb[6] | (hb[7] << 16)};
  *reinterpret_cast<uint4*>(lo_dst) =
      uint4{lb[0] | (lb[1] << 16), lb[2] | (lb[3] << 16), lb[4] | (lb[5] << 16), lb[6] | (lb[7] << 16)};
}

// Byte offset of row sub-tile r inside a lane slice of a b-bit chunk (the
// word(s) holding its codes; 3-bit slices are read whole).
__device__ __forceinline__ int sub_offset(int b, int r) {
  return b == 2 ? (r >> 1) * 4 : b == 4 ? r * 4 : b == 8 ? r * 8 : b == 16 ? r * 16 : 0;
}

template <int V>
using Int = std::integral_constant<int, V>;

__global__ __launch_bounds__(kThreads) void gemm_kernel(const GemmBatchArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t lds_a[2 * kStageA];      // [stage][token][channel]
  __shared__ __attribute__((aligned(16))) uint16_t lds_b[2 * 2 * kStageB];  // [stage][hi, lo][row][channel]
  __shared__ __attribute__((aligned(16))) float lds_r[2 * kRowsWG];         // [stage][row] group scale
  __shared__ int lds_tag[2];  // chunk index + 1 when the stage holds a nonzero lo tile

  const int tid = threadIdx.x, lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int tq = wv & 3, rt = wv >> 2;  // MFMA role: token quarter, packed tile
  // Token tile fastest: neighbouring work-groups (on different XCDs) share the
  // weight rows, and each XCD's work-groups keep to a subset of token tiles.
  int idx = 0;
#pragma unroll
  for (int i = 1; i < POLYQ_MAX_BATCH; ++i) idx += (i < a.count && static_cast<int>(blockIdx.x) >= a.wg_begin[i]) ? 1 : 0;
  const GemmItem& it = a.item[idx];
  const int local = static_cast<int>(blockIdx.x) - a.wg_begin[idx];
  const int mt = local % a.m_tiles, rest = local / a.m_tiles;
  const int ks = rest % a.splits, rp = rest / a.splits;
  const int m0 = mt * kTokWG;
  // this work-group's chunks [c0, C), c0 at a group boundary
  const int c0 = a.splits > 1 ? a.split_chunk[ks] : 0;
  const int C = a.splits > 1 ? a.split_chunk[ks + 1] : it.n_chunks;
  int b0 = 0;
#pragma unroll
  for (int j = 0; j < POLYQ_MAX_BLOCKS - 1; ++j) b0 += (j + 1 < it.nblocks && c0 >= it.ce[j]) ? 1 : 0;

  // Dequantization role: packed tile dp, row sub-tile dr (wave-uniform), lane
  // slice `lane`: row drow of the tile, channels 8 (lane / 16) .. + 7.
  const int dp = wv >> 2, dr = wv & 3;
  const int dt = rp * 2 + dp;
  const bool dtile_ok = dt < it.n_tiles;
  const int drow = 16 * dr + (lane & 15);
  const int bst = (dp * 64 + drow) * kLdsRow + 8 * (lane >> 4);  // LDS slot of its 8 weights
  const int sst = dp * 64 + drow;                                  // LDS slot of its row's scale

  // Activations: buffer over rows m0 .. m0 + 255 of x' (reads past row m - 1
  // return zero); piece j of this thread is token piece/4, 16-byte segment piece%4.
  const __amdgpu_buffer_rsrc_t xrs =
      make_rsrc(it.x + static_cast<int64_t>(m0) * it.k, static_cast<uint32_t>(min(a.m - m0, kTokWG)) * it.k * 2u);
  uint32_t avoff[2];
  int ast[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int piece = tid + j * kThreads;
    avoff[j] = (static_cast<uint32_t>(piece >> 2) * it.k + (piece & 3) * 8) * 2u;
    ast[j] = (piece >> 2) * kLdsRow + (piece & 3) * 8;
  }
  // MFMA fragment reads: tokens 64 tq + 16 j + lane%16 (B), rows 64 rt + 16 i + lane%16 (A)
  const int ard = (tq * 64 + (lane & 15)) * kLdsRow + 8 * (lane >> 4);
  const int brd = (rt * 64 + (lane & 15)) * kLdsRow + 8 * (lane >> 4);

  // Load cursor: the next chunk to fetch, its block and a buffer over this
  // thread's packed tile of that block (no records for a tile past the end,
  // so its reads return zero).  Block-generic: it runs ahead of the
  // bit-width-specialized loop across block boundaries.
  int lc = c0, lb = 0, lcl = 0, lbits = 0, lce = 0, lrb = 0;
  uint32_t lvoff = 0;
  __amdgpu_buffer_rsrc_t wrs;
  auto set_block = [&](int b) __attribute__((always_inline)) {
    lb = b;
    lbits = it.bits[b];
    lce = it.ce[b];
    lrb = static_cast<int>(it.rb[b]);
    const int64_t tb = it.tb[b];
    wrs = make_rsrc(it.packed + it.off[b] + static_cast<int64_t>(dtile_ok ? dt : 0) * tb,
                    dtile_ok ? static_cast<uint32_t>(tb) : 0u);
    lvoff = static_cast<uint32_t>(lane * 4 * lbits + sub_offset(lbits, dr));
    lcl = 0;
  };
  const uint32_t zvoff = 2 * meta_z_half(drow), svoff = 2 * meta_s_half(drow);
  auto load = [&](Pre& pr) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < 2; ++j)
      pr.av[j] = __builtin_bit_cast(u4v, __builtin_amdgcn_raw_buffer_load_b128(xrs, avoff[j], lc * 64, 0));
    const int rec = (lcl >> 2) * lrb;
    const int soff = rec + (lbits <= 8 ? kMetaBytes : 0) + (lcl & 3) * 256 * lbits;
    pr.w = __builtin_bit_cast(u4v, __builtin_amdgcn_raw_buffer_load_b128(wrs, lvoff, soff, 0));
    // the row's z and s of the chunk's group (used at a group's first chunk;
    // loaded for every chunk, so that every slot has the same loads in flight
    // and each wait can leave the younger slot's loads outstanding)
    pr.z = __builtin_amdgcn_raw_buffer_load_b16(wrs, zvoff, rec, 0);
    pr.s = __builtin_amdgcn_raw_buffer_load_b16(wrs, svoff, rec, 0);
    ++lc;
    ++lcl;
    if (lc == lce && lc < C) set_block(lb + 1);
  };
  // The same for a chunk known to lie in the current block, of bit-width B:
  // the packed words are fetched with a load of exactly their size (4, 8, 12
  // or 16 bytes), which the memory pipeline serves faster than a 16-byte load
  // at a 4-byte offset, and no block boundary is checked.  The row's z and s
  // are fetched only for a group's first chunk (`zs`, known at compile time
  // in the steady loop): their 2-byte loads, four lanes to an address, cost
  // the memory pipeline about as much as the activations' 16-byte loads.
  auto load_in_block = [&](auto b_tag, Pre& pr, bool zs) __attribute__((always_inline)) {
    constexpr int B = decltype(b_tag)::value;
#pragma unroll
    for (int j = 0; j < 2; ++j)
      pr.av[j] = __builtin_bit_cast(u4v, __builtin_amdgcn_raw_buffer_load_b128(xrs, avoff[j], lc * 64, 0));
    const int rec = (lcl >> 2) * lrb;
    const int soff = rec + (B <= 8 ? kMetaBytes : 0) + (lcl & 3) * 256 * B;
    if constexpr (B == 16) {
      pr.w = __builtin_bit_cast(u4v, __builtin_amdgcn_raw_buffer_load_b128(wrs, lvoff, soff, 0));
    } else if constexpr (B == 8) {
      const u2v v = __builtin_bit_cast(u2v, __builtin_amdgcn_raw_buffer_load_b64(wrs, lvoff, soff, 0));
      pr.w = u4v{v.x, v.y, 0u, 0u};
    } else if constexpr (B == 3) {
      const u3v v = __builtin_bit_cast(u3v, __builtin_amdgcn_raw_buffer_load_b96(wrs, lvoff, soff, 0));
      pr.w = u4v{v.x, v.y, v.z, 0u};
    } else {
      pr.w = u4v{__builtin_amdgcn_raw_buffer_load_b32(wrs, lvoff, soff, 0), 0u, 0u, 0u};
    }
    if (zs) {
      pr.z = __builtin_amdgcn_raw_buffer_load_b16(wrs, zvoff, rec, 0);
      pr.s = __builtin_amdgcn_raw_buffer_load_b16(wrs, svoff, rec, 0);
    }
    ++lc;
    ++lcl;
  };

  // Group state of the thread's row while its group is being stored: scale,
  // zero point, whether every zero point of the wave is an integer in
  // [0, 255] (wave-uniform), and the pair constants -(off[j] + z).
  float gs = 0.f, gz = 0.f;
  bool gexact = true;
  h2 gc[4];
  // bit st: this thread's lo slot of stage st may hold nonzero values (a
  // 16-bit chunk or a pair-stored group used it); cleared before an exact
  // store into the stage, since a stage's second MFMA pass reads every row.
  uint32_t lo_dirty = 0;

  // Dequantize one chunk (prefetched in pr) into stage st, with its rows'
  // group scales.  first: the chunk starts a group (its z and s are in pr).
  // The exact form (integer zero points) is always written, without
  // branches; store_fix then rewrites the chunk as hi + lo pairs in a wave
  // whose zero points are not all such integers.
  auto store_main = [&](auto b_tag, const Pre& pr, int c, int st, bool first) __attribute__((always_inline)) {
    constexpr int B = decltype(b_tag)::value;
    uint16_t* sa = lds_a + st * kStageA;
#pragma unroll
    for (int j = 0; j < 2; ++j) *reinterpret_cast<u4v*>(sa + ast[j]) = pr.av[j];
    uint16_t* hi = lds_b + st * 2 * kStageB + bst;
    uint16_t* lo = hi + kStageB;
    if constexpr (B == 16) {
      lds_r[st * kRowsWG + sst] = 1.f;  // the four threads of a row store the same value
      const uint32_t ww[4] = {pr.w.x, pr.w.y, pr.w.z, pr.w.w};
      float v[8];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const h2 h = __builtin_bit_cast(h2, ww[i]);
        v[2 * i] = static_cast<float>(h.x);
        v[2 * i + 1] = static_cast<float>(h.y);
      }
      store_pair(v, hi, lo);
      lo_dirty |= 1u << st;
      return;
    }
    if (first) {
      float off[4];
      pair_offsets<B>(dr, off);
      gz = static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(pr.z)));
      gs = static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(pr.s)));
      gexact = __all(gz == truncf(gz) && gz >= 0.f && gz <= 255.f);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const _Float16 cz = static_cast<_Float16>(-(off[j] + gz));  // exact when gexact
        gc[j] = h2{cz, cz};
      }
    }
    lds_r[st * kRowsWG + sst] = gs;
    uint32_t hp[4];
    unpack_sub_tile<B>(pr.w, dr, hp);
    // (off + q) - (off + z) = q - z exactly in fp16 (|q - z| <= 255), and
    // exactly again in fp32 and in its upper half (bf16)
    uint32_t o[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const h2 d = __builtin_bit_cast(h2, hp[j]) + gc[j];
      o[j] = hi_half_pair(static_cast<float>(d.x), static_cast<float>(d.y));
    }
    *reinterpret_cast<uint4*>(hi) = uint4{o[0], o[1], o[2], o[3]};
  };
  auto store_fix = [&](auto b_tag, const Pre& pr, int c, int st) __attribute__((always_inline)) {
    constexpr int B = decltype(b_tag)::value;
    uint16_t* hi = lds_b + st * 2 * kStageB + bst;
    uint16_t* lo = hi + kStageB;
    if constexpr (B == 16) {
      if (tid == 0) lds_tag[st] = c + 1;
      return;
    }
    if (__builtin_expect(gexact, 1)) {
      if (__builtin_expect(lo_dirty & (1u << st), 0)) {
        *reinterpret_cast<uint4*>(lo) = uint4{0u, 0u, 0u, 0u};
        lo_dirty &= ~(1u << st);
      }
      return;
    }
    // any other fp16 z: (off + q) - off = q exactly, then q - z rounds once
    float off[4];
    pair_offsets<B>(dr, off);
    uint32_t hp[4];
    unpack_sub_tile<B>(pr.w, dr, hp);
    float v[8];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const h2 h = __builtin_bit_cast(h2, hp[j]);
      v[2 * j] = (static_cast<float>(h.x) - off[j]) - gz;
      v[2 * j + 1] = (static_cast<float>(h.y) - off[j]) - gz;
    }
    store_pair(v, hi, lo);
    lo_dirty |= 1u << st;
    lds_tag[st] = c + 1;  // any thread; every writer stores the same value
  };

  f4 T[4][4], P[4][4];  // output accumulators, the group's partial sums
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) T[i][j] = f4{0.f, 0.f, 0.f, 0.f};

  // MFMA pass over stage st: the hi tile (first: fresh partial sums) or the
  // lo tile.
  auto mfma_pass = [&](int st, bool first, int tile) __attribute__((always_inline)) {
    const uint16_t* sa = lds_a + st * kStageA;
    const uint16_t* sb = lds_b + st * 2 * kStageB + tile * kStageB;
    bf16x8 af[4], bfr[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      af[i] = *reinterpret_cast<const bf16x8*>(sb + brd + i * 16 * kLdsRow);
      bfr[i] = *reinterpret_cast<const bf16x8*>(sa + ard + i * 16 * kLdsRow);
    }
    if (first) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          P[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[j], f4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) P[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[j], P[i][j], 0, 0, 0);
    }
  };
  // Group fold: total += s * part, s of rows 16 i + 4 (lane/16) + e
  // (stage st holds the group's last chunk and its scales).
  auto fold = [&](int st) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const f4 sv = *reinterpret_cast<const f4*>(&lds_r[st * kRowsWG + rt * 64 + 16 * i + 4 * (lane >> 4)]);
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int e = 0; e < 4; ++e) T[i][j][e] = fmaf(sv[e], P[i][j][e], T[i][j][e]);
    }
  };

  // A chunk sits in a register slot from its load (two chunks ahead) to its
  // store (one chunk ahead), and in an LDS stage from its store to its
  // multiply; both alternate chunk by chunk.  `sc` is the slot the next step
  // stores from, `sn` the other (it holds the chunk after that); a step that
  // ends a block leaves its slot, holding the next block's first chunk, for
  // that block's entry.  The slots are named, not indexed, so that they stay
  // in registers: after an odd number of steps their contents trade places.
  Pre sc, sn;
  if (tid < 2) lds_tag[tid] = 0;
  *reinterpret_cast<uint4*>(lds_b + kStageB + bst) = uint4{0u, 0u, 0u, 0u};  // lo slots of both stages
  *reinterpret_cast<uint4*>(lds_b + 3 * kStageB + bst) = uint4{0u, 0u, 0u, 0u};
  set_block(b0);
  lcl = c0 - it.cb[b0];
  load(sn);
  if (C - c0 > 1) load(sc);
  __syncthreads();  // the tags and cleared lo slots before the first store
  int c = c0;  // next chunk to multiply

  // Chunks [c, cend) of one block of bit-width B, from a group boundary.  The
  // loop is compiled per bit-width, one group of four chunks per iteration:
  // the unpack, the group start and the group end are fixed at compile time
  // and the common path of a step has no branch.
  auto run_block = [&](auto b_tag, int cend) __attribute__((always_inline)) {
    constexpr int B = decltype(b_tag)::value;
    // entry: the block's first chunk, still in sn, into stage 0 (the last
    // barrier left both stages free), so that stage indices are compile-time
    // constants: chunk i of a group sits in stage i & 1
    store_main(b_tag, sn, c, 0, true);
    store_fix(b_tag, sn, c, 0);
    if (c + 2 < C) load(sn);
    __syncthreads();
    // One step: multiply chunk c (stage st); if `more` (chunk c + 1 is in the
    // block) store chunk c + 1 (`nf`: it starts a group) from `slot` into the
    // other stage and fetch chunk c + 3 into it (`inner`: known to be in the
    // split); fold a group that ends with chunk c.  `two`: the group's chunks
    // carry lo tiles (every chunk of a group is stored the same way, since its
    // zero points are the group's, so the tag is read at its first chunk).
    bool two = B == 16;
    auto step = [&](Pre& slot, int st, bool first, bool last, bool nf, bool more, bool inner,
                    bool in_block = false, bool zs = true) __attribute__((always_inline)) {
      if (B != 16 && first) two = __builtin_expect(lds_tag[st] == c + 1, 0);
      mfma_pass(st, first, 0);
      if (more) store_main(b_tag, slot, c + 1, st ^ 1, nf);
      if (in_block) {
        // issue order of a steady step: the eight fragment reads, then each
        // MFMA followed by two VALU instructions of the next chunk's
        // dequantization and, every few MFMAs, one of its LDS stores (the
        // wave keeps its VALU and LDS work flowing while the matrix pipe is
        // busy, instead of leaving it all after the MFMAs)
        __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);
#pragma unroll
        for (int m = 0; m < 16; ++m) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x002, 2, 0);
          if (m == 3 || m == 7 || m == 11 || m == 13) __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);
        }
      }
      if (two) mfma_pass(st, false, 1);
      if (last) fold(st);
      if (more) {
        store_fix(b_tag, slot, c + 1, st ^ 1);
        if (in_block) load_in_block(b_tag, slot, zs);
        else if (inner || c + 3 < C) load(slot);
      }
      ++c;
      __syncthreads();
    };
    // Every group but the block's last: all four steps have their next chunk
    // in the block and (three chunks ahead) in the split, so every step
    // issues the same loads and each wait leaves the younger slot in flight.
    // In all but the last two groups the chunk fetched (at most six ahead of
    // the group's first) is in the block too.
    const int nch = cend - c;
    const int full = (nch - 1) / 4;
    // (step i fetches chunk i + 3 of the group: only step 1's starts a group)
    for (int g = full - 1; g > 0; --g) {
      step(sc, 0, true, false, false, true, true, true, false);
      step(sn, 1, false, false, false, true, true, true, true);
      step(sc, 0, false, false, false, true, true, true, false);
      step(sn, 1, false, true, true, true, true, true, false);
    }
    if (full > 0) {
      step(sc, 0, true, false, false, true, true);
      step(sn, 1, false, false, false, true, true);
      step(sc, 0, false, false, false, true, true);
      step(sn, 1, false, true, true, true, true);
    }
    // The block's last group: 1 .. 4 chunks.
    const int r = cend - c;
    step(sc, 0, true, r == 1, false, r > 1, false);
    if (r >= 2) step(sn, 1, false, r == 2, false, r > 2, false);
    if (r >= 3) step(sc, 0, false, r == 3, false, r > 3, false);
    if (r >= 4) step(sn, 1, false, true, false, false, false);
    if (r & 1) {
      const Pre t = sc;
      sc = sn;
      sn = t;
    }
  };
  // Blocks have strictly ascending bit-widths, so the work-group's blocks are
  // visited by one pass over the palette: straight-line code, no loop whose
  // registers every bit-width's copy would have to share.
  int bi = b0;
  auto visit = [&](auto b_tag) __attribute__((always_inline)) {
    constexpr int B = decltype(b_tag)::value;
    if (c < C && it.bits[bi] == B) {
      run_block(b_tag, min(it.ce[bi], C));
      ++bi;
    }
  };
  visit(Int<2>{});
  visit(Int<3>{});
  visit(Int<4>{});
  visit(Int<8>{});
  visit(Int<16>{});

  // D layout: lane holds weight rows 16 i + 4 (lane/16) + e of token 16 j + lane%16.
  const int row0 = (rp * 2 + rt) * kTileRows + 4 * (lane >> 4);
  float* ybase = a.splits > 1 ? a.partial + static_cast<int64_t>(ks) * a.m * it.n : it.y;
  const bool vec = a.splits > 1 ? (it.n & 3) == 0 : it.y_vec != 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int tok = m0 + tq * 64 + 16 * j + (lane & 15);
    if (tok >= a.m) continue;
    float* yr = ybase + static_cast<int64_t>(tok) * it.n;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = row0 + 16 * i;
      if (vec && row + 3 < it.n) {
        *reinterpret_cast<f4*>(yr + row) = T[i][j];
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (row + e < it.n) yr[row + e] = T[i][j][e];
      }
    }
  }
}

// y = partial[0] + partial[1] + ... (in split order), `count` elements each,
// four consecutive elements per thread (16-byte accesses when count is a
// multiple of 4 and y is 16-byte aligned; the partials always are).
__global__ __launch_bounds__(256) void sum_splits_kernel(const float* __restrict__ partial,
                                                         float* __restrict__ y, int splits,
                                                         int64_t count) {
  const int64_t i = (static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x) * 4;
  if (i >= count) return;
  if ((count & 3) == 0 && (reinterpret_cast<uintptr_t>(y) & 15) == 0) {
    float4 v = *reinterpret_cast<const float4*>(partial + i);
    for (int s = 1; s < splits; ++s) {
      const float4 w = *reinterpret_cast<const float4*>(partial + s * count + i);
      v.x += w.x;
      v.y += w.y;
      v.z += w.z;
      v.w += w.w;
    }
    *reinterpret_cast<float4*>(y + i) = v;
  } else {
    for (int64_t j = i; j < count && j < i + 4; ++j) {
      float v = partial[j];
      for (int s = 1; s < splits; ++s) v += partial[s * count + j];
      y[j] = v;
    }
  }
}

}  // namespace
}  // namespace polyq

using namespace polyq;

namespace {

size_t permuted_bytes(const polyq_layout& L, int32_t m) {
  return static_cast<size_t>(align_up(static_cast<int64_t>(m) * L.k * 2, 256));
}

// Work-groups of one linear (two packed tiles each) per K split.
int64_t tile_groups(const polyq_layout& L, int32_t m) {
  return static_cast<int64_t>((L.n_tiles + 1) / 2) * ((m + kTokWG - 1) / kTokWG);
}

// K splits of a single-linear launch whose work-groups would leave CUs idle:
// as many as keep the launch within one round of one work-group per CU (256),
// at least four groups per split, at most kMaxSplits.
int plan_splits(const polyq_layout& L, int32_t m, int32_t count) {
  const int64_t wg = tile_groups(L, m);
  if (count != 1 || wg >= 200) return 1;
  int groups = 0;
  for (int i = 0; i < L.nblocks; ++i) groups += (L.block[i].len / kChunk + kChunksPerGroup - 1) / kChunksPerGroup;
  return static_cast<int>(std::max<int64_t>(1, std::min<int64_t>({256 / wg, kMaxSplits, groups / 4})));
}

// Workspace of a batch: one clustered copy x' = x[:, perm] (times the channel
// factors of Eq. 8) per distinct (x, perm, factors) of the items with a
// permutation or factors (region[i] = byte offset of item i's copy, or -1),
// then the split partial sums of a single-linear launch (at *partial_off).
polyq_status plan_gemm_batch(const polyq_gemv_item* items, int32_t count, int32_t m,
                             int64_t* region, size_t* partial_off, int* splits, size_t* total) {
  if (items == nullptr || count < 1 || m < 1) return POLYQ_ERR_ARG;
  if (count > POLYQ_MAX_BATCH) return POLYQ_ERR_CAPACITY;
  size_t off = 0;
  for (int i = 0; i < count; ++i) {
    if (!layout_is_valid(items[i].layout)) return POLYQ_ERR_ARG;
    if (static_cast<int64_t>(m) * items[i].layout->k * 2 > 0x7FFFFFFFll) return POLYQ_ERR_CAPACITY;
    region[i] = -1;
    if (items[i].perm == nullptr && items[i].xscale == nullptr) continue;
    for (int j = 0; j < i; ++j)
      if (region[j] >= 0 && items[j].perm == items[i].perm && items[j].x == items[i].x &&
          items[j].xscale == items[i].xscale && items[j].layout->k == items[i].layout->k) {
        region[i] = region[j];
        break;
      }
    if (region[i] < 0) {
      region[i] = static_cast<int64_t>(off);
      off += permuted_bytes(*items[i].layout, m);
    }
  }
  *splits = plan_splits(*items[0].layout, m, count);
  *partial_off = off;
  if (*splits > 1)
    off += static_cast<size_t>(align_up(static_cast<int64_t>(*splits) * m * items[0].layout->n * 4, 256));
  *total = off;
  return POLYQ_OK;
}

}  // namespace

extern "C" size_t polyq_gemm_batch_workspace_bytes(const polyq_gemm_item* items, int32_t count,
                                                   int32_t m) {
  int64_t region[POLYQ_MAX_BATCH];
  size_t partial_off = 0, total = 0;
  int splits = 1;
  if (plan_gemm_batch(items, count, m, region, &partial_off, &splits, &total) != POLYQ_OK) return 0;
  return total;
}

extern "C" size_t polyq_gemm_workspace_bytes(const polyq_layout* layout, int32_t m, int perm_given) {
  if (!layout_is_valid(layout) || m < 1) return 0;
  const int32_t dummy = 0;
  const polyq_gemm_item item{layout, nullptr, perm_given ? &dummy : nullptr, nullptr, nullptr, nullptr};
  return polyq_gemm_batch_workspace_bytes(&item, 1, m);
}

extern "C" polyq_status polyq_gemm_batch(const polyq_gemm_item* items, int32_t count, int32_t m,
                                         void* workspace, size_t workspace_bytes, void* stream) {
  int64_t region[POLYQ_MAX_BATCH];
  size_t need = 0, partial_off = 0;
  int splits = 1;
  const polyq_status pst = plan_gemm_batch(items, count, m, region, &partial_off, &splits, &need);
  if (pst != POLYQ_OK) return pst;
  if (need > 0 && (workspace == nullptr || workspace_bytes < need)) return POLYQ_ERR_CAPACITY;
  if (need > 0 && reinterpret_cast<uintptr_t>(workspace) % 16 != 0) return POLYQ_ERR_ARG;
  hipStream_t st = static_cast<hipStream_t>(stream);
  GemmBatchArgs a;
  memset(&a, 0, sizeof(a));
  a.count = count;
  a.m = m;
  a.splits = splits;
  a.m_tiles = (m + kTokWG - 1) / kTokWG;
  for (int i = 0; i < count; ++i) {
    const polyq_gemv_item& itm = items[i];
    const polyq_layout& L = *itm.layout;
    if (itm.packed == nullptr || itm.x == nullptr || itm.y == nullptr) return POLYQ_ERR_ARG;
    if (reinterpret_cast<uintptr_t>(itm.packed) % 256 != 0 || reinterpret_cast<uintptr_t>(itm.y) % 4 != 0)
      return POLYQ_ERR_ARG;
    if (L.packed_bytes > 0x7FFFFFFFll) return POLYQ_ERR_CAPACITY;
    if (itm.perm == nullptr && itm.xscale == nullptr && reinterpret_cast<uintptr_t>(itm.x) % 16 != 0)
      return POLYQ_ERR_ARG;  // clustered activations are read as 16-byte vectors
  }
  // Every check above and here comes before the first launch.
  int64_t wg = 0;
  for (int i = 0; i < count; ++i) {
    a.wg_begin[i] = static_cast<int32_t>(wg);
    wg += tile_groups(*items[i].layout, m) * splits;
    if (wg > 0x7FFFFFFF) return POLYQ_ERR_CAPACITY;
  }
  for (int i = count; i <= POLYQ_MAX_BATCH; ++i) a.wg_begin[i] = static_cast<int32_t>(wg);
  // Permuted copies (one per distinct (x, perm, factors), all in one launch),
  // then the products.
  ShuffleJob jobs[POLYQ_MAX_BATCH];
  int njobs = 0;
  for (int i = 0; i < count; ++i) {
    if (region[i] < 0) continue;
    bool first = true;
    for (int j = 0; j < i; ++j) first = first && region[j] != region[i];
    if (first)
      jobs[njobs++] = ShuffleJob{items[i].perm, items[i].xscale, items[i].x,
                                 reinterpret_cast<uint16_t*>(static_cast<uint8_t*>(workspace) + region[i]),
                                 items[i].layout->k, 0};
  }
  launch_shuffle(jobs, njobs, m, true, st);
  for (int i = 0; i < count; ++i) {
    const polyq_gemv_item& itm = items[i];
    const polyq_layout& L = *itm.layout;
    const uint16_t* xp = itm.x;
    if (region[i] >= 0) xp = reinterpret_cast<const uint16_t*>(static_cast<uint8_t*>(workspace) + region[i]);
    GemmItem& g = a.item[i];
    g.packed = static_cast<const uint8_t*>(itm.packed);
    g.x = xp;
    g.y = itm.y;
    g.n = L.n;
    g.k = L.k;
    g.nblocks = L.nblocks;
    g.n_tiles = L.n_tiles;
    g.n_chunks = L.n_chunks;
    g.y_vec = (L.n % 4 == 0 && reinterpret_cast<uintptr_t>(itm.y) % 16 == 0) ? 1 : 0;
    for (int b = 0; b < POLYQ_MAX_BLOCKS; ++b) {
      const bool used = b < L.nblocks;
      g.bits[b] = used ? L.block[b].bits : 16;
      g.cb[b] = used ? L.k_begin[b] / kChunk : L.n_chunks;
      g.ce[b] = used ? (L.k_begin[b] + L.block[b].len) / kChunk : L.n_chunks;
      g.off[b] = used ? L.block_offset[b] : 0;
      g.tb[b] = used ? L.tile_bytes[b] : 0;
      g.rb[b] = used ? L.record_bytes[b] : 0;
    }
  }
  // split s covers groups [G s / S, G (s + 1) / S) of the group sequence
  {
    const polyq_layout& L = *items[0].layout;
    int gstart[POLYQ_MAX_K / POLYQ_GROUP + POLYQ_MAX_BLOCKS];
    int G = 0;
    if (splits > 1)
      for (int b = 0; b < L.nblocks; ++b)
        for (int c = L.k_begin[b] / kChunk; c < (L.k_begin[b] + L.block[b].len) / kChunk; c += kChunksPerGroup)
          gstart[G++] = c;
    for (int sp = 0; sp <= kMaxSplits; ++sp)
      a.split_chunk[sp] = splits == 1 ? (sp == 0 ? 0 : L.n_chunks)
                                      : (sp >= splits ? L.n_chunks : gstart[static_cast<int64_t>(G) * sp / splits]);
    a.partial = splits > 1 ? reinterpret_cast<float*>(static_cast<uint8_t*>(workspace) + partial_off) : nullptr;
  }
  hipLaunchKernelGGL(gemm_kernel, dim3(static_cast<unsigned>(wg)), dim3(kThreads), 0, st, a);
  if (splits > 1) {
    const int64_t n_el = static_cast<int64_t>(m) * items[0].layout->n;
    hipLaunchKernelGGL(sum_splits_kernel, dim3(static_cast<unsigned>((n_el + 1023) / 1024)), dim3(256), 0, st,
                       a.partial, items[0].y, splits, n_el);
  }
  return hipGetLastError() == hipSuccess ? POLYQ_OK : POLYQ_ERR_DEVICE;
}

extern "C" polyq_status polyq_gemm(const polyq_layout* layout, const void* packed,
                                   const int32_t* perm, const uint16_t* x, int32_t m, float* y,
                                   void* workspace, size_t workspace_bytes, void* stream) {
  const polyq_gemm_item item{layout, packed, perm, x, y, nullptr};
  return polyq_gemm_batch(&item, 1, m, workspace, workspace_bytes, stream);
}
