// Prefill GEMM over the mixed-bit clustered weight (Sec. 4.1-4.2), M tokens:
//   y[m][n] = sum_k' w_hat[n][k'] x'[m][k'],  x' = x[:, perm] (Eq. 9)
//
// Prefill is a dense contraction, so it runs on the bf16 matrix cores
// (v_mfma_f32_16x16x32_bf16, fp32 accumulation).  A work-group owns 256 tokens
// x 64*TN weight rows (TN packed tiles) and walks K one 32-channel chunk at a
// time through a two-stage LDS ring:
//   * every thread prefetches, two chunks ahead, 32 or 64 bytes of activations
//     and its share of the packed chunk (one row sub-tile of one lane slice,
//     4*b/4 .. 4*b bytes) plus that row's zero point;
//   * the packed share is dequantized once per work-group into a bf16 tile in
//     LDS that all waves of the work-group multiply (weights are the MFMA A
//     operand, activations the B operand);
//   * wave (tq, rt) multiplies rows 64*rt.. by tokens 64*tq..: 16 MFMAs per
//     chunk; one barrier per chunk.
// Group-fold numerics: the dequantized operand is (q - z), an integer of
// magnitude <= 255 that bf16 holds exactly when z is an integer; each
// 128-channel group accumulates into its own fp32 tile, which is then scaled
// by the row's fp16 scale s (fp32 FMA) into the output accumulator.  A 16-bit
// channel, or a group whose zero point is not an integer, enters as the pair
// hi + lo of bf16 values (two MFMAs); for 16-bit weights the pair is exact.
//
// Dequantization uses the fp16 exponent field: (1024 + q) is the fp16 with
// exponent 10 and mantissa q, so one AND-OR forms two codes of a pair as fp16.
// For an integer z in [0, 255] one fp32 subtract of (1024 + z) gives q - z
// exactly and the bf16 value is the fp32 value's upper half; for any other
// fp16 z, (1024 + q) - 1024 = q exactly and q - z rounds once in fp32 before
// the split into hi + lo.
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

constexpr int kTokWG = 256;   // tokens per work-group: 4 waves of 64 along M
constexpr int kLdsRow = 40;   // bf16 per LDS row: 32 channels + 8 pad against bank conflicts
constexpr uint32_t kMagic2 = 0x64006400u;  // two fp16 1024.0

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

// Position of a pipeline stage in the chunk sequence: chunk c, chunk cl of
// block bi (bit-width bits, ending at chunk ce).  Advanced one chunk at a
// time; the block table is read (from the kernel arguments) only when a block
// ends.
struct ChunkCursor {
  int c, bi, bits, cl, ce;
  __device__ __forceinline__ bool first() const { return (cl & 3) == 0; }
  __device__ __forceinline__ bool last() const { return (cl & 3) == 3 || c + 1 == ce; }
};

typedef uint32_t u4v __attribute__((ext_vector_type(4)));

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), static_cast<short>(0),
                                           static_cast<int>(bytes), 0x00020000);
}

// Prefetched data of one chunk for one thread.
template <int TN>
struct Pre {
  u4v av[4 / TN];  // activation pieces (16 bytes each)
  u4v w;           // 16 bytes from this thread's packed sub-tile (the first 4*b/4 .. 16 used)
  uint32_t z, s;   // its row's fp16 zero point and scale (bits), b <= 8
};

// Two codes of a pair as fp16 (1024 + q): the fields sit at bit offsets o and
// 16 + o of w.
__device__ __forceinline__ uint32_t pair_magic(uint32_t w, int o, uint32_t mask2) {
  return ((w >> o) & mask2) | kMagic2;
}

// The 4 code pairs (channels 2j, 2j+1) of row sub-tile r of a lane slice, in
// the slice arrangement of codec.h, as fp16 pairs (1024 + q).
template <int B>
__device__ __forceinline__ void sub_tile_pairs(const u4v w, int r, uint32_t* hp) {
  if constexpr (B == 2) {  // word r/2 (loaded as w.x) holds sub-tiles r & ~1 and r | 1
    const int sh = 8 * (r & 1);
#pragma unroll
    for (int j = 0; j < 4; ++j) hp[j] = pair_magic(w.x, sh + 2 * j, 0x00030003u);
  } else if constexpr (B == 4) {  // word r
#pragma unroll
    for (int j = 0; j < 4; ++j) hp[j] = pair_magic(w.x, 4 * j, 0x000F000Fu);
  } else if constexpr (B == 8) {  // words 2r, 2r+1
#pragma unroll
    for (int j = 0; j < 4; ++j) hp[j] = pair_magic((j >> 1) ? w.y : w.x, 8 * (j & 1), 0x00FF00FFu);
  } else {  // B == 3: all three words; pair P = 4r + j sits in word P/5 at f3(P%5)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int P = 4 * r + j;
      if (P < 15) {
        const int d = P / 5, p = P - 5 * d;
        const uint32_t wd = d == 0 ? w.x : (d == 1 ? w.y : w.z);
        hp[j] = pair_magic(wd, 3 * p + (p >= 3 ? 1 : 0), 0x00070007u);
      } else {  // codes 30, 31: bit d of each in bits 9 and 25 of word d
        const uint32_t t = ((w.x >> 9) & 0x00010001u) | ((w.y >> 8) & 0x00020002u) |
                           ((w.z >> 7) & 0x00040004u);
        hp[j] = t | kMagic2;
      }
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

// Eight values of one row, each exact in bf16, into the hi tile.
__device__ __forceinline__ void store_exact(const float* v, uint16_t* hi_dst) {
  uint4 o;
  o.x = hi_half_pair(v[0], v[1]);
  o.y = hi_half_pair(v[2], v[3]);
  o.z = hi_half_pair(v[4], v[5]);
  o.w = hi_half_pair(v[6], v[7]);
  *reinterpret_cast<uint4*>(hi_dst) = o;
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

template <int TN>
__global__ __launch_bounds__(256 * TN) void gemm_kernel(const GemmBatchArgs a) {
  constexpr int kThreads = 256 * TN, kRows = 64 * TN;
  constexpr int kAPieces = 4 / TN;  // 16-byte activation pieces per thread per chunk
  __shared__ __attribute__((aligned(16))) uint16_t lds_a[2][kTokWG * kLdsRow];
  __shared__ __attribute__((aligned(16))) uint16_t lds_b[2][2][kRows * kLdsRow];  // [stage][hi, lo]
  __shared__ __attribute__((aligned(16))) float lds_s[2][kRows];                 // row scales of the stage's group
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
  // this work-group's chunks [c0, C)
  const int c0 = a.splits > 1 ? a.split_chunk[ks] : 0;
  const int C = a.splits > 1 ? a.split_chunk[ks + 1] : it.n_chunks;
  int b0 = 0;
#pragma unroll
  for (int j = 0; j < POLYQ_MAX_BLOCKS - 1; ++j) b0 += (j + 1 < it.nblocks && c0 >= it.ce[j]) ? 1 : 0;
  auto cursor_at0 = [&]() { return ChunkCursor{c0, b0, it.bits[b0], c0 - it.cb[b0], it.ce[b0]}; };
  auto advance = [&](ChunkCursor& u) {
    ++u.c;
    ++u.cl;
    if (u.c == u.ce && u.c < C) {
      ++u.bi;
      u.bits = it.bits[u.bi];
      u.ce = it.ce[u.bi];
      u.cl = 0;
    }
  };

  // Dequantization role: packed tile dt, row sub-tile dr (wave-uniform), lane
  // slice lane; row drow of the tile.
  const int dp = wv >> 2, dr = wv & 3;
  const int dt = rp * TN + dp;
  const bool dtile_ok = dt < it.n_tiles;
  const int drow = 16 * dr + (lane & 15);
  const int bofs = (dp * 64 + drow) * kLdsRow + 8 * (lane >> 4);
  constexpr int kHalfB = kRows * kLdsRow;

  // Activations: buffer over rows m0 .. m0 + 255 of x' (reads past row m - 1
  // return zero); piece j of this thread is token piece/4, 16-byte segment piece%4.
  const __amdgpu_buffer_rsrc_t xrs =
      make_rsrc(it.x + static_cast<int64_t>(m0) * it.k, static_cast<uint32_t>(min(a.m - m0, kTokWG)) * it.k * 2u);
  uint32_t avoff[kAPieces];
#pragma unroll
  for (int j = 0; j < kAPieces; ++j) {
    const int piece = tid + j * kThreads;
    avoff[j] = (static_cast<uint32_t>(piece >> 2) * it.k + (piece & 3) * 8) * 2u;
  }

  // Load cursor: the next chunk to fetch, its block and a buffer over this
  // thread's packed tile of that block (no records for a tile past the end,
  // so its reads return zero).
  int lc = c0, lb = 0, lcl = 0, lbits = 0, lce = 0, lrb = 0;
  uint32_t lvoff = 0;
  __amdgpu_buffer_rsrc_t wrs;
  auto set_block = [&](int b) {
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
  auto load = [&](Pre<TN>& pr) {
#pragma unroll
    for (int j = 0; j < kAPieces; ++j)
      pr.av[j] = __builtin_bit_cast(u4v, __builtin_amdgcn_raw_buffer_load_b128(xrs, avoff[j], lc * 64, 0));
    const int rec = (lcl >> 2) * lrb;
    const int soff = rec + (lbits <= 8 ? kMetaBytes : 0) + (lcl & 3) * 256 * lbits;
    pr.w = __builtin_bit_cast(u4v, __builtin_amdgcn_raw_buffer_load_b128(wrs, lvoff, soff, 0));
    pr.z = __builtin_amdgcn_raw_buffer_load_b16(wrs, zvoff, rec, 0);
    pr.s = __builtin_amdgcn_raw_buffer_load_b16(wrs, svoff, rec, 0);
    ++lc;
    ++lcl;
    if (lc == lce && lc < C) set_block(lb + 1);
  };

  auto store = [&](const ChunkCursor& ci, const Pre<TN>& pr, int st) {
#pragma unroll
    for (int j = 0; j < kAPieces; ++j) {
      const int piece = tid + j * kThreads;
      *reinterpret_cast<u4v*>(&lds_a[st][(piece >> 2) * kLdsRow + (piece & 3) * 8]) = pr.av[j];
    }
    uint16_t* hi = &lds_b[st][0][bofs];
    uint16_t* lo = hi + kHalfB;
    float v[8];
    if (ci.bits == 16) {
      const uint32_t ww[4] = {pr.w.x, pr.w.y, pr.w.z, pr.w.w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const h2 h = __builtin_bit_cast(h2, ww[i]);
        v[2 * i] = static_cast<float>(h.x);
        v[2 * i + 1] = static_cast<float>(h.y);
      }
      lds_s[st][dp * 64 + drow] = 1.f;  // the four threads of a row store the same value
      store_pair(v, hi, lo);
      return;
    }
    const float zf = static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(pr.z)));
    lds_s[st][dp * 64 + drow] = static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(pr.s)));
    uint32_t hp[4];
    switch (ci.bits) {
      case 2: sub_tile_pairs<2>(pr.w, dr, hp); break;
      case 3: sub_tile_pairs<3>(pr.w, dr, hp); break;
      case 4: sub_tile_pairs<4>(pr.w, dr, hp); break;
      default: sub_tile_pairs<8>(pr.w, dr, hp); break;
    }
    if (__all(zf == truncf(zf) && zf >= 0.f && zf <= 255.f)) {  // wave-uniform
      // (1024 + q) - (1024 + z) = q - z: both sums are exact for such z, and
      // so is the difference, in fp32 and in bf16 (|q - z| <= 255)
      const float zoff = 1024.f + zf;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const h2 h = __builtin_bit_cast(h2, hp[j]);
        v[2 * j] = static_cast<float>(h.x) - zoff;
        v[2 * j + 1] = static_cast<float>(h.y) - zoff;
      }
      store_exact(v, hi);
      *reinterpret_cast<uint4*>(lo) = uint4{0u, 0u, 0u, 0u};
    } else {
      // any other fp16 z: ((1024 + q) - 1024) is q exactly, and q - z rounds
      // once in fp32 (1024 + z itself would round for small non-integer z)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const h2 h = __builtin_bit_cast(h2, hp[j]);
        v[2 * j] = (static_cast<float>(h.x) - 1024.f) - zf;
        v[2 * j + 1] = (static_cast<float>(h.y) - 1024.f) - zf;
      }
      store_pair(v, hi, lo);
      lds_tag[st] = ci.c + 1;  // any thread; every writer stores the same value
    }
  };

  f4 total[4][4], part[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) total[i][j] = f4{0.f, 0.f, 0.f, 0.f};

  const int aofs = (tq * 64 + (lane & 15)) * kLdsRow + 8 * (lane >> 4);
  const int bofs_m = (rt * 64 + (lane & 15)) * kLdsRow + 8 * (lane >> 4);
  // Chunk mc.c: multiply stage c&1, dequantize chunk c+1 (cursor sc) from
  // `slot` into the other stage, fetch chunk c+3 into `slot`, fold a finished
  // group.
  ChunkCursor mc = cursor_at0(), sc = cursor_at0();
  auto step = [&](Pre<TN>& slot, auto st_tag) {  // st = (c - c0) & 1, known at each call
    constexpr int st = decltype(st_tag)::value;
    const int c = mc.c;
    const bool two = mc.bits == 16 || lds_tag[st] == c + 1;
    bf16x8 af[4], bfr[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      af[i] = *reinterpret_cast<const bf16x8*>(&lds_b[st][0][bofs_m + i * 16 * kLdsRow]);
      bfr[i] = *reinterpret_cast<const bf16x8*>(&lds_a[st][aofs + i * 16 * kLdsRow]);
    }
    if (mc.first()) {  // first chunk of a group: fresh partial sums
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          part[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[j], f4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) part[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[j], part[i][j], 0, 0, 0);
    }
    if (two) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
        af[i] = *reinterpret_cast<const bf16x8*>(&lds_b[st][1][bofs_m + i * 16 * kLdsRow]);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) part[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[j], part[i][j], 0, 0, 0);
    }
    if (c + 1 < C) {
      advance(sc);
      store(sc, slot, st ^ 1);
    }
    if (c + 3 < C) load(slot);
    if (mc.last()) {  // group fold: total += s * part, s of rows 16 i + 4 (lane/16) + e
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const f4 sv = *reinterpret_cast<const f4*>(&lds_s[st][rt * 64 + 16 * i + 4 * (lane >> 4)]);
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int e = 0; e < 4; ++e) total[i][j][e] = fmaf(sv[e], part[i][j][e], total[i][j][e]);
      }
    }
    advance(mc);
    __syncthreads();
  };

  Pre<TN> s0, s1;
  if (tid < 2) lds_tag[tid] = 0;
  set_block(b0);
  lcl = c0 - it.cb[b0];
  load(s0);
  if (C - c0 > 1) load(s1);
  __syncthreads();
  store(sc, s0, 0);
  if (C - c0 > 2) load(s0);
  __syncthreads();
  int c = c0;
  for (; c + 1 < C; c += 2) {
    step(s1, std::integral_constant<int, 0>{});
    step(s0, std::integral_constant<int, 1>{});
  }
  if (c < C) step(s1, std::integral_constant<int, 0>{});

  // D layout: lane holds weight rows 16 i + 4 (lane/16) + e of token 16 j + lane%16.
  const int row0 = (rp * TN + rt) * kTileRows + 4 * (lane >> 4);
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int tok = m0 + tq * 64 + 16 * j + (lane & 15);
    if (tok >= a.m) continue;
    float* yr = a.splits > 1 ? a.partial + (static_cast<int64_t>(ks) * a.m + tok) * it.n
                             : it.y + static_cast<int64_t>(tok) * it.n;
    const bool vec = a.splits > 1 ? (it.n & 3) == 0 : it.y_vec != 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = row0 + 16 * i;
      if (vec && row + 3 < it.n) {
        *reinterpret_cast<f4*>(yr + row) = total[i][j];
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (row + e < it.n) yr[row + e] = total[i][j][e];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Wide-wave variant: a work-group of 4 waves owns 256 tokens x 128 rows (two
// packed tiles) and each wave 128 tokens x 64 rows, so a chunk costs a wave 32
// MFMAs against the same per-chunk bookkeeping.  To fit 128 accumulators per
// lane the group fold is replaced by a running rescale: the accumulator T of
// a row is kept in units of the current group's scale s_g (T = sum over
// earlier groups of s_g' P_g' / s_g); at a group's first chunk T is multiplied
// by s_{g-1} / s_g, the group's integer products (q - z) x are added by the
// MFMAs, and the output is T * s_last.  Each rescale rounds once (relative
// error below 2^-23 per group); a scale of 0 is treated as 1 with the row's
// dequantized values set to 0, so its products vanish exactly.  The activation
// tile is stored without padding, its 16-byte segments permuted per token
// (seg ^ swz(token)) so that both the stores and the fragment reads are free
// of bank conflicts.

__device__ __forceinline__ int swz(int t) { return ((t >> 1) ^ (t >> 3)) & 3; }

// Prefetched data of one chunk for one thread of the wide kernel.
struct PreW {
  u4v av[4];    // activation pieces
  u4v w0, w1;   // packed words of the thread's two row sub-tiles (w1: 16-bit only)
  uint32_t z2;  // fp16 zero points of the two rows (low, high half)
  uint32_t s0, s1;  // fp16 scales of the two rows
};

// The 4 code pairs of row sub-tile r from the 16 bytes `w` that hold it (the
// word(s) loaded at sub_offset(b, r) of the slice, or the whole 3-bit slice).
template <int B>
__device__ __forceinline__ void pairs_at(const u4v w, int r, int second, uint32_t* hp) {
  if constexpr (B == 2) {  // sub-tiles 2k and 2k+1 share word k (w.x)
    const int sh = 8 * second;
#pragma unroll
    for (int j = 0; j < 4; ++j) hp[j] = pair_magic(w.x, sh + 2 * j, 0x00030003u);
  } else if constexpr (B == 4) {  // word r (w.x for the first, w.y for the second)
    const uint32_t wd = second ? w.y : w.x;
#pragma unroll
    for (int j = 0; j < 4; ++j) hp[j] = pair_magic(wd, 4 * j, 0x000F000Fu);
  } else if constexpr (B == 8) {  // words 2r, 2r+1
#pragma unroll
    for (int j = 0; j < 4; ++j)
      hp[j] = pair_magic(second ? ((j >> 1) ? w.w : w.z) : ((j >> 1) ? w.y : w.x), 8 * (j & 1), 0x00FF00FFu);
  } else {
    sub_tile_pairs<3>(w, r, hp);
  }
}

__global__ __launch_bounds__(256) void gemm_wide_kernel(const GemmBatchArgs a) {
  constexpr int kRows = 128;
  __shared__ __attribute__((aligned(16))) uint16_t lds_a[2][kTokWG * kChunk];     // swizzled, no padding
  __shared__ __attribute__((aligned(16))) uint16_t lds_b[2][2][kRows * kLdsRow];  // [stage][hi, lo]
  __shared__ __attribute__((aligned(16))) float lds_r[2][kRows];  // rescale s_{g-1}/s_g at a group's first chunk
  __shared__ int lds_tag[2];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int th = wv & 1, rt = wv >> 1;  // MFMA role: token half, packed tile
  int idx = 0;
#pragma unroll
  for (int i = 1; i < POLYQ_MAX_BATCH; ++i) idx += (i < a.count && static_cast<int>(blockIdx.x) >= a.wg_begin[i]) ? 1 : 0;
  const GemmItem& it = a.item[idx];
  const int local = static_cast<int>(blockIdx.x) - a.wg_begin[idx];
  const int mt = local % a.m_tiles, rest = local / a.m_tiles;
  const int ks = rest % a.splits, rp = rest / a.splits;
  const int m0 = mt * kTokWG;
  const int c0 = a.splits > 1 ? a.split_chunk[ks] : 0;
  const int C = a.splits > 1 ? a.split_chunk[ks + 1] : it.n_chunks;
  int b0 = 0;
#pragma unroll
  for (int j = 0; j < POLYQ_MAX_BLOCKS - 1; ++j) b0 += (j + 1 < it.nblocks && c0 >= it.ce[j]) ? 1 : 0;
  auto cursor_at0 = [&]() { return ChunkCursor{c0, b0, it.bits[b0], c0 - it.cb[b0], it.ce[b0]}; };
  auto advance = [&](ChunkCursor& u) {
    ++u.c;
    ++u.cl;
    if (u.c == u.ce && u.c < C) {
      ++u.bi;
      u.bits = it.bits[u.bi];
      u.ce = it.ce[u.bi];
      u.cl = 0;
    }
  };

  // Dequantization role: packed tile dp, row sub-tiles dr and dr + 1, lane
  // slice `lane`; rows R0 = 16 dr + lane % 16 and R0 + 16.
  const int dp = wv >> 1, dr = 2 * (wv & 1);
  const int dt = rp * 2 + dp;
  const bool dtile_ok = dt < it.n_tiles;
  const int R0 = 16 * dr + (lane & 15);
  const int bofs = (dp * 64 + R0) * kLdsRow + 8 * (lane >> 4);
  constexpr int kHalfB = kRows * kLdsRow;

  const __amdgpu_buffer_rsrc_t xrs =
      make_rsrc(it.x + static_cast<int64_t>(m0) * it.k, static_cast<uint32_t>(min(a.m - m0, kTokWG)) * it.k * 2u);
  uint32_t avoff[4];
  int aofs_st[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int piece = tid + j * 256, t = piece >> 2, sg = piece & 3;
    avoff[j] = (static_cast<uint32_t>(t) * it.k + sg * 8) * 2u;
    aofs_st[j] = t * kChunk + 8 * (sg ^ swz(t));
  }

  int lc = c0, lb = 0, lcl = 0, lbits = 0, lce = 0, lrb = 0;
  uint32_t lvoff = 0;
  __amdgpu_buffer_rsrc_t wrs;
  auto set_block = [&](int b) {
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
  const uint32_t zvoff = 2 * meta_z_half(R0);  // both rows' z (halves 4 (lane%16) + dr, + 1)
  const uint32_t svoff0 = 2 * meta_s_half(R0), svoff1 = 2 * meta_s_half(R0 + 16);
  auto load = [&](PreW& pr) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
      pr.av[j] = __builtin_bit_cast(u4v, __builtin_amdgcn_raw_buffer_load_b128(xrs, avoff[j], lc * 64, 0));
    const int rec = (lcl >> 2) * lrb;
    const int soff = rec + (lbits <= 8 ? kMetaBytes : 0) + (lcl & 3) * 256 * lbits;
    pr.w0 = __builtin_bit_cast(u4v, __builtin_amdgcn_raw_buffer_load_b128(wrs, lvoff, soff, 0));
    pr.w1 = __builtin_bit_cast(u4v, __builtin_amdgcn_raw_buffer_load_b128(wrs, lvoff + 16, soff, 0));
    if ((lcl & 3) == 0) {  // z and s are read at a group's first chunk only
      pr.z2 = __builtin_amdgcn_raw_buffer_load_b32(wrs, zvoff, rec, 0);
      pr.s0 = __builtin_amdgcn_raw_buffer_load_b16(wrs, svoff0, rec, 0);
      pr.s1 = __builtin_amdgcn_raw_buffer_load_b16(wrs, svoff1, rec, 0);
    }
    ++lc;
    ++lcl;
    if (lc == lce && lc < C) set_block(lb + 1);
  };

  // Group scale of the two rows (0 read as 1), kept from the previous group,
  // and the values a group's first chunk derives from its metadata for the
  // group's other chunks: 1024 + z of both rows, rows whose scale is 0, and
  // whether every zero point of the wave is an integer in [0, 255].
  float sig_prev0 = 1.f, sig_prev1 = 1.f;
  float gz0 = 0.f, gz1 = 0.f;
  bool gdead0 = false, gdead1 = false, gdead = false, gexact = true;
  auto store = [&](const ChunkCursor& ci, const PreW& pr, int st) {
#pragma unroll
    for (int j = 0; j < 4; ++j) *reinterpret_cast<u4v*>(&lds_a[st][aofs_st[j]]) = pr.av[j];
    if ((ci.cl & 3) == 0) {  // first chunk of a group: its rows' scales and zero points
      float sg0 = 1.f, sg1 = 1.f;
      if (ci.bits <= 8) {
        const float s0 = static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(pr.s0)));
        const float s1 = static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(pr.s1)));
        gdead0 = s0 == 0.f;
        gdead1 = s1 == 0.f;
        sg0 = gdead0 ? 1.f : s0;
        sg1 = gdead1 ? 1.f : s1;
        const h2 zz = __builtin_bit_cast(h2, pr.z2);
        const float z0 = static_cast<float>(zz.x), z1 = static_cast<float>(zz.y);
        gz0 = z0;
        gz1 = z1;
        const bool ok0 = z0 == truncf(z0) && z0 >= 0.f && z0 <= 255.f;
        const bool ok1 = z1 == truncf(z1) && z1 >= 0.f && z1 <= 255.f;
        gexact = __all(ok0 && ok1);  // wave-uniform
        gdead = __any(gdead0 || gdead1);
      }
      lds_r[st][dp * 64 + R0] = sig_prev0 / sg0;  // rescale factors (the four threads of a row store the same value)
      lds_r[st][dp * 64 + R0 + 16] = sig_prev1 / sg1;
      sig_prev0 = sg0;
      sig_prev1 = sg1;
    }
    uint16_t* hi = &lds_b[st][0][bofs];
    uint16_t* lo = hi + kHalfB;
    constexpr int kRowStep = 16 * kLdsRow;  // row R0 + 16
    float v0[8], v1[8];
    if (ci.bits == 16) {
      const uint32_t ww[8] = {pr.w0.x, pr.w0.y, pr.w0.z, pr.w0.w, pr.w1.x, pr.w1.y, pr.w1.z, pr.w1.w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const h2 h = __builtin_bit_cast(h2, ww[i]), g = __builtin_bit_cast(h2, ww[4 + i]);
        v0[2 * i] = static_cast<float>(h.x);
        v0[2 * i + 1] = static_cast<float>(h.y);
        v1[2 * i] = static_cast<float>(g.x);
        v1[2 * i + 1] = static_cast<float>(g.y);
      }
      store_pair(v0, hi, lo);
      store_pair(v1, hi + kRowStep, lo + kRowStep);
      return;
    }
    uint32_t hp0[4], hp1[4];
    switch (ci.bits) {
      case 2: pairs_at<2>(pr.w0, dr, 0, hp0); pairs_at<2>(pr.w0, dr + 1, 1, hp1); break;
      case 3: pairs_at<3>(pr.w0, dr, 0, hp0); pairs_at<3>(pr.w0, dr + 1, 1, hp1); break;
      case 4: pairs_at<4>(pr.w0, dr, 0, hp0); pairs_at<4>(pr.w0, dr + 1, 1, hp1); break;
      default: pairs_at<8>(pr.w0, dr, 0, hp0); pairs_at<8>(pr.w0, dr + 1, 1, hp1); break;
    }
    if (gexact) {
      // (1024 + q) - (1024 + z) = q - z, all exact for an integer z in [0, 255]
      // (in bf16 too)
      const float zo0 = 1024.f + gz0, zo1 = 1024.f + gz1;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const h2 h = __builtin_bit_cast(h2, hp0[j]), g = __builtin_bit_cast(h2, hp1[j]);
        v0[2 * j] = static_cast<float>(h.x) - zo0;
        v0[2 * j + 1] = static_cast<float>(h.y) - zo0;
        v1[2 * j] = static_cast<float>(g.x) - zo1;
        v1[2 * j + 1] = static_cast<float>(g.y) - zo1;
      }
    } else {
      // any other fp16 z: (1024 + q) - 1024 = q exactly, then q - z rounds once
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const h2 h = __builtin_bit_cast(h2, hp0[j]), g = __builtin_bit_cast(h2, hp1[j]);
        v0[2 * j] = (static_cast<float>(h.x) - 1024.f) - gz0;
        v0[2 * j + 1] = (static_cast<float>(h.y) - 1024.f) - gz0;
        v1[2 * j] = (static_cast<float>(g.x) - 1024.f) - gz1;
        v1[2 * j + 1] = (static_cast<float>(g.y) - 1024.f) - gz1;
      }
    }
    if (gdead) {  // rows whose scale is 0 contribute nothing
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        v0[e] = gdead0 ? 0.f : v0[e];
        v1[e] = gdead1 ? 0.f : v1[e];
      }
    }
    if (gexact) {
      // lo is left as it is: zero, unless a chunk stored as pairs used this
      // stage last, and then the owner of each slot clears it before the
      // stage is stored again (clear_lo), because another wave may store its
      // rows of this chunk as pairs and the second MFMA pass reads all rows
      store_exact(v0, hi);
      store_exact(v1, hi + kRowStep);
    } else {
      store_pair(v0, hi, lo);
      store_pair(v1, hi + kRowStep, lo + kRowStep);
      lds_tag[st] = ci.c + 1;
    }
  };

  f4 T[4][8];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) T[i][j] = f4{0.f, 0.f, 0.f, 0.f};

  const int bofs_m = (rt * 64 + (lane & 15)) * kLdsRow + 8 * (lane >> 4);
  auto bfrag = [&](int st, int j) {
    const int t = th * 128 + 16 * j + (lane & 15);
    return *reinterpret_cast<const bf16x8*>(&lds_a[st][t * kChunk + 8 * ((lane >> 4) ^ swz(t))]);
  };
  ChunkCursor mc = cursor_at0(), sc = cursor_at0();
  // The lo tile of a stage is zero except where a chunk stored as pairs wrote
  // it; each thread clears its own two lo slots of a stage whose chunk used
  // the second pass, before it stores into that stage again.
  bool lo_dirty[2] = {false, false};
  auto clear_lo = [&](int st) {
    uint16_t* lo = &lds_b[st][1][bofs];
    *reinterpret_cast<uint4*>(lo) = uint4{0u, 0u, 0u, 0u};
    *reinterpret_cast<uint4*>(lo + 16 * kLdsRow) = uint4{0u, 0u, 0u, 0u};
  };
  // st: the LDS stage of chunk c (chunks alternate, starting with stage 0 at
  // c0), a compile-time constant in the loop below, which runs two chunks per
  // iteration.
  auto step = [&](PreW& slot, auto st_tag) {
    constexpr int st = decltype(st_tag)::value;
    const int c = mc.c;
    const bool two = mc.bits == 16 || lds_tag[st] == c + 1;
    if ((mc.cl & 3) == 0 && c != c0) {  // a new group: T to the new scale's units
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const f4 r = *reinterpret_cast<const f4*>(&lds_r[st][rt * 64 + 16 * i + 4 * (lane >> 4)]);
#pragma unroll
        for (int j = 0; j < 8; ++j)
#pragma unroll
          for (int e = 0; e < 4; ++e) T[i][j][e] *= r[e];
      }
    }
    bf16x8 af[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) af[i] = *reinterpret_cast<const bf16x8*>(&lds_b[st][0][bofs_m + i * 16 * kLdsRow]);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const bf16x8 b = bfrag(st, j);
#pragma unroll
      for (int i = 0; i < 4; ++i) T[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], b, T[i][j], 0, 0, 0);
    }
    if (two) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
        af[i] = *reinterpret_cast<const bf16x8*>(&lds_b[st][1][bofs_m + i * 16 * kLdsRow]);
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const bf16x8 b = bfrag(st, j);
#pragma unroll
        for (int i = 0; i < 4; ++i) T[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], b, T[i][j], 0, 0, 0);
      }
    }
    lo_dirty[st] = two;  // this chunk's pairs sit in stage st until cleared
    if (c + 1 < C) {
      advance(sc);
      if (lo_dirty[st ^ 1]) {  // read by the previous step, before this step's barrier
        clear_lo(st ^ 1);
        lo_dirty[st ^ 1] = false;
      }
      store(sc, slot, st ^ 1);
    }
    if (c + 2 < C) load(slot);
    advance(mc);
    __syncthreads();
  };

  PreW pre;
  if (tid < 2) lds_tag[tid] = 0;
  clear_lo(0);
  clear_lo(1);
  set_block(b0);
  lcl = c0 - it.cb[b0];
  load(pre);
  __syncthreads();
  store(sc, pre, 0);
  if (C - c0 > 1) load(pre);
  __syncthreads();
  {
    int c = c0;
    for (; c + 1 < C; c += 2) {
      step(pre, std::integral_constant<int, 0>{});
      step(pre, std::integral_constant<int, 1>{});
    }
    if (c < C) step(pre, std::integral_constant<int, 0>{});
  }

  // Output: T in units of the last group's scale; that scale goes through LDS.
  lds_r[0][dp * 64 + R0] = sig_prev0;
  lds_r[0][dp * 64 + R0 + 16] = sig_prev1;
  __syncthreads();
  const int row0 = (rp * 2 + rt) * kTileRows + 4 * (lane >> 4);
  float* ybase = a.splits > 1 ? a.partial + static_cast<int64_t>(ks) * a.m * it.n : it.y;
  const bool vec = a.splits > 1 ? (it.n & 3) == 0 : it.y_vec != 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const f4 sl = *reinterpret_cast<const f4*>(&lds_r[0][rt * 64 + 16 * i + 4 * (lane >> 4)]);
    const int row = row0 + 16 * i;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int tok = m0 + th * 128 + 16 * j + (lane & 15);
      if (tok >= a.m) continue;
      float* yr = ybase + static_cast<int64_t>(tok) * it.n;
      const f4 v = T[i][j] * sl;
      if (vec && row + 3 < it.n) {
        *reinterpret_cast<f4*>(yr + row) = v;
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (row + e < it.n) yr[row + e] = v[e];
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

// Work-groups of one linear with TN packed tiles per work-group.
int64_t tile_groups(const polyq_layout& L, int32_t m, int tn) {
  return static_cast<int64_t>((L.n_tiles + tn - 1) / tn) * ((m + kTokWG - 1) / kTokWG);
}

// K splits of a single-linear launch whose one-tile work-groups would leave
// CUs idle: enough wide-wave work-groups for two per CU (about 480), at least
// four groups per split, at most kMaxSplits.
int plan_splits(const polyq_layout& L, int32_t m, int32_t count) {
  if (count != 1 || tile_groups(L, m, 1) >= 240) return 1;
  const int64_t wg = tile_groups(L, m, 2);  // split launches run the wide-wave kernel
  int groups = 0;
  for (int i = 0; i < L.nblocks; ++i) groups += (L.block[i].len / kChunk + kChunksPerGroup - 1) / kChunksPerGroup;
  const int64_t want = (480 + wg - 1) / wg;
  return static_cast<int>(std::max<int64_t>(1, std::min<int64_t>({want, kMaxSplits, groups / 4})));
}

// Workspace of a batch: one permuted copy per distinct (x, perm) pair with
// perm != NULL (region[i] = byte offset of item i's copy, or -1), then the
// split partial sums of a single-linear launch (at *partial_off).
polyq_status plan_gemm_batch(const polyq_gemv_item* items, int32_t count, int32_t m,
                             int64_t* region, size_t* partial_off, int* splits, size_t* total) {
  if (items == nullptr || count < 1 || m < 1) return POLYQ_ERR_ARG;
  if (count > POLYQ_MAX_BATCH) return POLYQ_ERR_CAPACITY;
  size_t off = 0;
  for (int i = 0; i < count; ++i) {
    if (!layout_is_valid(items[i].layout)) return POLYQ_ERR_ARG;
    if (static_cast<int64_t>(m) * items[i].layout->k * 2 > 0x7FFFFFFFll) return POLYQ_ERR_CAPACITY;
    region[i] = -1;
    if (items[i].perm == nullptr) continue;
    for (int j = 0; j < i; ++j)
      if (items[j].perm == items[i].perm && items[j].x == items[i].x &&
          items[j].layout->k == items[i].layout->k) {
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
  const polyq_gemm_item item{layout, nullptr, perm_given ? &dummy : nullptr, nullptr, nullptr};
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
  int64_t tiles1 = 0;
  for (int i = 0; i < count; ++i) {
    const polyq_gemv_item& itm = items[i];
    const polyq_layout& L = *itm.layout;
    if (itm.packed == nullptr || itm.x == nullptr || itm.y == nullptr) return POLYQ_ERR_ARG;
    if (reinterpret_cast<uintptr_t>(itm.packed) % 256 != 0 || reinterpret_cast<uintptr_t>(itm.y) % 4 != 0)
      return POLYQ_ERR_ARG;
    if (L.packed_bytes > 0x7FFFFFFFll) return POLYQ_ERR_CAPACITY;
    if (itm.perm == nullptr && reinterpret_cast<uintptr_t>(itm.x) % 16 != 0)
      return POLYQ_ERR_ARG;  // clustered activations are read as 16-byte vectors
    tiles1 += L.n_tiles;
  }
  // Every check above and here comes before the first launch.  Work-group
  // shape by launch size: 4-wave work-groups of 256 tokens x 128
  // rows with 128 x 64 wave tiles (gemm_wide_kernel) when there are enough of
  // them for two per CU, or K is split; else 8-wave work-groups of the same tile
  // (gemm_kernel<2>) when those fill most CUs; else one packed tile per
  // 4-wave work-group (gemm_kernel<1>, two co-resident per CU).
  const int64_t wg2 = (tiles1 + count) / 2 * a.m_tiles;
  const int kind = splits > 1 || wg2 >= 400 ? 3 : wg2 >= 200 ? 2 : 1;
  const bool wide = kind >= 2;
  const int tn = wide ? 2 : 1;
  int64_t wg = 0;
  for (int i = 0; i < count; ++i) {
    a.wg_begin[i] = static_cast<int32_t>(wg);
    wg += static_cast<int64_t>((items[i].layout->n_tiles + tn - 1) / tn) * a.m_tiles * splits;
    if (wg > 0x7FFFFFFF) return POLYQ_ERR_CAPACITY;
  }
  for (int i = count; i <= POLYQ_MAX_BATCH; ++i) a.wg_begin[i] = static_cast<int32_t>(wg);
  // Permuted copies (one per distinct (x, perm)), then the products.
  for (int i = 0; i < count; ++i) {
    const polyq_gemv_item& itm = items[i];
    const polyq_layout& L = *itm.layout;
    const uint16_t* xp = itm.x;
    if (itm.perm != nullptr) {
      uint16_t* out = reinterpret_cast<uint16_t*>(static_cast<uint8_t*>(workspace) + region[i]);
      bool first = true;
      for (int j = 0; j < i; ++j) first = first && region[j] != region[i];
      if (first) launch_permute_rows(itm.perm, itm.x, out, m, L.k, st);
      xp = out;
    }
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
  if (kind == 3)
    hipLaunchKernelGGL(gemm_wide_kernel, dim3(static_cast<unsigned>(wg)), dim3(256), 0, st, a);
  else if (kind == 2)
    hipLaunchKernelGGL(gemm_kernel<2>, dim3(static_cast<unsigned>(wg)), dim3(512), 0, st, a);
  else
    hipLaunchKernelGGL(gemm_kernel<1>, dim3(static_cast<unsigned>(wg)), dim3(256), 0, st, a);
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
  const polyq_gemm_item item{layout, packed, perm, x, y};
  return polyq_gemm_batch(&item, 1, m, workspace, workspace_bytes, stream);
}
