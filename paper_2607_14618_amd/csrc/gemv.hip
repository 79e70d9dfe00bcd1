// Decode / small-batch GEMV over the mixed-bit clustered weight (Sec. 4.1-4.2),
// 1 <= M <= 16 tokens, on the matrix cores.
//
// Mapping on gfx950: a wave owns one 64-row tile and a contiguous range of
// 32-channel chunks.  For each chunk, lane l loads its 4b-byte slice (rows
// 16r + l%16, r = 0..3, channels 8(l/16) .. +7: one contiguous 512 B .. 4 KB
// run per wave), unpacks the 32 codes into exact fp16 (q - z) values -- the
// A fragments of four v_mfma_f32_16x16x32_f16, one per 16-row sub-tile -- and
// the B fragment is the 8 activations x'[token l%16][8(l/16) .. +7] from LDS.
// The 16 columns of the MFMA are the tokens, so M = 1 and M = 16 cost the same;
// the matrix pipe is otherwise idle, so the VALU only unpacks.
//
// Unpacking: a code field placed at mantissa bits [f, f+b) of an fp16 half is
// turned into the exact fp16 value (2^(10-f) + q) by OR-ing in the exponent
// field 25-f (one v_and_or_b32 for two codes); adding -(2^(10-f) + z) (exact
// for integer zero points) gives q - z exactly.  Each 128-channel group
// accumulates into its own fp32 tile, scaled once by the row's fp16 scale:
// y += s * sum_group (q - z) x'.  All products are exact; only fp32
// accumulation rounds.  16-bit channels enter the MFMA as their fp16 weights.
//
// A work-group (tile, split) stages its slice of the permuted activations
// x'[k'] = x[perm[k']] (Eq. 9) into LDS once, its waves take byte-balanced
// contiguous chunk ranges and reduce through LDS; splits of a tile across
// work-groups are combined by the last-arriving work-group (fixed order).
#include <hip/hip_runtime.h>

#include "codec.h"
#include "internal.h"

namespace polyq {
namespace {

typedef _Float16 h2 __attribute__((ext_vector_type(2)));
typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int kWaves = 4;  // waves per work-group (the host plan uses the same)

struct GemvArgs {
  const uint8_t* packed;
  const int32_t* perm;
  const uint16_t* x;
  float* y;
  float* partial;     // [S][m][rows_pad], only when S > 1
  uint32_t* counter;  // [n_tiles], only when S > 1
  int32_t n, k, m, nblocks, rows_pad, S;
  int32_t bits[POLYQ_MAX_BLOCKS];
  int32_t chunk_begin[POLYQ_MAX_BLOCKS];
  int32_t chunk_end[POLYQ_MAX_BLOCKS];
  int64_t block_offset[POLYQ_MAX_BLOCKS];
  int64_t tile_bytes[POLYQ_MAX_BLOCKS];
  int64_t record_bytes[POLYQ_MAX_BLOCKS];
  int32_t split[kMaxSplitEntries + 1];
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

// Load one lane slice (4*B bytes).
template <int B>
__device__ __forceinline__ void load_slice(const uint8_t* p, uint32_t* w) {
  if constexpr (B == 2) {
    const uint2 u = *reinterpret_cast<const uint2*>(p);
    w[0] = u.x; w[1] = u.y;
  } else if constexpr (B == 3) {
    const uint32_t* q = reinterpret_cast<const uint32_t*>(p);
    w[0] = q[0]; w[1] = q[1]; w[2] = q[2];
  } else {
#pragma unroll
    for (int i = 0; i < B / 4; ++i) {
      const uint4 u = reinterpret_cast<const uint4*>(p)[i];
      w[4 * i + 0] = u.x; w[4 * i + 1] = u.y; w[4 * i + 2] = u.z; w[4 * i + 3] = u.w;
    }
  }
}

// Batch geometry per bit-width: a batch is up to NB chunks of one group whose
// slices (16 dwords at most) are loaded together; two batches are in flight per
// wave (the next one is loaded while the current one is unpacked).
template <int B>
struct Geo {
  static constexpr int NB = B <= 4 ? 4 : (B == 8 ? 2 : 1);  // chunks per batch
  static constexpr int CB = 4 * B;                           // bytes per lane slice
  static constexpr int META = B <= 8 ? kMetaBytes : 0;
};

struct Buf {
  uint32_t w[16];  // NB slices of B dwords each
  uint32_t z[2];   // z of the lane's 4 dequantized rows (fp16), b <= 8
  uint32_t s[8];   // s of the lane's 16 accumulator rows (fp16), b <= 8
};

// End (exclusive) of the batch that starts at block-local chunk c.
template <int B>
__device__ __forceinline__ int batch_end(int c, int l1) {
  if constexpr (B == 16) {
    return c + 1;
  } else {
    return min(min(c + Geo<B>::NB, (c | 3) + 1), l1);
  }
}

// Issue the loads of the batch [c, cend) of one tile (slots past cend re-read chunk c).
template <int B>
__device__ __forceinline__ void issue(Buf& b, const uint8_t* __restrict__ tile_base,
                                      int64_t record_bytes, int c, int cend, int lane) {
  using G = Geo<B>;
  const uint8_t* rec = tile_base + (c >> 2) * record_bytes;
  if constexpr (B <= 8) {
    const uint2 zz = *reinterpret_cast<const uint2*>(rec + (lane & 15) * 8);
    b.z[0] = zz.x; b.z[1] = zz.y;
    const uint4* sp = reinterpret_cast<const uint4*>(rec + 128 + (lane >> 4) * 32);
    const uint4 s0 = sp[0], s1 = sp[1];
    b.s[0] = s0.x; b.s[1] = s0.y; b.s[2] = s0.z; b.s[3] = s0.w;
    b.s[4] = s1.x; b.s[5] = s1.y; b.s[6] = s1.z; b.s[7] = s1.w;
  }
  const uint8_t* slices = rec + G::META + lane * G::CB;
#pragma unroll
  for (int j = 0; j < G::NB; ++j) {
    const int cj = (c + j < cend) ? c + j : c;
    load_slice<B>(slices + (cj & 3) * (64 * G::CB), &b.w[j * B]);
  }
}

struct Group {
  h2 c1[16];     // per pair: -(offset + z_row) (integer z) or -offset
  h2 c2[4];      // per row: -z (non-integer z only)
  float s[16];   // scale of each accumulator row
  bool exact;
  f4 part[4];    // this group's accumulators, one per 16-row sub-tile
};

__device__ __forceinline__ h8 frag(const uint32_t* w4) {
  const uint4 u{w4[0], w4[1], w4[2], w4[3]};
  return __builtin_bit_cast(h8, u);
}

// Unpack one slice of a b <= 8 block into exact (q - z) fragments and run the
// four MFMAs of its 16-row sub-tiles against the activation fragment.
template <int B, bool kExactZ>
__device__ __forceinline__ void quant_slice(const uint32_t* w, h8 xb, Group& gs) {
  using U = Unpack<B>;
  uint32_t v[16];
  U::run(w, v);
  uint32_t d[16];
#pragma unroll
  for (int P = 0; P < 16; ++P) {
    h2 t = as_h2(v[P]) + gs.c1[P];
    if constexpr (!kExactZ) t = t + gs.c2[P >> 2];
    d[P] = as_u32(t);
  }
#pragma unroll
  for (int r = 0; r < 4; ++r)
    gs.part[r] = __builtin_amdgcn_mfma_f32_16x16x32_f16(frag(&d[4 * r]), xb, gs.part[r], 0, 0, 0);
}

// Unpack and accumulate the batch [c, cend) of a segment [l0, l1).  `xlane`
// points at this lane's activation fragment of block-local chunk l0 (LDS).
template <int B>
__device__ __forceinline__ void compute(const Buf& b, int c, int cend, int l0, int l1,
                                        const uint32_t* xlane, Group& gs, f4 (&acc)[4]) {
  using G = Geo<B>;
  if constexpr (B == 16) {
    const h8 xb = __builtin_bit_cast(h8, *reinterpret_cast<const uint4*>(xlane + (c - l0) * 16));
#pragma unroll
    for (int r = 0; r < 4; ++r)
      acc[r] = __builtin_amdgcn_mfma_f32_16x16x32_f16(frag(&b.w[4 * r]), xb, acc[r], 0, 0, 0);
  } else {
    using U = Unpack<B>;
    if ((c & 3) == 0 || c == l0) {  // first batch of a group (or of the segment)
      float z[4];
#pragma unroll
      for (int r = 0; r < 4; ++r)
        z[r] = static_cast<float>(__builtin_bit_cast(
            _Float16, static_cast<uint16_t>(b.z[r >> 1] >> (16 * (r & 1)))));
      bool ok = true;
#pragma unroll
      for (int r = 0; r < 4; ++r) ok = ok && (z[r] == truncf(z[r])) && fabsf(z[r]) <= 1023.f;
      // integer zero points (the asymmetric quantizer's): one exact add per pair
      gs.exact = __all(ok);
#pragma unroll
      for (int P = 0; P < 16; ++P)
        gs.c1[P] = gs.exact ? splat(-(U::offset[U::which[P]] + z[P >> 2])) : splat(-U::offset[U::which[P]]);
#pragma unroll
      for (int r = 0; r < 4; ++r) gs.c2[r] = splat(-z[r]);
#pragma unroll
      for (int i = 0; i < 16; ++i)
        gs.s[i] = static_cast<float>(__builtin_bit_cast(
            _Float16, static_cast<uint16_t>(b.s[i >> 1] >> (16 * (i & 1)))));
#pragma unroll
      for (int r = 0; r < 4; ++r) gs.part[r] = f4{0.f, 0.f, 0.f, 0.f};
    }
    if (gs.exact) {
#pragma unroll
      for (int j = 0; j < G::NB; ++j) {
        if (c + j < cend) {
          const h8 xb = __builtin_bit_cast(h8, *reinterpret_cast<const uint4*>(xlane + (c + j - l0) * 16));
          quant_slice<B, true>(&b.w[j * B], xb, gs);
        }
      }
    } else {
#pragma unroll
      for (int j = 0; j < G::NB; ++j) {
        if (c + j < cend) {
          const h8 xb = __builtin_bit_cast(h8, *reinterpret_cast<const uint4*>(xlane + (c + j - l0) * 16));
          quant_slice<B, false>(&b.w[j * B], xb, gs);
        }
      }
    }
    if ((cend & 3) == 0 || cend == l1) {  // group complete: apply its scales once
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[r][e] = fmaf(gs.s[4 * r + e], gs.part[r][e], acc[r][e]);
    }
  }
}

// Block-local chunks [l0, l1) of one tile: two batches in flight (ping-pong).
// `b0` already holds the first batch when `preloaded`.  The next batch is always
// issued (at the segment end it re-reads the current one, an L1/L2 hit), so the
// number of loads between a batch's issue and its use is fixed and the wait
// before each compute covers only the older batch.
template <int B>
__device__ __forceinline__ void run_segment(const uint8_t* __restrict__ tile_base,
                                            int64_t record_bytes, int l0, int l1,
                                            const uint32_t* xlane, int lane, Buf& b0,
                                            bool preloaded, f4 (&acc)[4]) {
  Buf b1;
  Group gs;
  int c = l0;
  int ce = batch_end<B>(c, l1);
  if (!preloaded) issue<B>(b0, tile_base, record_bytes, c, ce, lane);
  for (;;) {
    int cn = ce < l1 ? ce : c;
    int cne = ce < l1 ? batch_end<B>(cn, l1) : ce;
    issue<B>(b1, tile_base, record_bytes, cn, cne, lane);
    compute<B>(b0, c, ce, l0, l1, xlane, gs, acc);
    if (ce >= l1) break;
    c = cn;
    ce = cne;
    cn = ce < l1 ? ce : c;
    cne = ce < l1 ? batch_end<B>(cn, l1) : ce;
    issue<B>(b0, tile_base, record_bytes, cn, cne, lane);
    compute<B>(b1, c, ce, l0, l1, xlane, gs, acc);
    if (ce >= l1) break;
    c = cn;
    ce = cne;
  }
}

__global__ __launch_bounds__(kWaves * 64) void gemv_kernel(const GemvArgs a) {
  extern __shared__ uint32_t smem[];
  const int tile = blockIdx.x, s = blockIdx.y;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int m = a.m;
  const int cw0 = a.split[s * kWaves], cw1 = a.split[(s + 1) * kWaves];
  const int range = (cw1 - cw0) * kChunk;  // staged channels
  const int kbase = cw0 * kChunk;
  const int c0 = a.split[s * kWaves + wave], c1 = a.split[s * kWaves + wave + 1];

  // Start streaming this wave's first weight batch before staging x'.
  int first = 0;
  while (first < a.nblocks && a.chunk_end[first] <= c0) ++first;
  Buf b0;
  bool preloaded = false;
  if (c0 < c1 && first < a.nblocks) {
    const int l0 = c0 - a.chunk_begin[first];
    const int l1 = min(c1, a.chunk_end[first]) - a.chunk_begin[first];
    const uint8_t* tile_base = a.packed + a.block_offset[first] + tile * a.tile_bytes[first];
    const int64_t rb = a.record_bytes[first];
    preloaded = true;
    switch (a.bits[first]) {
      case 2: issue<2>(b0, tile_base, rb, l0, batch_end<2>(l0, l1), lane); break;
      case 3: issue<3>(b0, tile_base, rb, l0, batch_end<3>(l0, l1), lane); break;
      case 4: issue<4>(b0, tile_base, rb, l0, batch_end<4>(l0, l1), lane); break;
      case 8: issue<8>(b0, tile_base, rb, l0, batch_end<8>(l0, l1), lane); break;
      default: issue<16>(b0, tile_base, rb, l0, batch_end<16>(l0, l1), lane); break;
    }
  }

  // Stage x'[i][k'] = x[i][perm[k']] for this work-group's clustered channels
  // (rows 0..m-1) and a zero row m read by the MFMA columns of absent tokens.
  uint16_t* xs16 = reinterpret_cast<uint16_t*>(smem);
  for (int kk = threadIdx.x; kk < range; kk += blockDim.x) {
    const int kp = kbase + kk;
    const int src = a.perm != nullptr ? a.perm[kp] : kp;
    const bool ok = static_cast<unsigned>(src) < static_cast<unsigned>(a.k);
    for (int mi = 0; mi < m; ++mi) xs16[mi * range + kk] = ok ? a.x[static_cast<int64_t>(mi) * a.k + src] : 0;
    xs16[m * range + kk] = 0;
  }
  __syncthreads();

  f4 acc[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) acc[r] = f4{0.f, 0.f, 0.f, 0.f};
  const int tok = lane & 15;
  // this lane's activation row (token lane%16, or the zero row) and channel quarter
  const uint32_t* xrow = smem + ((tok < m ? tok : m) * range + 8 * (lane >> 4)) / 2;
  for (int bi = first; bi < a.nblocks; ++bi) {
    const int lo = max(c0, a.chunk_begin[bi]), hi = min(c1, a.chunk_end[bi]);
    if (lo >= hi) break;
    const uint8_t* tile_base = a.packed + a.block_offset[bi] + tile * a.tile_bytes[bi];
    const int l0 = lo - a.chunk_begin[bi], l1 = hi - a.chunk_begin[bi];
    const uint32_t* xlane = xrow + (lo - cw0) * 16;
    const int64_t rb = a.record_bytes[bi];
    const bool pre = preloaded && bi == first;
    switch (a.bits[bi]) {
      case 2: run_segment<2>(tile_base, rb, l0, l1, xlane, lane, b0, pre, acc); break;
      case 3: run_segment<3>(tile_base, rb, l0, l1, xlane, lane, b0, pre, acc); break;
      case 4: run_segment<4>(tile_base, rb, l0, l1, xlane, lane, b0, pre, acc); break;
      case 8: run_segment<8>(tile_base, rb, l0, l1, xlane, lane, b0, pre, acc); break;
      default: run_segment<16>(tile_base, rb, l0, l1, xlane, lane, b0, pre, acc); break;
    }
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
  if (wave != 0) return;
  const int row = tile * 64 + lane;
  if (a.S == 1) {
    for (int mi = 0; mi < m; ++mi) {
      float v = 0.f;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) v += red[(w * m + mi) * 64 + lane];
      if (row < a.n) a.y[static_cast<int64_t>(mi) * a.n + row] = v;
    }
    return;
  }
  // Split-K fix-up.  Each partial is written, and later read back and zeroed,
  // with a returning device-scope atomic swap, and a work-group takes its ticket
  // only after its swaps have returned: swaps and the ticket add on one address
  // are ordered at that address's device-wide point of coherence, so the
  // work-group whose ticket closes the round (ticket mod S == S-1, whatever the
  // counter held before) reads every partial of the round.  It sums them in
  // split order (deterministic), leaves them zero and resets the counter.  (A
  // release/acquire-fence version is both slower -- every fence writes back or
  // invalidates the XCD's whole L2 -- and was measured to read stale partials.)
  for (int mi = 0; mi < m; ++mi) {
    float v = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) v += red[(w * m + mi) * 64 + lane];
    float* p = &a.partial[(static_cast<int64_t>(s) * m + mi) * a.rows_pad + row];
    const float old = __hip_atomic_exchange(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    asm volatile("" ::"v"(old));  // keep the returning form of the swap
  }
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_waitcnt(0);  // the swaps have returned
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  uint32_t ticket = 0;
  if (lane == 0)
    ticket = __hip_atomic_fetch_add(&a.counter[tile], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  ticket = __shfl(ticket, 0);
  if (ticket % static_cast<uint32_t>(a.S) != static_cast<uint32_t>(a.S - 1)) return;
  for (int mi = 0; mi < m; ++mi) {
    float v = 0.f;
    for (int s2 = 0; s2 < a.S; ++s2)
      v += __hip_atomic_exchange(&a.partial[(static_cast<int64_t>(s2) * m + mi) * a.rows_pad + row],
                                 0.f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (row < a.n) a.y[static_cast<int64_t>(mi) * a.n + row] = v;
  }
  if (lane == 0) __hip_atomic_store(&a.counter[tile], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

}  // namespace
}  // namespace polyq

using namespace polyq;

extern "C" polyq_status polyq_gemv(const polyq_layout* layout, const void* packed,
                                   const int32_t* perm, const uint16_t* x, int32_t m, float* y,
                                   void* workspace, size_t workspace_bytes, void* stream) {
  if (!layout_is_valid(layout)) return POLYQ_ERR_ARG;
  const polyq_layout& L = *layout;
  if (packed == nullptr || x == nullptr || y == nullptr) return POLYQ_ERR_ARG;
  if (reinterpret_cast<uintptr_t>(packed) % 256 != 0) return POLYQ_ERR_ARG;
  if (reinterpret_cast<uintptr_t>(x) % 2 != 0 || reinterpret_cast<uintptr_t>(y) % 4 != 0)
    return POLYQ_ERR_ARG;
  if (m < 1) return POLYQ_ERR_ARG;
  if (m > POLYQ_MAX_M_GEMV) return POLYQ_ERR_CAPACITY;
  GemvPlan plan;
  if (plan_gemv(L, m, &plan) != 0) return POLYQ_ERR_CAPACITY;
  const size_t need = gemv_workspace_for(L, m, plan);
  if (need > 0 && (workspace == nullptr || workspace_bytes < need)) return POLYQ_ERR_CAPACITY;
  if (need > 0 && reinterpret_cast<uintptr_t>(workspace) % 256 != 0) return POLYQ_ERR_ARG;

  GemvArgs a;
  a.packed = static_cast<const uint8_t*>(packed);
  a.perm = perm;
  a.x = x;
  a.y = y;
  a.n = L.n;
  a.k = L.k;
  a.m = m;
  a.nblocks = L.nblocks;
  a.rows_pad = L.n_tiles * kTileRows;
  a.S = plan.S;
  if (plan.W != kWaves) return POLYQ_ERR_UNSUPPORTED;
  a.partial = nullptr;
  a.counter = nullptr;
  if (need > 0) {  // [counters: n_tiles x u32, 256-aligned][partials: S x m x rows_pad fp32]
    a.counter = static_cast<uint32_t*>(workspace);
    a.partial = reinterpret_cast<float*>(static_cast<uint8_t*>(workspace) +
                                         align_up(static_cast<int64_t>(L.n_tiles) * 4, 256));
  }
  for (int i = 0; i < POLYQ_MAX_BLOCKS; ++i) {
    const bool used = i < L.nblocks;
    a.bits[i] = used ? L.block[i].bits : 0;
    a.chunk_begin[i] = used ? L.k_begin[i] / kChunk : 0;
    a.chunk_end[i] = used ? (L.k_begin[i] + L.block[i].len) / kChunk : 0;
    a.block_offset[i] = used ? L.block_offset[i] : 0;
    a.tile_bytes[i] = used ? L.tile_bytes[i] : 0;
    a.record_bytes[i] = used ? L.record_bytes[i] : 0;
  }
  for (int i = 0; i <= plan.nsplit; ++i) a.split[i] = plan.split[i];
  for (int i = plan.nsplit + 1; i <= kMaxSplitEntries; ++i) a.split[i] = plan.split[plan.nsplit];

  const dim3 grid(L.n_tiles, plan.S), block(kWaves * 64);
  const size_t lds = gemv_lds_bytes(plan, m);
  hipLaunchKernelGGL(gemv_kernel, grid, block, lds, static_cast<hipStream_t>(stream), a);
  return hipGetLastError() == hipSuccess ? POLYQ_OK : POLYQ_ERR_DEVICE;
}
