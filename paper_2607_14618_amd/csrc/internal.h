// Internal definitions shared by the host planner and the HIP kernels of the
// mixed-bit linear-layer library.  Not part of the public ABI (include/polyq.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "polyq.h"

namespace polyq {

constexpr int kTileRows = POLYQ_TILE_ROWS;  // output rows per packed tile (one per lane)
constexpr int kChunk = POLYQ_QUANTUM;       // channels per chunk
constexpr int kGroup = POLYQ_GROUP;         // channels per quantization group
constexpr int kChunksPerGroup = kGroup / kChunk;
constexpr int kMetaBytes = kTileRows * 4;   // {fp16 s, fp16 z} per row of a tile

// Decode GEMV launch plan: the work-groups of one linear are n_tiles x S, each
// of W waves; wave w (0 <= w < S * W, across the tile's splits) covers the
// chunk range wave_range(w).  Every wave stays inside one block: block i gets
// waves[i] waves per tile.
constexpr int kMaxSplitEntries = 4096;  // S * W <= this

struct GemvPlan {
  int32_t S;                        // WG splits per 64-row tile
  int32_t W;                        // waves per WG
  int32_t waves[POLYQ_MAX_BLOCKS];  // waves per tile given to each block
  int32_t lds_chunks;               // largest chunk range of one wave
  int32_t lds_groups;               // most group records one wave stages (b <= 8 blocks)
};

// Exact floor(a / d) for 1 <= d and 0 <= a < 2^31 by a multiply and shifts
// (round-up multiplier, Granlund and Montgomery 1994): with l = floor(log2 d)
// and M = ceil(2^(32+l) / d), a M / 2^(32+l) = a / d + a e / (d 2^(32+l)) where
// e = M d - 2^(32+l) < d < 2^(l+1); since a e < 2^31 2^(l+1) = 2^(32+l) the
// excess stays below 1/d and cannot reach the next integer.  M < 2^32 unless d
// is a power of two, where div_magic returns 0 and the quotient is a >> l.
__host__ __device__ inline int div_log2(uint32_t d) { return d <= 1 ? 0 : 31 - __builtin_clz(d); }
__host__ __device__ inline uint32_t div_magic(uint32_t d) {
  if ((d & (d - 1)) == 0) return 0u;  // 0, 1 and powers of two
  return static_cast<uint32_t>(((1ull << (32 + div_log2(d))) + d - 1) / d);
}
__host__ __device__ inline uint32_t div_by_magic(uint32_t a, uint32_t magic, uint32_t d) {
  const uint32_t hi =
      magic == 0 ? a : static_cast<uint32_t>((static_cast<uint64_t>(a) * magic) >> 32);
  return hi >> div_log2(d);
}

// Chunk range [lo, hi) of wave w of every tile: waves are handed to the blocks
// in order (waves[i] to block i, starting at wave w0[i]) and a block's groups
// are split evenly among its waves, so that every wave starts and ends on a
// group boundary of one block.  Waves past the last block get an empty range
// at the end of the layer.  `blk` gives, for block i (a uniform run-time
// index), cb(i) / ce(i) (chunk range), w0(i), nw(i) and magic(i) =
// div_magic(nw(i)).  Shared by the host planner and the kernel, which must
// agree exactly; the kernel evaluates it in scalar registers, so the block is
// found with a handful of compares and read once.  `block` (optional) receives
// the block index i (or -1); the range is empty unless w < w0(i) + nw(i).
template <class Blk>
__host__ __device__ inline void wave_range(int w, int nblocks, int n_chunks, const Blk& blk,
                                           int* lo, int* hi, int* block = nullptr) {
  int i = -1;
#pragma unroll
  for (int b = 0; b < POLYQ_MAX_BLOCKS; ++b)
    if (b < nblocks && blk.w0(b) <= w) i = b;
  *lo = *hi = n_chunks;
  if (block) *block = i;
  if (i < 0) return;
  const int w0 = blk.w0(i), nw = blk.nw(i);
  if (w >= w0 + nw) return;
  const int cb = blk.cb(i), nch = blk.ce(i) - cb;
  const int ngr = (nch + kChunksPerGroup - 1) / kChunksPerGroup, j = w - w0;
  const uint32_t magic = blk.magic(i);
  const int a = kChunksPerGroup * static_cast<int>(div_by_magic(static_cast<uint32_t>(ngr * j), magic, nw));
  const int b = kChunksPerGroup * static_cast<int>(div_by_magic(static_cast<uint32_t>(ngr * (j + 1)), magic, nw));
  *lo = cb + (a < nch ? a : nch);
  *hi = cb + (b < nch ? b : nch);
}

// Returns 0 on success.  Chooses S, W and the waves per block for `m` tokens;
// `launch_tiles` is the number of 64-row tiles of every linear that shares the
// launch (the splits are sized so that the launch fills the GPU about once).
int plan_gemv(const polyq_layout& L, int32_t m, int32_t launch_tiles, GemvPlan* p);

// Bytes of GEMV workspace needed for plan p (0 when S == 1): one uint32 counter
// per tile (padded to 256 B) followed by the partials [S][m][n_tiles*64] fp32.
size_t gemv_workspace_for(const polyq_layout& L, int32_t m, const GemvPlan& p);

// True when `L` is exactly what polyq_plan produces for its own n, k, blocks.
bool layout_is_valid(const polyq_layout* L);

// LDS bytes of one GEMV wave's staging region (x' of m tokens, then group
// metadata), the offset of the work-group's shared zero row (after the W wave
// regions) and the LDS of a work-group, for plan p and m tokens.
size_t gemv_wave_lds_bytes(const GemvPlan& p, int32_t m);
size_t gemv_zero_offset(const GemvPlan& p, int32_t m);
size_t gemv_lds_bytes(const GemvPlan& p, int32_t m);

// Validation and workspace size of a polyq_gemv_batch request: every check
// polyq_gemv_batch makes before it launches, except the workspace's own.
// need: total bytes; zero: the leading bytes that must be zero on entry.
polyq_status gemv_batch_workspace_status(const polyq_gemv_item* items, int32_t count, int32_t m,
                                         size_t* need, size_t* zero);

// One copy of the explicit activation shuffle (Eq. 9, with Eq. 8's channel
// factors): out[i][j] = x[i][perm[j]] * f[j] for m rows of k 2-byte
// activations.  perm NULL: the identity; an entry outside [0, k) yields 0;
// f NULL: no factors (the values are copied bit for bit); otherwise fp16
// factors, the product rounded to the activation type.
struct ShuffleJob {
  const int32_t* perm;
  const uint16_t* f;
  const uint16_t* x;
  uint16_t* out;
  int32_t k, pad;
};
// All `count` (<= POLYQ_MAX_BATCH) copies in one launch on `stream` (fp16
// activations, or bf16 when `bf16`); rows are staged in LDS when there are
// many and k and the alignments allow.  Launch only: the caller has validated
// the arguments.
void launch_shuffle(const ShuffleJob* jobs, int count, int32_t m, bool bf16, hipStream_t stream);

// Block accessor of a layout for wave_range (host side).
struct LayoutBlocks {
  const polyq_layout* L;
  const int32_t* waves;
  int cb(int i) const { return L->k_begin[i] / kChunk; }
  int ce(int i) const { return (L->k_begin[i] + L->block[i].len) / kChunk; }
  int w0(int i) const {
    int first = 0;
    for (int j = 0; j < i; ++j) first += waves[j];
    return first;
  }
  int nw(int i) const { return waves[i]; }
  uint32_t magic(int i) const { return div_magic(static_cast<uint32_t>(waves[i])); }
};

inline int64_t align_up(int64_t v, int64_t a) { return (v + a - 1) / a * a; }

}  // namespace polyq
