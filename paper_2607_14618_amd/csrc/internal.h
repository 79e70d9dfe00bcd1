// Internal definitions shared by the host planner and the HIP kernels of the
// mixed-bit linear-layer library.  Not part of the public ABI (include/polyq.h).
#pragma once

#include <stdint.h>

#include "polyq.h"

namespace polyq {

constexpr int kTileRows = POLYQ_TILE_ROWS;  // output rows per packed tile (one per lane)
constexpr int kChunk = POLYQ_QUANTUM;       // channels per chunk
constexpr int kGroup = POLYQ_GROUP;         // channels per quantization group
constexpr int kChunksPerGroup = kGroup / kChunk;
constexpr int kMetaBytes = kTileRows * 4;   // {fp16 s, fp16 z} per row of a tile

// Decode GEMV launch plan: WGs = n_tiles x S, each of W waves; wave w of split
// s processes the global chunk range [split[s*W + w], split[s*W + w + 1]).
constexpr int kMaxSplitEntries = 256;  // S * W <= this

struct GemvPlan {
  int32_t S;                    // WG splits per 64-row tile
  int32_t W;                    // waves per WG
  int32_t lds_chunks;           // largest chunk range of one WG
  int32_t lds_groups;           // most group records one wave stages (b <= 8 blocks)
  int32_t nsplit;               // S * W
  int32_t split[kMaxSplitEntries + 1];
};

// Returns 0 on success.  Chooses S and W for `m` tokens and partitions the
// layer's chunks by bytes.
int plan_gemv(const polyq_layout& L, int32_t m, GemvPlan* p);

// Bytes of GEMV workspace needed for plan p (0 when S == 1): one uint32 counter
// per tile (padded to 256 B) followed by the partials [S][m][n_tiles*64] fp32.
size_t gemv_workspace_for(const polyq_layout& L, int32_t m, const GemvPlan& p);

// True when `L` is exactly what polyq_plan produces for its own n, k, blocks.
bool layout_is_valid(const polyq_layout* L);

// LDS bytes of a GEMV work-group for plan p and m tokens.
size_t gemv_lds_bytes(const GemvPlan& p, int32_t m);

inline int64_t align_up(int64_t v, int64_t a) { return (v + a - 1) / a * a; }

}  // namespace polyq
