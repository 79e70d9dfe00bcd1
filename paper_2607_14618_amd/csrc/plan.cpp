// Host-side planning: block-list validation, packed layout (polyq_plan),
// status strings and the decode-GEMV work split.  No HIP calls in this file.
#include <string.h>

#include <algorithm>
#include <vector>

#include "internal.h"

namespace {

bool bits_in_palette(int b) { return b == 2 || b == 3 || b == 4 || b == 8 || b == 16; }

// GEMV work split knobs.
constexpr int kWavesPerWG = 4;
constexpr int kResidentWGs = 512;        // 256 CUs x 2 co-resident 4-wave work-groups
constexpr int kMinChunksPerWave = 4;      // below this the per-wave setup dominates
constexpr size_t kLdsBudget = 64 * 1024;  // per work-group

}  // namespace

extern "C" polyq_status polyq_plan(int32_t n, int32_t k, const polyq_block* blocks,
                                   int32_t nblocks, polyq_layout* out) {
  if (blocks == nullptr || out == nullptr) return POLYQ_ERR_ARG;
  if (nblocks < 1 || nblocks > POLYQ_MAX_BLOCKS) return POLYQ_ERR_ARG;
  if (n < 1 || n > POLYQ_MAX_N || k < 1 || k > POLYQ_MAX_K) return POLYQ_ERR_SHAPE;
  int prev = 0;
  int64_t sum = 0;
  for (int i = 0; i < nblocks; ++i) {
    const int b = blocks[i].bits;
    if (!bits_in_palette(b) || b <= prev) return POLYQ_ERR_BITS;
    prev = b;
    const int len = blocks[i].len;
    if (len <= 0 || len % POLYQ_QUANTUM != 0) return POLYQ_ERR_QUANTUM;
    sum += len;
  }
  if (sum != k) return POLYQ_ERR_SHAPE;

  polyq_layout L;
  memset(&L, 0, sizeof(L));
  L.n = n;
  L.k = k;
  L.nblocks = nblocks;
  L.n_tiles = (n + polyq::kTileRows - 1) / polyq::kTileRows;
  L.n_chunks = k / polyq::kChunk;
  int64_t off = 0;
  int32_t k0 = 0, g0 = 0;
  int64_t code_bits = 0;
  for (int i = 0; i < nblocks; ++i) {
    const int b = blocks[i].bits, len = blocks[i].len;
    const int64_t chunk_row_bytes = 4 * b;  // 32 channels x b bits
    const int64_t meta = b <= 8 ? polyq::kMetaBytes : 0;
    const int64_t nch = len / polyq::kChunk;
    const int64_t ng = (len + polyq::kGroup - 1) / polyq::kGroup;
    L.block[i] = blocks[i];
    L.k_begin[i] = k0;
    L.group_begin[i] = g0;
    L.record_bytes[i] = meta + polyq::kChunksPerGroup * polyq::kTileRows * chunk_row_bytes;
    L.tile_bytes[i] = ng * meta + nch * polyq::kTileRows * chunk_row_bytes;
    L.block_offset[i] = off;
    off += static_cast<int64_t>(L.n_tiles) * L.tile_bytes[i];  // multiples of 256 B
    k0 += len;
    if (b <= 8) g0 += static_cast<int32_t>(ng);
    code_bits += static_cast<int64_t>(n) * b * len;
  }
  L.n_groups = g0;
  L.packed_bytes = off;
  L.code_bits = code_bits;
  L.weight_bytes = code_bits / 8 + static_cast<int64_t>(n) * g0 * 4;
  *out = L;
  return POLYQ_OK;
}

extern "C" const char* polyq_status_str(polyq_status s) {
  switch (s) {
    case POLYQ_OK: return "ok";
    case POLYQ_ERR_ARG: return "invalid argument (null pointer, bad size or bad layout)";
    case POLYQ_ERR_BITS: return "bit-widths must be strictly ascending values from {2,3,4,8,16}";
    case POLYQ_ERR_QUANTUM: return "block lengths must be positive multiples of 32";
    case POLYQ_ERR_SHAPE: return "block lengths must sum to k, with n and k in range";
    case POLYQ_ERR_CAPACITY: return "request exceeds a capacity limit (tokens or workspace)";
    case POLYQ_ERR_UNSUPPORTED: return "unsupported request";
    case POLYQ_ERR_DEVICE: return "a HIP runtime call failed";
  }
  return "unknown status";
}

namespace polyq {

bool layout_is_valid(const polyq_layout* L) {
  if (L == nullptr) return false;
  polyq_layout ref;
  if (polyq_plan(L->n, L->k, L->block, L->nblocks, &ref) != POLYQ_OK) return false;
  return memcmp(&ref, L, sizeof(ref)) == 0;
}

size_t gemv_lds_bytes(const GemvPlan& p, int32_t m) {
  // x' rows + a zero row (16-byte aligned), then every wave's group metadata;
  // reused for the reduction
  const size_t xs = static_cast<size_t>(align_up(static_cast<int64_t>(p.lds_chunks) * kChunk * (m + 1) * 2, 16)) +
                    static_cast<size_t>(p.W) * p.lds_groups * kMetaBytes;
  const size_t red = static_cast<size_t>(p.W) * m * kTileRows * 4;
  return std::max(xs, red);
}

// Group records of b <= 8 blocks that overlap the chunk range [lo, hi).
static int groups_touched(const polyq_layout& L, int lo, int hi) {
  int n = 0;
  for (int i = 0; i < L.nblocks; ++i) {
    if (L.block[i].bits > 8) continue;
    const int b0 = L.k_begin[i] / kChunk, b1 = b0 + L.block[i].len / kChunk;
    const int a = std::max(lo, b0), b = std::min(hi, b1);
    if (a < b) n += ((b - 1 - b0) >> 2) + 1 - ((a - b0) >> 2);
  }
  return n;
}

// The group boundary (block-relative multiple of 4 chunks, or the block end)
// nearest to chunk c.  GEMV waves start and end on these, so that every group
// record is processed whole by one wave.
static int snap_to_group(const polyq_layout& L, int c) {
  for (int i = 0; i < L.nblocks; ++i) {
    const int b0 = L.k_begin[i] / kChunk, b1 = b0 + L.block[i].len / kChunk;
    if (c < b0 || c >= b1) continue;
    const int down = b0 + (c - b0) / kChunksPerGroup * kChunksPerGroup;
    const int up = std::min(b1, down + kChunksPerGroup);
    return (c - down <= up - c) ? down : up;
  }
  return c;
}

static void partition(const polyq_layout& L, const std::vector<int64_t>& prefix, int parts,
                      int32_t* split) {
  const int C = static_cast<int>(prefix.size()) - 1;
  const int64_t total = prefix[C];
  split[0] = 0;
  int c = 0;
  for (int j = 1; j < parts; ++j) {
    const int64_t goal = (total * j + parts / 2) / parts;
    while (c < C && prefix[c] < goal) ++c;
    // pick the nearer of c-1 and c
    int best = c;
    if (c > 0 && goal - prefix[c - 1] < prefix[c] - goal) best = c - 1;
    best = std::max(snap_to_group(L, best), static_cast<int>(split[j - 1]));
    split[j] = best;
  }
  split[parts] = C;
}

// Cost of one 32-channel chunk of a 64-row tile, in units of 64 bytes (codes +
// the chunk's share of its group's 256-byte metadata).
static int64_t chunk_cost(int bits) { return 4 * bits + (bits <= 8 ? 1 : 0); }

// `parts` waves per tile with every wave inside one block: waves are given to
// blocks in proportion to their bytes (at least one each, at most one per
// group) and each block's groups are split evenly among its waves.  Returns
// false when there are fewer waves than blocks.
static bool partition_by_block(const polyq_layout& L, int parts, int32_t* split) {
  const int nb = L.nblocks;
  if (parts < nb) return false;
  int64_t cost[POLYQ_MAX_BLOCKS], total = 0;
  int nch[POLYQ_MAX_BLOCKS], ngr[POLYQ_MAX_BLOCKS], n[POLYQ_MAX_BLOCKS], used = 0;
  for (int i = 0; i < nb; ++i) {
    nch[i] = L.block[i].len / kChunk;
    ngr[i] = (nch[i] + kChunksPerGroup - 1) / kChunksPerGroup;
    cost[i] = nch[i] * chunk_cost(L.block[i].bits);
    total += cost[i];
  }
  for (int i = 0; i < nb; ++i) {
    n[i] = static_cast<int>(std::max<int64_t>(1, std::min<int64_t>(ngr[i], parts * cost[i] / total)));
    used += n[i];
  }
  while (used < parts) {  // next wave to the block with the most bytes per wave
    int best = -1;
    for (int i = 0; i < nb; ++i)
      if (n[i] < ngr[i] && (best < 0 || cost[i] * n[best] > cost[best] * n[i])) best = i;
    if (best < 0) break;
    ++n[best];
    ++used;
  }
  while (used > parts) {  // take a wave from the block with the fewest bytes per wave
    int best = -1;
    for (int i = 0; i < nb; ++i)
      if (n[i] > 1 && (best < 0 || cost[i] * n[best] < cost[best] * n[i])) best = i;
    --n[best];
    --used;
  }
  int u = 0;
  split[0] = 0;
  for (int i = 0; i < nb; ++i) {
    const int c0 = L.k_begin[i] / kChunk;
    for (int j = 0; j < n[i]; ++j) {
      const int g = static_cast<int>(static_cast<int64_t>(ngr[i]) * (j + 1) / n[i]);
      split[++u] = c0 + std::min(nch[i], g * kChunksPerGroup);
    }
  }
  for (; u < parts; ++u) split[u + 1] = L.n_chunks;  // waves left without work
  return true;
}

int plan_gemv(const polyq_layout& L, int32_t m, GemvPlan* p) {
  const int C = L.n_chunks, T = L.n_tiles;
  std::vector<int64_t> prefix(C + 1, 0);
  for (int i = 0; i < L.nblocks; ++i) {
    const int b = L.block[i].bits;
    const int c0 = L.k_begin[i] / kChunk, nc = L.block[i].len / kChunk;
    for (int c = 0; c < nc; ++c) prefix[c0 + c + 1] = prefix[c0 + c] + chunk_cost(b);
  }
  const int W = kWavesPerWG;
  // One round of co-resident work-groups: splits beyond that only add a second
  // round of prologue and fix-up latency.
  int S = std::max(1, kResidentWGs / T);
  S = std::min(S, std::max(1, C / (W * kMinChunksPerWave)));
  S = std::max(1, std::min(S, kMaxSplitEntries / W));
  for (;;) {
    p->S = S;
    p->W = W;
    p->nsplit = S * W;
    if (!partition_by_block(L, S * W, p->split)) partition(L, prefix, S * W, p->split);
    int worst = 0, worst_groups = 0;
    for (int s = 0; s < S; ++s) worst = std::max(worst, p->split[(s + 1) * W] - p->split[s * W]);
    for (int w = 0; w < S * W; ++w)
      worst_groups = std::max(worst_groups, groups_touched(L, p->split[w], p->split[w + 1]));
    p->lds_chunks = worst;
    p->lds_groups = worst_groups;
    if (gemv_lds_bytes(*p, m) <= kLdsBudget) return 0;
    if (S * W >= kMaxSplitEntries || S >= C) return 1;
    ++S;
  }
}

size_t gemv_workspace_for(const polyq_layout& L, int32_t m, const GemvPlan& p) {
  if (p.S <= 1) return 0;
  const size_t counters = static_cast<size_t>(align_up(static_cast<int64_t>(L.n_tiles) * 4, 256));
  return counters + static_cast<size_t>(p.S) * m * L.n_tiles * kTileRows * 4;
}

}  // namespace polyq

extern "C" size_t polyq_gemv_workspace_bytes(const polyq_layout* layout, int32_t m) {
  if (!polyq::layout_is_valid(layout) || m < 1 || m > POLYQ_MAX_M_GEMV) return 0;
  polyq::GemvPlan p;
  if (polyq::plan_gemv(*layout, m, &p) != 0) return 0;
  return polyq::gemv_workspace_for(*layout, m, p);
}
