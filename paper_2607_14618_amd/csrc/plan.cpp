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
constexpr int kResidentWGs = 768;        // 256 CUs x 3 co-resident 4-wave work-groups (<= 168 VGPRs)
constexpr int kMinChunksPerWave = 4;      // below this the per-wave setup dominates
// Per work-group, one token: a third of the CU's 160 KB, so that the three
// work-groups the VGPR budget allows stay co-resident.
constexpr size_t kLdsBudget = (160 * 1024 / 3) & ~static_cast<size_t>(15);
// With several tokens the staged activations grow with M; a larger budget
// (two work-groups per CU instead of three) keeps the split count, and with
// it the number of work-group rounds, down.
constexpr size_t kLdsBudgetTokens = 80 * 1024;

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

size_t gemv_wave_lds_bytes(const GemvPlan& p, int32_t m) {
  // x' rows of the wave's channels (16-byte aligned), then its group metadata
  return static_cast<size_t>(align_up(static_cast<int64_t>(p.lds_chunks) * kChunk * m * 2, 16)) +
         static_cast<size_t>(p.lds_groups) * kMetaBytes;
}

size_t gemv_zero_offset(const GemvPlan& p, int32_t m) {
  return static_cast<size_t>(p.W) * gemv_wave_lds_bytes(p, m);
}

size_t gemv_lds_bytes(const GemvPlan& p, int32_t m) {
  // every wave's staging region and the work-group's zero row; the start is
  // reused for the reduction
  const size_t zero = static_cast<size_t>(align_up(static_cast<int64_t>(p.lds_chunks) * kChunk * 2, 16));
  const size_t red = static_cast<size_t>(p.W) * m * kTileRows * 4;
  return std::max(gemv_zero_offset(p, m) + zero, red);
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

// Cost of one 32-channel chunk of a 64-row tile, in units of 64 bytes (codes +
// the chunk's share of its group's 256-byte metadata).
static int64_t chunk_cost(int bits) { return 4 * bits + (bits <= 8 ? 1 : 0); }

// `parts` (>= nblocks) waves per tile, every wave inside one block: waves are
// given to blocks in proportion to their bytes (at least one each, at most one
// per group); wave_range then splits each block's groups evenly among its
// waves.  Waves left over when every block has one wave per group stay idle.
static void waves_per_block(const polyq_layout& L, int parts, int32_t* n) {
  const int nb = L.nblocks;
  int64_t cost[POLYQ_MAX_BLOCKS], total = 0;
  int ngr[POLYQ_MAX_BLOCKS], used = 0;
  for (int i = 0; i < nb; ++i) {
    const int nch = L.block[i].len / kChunk;
    ngr[i] = (nch + kChunksPerGroup - 1) / kChunksPerGroup;
    cost[i] = nch * chunk_cost(L.block[i].bits);
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
  for (int i = nb; i < POLYQ_MAX_BLOCKS; ++i) n[i] = 0;
}

int plan_gemv(const polyq_layout& L, int32_t m, int32_t launch_tiles, GemvPlan* p) {
  const int C = L.n_chunks, W = kWavesPerWG;
  // One round of co-resident work-groups per launch: splits beyond that only
  // add prologue and fix-up latency.  Every block needs a wave of its own.
  int S = std::max(1, kResidentWGs / std::max(1, launch_tiles));
  S = std::min(S, std::max(1, C / (W * kMinChunksPerWave)));
  S = std::max(S, (L.nblocks + W - 1) / W);
  S = std::max(1, std::min(S, kMaxSplitEntries / W));
  for (;;) {
    p->S = S;
    p->W = W;
    waves_per_block(L, S * W, p->waves);
    const LayoutBlocks blk{&L, p->waves};
    int worst = 0, worst_groups = 0;
    for (int w = 0; w < S * W; ++w) {
      int a, b;
      wave_range(w, L.nblocks, C, blk, &a, &b);
      if (a < b) {
        worst = std::max(worst, b - a);
        worst_groups = std::max(worst_groups, groups_touched(L, a, b));
      }
    }
    p->lds_chunks = worst;
    p->lds_groups = worst_groups;
    if (gemv_lds_bytes(*p, m) <= (m > 1 ? kLdsBudgetTokens : kLdsBudget)) return 0;
    if (S * W >= kMaxSplitEntries || S >= C) return 1;
    // one split at a time while splits are few, then doubling (very long k)
    S = S < 64 ? S + 1 : std::min(std::min(2 * S, kMaxSplitEntries / W), C);
  }
}

size_t gemv_workspace_for(const polyq_layout& L, int32_t m, const GemvPlan& p) {
  if (p.S <= 1) return 0;
  const size_t counters = static_cast<size_t>(align_up(static_cast<int64_t>(L.n_tiles) * 4, 256));
  return counters + static_cast<size_t>(p.S) * m * L.n_tiles * kTileRows * 4;
}

}  // namespace polyq

extern "C" size_t polyq_gemv_workspace_bytes(const polyq_layout* layout, int32_t m) {
  // enough with or without a permutation: the split-K state, and for several
  // tokens the clustered copy of x that a call with a permutation makes first
  if (!polyq::layout_is_valid(layout) || m < 1 || m > POLYQ_MAX_M_GEMV) return 0;
  polyq::GemvPlan p;
  if (polyq::plan_gemv(*layout, m, layout->n_tiles, &p) != 0) return 0;
  size_t need = static_cast<size_t>(polyq::align_up(static_cast<int64_t>(polyq::gemv_workspace_for(*layout, m, p)), 256));
  if (m > 1) need += static_cast<size_t>(polyq::align_up(static_cast<int64_t>(m) * layout->k * 2, 256));
  return need;
}
