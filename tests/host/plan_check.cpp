// Host-only property check of the planner (plan.cpp) and the bit allocation
// (alloc.cpp): packed layouts of random valid block lists, the statuses of
// invalid ones, the decode-GEMV work split (every chunk of a layer covered by
// exactly one wave, each wave inside one block and starting on one of its
// group boundaries, LDS within the work-group budget), and the allocation's
// outputs (palette bit-widths, the budget never exceeded by waterfilling,
// counts on the quantum after matching, a permutation from clustering).
// Built with g++ and the address and undefined-behaviour sanitizers by
// tests/test_host_sanitizer.py; exits non-zero on the first violated
// property.
#include <math.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <vector>

#include "internal.h"

namespace {

int g_fail = 0;

#define CHECK(cond, ...)                                  \
  do {                                                    \
    if (!(cond)) {                                        \
      fprintf(stderr, "FAIL %s:%d: %s: ", __FILE__, __LINE__, #cond); \
      fprintf(stderr, __VA_ARGS__);                       \
      fprintf(stderr, "\n");                              \
      ++g_fail;                                           \
      return;                                             \
    }                                                     \
  } while (0)

// splitmix64 (Steele, Lea and Flood 2014): a seeded, portable stream
struct Rng {
  uint64_t s;
  uint64_t next() {
    uint64_t z = (s += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
  }
  int uniform(int lo, int hi) { return lo + static_cast<int>(next() % static_cast<uint64_t>(hi - lo + 1)); }
};

const int kPalette[5] = {2, 3, 4, 8, 16};

// A random valid block list: a random ascending subset of the palette, each
// block a positive multiple of 32 channels.
int random_blocks(Rng& r, int max_units, polyq_block* b) {
  int nb = 0;
  for (int i = 0; i < 5; ++i)
    if (r.next() % 2) b[nb++] = polyq_block{kPalette[i], 0};
  if (nb == 0) b[nb++] = polyq_block{kPalette[r.uniform(0, 4)], 0};
  for (int i = 0; i < nb; ++i) b[i].len = 32 * r.uniform(1, max_units);
  return nb;
}

void check_layout(const polyq_layout& L, const polyq_block* b, int nb, int n, int k) {
  CHECK(L.n == n && L.k == k && L.nblocks == nb, "header");
  CHECK(L.n_tiles == (n + 63) / 64 && L.n_chunks == k / 32, "tiles %d chunks %d", L.n_tiles, L.n_chunks);
  int64_t off = 0, bits = 0;
  int k0 = 0, g0 = 0;
  for (int i = 0; i < nb; ++i) {
    const int64_t ng = (b[i].len + 127) / 128, nch = b[i].len / 32;
    const int64_t meta = b[i].bits <= 8 ? 256 : 0;
    CHECK(L.block[i].bits == b[i].bits && L.block[i].len == b[i].len, "block %d", i);
    CHECK(L.k_begin[i] == k0 && L.group_begin[i] == g0, "block %d begins", i);
    CHECK(L.block_offset[i] == off && off % 256 == 0, "block %d offset %lld", i, (long long)L.block_offset[i]);
    CHECK(L.tile_bytes[i] == ng * meta + nch * 64 * 4 * b[i].bits && L.tile_bytes[i] % 256 == 0,
          "block %d tile bytes %lld", i, (long long)L.tile_bytes[i]);
    off += static_cast<int64_t>(L.n_tiles) * L.tile_bytes[i];
    k0 += b[i].len;
    if (b[i].bits <= 8) g0 += static_cast<int>(ng);
    bits += static_cast<int64_t>(n) * b[i].bits * b[i].len;
  }
  CHECK(L.packed_bytes == off && L.n_groups == g0 && L.code_bits == bits, "totals");
  CHECK(L.weight_bytes == bits / 8 + static_cast<int64_t>(n) * g0 * 4, "weight bytes");
  CHECK(polyq::layout_is_valid(&L), "a planned layout is valid");
  polyq_layout bad = L;
  bad.packed_bytes += 256;
  CHECK(!polyq::layout_is_valid(&bad), "a changed layout is not valid");
}

// The decode split for m tokens: coverage, block and group alignment, budgets.
void check_gemv_plan(const polyq_layout& L, int m, int launch_tiles) {
  polyq::GemvPlan p;
  CHECK(polyq::plan_gemv(L, m, launch_tiles, &p) == 0, "no plan for k=%d m=%d", L.k, m);
  CHECK(p.W == 4 && p.S >= 1 && p.S * p.W <= polyq::kMaxSplitEntries, "S=%d W=%d", p.S, p.W);
  int sum = 0;
  for (int i = 0; i < L.nblocks; ++i) {
    CHECK(p.waves[i] >= 1, "block %d has no wave", i);
    sum += p.waves[i];
  }
  CHECK(sum <= p.S * p.W, "waves %d > %d", sum, p.S * p.W);
  const polyq::LayoutBlocks blk{&L, p.waves};
  std::vector<int> seen(L.n_chunks, 0);
  int worst = 0;
  for (int w = 0; w < p.S * p.W; ++w) {
    int a = 0, b = 0, bi = -2;
    polyq::wave_range(w, L.nblocks, L.n_chunks, blk, &a, &b, &bi);
    CHECK(0 <= a && a <= b && b <= L.n_chunks, "wave %d range [%d, %d)", w, a, b);
    if (a == b) continue;
    CHECK(bi >= 0 && bi < L.nblocks, "wave %d block %d", w, bi);
    const int cb = L.k_begin[bi] / 32, ce = cb + L.block[bi].len / 32;
    CHECK(cb <= a && b <= ce, "wave %d leaves block %d", w, bi);
    CHECK((a - cb) % 4 == 0 && (b == ce || (b - cb) % 4 == 0), "wave %d not on group boundaries", w);
    for (int c = a; c < b; ++c) ++seen[c];
    worst = b - a > worst ? b - a : worst;
  }
  for (int c = 0; c < L.n_chunks; ++c) CHECK(seen[c] == 1, "chunk %d covered %d times (m=%d)", c, seen[c], m);
  CHECK(worst == p.lds_chunks, "lds_chunks %d, widest range %d", p.lds_chunks, worst);
  CHECK(polyq::gemv_lds_bytes(p, m) <= 80 * 1024, "LDS %zu", polyq::gemv_lds_bytes(p, m));
  const size_t ws = polyq_gemv_workspace_bytes(&L, m);
  CHECK(ws >= polyq::gemv_workspace_for(L, m, p) || launch_tiles != L.n_tiles, "workspace %zu", ws);
}

void check_invalid() {
  polyq_layout L;
  polyq_block ok[2] = {{2, 64}, {16, 64}};
  CHECK(polyq_plan(64, 128, nullptr, 2, &L) == POLYQ_ERR_ARG, "null blocks");
  CHECK(polyq_plan(64, 128, ok, 2, nullptr) == POLYQ_ERR_ARG, "null out");
  CHECK(polyq_plan(64, 128, ok, 0, &L) == POLYQ_ERR_ARG, "no blocks");
  CHECK(polyq_plan(64, 128, ok, POLYQ_MAX_BLOCKS + 1, &L) == POLYQ_ERR_ARG, "too many blocks");
  CHECK(polyq_plan(0, 128, ok, 2, &L) == POLYQ_ERR_SHAPE, "n = 0");
  CHECK(polyq_plan(POLYQ_MAX_N + 1, 128, ok, 2, &L) == POLYQ_ERR_SHAPE, "n too large");
  CHECK(polyq_plan(64, POLYQ_MAX_K + 32, ok, 2, &L) == POLYQ_ERR_SHAPE, "k too large");
  CHECK(polyq_plan(64, 160, ok, 2, &L) == POLYQ_ERR_SHAPE, "sum != k");
  polyq_block desc[2] = {{4, 64}, {2, 64}};
  CHECK(polyq_plan(64, 128, desc, 2, &L) == POLYQ_ERR_BITS, "descending bits");
  polyq_block dup[2] = {{4, 64}, {4, 64}};
  CHECK(polyq_plan(64, 128, dup, 2, &L) == POLYQ_ERR_BITS, "repeated bits");
  polyq_block five[1] = {{5, 128}};
  CHECK(polyq_plan(64, 128, five, 1, &L) == POLYQ_ERR_BITS, "5 bits");
  polyq_block odd[2] = {{2, 48}, {16, 80}};
  CHECK(polyq_plan(64, 128, odd, 2, &L) == POLYQ_ERR_QUANTUM, "not a multiple of 32");
  polyq_block neg[2] = {{2, -32}, {16, 160}};
  CHECK(polyq_plan(64, 128, neg, 2, &L) == POLYQ_ERR_QUANTUM, "negative length");
  for (int s = -2; s < 10; ++s) CHECK(polyq_status_str(static_cast<polyq_status>(s)) != nullptr, "status %d", s);
  CHECK(polyq_gemv_workspace_bytes(nullptr, 1) == 0, "null layout");
  polyq_block one[1] = {{3, 256}};
  CHECK(polyq_plan(64, 256, one, 1, &L) == POLYQ_OK, "plan");
  CHECK(polyq_gemv_workspace_bytes(&L, 0) == 0 && polyq_gemv_workspace_bytes(&L, POLYQ_MAX_M_GEMV + 1) == 0,
        "m out of range");
}

void check_alloc(Rng& r, int iter) {
  const int n = r.uniform(1, 40), k = 32 * r.uniform(1, 40);
  std::vector<float> w(static_cast<size_t>(n) * k), s(k);
  std::vector<double> x2(k), err(static_cast<size_t>(POLYQ_NUM_BITS) * k);
  for (auto& v : w) v = static_cast<float>((static_cast<int64_t>(r.next() % 2001) - 1000) * 2e-5);
  for (int j = 0; j < k; ++j) {
    x2[j] = 1.0 + static_cast<double>(r.next() % 1000);
    s[j] = 0.5f + static_cast<float>(r.next() % 100) / 50.0f;
  }
  CHECK(polyq_channel_error(w.data(), n, k, x2.data(), iter % 2 ? s.data() : nullptr, err.data()) == POLYQ_OK,
        "channel_error");
  for (int j = 0; j < k; ++j) CHECK(err[4 * static_cast<size_t>(k) + j] == 0.0 && err[j] >= 0.0, "E_16 = 0, E >= 0");
  const double budget = 2.0 + static_cast<double>(r.next() % 1400) / 100.0;
  std::vector<int32_t> bits(k), perm(k);
  CHECK(polyq_waterfill(err.data(), k, budget, bits.data()) == POLYQ_OK, "waterfill");
  int64_t sum = 0;
  for (int j = 0; j < k; ++j) sum += bits[j];
  CHECK(sum <= static_cast<int64_t>(nearbyint(budget * k)) || sum == 2 * k, "budget exceeded: %lld", (long long)sum);
  int32_t counts[POLYQ_NUM_BITS];
  CHECK(polyq_quanta_match(err.data(), k, 32, budget, bits.data(), counts) == POLYQ_OK, "quanta_match");
  int32_t total = 0;
  for (int i = 0; i < POLYQ_NUM_BITS; ++i) {
    CHECK(counts[i] % 32 == 0, "count %d off the quantum", counts[i]);
    total += counts[i];
  }
  CHECK(total == k, "counts sum to %d, k %d", total, k);
  polyq_block blocks[POLYQ_MAX_BLOCKS];
  int32_t nb = 0;
  CHECK(polyq_cluster(bits.data(), k, perm.data(), blocks, &nb) == POLYQ_OK, "cluster");
  std::vector<int> seen(k, 0);
  for (int j = 0; j < k; ++j) ++seen[perm[j]];
  for (int j = 0; j < k; ++j) CHECK(seen[j] == 1, "perm is not a permutation");
  polyq_layout L;
  CHECK(polyq_plan(n, k, blocks, nb, &L) == POLYQ_OK, "clustered blocks plan");
  // Eq. 8 scales on the final bit map: powers of two, 16-bit channels at 1
  std::vector<double> sal(k);
  for (int j = 0; j < k; ++j) sal[j] = 0.05 + static_cast<double>(r.next() % 4000) / 100.0;
  const float grid[4] = {0.0f, 0.3f, 0.7f, 1.0f};
  float alpha[POLYQ_NUM_BITS];
  CHECK(polyq_bit_scaling(w.data(), n, k, x2.data(), sal.data(), bits.data(), grid, 4, s.data(), alpha) ==
            POLYQ_OK, "bit_scaling");
  for (int j = 0; j < k; ++j) {
    int e = 0;
    CHECK(frexpf(s[j], &e) == 0.5f, "scale %g is not a power of two", static_cast<double>(s[j]));
    CHECK(bits[j] != 16 || s[j] == 1.0f, "16-bit channel scaled");
  }
  CHECK(alpha[POLYQ_NUM_BITS - 1] == 0.0f, "alpha_16 = 0");
  const float bad_grid[1] = {1.5f};
  CHECK(polyq_bit_scaling(w.data(), n, k, x2.data(), sal.data(), bits.data(), bad_grid, 1, s.data(), nullptr) ==
            POLYQ_ERR_ARG, "grid out of [0, 1] refused");
  CHECK(polyq_waterfill(err.data(), k, NAN, bits.data()) == POLYQ_ERR_ARG, "NaN budget refused");
  CHECK(polyq_quanta_match(err.data(), k, 7, budget, bits.data(), counts) ==
            (k % 7 ? POLYQ_ERR_QUANTUM : POLYQ_OK), "quantum check");
}

}  // namespace

int main(int argc, char** argv) {
  const uint64_t seed = argc > 1 ? strtoull(argv[1], nullptr, 10) : 1;
  const int iters = argc > 2 ? atoi(argv[2]) : 300;
  Rng r{seed};
  check_invalid();
  for (int it = 0; it < iters && !g_fail; ++it) {
    polyq_block b[POLYQ_MAX_BLOCKS];
    // mostly short layers, some long ones up to the largest k
    const int max_units = it % 25 == 0 ? (POLYQ_MAX_K / 32) / 5 : (it % 5 == 0 ? 200 : 24);
    const int nb = random_blocks(r, max_units, b);
    int k = 0;
    for (int i = 0; i < nb; ++i) k += b[i].len;
    const int n = r.uniform(1, 5 * 64 + 7);
    polyq_layout L;
    const polyq_status st = polyq_plan(n, k, b, nb, &L);
    if (k > POLYQ_MAX_K) {
      if (st != POLYQ_ERR_SHAPE) { fprintf(stderr, "FAIL k=%d status %d\n", k, st); ++g_fail; }
      continue;
    }
    if (st != POLYQ_OK) { fprintf(stderr, "FAIL plan status %d (k=%d)\n", st, k); ++g_fail; break; }
    check_layout(L, b, nb, n, k);
    const int ms[4] = {1, 2, 5, 16};
    for (int j = 0; j < 4 && !g_fail; ++j) {
      check_gemv_plan(L, ms[j], L.n_tiles);
      check_gemv_plan(L, ms[j], L.n_tiles * r.uniform(1, 40));
    }
  }
  for (int it = 0; it < iters / 10 + 1 && !g_fail; ++it) check_alloc(r, it);
  if (g_fail) return 1;
  printf("plan_check ok: seed %llu, %d layouts\n", static_cast<unsigned long long>(seed), iters);
  return 0;
}
