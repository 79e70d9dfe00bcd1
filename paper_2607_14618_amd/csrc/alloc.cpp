// Compile-time bit allocation (Sec. 3.1-3.4): the activation-aware error
// proxy (Eq. 1-2), per-layer waterfilling under a fractional budget (Eq. 3-5),
// ISA-aware quanta matching (Eq. 6-7), channel clustering (Sec. 4.1) and the
// bit-specific activation-aware scales (Eq. 8).
// Host code on host memory; no HIP calls in this file.
#include <math.h>
#include <stdint.h>
#include <string.h>

#include <algorithm>
#include <queue>
#include <vector>

#include "polyq.h"

namespace {

constexpr int kBits[POLYQ_NUM_BITS] = {2, 3, 4, 8, 16};
constexpr int kProxyGroup = 128;  // input channels per quantization group of the proxy
constexpr int kScaleExp = 14;     // |log2 s| of the Eq. 8 scales: 1/s stays a normal fp16 value

int bit_index(int b) {
  for (int i = 0; i < POLYQ_NUM_BITS; ++i)
    if (kBits[i] == b) return i;
  return -1;
}

// The fp16 value nearest to v (ties to even), as a double; beyond the fp16
// range it is +-inf.  Normal range: a spacing of 2^(e - 10) for |v| in
// [2^e, 2^(e+1)); below 2^-14 the subnormal spacing 2^-24.  v / spacing is
// exact (a power of two), so one rint gives the nearest multiple.
double round_to_half(double v) {
  if (v == 0.0 || !isfinite(v)) return v;
  int e2 = 0;
  frexp(v, &e2);  // |v| = m 2^e2, m in [0.5, 1): |v| in [2^(e2-1), 2^e2)
  const int e = std::max(e2 - 1, -14);
  const double spacing = ldexp(1.0, e - 10);
  const double r = rint(v / spacing) * spacing;
  return fabs(r) >= 65536.0 ? copysign(INFINITY, v) : r;  // 65504 is the largest fp16
}

// Eq. 3: the gain per extra bit of moving channel j from palette index i to i + 1.
inline double gain(const double* err, int32_t k, int i, int32_t j) {
  return (err[static_cast<int64_t>(i) * k + j] - err[static_cast<int64_t>(i + 1) * k + j]) /
         static_cast<double>(kBits[i + 1] - kBits[i]);
}

// Squared reconstruction error, weighted by x2 and summed over the channels
// `idx` (in that order) and the n rows, of Q_b applied to W[:, idx] diag(s)
// in groups of 128 consecutive listed channels per row (b = kBits[bi]).
double block_error(const float* w, int32_t n, int32_t k, const double* x2, const int32_t* idx,
                   int32_t cnt, const double* s, int bi) {
  const double qmax = static_cast<double>((1 << kBits[bi]) - 1);
  std::vector<double> sq(cnt, 0.0), ws(kProxyGroup);
  for (int32_t r = 0; r < n; ++r) {
    const float* row = w + static_cast<int64_t>(r) * k;
    for (int32_t a = 0; a < cnt; a += kProxyGroup) {
      const int32_t len = std::min(kProxyGroup, cnt - a);
      double mn = INFINITY, mx = -INFINITY;
      for (int32_t t = 0; t < len; ++t) {
        ws[t] = static_cast<double>(row[idx[a + t]]) * s[a + t];
        mn = std::min(mn, ws[t]);
        mx = std::max(mx, ws[t]);
      }
      const double s16 = round_to_half((mx - mn) / qmax);
      const bool dead = s16 == 0.0;
      const double st = dead ? 1.0 : s16;
      const double z = std::min(std::max(rint(-mn / st), 0.0), qmax);
      for (int32_t t = 0; t < len; ++t) {
        const double q = std::min(std::max(rint(ws[t] / st) + z, 0.0), qmax);
        const double val = dead ? 0.0 : st * (q - z);
        const double d = val / s[a + t] - static_cast<double>(row[idx[a + t]]);
        sq[a + t] += d * d;
      }
    }
  }
  double e = 0.0;
  for (int32_t t = 0; t < cnt; ++t) e += sq[t] * x2[idx[t]];
  return e;
}

}  // namespace

extern "C" polyq_status polyq_channel_error(const float* w, int32_t n, int32_t k, const double* x2,
                                            const float* scale, double* err) {
  if (w == nullptr || x2 == nullptr || err == nullptr || n < 1 || k < 1) return POLYQ_ERR_ARG;
  if (static_cast<int64_t>(n) * k > (int64_t{1} << 31)) return POLYQ_ERR_SHAPE;
  for (int32_t j = 0; j < k; ++j) {
    if (!(x2[j] >= 0.0) || !isfinite(x2[j])) return POLYQ_ERR_ARG;
    if (scale != nullptr && (!(scale[j] > 0.0f) || !isfinite(scale[j]))) return POLYQ_ERR_ARG;
  }
  std::vector<double> s(k, 1.0);
  if (scale != nullptr)
    for (int32_t j = 0; j < k; ++j) s[j] = scale[j];
  // squared reconstruction error per channel, summed over the rows in order
  std::vector<double> sq(static_cast<size_t>(POLYQ_NUM_BITS) * k, 0.0);
  std::vector<double> ws(kProxyGroup);
  for (int32_t r = 0; r < n; ++r) {
    const float* row = w + static_cast<int64_t>(r) * k;
    for (int32_t a = 0; a < k; a += kProxyGroup) {
      const int32_t e = std::min(a + kProxyGroup, k), len = e - a;
      double mn = INFINITY, mx = -INFINITY;
      for (int32_t j = 0; j < len; ++j) {
        ws[j] = static_cast<double>(row[a + j]) * s[a + j];  // diag(s) W (exact in fp64)
        mn = std::min(mn, ws[j]);
        mx = std::max(mx, ws[j]);
      }
      for (int i = 0; i + 1 < POLYQ_NUM_BITS; ++i) {  // b = 2, 3, 4, 8
        const double qmax = static_cast<double>((1 << kBits[i]) - 1);
        const double s16 = round_to_half((mx - mn) / qmax);
        const bool dead = s16 == 0.0;
        const double st = dead ? 1.0 : s16;
        const double z = std::min(std::max(rint(-mn / st), 0.0), qmax);
        double* acc = sq.data() + static_cast<int64_t>(i) * k + a;
        for (int32_t j = 0; j < len; ++j) {
          const double q = std::min(std::max(rint(ws[j] / st) + z, 0.0), qmax);
          const double val = dead ? 0.0 : st * (q - z);
          const double d = val / s[a + j] - static_cast<double>(row[a + j]);  // diag(s)^-1 Q_b(...) - W
          acc[j] += d * d;
        }
      }
    }
  }
  for (int i = 0; i < POLYQ_NUM_BITS; ++i)
    for (int32_t j = 0; j < k; ++j)
      err[static_cast<int64_t>(i) * k + j] =
          kBits[i] == 16 ? 0.0 : sq[static_cast<int64_t>(i) * k + j] * x2[j];
  return POLYQ_OK;
}

extern "C" polyq_status polyq_waterfill(const double* err, int32_t k, double budget, int32_t* bits) {
  if (err == nullptr || bits == nullptr || k < 1 || !isfinite(budget) || budget > 16.0)
    return POLYQ_ERR_ARG;
  for (int32_t j = 0; j < k; ++j) bits[j] = 2;
  int64_t remaining = static_cast<int64_t>(nearbyint(budget * k)) - 2 * static_cast<int64_t>(k);
  if (remaining <= 0) return POLYQ_OK;
  // max-heap of (gain, channel, from-index): larger gain first, then lower channel
  struct Cand {
    double g;
    int32_t j;
    int i;
  };
  auto below = [](const Cand& x, const Cand& y) { return x.g < y.g || (x.g == y.g && x.j > y.j); };
  std::priority_queue<Cand, std::vector<Cand>, decltype(below)> heap(below);
  for (int32_t j = 0; j < k; ++j) heap.push(Cand{gain(err, k, 0, j), j, 0});
  while (remaining > 0 && !heap.empty()) {
    const Cand c = heap.top();
    heap.pop();
    if (bits[c.j] != kBits[c.i]) continue;  // stale (one entry per channel: cannot happen)
    const int step = kBits[c.i + 1] - kBits[c.i];
    if (step > remaining) continue;  // does not fit, and never will
    bits[c.j] = kBits[c.i + 1];
    remaining -= step;
    if (c.i + 2 < POLYQ_NUM_BITS) heap.push(Cand{gain(err, k, c.i + 1, c.j), c.j, c.i + 1});
  }
  return POLYQ_OK;
}

extern "C" polyq_status polyq_quanta_match(const double* err, int32_t k, int32_t quantum, double budget,
                                           int32_t* bits, int32_t* counts) {
  if (err == nullptr || bits == nullptr || k < 1 || quantum < 1 || !isfinite(budget) || budget > 16.0)
    return POLYQ_ERR_ARG;
  for (int32_t j = 0; j < k; ++j)
    if (bit_index(bits[j]) < 0) return POLYQ_ERR_ARG;
  if (k % quantum != 0) return POLYQ_ERR_QUANTUM;
  int64_t c[POLYQ_NUM_BITS] = {};
  for (int32_t j = 0; j < k; ++j) ++c[bit_index(bits[j])];
  // (1) round to the quantum: floors, then the units left to the largest
  // remainders (ties to the higher bit-width)
  int64_t t[POLYQ_NUM_BITS];
  int64_t left = k / quantum;
  for (int i = 0; i < POLYQ_NUM_BITS; ++i) {
    t[i] = c[i] / quantum;
    left -= t[i];
  }
  int order[POLYQ_NUM_BITS] = {4, 3, 2, 1, 0};  // higher bit-width first among equal remainders
  std::stable_sort(order, order + POLYQ_NUM_BITS,
                   [&](int x, int y) { return c[x] % quantum > c[y] % quantum; });
  for (int u = 0; u < left; ++u) ++t[order[u]];
  // (2) budget repair: whole-quantum moves between neighbouring levels while
  // one brings the total strictly closer to round(B k)
  const int64_t target = static_cast<int64_t>(nearbyint(budget * k));
  for (;;) {
    int64_t cur = 0;
    for (int i = 0; i < POLYQ_NUM_BITS; ++i) cur += static_cast<int64_t>(kBits[i]) * t[i] * quantum;
    int64_t best = 0;
    int bs = -1, bd = -1;
    for (int i = 0; i + 1 < POLYQ_NUM_BITS; ++i) {
      const int pairs[2][2] = {{i, i + 1}, {i + 1, i}};  // promotion, then demotion
      for (const auto& p : pairs) {
        if (t[p[0]] == 0) continue;
        const int64_t nw = cur + static_cast<int64_t>(kBits[p[1]] - kBits[p[0]]) * quantum;
        const int64_t better = std::llabs(cur - target) - std::llabs(nw - target);
        if (better > best) {
          best = better;
          bs = p[0];
          bd = p[1];
        }
      }
    }
    if (bs < 0) break;
    --t[bs];
    ++t[bd];
  }
  // (3) single-channel moves between neighbouring levels until the counts match
  int64_t target_count[POLYQ_NUM_BITS];
  for (int i = 0; i < POLYQ_NUM_BITS; ++i) target_count[i] = t[i] * quantum;
  for (;;) {
    bool moved = false;
    for (int i = 0; i + 1 < POLYQ_NUM_BITS && !moved; ++i) {
      int64_t flow = 0;  // channels that must cross the boundary above level i upwards
      for (int l = i + 1; l < POLYQ_NUM_BITS; ++l) flow += target_count[l] - c[l];
      if (flow == 0) continue;
      const int src = flow > 0 ? i : i + 1, dst = flow > 0 ? i + 1 : i;
      int32_t pick = -1;
      double pg = 0.0;
      for (int32_t j = 0; j < k; ++j) {
        if (bits[j] != kBits[src]) continue;
        const double g = gain(err, k, i, j);
        if (pick < 0 || (flow > 0 ? g > pg : g < pg)) {
          pick = j;
          pg = g;
        }
      }
      if (pick < 0) continue;  // source level empty: a lower boundary moves first
      bits[pick] = kBits[dst];
      --c[src];
      ++c[dst];
      moved = true;
    }
    if (!moved) break;
  }
  if (counts != nullptr)
    for (int i = 0; i < POLYQ_NUM_BITS; ++i) counts[i] = static_cast<int32_t>(c[i]);
  return POLYQ_OK;
}

extern "C" polyq_status polyq_cluster(const int32_t* bits, int32_t k, int32_t* perm, polyq_block* blocks,
                                      int32_t* nblocks) {
  if (bits == nullptr || perm == nullptr || blocks == nullptr || nblocks == nullptr || k < 1)
    return POLYQ_ERR_ARG;
  for (int32_t j = 0; j < k; ++j)
    if (bit_index(bits[j]) < 0) return POLYQ_ERR_ARG;
  int32_t pos = 0, nb = 0;
  for (int i = 0; i < POLYQ_NUM_BITS; ++i) {
    const int32_t start = pos;
    for (int32_t j = 0; j < k; ++j)
      if (bits[j] == kBits[i]) perm[pos++] = j;
    if (pos > start) blocks[nb++] = polyq_block{kBits[i], pos - start};
  }
  for (int i = nb; i < POLYQ_MAX_BLOCKS; ++i) blocks[i] = polyq_block{0, 0};
  *nblocks = nb;
  return POLYQ_OK;
}

extern "C" polyq_status polyq_bit_scaling(const float* w, int32_t n, int32_t k, const double* x2,
                                          const double* saliency, const int32_t* bits, const float* grid,
                                          int32_t ngrid, float* scale, float* alpha) {
  if (w == nullptr || x2 == nullptr || saliency == nullptr || bits == nullptr || grid == nullptr ||
      scale == nullptr || n < 1 || k < 1 || ngrid < 1)
    return POLYQ_ERR_ARG;
  if (static_cast<int64_t>(n) * k > (int64_t{1} << 31)) return POLYQ_ERR_SHAPE;
  for (int32_t j = 0; j < k; ++j) {
    if (bit_index(bits[j]) < 0) return POLYQ_ERR_ARG;
    if (!(x2[j] >= 0.0) || !isfinite(x2[j])) return POLYQ_ERR_ARG;
    if (!(saliency[j] > 0.0) || !isfinite(saliency[j])) return POLYQ_ERR_ARG;
  }
  for (int32_t g = 0; g < ngrid; ++g)
    if (!(grid[g] >= 0.0f && grid[g] <= 1.0f)) return POLYQ_ERR_ARG;
  for (int32_t j = 0; j < k; ++j) scale[j] = 1.0f;
  float al[POLYQ_NUM_BITS] = {0.f, 0.f, 0.f, 0.f, 0.f};
  std::vector<int32_t> idx;
  std::vector<double> s, best_s;
  for (int bi = 0; bi + 1 < POLYQ_NUM_BITS; ++bi) {  // 16-bit channels are unquantized: s = 1
    idx.clear();
    for (int32_t j = 0; j < k; ++j)
      if (bits[j] == kBits[bi]) idx.push_back(j);
    if (idx.empty()) continue;
    const int32_t cnt = static_cast<int32_t>(idx.size());
    s.assign(cnt, 1.0);
    double best = INFINITY;
    for (int32_t g = 0; g < ngrid; ++g) {
      // s_j = 2^rint(alpha log2 m_j): Eq. 8's power law, kept to powers of two,
      // the exponent clamped to [-kScaleExp, kScaleExp] so that 1/s_j is a
      // normal fp16 value
      for (int32_t t = 0; t < cnt; ++t) {
        const double e = rint(static_cast<double>(grid[g]) * log2(saliency[idx[t]]));
        s[t] = ldexp(1.0, static_cast<int>(std::min(std::max(e, -1.0 * kScaleExp), 1.0 * kScaleExp)));
      }
      const double e = block_error(w, n, k, x2, idx.data(), cnt, s.data(), bi);
      if (e < best) {  // ties keep the earlier grid point
        best = e;
        best_s = s;
        al[bi] = grid[g];
      }
    }
    for (int32_t t = 0; t < cnt; ++t) scale[idx[t]] = static_cast<float>(best_s[t]);
  }
  if (alpha != nullptr)
    for (int i = 0; i < POLYQ_NUM_BITS; ++i) alpha[i] = al[i];
  return POLYQ_OK;
}
