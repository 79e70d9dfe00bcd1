// Pack / unpack of the clustered quantized weight (Sec. 4.1: the clustered
// weight P W is materialized once, at compile time) and the explicit activation
// shuffle of Eq. 9.  Memory-bound helper kernels; the packed layout is the one
// declared in include/polyq.h.  Packing can also reorder the output rows
// (Sec. 4.3, Eq. 10): packed row r then holds source row row_perm[r], so the
// layer emits its output directly in a consumer's clustered channel basis.
#include <hip/hip_runtime.h>

#include "codec.h"
#include "internal.h"

namespace polyq {
namespace {

constexpr int kThreads = 256;

constexpr int64_t kMaxPermuteElems = (static_cast<int64_t>(1) << 31) - 1;  // m * k of polyq_permute

inline unsigned grid_for(int64_t items) {
  return static_cast<unsigned>((items + kThreads - 1) / kThreads);
}

// Source row of packed row R (R < n): R itself, or row_perm[R]; -1 (a zero
// row) for an entry outside [0, n).
__device__ __forceinline__ int source_row(const int32_t* __restrict__ row_perm, int R, int n) {
  if (row_perm == nullptr) return R;
  const int src = row_perm[R];
  return static_cast<unsigned>(src) < static_cast<unsigned>(n) ? src : -1;
}

// One thread per (tile, chunk, lane slice): gathers the slice's 4 rows x 8
// channels from the row-major codes and writes its 4*B bytes.
template <int B>
__global__ __launch_bounds__(kThreads) void pack_codes_kernel(
    const uint16_t* __restrict__ codes, const int32_t* __restrict__ row_perm, int n, int k, int k0,
    int nch, int n_tiles, int64_t tile_bytes, int64_t record_bytes, uint8_t* __restrict__ region) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (idx >= static_cast<int64_t>(n_tiles) * nch * 64) return;
  const int lane = static_cast<int>(idx % 64);
  const int64_t rest = idx / 64;
  const int t = static_cast<int>(rest % n_tiles), c = static_cast<int>(rest / n_tiles);
  uint16_t q[32];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int R = t * 64 + 16 * r + (lane % 16);
    const int src = R < n ? source_row(row_perm, R, n) : -1;
    if (src >= 0) {
      const uint4 u = *reinterpret_cast<const uint4*>(codes + static_cast<int64_t>(src) * k + k0 +
                                                      c * 32 + 8 * (lane / 16));
      const uint32_t wd[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        q[slice_index(r, 2 * j)] = static_cast<uint16_t>(wd[j] & 0xFFFFu);
        q[slice_index(r, 2 * j + 1)] = static_cast<uint16_t>(wd[j] >> 16);
      }
    } else {
#pragma unroll
      for (int j = 0; j < 8; ++j) q[slice_index(r, j)] = 0;
    }
  }
  uint32_t w[B];
  encode_slice<B>(q, w);
  uint32_t* dst = reinterpret_cast<uint32_t*>(
      region + slice_offset(tile_bytes, record_bytes, B <= 8 ? kMetaBytes : 0, B, t, c, lane));
#pragma unroll
  for (int d = 0; d < B; ++d) dst[d] = w[d];
}

template <int B>
__global__ __launch_bounds__(kThreads) void unpack_codes_kernel(
    const uint8_t* __restrict__ region, int n, int k, int k0, int nch, int n_tiles,
    int64_t tile_bytes, int64_t record_bytes, uint16_t* __restrict__ codes) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (idx >= static_cast<int64_t>(n_tiles) * nch * 64) return;
  const int lane = static_cast<int>(idx % 64);
  const int64_t rest = idx / 64;
  const int t = static_cast<int>(rest % n_tiles), c = static_cast<int>(rest / n_tiles);
  const uint32_t* src = reinterpret_cast<const uint32_t*>(
      region + slice_offset(tile_bytes, record_bytes, B <= 8 ? kMetaBytes : 0, B, t, c, lane));
  uint32_t w[B];
#pragma unroll
  for (int d = 0; d < B; ++d) w[d] = src[d];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int R = t * 64 + 16 * r + (lane % 16);
    if (R >= n) continue;
    uint32_t out[4];
#pragma unroll
    for (int j = 0; j < 4; ++j)
      out[j] = slice_code<B>(w, slice_index(r, 2 * j)) | (slice_code<B>(w, slice_index(r, 2 * j + 1)) << 16);
    *reinterpret_cast<uint4*>(codes + static_cast<int64_t>(R) * k + k0 + c * 32 + 8 * (lane / 16)) =
        uint4{out[0], out[1], out[2], out[3]};
  }
}

// One thread per (row, block-local group): scale and zero point into the group's metadata.
__global__ __launch_bounds__(kThreads) void pack_meta_kernel(
    const uint16_t* __restrict__ scales, const uint16_t* __restrict__ zeros,
    const int32_t* __restrict__ row_perm, int n, int G, int g0, int ng, int64_t tile_bytes,
    int64_t record_bytes, int rows_total, uint8_t* __restrict__ region) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (idx >= static_cast<int64_t>(rows_total) * ng) return;
  const int R = static_cast<int>(idx % rows_total);
  const int g = static_cast<int>(idx / rows_total);
  uint16_t sv = 0, zv = 0;
  const int src = R < n ? source_row(row_perm, R, n) : -1;
  if (src >= 0) {
    const int64_t at = static_cast<int64_t>(src) * G + g0 + g;
    sv = scales[at];
    zv = zeros[at];
  }
  uint16_t* meta = reinterpret_cast<uint16_t*>(region + (R / 64) * tile_bytes + g * record_bytes);
  meta[meta_z_half(R % 64)] = zv;
  meta[meta_s_half(R % 64)] = sv;
}

__global__ __launch_bounds__(kThreads) void unpack_meta_kernel(
    const uint8_t* __restrict__ region, int n, int G, int g0, int ng, int64_t tile_bytes,
    int64_t record_bytes, uint16_t* __restrict__ scales, uint16_t* __restrict__ zeros) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (idx >= static_cast<int64_t>(n) * ng) return;
  const int R = static_cast<int>(idx % n);
  const int g = static_cast<int>(idx / n);
  const uint16_t* meta =
      reinterpret_cast<const uint16_t*>(region + (R / 64) * tile_bytes + g * record_bytes);
  const int64_t at = static_cast<int64_t>(R) * G + g0 + g;
  if (scales) scales[at] = meta[meta_s_half(R % 64)];
  if (zeros) zeros[at] = meta[meta_z_half(R % 64)];
}

__global__ __launch_bounds__(kThreads) void permute_kernel(const int32_t* __restrict__ perm,
                                                           const uint16_t* __restrict__ x,
                                                           uint16_t* __restrict__ out, int m, int k) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (idx >= static_cast<int64_t>(m) * k) return;
  const int i = static_cast<int>(idx / k), kp = static_cast<int>(idx % k);
  const int p = perm[kp];
  out[idx] = static_cast<unsigned>(p) < static_cast<unsigned>(k) ? x[static_cast<int64_t>(i) * k + p] : 0;
}

// The explicit shuffle x'[i][j] = x[i][perm[j]] * f[j] of several copies in one
// launch (grid.y = copy).  perm NULL: the identity; an entry outside [0, k)
// yields 0; f NULL: no factors, the 2-byte values are copied as they are;
// otherwise f holds Eq. 8's fp16 channel factors 1/s_j and the product is
// formed in fp32 and rounded (nearest even) to the activation type (fp16, or
// bf16 when `bf16`): exact for a power-of-two factor.
constexpr int kPermLdsK = 32768;   // longest row staged in LDS
constexpr int kPermLdsMinRows = 64;

struct ShuffleArgs {
  ShuffleJob job[POLYQ_MAX_BATCH];
  int32_t m, bf16;
};

__device__ __forceinline__ float act_to_f32(uint16_t h, bool bf16) {
  return bf16 ? __builtin_bit_cast(float, static_cast<uint32_t>(h) << 16)
              : static_cast<float>(__builtin_bit_cast(_Float16, h));
}
__device__ __forceinline__ uint16_t f32_to_act(float v, bool bf16) {
  if (!bf16) return __builtin_bit_cast(uint16_t, static_cast<_Float16>(v));
  const uint32_t u = __builtin_bit_cast(uint32_t, v);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return static_cast<uint16_t>((u >> 16) | 0x40u);  // NaN stays NaN
  return static_cast<uint16_t>((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}
__device__ __forceinline__ uint16_t scaled(uint16_t v, uint16_t f, bool bf16) {
  return f32_to_act(act_to_f32(v, bf16) * static_cast<float>(__builtin_bit_cast(_Float16, f)), bf16);
}

// A few rows (decode tokens): one element per thread, spread over the chip.
__global__ __launch_bounds__(256) void shuffle_elems_kernel(const ShuffleArgs a) {
  const ShuffleJob& jb = a.job[blockIdx.y];
  const int k = jb.k;
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (idx >= static_cast<int64_t>(a.m) * k) return;
  const int i = static_cast<int>(idx / k), j = static_cast<int>(idx % k);
  const int p = jb.perm != nullptr ? jb.perm[j] : j;
  uint16_t v = static_cast<unsigned>(p) < static_cast<unsigned>(k) ? jb.x[static_cast<int64_t>(i) * k + p] : 0;
  if (jb.f != nullptr) v = scaled(v, jb.f[j], a.bf16 != 0);
  jb.out[idx] = v;
}

// Many rows (prefill): one row per work-group, staged in LDS with 16-byte loads
// (k <= kPermLdsK, k % 8 == 0, 16-byte aligned rows, permutation and
// factors), then 8 channels per thread and pass: the permutation and factors
// as 16-byte loads, one 16-byte store.  The indices and factors of the first
// kPre passes (k <= 16384) are loaded together with the row (one memory round
// trip).
__global__ __launch_bounds__(256) void shuffle_rows_lds_kernel(const ShuffleArgs a) {
  extern __shared__ uint4 row4[];
  const ShuffleJob& jb = a.job[blockIdx.y];
  const int k = jb.k, k8 = k / 8;
  const bool has_perm = jb.perm != nullptr, has_f = jb.f != nullptr, bf16 = a.bf16 != 0;
  const uint16_t* row = reinterpret_cast<const uint16_t*>(row4);
  const int64_t base = static_cast<int64_t>(blockIdx.x) * k;
  const uint4* src = reinterpret_cast<const uint4*>(jb.x + base);
  const int4* p4 = reinterpret_cast<const int4*>(jb.perm);
  const uint4* f4 = reinterpret_cast<const uint4*>(jb.f);
  constexpr int kPre = 8;  // passes whose indices come with the row (k <= 16384 in one round trip)
  int4 pp[kPre][2];
  uint4 ff[kPre];
#pragma unroll
  for (int u = 0; u < kPre; ++u) {
    const int j = threadIdx.x + u * 256;
    if (j < k8) {
      if (has_perm) {
        pp[u][0] = p4[2 * j];
        pp[u][1] = p4[2 * j + 1];
      }
      if (has_f) ff[u] = f4[j];
    }
  }
  for (int j = threadIdx.x; j < k8; j += 256) row4[j] = src[j];
  __syncthreads();
  uint4* dst = reinterpret_cast<uint4*>(jb.out + base);
  auto gather = [&](int j, int4 p0, int4 p1, uint4 fv) {
    int p[8] = {p0.x, p0.y, p0.z, p0.w, p1.x, p1.y, p1.z, p1.w};
    if (!has_perm) {
#pragma unroll
      for (int e = 0; e < 8; ++e) p[e] = 8 * j + e;
    }
    const uint32_t fw[4] = {fv.x, fv.y, fv.z, fv.w};
    uint32_t h[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      uint16_t v = static_cast<unsigned>(p[e]) < static_cast<unsigned>(k) ? row[p[e]] : 0;
      if (has_f) v = scaled(v, static_cast<uint16_t>(fw[e / 2] >> (16 * (e & 1))), bf16);
      h[e] = v;
    }
    dst[j] = uint4{h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16)};
  };
  const int4 z4{0, 0, 0, 0};
  const uint4 zf{0u, 0u, 0u, 0u};
#pragma unroll
  for (int u = 0; u < kPre; ++u) {
    const int j = threadIdx.x + u * 256;
    if (j < k8) gather(j, has_perm ? pp[u][0] : z4, has_perm ? pp[u][1] : z4, has_f ? ff[u] : zf);
  }
  for (int j = threadIdx.x + kPre * 256; j < k8; j += 256)
    gather(j, has_perm ? p4[2 * j] : z4, has_perm ? p4[2 * j + 1] : z4, has_f ? f4[j] : zf);
}

template <int B>
void launch_pack(const polyq_layout& L, int i, const uint16_t* codes, const int32_t* row_perm,
                 uint8_t* region, hipStream_t st) {
  const int nch = L.block[i].len / kChunk;
  hipLaunchKernelGGL(pack_codes_kernel<B>,
                     dim3(grid_for(static_cast<int64_t>(L.n_tiles) * nch * 64)), dim3(kThreads), 0,
                     st, codes, row_perm, L.n, L.k, L.k_begin[i], nch, L.n_tiles, L.tile_bytes[i],
                     L.record_bytes[i], region);
}

template <int B>
void launch_unpack(const polyq_layout& L, int i, const uint8_t* region, uint16_t* codes,
                   hipStream_t st) {
  const int nch = L.block[i].len / kChunk;
  hipLaunchKernelGGL(unpack_codes_kernel<B>,
                     dim3(grid_for(static_cast<int64_t>(L.n_tiles) * nch * 64)), dim3(kThreads), 0,
                     st, region, L.n, L.k, L.k_begin[i], nch, L.n_tiles, L.tile_bytes[i],
                     L.record_bytes[i], codes);
}

}  // namespace

void launch_shuffle(const ShuffleJob* jobs, int count, int32_t m, bool bf16, hipStream_t st) {
  if (count < 1) return;
  ShuffleArgs a{};
  bool lds = m >= kPermLdsMinRows;
  int kmax = 0;
  for (int i = 0; i < count; ++i) {
    const ShuffleJob& j = jobs[i];
    a.job[i] = j;
    kmax = std::max(kmax, static_cast<int>(j.k));
    lds = lds && j.k <= kPermLdsK && j.k % 8 == 0 && reinterpret_cast<uintptr_t>(j.x) % 16 == 0 &&
          reinterpret_cast<uintptr_t>(j.perm) % 16 == 0 && reinterpret_cast<uintptr_t>(j.f) % 16 == 0 &&
          reinterpret_cast<uintptr_t>(j.out) % 16 == 0;
  }
  a.m = m;
  a.bf16 = bf16 ? 1 : 0;
  if (lds) {
    hipLaunchKernelGGL(shuffle_rows_lds_kernel, dim3(static_cast<unsigned>(m), static_cast<unsigned>(count)),
                       dim3(256), static_cast<size_t>(kmax) * 2, st, a);
  } else {
    const int64_t n_el = static_cast<int64_t>(m) * kmax;
    hipLaunchKernelGGL(shuffle_elems_kernel, dim3(static_cast<unsigned>((n_el + 255) / 256), static_cast<unsigned>(count)),
                       dim3(256), 0, st, a);
  }
}

}  // namespace polyq

using namespace polyq;

namespace {
polyq_status pack_impl(const polyq_layout* layout, const uint16_t* codes, const uint16_t* scales,
                       const uint16_t* zeros, const int32_t* row_perm, void* packed, void* stream) {
  if (!layout_is_valid(layout)) return POLYQ_ERR_ARG;
  const polyq_layout& L = *layout;
  if (codes == nullptr || packed == nullptr) return POLYQ_ERR_ARG;
  if (L.n_groups > 0 && (scales == nullptr || zeros == nullptr)) return POLYQ_ERR_ARG;
  if (reinterpret_cast<uintptr_t>(packed) % 256 != 0 || reinterpret_cast<uintptr_t>(codes) % 16 != 0)
    return POLYQ_ERR_ARG;
  hipStream_t st = static_cast<hipStream_t>(stream);
  uint8_t* base = static_cast<uint8_t*>(packed);
  const int rows_total = L.n_tiles * kTileRows;
  for (int i = 0; i < L.nblocks; ++i) {
    uint8_t* region = base + L.block_offset[i];
    switch (L.block[i].bits) {
      case 2: launch_pack<2>(L, i, codes, row_perm, region, st); break;
      case 3: launch_pack<3>(L, i, codes, row_perm, region, st); break;
      case 4: launch_pack<4>(L, i, codes, row_perm, region, st); break;
      case 8: launch_pack<8>(L, i, codes, row_perm, region, st); break;
      case 16: launch_pack<16>(L, i, codes, row_perm, region, st); break;
      default: return POLYQ_ERR_BITS;
    }
    if (L.block[i].bits <= 8) {
      const int ng = (L.block[i].len + kGroup - 1) / kGroup;
      hipLaunchKernelGGL(pack_meta_kernel, dim3(grid_for(static_cast<int64_t>(rows_total) * ng)),
                         dim3(kThreads), 0, st, scales, zeros, row_perm, L.n, L.n_groups, L.group_begin[i],
                         ng, L.tile_bytes[i], L.record_bytes[i], rows_total, region);
    }
  }
  return hipGetLastError() == hipSuccess ? POLYQ_OK : POLYQ_ERR_DEVICE;
}

}  // namespace

extern "C" polyq_status polyq_pack(const polyq_layout* layout, const uint16_t* codes,
                                   const uint16_t* scales, const uint16_t* zeros, void* packed,
                                   void* stream) {
  return pack_impl(layout, codes, scales, zeros, nullptr, packed, stream);
}

extern "C" polyq_status polyq_pack_rows(const polyq_layout* layout, const uint16_t* codes,
                                        const uint16_t* scales, const uint16_t* zeros,
                                        const int32_t* row_perm, void* packed, void* stream) {
  if (row_perm == nullptr) return POLYQ_ERR_ARG;
  return pack_impl(layout, codes, scales, zeros, row_perm, packed, stream);
}

extern "C" polyq_status polyq_unpack(const polyq_layout* layout, const void* packed,
                                     uint16_t* codes, uint16_t* scales, uint16_t* zeros,
                                     void* stream) {
  if (!layout_is_valid(layout)) return POLYQ_ERR_ARG;
  const polyq_layout& L = *layout;
  if (packed == nullptr || reinterpret_cast<uintptr_t>(packed) % 256 != 0) return POLYQ_ERR_ARG;
  if (codes != nullptr && reinterpret_cast<uintptr_t>(codes) % 16 != 0) return POLYQ_ERR_ARG;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const uint8_t* base = static_cast<const uint8_t*>(packed);
  for (int i = 0; i < L.nblocks; ++i) {
    const uint8_t* region = base + L.block_offset[i];
    if (codes != nullptr) {
      switch (L.block[i].bits) {
        case 2: launch_unpack<2>(L, i, region, codes, st); break;
        case 3: launch_unpack<3>(L, i, region, codes, st); break;
        case 4: launch_unpack<4>(L, i, region, codes, st); break;
        case 8: launch_unpack<8>(L, i, region, codes, st); break;
        case 16: launch_unpack<16>(L, i, region, codes, st); break;
        default: return POLYQ_ERR_BITS;
      }
    }
    if (L.block[i].bits <= 8 && (scales != nullptr || zeros != nullptr)) {
      const int ng = (L.block[i].len + kGroup - 1) / kGroup;
      hipLaunchKernelGGL(unpack_meta_kernel, dim3(grid_for(static_cast<int64_t>(L.n) * ng)),
                         dim3(kThreads), 0, st, region, L.n, L.n_groups, L.group_begin[i], ng,
                         L.tile_bytes[i], L.record_bytes[i], scales, zeros);
    }
  }
  return hipGetLastError() == hipSuccess ? POLYQ_OK : POLYQ_ERR_DEVICE;
}

extern "C" polyq_status polyq_permute(const int32_t* perm, const uint16_t* x, uint16_t* x_out,
                                      int32_t m, int32_t k, void* stream) {
  if (perm == nullptr || x == nullptr || x_out == nullptr) return POLYQ_ERR_ARG;
  if (m < 1 || k < 1 || k > POLYQ_MAX_K) return POLYQ_ERR_ARG;
  // one thread per element: the grid's thread count must stay below 2^32
  if (static_cast<int64_t>(m) * k > kMaxPermuteElems) return POLYQ_ERR_CAPACITY;
  hipLaunchKernelGGL(permute_kernel, dim3(grid_for(static_cast<int64_t>(m) * k)), dim3(kThreads), 0,
                     static_cast<hipStream_t>(stream), perm, x, x_out, m, k);
  return hipGetLastError() == hipSuccess ? POLYQ_OK : POLYQ_ERR_DEVICE;
}
