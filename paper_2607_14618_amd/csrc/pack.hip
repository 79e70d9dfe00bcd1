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

// x'[i][j] = x[i][perm[j]] for one token row per work-group: the row is staged
// in LDS with 16-byte loads, then gathered there and written with 16-byte
// stores (k <= kPermLdsK, rows 16-byte aligned).
constexpr int kPermLdsK = 32768;
constexpr int kPermLdsMinRows = 64;

__global__ __launch_bounds__(256) void permute_rows_lds_kernel(const int32_t* __restrict__ perm,
                                                               const uint16_t* __restrict__ x,
                                                               uint16_t* __restrict__ out, int k) {
  extern __shared__ uint4 row4[];
  const uint16_t* row = reinterpret_cast<const uint16_t*>(row4);
  const int64_t base = static_cast<int64_t>(blockIdx.x) * k;
  const uint4* src = reinterpret_cast<const uint4*>(x + base);
  const int4* p4 = reinterpret_cast<const int4*>(perm);
  // The indices of the first kPre passes are loaded together with the row (one
  // memory round trip for both).
  constexpr int kPre = 4;
  int4 pp[kPre][2];
#pragma unroll
  for (int u = 0; u < kPre; ++u) {
    const int j = threadIdx.x + u * 256;
    if (j < k / 8) {
      pp[u][0] = p4[2 * j];
      pp[u][1] = p4[2 * j + 1];
    }
  }
  for (int j = threadIdx.x; j < k / 8; j += 256) row4[j] = src[j];
  __syncthreads();
  uint4* dst = reinterpret_cast<uint4*>(out + base);
  auto gather = [&](int j, int4 p0, int4 p1) {
    const int p[8] = {p0.x, p0.y, p0.z, p0.w, p1.x, p1.y, p1.z, p1.w};
    uint32_t h[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) h[e] = static_cast<unsigned>(p[e]) < static_cast<unsigned>(k) ? row[p[e]] : 0u;
    dst[j] = uint4{h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16)};
  };
#pragma unroll
  for (int u = 0; u < kPre; ++u) {
    const int j = threadIdx.x + u * 256;
    if (j < k / 8) gather(j, pp[u][0], pp[u][1]);
  }
  for (int j = threadIdx.x + kPre * 256; j < k / 8; j += 256) gather(j, p4[2 * j], p4[2 * j + 1]);
}

// Fallback gather, one element per thread (any k, any alignment).
__global__ __launch_bounds__(256) void permute_rows_kernel(const int32_t* __restrict__ perm,
                                                           const uint16_t* __restrict__ x,
                                                           uint16_t* __restrict__ out, int m, int k) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (idx >= static_cast<int64_t>(m) * k) return;
  const int i = static_cast<int>(idx / k), kp = static_cast<int>(idx % k);
  const int p = perm[kp];
  out[idx] = static_cast<unsigned>(p) < static_cast<unsigned>(k) ? x[static_cast<int64_t>(i) * k + p] : 0;
}

// x'[i][j] = x[i][perm[j]] * f[j] (perm NULL: the identity), f the fp16
// channel factors of Eq. 8 (1/s_j).  The product is formed in fp32 and
// rounded to the activation type (fp16, or bf16 when `bf16`), nearest even:
// exact for a power-of-two factor.  One thread per E channels of a row (E = 8
// for many rows, 1 for a few decode tokens, so that the grid fills the chip).
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

template <int E>
__global__ __launch_bounds__(256) void scale_rows_kernel(const int32_t* __restrict__ perm,
                                                         const uint16_t* __restrict__ f,
                                                         const uint16_t* __restrict__ x,
                                                         uint16_t* __restrict__ out, int m, int k, int bf16) {
  const int kp = (k + E - 1) / E;  // pieces per row
  const int64_t t = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (t >= static_cast<int64_t>(m) * kp) return;
  const int i = static_cast<int>(t / kp), j0 = static_cast<int>(t % kp) * E;
  const uint16_t* row = x + static_cast<int64_t>(i) * k;
  uint16_t* dst = out + static_cast<int64_t>(i) * k;
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int j = j0 + e;
    if (j < k) {
      const int src = perm != nullptr ? perm[j] : j;
      const float v = static_cast<unsigned>(src) < static_cast<unsigned>(k) ? act_to_f32(row[src], bf16 != 0) : 0.f;
      const float fj = static_cast<float>(__builtin_bit_cast(_Float16, f[j]));
      dst[j] = f32_to_act(v * fj, bf16 != 0);
    }
  }
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

void launch_permute_rows(const int32_t* perm, const uint16_t* x, uint16_t* out, int32_t m, int32_t k,
                         hipStream_t st) {
  // one work-group per row only when there are enough rows to fill the chip;
  // a few decode tokens spread one element per thread over the whole chip
  if (m >= kPermLdsMinRows && k <= kPermLdsK && k % 8 == 0 && reinterpret_cast<uintptr_t>(x) % 16 == 0 &&
      reinterpret_cast<uintptr_t>(perm) % 16 == 0 && reinterpret_cast<uintptr_t>(out) % 16 == 0) {
    hipLaunchKernelGGL(permute_rows_lds_kernel, dim3(static_cast<unsigned>(m)), dim3(256),
                       static_cast<size_t>(k) * 2, st, perm, x, out, k);
  } else {
    const int64_t n_el = static_cast<int64_t>(m) * k;
    hipLaunchKernelGGL(permute_rows_kernel, dim3(static_cast<unsigned>((n_el + 255) / 256)), dim3(256), 0,
                       st, perm, x, out, m, k);
  }
}

// The same for many rows: one token row per work-group, staged in LDS with
// 16-byte loads (k <= kPermLdsK, k % 8 == 0, 16-byte aligned rows, factors and
// permutation), then 8 channels per thread: the permutation and factors as
// 16-byte loads, one 16-byte store.
template <bool HasPerm>
__global__ __launch_bounds__(256) void scale_rows_lds_kernel(const int32_t* __restrict__ perm,
                                                             const uint16_t* __restrict__ f,
                                                             const uint16_t* __restrict__ x,
                                                             uint16_t* __restrict__ out, int k, int bf16) {
  extern __shared__ uint4 row4[];
  const uint16_t* row = reinterpret_cast<const uint16_t*>(row4);
  const int64_t base = static_cast<int64_t>(blockIdx.x) * k;
  const uint4* src = reinterpret_cast<const uint4*>(x + base);
  for (int j = threadIdx.x; j < k / 8; j += 256) row4[j] = src[j];
  __syncthreads();
  const int4* p4 = reinterpret_cast<const int4*>(perm);
  const uint4* f4 = reinterpret_cast<const uint4*>(f);
  uint4* dst = reinterpret_cast<uint4*>(out + base);
  for (int j = threadIdx.x; j < k / 8; j += 256) {
    int p[8];
    if constexpr (HasPerm) {
      const int4 a = p4[2 * j], b = p4[2 * j + 1];
      p[0] = a.x; p[1] = a.y; p[2] = a.z; p[3] = a.w; p[4] = b.x; p[5] = b.y; p[6] = b.z; p[7] = b.w;
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) p[e] = 8 * j + e;
    }
    const uint4 fv = f4[j];
    const uint32_t fw[4] = {fv.x, fv.y, fv.z, fv.w};
    uint32_t h[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float v = static_cast<unsigned>(p[e]) < static_cast<unsigned>(k) ? act_to_f32(row[p[e]], bf16 != 0) : 0.f;
      const float fj = static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(fw[e / 2] >> (16 * (e & 1)))));
      h[e] = f32_to_act(v * fj, bf16 != 0);
    }
    dst[j] = uint4{h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16)};
  }
}

void launch_scale_rows(const int32_t* perm, const uint16_t* f, const uint16_t* x, uint16_t* out, int32_t m,
                       int32_t k, bool bf16, hipStream_t st) {
  const bool lds = m >= kPermLdsMinRows && k <= kPermLdsK && k % 8 == 0 &&
                   reinterpret_cast<uintptr_t>(x) % 16 == 0 && reinterpret_cast<uintptr_t>(f) % 16 == 0 &&
                   reinterpret_cast<uintptr_t>(perm) % 16 == 0 && reinterpret_cast<uintptr_t>(out) % 16 == 0;
  if (lds) {
    const size_t shm = static_cast<size_t>(k) * 2;
    if (perm != nullptr)
      hipLaunchKernelGGL(scale_rows_lds_kernel<true>, dim3(static_cast<unsigned>(m)), dim3(256), shm, st, perm, f, x,
                         out, k, bf16 ? 1 : 0);
    else
      hipLaunchKernelGGL(scale_rows_lds_kernel<false>, dim3(static_cast<unsigned>(m)), dim3(256), shm, st, perm, f,
                         x, out, k, bf16 ? 1 : 0);
  } else if (m >= kPermLdsMinRows) {
    const int64_t threads = static_cast<int64_t>(m) * ((k + 7) / 8);
    hipLaunchKernelGGL(scale_rows_kernel<8>, dim3(static_cast<unsigned>((threads + 255) / 256)), dim3(256), 0, st,
                       perm, f, x, out, m, k, bf16 ? 1 : 0);
  } else {
    const int64_t threads = static_cast<int64_t>(m) * k;
    hipLaunchKernelGGL(scale_rows_kernel<1>, dim3(static_cast<unsigned>((threads + 255) / 256)), dim3(256), 0, st,
                       perm, f, x, out, m, k, bf16 ? 1 : 0);
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
