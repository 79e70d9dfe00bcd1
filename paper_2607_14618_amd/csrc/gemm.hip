// Prefill GEMM over the mixed-bit clustered weight (Sec. 4.1-4.2), M tokens:
//   y[m][n] = sum_k' w_hat[n][k'] x'[m][k'],  x' = x[:, perm] (Eq. 9)
//
// Prefill is a dense contraction, so it runs on the bf16 matrix cores
// (v_mfma_f32_16x16x32_bf16, fp32 accumulation).  Each work-group owns a
// 128-token x 64-row output tile (one packed tile); per 32-channel chunk the
// work-group dequantizes the chunk of its 64 rows into LDS and its four waves
// multiply it with their 32 tokens each.  Group-fold numerics: the dequantized
// operand is (q - z), an integer of magnitude <= 255 that bf16 holds exactly;
// each 128-channel group accumulates into its own fp32 tile, which is then
// scaled by the row's fp16 scale s and added to the output accumulator.  A
// 16-bit channel enters as the exact pair hi + lo of bf16 values of its fp16
// weight (two MFMAs), so every product is exact before fp32 accumulation.
#include <hip/hip_runtime.h>

#include "codec.h"
#include "internal.h"

namespace polyq {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kBM = 128;          // tokens per work-group
constexpr int kBN = kTileRows;    // rows per work-group (one packed tile)
constexpr int kWaves = 4;         // each wave: 32 tokens x 64 rows
constexpr int kLdsRow = 40;       // bf16 per LDS row (32 + 8 pad against bank conflicts)

struct GemmArgs {
  const uint8_t* packed;
  const uint16_t* x;  // bf16 [m][k], clustered order
  float* y;           // fp32 [m][n]
  int32_t n, k, m, nblocks;
  int32_t bits[POLYQ_MAX_BLOCKS];
  int32_t chunk_begin[POLYQ_MAX_BLOCKS];
  int32_t chunk_end[POLYQ_MAX_BLOCKS];
  int64_t block_offset[POLYQ_MAX_BLOCKS];
  int64_t tile_bytes[POLYQ_MAX_BLOCKS];
  int64_t record_bytes[POLYQ_MAX_BLOCKS];
};

// fp32 -> bf16 bits, round to nearest even (inputs here are finite).
__device__ __forceinline__ uint32_t bf16_bits(float f) {
  const uint32_t u = __builtin_bit_cast(uint32_t, f);
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}
__device__ __forceinline__ float bf16_value(uint32_t b) { return __builtin_bit_cast(float, b << 16); }
__device__ __forceinline__ uint32_t pack2(uint32_t lo, uint32_t hi) { return lo | (hi << 16); }

// Thread (row R, quarter j) dequantizes channels 8j .. 8j+7 of tile row R of one
// chunk into bf16 (q - z) in LDS row R, columns 8j .. 8j+7.  They sit in lane
// slice 16j + R%16, row sub-tile R/16 (slice codes 8(R/16) .. +7).
template <int B>
__device__ __forceinline__ void dequant_chunk(const uint8_t* chunk, int R, int j, float z,
                                              uint16_t* lds_b) {
  uint32_t w[B];
  const uint32_t* src = reinterpret_cast<const uint32_t*>(chunk + (16 * j + (R & 15)) * 4 * B);
#pragma unroll
  for (int d = 0; d < B; ++d) w[d] = src[d];
  const int r = R >> 4;
  uint32_t out[4];
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    const float a = static_cast<float>(slice_code<B>(w, slice_index(r, 2 * p))) - z;
    const float b = static_cast<float>(slice_code<B>(w, slice_index(r, 2 * p + 1))) - z;
    out[p] = pack2(bf16_bits(a), bf16_bits(b));
  }
  *reinterpret_cast<uint4*>(lds_b + R * kLdsRow + 8 * j) = uint4{out[0], out[1], out[2], out[3]};
}

// 16-bit chunk: hi = bf16(w), lo = bf16(w - hi) (exact), into two LDS tiles.
__device__ __forceinline__ void split_fp16_chunk(const uint8_t* chunk, int R, int j,
                                                 uint16_t* lds_hi, uint16_t* lds_lo) {
  const uint4 u = *reinterpret_cast<const uint4*>(chunk + (16 * j + (R & 15)) * 64 + 16 * (R >> 4));
  const uint32_t wd[4] = {u.x, u.y, u.z, u.w};
  uint32_t hi[4], lo[4];
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    uint32_t h2[2], l2[2];
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const uint16_t bits = static_cast<uint16_t>(e == 0 ? (wd[p] & 0xFFFFu) : (wd[p] >> 16));
      const float v = static_cast<float>(__builtin_bit_cast(_Float16, bits));
      h2[e] = bf16_bits(v);
      l2[e] = bf16_bits(v - bf16_value(h2[e]));
    }
    hi[p] = pack2(h2[0], h2[1]);
    lo[p] = pack2(l2[0], l2[1]);
  }
  *reinterpret_cast<uint4*>(lds_hi + R * kLdsRow + 8 * j) = uint4{hi[0], hi[1], hi[2], hi[3]};
  *reinterpret_cast<uint4*>(lds_lo + R * kLdsRow + 8 * j) = uint4{lo[0], lo[1], lo[2], lo[3]};
}

__device__ __forceinline__ bf16x8 load_frag(const uint16_t* p) {
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(p));
}

__global__ __launch_bounds__(kWaves * 64) void gemm_kernel(const GemmArgs a) {
  __shared__ uint16_t lds_b[2][kBN * kLdsRow];  // [0]: (q - z) or hi, [1]: lo
  __shared__ float lds_s[kBN];

  const int mt = blockIdx.x, tile = blockIdx.y;
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int dq_row = tid & 63, dq_q = wave;  // dequant assignment: row, quarter of the chunk
  const int m_wave = mt * kBM + wave * 32;   // first token of this wave

  floatx4 total[2][4], part[2][4];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int jn = 0; jn < 4; ++jn) total[i][jn] = floatx4{0.f, 0.f, 0.f, 0.f};

  // A fragment source rows (tokens) of this lane; rows >= m read as zero
  const int arow0 = m_wave + (lane & 15), arow1 = arow0 + 16;
  const int acol = 8 * (lane >> 4);

  for (int bi = 0; bi < a.nblocks; ++bi) {
    const int B = a.bits[bi];
    const int cb0 = a.chunk_begin[bi], nch = a.chunk_end[bi] - cb0;
    const uint8_t* tile_base = a.packed + a.block_offset[bi] + tile * a.tile_bytes[bi];
    const int meta = B <= 8 ? kMetaBytes : 0;
    for (int g = 0; g * 4 < nch; ++g) {
      const uint8_t* rec = tile_base + g * a.record_bytes[bi];
      float z = 0.f;
      if (B <= 8)
        z = static_cast<float>(reinterpret_cast<const _Float16*>(rec)[meta_z_half(dq_row)]);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int jn = 0; jn < 4; ++jn) part[i][jn] = floatx4{0.f, 0.f, 0.f, 0.f};
      const int cend = min(nch, 4 * g + 4);
      for (int c = 4 * g; c < cend; ++c) {
        __syncthreads();  // the previous chunk's LDS tile is consumed
        const uint8_t* chunk_rows = rec + meta + (c & 3) * (64 * 4 * B);
        switch (B) {
          case 2: dequant_chunk<2>(chunk_rows, dq_row, dq_q, z, lds_b[0]); break;
          case 3: dequant_chunk<3>(chunk_rows, dq_row, dq_q, z, lds_b[0]); break;
          case 4: dequant_chunk<4>(chunk_rows, dq_row, dq_q, z, lds_b[0]); break;
          case 8: dequant_chunk<8>(chunk_rows, dq_row, dq_q, z, lds_b[0]); break;
          default: split_fp16_chunk(chunk_rows, dq_row, dq_q, lds_b[0], lds_b[1]); break;
        }
        if (B <= 8 && c == 4 * g && tid < kBN)
          lds_s[tid] = static_cast<float>(reinterpret_cast<const _Float16*>(rec)[meta_s_half(tid)]);
        __syncthreads();
        const int kc = (cb0 + c) * kChunk + acol;
        bf16x8 afr[2];
        afr[0] = arow0 < a.m ? load_frag(a.x + static_cast<int64_t>(arow0) * a.k + kc)
                             : __builtin_bit_cast(bf16x8, uint4{0, 0, 0, 0});
        afr[1] = arow1 < a.m ? load_frag(a.x + static_cast<int64_t>(arow1) * a.k + kc)
                             : __builtin_bit_cast(bf16x8, uint4{0, 0, 0, 0});
#pragma unroll
        for (int jn = 0; jn < 4; ++jn) {
          const bf16x8 bfr = load_frag(lds_b[0] + (jn * 16 + (lane & 15)) * kLdsRow + acol);
#pragma unroll
          for (int i = 0; i < 2; ++i)
            part[i][jn] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(afr[i], bfr, part[i][jn], 0, 0, 0);
        }
        if (B == 16) {
#pragma unroll
          for (int jn = 0; jn < 4; ++jn) {
            const bf16x8 bfr = load_frag(lds_b[1] + (jn * 16 + (lane & 15)) * kLdsRow + acol);
#pragma unroll
            for (int i = 0; i < 2; ++i)
              part[i][jn] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(afr[i], bfr, part[i][jn], 0, 0, 0);
          }
        }
      }
      // group fold: total += s[n] * part (16-bit channels: scale 1)
#pragma unroll
      for (int jn = 0; jn < 4; ++jn) {
        const float s = B <= 8 ? lds_s[jn * 16 + (lane & 15)] : 1.f;
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int e = 0; e < 4; ++e) total[i][jn][e] = fmaf(s, part[i][jn][e], total[i][jn][e]);
      }
    }
  }
  // D layout: lane holds rows 4*(lane/16)+e of the 16x16 tile, column lane%16
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int jn = 0; jn < 4; ++jn) {
      const int col = tile * kBN + jn * 16 + (lane & 15);
      if (col >= a.n) continue;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int row = m_wave + i * 16 + 4 * (lane >> 4) + e;
        if (row < a.m) a.y[static_cast<int64_t>(row) * a.n + col] = total[i][jn][e];
      }
    }
}

__global__ __launch_bounds__(256) void permute_rows_kernel(const int32_t* __restrict__ perm,
                                                           const uint16_t* __restrict__ x,
                                                           uint16_t* __restrict__ out, int m, int k) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (idx >= static_cast<int64_t>(m) * k) return;
  const int i = static_cast<int>(idx / k), kp = static_cast<int>(idx % k);
  const int p = perm[kp];
  out[idx] = static_cast<unsigned>(p) < static_cast<unsigned>(k) ? x[static_cast<int64_t>(i) * k + p] : 0;
}

}  // namespace
}  // namespace polyq

using namespace polyq;

extern "C" size_t polyq_gemm_workspace_bytes(const polyq_layout* layout, int32_t m, int perm_given) {
  if (!layout_is_valid(layout) || m < 1) return 0;
  if (!perm_given) return 0;
  return static_cast<size_t>(align_up(static_cast<int64_t>(m) * layout->k * 2, 256));
}

extern "C" polyq_status polyq_gemm(const polyq_layout* layout, const void* packed,
                                   const int32_t* perm, const uint16_t* x, int32_t m, float* y,
                                   void* workspace, size_t workspace_bytes, void* stream) {
  if (!layout_is_valid(layout)) return POLYQ_ERR_ARG;
  const polyq_layout& L = *layout;
  if (packed == nullptr || x == nullptr || y == nullptr || m < 1) return POLYQ_ERR_ARG;
  if (reinterpret_cast<uintptr_t>(packed) % 256 != 0 || reinterpret_cast<uintptr_t>(y) % 4 != 0)
    return POLYQ_ERR_ARG;
  if (static_cast<int64_t>(m) * L.k > (static_cast<int64_t>(1) << 40)) return POLYQ_ERR_CAPACITY;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const uint16_t* xp = x;
  if (perm != nullptr) {
    const size_t need = polyq_gemm_workspace_bytes(layout, m, 1);
    if (workspace == nullptr || workspace_bytes < need) return POLYQ_ERR_CAPACITY;
    if (reinterpret_cast<uintptr_t>(workspace) % 16 != 0) return POLYQ_ERR_ARG;
    const int64_t items = static_cast<int64_t>(m) * L.k;
    hipLaunchKernelGGL(permute_rows_kernel, dim3(static_cast<unsigned>((items + 255) / 256)),
                       dim3(256), 0, st, perm, x, static_cast<uint16_t*>(workspace), m, L.k);
    xp = static_cast<const uint16_t*>(workspace);
  } else if (reinterpret_cast<uintptr_t>(x) % 16 != 0) {
    return POLYQ_ERR_ARG;  // fragments are read as 16-byte vectors
  }
  GemmArgs a;
  a.packed = static_cast<const uint8_t*>(packed);
  a.x = xp;
  a.y = y;
  a.n = L.n;
  a.k = L.k;
  a.m = m;
  a.nblocks = L.nblocks;
  for (int i = 0; i < POLYQ_MAX_BLOCKS; ++i) {
    const bool used = i < L.nblocks;
    a.bits[i] = used ? L.block[i].bits : 0;
    a.chunk_begin[i] = used ? L.k_begin[i] / kChunk : 0;
    a.chunk_end[i] = used ? (L.k_begin[i] + L.block[i].len) / kChunk : 0;
    a.block_offset[i] = used ? L.block_offset[i] : 0;
    a.tile_bytes[i] = used ? L.tile_bytes[i] : 0;
    a.record_bytes[i] = used ? L.record_bytes[i] : 0;
  }
  const dim3 grid((m + kBM - 1) / kBM, L.n_tiles);
  hipLaunchKernelGGL(gemm_kernel, grid, dim3(kWaves * 64), 0, st, a);
  return hipGetLastError() == hipSuccess ? POLYQ_OK : POLYQ_ERR_DEVICE;
}
