// Device-side helpers shared by the gfx950 kernels of the decoder runtime:
// 16-byte vector loads that widen bf16 / fp16 / fp32 storage to fp32,
// wave64 reductions, and the paged KV-cache addressing.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hh {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));

constexpr int kHeadDim = 64;   // head dimension the kernels are written for
constexpr int kPage = 16;      // tokens per KV page
constexpr int kWave = 64;      // CDNA wavefront width

// Elements of T in one 16-byte load.
template <typename T> struct Vec16 { static constexpr int n = 16 / sizeof(T); };

// Widen one 16-byte chunk of T to fp32 (n = 4 for float, 8 for 16-bit types).
__device__ __forceinline__ void widen16(const u32x4 v, float* f, float) {
#pragma unroll
  for (int i = 0; i < 4; ++i) f[i] = __uint_as_float(v[i]);
}
__device__ __forceinline__ void widen16(const u32x4 v, float* f, __bf16) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = __uint_as_float(v[i] << 16);
    f[2 * i + 1] = __uint_as_float(v[i] & 0xffff0000u);
  }
}
__device__ __forceinline__ void widen16(const u32x4 v, float* f, _Float16) {
  const f16x8 h = __builtin_bit_cast(f16x8, v);
#pragma unroll
  for (int i = 0; i < 8; ++i) f[i] = (float)h[i];
}

// 16-byte load widened to fp32; `stream` marks data read exactly once
// (weights), which is loaded non-temporally so it does not evict reused lines.
template <typename T, bool stream = false>
__device__ __forceinline__ void load16(const T* p, float* f) {
  u32x4 v;
  if constexpr (stream) v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  else v = *reinterpret_cast<const u32x4*>(p);
  widen16(v, f, T());
}

template <typename T> __device__ __forceinline__ T from_f32(float x) { return (T)x; }

// DPP lane moves (VALU, no LDS round trip).  CTRL: 0xB1 quad_perm [1,0,3,2]
// (partner lane ^ 1), 0x4E quad_perm [2,3,0,1] (lane ^ 2), 0x120 + n row_ror:n
// (rotate right by n within each row of 16 lanes).
template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float lane_read(float v, int lane) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), lane));
}
// Sum / max over the 16 lanes of each row (every lane of the row gets it).
__device__ __forceinline__ float row_sum16(float v) {
  v += dpp<0xB1>(v);
  v += dpp<0x4E>(v);
  v += dpp<0x124>(v);
  v += dpp<0x128>(v);
  return v;
}
__device__ __forceinline__ float row_max16(float v) {
  v = fmaxf(v, dpp<0xB1>(v));
  v = fmaxf(v, dpp<0x4E>(v));
  v = fmaxf(v, dpp<0x124>(v));
  v = fmaxf(v, dpp<0x128>(v));
  return v;
}
// Wave-wide sum / max, returned uniformly (row totals combined by readlane).
__device__ __forceinline__ float wave_sum_u(float v) {
  v = row_sum16(v);
  return (lane_read(v, 0) + lane_read(v, 16)) + (lane_read(v, 32) + lane_read(v, 48));
}
__device__ __forceinline__ float wave_max_u(float v) {
  v = row_max16(v);
  return fmaxf(fmaxf(lane_read(v, 0), lane_read(v, 16)), fmaxf(lane_read(v, 32), lane_read(v, 48)));
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}

// Sum over a 256-thread block; `red` is >= 4 floats of LDS.  All threads get it.
__device__ __forceinline__ float block_sum256(float v, float* red) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  const float s = red[0] + red[1] + red[2] + red[3];
  __syncthreads();
  return s;
}

// SiLU written from its definition z * sigmoid(z).
__device__ __forceinline__ float silu(float z) { return z / (1.0f + __expf(-z)); }

// Paged KV cache: per layer, n_pages pages of [K|V][n_kv_heads][16][64].
struct KvLayout {
  int n_pages;     // physical pages per layer
  int n_kv_heads;
  int max_pages;   // page-table columns per stream
  __device__ __forceinline__ size_t head_tile(int layer, int page, int kind, int g) const {
    return ((((size_t)layer * n_pages + page) * 2 + kind) * n_kv_heads + g) * (kPage * kHeadDim);
  }
};

// Order-preserving map of an fp32 value to uint32 (larger float -> larger int).
__device__ __forceinline__ uint32_t ordered_bits(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
// Argmax key: the larger value wins, and among equal values the lower index.
__device__ __forceinline__ unsigned long long argmax_key(float v, uint32_t idx) {
  return ((unsigned long long)ordered_bits(v) << 32) | (unsigned long long)(0xffffffffu - idx);
}
__device__ __forceinline__ int argmax_index(unsigned long long key) {
  return (int)(0xffffffffu - (uint32_t)(key & 0xffffffffull));
}

}  // namespace hh
