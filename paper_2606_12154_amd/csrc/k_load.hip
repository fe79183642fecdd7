// Load-time weight preparation kernels: widen bf16 norm gains to fp32, find
// the largest |w| of the bf16 matrices, repack them to fp16 times 2^s for
// the MFMA path, and quantize them to the 4-bit group format.  A bf16 value v with |v| * 2^s <= 2^14 converts exactly to
// fp16 whenever |v| * 2^s >= 2^-24 (fp16 subnormals are multiples of 2^-24 and
// a bf16 value carries 8 significant bits), so the repack is exact for every
// weight except magnitudes below 2^-(24 + s - 7).
#include "hh_kernels.h"

namespace hh {

__global__ void k_widen_bf16(const __bf16* __restrict__ src, float* __restrict__ dst, size_t n) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    dst[i] = (float)src[i];
}

__global__ void k_absmax_bf16(const __bf16* __restrict__ src, size_t n, unsigned int* __restrict__ out) {
  float mx = 0.f;
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    mx = fmaxf(mx, fabsf((float)src[i]));
  mx = wave_max(mx);
  // Non-negative floats order like their bit patterns.
  if ((threadIdx.x & 63) == 0) atomicMax(out, __float_as_uint(mx));
}

__global__ void k_bf16_to_f16_scaled(const __bf16* __restrict__ src, _Float16* __restrict__ dst, size_t n,
                                     float scale) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    dst[i] = (_Float16)((float)src[i] * scale);
}

// dst[c][r] = src[r][c] for a rows x cols matrix, through 32 x 32 LDS tiles.
template <typename T>
__global__ __launch_bounds__(256) void k_transpose(const T* __restrict__ src, T* __restrict__ dst, int rows, int cols) {
  __shared__ T tile[32][33];
  const int c0 = blockIdx.x * 32, r0 = blockIdx.y * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  for (int i = ty; i < 32; i += 8) {
    const int r = r0 + i, c = c0 + tx;
    if (r < rows && c < cols) tile[i][tx] = src[(size_t)r * cols + c];
  }
  __syncthreads();
  for (int i = ty; i < 32; i += 8) {
    const int c = c0 + i, r = r0 + tx;
    if (c < cols && r < rows) dst[(size_t)c * rows + r] = tile[tx][i];
  }
}

static int grid_for(size_t n) {
  const size_t b = (n + 255) / 256;
  return (int)(b < 4096 ? (b > 0 ? b : 1) : 4096);
}

void widen_bf16(hipStream_t st, const __bf16* src, float* dst, size_t n) {
  k_widen_bf16<<<grid_for(n), 256, 0, st>>>(src, dst, n);
}
void absmax_bf16(hipStream_t st, const __bf16* src, size_t n, unsigned int* out_bits) {
  k_absmax_bf16<<<grid_for(n), 256, 0, st>>>(src, n, out_bits);
}
void bf16_to_f16_scaled(hipStream_t st, const __bf16* src, _Float16* dst, size_t n, float scale) {
  k_bf16_to_f16_scaled<<<grid_for(n), 256, 0, st>>>(src, dst, n, scale);
}

template <typename T>
void transpose(hipStream_t st, const T* src, T* dst, int rows, int cols) {
  dim3 grid((cols + 31) / 32, (rows + 31) / 32);
  k_transpose<T><<<grid, 256, 0, st>>>(src, dst, rows, cols);
}
// Operand tiles for the 32-row GEMM: dst[(rb * (K / 32) + kb) * 64 + l] (16
// bytes each) = row 16 rb + l % 16, columns 32 kb + 8 (l / 16) .. + 8 of the
// logical matrix, whose row n is source row n (interleave_f == 0) or, for
// the gate/up matrix in groups of 32 gate + 32 up rows, row j or F + j with
// j = 32 (n / 64) + n % 32 (interleave_f == F); rows past the matrix are zero.
__global__ void k_tile16(const _Float16* __restrict__ src, _Float16* __restrict__ dst, int rows, int K, int interleave_f,
                         size_t n_chunks) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n_chunks) return;
  const int l = (int)(i & 63);
  const size_t t = i >> 6;
  const int nkb = K / 32;
  const int kb = (int)(t % nkb), rb = (int)(t / nkb);
  const int n = 16 * rb + (l & 15), k = 32 * kb + 8 * (l >> 4);
  int row = n;
  if (interleave_f > 0) {
    const int c = n & 63, j = (n >> 6) * 32 + (c & 31);
    row = j < interleave_f ? (c < 32 ? j : interleave_f + j) : -1;
  }
  u32x4 v = {0u, 0u, 0u, 0u};
  if (row >= 0 && row < rows) v = *reinterpret_cast<const u32x4*>(src + (size_t)row * K + k);
  reinterpret_cast<u32x4*>(dst)[i] = v;
}

void tile16(hipStream_t st, const _Float16* src, _Float16* dst, int rows, int K, int logical_rows, int interleave_f) {
  const size_t n_chunks = (size_t)((logical_rows + 15) / 16) * 16 * K / 8;
  k_tile16<<<(unsigned)((n_chunks + 255) / 256), 256, 0, st>>>(src, dst, rows, K, interleave_f, n_chunks);
}

// The 4-bit group format: one thread per group of 32 consecutive elements of
// a row.  Scale s = bf16(max|w| / 7), codes q = clamp(rint(w / s), -8, 7)
// (fp32 divisions, both roundings to nearest even; s = 0 gives q = 0).  q4
// (optional) receives the stored row: nibbles n = q + 8 (even element low),
// then the row's scales as bf16; deq (optional) receives q * s * scale as fp16
// -- exact, a 4-bit code times an 8-bit significand, for |q s| scale in the
// fp16 normal range.  deq may be src (each thread reads its whole group before
// writing it), so neither is declared restrict.
__global__ void k_q4g32(const __bf16* src, size_t n_groups, int K, unsigned char* __restrict__ q4, _Float16* deq,
                        float scale) {
  const size_t gi = blockIdx.x * (size_t)blockDim.x + threadIdx.x;
  if (gi >= n_groups) return;
  const int gpr = K / 32;
  const size_t row = gi / gpr;
  const int g = (int)(gi % gpr);
  const size_t e0 = row * (size_t)K + 32 * (size_t)g;
  float v[32];
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const u32x4 t = *reinterpret_cast<const u32x4*>(src + e0 + 8 * c);
    float f[8];
    widen16(t, f, __bf16());
#pragma unroll
    for (int i = 0; i < 8; ++i) v[8 * c + i] = f[i];
  }
  float a = 0.f;
#pragma unroll
  for (int i = 0; i < 32; ++i) a = fmaxf(a, fabsf(v[i]));
  const __bf16 sb = (__bf16)(a / 7.0f);
  const float sf = (float)sb;
  unsigned nib[4] = {0u, 0u, 0u, 0u};
  _Float16 dq[32];
#pragma unroll
  for (int i = 0; i < 32; ++i) {
    const float r = sf > 0.f ? v[i] / sf : 0.f;
    const int q = min(7, max(-8, (int)rintf(r)));
    nib[i >> 3] |= (unsigned)(q + 8) << (4 * (i & 7));
    dq[i] = (_Float16)((float)q * sf * scale);
  }
  if (q4) {
    unsigned char* rb = q4 + row * (size_t)(K / 2 + K / 16);
    *reinterpret_cast<u32x4*>(rb + 16 * g) = u32x4{nib[0], nib[1], nib[2], nib[3]};
    *reinterpret_cast<__bf16*>(rb + K / 2 + 2 * g) = sb;
  }
  if (deq) {
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      typedef _Float16 f16x8l __attribute__((ext_vector_type(8)));
      f16x8l o;
#pragma unroll
      for (int i = 0; i < 8; ++i) o[i] = dq[8 * c + i];
      *reinterpret_cast<f16x8l*>(deq + e0 + 8 * c) = o;
    }
  }
}

void q4g32(hipStream_t st, const __bf16* src, size_t rows, int K, unsigned char* q4, _Float16* deq, float scale) {
  const size_t n = rows * (size_t)(K / 32);
  k_q4g32<<<(unsigned)((n + 255) / 256), 256, 0, st>>>(src, n, K, q4, deq, scale);
}

template void transpose<__bf16>(hipStream_t, const __bf16*, __bf16*, int, int);
template void transpose<float>(hipStream_t, const float*, float*, int, int);
template void transpose<_Float16>(hipStream_t, const _Float16*, _Float16*, int, int);

// ---------------------------------------------------------------- read probe

// Streams n 16-byte vectors once (non-temporal loads, eight in flight per
// thread, 32768 workgroups: the fastest of the shapes tried) and folds them
// into a value that is stored only if it matches a constant, so the loads
// cannot be dropped.
__device__ unsigned g_probe_sink;

__global__ __launch_bounds__(256) void k_read_probe(const u32x4* __restrict__ p, size_t n) {
  constexpr int U = 8;
  const size_t stride = (size_t)gridDim.x * 256;
  size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  unsigned acc = 0;
  for (; i + (U - 1) * stride < n; i += U * stride) {
    u32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = __builtin_nontemporal_load(p + i + u * stride);
#pragma unroll
    for (int u = 0; u < U; ++u) acc ^= v[u].x + v[u].y + v[u].z + v[u].w;
  }
  for (; i < n; i += stride) {
    const u32x4 a = __builtin_nontemporal_load(p + i);
    acc ^= a.x + a.y + a.z + a.w;
  }
  if (acc == 0x9E3779B9u) g_probe_sink = acc;
}

void read_probe(hipStream_t st, const void* src, size_t bytes) {
  const size_t n = bytes / 16;
  k_read_probe<<<32768, 256, 0, st>>>(reinterpret_cast<const u32x4*>(src), n);
}

}  // namespace hh
