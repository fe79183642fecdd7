// Load-time weight preparation kernels: widen bf16 norm gains to fp32, find
// the largest |w| of the bf16 matrices, and repack them to fp16 times 2^s for
// the MFMA path.  A bf16 value v with |v| * 2^s <= 2^14 converts exactly to
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

template void transpose<__bf16>(hipStream_t, const __bf16*, __bf16*, int, int);
template void transpose<float>(hipStream_t, const float*, float*, int, int);
template void transpose<_Float16>(hipStream_t, const _Float16*, _Float16*, int, int);

}  // namespace hh
