// MFMA GEMM for gfx950 with fused epilogues, used where the decoder's work is a
// dense contraction: prompt prefill (M = prompt rows) and lockstep multi-stream
// decode (M = streams).  C[M, N] = A[M, K] * W[N, K]^T with fp32 accumulation.
//
// Operands are of type TM: _Float16 for bf16 models (the bf16 weights are
// repacked at load time to fp16 times a power-of-two scale, exact for this
// weight range, and activations are rounded to fp16 once), float for fp32
// models (v_mfma_f32_16x16x4_f32).  A 256-thread block computes a 64x64 tile:
// four waves in a 2x2 arrangement each own a 32x32 quarter as 2x2 MFMA 16x16
// fragments; K advances in steps of 32 through LDS.  The finished tile is
// staged in LDS so the epilogue can use any column pairing (rotary pairs
// i / i + 32 of a head, gate / up columns) without shuffles.
#include "hh_kernels.h"

namespace hh {

constexpr int GBM = 64, GBN = 64, GBK = 32;
constexpr int GLDC = GBN + 4;

// ---------------------------------------------------------------- epilogues

// Columns of W for tile nt: head nt of [Wq; Wk; Wv] (64 rows).  Rotates query
// heads into q and key heads into the KV page slot of each row; copies values.
template <typename TKV>
struct EpiQKV {
  int hq, hkv;
  float scale;
  const int* row_stream;
  const int* row_pos;
  const float2* rope;
  float* q;
  TKV* kv;
  KvLayout L;
  int layer;
  const int* page_table;
  __device__ int b_row(int nt, int c) const { return nt * 64 + c; }
  __device__ void operator()(const float* Cs, int m0, int M, int nt) const {
    const int head = nt;
    for (int idx = threadIdx.x; idx < GBM * 32; idx += 256) {
      const int r = idx >> 5, i = idx & 31, row = m0 + r;
      if (row >= M) continue;
      const float y0 = Cs[r * GLDC + i] * scale, y1 = Cs[r * GLDC + i + 32] * scale;
      const int s = row_stream[row], p = row_pos[row];
      if (head < hq + hkv) {
        const float2 cs = rope[(size_t)p * 32 + i];
        const float r0 = y0 * cs.x - y1 * cs.y, r1 = y1 * cs.x + y0 * cs.y;
        if (head < hq) {
          q[((size_t)row * hq + head) * 64 + i] = r0;
          q[((size_t)row * hq + head) * 64 + i + 32] = r1;
        } else {
          const int page = page_table[(size_t)s * L.max_pages + p / kPage];
          TKV* dst = kv + L.head_tile(layer, page, 0, head - hq) + (p % kPage) * 64;
          dst[i] = (TKV)r0;
          dst[i + 32] = (TKV)r1;
        }
      } else {
        const int page = page_table[(size_t)s * L.max_pages + p / kPage];
        TKV* dst = kv + L.head_tile(layer, page, 1, head - hq - hkv) + (p % kPage) * 64;
        dst[i] = (TKV)y0;
        dst[i + 32] = (TKV)y1;
      }
    }
  }
};

// x[row, col] += C (residual add of the O and down projections).
struct EpiResid {
  int N;
  float scale;
  float* x;
  __device__ int b_row(int nt, int c) const { return nt * 64 + c < N ? nt * 64 + c : -1; }
  __device__ void operator()(const float* Cs, int m0, int M, int nt) const {
    for (int idx = threadIdx.x; idx < GBM * GBN; idx += 256) {
      const int r = idx >> 6, c = idx & 63, row = m0 + r, col = nt * 64 + c;
      if (row < M && col < N) x[(size_t)row * N + col] += Cs[r * GLDC + c] * scale;
    }
  }
};

// Tile nt covers gate columns [32nt, 32nt + 32) and the matching up columns
// (rows F + j of [Wg; Wu]); m[row, j] = silu(gate) * up.
template <typename TM>
struct EpiGateUp {
  int F;
  float scale;
  TM* m;
  __device__ int b_row(int nt, int c) const {
    const int j = nt * 32 + (c & 31);
    return j < F ? (c < 32 ? j : F + j) : -1;
  }
  __device__ void operator()(const float* Cs, int m0, int M, int nt) const {
    for (int idx = threadIdx.x; idx < GBM * 32; idx += 256) {
      const int r = idx >> 5, j = idx & 31, row = m0 + r, col = nt * 32 + j;
      if (row >= M || col >= F) continue;
      const float g = Cs[r * GLDC + j] * scale, u = Cs[r * GLDC + 32 + j] * scale;
      m[(size_t)row * F + col] = (TM)(silu(g) * u);
    }
  }
};

// LM head rows: optional fp32 logits and the per-row packed argmax into the
// row's stream slot.
struct EpiLogits {
  int V;
  float scale;
  float* logits;
  unsigned long long* slot;
  const int* row_stream;
  __device__ int b_row(int nt, int c) const { return nt * 64 + c < V ? nt * 64 + c : -1; }
  __device__ void operator()(const float* Cs, int m0, int M, int nt) const {
    if (logits)
      for (int idx = threadIdx.x; idx < GBM * GBN; idx += 256) {
        const int r = idx >> 6, c = idx & 63, row = m0 + r, col = nt * 64 + c;
        if (row < M && col < V) logits[(size_t)row * V + col] = Cs[r * GLDC + c] * scale;
      }
    if (slot && threadIdx.x < GBM && m0 + threadIdx.x < M) {
      const int r = threadIdx.x;
      unsigned long long best = 0ull;
      for (int c = 0; c < GBN && nt * 64 + c < V; ++c) {
        const unsigned long long k = argmax_key(Cs[r * GLDC + c] * scale, (uint32_t)(nt * 64 + c));
        best = k > best ? k : best;
      }
      atomicMax(slot + row_stream[m0 + r], best);
    }
  }
};

// ---------------------------------------------------------------- kernel

template <typename TM, typename Epi>
__global__ __launch_bounds__(256) void k_gemm(const TM* __restrict__ A, int M, const TM* __restrict__ W, int K,
                                              Epi epi) {
  constexpr int V = Vec16<TM>::n;  // elements per 16-byte chunk
  constexpr int CPR = GBK / V;     // chunks per tile row
  constexpr int LDK = GBK + V;     // padded LDS row (elements)
  __shared__ __attribute__((aligned(16))) TM As[GBM * LDK];
  __shared__ __attribute__((aligned(16))) TM Bs[GBN * LDK];
  __shared__ float Cs[GBM * GLDC];
  const int nt = blockIdx.x, m0 = blockIdx.y * GBM;
  const int tid = threadIdx.x, wv = tid >> 6, lane = tid & 63;
  const int wm = wv >> 1, wn = wv & 1;
  const int lr = lane & 15, lk = lane >> 4;
  f32x4 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int k0 = 0; k0 < K; k0 += GBK) {
    for (int c = tid; c < GBM * CPR; c += 256) {
      const int r = c / CPR, kc = (c % CPR) * V;
      u32x4 va = {0u, 0u, 0u, 0u}, vb = {0u, 0u, 0u, 0u};
      if (m0 + r < M && k0 + kc < K) va = *reinterpret_cast<const u32x4*>(A + (size_t)(m0 + r) * K + k0 + kc);
      const int br = epi.b_row(nt, r);
      if (br >= 0 && k0 + kc < K) vb = *reinterpret_cast<const u32x4*>(W + (size_t)br * K + k0 + kc);
      *reinterpret_cast<u32x4*>(As + r * LDK + kc) = va;
      *reinterpret_cast<u32x4*>(Bs + r * LDK + kc) = vb;
    }
    __syncthreads();
    if constexpr (sizeof(TM) == 2) {
      // 16x16x32 f16: lane supplies A[lr][8lk..8lk+8) and W[lr][8lk..8lk+8).
      f16x8 a[2], b[2];
#pragma unroll
      for (int i = 0; i < 2; ++i)
        a[i] = *reinterpret_cast<const f16x8*>(As + (wm * 32 + i * 16 + lr) * LDK + 8 * lk);
#pragma unroll
      for (int j = 0; j < 2; ++j)
        b[j] = *reinterpret_cast<const f16x8*>(Bs + (wn * 32 + j * 16 + lr) * LDK + 8 * lk);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a[i], b[j], acc[i][j], 0, 0, 0);
    } else {
      // 16x16x4 f32: lane supplies A[lr][kk + lk] and W[lr][kk + lk].
#pragma unroll
      for (int kk = 0; kk < GBK; kk += 4) {
        float a[2], b[2];
#pragma unroll
        for (int i = 0; i < 2; ++i) a[i] = As[(wm * 32 + i * 16 + lr) * LDK + kk + lk];
#pragma unroll
        for (int j = 0; j < 2; ++j) b[j] = Bs[(wn * 32 + j * 16 + lr) * LDK + kk + lk];
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i], b[j], acc[i][j], 0, 0, 0);
      }
    }
    __syncthreads();
  }
  // Output fragment layout: lane holds C[4 * lk + e][lr] of its 16x16 fragment.
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e)
        Cs[(wm * 32 + i * 16 + 4 * lk + e) * GLDC + wn * 32 + j * 16 + lr] = acc[i][j][e];
  __syncthreads();
  epi(Cs, m0, M, nt);
}

// ---------------------------------------------------------------- launchers

template <typename TM, typename TKV>
void GemmKernels<TM, TKV>::qkv(hipStream_t st, const TM* A, int M, const TM* W, int d, int hq, int hkv, float scale,
                               const int* row_stream, const int* row_pos, const float2* rope, float* q, TKV* kv,
                               KvLayout L, int layer, const int* page_table) {
  EpiQKV<TKV> e{hq, hkv, scale, row_stream, row_pos, rope, q, kv, L, layer, page_table};
  k_gemm<TM, EpiQKV<TKV>><<<dim3(hq + 2 * hkv, (M + GBM - 1) / GBM), 256, 0, st>>>(A, M, W, d, e);
}

template <typename TM, typename TKV>
void GemmKernels<TM, TKV>::resid(hipStream_t st, const TM* A, int M, const TM* W, int K, int N, float scale,
                                 float* x) {
  EpiResid e{N, scale, x};
  k_gemm<TM, EpiResid><<<dim3((N + 63) / 64, (M + GBM - 1) / GBM), 256, 0, st>>>(A, M, W, K, e);
}

template <typename TM, typename TKV>
void GemmKernels<TM, TKV>::gateup(hipStream_t st, const TM* A, int M, const TM* W, int d, int F, float scale,
                                  TM* m) {
  EpiGateUp<TM> e{F, scale, m};
  k_gemm<TM, EpiGateUp<TM>><<<dim3((F + 31) / 32, (M + GBM - 1) / GBM), 256, 0, st>>>(A, M, W, d, e);
}

template <typename TM, typename TKV>
void GemmKernels<TM, TKV>::logits(hipStream_t st, const TM* A, int M, const TM* W, int d, int V, float scale,
                                  float* logits, unsigned long long* slot, const int* row_stream) {
  EpiLogits e{V, scale, logits, slot, row_stream};
  k_gemm<TM, EpiLogits><<<dim3((V + 63) / 64, (M + GBM - 1) / GBM), 256, 0, st>>>(A, M, W, d, e);
}

template struct GemmKernels<float, float>;
template struct GemmKernels<_Float16, _Float16>;

}  // namespace hh
