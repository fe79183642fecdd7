// MFMA GEMM for gfx950 with fused epilogues, used where the decoder's work is a
// dense contraction: prompt prefill (M = prompt rows) and lockstep multi-stream
// decode (M = streams).  C[M, N] = A[M, K] * W[N, K]^T with fp32 accumulation.
//
// Operands are of type TM: _Float16 for bf16 models (the bf16 weights are
// repacked at load time to fp16 times a power-of-two scale, exact for this
// weight range, and activations are rounded to fp16 once), float for fp32
// models (v_mfma_f32_16x16x4_f32).  The finished tile is staged in LDS so the
// epilogue can use any column pairing (rotary pairs i / i + 32 of a head,
// gate / up columns) without shuffles.
#include "hh_kernels.h"

#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <type_traits>

namespace hh {

enum class GemmKind { QKV = 0, Resid = 1, GateUp = 2, Logits = 3 };

typedef float f32x16 __attribute__((ext_vector_type(16)));

// ---------------------------------------------------------------- epilogues
//
// The GEMM works on logical columns n; epi.b_row(n) names the weight row of
// column n (-1: none).  A tile covers logical columns [n0, n0 + BN) and the
// epilogue receives the finished fp32 tile Cs[BM][ldc] in LDS.

// Columns = rows of [Wq; Wk; Wv]; a tile holds whole heads (BN % 64 == 0).
// Rotates query heads into q (and qM), key heads into the KV page slot of
// each row; copies value heads.
template <typename TKV>
struct EpiQKV {
  int hq, hkv;
  float scale;
  const int* row_stream;
  const int* row_pos;
  const float2* rope;
  float* q;
  TKV* qM;  // nullptr, or rotated queries again in the MFMA operand type
  TKV* kv;
  KvLayout L;
  int layer;
  const int* page_table;
  __device__ int b_row(int n) const { return n < (hq + 2 * hkv) * 64 ? n : -1; }
  // Rotary pair (i, i + 32) of head `head` in row `row`, unscaled.
  __device__ void head_pair(int row, int head, int i, float y0, float y1) const {
    const int p = row_pos[row];
    head_pair_at(row, head, i, y0, y1, p, page_table[(size_t)row_stream[row] * L.max_pages + p / kPage]);
  }
  // The same with the row's position p and the KV page holding it given.
  __device__ void head_pair_at(int row, int head, int i, float y0, float y1, int p, int page) const {
    head_pair_cs(row, head, i, y0, y1, p, page, head < hq + hkv ? rope[(size_t)p * 32 + i] : make_float2(1.f, 0.f));
  }
  // ... and with the rotation's (cos, sin) at (p, i) given.
  __device__ void head_pair_cs(int row, int head, int i, float y0, float y1, int p, int page, float2 cs) const {
    y0 *= scale;
    y1 *= scale;
    if (head < hq + hkv) {
      const float r0 = y0 * cs.x - y1 * cs.y, r1 = y1 * cs.x + y0 * cs.y;
      if (head < hq) {
        if (q) {
          q[((size_t)row * hq + head) * 64 + i] = r0;
          q[((size_t)row * hq + head) * 64 + i + 32] = r1;
        }
        if (qM) {
          qM[((size_t)row * hq + head) * 64 + i] = (TKV)r0;
          qM[((size_t)row * hq + head) * 64 + i + 32] = (TKV)r1;
        }
      } else {
        TKV* dst = kv + L.head_tile(layer, page, 0, head - hq) + (p % kPage) * 64;
        dst[i] = (TKV)r0;
        dst[i + 32] = (TKV)r1;
      }
    } else {
      TKV* dst = kv + L.head_tile(layer, page, 1, head - hq - hkv) + (p % kPage) * 64;
      dst[i] = (TKV)y0;
      dst[i + 32] = (TKV)y1;
    }
  }
  // Register epilogue: logical columns cb + c and cb + 32 + c (cb % 64 == 0).
  __device__ void pair(int row, int cb, int c, float v0, float v1) const {
    const int head = cb / 64;
    if (head < hq + 2 * hkv) head_pair(row, head, c, v0, v1);
  }
  // A wave's whole in-range 64-column group (one head) for FM x 16 rows:
  // element e of accumulator block i is row rb + 32 i + 8 (e / 4) + e % 4.
  // The head's kind is decided once for all its rows.  Per block of 16 rows,
  // every lookup (positions, rotations, KV pages) is loaded before any
  // store: the stores may alias the tables as far as the compiler can tell,
  // so interleaved they would serialise one round trip per element.
  template <int FM>
  __device__ void group_full(int rb, int cb, int c, const f32x16* a0, const f32x16* a1) const {
    const int head = cb / 64;
    const bool isq = head < hq, isk = !isq && head < hq + hkv;
    const int kvh = isq ? 0 : isk ? head - hq : head - hq - hkv;
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      int p[16], sr[16], pg[16];
      float2 cs[16];
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int row = rb + 32 * i + 8 * (e >> 2) + (e & 3);
        p[e] = row_pos[row];
        if (!isq) sr[e] = row_stream[row];
      }
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        cs[e] = isq || isk ? rope[(size_t)p[e] * 32 + c] : make_float2(1.f, 0.f);
        if (!isq) pg[e] = page_table[(size_t)sr[e] * L.max_pages + p[e] / kPage];
      }
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int row = rb + 32 * i + 8 * (e >> 2) + (e & 3);
        float y0 = a0[i][e] * scale, y1 = a1[i][e] * scale;
        if (isq || isk) {
          const float r0 = y0 * cs[e].x - y1 * cs[e].y, r1 = y1 * cs[e].x + y0 * cs[e].y;
          y0 = r0;
          y1 = r1;
        }
        if (isq) {
          const size_t o = ((size_t)row * hq + head) * 64 + c;
          if (q) {
            q[o] = y0;
            q[o + 32] = y1;
          }
          if (qM) {
            qM[o] = (TKV)y0;
            qM[o + 32] = (TKV)y1;
          }
        } else {
          TKV* dst = kv + L.head_tile(layer, pg[e], isk ? 0 : 1, kvh) + (p[e] % kPage) * 64 + c;
          dst[0] = (TKV)y0;
          dst[32] = (TKV)y1;
        }
      }
    }
  }
  __device__ void operator()(const float* Cs, int ldc, int m0, int M, int n0, int BM, int BN) const {
    // Each row's position and KV page are looked up once per tile and kept
    // in the row's padding of the tile (ldc >= BN + 2): the element loop
    // then has no chain of dependent global loads per element.
    int* info = const_cast<int*>(reinterpret_cast<const int*>(Cs));
    for (int r = threadIdx.x; r < BM; r += blockDim.x) {
      const int row = m0 + r;
      if (row < M) {
        const int p = row_pos[row];
        info[r * ldc + BN] = p;
        info[r * ldc + BN + 1] = page_table[(size_t)row_stream[row] * L.max_pages + p / kPage];
      }
    }
    __syncthreads();
    // U pairs per thread at a time: their rotations are loaded before any
    // of their stores.
    constexpr int U = 8;
    const int nh = BN / 64, total = BM * 32 * nh;
    for (int base = threadIdx.x; base < total; base += U * (int)blockDim.x) {
      float2 cs[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int idx = base + u * (int)blockDim.x;
        const int r = idx / (32 * nh), head = n0 / 64 + (idx / 32) % nh;
        cs[u] = make_float2(1.f, 0.f);
        if (idx < total && m0 + r < M && head < hq + hkv) cs[u] = rope[(size_t)info[r * ldc + BN] * 32 + (idx & 31)];
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int idx = base + u * (int)blockDim.x;
        const int r = idx / (32 * nh), hh = (idx / 32) % nh, i = idx & 31, row = m0 + r;
        const int head = n0 / 64 + hh;
        if (idx >= total || row >= M || head >= hq + 2 * hkv) continue;
        head_pair_cs(row, head, i, Cs[r * ldc + hh * 64 + i], Cs[r * ldc + hh * 64 + i + 32], info[r * ldc + BN],
                     info[r * ldc + BN + 1], cs[u]);
      }
    }
  }
};

// x[row, col] += C (residual add of the O and down projections).
struct EpiResid {
  int N;
  float scale;
  float* x;
  __device__ int b_row(int n) const { return n < N ? n : -1; }
  __device__ void pair(int row, int cb, int c, float v0, float v1) const {
    float* xr = x + (size_t)row * N + cb + c;
    if (cb + c < N) xr[0] += v0 * scale;
    if (cb + 32 + c < N) xr[32] += v1 * scale;
  }
  template <int FM>
  __device__ void group_full(int rb, int cb, int c, const f32x16* a0, const f32x16* a1) const {
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        float* xr = x + (size_t)(rb + 32 * i + 8 * (e >> 2) + (e & 3)) * N + cb + c;
        xr[0] += a0[i][e] * scale;
        xr[32] += a1[i][e] * scale;
      }
  }
  __device__ void operator()(const float* Cs, int ldc, int m0, int M, int n0, int BM, int BN) const {
    for (int idx = threadIdx.x; idx < BM * BN; idx += blockDim.x) {
      const int r = idx / BN, c = idx % BN, row = m0 + r, col = n0 + c;
      if (row < M && col < N) x[(size_t)row * N + col] += Cs[r * ldc + c] * scale;
    }
  }
};

// Logical columns come in groups of 2 * half: gate columns j = group * half + c
// (c < half), then the matching up columns (rows F + j of [Wg; Wu]);
// m[row, j] = silu(gate) * up.
template <typename TM>
struct EpiGateUp {
  int F, half;
  float scale;
  TM* m;
  __device__ int b_row(int n) const {
    const int c = n % (2 * half), j = (n / (2 * half)) * half + (c < half ? c : c - half);
    return j < F ? (c < half ? j : F + j) : -1;
  }
  // Register epilogue (half == 32): gate column cb + c, up column cb + 32 + c.
  __device__ void pair(int row, int cb, int c, float v0, float v1) const {
    const int col = (cb / 64) * 32 + c;
    if (col < F) m[(size_t)row * F + col] = (TM)(silu(v0 * scale) * (v1 * scale));
  }
  // In-range group; SiLU with the hardware reciprocal (the result is rounded
  // to fp16 right after, far coarser than its 1-ulp error).
  template <int FM>
  __device__ void group_full(int rb, int cb, int c, const f32x16* a0, const f32x16* a1) const {
    TM* mc = m + (cb / 64) * 32 + c;
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const float gt = a0[i][e] * scale;
        mc[(size_t)(rb + 32 * i + 8 * (e >> 2) + (e & 3)) * F] =
            (TM)(gt * __builtin_amdgcn_rcpf(1.0f + __expf(-gt)) * (a1[i][e] * scale));
      }
  }
  __device__ void operator()(const float* Cs, int ldc, int m0, int M, int n0, int BM, int BN) const {
    const int j0 = (n0 / (2 * half)) * half, nc = BN / 2;
    for (int idx = threadIdx.x; idx < BM * nc; idx += blockDim.x) {
      const int r = idx / nc, c = idx % nc, row = m0 + r, col = j0 + c;
      if (row >= M || col >= F) continue;
      const int cg = (c / half) * 2 * half + c % half;  // gate column in the tile; up is half later
      const float g = Cs[r * ldc + cg] * scale, u = Cs[r * ldc + cg + half] * scale;
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
  __device__ int b_row(int n) const { return n < V ? n : -1; }
  __device__ void operator()(const float* Cs, int ldc, int m0, int M, int n0, int BM, int BN) const {
    if (logits)
      for (int idx = threadIdx.x; idx < BM * BN; idx += blockDim.x) {
        const int r = idx / BN, c = idx % BN, row = m0 + r, col = n0 + c;
        if (row < M && col < V) logits[(size_t)row * V + col] = Cs[r * ldc + c] * scale;
      }
    if (slot && (int)threadIdx.x < BM && m0 + (int)threadIdx.x < M) {
      const int r = threadIdx.x;
      unsigned long long best = 0ull;
      for (int c = 0; c < BN && n0 + c < V; ++c) {
        const unsigned long long k = argmax_key(Cs[r * ldc + c] * scale, (uint32_t)(n0 + c));
        best = k > best ? k : best;
      }
      atomicMax(slot + row_stream[m0 + r], best);
    }
  }
};

// ---------------------------------------------------------------- generic kernel (64 x 64)

// Any operand type and any K % 8 == 0 (fp32 models, odd shapes): 64x64 tile,
// four waves of 32x32 as 16x16 MFMA fragments, K in steps of 32 through LDS.
constexpr int GBM = 64, GBN = 64, GBK = 32;
constexpr int GLDC = GBN + 4;

template <typename TM, typename Epi>
__global__ __launch_bounds__(256) void k_gemm(const TM* __restrict__ A, int M, const TM* __restrict__ W, int K,
                                              Epi epi) {
  constexpr int V = Vec16<TM>::n;  // elements per 16-byte chunk
  constexpr int CPR = GBK / V;     // chunks per tile row
  constexpr int LDK = GBK + V;     // padded LDS row (elements)
  __shared__ __attribute__((aligned(16))) TM As[GBM * LDK];
  __shared__ __attribute__((aligned(16))) TM Bs[GBN * LDK];
  __shared__ float Cs[GBM * GLDC];
  const int n0 = blockIdx.x * GBN, m0 = blockIdx.y * GBM;
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
      const int br = epi.b_row(n0 + r);
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
  epi(Cs, GLDC, m0, M, n0, GBM, GBN);
}

// ---------------------------------------------------------------- fp16 kernel (BM x 128 x 64)

// fp16 operands, K % 64 == 0.  Tile BM x 128 (BM = 128, 64 or 32), K step 64;
// four waves (2 x 2 for BM >= 64, else 1 x 4), each a block of 32x32x16
// MFMAs.  Operands go global -> LDS with direct 16-byte loads, a wave
// instruction moving 8 whole rows of the step (8 cache lines) into an
// XOR-swizzled row-major stage, so every MFMA fragment read is a
// conflict-free 16-byte read.
// NSTAGE stages: the loads of the next NSTAGE-1 steps are in flight while a
// step computes; two workgroups per CU hide the rest of the latency.  Split-K
// workgroups write fp32 partial tiles that k_splitk_finalize sums in a fixed
// order (bitwise reproducible) before applying the epilogue.  Tiles are
// numbered with the column index fastest, so (with workgroups dealt
// round-robin to the 8 XCDs) row blocks that share a weight tile run on the
// same XCD and reuse it from its L2.
template <int BM>
struct F16Tile {
  static constexpr int BN = 128, BK = 64;
  // Four waves; two workgroups per CU fit in LDS (two independent
  // workgroups hide each other's barrier and load stalls better than one
  // workgroup of eight waves with a deeper pipeline).
  static constexpr int NW = 4;
  static constexpr int THREADS = 64 * NW;
  static constexpr int OCC = 2;
  static constexpr int NSTAGE = BM == 128 ? 2 : 3;
  static constexpr int WGM = BM >= 64 ? 2 : 1, WGN = NW / WGM;  // wave grid
  static constexpr int FM = BM / WGM / 32, FN = BN / WGN / 32;  // 32x32 blocks per wave
  static constexpr int GROUPS = (BM + BN) / 8;        // 1 KiB row groups (8 rows x 64 k) per stage
  static constexpr int NI = GROUPS / NW;               // loads per wave per stage
  static constexpr int STAGE = GROUPS * 1024;
  static constexpr int LDC = BN + 4;
  static constexpr int CS = BM * LDC * 4;
  static constexpr int LDS = (NSTAGE * STAGE > CS ? NSTAGE * STAGE : CS);
  static_assert(GROUPS % NW == 0, "row groups split evenly over the waves");
};


// Workgroup barrier without the memory fence __syncthreads() adds (waits are
// explicit in the caller).
__device__ __forceinline__ void bare_barrier() { asm volatile("s_barrier" ::: "memory"); }

// One 16-byte direct global -> LDS load per lane (wave-uniform LDS base).
// Kept in a device function: the builtin written directly in a kernel body
// makes the host pass drop the kernel's launch stub without a diagnostic.
__device__ __forceinline__ void load_lds16(const _Float16* src, char* dst) {
  __builtin_amdgcn_global_load_lds(src, dst, 16, 0, 0);
}

template <int NI, int NW>
__device__ __forceinline__ void issue_stage(const _Float16* const* src, int koff, char* dst, int wave) {
#pragma unroll
  for (int q = 0; q < NI; ++q)
    __builtin_amdgcn_global_load_lds(src[q] + koff, dst + (wave + NW * q) * 1024, 16, 0, 0);
}

// Wait until at most n * NI of this wave's loads are outstanding (n <= 3).
template <int NI>
__device__ __forceinline__ void wait_stages(int n) {
#define HH_VMWAIT(c) __builtin_amdgcn_s_waitcnt(((c) & 15) | (0x7 << 4) | (0xF << 8) | (((c) >> 4) << 14))
  switch (n) {
    case 0: HH_VMWAIT(0); break;
    case 1: HH_VMWAIT(NI); break;
    case 2: HH_VMWAIT(2 * NI); break;
    default: HH_VMWAIT(3 * NI); break;
  }
#undef HH_VMWAIT
}

template <int BM, class Epi>
__global__ __launch_bounds__(F16Tile<BM>::THREADS, F16Tile<BM>::OCC) void k_gemm_f16(const _Float16* __restrict__ A, int M,
                                                  const _Float16* __restrict__ W, int K, int ntn, int ntiles,
                                                  int steps_per_split, float* __restrict__ partial, int ncols,
                                                  Epi epi) {
  using T = F16Tile<BM>;
  static_assert((T::NSTAGE - 1) * T::NI <= 63, "in-flight loads exceed the vmcnt range");
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int tile = blockIdx.x % ntiles, split = blockIdx.x / ntiles;
  const int tn = tile % ntn, tm = tile / ntn;
  const int m0 = tm * BM, n0 = tn * T::BN;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int wm = wave / T::WGN, wn = wave % T::WGN;
  const int nk_all = K / T::BK;
  const int s0 = split * steps_per_split;
  const int nk = min(nk_all, s0 + steps_per_split) - s0;

  // Per-lane source addresses of the row groups this wave loads (fixed over
  // K).  A stage holds the BM rows of A then the BN rows of W, 128 bytes (the
  // step's 64 k) each; instruction q of wave w fills row group g = w + 4q
  // (rows 8g .. 8g + 7, 1 KiB; g = w + NW q): lane l takes row r = 8g + l/8 and stores it
  // in slot l%8, which holds the row's k chunk (l%8) ^ swz(r), swz(r) =
  // (r/2)%8.  Each instruction thus reads 8 whole cache lines, and an MFMA
  // fragment read (16 consecutive rows, one chunk, per 64-bank cycle) hits
  // 16 distinct bank quads.
  const _Float16* src[T::NI];
#pragma unroll
  for (int q = 0; q < T::NI; ++q) {
    const int rr = 8 * (wave + T::NW * q) + (lane >> 3);  // row within the stage
    const int chunk = (lane & 7) ^ ((rr >> 1) & 7);
    if (rr < BM) {
      const int row = min(m0 + rr, M - 1);  // rows past M: computed, never stored
      src[q] = A + (size_t)row * K + (size_t)s0 * T::BK + chunk * 8;
    } else {
      const int br = epi.b_row(n0 + rr - BM);
      src[q] = W + (size_t)(br < 0 ? 0 : br) * K + (size_t)s0 * T::BK + chunk * 8;
    }
  }

  f32x16 acc[T::FM][T::FN];
#pragma unroll
  for (int i = 0; i < T::FM; ++i)
#pragma unroll
    for (int j = 0; j < T::FN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  // Waits are explicit: __syncthreads() would add a workgroup release fence,
  // i.e. vmcnt(0), and stall on the later steps' loads as well.
  constexpr int kWaitLds = 0xF | (0x7 << 4) | (0x3 << 14);  // lgkmcnt(0)
  for (int i = 0; i < T::NSTAGE - 1 && i < nk; ++i)
    issue_stage<T::NI, T::NW>(src, i * T::BK, smem + i * T::STAGE, wave);
  for (int step = 0; step < nk; ++step) {
    const int ahead = step + T::NSTAGE - 1;
    if (ahead < nk) issue_stage<T::NI, T::NW>(src, ahead * T::BK, smem + (ahead % T::NSTAGE) * T::STAGE, wave);
    const int later = min(T::NSTAGE - 1, nk - 1 - step);  // stages after `step` in flight
    wait_stages<T::NI>(later);   // this wave's loads of `step` have landed
    bare_barrier();              // ... and every other wave's
    const char* sb = smem + (step % T::NSTAGE) * T::STAGE;
    // Fragment of rows r0 .. r0 + 31, k 16 kb .. + 16: lane l reads row
    // r0 + l%32, chunk 2 kb + l/32, from its swizzled slot.
    auto frag = [&](int r0, int kb) {
      const int r = r0 + (lane & 31), c = 2 * kb + (lane >> 5);
      return *reinterpret_cast<const f16x8*>(sb + r * 128 + 16 * (c ^ ((r >> 1) & 7)));
    };
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      f16x8 a[T::FM], b[T::FN];
#pragma unroll
      for (int i = 0; i < T::FM; ++i) a[i] = frag((wm * T::FM + i) * 32, kb);
#pragma unroll
      for (int j = 0; j < T::FN; ++j) b[j] = frag(BM + (wn * T::FN + j) * 32, kb);
#pragma unroll
      for (int i = 0; i < T::FM; ++i)
#pragma unroll
        for (int j = 0; j < T::FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
    __builtin_amdgcn_s_waitcnt(kWaitLds);  // this wave's reads of the stage are done ...
    bare_barrier();                         // ... and every wave's, before it is refilled
  }
  // Result element e of lane l in a 32x32 block: row 8(e/4) + 4(l/32) + e%4, column l%32.
  if (partial) {
    float* dst = partial + (size_t)split * M * ncols;
#pragma unroll
    for (int i = 0; i < T::FM; ++i)
#pragma unroll
      for (int j = 0; j < T::FN; ++j)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int r = m0 + (wm * T::FM + i) * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
          const int c = n0 + (wn * T::FN + j) * 32 + (lane & 31);
          if (r < M && c < ncols) dst[(size_t)r * ncols + c] = acc[i][j][e];
        }
    return;
  }
  float* Cs = reinterpret_cast<float*>(smem);
#pragma unroll
  for (int i = 0; i < T::FM; ++i)
#pragma unroll
    for (int j = 0; j < T::FN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int r = (wm * T::FM + i) * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
        const int c = (wn * T::FN + j) * 32 + (lane & 31);
        Cs[r * T::LDC + c] = acc[i][j][e];
      }
  __syncthreads();
  epi(Cs, T::LDC, m0, M, n0, BM, T::BN);
}

// Sum the split-K partials of a 2-row block in split order and apply the
// epilogue (small blocks give the reduction enough workgroups; each thread
// sums one element's partials with independent loads).
constexpr int kFinRows = 2;
template <class Epi>
__global__ __launch_bounds__(256) void k_splitk_finalize(const float* __restrict__ partial, int splits, int M,
                                                         int ncols, int ntn, Epi epi) {
  constexpr int BN = 128, LDC = BN + 4;
  __shared__ float Cs[kFinRows * LDC];
  const int tn = blockIdx.x % ntn, tm = blockIdx.x / ntn;
  const int m0 = tm * kFinRows, n0 = tn * BN;
  for (int idx = threadIdx.x; idx < kFinRows * BN; idx += 256) {
    const int r = idx / BN, c = idx % BN;
    float v = 0.f;
    if (m0 + r < M && n0 + c < ncols) {
      const float* pp = partial + (size_t)(m0 + r) * ncols + n0 + c;
      const size_t stride = (size_t)M * ncols;
      int sp = 0;
      for (; sp + 4 <= splits; sp += 4) {
        const float a = pp[sp * stride], b = pp[(sp + 1) * stride], c2 = pp[(sp + 2) * stride], d = pp[(sp + 3) * stride];
        v += a;  // split order, as in the loop below
        v += b;
        v += c2;
        v += d;
      }
      for (; sp < splits; ++sp) v += pp[sp * stride];
    }
    Cs[r * LDC + c] = v;
  }
  __syncthreads();
  epi(Cs, LDC, m0, M, n0, kFinRows, BN);
}

// ---------------------------------------------------------------- wide-tile fp16 kernel (prompt prefill)

// Prompt-sized GEMMs (M >= 256): BM x BN x 64 tiles, one 256-thread workgroup
// per CU, four waves in a 2 x 2 grid each owning a (BM/2) x (BN/2) block of
// 32x32x16 MFMAs.  A wave's LDS traffic per MFMA falls with the size of its
// block (a 128 x 128 block reads 8 KiB of fragments per 16 MFMAs, a 64 x 64
// block 4 KiB per 4), so large wave blocks keep the LDS well below its
// bandwidth.  Staging is the same as k_gemm_f16's (whole-line direct loads,
// (row/2)-swizzled chunks), one barrier per K step: the loads of a step are
// issued right after the barrier that retires the stage they overwrite.  The
// epilogue runs from the accumulators: column pairs (c, c + 32) of a 64-column
// group sit in one lane (blocks 2g and 2g + 1 of the wave), which is the pairing
// every register epilogue needs (rotary halves, gate / up).
template <int BM, int BN, int NW_ = 4>
struct WideTile {
  static constexpr int BK = 64, NW = NW_, THREADS = 64 * NW_;
  // Wave grid: 2 x 2 with four waves; with eight (two per SIMD, so one
  // wave's MFMAs run while the other waits on LDS or a barrier) 2 x 4 for
  // 256-wide tiles, else 4 x 2, so a wave block keeps whole 64-column groups.
  static constexpr int WGM = NW == 4 ? 2 : (BN >= 256 ? 2 : 4), WGN = NW / WGM;
  static constexpr int WM = BM / WGM, WN = BN / WGN;  // wave block
  static constexpr int FM = WM / 32, FN = WN / 32;   // 32x32 MFMA blocks per wave
  static constexpr int GROUPS = (BM + BN) / 8;       // 1 KiB row groups per stage
  static constexpr int NI = GROUPS / NW;             // load instructions per wave per stage
  static constexpr int STAGE = GROUPS * 1024;
  static constexpr int NSTAGE = (160 * 1024) / STAGE >= 3 ? 3 : 2;
  static constexpr int LDS = NSTAGE * STAGE;
  static_assert(FN % 2 == 0, "a wave block holds whole 64-column groups");
  static_assert(GROUPS % NW == 0, "row groups split evenly over the waves");
  static_assert(NSTAGE * STAGE <= 160 * 1024, "stages fit the LDS");
  static_assert((NSTAGE - 1) * NI <= 63, "in-flight loads fit the vmcnt range");
};

template <int BM, int BN, int NW, class Epi>
__global__ __launch_bounds__(64 * NW, 1) void k_gemm_wide(const _Float16* __restrict__ A, int M,
                                                          const _Float16* __restrict__ W, int K, int ntn, int ntiles,
                                                          int steps_per_split, float* __restrict__ partial, int ncols,
                                                          Epi epi) {
  using T = WideTile<BM, BN, NW>;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int tile = blockIdx.x % ntiles, split = blockIdx.x / ntiles;
  const int tn = tile % ntn, tm = tile / ntn;
  const int m0 = tm * BM, n0 = tn * BN;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int wm = wave / T::WGN, wn = wave % T::WGN;
  const int nk_all = K / T::BK;
  const int s0 = split * steps_per_split;
  const int nk = min(nk_all, s0 + steps_per_split) - s0;

  // Instruction q of wave w fills row group g = w + NW q (stage rows 8g .. 8g + 7):
  // lane l takes row 8g + l/8, k chunk (l%8) ^ swz(row), swz(r) = (r/2) % 8.
  const _Float16* src[T::NI];
#pragma unroll
  for (int q = 0; q < T::NI; ++q) {
    const int rr = 8 * (wave + T::NW * q) + (lane >> 3);
    const int chunk = (lane & 7) ^ ((rr >> 1) & 7);
    if (rr < BM) {
      const int row = min(m0 + rr, M - 1);  // rows past M: computed, never stored
      src[q] = A + (size_t)row * K + (size_t)s0 * T::BK + chunk * 8;
    } else {
      const int br = epi.b_row(n0 + rr - BM);
      src[q] = W + (size_t)(br < 0 ? 0 : br) * K + (size_t)s0 * T::BK + chunk * 8;
    }
  }

  f32x16 acc[T::FM][T::FN];
#pragma unroll
  for (int i = 0; i < T::FM; ++i)
#pragma unroll
    for (int j = 0; j < T::FN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  // Loads are issued unconditionally (K steps past the end re-read the last
  // one into a stage nobody reads again), so exactly NSTAGE - 2 stages are in
  // flight behind the current one at every wait, and the scheduling groups
  // below see one basic block per step.
  constexpr int kWaitLds = 0xF | (0x7 << 4) | (0x3 << 14);  // lgkmcnt(0)
#pragma unroll
  for (int i = 0; i < T::NSTAGE - 1; ++i)
    issue_stage<T::NI, T::NW>(src, min(i, nk - 1) * T::BK, smem + i * T::STAGE, wave);
  for (int step = 0; step < nk; ++step) {
    wait_stages<T::NI>(T::NSTAGE - 2);  // this wave's loads of `step` have landed
    __builtin_amdgcn_s_waitcnt(kWaitLds);
    bare_barrier();                     // every wave's have, and every wave is done with step - 1
    const int ahead = step + T::NSTAGE - 1;
    const char* sb = smem + (step % T::NSTAGE) * T::STAGE;
    char* nb = smem + (ahead % T::NSTAGE) * T::STAGE;
    const int koff = min(ahead, nk - 1) * T::BK;
    auto frag = [&](int r0, int kb) {
      const int r = r0 + (lane & 31), c = 2 * kb + (lane >> 5);
      return *reinterpret_cast<const f16x8*>(sb + r * 128 + 16 * (c ^ ((r >> 1) & 7)));
    };
    // Fragments of k block kb + 1 are read while the MFMAs of kb run; the
    // next stage's global loads are spread over the step's MFMAs.
    f16x8 a[2][T::FM], b[2][T::FN];
#pragma unroll
    for (int i = 0; i < T::FM; ++i) a[0][i] = frag(wm * T::WM + i * 32, 0);
#pragma unroll
    for (int j = 0; j < T::FN; ++j) b[0][j] = frag(BM + wn * T::WN + j * 32, 0);
    constexpr int kLoadsPerKb = (T::NI + 3) / 4;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      const int cur = kb & 1, nxt = cur ^ 1;
      if (kb < 3) {
#pragma unroll
        for (int i = 0; i < T::FM; ++i) a[nxt][i] = frag(wm * T::WM + i * 32, kb + 1);
#pragma unroll
        for (int j = 0; j < T::FN; ++j) b[nxt][j] = frag(BM + wn * T::WN + j * 32, kb + 1);
      }
#pragma unroll
      for (int q = kb * kLoadsPerKb; q < (kb + 1) * kLoadsPerKb && q < T::NI; ++q)
        load_lds16(src[q] + koff, nb + (wave + T::NW * q) * 1024);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < T::FM; ++i)
#pragma unroll
        for (int j = 0; j < T::FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a[cur][i], b[cur][j], acc[i][j], 0, 0, 0);
      // Keep the reads and loads of this block ahead of its MFMAs (the
      // scheduler would otherwise sink each read to just before its first use).
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  wait_stages<T::NI>(0);  // no direct-to-LDS load outlives the workgroup
  // Element e of lane l in a 32x32 block: row 8(e/4) + 4(l/32) + e%4, column l%32.
  const int rbase = m0 + wm * T::WM + 4 * (lane >> 5), c = lane & 31;
  if (partial) {
    float* dst = partial + (size_t)split * M * ncols;
#pragma unroll
    for (int i = 0; i < T::FM; ++i)
#pragma unroll
      for (int j = 0; j < T::FN; ++j)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int r = rbase + i * 32 + 8 * (e >> 2) + (e & 3);
          const int col = n0 + wn * T::WN + j * 32 + c;
          if (r < M && col < ncols) dst[(size_t)r * ncols + col] = acc[i][j][e];
        }
    return;
  }
  if (m0 + BM <= M && n0 + BN <= ncols) {
    // Whole tile in range (every tile of a prompt whose length is a multiple
    // of BM): no per-element guards, which would otherwise turn the unrolled
    // epilogue into thousands of exec-mask branches.
#pragma unroll
    for (int g = 0; g < T::FN / 2; ++g) {
      f32x16 a0[T::FM], a1[T::FM];
#pragma unroll
      for (int i = 0; i < T::FM; ++i) {
        a0[i] = acc[i][2 * g];
        a1[i] = acc[i][2 * g + 1];
      }
      epi.template group_full<T::FM>(rbase, n0 + wn * T::WN + 64 * g, c, a0, a1);
    }
    return;
  }
#pragma unroll
  for (int i = 0; i < T::FM; ++i)
#pragma unroll
    for (int g = 0; g < T::FN / 2; ++g)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int r = rbase + i * 32 + 8 * (e >> 2) + (e & 3);
        if (r < M) epi.pair(r, n0 + wn * T::WN + 64 * g, c, acc[i][2 * g][e], acc[i][2 * g + 1][e]);
      }
}

// ---------------------------------------------------------------- launchers

// Launchers return the number of K splits used.  With defer set, split
// partials are left in the workspace for the caller to reduce (1: the
// epilogue already ran).
template <int BM, class Epi>
static int launch_f16(hipStream_t st, GemmWorkspace ws, const _Float16* A, int M, const _Float16* W, int K, int n_cols,
                      const Epi& e, bool defer) {
  using T = F16Tile<BM>;
  static bool attr = false;
  if (!attr) {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(k_gemm_f16<BM, Epi>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, T::LDS);
    attr = true;
  }
  const int ntn = (n_cols + T::BN - 1) / T::BN;
  const int ntiles = ((M + BM - 1) / BM) * ntn;
  const int nk = K / T::BK;
  // Split K only when tiles alone leave most CUs idle: then aim at 256
  // workgroups, at least 4 K steps each, with partials that fit the workspace.
  int splits = ntiles < 128 ? (256 + ntiles - 1) / ntiles : 1;
  splits = std::min(splits, std::max(1, nk / 4));
  while (splits > 1 && (size_t)splits * M * n_cols * sizeof(float) > ws.bytes) --splits;
  const int per = (nk + splits - 1) / splits;
  splits = (nk + per - 1) / per;
  float* part = splits > 1 ? ws.ptr : nullptr;
  k_gemm_f16<BM, Epi><<<ntiles * splits, T::THREADS, T::LDS, st>>>(A, M, W, K, ntn, ntiles, per, part, n_cols, e);
  if (splits > 1 && !defer)
    k_splitk_finalize<Epi><<<((M + kFinRows - 1) / kFinRows) * ntn, 256, 0, st>>>(part, splits, M, n_cols, ntn, e);
  return splits;
}

template <int BM, int BN, int NW = 4, class Epi>
static int launch_wide(hipStream_t st, GemmWorkspace ws, const _Float16* A, int M, const _Float16* W, int K, int n_cols,
                       int splits, const Epi& e, bool defer) {
  using T = WideTile<BM, BN, NW>;
  static bool attr = false;
  if (!attr) {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(k_gemm_wide<BM, BN, NW, Epi>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, T::LDS);
    attr = true;
  }
  const int ntn = (n_cols + BN - 1) / BN;
  const int ntiles = ((M + BM - 1) / BM) * ntn;
  const int nk = K / T::BK;
  splits = std::max(1, std::min(splits, nk / 4));
  while (splits > 1 && (size_t)splits * M * n_cols * sizeof(float) > ws.bytes) --splits;
  const int per = (nk + splits - 1) / splits;
  splits = (nk + per - 1) / per;
  float* part = splits > 1 ? ws.ptr : nullptr;
  k_gemm_wide<BM, BN, NW, Epi><<<ntiles * splits, T::THREADS, T::LDS, st>>>(A, M, W, K, ntn, ntiles, per, part, n_cols,
                                                                            e);
  if (splits > 1 && !defer)
    k_splitk_finalize<Epi><<<((M + kFinRows - 1) / kFinRows) * ntn * (BN / 128), 256, 0, st>>>(part, splits, M, n_cols,
                                                                                             ntn * (BN / 128), e);
  return splits;
}

// ---------------------------------------------------------------- skinny kernel (<= 32 rows)

// Lockstep multi-stream decode: C[M <= 32, N] = A W^T is weight streaming, not
// arithmetic.  A workgroup owns 64 logical columns (one QKV head, 32 gate + 32
// up columns, or 64 residual columns) and one K range; each group of four
// waves takes 16 weight rows per wave (KW groups split the K range).  Weights
// go from HBM straight into registers as the A operand of 16x16x32 MFMAs (lane
// l: row l%16, k 8(l/16) .. + 8), from a copy laid out as 16 x 32 operand
// tiles, in batches of eight K blocks with the next batch loading while one
// computes; the activations (at most 32 rows) of each batch are loaded once per
// K group, coalesced, into double-buffered LDS (16-byte row padding keeps the
// B fragment reads conflict-free).  The finished 64-column tile goes through
// LDS into the usual epilogue, or into split partials when K is split to give
// every CU work.
// RowNorm consumer of the 32-row kernels: thread t < 256 loads float4 t % 8
// of row t / 8's block sums (nss <= 32, a multiple of 4; eight consecutive
// lanes read one row's 128 bytes) first thing, so that the tail finds them
// landed (zeros past M rows or nss sums).
__device__ __forceinline__ void row_norm_loads(float4& ssv, const RowNorm& rn, int M) {
  if (!rn.ss_in || threadIdx.x >= 256) return;
  const __amdgpu_buffer_rsrc_t res =
      __builtin_amdgcn_make_buffer_rsrc((void*)rn.ss_in, (short)0, (int)((size_t)M * rn.nss * 4), 0x00020000);
  const int r = threadIdx.x >> 3, q = threadIdx.x & 7;
  ssv = __builtin_bit_cast(
      float4, __builtin_amdgcn_raw_buffer_load_b128(
                  res, r < M && 4 * q < rn.nss ? (unsigned)((r * rn.nss + 4 * q) * 4) : 0x80000000u, 0, 0));
}

// acc0[j] of lane l: column 16 rw + 4 (l / 16) + j, row l % 16 (acc1: row
// + 16).  K groups add into the LDS tile Cs (32 x 68 floats, which the caller's
// activation buffer holds once every wave is done with it) in group order;
// rows are scaled by their norm factors (RowNorm consumer), then the tile
// goes to the split partials or through the epilogue.  A RowNorm producer's
// last split of the column block then finishes the residual (rs, flag: LDS
// scratch of 32 floats and one int).
template <class Epi, int KW>
__device__ __forceinline__ void skinny_tail(float* Cs, const f32x4& acc0, const f32x4& acc1, int rw, int kg, int lane,
                                            float* __restrict__ partial, int split, int splits, int cb, int M,
                                            int ncols, int n0, const Epi& epi, const RowNorm& rn,
                                            const float4& ssv, float* rs, int* flag) {
  constexpr int LDC = 68;
  const int col = 16 * rw + 4 * (lane >> 4), r = lane & 15;
  float f0 = 1.f, f1 = 1.f;  // norm factors of rows r and r + 16
  if (rn.ss_in) {
    if (threadIdx.x < 256) {
      float v = (ssv.x + ssv.y) + (ssv.z + ssv.w);
      v += __shfl_xor(v, 1);
      v += __shfl_xor(v, 2);
      v += __shfl_xor(v, 4);
      if ((threadIdx.x & 7) == 0) rs[threadIdx.x >> 3] = rsqrtf(v / rn.n + rn.eps);
    }
    __syncthreads();
    f0 = rs[r];
    f1 = rs[r + 16];
  }
#pragma unroll
  for (int g = 0; g < KW; ++g) {
    if (kg == g) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        Cs[r * LDC + col + j] = (g ? Cs[r * LDC + col + j] : 0.f) + acc0[j] * f0;
        Cs[(r + 16) * LDC + col + j] = (g ? Cs[(r + 16) * LDC + col + j] : 0.f) + acc1[j] * f1;
      }
    }
    __syncthreads();
  }
  if (partial) {
    bool producer = false;
    if constexpr (std::is_same<Epi, EpiResid>::value) producer = rn.cnt != nullptr;
    if (!producer) {
      float* dst = partial + (size_t)split * M * ncols;
      for (int i = threadIdx.x; i < M * 64; i += blockDim.x) {
        const int rr = i / 64, c = i % 64;
        if (n0 + c < ncols) dst[(size_t)rr * ncols + n0 + c] = Cs[rr * LDC + c];
      }
      return;
    }
    if constexpr (std::is_same<Epi, EpiResid>::value) {
      // RowNorm producer.  The partials go out and come back with the
      // agent-coherent cache policy, so that no fence (and no writeback or
      // invalidation of a whole L2) is needed: a split's stores have
      // completed before it counts itself in, and the last split to arrive
      // reads every split's partials from the coherent level.
      constexpr int kSc1 = 16;
      const int N = epi.N;
      const __amdgpu_buffer_rsrc_t pres = __builtin_amdgcn_make_buffer_rsrc(
          (void*)partial, (short)0, (int)((size_t)splits * M * ncols * 4), 0x00020000);
      const unsigned sstride = (unsigned)M * ncols * 4;  // bytes of one split's partials
      // Items: row rr = it / 16, four columns n0 + 4 (it % 16); a row's 16
      // items are 16 aligned lanes of one wave (M * 16 <= 512 <= 2 blockDim).
      // Every split loads its items' x and gains before counting itself in,
      // so the last one does not wait for them afterwards.
      float4 xa[2], ga[2];
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        const int it = threadIdx.x + blockDim.x * k, rr = it >> 4, c = n0 + 4 * (it & 15);
        if (it < M * 16 && c < N) {
          xa[k] = *reinterpret_cast<const float4*>(epi.x + (size_t)rr * N + c);
          ga[k] = *reinterpret_cast<const float4*>(rn.gain + c);
        }
      }
      for (int it = threadIdx.x; it < M * 16; it += blockDim.x) {
        const int rr = it >> 4, c = n0 + 4 * (it & 15);
        if (c < ncols) {
          const float4 v = *reinterpret_cast<const float4*>(Cs + rr * LDC + 4 * (it & 15));
          __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), pres,
                                                 (unsigned)split * sstride + (unsigned)(rr * ncols + c) * 4, 0, kSc1);
        }
      }
      __builtin_amdgcn_s_waitcnt(0);  // every store of this thread acknowledged
      __syncthreads();
      if (threadIdx.x == 0) *flag = atomicAdd(rn.cnt + cb, 1) == splits - 1;
      __syncthreads();
      if (!*flag) return;
      // Up to 8 splits: both items' partials are loaded at once; more splits
      // go 8 at a time.  Either way they are summed in split order.
      float4 t[2];
#pragma unroll
      for (int k = 0; k < 2; ++k) t[k] = make_float4(0.f, 0.f, 0.f, 0.f);
      for (int s0 = 0; s0 < splits; s0 += 8) {
        float4 u[2][8];
#pragma unroll
        for (int k = 0; k < 2; ++k) {
          const int it = threadIdx.x + blockDim.x * k, rr = it >> 4, c = n0 + 4 * (it & 15);
          const bool ok = it < M * 16 && c < N;
#pragma unroll
          for (int j = 0; j < 8; ++j)
            u[k][j] = __builtin_bit_cast(
                float4, __builtin_amdgcn_raw_buffer_load_b128(
                            pres, ok && s0 + j < splits ? (unsigned)(s0 + j) * sstride + (unsigned)(rr * ncols + c) * 4
                                                        : 0x80000000u,
                            0, kSc1));
        }
#pragma unroll
        for (int k = 0; k < 2; ++k)
#pragma unroll
          for (int j = 0; j < 8; ++j)
            if (s0 + j < splits) {
              t[k].x += u[k][j].x;
              t[k].y += u[k][j].y;
              t[k].z += u[k][j].z;
              t[k].w += u[k][j].w;
            }
      }
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        const int it = threadIdx.x + blockDim.x * k, rr = it >> 4, c = n0 + 4 * (it & 15);
        float sq = 0.f;
        if (it < M * 16 && c < N) {
          float4 a = xa[k];
          a.x += t[k].x * epi.scale;
          a.y += t[k].y * epi.scale;
          a.z += t[k].z * epi.scale;
          a.w += t[k].w * epi.scale;
          *reinterpret_cast<float4*>(epi.x + (size_t)rr * N + c) = a;
          const float4 g = ga[k];
          typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
          const f16x4 o = {(_Float16)(a.x * g.x), (_Float16)(a.y * g.y), (_Float16)(a.z * g.z), (_Float16)(a.w * g.w)};
          *reinterpret_cast<f16x4*>(rn.y + (size_t)rr * N + c) = o;
          sq = a.x * a.x + a.y * a.y + a.z * a.z + a.w * a.w;
        }
        sq += __shfl_xor(sq, 8);
        sq += __shfl_xor(sq, 4);
        sq += __shfl_xor(sq, 2);
        sq += __shfl_xor(sq, 1);
        if (it < M * 16 && (it & 15) == 0) rn.ss_out[(size_t)rr * ((N + 63) / 64) + cb] = sq;
      }
      if (threadIdx.x == 0) __hip_atomic_store(rn.cnt + cb, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    return;
  }
  epi(Cs, LDC, 0, M, n0, 32, 64);
}
constexpr int kSkinnyTileBytes = 32 * 68 * 4;
// LDS row pitch (halfs) of the activation-resident skinny kernel: a K group's
// largest block count rounded up to 4 blocks (256 bytes), plus 16 bytes.
__host__ __device__ constexpr int skinny_res_pitch(int steps_per_split, int kw) {
  return 32 * ((((steps_per_split + kw - 1) / kw) + 3) & ~3) + 8;
}

template <class Epi, int U, int KW>
__global__ __launch_bounds__(256 * KW) void k_gemm_skinny(const _Float16* __restrict__ A, int M,
                                                          const _Float16* __restrict__ Wt, int K, int nb,
                                                          int steps_per_split, float* __restrict__ partial, int ncols,
                                                          Epi epi, RowNorm rn) {
  constexpr int XP = 32 * U + 8;              // LDS row pitch of an activation chunk (halfs; 16 bytes of padding)
  constexpr int XCH = 32 * (32 * U / 8);      // 16-byte chunks per activation batch (32 rows)
  static_assert(XCH % 256 == 0, "activation chunks split evenly over a group's threads");
  __shared__ __attribute__((aligned(16))) _Float16 xs[KW][2][32 * XP];
  static_assert(sizeof(xs) >= kSkinnyTileBytes, "the tile fits the activation buffers");
  __shared__ float rs[32];
  __shared__ int flag;
  float4 ssv = make_float4(0.f, 0.f, 0.f, 0.f);
  row_norm_loads(ssv, rn, M);
  const int cb = blockIdx.x % nb, split = blockIdx.x / nb;
  const int n0 = cb * 64;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int rw = wave & 3, kg = wave >> 2;  // 16-row group, K group
  const int gt = threadIdx.x & 255;         // thread index within the K group
  const int k0 = split * steps_per_split * 32;
  const int nkb_all = min(K - k0, steps_per_split * 32) / 32;  // K blocks of 32 in this range
  // K group kg takes blocks [kb_lo, kb_lo + nkb) of the range.
  const int kb_lo = (nkb_all * kg) / KW, nkb = (nkb_all * (kg + 1)) / KW - kb_lo;
  const int kbase = k0 + 32 * kb_lo;

  // Weights (16 x 32 operand tiles, 1 KiB each in lane order, so a load
  // instruction reads one contiguous KiB) and activations both come through
  // range-checked buffer loads: the batches need no clamping (blocks past this
  // range read further on, or zeros past the matrix, and are never used), and
  // activation rows past M read zeros.
  const int nkbt = K / 32;  // tiles per 16-row block
  const int rb = 4 * cb + rw;
  const __amdgpu_buffer_rsrc_t wres = __builtin_amdgcn_make_buffer_rsrc(
      (void*)Wt, (short)0, (int)((size_t)((ncols + 15) / 16) * 16 * K * 2), 0x00020000);
  const __amdgpu_buffer_rsrc_t xres =
      __builtin_amdgcn_make_buffer_rsrc((void*)A, (short)0, (int)((size_t)M * K * 2), 0x00020000);
  const unsigned wvoff = (unsigned)((((size_t)rb * nkbt + kbase / 32) * 64 + lane) * 16);
  // Activation batch: group thread t loads chunks t + 256 j (row c / (4 U), 8
  // halfs at 8 (c % (4 U))), consecutive threads reading consecutive 16 bytes.
  constexpr int XJ = XCH / 256;
  auto xload = [&](f16x8* v, int kb0) {
#pragma unroll
    for (int j = 0; j < XJ; ++j) {
      const int c = gt + 256 * j, r = c / (4 * U), kc = c % (4 * U);
      v[j] = __builtin_bit_cast(
          f16x8, __builtin_amdgcn_raw_buffer_load_b128(xres, (unsigned)((r * K + kbase + 32 * kb0 + 8 * kc) * 2), 0, 0));
    }
  };
  auto xstore = [&](const f16x8* v, int buf) {
#pragma unroll
    for (int j = 0; j < XJ; ++j) {
      const int c = gt + 256 * j, r = c / (4 * U), kc = c % (4 * U);
      *reinterpret_cast<f16x8*>(&xs[kg][buf][r * XP + 8 * kc]) = v[j];
    }
  };
  // Weights are read once per step: non-temporal loads (streaming policy in
  // the caches) measured 15.9 -> 15.1 us for gate/up and 98 -> 93 us for the
  // LM head at 32 rows.
  constexpr int kNt = 2;
  auto wload = [&](f16x8* w, int kb0) {
#pragma unroll
    for (int u = 0; u < U; ++u)
      w[u] = __builtin_bit_cast(f16x8, __builtin_amdgcn_raw_buffer_load_b128(wres, wvoff + 1024u * (kb0 + u), 0, kNt));
  };
  f32x4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
  auto compute = [&](const f16x8* w, int buf, int kb0) {
    const _Float16* xb = &xs[kg][buf][(lane & 15) * XP + 8 * (lane >> 4)];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (kb0 + u < nkb) {
        const f16x8 b0 = *reinterpret_cast<const f16x8*>(xb + 32 * u);
        const f16x8 b1 = *reinterpret_cast<const f16x8*>(xb + 16 * XP + 32 * u);
        acc0 = __builtin_amdgcn_mfma_f32_16x16x32_f16(w[u], b0, acc0, 0, 0, 0);
        acc1 = __builtin_amdgcn_mfma_f32_16x16x32_f16(w[u], b1, acc1, 0, 0, 0);
      }
    }
  };
  // Batch i computes from xs[kg][i & 1] and registers wa / wb while batch
  // i + 1's activations and weights load; one barrier per batch (the same
  // count in every K group) orders the LDS reuse.
  const int nbatch = ((nkb_all + KW - 1) / KW + U - 1) / U;
  f16x8 wa[U], wb[U], xv[XJ];
  xload(xv, 0);
  wload(wa, 0);
  xstore(xv, 0);
  __syncthreads();
  for (int bt = 0; bt < nbatch; bt += 2) {
    if (bt + 1 < nbatch) {
      xload(xv, (bt + 1) * U);  // issued before the weights, so waiting for it leaves them in flight
      wload(wb, (bt + 1) * U);
    }
    compute(wa, 0, bt * U);
    if (bt + 1 >= nbatch) break;
    xstore(xv, 1);
    __syncthreads();
    if (bt + 2 < nbatch) {
      xload(xv, (bt + 2) * U);
      wload(wa, (bt + 2) * U);
    }
    compute(wb, 1, (bt + 1) * U);
    if (bt + 2 >= nbatch) break;
    xstore(xv, 0);
    __syncthreads();
  }

  __syncthreads();  // every wave is done with the activations
  skinny_tail<Epi, KW>(reinterpret_cast<float*>(&xs[0][0][0]), acc0, acc1, rw, kg, lane, partial, split, gridDim.x / nb,
                       cb, M, ncols, n0, epi, rn, ssv, rs, &flag);
}

// Activation-resident variant, for grids of at most two workgroups per CU:
// every wave issues its first weight loads with the activations and the rest
// (at most 32 K blocks, 32 KiB per wave, in all) once those have landed, the workgroup's activation range (32 rows x at most 1024 K
// per K group) goes into LDS once, and each block's MFMAs wait only for that
// block's weights.  The batched kernel above pays an L2 round trip and a
// barrier per 256 K of activations, and keeps two batches in flight: at 32
// rows its gate/up launch took 7.3 us with no weight loads at all.  Loads a
// wave does not need (blocks past its range, chunks past the group's K) take
// an offset past the buffer's range, which returns zeros without a memory
// access, so the issue order stays branch-free.  Wave rw of a K group loads
// rows rw, rw + 4, ... (16-byte chunks lane + 64 q along the row); the LDS row
// pitch is 16 bytes past a multiple of 256 bytes, as in the batched kernel,
// so the B fragment reads stay conflict-free.
template <class Epi, int NB, int KW>
__global__ __launch_bounds__(256 * KW) void k_gemm_skinny_res(const _Float16* __restrict__ A, int M,
                                                              const _Float16* __restrict__ Wt, int K, int nb,
                                                              int steps_per_split, float* __restrict__ partial,
                                                              int ncols, Epi epi, RowNorm rn) {
  constexpr int XQ = (4 * NB + 63) / 64;  // activation chunks per lane and row
  constexpr unsigned kOob = 0x80000000u;  // past every buffer range here (ranges stay below 2^31 bytes)
  extern __shared__ __attribute__((aligned(16))) _Float16 xsd[];
  __shared__ float rs[32];
  __shared__ int flag;
  float4 ssv = make_float4(0.f, 0.f, 0.f, 0.f);
  row_norm_loads(ssv, rn, M);  // first, so that no later wait covers them
  const int cb = blockIdx.x % nb, split = blockIdx.x / nb;
  const int n0 = cb * 64;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int rw = wave & 3, kg = wave >> 2;
  const int k0 = split * steps_per_split * 32;
  const int nkb_all = min(K - k0, steps_per_split * 32) / 32;
  const int kb_lo = (nkb_all * kg) / KW, nkb = (nkb_all * (kg + 1)) / KW - kb_lo;
  const int kbase = k0 + 32 * kb_lo;
  const int pitch = skinny_res_pitch(steps_per_split, KW);
  _Float16* xs = xsd + (size_t)kg * 32 * pitch;
  // Chunks past the group's K are stored to a 16-byte slot past the tiles.
  _Float16* sink = xsd + (size_t)KW * 32 * pitch;

  const int nkbt = K / 32;
  const int rb = 4 * cb + rw;
  const __amdgpu_buffer_rsrc_t wres = __builtin_amdgcn_make_buffer_rsrc(
      (void*)Wt, (short)0, (int)((size_t)((ncols + 15) / 16) * 16 * K * 2), 0x00020000);
  const __amdgpu_buffer_rsrc_t xres =
      __builtin_amdgcn_make_buffer_rsrc((void*)A, (short)0, (int)((size_t)M * K * 2), 0x00020000);
  const unsigned wvoff = (unsigned)((((size_t)rb * nkbt + kbase / 32) * 64 + lane) * 16);
  constexpr int kNt = 2;  // weights are read once per step: streaming policy
  // Activations first, so that the wait before their LDS stores leaves the
  // weights in flight.  Rows past M read zeros.
  f16x8 xv[8][XQ];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int q = 0; q < XQ; ++q) {
      const int kc = lane + 64 * q;
      const unsigned off = kc < 4 * nkb ? (unsigned)(((rw + 4 * i) * K + kbase + 8 * kc) * 2) : kOob;
      xv[i][q] = __builtin_bit_cast(f16x8, __builtin_amdgcn_raw_buffer_load_b128(xres, off, 0, 0));
    }
  // The scheduler would otherwise start the LDS stores (and so wait for the
  // activations) before issuing the first weight loads.
  __builtin_amdgcn_sched_barrier(0);
  // Wave (rb, kg) starts its tiles at block `rot` of its range and wraps
  // around, so that the waves' first requests do not all fall on 32 KiB
  // boundaries (every range starts on one).
  const int rot = nkb > 0 ? (rb * 13 + kg * 7) % nkb : 0;
  auto blk = [&](int u) { return u + rot < nkb ? u + rot : u + rot - nkb; };
  // Only the first W0 weight blocks go out with the activations: with every
  // block issued at once, the activations (a shared 128 KiB per workgroup,
  // from memory after the producing launch) came back behind the weight
  // stream, ~10 us into a 13.5 us gate/up launch, and every MFMA waited for
  // them.  The rest of the weights follow once the activations have landed
  // (the 32-row step 0.957 -> 0.947 ms; 4, 12 and 16 blocks first measured
  // 0.948, 0.951 and 0.954).
  constexpr int W0 = NB < 8 ? NB : 8;
  f16x8 w[NB];
#pragma unroll
  for (int u = 0; u < W0; ++u)
    w[u] = __builtin_bit_cast(
        f16x8, __builtin_amdgcn_raw_buffer_load_b128(wres, u < nkb ? wvoff + 1024u * blk(u) : kOob, 0, kNt));
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int q = 0; q < XQ; ++q) {
      const int kc = lane + 64 * q;
      _Float16* dst = kc < 4 * nkb ? xs + (rw + 4 * i) * pitch + 8 * kc : sink;
      *reinterpret_cast<f16x8*>(dst) = xv[i][q];
    }
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int u = W0; u < NB; ++u)
    w[u] = __builtin_bit_cast(
        f16x8, __builtin_amdgcn_raw_buffer_load_b128(wres, u < nkb ? wvoff + 1024u * blk(u) : kOob, 0, kNt));
  __builtin_amdgcn_sched_barrier(0);
  __syncthreads();

  f32x4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
  const _Float16* xb = xs + (lane & 15) * pitch + 8 * (lane >> 4);
#pragma unroll
  for (int u = 0; u < NB; ++u) {
    if (u < nkb) {
      const int kb = blk(u);
      const f16x8 b0 = *reinterpret_cast<const f16x8*>(xb + 32 * kb);
      const f16x8 b1 = *reinterpret_cast<const f16x8*>(xb + 16 * pitch + 32 * kb);
      acc0 = __builtin_amdgcn_mfma_f32_16x16x32_f16(w[u], b0, acc0, 0, 0, 0);
      acc1 = __builtin_amdgcn_mfma_f32_16x16x32_f16(w[u], b1, acc1, 0, 0, 0);
    }
  }

  __syncthreads();  // every wave is done with the activations
  skinny_tail<Epi, KW>(reinterpret_cast<float*>(xsd), acc0, acc1, rw, kg, lane, partial, split, gridDim.x / nb, cb, M,
                       ncols, n0, epi, rn, ssv, rs, &flag);
}

constexpr int kSkinnyResLds = 159 * 1024;  // dynamic LDS limit of the resident kernel

template <class Epi, int NB, int KW>
static bool skinny_res_go(hipStream_t st, unsigned bytes, const _Float16* A, int M, const _Float16* Wt, int K, int nb,
                          int splits, int per, float* part, int n_cols, const Epi& e, const RowNorm& rn) {
  // Once per instantiation, to the largest size the launcher allows (the
  // kernel's static LDS takes the rest of the 160 KiB).
  static const hipError_t attr = [] {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(k_gemm_skinny_res<Epi, NB, KW>),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, kSkinnyResLds);
    if (e != hipSuccess) (void)hipGetLastError();  // the batched kernel runs instead
    return e;
  }();
  if (attr != hipSuccess) return false;
  k_gemm_skinny_res<Epi, NB, KW><<<nb * splits, 256 * KW, bytes, st>>>(A, M, Wt, K, nb, per, part, n_cols, e, rn);
  return true;
}

// The activation-resident kernel takes grids of at most two workgroups per CU
// whose K groups hold at most 32 K blocks (1024 K) each (HH_SKINNY_RES=0 turns
// it off, for comparison); returns false when the batched kernel is to run.
template <class Epi>
static bool launch_skinny_res(hipStream_t st, const _Float16* A, int M, const _Float16* Wt, int K, int nb, int splits,
                              int per, float* part, int n_cols, int kw, const Epi& e, const RowNorm& rn) {
  if constexpr (std::is_same<Epi, EpiLogits>::value) {
    return false;
  } else {
    const char* v = getenv("HH_SKINNY_RES");
    const bool on = !(v && v[0] == '0');
    const int gmax = (per + kw - 1) / kw;
    // K-group tiles plus the 16-byte sink for unused chunks.
    const size_t lds = (size_t)kw * 32 * skinny_res_pitch(per, kw) * 2 + 16;
    if (!on || (long long)nb * splits > 2 * 256 || gmax > 32 || lds > (size_t)kSkinnyResLds) return false;
    const unsigned bytes = (unsigned)std::max<size_t>(lds, kSkinnyTileBytes);
    auto go = [&](auto nbc, auto kwc) {
      return skinny_res_go<Epi, decltype(nbc)::value, decltype(kwc)::value>(st, bytes, A, M, Wt, K, nb, splits, per,
                                                                            part, n_cols, e, rn);
    };
    using I1 = std::integral_constant<int, 1>;
    using I2 = std::integral_constant<int, 2>;
    if (kw == 2) {
      if (gmax <= 8) return go(std::integral_constant<int, 8>(), I2());
      if (gmax <= 16) return go(std::integral_constant<int, 16>(), I2());
      return go(std::integral_constant<int, 32>(), I2());
    }
    if (gmax <= 8) return go(std::integral_constant<int, 8>(), I1());
    if (gmax <= 16) return go(std::integral_constant<int, 16>(), I1());
    return go(std::integral_constant<int, 32>(), I1());
  }
}

// Returns the K splits, 0 when the shape does not fit the 32-row kernels.
// rn: see RowNorm; its producer half runs only in the activation-resident
// kernel of a split residual product (*fused = 1 then, and the partials are
// consumed in the kernel).
template <class Epi>
static int launch_skinny(hipStream_t st, GemmWorkspace ws, const _Float16* A, int M, const _Float16* Wt, int K,
                         int n_cols, const Epi& e, bool defer, RowNorm rn, int* fused) {
  if (fused) *fused = 0;
  // Buffer ranges take 31-bit byte offsets.
  if ((size_t)((n_cols + 15) / 16) * 16 * K * 2 >= ((size_t)1 << 31) || (size_t)32 * K * 2 >= ((size_t)1 << 31)) return 0;
  // The consumer half reads at most 32 block sums per row (a multiple of 4).
  if (rn.ss_in && (rn.nss > 32 || rn.nss % 4)) return 0;
  const int nb = (n_cols + 63) / 64;
  const int nk = K / 32;
  // Split K only to give about 256 workgroups, with at least 16 K blocks
  // (512 K) per split: at 32 rows the O and QKV products (64 K blocks) run
  // 4 splits, not 8 and 6 (step 1.002 -> 0.978 ms; the down projection keeps
  // 8, which 4 slowed).
  int splits = std::max(1, std::min((256 + nb - 1) / nb, nk / 16));
  while (splits > 1 && (size_t)splits * M * n_cols * sizeof(float) > ws.bytes) --splits;
  const int per = (nk + splits - 1) / splits;
  splits = (nk + per - 1) / per;
  float* part = splits > 1 ? ws.ptr : nullptr;
  if (!(std::is_same<Epi, EpiResid>::value && splits > 1 && n_cols % 64 == 0 && nb <= rn.ncnt)) rn.cnt = nullptr;
  // Unsplit (long) K ranges take two K groups per workgroup: eight waves per
  // CU keep more weight loads in flight (gate/up 17.0 -> 15.9 us at 32 rows).
  const int kw = splits == 1 ? 2 : 1;
  if (!launch_skinny_res<Epi>(st, A, M, Wt, K, nb, splits, per, part, n_cols, kw, e, rn)) {
    rn.cnt = nullptr;
    if (kw == 2)
      k_gemm_skinny<Epi, 8, 2><<<nb * splits, 512, 0, st>>>(A, M, Wt, K, nb, per, part, n_cols, e, rn);
    else
      k_gemm_skinny<Epi, 8, 1><<<nb * splits, 256, 0, st>>>(A, M, Wt, K, nb, per, part, n_cols, e, rn);
  }
  if (rn.cnt) {
    if (fused) *fused = 1;
    return splits;
  }
  if (splits > 1 && !defer)
    k_splitk_finalize<Epi><<<((M + kFinRows - 1) / kFinRows) * ((n_cols + 127) / 128), 256, 0, st>>>(
        part, splits, M, n_cols, (n_cols + 127) / 128, e);
  return splits;
}

// RowNorm consumer fallback for products that no 32-row kernel takes: scale
// the rows of A (x * gain as fp16) in place by their norm factors.
__global__ __launch_bounds__(256) void k_rownorm_apply(_Float16* __restrict__ A, int K, RowNorm rn) {
  __shared__ float red[4];
  const int row = blockIdx.x;
  float v = 0.f;
  if (threadIdx.x == 0)
    for (int j = 0; j < rn.nss; ++j) v += rn.ss_in[(size_t)row * rn.nss + j];
  const float inv = rsqrtf(block_sum256(v, red) / rn.n + rn.eps);
  for (int k = threadIdx.x; k < K; k += 256) A[(size_t)row * K + k] = (_Float16)((float)A[(size_t)row * K + k] * inv);
}

// Tile choice of a prompt-sized GEMM: {BM, BN, splits}, BM == 0 for the
// small-tile kernel.  HH_GEMM_QKV / _RESID (O projection) / _DOWN / _GATEUP =
// "BMxBNxS" (or "0") overrides it, for tuning.
struct WideCfg {
  int bm, bn, splits, nw;  // nw: waves per workgroup (4 or 8)
};

static WideCfg wide_choice(GemmKind kind, int M, int n_cols, int K) {
  static const char* names[4] = {"HH_GEMM_QKV", "HH_GEMM_RESID", "HH_GEMM_GATEUP", "HH_GEMM_LOGITS"};
  // The down projection (K > N) has a knob of its own.
  const char* env = getenv(kind == GemmKind::Resid && K > n_cols ? "HH_GEMM_DOWN" : names[(int)kind]);
  if (env) {
    WideCfg c{0, 0, 1, 4};
    if (sscanf(env, "%dx%dx%dx%d", &c.bm, &c.bn, &c.splits, &c.nw) >= 2) return c;
    return WideCfg{0, 0, 1, 4};
  }
  // Measured on the 1B prompt shapes (d 2048, FFN 8192): gate/up at 1024 rows
  // takes 256 x 128 tiles (512 tiles, two rounds of the CUs; TTFT 3.74 ->
  // 3.44 ms against 256 x 256, one tile per CU); the down and O projections
  // (only 128 tiles of 128 x 128) gain most from a 2-way K split; everything
  // at 256 rows stays on the small-tile kernel, whose two workgroups per CU
  // suit these few-tile shapes better.
  if (kind == GemmKind::GateUp && n_cols >= 8192) {
    // Eight waves (two per SIMD) here: TTFT at 1024 rows 3.66 -> 3.57 ms;
    // every other shape was slower with eight.
    if (M >= 512) return WideCfg{256, 128, 1, 8};
    if (M >= 256) return WideCfg{128, 128, 1, 4};
  }
  // O and down at >= 512 rows: 128 x 128 tiles, 2-way K split, eight waves
  // (O 17.5 -> 16.3 us, down 45.6 -> 44.2 us at 1024 rows against four).
  if (kind == GemmKind::Resid && M >= 512) return WideCfg{128, 128, 2, 8};
  // QKV at >= 512 rows: 128 x 128 tiles, no split (its epilogue loads its
  // rotations and KV pages ahead of the stores): TTFT at 1024 rows 3.41 ->
  // 3.34 ms against the small-tile kernel, which stays better at 256 rows;
  // eight waves 29.3 -> 28.1 us.
  if (kind == GemmKind::QKV && M >= 512) return WideCfg{128, 128, 1, 8};
  // QKV at 256 .. 511 rows: the same tiles with a 4-way K split (192
  // workgroups; the split-K reduction applies the epilogue): TTFT at 256
  // rows 1.68-1.69 -> 1.64 ms against the small-tile kernel's 3-way split
  // (2-, 3- and 6-way splits, four waves and 128 x 256 tiles all slower).
  if (kind == GemmKind::QKV && M >= 256) return WideCfg{128, 128, 4, 8};
  return WideCfg{0, 0, 1, 4};
}

// Returns the splits used, 0 when the shape is left to the small-tile kernel.
template <class Epi>
static int run_wide(hipStream_t st, GemmWorkspace ws, const _Float16* A, int M, const _Float16* W, int K, int n_cols,
                    const Epi& e, GemmKind kind, bool defer) {
  if (kind == GemmKind::Logits || M < 128) return 0;
  const WideCfg c = wide_choice(kind, M, n_cols, K);
  if (c.nw == 8) {
    if (c.bm == 256 && c.bn == 256) return launch_wide<256, 256, 8>(st, ws, A, M, W, K, n_cols, c.splits, e, defer);
    if (c.bm == 256 && c.bn == 128) return launch_wide<256, 128, 8>(st, ws, A, M, W, K, n_cols, c.splits, e, defer);
    if (c.bm == 128 && c.bn == 256) return launch_wide<128, 256, 8>(st, ws, A, M, W, K, n_cols, c.splits, e, defer);
    if (c.bm == 128 && c.bn == 128) return launch_wide<128, 128, 8>(st, ws, A, M, W, K, n_cols, c.splits, e, defer);
    return 0;
  }
  if (c.bm == 256 && c.bn == 256) return launch_wide<256, 256>(st, ws, A, M, W, K, n_cols, c.splits, e, defer);
  if (c.bm == 256 && c.bn == 128) return launch_wide<256, 128>(st, ws, A, M, W, K, n_cols, c.splits, e, defer);
  if (c.bm == 128 && c.bn == 256) return launch_wide<128, 256>(st, ws, A, M, W, K, n_cols, c.splits, e, defer);
  if (c.bm == 128 && c.bn == 128) return launch_wide<128, 128>(st, ws, A, M, W, K, n_cols, c.splits, e, defer);
  return 0;
}

// Run C = A W^T over n_cols logical columns with epilogue e; returns the K
// splits used (with defer, partials of a split run are left in ws.ptr).
// rn (fp16 operands only): RowNorm's consumer and producer halves, honoured
// by the 32-row kernels; a consumer request that no 32-row kernel takes
// scales A's rows first, and *fused says whether the producer half ran.
template <typename TM, class Epi>
static int run_gemm(hipStream_t st, GemmWorkspace ws, const TM* A, int M, const TM* W, int K, int n_cols, const Epi& e,
                    GemmKind kind, bool defer = false, const TM* Wt = nullptr, const RowNorm& rn = RowNorm(),
                    int* fused = nullptr) {
  if (fused) *fused = 0;
  if constexpr (sizeof(TM) == 2) {
    if (M <= 32 && Wt && K % 64 == 0) {
      const int sp = launch_skinny(st, ws, reinterpret_cast<const _Float16*>(A), M,
                                   reinterpret_cast<const _Float16*>(Wt), K, n_cols, e, defer, rn, fused);
      if (sp > 0) return sp;
    }
    if (rn.ss_in)
      k_rownorm_apply<<<M, 256, 0, st>>>(reinterpret_cast<_Float16*>(const_cast<TM*>(A)), K, rn);
    if (K % 64 == 0) {
      const _Float16* Ah = reinterpret_cast<const _Float16*>(A);
      const _Float16* Wh = reinterpret_cast<const _Float16*>(W);
      if constexpr (!std::is_same<Epi, EpiLogits>::value) {
        const int sp = run_wide(st, ws, Ah, M, Wh, K, n_cols, e, kind, defer);
        if (sp > 0) return sp;
      }
      const long long ntn = (n_cols + 127) / 128;
      if (M <= 32) return launch_f16<32>(st, ws, Ah, M, Wh, K, n_cols, e, defer);
      if (M <= 64 || ((M + 127) / 128) * ntn < 256) return launch_f16<64>(st, ws, Ah, M, Wh, K, n_cols, e, defer);
      return launch_f16<128>(st, ws, Ah, M, Wh, K, n_cols, e, defer);
    }
  }
  k_gemm<TM, Epi><<<dim3((n_cols + GBN - 1) / GBN, (M + GBM - 1) / GBM), 256, 0, st>>>(A, M, W, K, e);
  return 1;
}

// ---------------------------------------------------------------- residual + RMSNorm

// One row per workgroup: x[row] += (sum of the split partials, in split
// order) * scale when splits > 0, then h[row] = x[row] * rsqrt(mean(x^2) +
// eps) * gain in the MFMA operand type.  The row (N % 4 == 0, N <= 4096) stays
// in registers between the two halves.
constexpr int kNormMaxChunks = 4;  // float4 chunks per thread: N <= 4096
constexpr int kNormSplitBatch = 8;  // split partials in flight per chunk
template <typename TM>
__global__ __launch_bounds__(256) void k_resid_norm(const float* __restrict__ partial, int splits, int M, int N, float scale,
                                                    float* __restrict__ x, const float* __restrict__ gain, float eps,
                                                    TM* __restrict__ h) {
  __shared__ float red[4];
  const int row = blockIdx.x, nc = N >> 2;
  float4* xr = reinterpret_cast<float4*>(x + (size_t)row * N);
  float4 v[kNormMaxChunks], g[kNormMaxChunks];
  // The gains load with the row, so the second half waits on no global load.
#pragma unroll
  for (int k = 0; k < kNormMaxChunks; ++k) {
    const int ch = threadIdx.x + 256 * k;
    if (ch < nc) g[k] = reinterpret_cast<const float4*>(gain)[ch];
  }
  float ss = 0.f;
#pragma unroll
  for (int k = 0; k < kNormMaxChunks; ++k) {
    const int ch = threadIdx.x + 256 * k;
    if (ch < nc) {
      float4 a = xr[ch];
      if (splits > 0) {
        const float4* pp = reinterpret_cast<const float4*>(partial + (size_t)row * N) + ch;
        const size_t stride = (size_t)M * nc;  // one split's partials, in float4
        // Up to kNormSplitBatch partials are loaded at once (clamped indices,
        // unused ones dropped), then summed in split order.
        float4 t = pp[0];
        for (int s0 = 1; s0 < splits; s0 += kNormSplitBatch) {
          float4 u[kNormSplitBatch];
#pragma unroll
          for (int j = 0; j < kNormSplitBatch; ++j) u[j] = pp[min(s0 + j, splits - 1) * stride];
#pragma unroll
          for (int j = 0; j < kNormSplitBatch; ++j)
            if (s0 + j < splits) {
              t.x += u[j].x;
              t.y += u[j].y;
              t.z += u[j].z;
              t.w += u[j].w;
            }
        }
        a.x += t.x * scale;
        a.y += t.y * scale;
        a.z += t.z * scale;
        a.w += t.w * scale;
        xr[ch] = a;
      }
      v[k] = a;
      ss += a.x * a.x + a.y * a.y + a.z * a.z + a.w * a.w;
    }
  }
  const float inv = rsqrtf(block_sum256(ss, red) / (float)N + eps);
#pragma unroll
  for (int k = 0; k < kNormMaxChunks; ++k) {
    const int ch = threadIdx.x + 256 * k;
    if (ch < nc) {
      const float4 gk = g[k];
      TM* hr = h + (size_t)row * N + 4 * ch;
      if constexpr (sizeof(TM) == 2) {
        typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
        const f16x4 o = {(_Float16)(v[k].x * inv * gk.x), (_Float16)(v[k].y * inv * gk.y),
                         (_Float16)(v[k].z * inv * gk.z), (_Float16)(v[k].w * inv * gk.w)};
        *reinterpret_cast<f16x4*>(hr) = o;
      } else {
        *reinterpret_cast<float4*>(hr) = make_float4(v[k].x * inv * gk.x, v[k].y * inv * gk.y, v[k].z * inv * gk.z,
                                                     v[k].w * inv * gk.w);
      }
    }
  }
}

template <typename TM, typename TKV>
void GemmKernels<TM, TKV>::qkv(hipStream_t st, GemmWorkspace ws, const TM* A, int M, const TM* W, int d, int hq, int hkv, float scale,
                               const int* row_stream, const int* row_pos, const float2* rope, float* q, TM* qM,
                               TKV* kv, KvLayout L, int layer, const int* page_table, const TM* Wt) {
  EpiQKV<TKV> e{hq, hkv, scale, row_stream, row_pos, rope, q, reinterpret_cast<TKV*>(qM), kv, L, layer, page_table};
  run_gemm<TM>(st, ws, A, M, W, d, (hq + 2 * hkv) * 64, e, GemmKind::QKV, false, Wt);
}

template <typename TM, typename TKV>
int GemmKernels<TM, TKV>::qkv_deferred(hipStream_t st, GemmWorkspace ws, const TM* A, int M, const TM* W, int d, int hq,
                                       int hkv, float scale, const int* row_stream, const int* row_pos,
                                       const float2* rope, float* q, TKV* kv, KvLayout L, int layer,
                                       const int* page_table, const TM* Wt, const RowNorm& rn) {
  EpiQKV<TKV> e{hq, hkv, scale, row_stream, row_pos, rope, q, nullptr, kv, L, layer, page_table};
  return run_gemm<TM>(st, ws, A, M, W, d, (hq + 2 * hkv) * 64, e, GemmKind::QKV, true, Wt, rn);
}

template <typename TM, typename TKV>
bool GemmKernels<TM, TKV>::norm_fusable(int N) {
  return N % 4 == 0 && N <= 4 * 256 * kNormMaxChunks;
}

template <typename TM, typename TKV>
bool GemmKernels<TM, TKV>::resid(hipStream_t st, GemmWorkspace ws, const TM* A, int M, const TM* W, int K, int N,
                                 float scale, float* x, const float* gain, float eps, TM* h, const TM* Wt, float* ss,
                                 int* cnt, int ncnt) {
  EpiResid e{N, scale, x};
  const bool norm = gain != nullptr;
  RowNorm rn;
  if constexpr (sizeof(TM) == 2) {
    if (norm && ss && cnt) {
      rn.cnt = cnt;
      rn.ncnt = ncnt;
      rn.gain = gain;
      rn.y = reinterpret_cast<_Float16*>(h);
      rn.ss_out = ss;
    }
  }
  int fused = 0;
  const int sp = run_gemm<TM>(st, ws, A, M, W, K, N, e, GemmKind::Resid, norm, Wt, rn, &fused);
  if (norm && !fused) k_resid_norm<TM><<<M, 256, 0, st>>>(ws.ptr, sp > 1 ? sp : 0, M, N, scale, x, gain, eps, h);
  return fused != 0;
}

template <typename TM, typename TKV>
void GemmKernels<TM, TKV>::rmsnorm(hipStream_t st, int M, float* x, int N, const float* gain, float eps, TM* h) {
  k_resid_norm<TM><<<M, 256, 0, st>>>(nullptr, 0, M, N, 1.f, x, gain, eps, h);
}

template <typename TM, typename TKV>
void GemmKernels<TM, TKV>::gateup(hipStream_t st, GemmWorkspace ws, const TM* A, int M, const TM* W, int d, int F, float scale,
                                  TM* m, const TM* Wt, const RowNorm& rn) {
  // Groups of 32 gate + 32 up columns: every tile width here is a multiple of 64.
  EpiGateUp<TM> e{F, 32, scale, m};
  run_gemm<TM>(st, ws, A, M, W, d, ((F + 31) / 32) * 64, e, GemmKind::GateUp, false, Wt, rn);
}

template <typename TM, typename TKV>
void GemmKernels<TM, TKV>::logits(hipStream_t st, GemmWorkspace ws, const TM* A, int M, const TM* W, int d, int V, float scale,
                                  float* logits, unsigned long long* slot, const int* row_stream, const TM* Wt,
                                  const RowNorm& rn) {
  EpiLogits e{V, scale, logits, slot, row_stream};
  run_gemm<TM>(st, ws, A, M, W, d, V, e, GemmKind::Logits, false, Wt, rn);
}

template struct GemmKernels<float, float>;
template struct GemmKernels<_Float16, _Float16>;

}  // namespace hh
