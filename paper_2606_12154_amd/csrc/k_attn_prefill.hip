// Causal GQA flash attention for prompt prefill on gfx950 MFMA (fp16 KV).
//
// A workgroup owns one block of 32 query positions and one kv head g; wave w
// serves query head g * G + w.  Per block of 32 keys (two KV pages):
//   S^T[key][query] = K[key][:] . Q[query][:]      4 x mfma_f32_32x32x16_f16
// so a lane holds 16 keys of ONE query column (lane % 32), and the row max /
// sum of the online softmax need a single exchange with lane ^ 32.  Then
//   O^T[dim][query] += V^T[dim][key] P^T[key][query]   4 x mfma 32x32x16
// where the second contraction's K index is ordered to match the keys each
// lane already holds in S^T (j -> key 16t + 8(j/4) + 4h + j%4 for lane half h),
// so P goes from the accumulator straight into the B operand.  K and V^T of
// a key block are staged once per workgroup in LDS (all waves read them), so
// each lane's K operand is one 16-byte read and its V^T operand two 8-byte
// reads.
// Result lane layout of a 32x32 MFMA: element i of lane l is row
// 8(i/4) + 4(l/32) + i%4, column l%32.
#include "hh_kernels.h"

namespace hh {

constexpr int kFlashMaxPages = 2048;  // pages of keys per prefill attention (32768 positions)

typedef float f32x16 __attribute__((ext_vector_type(16)));

// The next key blocks' K fragments and V slices are loaded into further
// register sets while the current block is processed (sets in strict
// rotation, loads issued unconditionally with clamped keys, so the compiler
// waits for exactly the oldest set), and V^T is double-buffered in LDS so each
// block needs a single barrier.
struct KvRegs {
  f16x8 k, v;  // key idx / 8 of the block, dims (idx % 8) * 8 .. + 8, for this thread's idx
};

// pt: the stream's page-table slice in LDS (a global read here would make
// every prefetch wait, in order, for all loads before it).
__device__ __forceinline__ void flash_load(KvRegs& R, const _Float16* __restrict__ kv, const KvLayout& L, int layer,
                                           const int* pt, int g, int k0, int kend) {
  const int idx = threadIdx.x & 255;
  const int key = min(k0 + (idx >> 3), kend - 1), dc = idx & 7;
  const size_t off = (size_t)(key & 15) * 64 + dc * 8;
  const int page = pt[key >> 4];
  R.k = *reinterpret_cast<const f16x8*>(kv + L.head_tile(layer, page, 0, g) + off);
  R.v = *reinterpret_cast<const f16x8*>(kv + L.head_tile(layer, page, 1, g) + off);
}

template <int G>
__global__ __launch_bounds__(64 * G) void k_flash_prefill(const _Float16* __restrict__ qM, const _Float16* __restrict__ kv,
                                                          KvLayout L, int layer, const int* __restrict__ page_table,
                                                          int s, int p0, int n_rows, int hq, _Float16* __restrict__ oM) {
  static_assert(G >= 4, "the V slice of a key block needs 256 threads");
  constexpr int VT_LD = 32 + 8;  // padded row of V^T (halfs)
  constexpr int KT_LD = 64 + 8;  // padded row of K (halfs)
  __shared__ __attribute__((aligned(16))) _Float16 vt[2][64 * VT_LD];
  __shared__ __attribute__((aligned(16))) _Float16 kt[2][32 * KT_LD];
  __shared__ int pt[kFlashMaxPages];  // physical pages of keys 0 .. kend-1
  const int g = blockIdx.y;
  const int qb = gridDim.x - 1 - blockIdx.x;  // longest (latest) query blocks first
  const int q0 = qb * 32;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int j = g * G + wave;
  const int h = lane >> 5, c = lane & 31;
  const int qrow = q0 + c;
  const bool qvalid = qrow < n_rows;
  const int qpos = p0 + qrow;
  const float scale = 0.125f * 1.4426950408889634f;  // 1/sqrt(64) * log2(e)

  f16x8 qf[4];
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) {
    if (qvalid) qf[ks] = *reinterpret_cast<const f16x8*>(qM + ((size_t)qrow * hq + j) * 64 + 16 * ks + 8 * h);
    else qf[ks] = f16x8{0, 0, 0, 0, 0, 0, 0, 0};
  }
  float m = -INFINITY, lsum = 0.f;
  f32x16 o0, o1;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    o0[i] = 0.f;
    o1[i] = 0.f;
  }
  const int kend = min(p0 + q0 + 32, p0 + n_rows);  // keys 0 .. kend-1 exist for this block
  const int nkb = (kend + 31) / 32;
  {
    const int* src = page_table + (size_t)s * L.max_pages;
    for (int i = threadIdx.x; i < (kend + kPage - 1) / kPage; i += blockDim.x) pt[i] = src[i];
    __syncthreads();
  }

  auto process = [&](const KvRegs& R, int kb) {
    const int k0 = kb * 32;
    _Float16* vb = vt[kb & 1];
    _Float16* kbuf = kt[kb & 1];
    // Stage K and V^T of this key block once for all waves (threads 0..255:
    // key idx / 8, dims (idx % 8) * 8 .. + 8).
    if (threadIdx.x < 256) {
      const int key = threadIdx.x >> 3, dc = threadIdx.x & 7;
      const bool ok = k0 + key < kend;
      *reinterpret_cast<f16x8*>(kbuf + key * KT_LD + dc * 8) = R.k;
#pragma unroll
      for (int e = 0; e < 8; ++e) vb[(dc * 8 + e) * VT_LD + key] = ok ? R.v[e] : (_Float16)0.f;
    }
    __syncthreads();

    f32x16 sacc;
#pragma unroll
    for (int i = 0; i < 16; ++i) sacc[i] = 0.f;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const f16x8 kf = *reinterpret_cast<const f16x8*>(kbuf + c * KT_LD + 16 * ks + 8 * h);
      sacc = __builtin_amdgcn_mfma_f32_32x32x16_f16(kf, qf[ks], sacc, 0, 0, 0);
    }

    float bm = -INFINITY;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int kk = k0 + 8 * (i >> 2) + 4 * h + (i & 3);
      float v = sacc[i] * scale;
      if (kk > qpos || kk >= kend) v = -INFINITY;
      sacc[i] = v;
      bm = fmaxf(bm, v);
    }
    bm = fmaxf(bm, __shfl_xor(bm, 32, 64));
    const float mn = fmaxf(m, bm);  // finite: key 0 of block 0 is visible to every query
    const float alpha = exp2f(m - mn);
    float ls = 0.f;
    f16x8 pb[2];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const float pv = exp2f(sacc[i] - mn);
      ls += pv;
      pb[i >> 3][i & 7] = (_Float16)pv;
    }
    lsum = lsum * alpha + ls;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      o0[i] *= alpha;
      o1[i] *= alpha;
    }
#pragma unroll
    for (int t2 = 0; t2 < 2; ++t2) {
      // A operand: V^T[dim][keys 16 t2 + 4 h + {0..3, 8..11}] for dims c and c + 32.
      f16x8 a0, a1;
      const _Float16* r0 = vb + c * VT_LD + 16 * t2 + 4 * h;
      const _Float16* r1 = vb + (c + 32) * VT_LD + 16 * t2 + 4 * h;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        a0[e] = r0[e];
        a0[4 + e] = r0[8 + e];
        a1[e] = r1[e];
        a1[4 + e] = r1[8 + e];
      }
      o0 = __builtin_amdgcn_mfma_f32_32x32x16_f16(a0, pb[t2], o0, 0, 0, 0);
      o1 = __builtin_amdgcn_mfma_f32_32x32x16_f16(a1, pb[t2], o1, 0, 0, 0);
    }
    m = mn;
  };

  // Three register sets in rotation: blocks kb + 1 and kb + 2 are in flight
  // while block kb is processed.
  KvRegs A, B, C;
  flash_load(A, kv, L, layer, pt, g, 0, kend);
  flash_load(B, kv, L, layer, pt, g, min(1, nkb - 1) * 32, kend);
  for (int kb = 0; kb < nkb; kb += 3) {
    flash_load(C, kv, L, layer, pt, g, min(kb + 2, nkb - 1) * 32, kend);
    process(A, kb);
    if (kb + 1 >= nkb) break;
    flash_load(A, kv, L, layer, pt, g, min(kb + 3, nkb - 1) * 32, kend);
    process(B, kb + 1);
    if (kb + 2 >= nkb) break;
    flash_load(B, kv, L, layer, pt, g, min(kb + 4, nkb - 1) * 32, kend);
    process(C, kb + 2);
  }
  const float ltot = lsum + __shfl_xor(lsum, 32, 64);
  if (qvalid) {
    const float inv = 1.f / ltot;
    _Float16* dst = oM + ((size_t)qrow * hq + j) * 64;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int dim = 8 * (i >> 2) + 4 * h + (i & 3);
      dst[dim] = (_Float16)(o0[i] * inv);
      dst[dim + 32] = (_Float16)(o1[i] * inv);
    }
  }
}

bool flash_prefill_supported(int G, int max_context) {
  return (G == 4 || G == 8) && (max_context + kPage - 1) / kPage <= kFlashMaxPages;
}

void flash_prefill(hipStream_t st, const _Float16* qM, const _Float16* kv, KvLayout L, int layer,
                   const int* page_table, int s, int p0, int n_rows, int hq, int hkv, _Float16* oM) {
  const int G = hq / hkv;
  dim3 grid((n_rows + 31) / 32, hkv);
  switch (G) {
    case 4: k_flash_prefill<4><<<grid, 256, 0, st>>>(qM, kv, L, layer, page_table, s, p0, n_rows, hq, oM); break;
    default: k_flash_prefill<8><<<grid, 512, 0, st>>>(qM, kv, L, layer, page_table, s, p0, n_rows, hq, oM); break;
  }
}

}  // namespace hh
