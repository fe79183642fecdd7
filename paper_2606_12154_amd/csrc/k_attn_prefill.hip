// Causal GQA flash attention for prompt prefill on gfx950 MFMA (fp16 KV).
//
// A workgroup owns two blocks of 32 query positions, p and the mirror block
// from the end (so every workgroup has the same causal work), and half of kv
// head g's query heads.  Its waves form NS key-split groups of G waves; a
// group's waves serve (query block, head) pairs, and group s takes key blocks
// s, s + NS, s + 2 NS, ... of 32 keys (two KV pages) of the longer block, so
// the longest dependency chain is 1/NS of the keys and every SIMD runs four
// waves that hide each other's latencies.  Per key block:
//   S^T[key][query] = K[key][:] . Q[query][:]      4 x mfma_f32_32x32x16_f16
// so a lane holds 16 keys of ONE query column (lane % 32), and the row max /
// sum of the online softmax need a single exchange with lane ^ 32.  Then
//   O^T[dim][query] += V^T[dim][key] P^T[key][query]   4 x mfma 32x32x16
// where the second contraction's K index is ordered to match the keys each
// lane already holds in S^T (j -> key 16t + 8(j/4) + 4h + j%4 for lane half h),
// so P goes from the accumulator straight into the B operand.  K and V^T of a
// key block are staged once per group in LDS (the group's waves all read
// them).  At the end the groups' (max, sum, output) triples are merged in LDS
// by group 0 in split order.
// Result lane layout of a 32x32 MFMA: element i of lane l is row
// 8(i/4) + 4(l/32) + i%4, column l%32.
#include "hh_kernels.h"

namespace hh {

constexpr int kFlashMaxPages = 8192;  // pages of keys per prefill attention (131072 positions)

typedef float f32x16 __attribute__((ext_vector_type(16)));

// Thread idx of a group stages, of the block's 32 keys,
//   K: key idx / 8, dims 8 (idx % 8) .. + 8 (a wave reads 8 whole 128-byte rows);
//   V: key idx % 32, dims 8 (idx / 32) .. + 8, so a wave's transposed V^T
//      stores (one half per lane and dim) cover all 32 keys of two dim chunks
//      and spread over every LDS bank instead of piling onto four.
struct KvRegs {
  f16x8 k, v;
};

// pt: the stream's page-table slice in LDS (a global read here would make
// every prefetch wait, in order, for all loads before it).  idx: the thread's
// index within its group (0 .. 255 stage a block).
// Keys of kv head g in one layer, addressed with 32-bit element offsets from
// the head's first tile (flash_prefill_supported bounds a layer's cache).
struct FlashKv {
  const _Float16* base;   // head_tile(layer, 0, 0, g)
  unsigned page_stride;   // elements between pages: 2 (K, V) x heads x one tile
  unsigned v_off;         // V tile of a page after its K tile
};
__device__ __forceinline__ void flash_load(KvRegs& R, const FlashKv& A, const int* pt, int idx, int k0, int kend) {
  const int kk = min(k0 + (idx >> 3), kend - 1), kd = idx & 7;
  const int vk = min(k0 + (idx & 31), kend - 1), vd = idx >> 5;
  const unsigned ko = (unsigned)pt[kk >> 4] * A.page_stride + (unsigned)((kk & 15) * 64 + kd * 8);
  const unsigned vo = (unsigned)pt[vk >> 4] * A.page_stride + A.v_off + (unsigned)((vk & 15) * 64 + vd * 8);
  R.k = *reinterpret_cast<const f16x8*>(A.base + ko);
  R.v = *reinterpret_cast<const f16x8*>(A.base + vo);
}

template <int G, int NS>
struct FlashCfg {
  static constexpr int THREADS = 64 * G * NS;
  // Padded row of V^T (halfs): 18 banks per row, so the two dim chunks of a
  // wave's transposed stores (rows 8 apart) fall 16 banks apart, and the
  // fragment reads (8 bytes, rows c = 0..31) cover every bank equally.
  static constexpr int VT_LD = 32 + 4;
  static constexpr int KT_LD = 64 + 8;                 // padded row of K (halfs)
  static constexpr int BUF = (64 * VT_LD + 32 * KT_LD) * 2;  // one staged key block, bytes
  static constexpr int STAGE = NS * 2 * BUF;           // double-buffered, per group
  // Merge area: groups 1 .. NS-1 leave m, l (64 lanes) and o (32 values x 64 lanes) per wave.
  static constexpr int MERGE = (NS - 1) * G * (2 + 32) * 64 * 4;
  static constexpr int PT = kFlashMaxPages * 4;
  static constexpr int LDS = (STAGE > MERGE ? STAGE : MERGE) + PT;
  static_assert(G * 64 >= 256, "a group stages a key block with 256 threads");
  static_assert(THREADS <= 1024, "workgroup size");
  static_assert(LDS <= 160 * 1024, "LDS");
};

template <int G, int NS>
__global__ __launch_bounds__(64 * G * NS) void k_flash_prefill(const _Float16* __restrict__ qM,
                                                               const _Float16* __restrict__ kv, KvLayout L, int layer,
                                                               const int* __restrict__ page_table, int s, int p0,
                                                               int n_rows, int hq, _Float16* __restrict__ oM) {
  using C = FlashCfg<G, NS>;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  int* pt = reinterpret_cast<int*>(smem + (C::LDS - C::PT));  // physical pages of keys 0 .. kend-1
  // Causal work is balanced by pairing query blocks: workgroup (p, g, hh)
  // serves query blocks p and nqb - 1 - p (together nqb + 1 key blocks, the
  // same for every pair) for the query heads g G + hh G/2 .. + G/2 - 1.  In
  // each group, waves 0 .. G/2 - 1 take one block and the others the second,
  // alternating with the group index: a SIMD runs wave w of every group, so
  // each SIMD gets waves of both blocks and none idles once the short block
  // is done.
  constexpr int GH = G / 2;  // query heads per workgroup
  const int g = blockIdx.y, hh = blockIdx.z;
  const int nqb = (n_rows + 31) / 32;
  const int p = blockIdx.x;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int hi = wave % G, grp = wave / G;
  const int qsel = ((hi / GH) + grp) & 1;                  // 0: block p, 1: block nqb - 1 - p
  const int qb = qsel ? nqb - 1 - p : p;
  const bool active = qsel == 0 || nqb - 1 - p != p;     // an odd count's middle block is served once
  const int q0 = qb * 32;
  const int idx = threadIdx.x - grp * 64 * G;  // thread index within the group
  // Threads 0..255 of a group load and stage its key blocks.  With 256-thread
  // groups that is every thread, and the condition must be visibly true:
  // loads under a runtime branch make the compiler's wait counts assume the
  // branch skipped them, so each block's wait would also wait for the next
  // block's loads.
  const bool stager = G * 64 == 256 || idx < 256;
  const int j = g * G + hh * GH + hi % GH;
  const int h = lane >> 5, c = lane & 31;
  const int qrow = q0 + c;
  const bool qvalid = active && qrow < n_rows;
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
  // This wave's query block sees keys 0 .. kend - 1; the workgroup stages
  // key blocks for the longer block of the pair (keys 0 .. kend_all - 1).
  const int kend = min(p0 + q0 + 32, p0 + n_rows);
  const int nkb = active ? (kend + 31) / 32 : 0;
  const int kend_all = min(p0 + (nqb - 1 - p) * 32 + 32, p0 + n_rows);
  const int nkb_all = (kend_all + 31) / 32;
  const int niter = (nkb_all + NS - 1) / NS;        // the same for every group (uniform barriers)
  // Arrival counters of the NS groups' per-iteration barriers.
  __shared__ int gsync[NS];
  if (threadIdx.x < NS) gsync[threadIdx.x] = 0;
  {
    const int* src = page_table + (size_t)s * L.max_pages;
    for (int i = threadIdx.x; i < (kend_all + kPage - 1) / kPage; i += blockDim.x) pt[i] = src[i];
    __syncthreads();
  }
  // Barrier among the G waves of this thread's group only: groups share no
  // staging buffer, so each runs at its own pace and a SIMD (one wave of
  // every group) overlaps one group's MFMAs with another's softmax instead of
  // running them in lock step.  The arrival is counted once this wave's LDS
  // stores have completed; the wait is bounded (it cannot miss in a correct
  // run: every wave of a group arrives once per iteration).
  auto group_sync = [&](int it) {
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): this wave's staging stores are done
    if (lane == 0) __hip_atomic_fetch_add(&gsync[grp], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    const int target = G * (it + 1);
    for (int spin = 0; spin < (1 << 24); ++spin) {
      if (__hip_atomic_load(&gsync[grp], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP) >= target) break;
      __builtin_amdgcn_s_sleep(1);
    }
    asm volatile("" ::: "memory");  // the staged block is read only after the wait
  };

  char* gbase = smem + grp * 2 * C::BUF;
  auto process = [&](const KvRegs& R, int it) {
    const int kb = it * NS + grp;
    const int k0 = kb * 32;
    const bool staged = kb < nkb_all, have = kb < nkb;
    _Float16* vb = reinterpret_cast<_Float16*>(gbase + (it & 1) * C::BUF);
    _Float16* kbuf = vb + 64 * C::VT_LD;
    // Stage K and V^T of this key block once for the group's waves (the
    // thread-to-key maps of flash_load).
    if (staged && stager) {
      *reinterpret_cast<f16x8*>(kbuf + (idx >> 3) * C::KT_LD + (idx & 7) * 8) = R.k;
      const int vk = idx & 31, vd = idx >> 5;
      const bool ok = k0 + vk < kend_all;
#pragma unroll
      for (int e = 0; e < 8; ++e) vb[(vd * 8 + e) * C::VT_LD + vk] = ok ? R.v[e] : (_Float16)0.f;
    }
    // Buffers alternate, so one barrier per iteration orders this write
    // after every read of the same buffer two iterations ago.
    group_sync(it);
    if (!have) return;

    f32x16 sacc;
#pragma unroll
    for (int i = 0; i < 16; ++i) sacc[i] = 0.f;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const f16x8 kf = *reinterpret_cast<const f16x8*>(kbuf + c * C::KT_LD + 16 * ks + 8 * h);
      sacc = __builtin_amdgcn_mfma_f32_32x32x16_f16(kf, qf[ks], sacc, 0, 0, 0);
    }

    // The softmax is the VALU side of the loop (four waves per SIMD share it
    // while the MFMAs are short), so it does only what a block needs: keys
    // past a query (causal) or past the block's end exist only in blocks
    // that reach the diagonal (wave-uniform test), the scale folds into the
    // exponent's FMA (the max is taken on raw scores: scaling by a positive
    // factor keeps the order), and a query's reference m moves only when
    // the block's max exceeds it by more than kLazy (log2 units), so the
    // output is rescaled in few blocks (alpha is exactly 1 otherwise).
    // Weights are then at most 2^kLazy, which fp16 holds with its full
    // relative precision; the final (m, l, o) stay consistent.
    if (k0 + 31 > p0 + q0 || k0 + 32 > kend) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int kk = k0 + 8 * (i >> 2) + 4 * h + (i & 3);
        if (kk > qpos || kk >= kend) sacc[i] = -INFINITY;
      }
    }
    float bm = -INFINITY;
#pragma unroll
    for (int i = 0; i < 16; ++i) bm = fmaxf(bm, sacc[i]);
    bm = fmaxf(bm, __shfl_xor(bm, 32, 64)) * scale;
    // A group's first blocks may hide every key from some query of an
    // appended chunk: keep such a query's state at (-inf, 0, 0).
    constexpr float kLazy = 8.f;
    const float mn = bm > m + kLazy ? bm : m;  // m = -inf: any finite bm
    const float mref = mn == -INFINITY ? 0.f : mn;
    // Hardware exp2 (arguments are <= 0 up to the product's rounding; results
    // below the normal range flush to zero, which a softmax weight can take).
    const float alpha = __builtin_amdgcn_exp2f(m - mref);
    float ls = 0.f;
    f16x8 pb[2];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const float pv = __builtin_amdgcn_exp2f(fmaf(sacc[i], scale, -mref));
      ls += pv;
      pb[i >> 3][i & 7] = (_Float16)pv;
    }
    lsum = lsum * alpha + ls;
    if (__builtin_amdgcn_ballot_w64(alpha != 1.f)) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        o0[i] *= alpha;
        o1[i] *= alpha;
      }
    }
#pragma unroll
    for (int t2 = 0; t2 < 2; ++t2) {
      // A operand: V^T[dim][keys 16 t2 + 4 h + {0..3, 8..11}] for dims c and c + 32.
      f16x8 a0, a1;
      const _Float16* r0 = vb + c * C::VT_LD + 16 * t2 + 4 * h;
      const _Float16* r1 = vb + (c + 32) * C::VT_LD + 16 * t2 + 4 * h;
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

  // Three register sets in rotation: blocks it + 1 and it + 2 are in flight
  // while block it is processed (loads of absent blocks are clamped, never
  // used).
  KvRegs R0, R1, R2;
  const FlashKv fkv{kv + L.head_tile(layer, 0, 0, g), (unsigned)(2 * L.n_kv_heads * kPage * kHeadDim),
                    (unsigned)(L.n_kv_heads * kPage * kHeadDim)};
  const int kcl = (nkb_all - 1) * 32;
  auto blk = [&](int it) { return min((it * NS + grp) * 32, kcl); };
  if (stager) {
    flash_load(R0, fkv, pt, idx, blk(0), kend_all);
    flash_load(R1, fkv, pt, idx, blk(1), kend_all);
  }
  for (int it = 0; it < niter; it += 3) {
    if (stager) flash_load(R2, fkv, pt, idx, blk(it + 2), kend_all);
    process(R0, it);
    if (it + 1 >= niter) break;
    if (stager) flash_load(R0, fkv, pt, idx, blk(it + 3), kend_all);
    process(R1, it + 1);
    if (it + 2 >= niter) break;
    if (stager) flash_load(R1, fkv, pt, idx, blk(it + 4), kend_all);
    process(R2, it + 2);
  }
  lsum += __shfl_xor(lsum, 32, 64);

  // Merge the groups in split order (group 0 holds key block 0, so its max is
  // finite for every query).
  if constexpr (NS > 1) {
    float* mg = reinterpret_cast<float*>(smem);
    __syncthreads();  // every group is done with its staging buffers
    if (grp > 0) {
      float* r = mg + ((grp - 1) * G + hi) * (2 + 32) * 64;
      r[lane] = m;
      r[64 + lane] = lsum;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        r[(2 + i) * 64 + lane] = o0[i];
        r[(18 + i) * 64 + lane] = o1[i];
      }
    }
    __syncthreads();
    if (grp > 0) return;
    // Group sp keeps this wave's (query block, head) at position hs(sp).
    auto hs = [&](int sp) { return (((qsel + sp) & 1) * GH) + hi % GH; };
    float mx = m;
#pragma unroll
    for (int sp = 1; sp < NS; ++sp) mx = fmaxf(mx, mg[((sp - 1) * G + hs(sp)) * (2 + 32) * 64 + lane]);
    const float w0 = __builtin_amdgcn_exp2f(m - mx);
    lsum *= w0;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      o0[i] *= w0;
      o1[i] *= w0;
    }
#pragma unroll
    for (int sp = 1; sp < NS; ++sp) {
      const float* r = mg + ((sp - 1) * G + hs(sp)) * (2 + 32) * 64;
      const float w = __builtin_amdgcn_exp2f(r[lane] - mx);  // 0 for a split that saw no key
      lsum += w * r[64 + lane];
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        o0[i] += w * r[(2 + i) * 64 + lane];
        o1[i] += w * r[(18 + i) * 64 + lane];
      }
    }
  }
  if (qvalid) {
    const float inv = 1.f / lsum;
    _Float16* dst = oM + ((size_t)qrow * hq + j) * 64;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int dim = 8 * (i >> 2) + 4 * h + (i & 3);
      dst[dim] = (_Float16)(o0[i] * inv);
      dst[dim + 32] = (_Float16)(o1[i] * inv);
    }
  }
}

bool flash_prefill_supported(int G, int max_context, size_t layer_kv_elems) {
  return (G == 4 || G == 8) && (max_context + kPage - 1) / kPage <= kFlashMaxPages &&
         layer_kv_elems <= 0xFFFFFFFFull;
}

template <int G, int NS>
static void launch_flash(hipStream_t st, dim3 grid, const _Float16* qM, const _Float16* kv, KvLayout L, int layer,
                         const int* page_table, int s, int p0, int n_rows, int hq, _Float16* oM) {
  using C = FlashCfg<G, NS>;
  static bool attr = false;
  if (!attr) {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(k_flash_prefill<G, NS>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS);
    attr = true;
  }
  k_flash_prefill<G, NS><<<grid, C::THREADS, C::LDS, st>>>(qM, kv, L, layer, page_table, s, p0, n_rows, hq, oM);
}

void flash_prefill(hipStream_t st, const _Float16* qM, const _Float16* kv, KvLayout L, int layer,
                   const int* page_table, int s, int p0, int n_rows, int hq, int hkv, _Float16* oM) {
  const int G = hq / hkv;
  // Pairs of query blocks x kv heads x two halves of each kv head's query heads.
  dim3 grid(((n_rows + 31) / 32 + 1) / 2, hkv, 2);
  switch (G) {
    case 4: launch_flash<4, 4>(st, grid, qM, kv, L, layer, page_table, s, p0, n_rows, hq, oM); break;
    default: launch_flash<8, 2>(st, grid, qM, kv, L, layer, page_table, s, p0, n_rows, hq, oM); break;
  }
}

}  // namespace hh
