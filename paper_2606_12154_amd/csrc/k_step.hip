// Batch-1 decode step as ONE persistent kernel for gfx950.
//
// One 512-thread workgroup per CU runs the whole token: embedding, then per
// layer the fused RMSNorm+QKV+RoPE+KV-append phase, paged GQA attention
// (split over pages; split 0 of each kv head combines), O projection +
// residual, RMSNorm+gate/up+SwiGLU, down projection + residual, and finally
// RMSNorm + LM head + argmax, reduced by workgroup 0 which publishes the token.
//
// Batch-1 decode is bound by reading every weight once from HBM.  Each phase
// splits its weight rows evenly over the workgroups; a wave owns whole rows and
// streams them with coalesced 16-byte non-temporal loads (a wave instruction
// reads 1 KiB of a row), double-buffered in registers, with the fp32 input
// vector staged in LDS.  Each output row is produced by exactly one wave, so
// results are bitwise reproducible.
//
// Workgroups exchange activations without grid barriers or memory fences:
// every value crossing workgroups travels as one 64-bit word (fp32 bits | a
// 32-bit epoch naming the step, layer and phase), written with a single
// relaxed agent-scope store, so a reader that sees the expected epoch also
// sees the value.  A consumer polls exactly the words it needs.  On this chip
// an agent-scope fence (an L2 write-back/invalidate) costs several
// microseconds while a flag crosses CUs in about half a microsecond, so this
// turns each phase boundary into one flag latency.  Because weights do not
// depend on activations, every wave issues its first batch of a phase's weight
// loads BEFORE polling that phase's input, so the wait overlaps HBM streaming.
#include "hh_kernels.h"

namespace hh {

constexpr int kStepWaves = kStepThreads / 64;
constexpr unsigned kSpinLimit = 1u << 20;  // polls (~1 s) before a wait gives up

// ---------------------------------------------------------------- epoch words

__device__ __forceinline__ void ll_put(unsigned long long* p, float v, unsigned ep) {
  __hip_atomic_store(p, ((unsigned long long)ep << 32) | __float_as_uint(v), __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void ll_put_u(unsigned long long* p, unsigned v, unsigned ep) {
  __hip_atomic_store(p, ((unsigned long long)ep << 32) | v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ unsigned long long ll_get(const unsigned long long* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Poll word p (first read already in w) until it carries epoch ep; returns
// its 32-bit payload.  A wait longer than kSpinLimit polls, or any wait after
// another one timed out, sets *err and returns the stale payload, so every
// wave always terminates.
__device__ __forceinline__ unsigned ll_wait(const unsigned long long* p, unsigned ep, unsigned long long w,
                                            int* err) {
  unsigned spins = 0;
  while ((unsigned)(w >> 32) != ep) {
    __builtin_amdgcn_s_sleep(1);
    w = ll_get(p);
    if ((++spins & 255u) == 0) {
      if (spins > kSpinLimit || __hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) {
        __hip_atomic_store(err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        break;
      }
    }
  }
  return (unsigned)w;
}

// xs[i] = value of word src[i] at epoch ep for i < n (all threads of the
// block); returns the block-wide sum of squares.  A thread loads all of its
// (up to U) words at once and, while any is stale, re-polls only the stale
// ones together, so a late producer costs one round trip, not one per word.
__device__ __forceinline__ float ll_stage(const unsigned long long* __restrict__ src, int n, unsigned ep, float* xs,
                                          float* red, int* err) {
  constexpr int U = 16;
  float ss = 0.f;
  for (int base = threadIdx.x; base < n; base += kStepThreads * U) {
    unsigned long long w[U];
    unsigned stale = 0;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = base + u * kStepThreads;
      w[u] = i < n ? ll_get(src + i) : ((unsigned long long)ep << 32);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) stale |= ((unsigned)(w[u] >> 32) != ep ? 1u : 0u) << u;
    unsigned spins = 0;
    while (stale) {
      __builtin_amdgcn_s_sleep(1);
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (stale & (1u << u)) w[u] = ll_get(src + base + u * kStepThreads);
#pragma unroll
      for (int u = 0; u < U; ++u)
        if ((stale & (1u << u)) && (unsigned)(w[u] >> 32) == ep) stale &= ~(1u << u);
      if ((++spins & 255u) == 0 && stale) {
        if (spins > kSpinLimit || __hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) {
          __hip_atomic_store(err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          break;
        }
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = base + u * kStepThreads;
      if (i < n) {
        const float v = __uint_as_float((unsigned)w[u]);
        xs[i] = v;
        ss += v * v;
      }
    }
  }
  ss = wave_sum(ss);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int w = 0; w < kStepWaves; ++w) tot += red[w];
  __syncthreads();
  return tot;
}

// In-place RMSNorm of the staged vector: xs *= rsqrt(ss / n + eps) * gain,
// with this thread's gains (elements tid + 512 k) already in registers.
template <int NR>
__device__ __forceinline__ void norm_staged(float* xs, int n, float ss, float eps, const float* gr) {
  const float inv = rsqrtf(ss / (float)n + eps);
#pragma unroll
  for (int k = 0; k < NR; ++k) {
    const int i = threadIdx.x + k * kStepThreads;
    if (i < n) xs[i] = xs[i] * inv * gr[k];
  }
  __syncthreads();
}

// ---------------------------------------------------------------- row streaming

// Sum RB per-lane partials over the wave.  Returns, in lane l, the total of
// row l >> (6 - log2 RB); a butterfly halves the row set at each of the first
// log2 RB exchange steps, so RB rows cost log2 RB + 6 - log2 RB + (RB - 1)
// shuffles instead of 6 RB.
template <int RB>
__device__ __forceinline__ float reduce_rows(float* v) {
  constexpr int LOG = RB == 1 ? 0 : RB == 2 ? 1 : RB == 4 ? 2 : RB == 8 ? 3 : 4;
  static_assert((1 << LOG) == RB, "RB must be 1, 2, 4, 8 or 16");
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int s = 0; s < LOG; ++s) {
    const int off = 32 >> s;
    const bool upper = (lane & off) != 0;
    const int half = RB >> (s + 1);
#pragma unroll
    for (int i = 0; i < (RB >> 1); ++i) {
      if (i < half) {
        const float send = upper ? v[i] : v[i + half];
        const float keep = upper ? v[i + half] : v[i];
        v[i] = keep + __shfl_xor(send, off, 64);
      }
    }
  }
  float r = v[0];
#pragma unroll
  for (int off = 32 >> LOG; off > 0; off >>= 1) r += __shfl_xor(r, off, 64);
  return r;
}

constexpr int pow2_floor(int v) { return v >= 16 ? 16 : v >= 8 ? 8 : v >= 4 ? 4 : v >= 2 ? 2 : 1; }

// One register batch of a wave: RB rows x CHB 16-byte chunks per lane
// (RB * CHB <= 8 outstanding loads per lane).  A row has CH chunks per lane
// (lane l reads chunks l, l + 64, ...), taken in NCB = CH / CHB blocks; batch
// b covers row group b / NCB and chunk block b % NCB.  Wave w of a workgroup
// owns the local rows w, w + 8, w + 16, ...; row group g holds its rows
// g*RB .. g*RB + RB - 1.
// Registers of one wave's in-flight weight loads: 8 x 16 bytes per lane.
struct WBuf {
  u32x4 w[8];
};

// View of a WBuf for rows of CH chunks per lane: RB rows x CHB chunks
// (RB * CHB = 8, RB a power of two).  A row's CH chunks (lane l reads chunks
// l, l + 64, ...) are taken in NCB = CH / CHB blocks; batch b covers row group
// b / NCB and chunk block b % NCB.  Wave w of a workgroup owns the local rows
// w, w + 8, w + 16, ...; row group g holds its rows g*RB .. g*RB + RB - 1.
template <typename TW, int CH>
struct RowBatch {
  static constexpr int CHB = CH >= 8 ? 8 : CH;
  static constexpr int NCB = CH / CHB;
  static constexpr int RB = pow2_floor(8 / CHB);
  static constexpr int LOG = RB == 1 ? 0 : RB == 2 ? 1 : RB == 4 ? 2 : RB == 8 ? 3 : 4;
  static_assert(CH % CHB == 0, "chunk blocks must tile the row");
  static_assert(RB * CHB <= 8, "batch exceeds the register buffer");

  template <class Map>
  static __device__ __forceinline__ void issue(WBuf& B, const TW* __restrict__ W, int K, const Map& map, int n_local,
                                               int b) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int nch = K / Vec16<TW>::n;
    const int grp = b / NCB, cb = b % NCB;
#pragma unroll
    for (int r = 0; r < RB; ++r) {
      const int lr = wave + kStepWaves * (grp * RB + r);
      const int row = lr < n_local ? map(lr) : -1;
      const u32x4* src = reinterpret_cast<const u32x4*>(W + (size_t)(row < 0 ? 0 : row) * K);
#pragma unroll
      for (int c = 0; c < CHB; ++c) {
        const int ch = lane + 64 * (cb * CHB + c);
        if (row >= 0 && ch < nch) B.w[r * CHB + c] = __builtin_nontemporal_load(src + ch);
        else B.w[r * CHB + c] = u32x4{0u, 0u, 0u, 0u};
      }
    }
  }

  // Accumulate the batch's dot products with the LDS vector xs into acc; on
  // the row group's last chunk block, reduce and store res[lr] = row total.
  static __device__ __forceinline__ void consume(const WBuf& B, const float* xs, int K, int n_local, int b,
                                                 float* acc, float* res) {
    constexpr int V = Vec16<TW>::n;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int nch = K / V;
    const int grp = b / NCB, cb = b % NCB;
#pragma unroll
    for (int c = 0; c < CHB; ++c) {
      const int ch = lane + 64 * (cb * CHB + c);
      if (ch < nch) {
        float xv[V];
#pragma unroll
        for (int e = 0; e < V; e += 4) {
          const float4 t = *reinterpret_cast<const float4*>(xs + ch * V + e);
          xv[e] = t.x;
          xv[e + 1] = t.y;
          xv[e + 2] = t.z;
          xv[e + 3] = t.w;
        }
#pragma unroll
        for (int r = 0; r < RB; ++r) {
          float wf[V];
          widen16(B.w[r * CHB + c], wf, TW());
#pragma unroll
          for (int e = 0; e < V; ++e) acc[r] = fmaf(wf[e], xv[e], acc[r]);
        }
      }
    }
    if (cb == NCB - 1) {
      const float tot = reduce_rows<RB>(acc);
      const int r = lane >> (6 - LOG);
      if ((lane & ((64 >> LOG) - 1)) == 0) {
        const int lr = wave + kStepWaves * (grp * RB + r);
        if (lr < n_local) res[lr] = tot;
      }
#pragma unroll
      for (int i = 0; i < RB; ++i) acc[i] = 0.f;
    }
  }
};

// Stream the workgroup's n_local rows; `cur` already holds batch 0.
template <typename TW, int CH, class Map>
__device__ __forceinline__ void run_rows(WBuf& cur, const TW* __restrict__ W, int K, const Map& map, int n_local,
                                         const float* xs, float* res) {
  using B = RowBatch<TW, CH>;
  const int per_wave = (n_local + kStepWaves - 1) / kStepWaves;
  const int nb = (per_wave + B::RB - 1) / B::RB * B::NCB;
  float acc[B::RB];
#pragma unroll
  for (int i = 0; i < B::RB; ++i) acc[i] = 0.f;
  WBuf nxt;
  for (int b = 0; b < nb; ++b) {
    if (b + 1 < nb) B::issue(nxt, W, K, map, n_local, b + 1);
    B::consume(cur, xs, K, n_local, b, acc, res);
    cur = nxt;
  }
}

// ---------------------------------------------------------------- row maps

// Weight rows of a GEMV phase as a function of the workgroup-local row index.
// One map type for every phase keeps a single copy of the streaming code.
struct RowMap {
  int mode;  // 0: r0 + lr; 1: rotary pairs from pair r0; 2: gate/up outputs from r0
  int r0, nj, F;
  __device__ __forceinline__ int operator()(int lr) const {
    if (mode == 0) return r0 + lr;
    if (mode == 1) {  // pair gp = r0 + lr/2 is (head gp/32, i = gp%32): rows i and i + 32
      const int gp = r0 + (lr >> 1);
      return (gp >> 5) * 64 + (gp & 31) + 32 * (lr & 1);
    }
    return lr < nj ? r0 + lr : F + r0 + lr - nj;  // gate row j, or up row F + j
  }
};

__device__ __forceinline__ void split_range(int n, int parts, int i, int& b, int& e) {
  b = (int)(((long long)n * i) / parts);
  e = (int)(((long long)n * (i + 1)) / parts);
}


// ---------------------------------------------------------------- kernel

// Optional phase timestamps (100 MHz s_memrealtime), one row per workgroup.
#define STEP_MARK(l, ev)                                                                           \
  do {                                                                                             \
    if (P.trace && tid == 0) P.trace[((size_t)wg * (L + 1) + (l)) * 32 + (ev)] = wall_clock64();   \
  } while (0)

// Epoch of (layer, phase) in this step; phases: 0 q/k/v, 1 attention
// partials, 2 attention output, 3 x after O, 4 SwiGLU output, 5 x after down,
// 6 argmax keys.  The layer field is 6 bits wide (at most 63 layers + head).
__device__ __forceinline__ unsigned ep_of(unsigned base, int l, int ph) { return base + (unsigned)l * 8u + ph; }

enum : int { PH_QKV = 0, PH_O = 1, PH_GU = 2, PH_DOWN = 3, PH_HEAD = 4 };
constexpr int kKvStageBytes = 72 * 1024;  // LDS holding an attention item's K/V pages
constexpr int kNormRegs = 8;              // gain values per thread (d <= 8 * 512)
constexpr int kMaxSplitsPerWave = 8;  // split partials one combiner wave loads per round

template <typename TW, typename TKV, int CHD, int CHF>
__global__ __launch_bounds__(kStepThreads) void k_decode_step(StepParams<TW, TKV> P) {
  extern __shared__ float smem[];
  float* xs = smem;                      // [stage_floats] staged input vector
  float* res = xs + P.stage_floats;      // [kStepResFloats] row results
  float* st = res + kStepResFloats;      // [8 waves][4 rows][66] attention states
  float* qs = st + kStepWaves * 4 * 66;  // [8][64] query heads of a kv group
  float* kn = qs + kStepWaves * 64;      // [64] key of the current position
  float* vn = kn + 64;                   // [64] value of the current position
  float* xown = vn + 64;                 // [kStepResFloats] this workgroup's rows of x
  TKV* kvs = reinterpret_cast<TKV*>(xown + kStepResFloats);  // [pages][K|V][16][64] staged K/V
  __shared__ float red[kStepWaves];
  __shared__ unsigned long long kred[kStepWaves];
  __shared__ float2 rope_p[32];  // cos/sin of this step's position
  __shared__ LayerPtrs<TW> lptr[kStepMaxLayers];  // per-layer weight pointers
  __shared__ int item_pages[kStepMaxItemPages];   // physical pages of this workgroup's attention item

  const int wg = blockIdx.x, nwg = gridDim.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int d = P.d, F = P.F, hq = P.hq, hkv = P.hkv, G = hq / hkv, L = P.n_layers;
  const int s = P.stream;
  const int p = P.pos[s];
  const int tok = P.feed ? P.feed[0] : P.pending[s];
  const int t = p + 1;  // keys attended this step
  const unsigned E0 = P.epoch;

  int pq0, pq1, rd0, rd1, j0, j1, v0, v1;
  split_range((hq + 2 * hkv) * 32, nwg, wg, pq0, pq1);  // rotary pairs of [Wq; Wk; Wv]
  split_range(d, nwg, wg, rd0, rd1);                     // rows of Wo / Wdown / x
  split_range(F, nwg, wg, j0, j1);                       // SwiGLU outputs
  split_range(P.V, nwg, wg, v0, v1);                     // LM head rows
  const int nd = rd1 - rd0;

  // Attention plan (identical in every workgroup).  An item is a set of nh
  // query heads of kv head g over the pages of split sp; its K/V pages are
  // staged in LDS (at most kv_cap per stage).  Short contexts use one item
  // per query head (nh = 1, all waves split the pages, no combine step);
  // long ones use items per kv head (nh = G) split over up to nwg / Hkv
  // workgroups, whose partials the item of split 0 combines.
  const int npg = (t + kPage - 1) / kPage;
  const int kv_cap = kKvStageBytes / (2 * kPage * 64 * (int)sizeof(TKV));
  const int s_cap = nwg / hkv;
  const int nsplit_min = (npg + kv_cap - 1) / kv_cap;
  const bool per_q = hq * nsplit_min <= nwg;
  const int nh = per_q ? 1 : G;                 // query heads per item
  int nspl = per_q ? nsplit_min : (nsplit_min < s_cap ? nsplit_min : s_cap);
  const int pps = (npg + nspl - 1) / nspl;      // pages per split
  nspl = (npg + pps - 1) / pps;
  const int n_items = (hq / nh) * nspl;
  const bool has_item = wg < n_items;
  const int it_h = wg / nspl, it_sp = wg % nspl;          // head set, split
  const int it_g = per_q ? it_h / G : it_h;               // kv head
  const int it_j0 = per_q ? it_h : it_h * G;              // first query head
  const int ngrp = kStepWaves / nh;                       // waves per query head
  const int it_pg0 = it_sp * pps, it_pg1 = min(npg, it_pg0 + pps);

  // Phase table: sequence index i -> (layer, kind) with four GEMV phases per
  // layer and the LM head last.
  auto phase_w = [&](int l, int kind) -> const TW* {
    if (kind == PH_HEAD) return P.head;
    const LayerPtrs<TW>& Lw = lptr[l];
    return kind == PH_QKV ? Lw.wqkv : kind == PH_O ? Lw.wo : kind == PH_GU ? Lw.wgu : Lw.wdown;
  };
  auto phase_k = [&](int kind) { return kind == PH_DOWN ? F : kind == PH_O ? hq * 64 : d; };
  auto phase_map = [&](int kind) -> RowMap {
    if (kind == PH_QKV) return RowMap{1, pq0, 0, F};
    if (kind == PH_GU) return RowMap{2, j0, j1 - j0, F};
    return RowMap{0, kind == PH_HEAD ? v0 : rd0, 0, F};
  };
  auto phase_n = [&](int kind) {
    return kind == PH_QKV ? 2 * (pq1 - pq0) : kind == PH_GU ? 2 * (j1 - j0) : kind == PH_HEAD ? v1 - v0 : nd;
  };

  WBuf wb;              // the next phase's first weight batch, in flight
  float gr[kNormRegs];  // the next phase's RMSNorm gains, elements tid + 512 k
  auto issue_first = [&](int l2, int k2) {
    // Gains first: the norm needs them as soon as the input arrives, and a
    // wave's loads complete in order.
    const float* gsrc = k2 == PH_QKV ? lptr[l2].attn_norm
                        : k2 == PH_GU ? lptr[l2].mlp_norm
                        : k2 == PH_HEAD ? P.final_norm : nullptr;
    if (gsrc) {
#pragma unroll
      for (int k = 0; k < kNormRegs; ++k) {
        const int i = tid + k * kStepThreads;
        gr[k] = i < d ? gsrc[i] : 0.f;
      }
    }
    if (k2 == PH_DOWN) RowBatch<TW, CHF>::issue(wb, phase_w(l2, k2), F, phase_map(k2), phase_n(k2), 0);
    else RowBatch<TW, CHD>::issue(wb, phase_w(l2, k2), phase_k(k2), phase_map(k2), phase_n(k2), 0);
  };
  // Everything the epilogues read from memory is loaded now, so no epilogue
  // load ever queues behind a phase's weight or KV stream.
  const int page_p = P.page_table[(size_t)s * P.kv.max_pages + p / kPage];  // page of this position
  if (tid < 32) rope_p[tid] = P.rope[(size_t)p * 32 + tid];
  for (int i = tid; i < L; i += kStepThreads) lptr[i] = P.layer[i];
  if (has_item)
    for (int i = tid; i < it_pg1 - it_pg0; i += kStepThreads)
      item_pages[i] = P.page_table[(size_t)s * P.kv.max_pages + it_pg0 + i];
  const TW* erow = P.embed + (size_t)tok * d;
  for (int i = tid; i < nd; i += kStepThreads) xown[i] = (float)erow[rd0 + i];
  __syncthreads();
  issue_first(0, L > 0 ? PH_QKV : PH_HEAD);

  // Issue direct global->LDS loads of pages [pa, pb) of kv head it_g, layer
  // l: wave instruction q moves 1 KiB (lane i: 16 bytes at offset 16 i).
  auto stage_kv = [&](int l, int pa, int pb) {
    constexpr int tile_kib = kPage * 64 * (int)sizeof(TKV) / 1024;  // 1 KiB pieces per K or V tile
    const int n_instr = (pb - pa) * 2 * tile_kib;
    for (int q = wave; q < n_instr; q += kStepWaves) {
      const int tile = q / tile_kib, piece = q % tile_kib;
      const int pl = tile >> 1, kind2 = tile & 1;
      const int page = item_pages[pa + pl - it_pg0];
      const char* src = reinterpret_cast<const char*>(P.kvc + P.kv.head_tile(l, page, kind2, it_g)) +
                        piece * 1024 + lane * 16;
      char* dst = reinterpret_cast<char*>(kvs + (size_t)tile * kPage * 64) + piece * 1024;
      __builtin_amdgcn_global_load_lds(src, dst, 16, 0, 0);
    }
  };

  const int nphase = 4 * L + 1;
  for (int ip = 0; ip < nphase; ++ip) {
    const int l = ip == 4 * L ? L : ip >> 2;
    const int kind = ip == 4 * L ? PH_HEAD : ip & 3;

    // ---- paged GQA attention, before the O projection (workgroups with an
    // item; a wave's loads complete in order, so these workgroups issue their
    // O-projection prefetch only after it).
    if (kind == PH_O && has_item) {
      const int g = it_g, sp = it_sp;
      const unsigned e0 = ep_of(E0, l, 0);
      const int jj = wave % nh, grp = wave / nh;
      const int key = lane >> 2, quarter = lane & 3;
      // The item's query heads and the current position's k, v.
      for (int i = tid; i < nh * 64 + 128; i += kStepThreads) {
        const unsigned long long* src = i < nh * 64 ? P.ll_q + it_j0 * 64 + i
                                        : i < nh * 64 + 64 ? P.ll_kn + g * 64 + (i - nh * 64)
                                                           : P.ll_vn + g * 64 + (i - nh * 64 - 64);
        const float v = __uint_as_float(ll_wait(src, e0, ll_get(src), P.err));
        if (i < nh * 64) qs[i] = v;
        else if (i < nh * 64 + 64) kn[i - nh * 64] = v;
        else vn[i - nh * 64 - 64] = v;
      }
      STEP_MARK(l, 12);
      const float qscale = 0.125f * 1.4426950408889634f;  // 1/sqrt(64) * log2(e)
      float m = -INFINITY, lsum = 0.f, o[16], qv[16];
#pragma unroll
      for (int e = 0; e < 16; ++e) o[e] = 0.f;
      for (int ca = it_pg0; ca < it_pg1; ca += kv_cap) {
        const int cb = min(it_pg1, ca + kv_cap);
        if (ca != it_pg0) stage_kv(l, ca, cb);
        __builtin_amdgcn_s_waitcnt(0);  // this wave's direct LDS loads have landed
        __syncthreads();
        if (ca == it_pg0) STEP_MARK(l, 16);
#pragma unroll
        for (int e = 0; e < 16; ++e) qv[e] = qs[jj * 64 + quarter * 16 + e] * qscale;
        for (int pg = ca + grp; pg < cb; pg += ngrp) {
          const TKV* Kl = kvs + (size_t)((pg - ca) * 2) * kPage * 64 + key * 64 + quarter * 16;
          const TKV* Vl = Kl + kPage * 64;
          float kf[16], vf[16];
#pragma unroll
          for (int e = 0; e < 16; e += Vec16<TKV>::n) {
            widen16(*reinterpret_cast<const u32x4*>(Kl + e), kf + e, TKV());
            widen16(*reinterpret_cast<const u32x4*>(Vl + e), vf + e, TKV());
          }
          if (pg * kPage + key == p) {  // written this step: take the exchanged copy
#pragma unroll
            for (int e = 0; e < 16; ++e) {
              kf[e] = kn[quarter * 16 + e];
              vf[e] = vn[quarter * 16 + e];
            }
          }
          float sc = 0.f;
#pragma unroll
          for (int e = 0; e < 16; ++e) sc = fmaf(qv[e], kf[e], sc);
          sc += dpp<0xB1>(sc);  // the 4 lanes of a key hold quarters of its dot product
          sc += dpp<0x4E>(sc);
          if (pg * kPage + key >= t) {  // a slot past the length: stale data, weight 0 (and 0 * NaN is NaN)
            sc = -INFINITY;
#pragma unroll
            for (int e = 0; e < 16; ++e) vf[e] = 0.f;
          }
          const float mn = fmaxf(m, wave_max_u(sc));
          const float alpha = exp2f(m - mn);
          const float pk = exp2f(sc - mn);
          lsum = lsum * alpha + (quarter == 0 ? pk : 0.f);
#pragma unroll
          for (int e = 0; e < 16; ++e) o[e] = fmaf(pk, vf[e], o[e] * alpha);
          m = mn;
        }
        __syncthreads();  // the stage is reused by the next chunk
      }
      // Reduce over the keys of each row (lanes of a row sharing `quarter`;
      // row_ror by 4 and 8 keeps lane bits 0-1), then across the 4 rows in
      // the merge below: lanes 0-3 of row r leave o[quarter*16 .. +16] in
      // the wave's state slot for row r.
      lsum = wave_sum_u(lsum);
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        float v = o[e];
        v += dpp<0x124>(v);
        v += dpp<0x128>(v);
        o[e] = v;
      }
      {
        float* sw = st + wave * 4 * 66 + (lane >> 4) * 66;
        if ((lane & 15) == 0) {
          sw[0] = m;
          sw[1] = lsum;
        }
        if ((lane & 15) < 4) {
#pragma unroll
          for (int e = 0; e < 16; ++e) sw[2 + quarter * 16 + e] = o[e];
        }
      }
      __syncthreads();
      // Merge the wave groups of each query head (one wave per head).
      if (wave < nh) {
        const int j = it_j0 + wave;
        float M = -INFINITY;
        for (int gr = 0; gr < ngrp; ++gr) M = fmaxf(M, st[(gr * nh + wave) * 4 * 66]);
        float Ls = 0.f, O = 0.f;
        for (int gr = 0; gr < ngrp; ++gr) {
          const float* sw = st + (gr * nh + wave) * 4 * 66;
          const float f = exp2f(sw[0] - M);
          Ls = fmaf(sw[1], f, Ls);
          const float ow = (sw[2 + lane] + sw[66 + 2 + lane]) + (sw[132 + 2 + lane] + sw[198 + 2 + lane]);
          O = fmaf(ow, f, O);
        }
        if (nspl == 1) {
          ll_put(P.ll_o + j * 64 + lane, O / Ls, ep_of(E0, l, 2));
        } else {
          unsigned long long* pp = P.ll_part + ((size_t)j * s_cap + sp) * 66;
          const unsigned e1 = ep_of(E0, l, 1);
          if (lane == 0) {
            ll_put(pp, M, e1);
            ll_put(pp + 1, Ls, e1);
          }
          ll_put(pp + 2 + lane, O, e1);
        }
      }
      __syncthreads();
      STEP_MARK(l, 13);
      // Split 0 combines the splits of its query heads: wave (head jj, group
      // grp) loads splits grp, grp + ngrp, ... a round of 8 at a time (lane =
      // head dimension), then the groups merge through LDS.
      if (nspl > 1 && sp == 0) {
        const unsigned e1 = ep_of(E0, l, 1);
        float M = -INFINITY, Ls = 0.f, O = 0.f;
        {
          const int j = it_j0 + jj;
          const unsigned long long* pp = P.ll_part + (size_t)j * s_cap * 66;
          for (int r0 = grp; r0 < nspl; r0 += kMaxSplitsPerWave * ngrp) {
            unsigned long long w[kMaxSplitsPerWave][3];
            unsigned stale = 0;
#pragma unroll
            for (int u = 0; u < kMaxSplitsPerWave; ++u) {
              const int i = r0 + u * ngrp;
              const unsigned long long* q0 = pp + (size_t)i * 66;
              w[u][0] = w[u][1] = w[u][2] = (unsigned long long)e1 << 32;
              if (i < nspl) {
                w[u][0] = ll_get(q0);
                w[u][1] = ll_get(q0 + 1);
                w[u][2] = ll_get(q0 + 2 + lane);
              }
            }
#pragma unroll
            for (int u = 0; u < kMaxSplitsPerWave; ++u)
              stale |= ((unsigned)(w[u][0] >> 32) != e1 || (unsigned)(w[u][1] >> 32) != e1 ||
                                (unsigned)(w[u][2] >> 32) != e1
                            ? 1u
                            : 0u)
                       << u;
            unsigned spins = 0;
            while (stale) {
              __builtin_amdgcn_s_sleep(1);
#pragma unroll
              for (int u = 0; u < kMaxSplitsPerWave; ++u)
                if (stale & (1u << u)) {
                  const unsigned long long* q0 = pp + (size_t)(r0 + u * ngrp) * 66;
                  w[u][0] = ll_get(q0);
                  w[u][1] = ll_get(q0 + 1);
                  w[u][2] = ll_get(q0 + 2 + lane);
                  if ((unsigned)(w[u][0] >> 32) == e1 && (unsigned)(w[u][1] >> 32) == e1 &&
                      (unsigned)(w[u][2] >> 32) == e1)
                    stale &= ~(1u << u);
                }
              if ((++spins & 255u) == 0 && stale) {
                if (spins > kSpinLimit || __hip_atomic_load(P.err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) {
                  __hip_atomic_store(P.err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                  break;
                }
              }
            }
#pragma unroll
            for (int u = 0; u < kMaxSplitsPerWave; ++u) {
              if (r0 + u * ngrp >= nspl) break;
              const float mi = __uint_as_float((unsigned)w[u][0]);
              const float li = __uint_as_float((unsigned)w[u][1]);
              const float oi = __uint_as_float((unsigned)w[u][2]);
              const float Mn = fmaxf(M, mi);
              const float a = exp2f(M - Mn), b = exp2f(mi - Mn);
              Ls = Ls * a + li * b;
              O = O * a + oi * b;
              M = Mn;
            }
          }
        }
        float* sw = st + wave * 4 * 66;
        if (lane == 0) {
          sw[0] = M;
          sw[1] = Ls;
        }
        sw[2 + lane] = O;
        __syncthreads();
        if (wave < nh) {
          float Mx = -INFINITY;
          for (int gr = 0; gr < ngrp; ++gr) Mx = fmaxf(Mx, st[(gr * nh + wave) * 4 * 66]);
          float Lt = 0.f, Ot = 0.f;
          for (int gr = 0; gr < ngrp; ++gr) {
            const float* sv = st + (gr * nh + wave) * 4 * 66;
            const float f = exp2f(sv[0] - Mx);
            Lt = fmaf(sv[1], f, Lt);
            Ot = fmaf(sv[2 + lane], f, Ot);
          }
          ll_put(P.ll_o + (it_j0 + wave) * 64 + lane, Ot / Lt, ep_of(E0, l, 2));
        }
        __syncthreads();
        STEP_MARK(l, 14);
      }
      issue_first(l, PH_O);
    }

    // ---- stage this phase's input vector into LDS (normalised where needed)
    STEP_MARK(l, kind * 3);
    {
      const bool normed = kind == PH_QKV || kind == PH_GU || kind == PH_HEAD;
      float ss;
      if ((kind == PH_QKV && l == 0) || (kind == PH_HEAD && L == 0)) {  // the embedding row itself
        ss = 0.f;
        for (int i = tid; i < d; i += kStepThreads) {
          const float v = (float)erow[i];
          xs[i] = v;
          ss += v * v;
        }
        ss = wave_sum(ss);
        if (lane == 0) red[wave] = ss;
        __syncthreads();
        ss = 0.f;
        for (int w = 0; w < kStepWaves; ++w) ss += red[w];
        __syncthreads();
      } else {
        const unsigned long long* src = kind == PH_QKV || kind == PH_HEAD ? P.ll_xb
                                        : kind == PH_O ? P.ll_o : kind == PH_GU ? P.ll_xa : P.ll_m;
        const int n = kind == PH_O ? hq * 64 : kind == PH_DOWN ? F : d;
        const unsigned e = kind == PH_QKV || kind == PH_HEAD ? ep_of(E0, l - 1, 5)
                           : ep_of(E0, l, kind == PH_O ? 2 : kind == PH_GU ? 3 : 4);
        ss = ll_stage(src, n, e, xs, red, P.err);
      }
      if (normed) norm_staged<kNormRegs>(xs, d, ss, P.eps, gr);
    }
    STEP_MARK(l, kind * 3 + 1);

    // ---- stream this workgroup's weight rows
    const int nl = phase_n(kind);
    if (kind == PH_DOWN) run_rows<TW, CHF>(wb, phase_w(l, kind), F, phase_map(kind), nl, xs, res);
    else run_rows<TW, CHD>(wb, phase_w(l, kind), phase_k(kind), phase_map(kind), nl, xs, res);
    __syncthreads();
    STEP_MARK(l, kind * 3 + 2);
    // Cached pages do not depend on this step: start staging this layer's
    // attention K/V now, so it streams during the epilogue and the q wait.
    if (kind == PH_QKV && has_item) stage_kv(l, it_pg0, min(it_pg1, it_pg0 + kv_cap));

    // ---- epilogue
    if (kind == PH_QKV) {
      const unsigned e = ep_of(E0, l, 0);
      for (int lp = tid; lp < (pq1 - pq0); lp += kStepThreads) {
        const int gp = pq0 + lp, head = gp >> 5, i = gp & 31;
        const float y0 = res[2 * lp], y1 = res[2 * lp + 1];
        if (head < hq + hkv) {
          const float2 cs = rope_p[i];
          const float r0 = y0 * cs.x - y1 * cs.y, r1 = y1 * cs.x + y0 * cs.y;
          if (head < hq) {
            ll_put(P.ll_q + head * 64 + i, r0, e);
            ll_put(P.ll_q + head * 64 + i + 32, r1, e);
          } else {
            const int g = head - hq;
            TKV* dst = P.kvc + P.kv.head_tile(l, page_p, 0, g) + (p % kPage) * 64;
            dst[i] = (TKV)r0;
            dst[i + 32] = (TKV)r1;
            ll_put(P.ll_kn + g * 64 + i, (float)(TKV)r0, e);
            ll_put(P.ll_kn + g * 64 + i + 32, (float)(TKV)r1, e);
          }
        } else {
          const int g = head - hq - hkv;
          TKV* dst = P.kvc + P.kv.head_tile(l, page_p, 1, g) + (p % kPage) * 64;
          dst[i] = (TKV)y0;
          dst[i + 32] = (TKV)y1;
          ll_put(P.ll_vn + g * 64 + i, (float)(TKV)y0, e);
          ll_put(P.ll_vn + g * 64 + i + 32, (float)(TKV)y1, e);
        }
      }
    } else if (kind == PH_O || kind == PH_DOWN) {
      unsigned long long* dst = kind == PH_O ? P.ll_xa : P.ll_xb;
      const unsigned e = ep_of(E0, l, kind == PH_O ? 3 : 5);
      for (int i = tid; i < nd; i += kStepThreads) {
        const float xn = xown[i] + res[i];
        xown[i] = xn;
        ll_put(dst + rd0 + i, xn, e);
      }
    } else if (kind == PH_GU) {
      const unsigned e = ep_of(E0, l, 4);
      for (int i = tid; i < j1 - j0; i += kStepThreads) ll_put(P.ll_m + j0 + i, silu(res[i]) * res[(j1 - j0) + i], e);
    } else {  // PH_HEAD: logits, argmax; workgroup 0 publishes the token
      const int nv = v1 - v0;
      unsigned long long best = 0ull;
      for (int i = tid; i < nv; i += kStepThreads) {
        const float v = res[i];
        if (P.logits) P.logits[v0 + i] = v;
        const unsigned long long k = argmax_key(v, (uint32_t)(v0 + i));
        best = k > best ? k : best;
      }
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) {
        const unsigned long long o2 = __shfl_xor(best, off, 64);
        best = o2 > best ? o2 : best;
      }
      if (lane == 0) kred[wave] = best;
      __syncthreads();
      const unsigned e6 = ep_of(E0, L, 6);
      if (tid == 0) {
        for (int w = 1; w < kStepWaves; ++w) best = kred[w] > best ? kred[w] : best;
        ll_put_u(P.ll_keys + 2 * wg, (unsigned)(best >> 32), e6);
        ll_put_u(P.ll_keys + 2 * wg + 1, (unsigned)best, e6);
      }
      if (wg == 0 && wave == 0) {
        unsigned long long b = 0ull;
        for (int i = lane; i < nwg; i += 64) {
          const unsigned hi = ll_wait(P.ll_keys + 2 * i, e6, ll_get(P.ll_keys + 2 * i), P.err);
          const unsigned lo = ll_wait(P.ll_keys + 2 * i + 1, e6, ll_get(P.ll_keys + 2 * i + 1), P.err);
          const unsigned long long k = ((unsigned long long)hi << 32) | lo;
          b = k > b ? k : b;
        }
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) {
          const unsigned long long o2 = __shfl_xor(b, off, 64);
          b = o2 > b ? o2 : b;
        }
        if (lane == 0) {
          STEP_MARK(L, 15);
          const int nt = argmax_index(b);
          P.pending[s] = nt;
          P.hist[(size_t)s * P.max_ctx + p] = nt;
          P.pos[s] = p + 1;
        }
      }
    }

    STEP_MARK(l, 17 + kind);
    // ---- first weight batch of the next phase (it streams during the wait)
    if (ip + 1 < nphase) {
      const int l2 = ip + 1 == 4 * L ? L : (ip + 1) >> 2;
      const int k2 = ip + 1 == 4 * L ? PH_HEAD : (ip + 1) & 3;
      if (!(k2 == PH_O && has_item)) issue_first(l2, k2);
    }
    STEP_MARK(l, 22 + kind);
  }
}

// ---------------------------------------------------------------- launcher

template <typename TW, typename TKV>
size_t StepKernel<TW, TKV>::lds_bytes(int d, int F, int hq) {
  const int stage = d > F ? (d > hq * 64 ? d : hq * 64) : (F > hq * 64 ? F : hq * 64);
  return (size_t)(stage + 2 * kStepResFloats + kStepWaves * 4 * 66 + kStepWaves * 64 + 128) * sizeof(float) +
         kKvStageBytes;
}

template <typename TW, typename TKV, int CHD, int CHF>
static hipError_t launch_step(const StepParams<TW, TKV>& P, int nwg, hipStream_t st) {
  const size_t lds = StepKernel<TW, TKV>::lds_bytes(P.d, P.F, P.hq);
  auto kern = k_decode_step<TW, TKV, CHD, CHF>;
  if (lds > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  kern<<<nwg, kStepThreads, lds, st>>>(P);
  return hipGetLastError();
}

template <typename TW, typename TKV>
bool StepKernel<TW, TKV>::supports(int d, int F, int hq, int hkv, int V, int n_layers, int nwg) {
  constexpr int Vn = Vec16<TW>::n;
  const int chd = (d + 64 * Vn - 1) / (64 * Vn), chf = (F + 64 * Vn - 1) / (64 * Vn);
  if (hq * 64 != d || hq % hkv || hq / hkv > kStepWaves || nwg / hkv < 1 || n_layers > kStepMaxLayers) return false;
  if (d > kNormRegs * kStepThreads) return false;
  const int pairs = (hq + 2 * hkv) * 32;
  if ((V + nwg - 1) / nwg > kStepResFloats || 2 * ((F + nwg - 1) / nwg) > kStepResFloats ||
      2 * ((pairs + nwg - 1) / nwg) > kStepResFloats || (d + nwg - 1) / nwg > kStepResFloats)
    return false;
  if (lds_bytes(d, F, hq) > 144 * 1024) return false;  // plus ~12 KiB of static LDS
  if (sizeof(TW) == 2) return chd <= 4 && chf <= 16;
  return chd <= 1 && chf <= 3;
}

template <typename TW, typename TKV>
hipError_t StepKernel<TW, TKV>::launch(const StepParams<TW, TKV>& P, int nwg, hipStream_t st) {
  if constexpr (sizeof(TW) == 2) return launch_step<TW, TKV, 4, 16>(P, nwg, st);
  else return launch_step<TW, TKV, 1, 3>(P, nwg, st);
}

template <typename TW, typename TKV>
int StepKernel<TW, TKV>::max_blocks_per_cu(int d, int F, int hq) {
  const size_t lds = lds_bytes(d, F, hq);
  int nb = 0;
  hipError_t e;
  if constexpr (sizeof(TW) == 2)
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, k_decode_step<TW, TKV, 4, 16>, kStepThreads, lds);
  else
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, k_decode_step<TW, TKV, 1, 3>, kStepThreads, lds);
  return e == hipSuccess ? nb : 0;
}

template struct StepKernel<__bf16, _Float16>;
template struct StepKernel<float, float>;

}  // namespace hh
