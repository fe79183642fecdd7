// Batch-1 decode step as ONE persistent kernel for gfx950.
//
// One 512-thread workgroup per CU runs the whole token: embedding, then per
// layer RMSNorm + QKV + RoPE + KV append, paged GQA attention, O projection +
// residual, RMSNorm + gate/up + SwiGLU, down projection + residual, and
// finally RMSNorm + LM head + argmax, reduced by workgroup 0 which publishes
// the token.
//
// Batch-1 decode is bound by reading every weight once from HBM, but its
// phases are chained: every phase needs the whole output of the phase before,
// computed by all CUs.  The kernel therefore separates streaming from
// computing inside each workgroup:
//
//  * waves 0..2 (the streaming waves) walk the workgroup's whole byte stream
//    for the token -- its rows of every weight matrix, layer by layer, plus
//    the K/V pages of its attention item -- and copy it with direct
//    global->LDS loads into a ring of 8 KiB slots (slot n by wave n % 3).
//    Each keeps only a few slots in flight (together enough to saturate HBM,
//    few enough that the memory queues stay short), and none waits for
//    activations: they only wait for free ring slots.
//  * waves 3..7 (the five compute waves) wait for a phase's input vector,
//    then consume the phase's ring slots (dot products of staged rows with
//    the input, or attention over staged K/V pages), and publish the phase's
//    outputs.
//
// While compute waves wait for other CUs at a phase boundary, the streaming
// waves keep filling the ring with the next phases' weights, so HBM stays
// busy through the exchange latency instead of idling.
//
// Workgroups exchange activations without grid barriers or memory fences:
// every value crossing workgroups travels as one 64-bit word (fp32 bits | a
// 32-bit epoch naming the step, layer and phase), written with a single
// relaxed agent-scope store, so a reader that sees the expected epoch also
// sees the value.  Inside a workgroup, the streaming and compute waves
// synchronise through LDS counters (slots landed, slots consumed, a barrier
// among compute waves); every wait is bounded in time and gives up through a
// shared error flag, so every wave always terminates.
//
// Attention: an item is one kv head over a range of pages (all query heads of
// the group together, so K/V are read once).  For fp16 K/V the scores and the
// weighted sum use 16x16x32 fp16 MFMAs (queries split into fp16 high and low
// parts, so the scores keep fp32 accuracy); fp32 K/V use the VALU.  Items of
// at most two splits per kv head are combined by the consumers while they
// stage the O-projection input; longer contexts combine in split 0's
// workgroup.
#include "hh_kernels.h"

#include <type_traits>

namespace hh {

constexpr int kWaves = kStepThreads / 64;  // 8
constexpr int kLoaders = 3;                // streaming waves (one wave's direct-to-LDS loads top out near 13 GB/s)
constexpr int kNC = kWaves - kLoaders;     // compute waves
// Poll widths (words per compute thread) that cover the 1B shapes in one round.
constexpr int kPollX = (2048 + 64 * kNC - 1) / (64 * kNC);
constexpr int kHeadsPerWave = (32 + kNC - 1) / kNC;
constexpr int kSlot = 8192;                // ring slot: 8 pieces of 1 KiB
// 4-bit rows (d = 2048): 1024 bytes of codes + 64 bf16 scales.  A slot holds
// seven: codes of row r at 1024 r, all scales from kQ4ScaleOff (128 B a row).
constexpr int kQ4Rows = 7;
constexpr int kQ4RowBytes = 1152;
constexpr int kQ4ScaleOff = kQ4Rows * 1024;

// Rows per 4-bit slot for a segment of n rows: short segments (the q/k/v and
// O rows of one workgroup) are cut into thinner slots so that every compute
// wave gets some; the three sizes are the compiled variants of the row code.
__host__ __device__ constexpr int q4_rows(int n) { return n <= 2 * kNC ? 2 : n <= 3 * kNC ? 3 : kQ4Rows; }
constexpr int kMaxRing = 16;               // ring slots supported
constexpr int kItemKvBytes = 32 * 1024;    // K/V bytes aimed at per attention item (swept: 16-64 KiB)
constexpr int kMaxItemPages = 256;         // pages of one attention item
constexpr int kMaxConsumerSplits = 2;      // splits per kv head merged by the O-phase consumers
constexpr int kMaxGroup = 8;               // query heads per kv head (fp16 K/V)
constexpr int kMaxGroupF32 = 4;            // query heads per kv head (fp32 K/V)
constexpr int kStRow = 68;                 // LDS floats per (wave, head) attention state: m, l, o[64], pad
constexpr unsigned long long kWaitTicks = 100000000ull;  // 1 s of the 100 MHz real-time clock

typedef _Float16 f16x8v __attribute__((ext_vector_type(8)));

// Explicit address spaces: a generic (flat) access to LDS goes through the
// vector-memory path and is ordered behind the CU's in-flight global loads,
// so every LDS flag and every global pointer read from LDS is typed here.
#define HH_LDS __attribute__((address_space(3)))
#define HH_GLB __attribute__((address_space(1)))

// Floats of the second staging buffer: the down-projection input [F], or the
// O-projection input [Hq * 64] followed by the attention states of the
// compute waves.
__host__ __device__ constexpr int step_xc_floats(int d, int hq, int hkv) {
  return (kNC - 1) * d > hq * 64 + kNC * (hq / hkv) * kStRow ? (kNC - 1) * d : hq * 64 + kNC * (hq / hkv) * kStRow;
}

// ---------------------------------------------------------------- waits

// LDS block shared by the streaming and compute waves.
struct RingSync {
  unsigned long long wait_ticks;  // a wait gives up after this many ticks of the 100 MHz clock
  int cbar;      // arrivals at compute-wave barriers
  int abort;     // set when a wait gave up: every later wait returns at once
  int quiet;     // compute waves are waiting for another workgroup's outputs
  int landed[kMaxRing];    // per ring position: stream index of the last slot landed there
  int consumed[kMaxRing];  // per ring position: stream index of the last slot consumed there
  float ss[kNC];           // per compute wave: partial sum of squares of a staged vector
};

// Called in a wait loop: true once the wait must give up (after wait_ticks,
// 1 s unless the host sets a shorter limit, or once any wait of this
// workgroup or of another one has given up).
__device__ __forceinline__ bool give_up(unsigned& spins, unsigned long long& t0, RingSync HH_LDS* sy, int HH_GLB* err) {
  if ((++spins & 63u) != 0) return false;
  if (*(volatile int HH_LDS*)&sy->abort) return true;
  const unsigned long long t = wall_clock64();
  if (t0 == 0) {
    t0 = t;
    return false;
  }
  if (t - t0 > sy->wait_ticks || __hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) {
    *(volatile int HH_LDS*)&sy->abort = 1;
    __hip_atomic_store(err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return true;
  }
  return false;
}

__device__ __forceinline__ void compiler_fence() { asm volatile("" ::: "memory"); }
// s_waitcnt lgkmcnt(0) (vmcnt and expcnt left at their maxima).
__device__ __forceinline__ void wait_lds() { __builtin_amdgcn_s_waitcnt(0xC07F); }
#define HH_STEP_VMWAIT(c) __builtin_amdgcn_s_waitcnt(((c) & 15) | (0x7 << 4) | (0xF << 8) | (((c) >> 4) << 14))

// Barrier among the compute waves (the streaming wave never joins one).
__device__ __forceinline__ void cbar(RingSync HH_LDS* sy, int& gen, int HH_GLB* err) {
  gen += 1;
  compiler_fence();
  wait_lds();
  if ((threadIdx.x & 63) == 0) __hip_atomic_fetch_add(&sy->cbar, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  unsigned spins = 0;
  unsigned long long t0 = 0;
  while (*(volatile int HH_LDS*)&sy->cbar < gen * kNC) {
    __builtin_amdgcn_s_sleep(1);
    if (give_up(spins, t0, sy, err)) break;
  }
  compiler_fence();
}

__device__ __forceinline__ void wait_landed(RingSync HH_LDS* sy, int n, int pos, int HH_GLB* err) {
  if (*(volatile int HH_LDS*)&sy->landed[pos] < n) {
    unsigned spins = 0;
    unsigned long long t0 = 0;
    while (*(volatile int HH_LDS*)&sy->landed[pos] < n) {
      __builtin_amdgcn_s_sleep(1);
      if (give_up(spins, t0, sy, err)) break;
    }
  }
  compiler_fence();
}

// This wave's LDS reads of ring slot n are complete: hand it back.
__device__ __forceinline__ void release_slot(RingSync HH_LDS* sy, int pos, int n) {
  compiler_fence();
  wait_lds();
  if ((threadIdx.x & 63) == 0) *(volatile int HH_LDS*)&sy->consumed[pos] = n;
}

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

// Compute-wave threads (index tc = tid - 128 of NT = 384) read the words
// addr(i), i < n, at epoch ep and pass (i, value) to f.  A thread issues all
// of its (at most U per round) loads at once and then re-polls only the stale
// ones, so a late producer costs one more round trip, not one per word.
// Diagnostic record of one poll (thread 0 of the compute waves): when the
// first round returned and how many rounds ran.
struct PollTrace {
  unsigned long long* rec;  // nullptr, or 2 words: first-return time, rounds
};

template <int U, class A, class F>
__device__ __forceinline__ void poll_words(A&& addr, int n, unsigned ep, RingSync HH_LDS* sy, int HH_GLB* err, F&& f,
                                           PollTrace pt = PollTrace{nullptr}) {
  constexpr int NT = kNC * 64;
  const int tc = (int)threadIdx.x - 64 * kLoaders;
  for (int base = tc; base < n; base += NT * U) {
    unsigned long long w[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = base + u * NT;
      w[u] = i < n ? ll_get(addr(i)) : ((unsigned long long)ep << 32);
    }
    unsigned stale = 0;
#pragma unroll
    for (int u = 0; u < U; ++u) stale |= ((unsigned)(w[u] >> 32) != ep ? 1u : 0u) << u;
    if (pt.rec && tc == 0) pt.rec[0] = wall_clock64();
    unsigned rounds = 1;
    unsigned spins = 0;
    unsigned long long t0 = 0;
    while (stale) {
      ++rounds;
      __builtin_amdgcn_s_sleep(1);
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (stale & (1u << u)) w[u] = ll_get(addr(base + u * NT));
#pragma unroll
      for (int u = 0; u < U; ++u)
        if ((stale & (1u << u)) && (unsigned)(w[u] >> 32) == ep) stale &= ~(1u << u);
      if (stale && give_up(spins, t0, sy, err)) break;
    }
    if (pt.rec && tc == 0) pt.rec[1] = rounds;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = base + u * NT;
      if (i < n) f(i, __uint_as_float((unsigned)w[u]));
    }
  }
}
template <int U, class F>
__device__ __forceinline__ void poll_span(const unsigned long long* __restrict__ src, int n, unsigned ep, RingSync HH_LDS* sy,
                                          int HH_GLB* err, F&& f, PollTrace pt = PollTrace{nullptr}) {
  poll_words<U>([=](int i) { return src + i; }, n, ep, sy, err, f, pt);
}

// ---------------------------------------------------------------- row dot products

// Sum RB per-lane partials over the wave.  Returns, in lane l, the total of
// row l >> (6 - log2 RB); a butterfly halves the row set at each of the first
// log2 RB exchange steps.
template <int RB>
__device__ __forceinline__ float reduce_rows(float* v) {
  constexpr int LOG = RB == 1 ? 0 : RB == 2 ? 1 : RB == 4 ? 2 : 3;
  static_assert((1 << LOG) == RB, "RB must be 1, 2, 4 or 8");
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

constexpr int rows_per_slot(int np) { return np >= 8 ? 1 : 8 / np; }
constexpr int log2_small(int v) { return v >= 8 ? 3 : v >= 4 ? 2 : v >= 2 ? 1 : 0; }

// Slots of a segment of n rows with np 1 KiB pieces per row: a slot holds
// 8 / np whole rows (np <= 8) or 8 pieces of one row (np > 8, np % 8 == 0).
__device__ __forceinline__ int row_slots(int n, int np) {
  return np <= 8 ? (n + (8 / np) - 1) / (8 / np) : n * (np / 8);
}

// One ring slot of weight rows (slot index k of its segment) against the
// staged fp32 vector xs of K elements.  Lane l reads the 16 bytes at offset
// 16 l of every piece.  NP <= 8: writes res[row] for the slot's rows; NP > 8:
// writes the partial res[row * (NP / 8) + chunk].  FULL: K fills the pieces
// exactly, so every read is issued up front with no per-piece branch (rows
// missing from the slot hold a copy of its first row and are read but not
// written back).
template <typename TW, int NP, bool FULL>
__device__ __forceinline__ void slot_rows(const char* slot, const float* xs, int K, int k, int n_rows, float* res) {
  constexpr int E = 16 / (int)sizeof(TW);     // elements per lane per piece
  constexpr int PE = 1024 / (int)sizeof(TW);  // elements per piece
  const int lane = threadIdx.x & 63;
  if constexpr (NP <= 8) {
    constexpr int RPS = rows_per_slot(NP);
    constexpr int LOG = log2_small(RPS);
    static_assert((1 << LOG) == RPS, "rows per slot must be a power of two");
    const int r0 = k * RPS;
    // One accumulator per (row, piece): independent FMA chains interleave
    // instead of serialising on the FMA latency.
    float acc[RPS][NP];
#pragma unroll
    for (int r = 0; r < RPS; ++r)
#pragma unroll
      for (int c = 0; c < NP; ++c) acc[r][c] = 0.f;
#pragma unroll
    for (int c = 0; c < NP; ++c) {
      const int e0 = c * PE + lane * E;
      const bool ok = FULL || e0 < K;
      float xv[E];
#pragma unroll
      for (int e = 0; e < E; e += 4) {
        const float4 t = *reinterpret_cast<const float4*>(xs + e0 + e);
        xv[e] = ok ? t.x : 0.f;
        xv[e + 1] = ok ? t.y : 0.f;
        xv[e + 2] = ok ? t.z : 0.f;
        xv[e + 3] = ok ? t.w : 0.f;
      }
#pragma unroll
      for (int r = 0; r < RPS; ++r) {
        const u32x4 w = *reinterpret_cast<const u32x4*>(slot + (r * NP + c) * 1024 + lane * 16);
        float wf[E];
        widen16(w, wf, TW());
#pragma unroll
        for (int e = 0; e < E; ++e) acc[r][c] = fmaf(ok ? wf[e] : 0.f, xv[e], acc[r][c]);
      }
    }
    // Row totals by DPP row sums and lane reads (VALU only: a chain of
    // LDS-routed shuffles would dominate the latency of a small phase).
#pragma unroll
    for (int r = 0; r < RPS; ++r) {
      float a = 0.f;
#pragma unroll
      for (int c = 0; c < NP; ++c) a += acc[r][c];
      const float tot = wave_sum_u(a);
      if (lane == 0 && r0 + r < n_rows) res[r0 + r] = tot;
    }
  } else {
    static_assert(NP % 8 == 0, "long rows must be whole slots");
    constexpr int CPR = NP / 8;
    const int row = k / CPR, ch = k % CPR;
    float acc = 0.f;
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      const int e0 = (ch * 8 + c) * PE + lane * E;
      const bool ok = FULL || e0 < K;
      const u32x4 w = *reinterpret_cast<const u32x4*>(slot + c * 1024 + lane * 16);
      float wf[E];
      widen16(w, wf, TW());
#pragma unroll
      for (int e = 0; e < E; e += 4) {
        const float4 t = *reinterpret_cast<const float4*>(xs + e0 + e);
        acc = fmaf(ok ? wf[e] : 0.f, ok ? t.x : 0.f, acc);
        acc = fmaf(ok ? wf[e + 1] : 0.f, ok ? t.y : 0.f, acc);
        acc = fmaf(ok ? wf[e + 2] : 0.f, ok ? t.z : 0.f, acc);
        acc = fmaf(ok ? wf[e + 3] : 0.f, ok ? t.w : 0.f, acc);
      }
    }
    acc = wave_sum_u(acc);
    if (lane == 0 && row < n_rows) res[row * CPR + ch] = acc;
  }
}

// ---------------------------------------------------------------- the plan

// Weight rows of a GEMV phase as a function of the workgroup-local row index.
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

enum : int { SG_QKV = 0, SG_KV = 1, SG_O = 2, SG_GU = 3, SG_DOWN = 4, SG_HEAD = 5 };

// The workgroup's share of the step (identical arithmetic in every wave).
struct Plan {
  int pq0, pq1;  // rotary pairs of [Wq; Wk; Wv]
  int rd0, rd1;  // rows of Wo / Wdown / x
  int j0, j1;    // SwiGLU outputs (gate and up rows)
  int v0, v1;    // LM head rows
  // attention: items are (kv head, split) on workgroups 0 .. n_items - 1
  int nspl, pps, n_items, has_item, it_g, it_sp, it_pg0, it_pg1, consumer_comb;
  // Ring slots per layer of each segment, and the segment's first slot
  // within the layer (named fields: an array indexed at run time would live
  // in scratch memory).
  int n_qkv, n_kv, n_o, n_gu, n_down;
  int o_qkv, o_kv, o_o, o_gu, o_down;
  int per_layer, head_slots;
  __device__ __forceinline__ int slots(int sg) const {
    switch (sg) {
      case SG_QKV: return n_qkv;
      case SG_KV: return n_kv;
      case SG_O: return n_o;
      case SG_GU: return n_gu;
      case SG_DOWN: return n_down;
      default: return head_slots;
    }
  }
};

template <typename TW, typename TKV, int NPD>
__device__ __forceinline__ void make_plan(Plan& pl, const StepParams<TW, TKV>& P, int wg, int nwg, int t) {
  const int d = P.d, F = P.F, hq = P.hq, hkv = P.hkv;
  split_range((hq + 2 * hkv) * 32, nwg, wg, pl.pq0, pl.pq1);
  split_range(d, nwg, wg, pl.rd0, pl.rd1);
  split_range(P.V, nwg, wg, pl.v0, pl.v1);
  // Attention items: split the t positions' pages so an item streams about
  // kItemKvBytes of K/V.
  constexpr int page_bytes = 2 * kPage * 64 * (int)sizeof(TKV);  // K and V of one page, one kv head
  constexpr int pps = kSlot / page_bytes;                          // pages per ring slot
  const int npg = (t + kPage - 1) / kPage;
  // Items of kItemKvBytes while that makes at most 16 splits per kv head;
  // longer caches keep about 16 splits with items of up to four times that
  // size, and beyond that as many splits as there are workgroups per kv
  // head.  Measured, tok/s at 2,048 / 8,192 / 16,384 cached positions:
  // 1,505 / 1,360 / 1,305; 1,499 / 1,351 / 1,305 with 64 KiB items past 16
  // splits; 1,507 / 1,371 / 1,225 with 16 splits at every length (too few
  // workgroups streaming the longest caches).
  int cap = kItemKvBytes / page_bytes;
  if (npg > 16 * cap) cap = min((npg + 15) / 16, 4 * cap);
  const int s_cap = nwg / hkv;
  int nspl = (npg + cap - 1) / cap;
  nspl = nspl < s_cap ? nspl : s_cap;
  int per = (npg + nspl - 1) / nspl;
  nspl = (npg + per - 1) / per;
  pl.nspl = nspl;
  pl.pps = pps;
  pl.n_items = hkv * nspl;
  pl.has_item = wg < pl.n_items;
  pl.it_g = wg / nspl;
  pl.it_sp = wg % nspl;
  pl.it_pg0 = pl.it_sp * per;
  pl.it_pg1 = pl.it_pg0 + per < npg ? pl.it_pg0 + per : npg;
  pl.consumer_comb = nspl <= kMaxConsumerSplits;
  // SwiGLU outputs: item workgroups take fewer, so every workgroup streams
  // about the same bytes per layer.  An output is three d-rows (gate, up,
  // and the Wdown^T row it multiplies).
  constexpr bool q4 = std::is_same<TW, Q4Row>::value;
  const int kv_slots = (per + pps - 1) / pps;
  // Bytes of one output's rows: gate, up and its Wdown^T row.
  const int gu_unit = 3 * (q4 ? kQ4RowBytes : NPD * 1024);
  int kvu = (kv_slots * kSlot + gu_unit / 2) / gu_unit;
  long long tot = (long long)F + (long long)pl.n_items * kvu;
  if (tot < (long long)kvu * nwg) {  // items would get a negative share: plain split
    kvu = 0;
    tot = F;
  }
  auto cum = [&](int w) -> int {
    const int wi = w < pl.n_items ? w : pl.n_items;
    return (int)(((long long)w * tot - (long long)wi * kvu * nwg) / nwg);
  };
  pl.j0 = cum(wg);
  pl.j1 = cum(wg + 1);
  auto slots = [&](int n) { return q4 ? (n + q4_rows(n) - 1) / q4_rows(n) : row_slots(n, NPD); };
  pl.n_qkv = slots(2 * (pl.pq1 - pl.pq0));
  pl.n_kv = pl.has_item ? (pl.it_pg1 - pl.it_pg0 + pps - 1) / pps : 0;
  pl.n_o = slots(pl.rd1 - pl.rd0);
  pl.n_gu = slots(2 * (pl.j1 - pl.j0));
  pl.n_down = slots(pl.j1 - pl.j0);
  pl.o_qkv = 0;
  pl.o_kv = pl.n_qkv;
  pl.o_o = pl.o_kv + pl.n_kv;
  pl.o_gu = pl.o_o + pl.n_o;
  pl.o_down = pl.o_gu + pl.n_gu;
  pl.per_layer = pl.o_down + pl.n_down;
  pl.head_slots = slots(pl.v1 - pl.v0);
}

// ---------------------------------------------------------------- streaming

// Issue the 8 direct global->LDS loads (1 KiB each, lane l: 16 bytes at
// 16 l) of ring slot k of a row segment: 8 / NP whole rows (NP <= 8, rows
// missing at the end repeat the slot's first row; pieces beyond 8 / NP * NP
// repeat its first piece) or 8 pieces of one row (NP > 8).  full: rows are a
// whole number of pieces (no lane reads past the end of a row).
template <int NP>
__device__ __forceinline__ void issue_row_slot(char* dst, const char* W, const RowMap& map, int rowb, int nrows, int k,
                                               bool full) {
  const int lane = threadIdx.x & 63;
  if constexpr (NP <= 8) {
    constexpr int RPS = rows_per_slot(NP);
    const int lr0 = k * RPS;
    const char* first = W + (size_t)map(lr0) * rowb;
#pragma unroll
    for (int r = 0; r < RPS; ++r) {
      const char* row = r == 0 ? first : lr0 + r < nrows ? W + (size_t)map(lr0 + r) * rowb : first;
#pragma unroll
      for (int c = 0; c < NP; ++c) {
        int off = c * 1024 + lane * 16;
        if (!full && off + 16 > rowb) off = 0;
        __builtin_amdgcn_global_load_lds(row + off, dst + (r * NP + c) * 1024, 16, 0, 2);
      }
    }
#pragma unroll
    for (int q = RPS * NP; q < 8; ++q) __builtin_amdgcn_global_load_lds(first, dst + q * 1024, 16, 0, 2);
  } else {
    constexpr int CPR = NP / 8;
    const int row = k / CPR, ch = k - row * CPR;
    const char* src = W + (size_t)map(row) * rowb + ch * 8 * 1024;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      int off = q * 1024 + lane * 16;
      if (!full && ch * 8 * 1024 + off + 16 > rowb) off = 0;
      __builtin_amdgcn_global_load_lds(src + off, dst + q * 1024, 16, 0, 2);
    }
  }
}

// The 8 direct global->LDS loads of a slot of 4-bit rows: up to seven rows'
// codes (lane l: 16 bytes at 16 l), then their scales (lane l < 56: bytes
// 16 (l % 8) .. + 16 of row l / 8's scales).  The slot holds rows R k ..
// R k + R - 1 of the segment (R = q4_rows(nrows)); its other row places, and
// rows missing at the end of the segment, repeat the slot's first row, so
// every slot costs the same 8 loads.
__device__ __forceinline__ void issue_q4_slot(char* dst, const char* W, const RowMap& map, int nrows, int k) {
  const int lane = threadIdx.x & 63;
  const int R = q4_rows(nrows);
  const int lr0 = k * R;
  const char* first = W + (size_t)map(lr0) * kQ4RowBytes;
  auto row_ptr = [&](int r) {
    return r == 0 ? first : r < R && lr0 + r < nrows ? W + (size_t)map(lr0 + r) * kQ4RowBytes : first;
  };
#pragma unroll
  for (int r = 0; r < kQ4Rows; ++r) __builtin_amdgcn_global_load_lds(row_ptr(r) + lane * 16, dst + r * 1024, 16, 0, 2);
  const int rs = lane >> 3;
  const char* srow = row_ptr(rs < kQ4Rows ? rs : 0);
  if (lane < 8 * kQ4Rows) __builtin_amdgcn_global_load_lds(srow + 1024 + (lane & 7) * 16, dst + kQ4ScaleOff, 16, 0, 2);
}

typedef _Float16 h2x __attribute__((ext_vector_type(2)));

__device__ __forceinline__ unsigned and_or(unsigned a, unsigned m, unsigned o) {
  unsigned r;
  asm("v_and_or_b32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "s"(m), "v"(o));
  return r;
}

// A code word (byte b: element 2 b in the low nibble, 2 b + 1 in the high
// one) as four fp16 pairs, pair j holding elements j and j + 4.  A nibble n
// placed in the low mantissa bits of 1024 reads 1024 + n, one nibble up
// 1024 + 16 n (pairs 1 and 3).  q4_biased returns these raw pairs; q4_codes
// turns them into q = n - 8 exactly (a subtraction, or a fused scale and
// subtraction).
__device__ __forceinline__ void q4_biased(unsigned wd, unsigned* p) {
  const unsigned mg = 0x64006400u, w8 = wd >> 8;
  p[0] = and_or(wd, 0x000F000Fu, mg);
  p[1] = and_or(wd, 0x00F000F0u, mg);
  p[2] = and_or(w8, 0x000F000Fu, mg);
  p[3] = and_or(w8, 0x00F000F0u, mg);
}
__device__ __forceinline__ void q4_codes(unsigned wd, h2x* q) {
  unsigned p[4];
  q4_biased(wd, p);
  const h2x c0 = {(_Float16)-1032.f, (_Float16)-1032.f};
  const h2x sc = {(_Float16)0.0625f, (_Float16)0.0625f}, c1 = {(_Float16)-72.f, (_Float16)-72.f};
  q[0] = __builtin_bit_cast(h2x, p[0]) + c0;
  q[1] = __builtin_elementwise_fma(__builtin_bit_cast(h2x, p[1]), sc, c1);
  q[2] = __builtin_bit_cast(h2x, p[2]) + c0;
  q[3] = __builtin_elementwise_fma(__builtin_bit_cast(h2x, p[3]), sc, c1);
}

// R 4-bit rows of one slot against the staged input.  Lane l takes, as the
// 16-bit rows do, elements 512 c + 8 l .. + 8 (c < 4): code word c is the 4
// bytes at 256 c + 4 l of the row's codes (consecutive lanes, consecutive
// words) and its group is 16 c + l / 4.  The input comes in the layout of
// the biased code pairs: xh[4 c + j] holds the lane's inputs j and j + 4 of
// chunk c in fp16, divided by 16 for j = 1, 3, and xb[c] = -(1032 (sum of
// the j = 0, 2 halves) + 1152 (sum of the j = 1, 3 halves)), so that four
// 2-term dot products started from xb[c] give sum x q for the word, which
// its group's scale multiplies.  Row totals: a transposed reduction (lane
// swaps across the wave halves and 16-lane rows, then DPP within 8 lanes)
// leaves row bitrev3(l / 8) in lanes l.
template <int R>
__device__ __forceinline__ void q4_slot_rows(const char* slot, const h2x* xh, const float* xb, int k, int n_rows,
                                             float* res) {
  static_assert(R >= 1 && R <= kQ4Rows, "rows per slot");
  const int lane = threadIdx.x & 63;
  // All of the slot's words and scales are read before any is used, so the
  // LDS reads overlap instead of each waiting for the one before.
  unsigned wds[R][4];
  float scs[R][4];
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      wds[r][c] = *reinterpret_cast<const unsigned*>(slot + r * 1024 + 256 * c + 4 * lane);
      scs[r][c] = (float)*reinterpret_cast<const __bf16*>(slot + kQ4ScaleOff + r * 128 + 2 * (16 * c + (lane >> 2)));
    }
  float v[8];
#pragma unroll
  for (int r = 0; r < 8; ++r) v[r] = 0.f;
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int r = 0; r < R; ++r) {
      unsigned p[4];
      q4_biased(wds[r][c], p);
      float t = xb[c];
#pragma unroll
      for (int j = 0; j < 4; ++j) t = __builtin_amdgcn_fdot2(xh[4 * c + j], __builtin_bit_cast(h2x, p[j]), t, false);
      v[r] = fmaf(t, scs[r][c], v[r]);
    }
  // Rows (2 i, 2 i + 1) -> wave halves, then pairs of those -> 16-lane rows:
  // w[0] holds rows 0, 2, 1, 3 and w[1] rows 4, 6, 5, 7 in lane rows 0..3.
  float u[4], w[2];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(v[2 * i]), __float_as_uint(v[2 * i + 1]), false,
                                                     false);
    u[i] = __uint_as_float(sw[0]) + __uint_as_float(sw[1]);
  }
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const auto sw = __builtin_amdgcn_permlane16_swap(__float_as_uint(u[2 * i]), __float_as_uint(u[2 * i + 1]), false,
                                                     false);
    w[i] = __uint_as_float(sw[0]) + __uint_as_float(sw[1]);
  }
  // Halves of each 16-lane row: w[0] stays in lanes 0..7, w[1] in 8..15.
  const bool hi8 = (lane & 8) != 0;
  float tot = (hi8 ? w[1] : w[0]) + dpp<0x128>(hi8 ? w[0] : w[1]);
  tot += dpp<0xB1>(tot);   // lane ^ 1
  tot += dpp<0x4E>(tot);   // lane ^ 2
  tot += dpp<0x141>(tot);  // mirror within 8 lanes
  const int g = lane >> 3;
  const int r = ((g & 1) << 2) | (g & 2) | (g >> 2);
  if ((lane & 7) == 0 && r < R && k * R + r < n_rows) res[k * R + r] = tot;
}

// ---------------------------------------------------------------- kernel

// Optional timestamps (100 MHz s_memrealtime), [workgroup][layer][32 events].
#define STEP_MARK(l, ev)                                                                           \
  do {                                                                                             \
    if (P.trace && threadIdx.x == 64 * kLoaders) P.trace[((size_t)wg * (L + 1) + (l)) * 32 + (ev)] = wall_clock64(); \
  } while (0)

// Epoch of (layer, phase) in this step; phases: 0 q/k/v, 1 attention
// partials, 2 combined attention output, 3 x after O, 4 SwiGLU output, 5 x
// after down, 6 argmax keys.  The layer field is 6 bits wide.
__device__ __forceinline__ unsigned ep_of(unsigned base, int l, int ph) { return base + (unsigned)l * 8u + ph; }

template <typename TW, typename TKV, int NPD, bool FD>
__global__ __launch_bounds__(kStepThreads) void k_decode_step(StepParams<TW, TKV> P) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  __shared__ RingSync sy;
  RingSync HH_LDS* const syp = (RingSync HH_LDS*)&sy;
  __shared__ float2 rope_p[32];                    // cos/sin of this step's position
  __shared__ LayerPtrs<TW> lptr[kStepMaxLayers];   // per-layer weight pointers
  __shared__ int item_pages[kMaxItemPages];        // physical pages of this workgroup's attention item
  __shared__ float qs[kMaxGroup * 64];             // the item's query heads, pre-scaled
  __shared__ float kn[64], vn[64];                 // key / value of the current position (kv head of the item)
  __shared__ unsigned long long kred[kNC];

  const int wg = blockIdx.x, nwg = gridDim.x;
  // The wave index is uniform; read into a scalar register, every per-wave
  // choice (role, rows, slots) becomes a scalar branch.  The 4-bit kernel
  // runs 6 % faster for it (0.516 against 0.548 ms per token).
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int d = P.d, F = P.F, hq = P.hq, hkv = P.hkv, G = hq / hkv, L = P.n_layers;
  const int S = P.ring_slots;
  const int s = P.stream;
  const int p = P.pos[s];
  const int tok = P.feed ? P.feed[0] : P.pending[s];
  const int t = p + 1;  // keys attended this step
  const unsigned E0 = P.epoch;
  const int s_cap = nwg / hkv;
  // A step whose input is the -1 left by an abandoned step, or that starts
  // after a wait of this context gave up, computes nothing: the stream
  // records -1 at this position and moves on, so device-fed consumers see
  // the failure instead of a plausible token.
  // (One thread decides, so the whole workgroup takes the same branch.)
  __shared__ int dead;
  if (tid == 0) dead = tok < 0 || __hip_atomic_load((int*)P.err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0;
  __syncthreads();
  if (dead) {
    if (wg == 0 && tid == 0) {
      P.pending[s] = -1;
      P.hist[(size_t)s * P.max_ctx + p] = -1;
      P.pos[s] = p + 1;
    }
    return;
  }

  char* ring = smem;
  float* xa = reinterpret_cast<float*>(smem + (size_t)S * kSlot);  // [d] normalised inputs (QKV, GU, head)
  float* xc = xa + d;                                               // [F] or [Hq*64] + attention states
  float* res = xc + step_xc_floats(d, hq, hkv);  // [kStepResFloats] phase results
  float* xown = res + kStepResFloats;                               // [kStepResFloats] this workgroup's rows of x
  float* st = xc + hq * 64;                                         // [kNC][G][kStRow] attention states

  Plan pl;
  make_plan<TW, TKV, NPD>(pl, P, wg, nwg, t);
  const int nd = pl.rd1 - pl.rd0;

  if (tid < kMaxRing) {
    syp->consumed[tid] = tid - S;
    syp->landed[tid] = tid - S;
  }
  if (tid == 0) {
    syp->wait_ticks = P.wait_ticks > 0 ? P.wait_ticks : kWaitTicks;
    syp->quiet = 0;
    syp->cbar = 0;
    syp->abort = 0;
  }
  if (tid < 32) rope_p[tid] = P.rope[(size_t)p * 32 + tid];
  for (int i = tid; i < L; i += kStepThreads) lptr[i] = P.layer[i];
  if (pl.has_item)
    for (int i = tid; i < pl.it_pg1 - pl.it_pg0; i += kStepThreads)
      item_pages[i] = P.page_table[(size_t)s * P.kv.max_pages + pl.it_pg0 + i];
  const typename StepEmbed<TW>::type* erow = P.embed + (size_t)tok * d;
  const float ws = P.wscale_inv;
  for (int i = tid; i < nd; i += kStepThreads) xown[i] = (float)erow[pl.rd0 + i];
  const int page_p = P.page_table[(size_t)s * P.kv.max_pages + p / kPage];  // page receiving this position
  __syncthreads();

  // ================================================================ streaming waves
  // Wave lw streams the slots n with n % kLoaders == lw.  After issuing one,
  // it waits until at most `depth` of its slots are in flight and marks the
  // oldest as landed.
  if (wave < kLoaders) {
    __builtin_amdgcn_s_setprio(3);  // issue ahead of the compute wave sharing this SIMD
    const int lw = wave;
    const int depth = P.load_depth < 1 ? 1 : P.load_depth > 7 ? 7 : P.load_depth;
    int n = 0;                      // slot index in the stream
    int mypub = lw - kLoaders;      // this wave's last slot marked landed
    unsigned long long stall = 0;
    auto publish_upto = [&](int upto) {  // mark this wave's slots <= upto landed
      while (mypub + kLoaders <= upto) {
        mypub += kLoaders;
        if (lane == 0) *(volatile int HH_LDS*)&syp->landed[mypub % S] = mypub;
      }
    };
    // Per-lane byte offsets of the two 1 KiB halves of a swizzled fp16 K/V
    // tile: lane i fills LDS chunk i, i.e. key 8 h + i / 8, chunk position
    // i % 8, which holds the key's source chunk (i % 8) ^ ((key / 2) % 8).
    int kvoff[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int key = 8 * h + (lane >> 3);
      kvoff[h] = key * 128 + (((lane & 7) ^ ((key >> 1) & 7)) << 4);
    }
    for (int l = 0; l <= L; ++l) {
      if (lw == 0 && P.trace && lane == 0) P.trace[((size_t)wg * (L + 1) + l) * 32 + 20] = wall_clock64();
      stall = 0;
      for (int sg = (l < L ? SG_QKV : SG_HEAD); sg <= (l < L ? SG_DOWN : SG_HEAD); ++sg) {
        const int nsl = pl.slots(sg);
        if (nsl == 0) continue;
        // The segment's matrix, rows and row size.
        const char* W = nullptr;
        RowMap map{0, 0, 0, F};
        int nrows = 0, rowb = 0;
        if (sg != SG_KV) {
          rowb = std::is_same<TW, Q4Row>::value ? kQ4RowBytes : d * (int)sizeof(TW);
          if (sg == SG_QKV) {
            W = reinterpret_cast<const char*>(lptr[l].wqkv);
            map = RowMap{1, pl.pq0, 0, F};
            nrows = 2 * (pl.pq1 - pl.pq0);
          } else if (sg == SG_O) {
            W = reinterpret_cast<const char*>(lptr[l].wo);
            map = RowMap{0, pl.rd0, 0, F};
            nrows = nd;
          } else if (sg == SG_GU) {
            W = reinterpret_cast<const char*>(lptr[l].wgu);
            map = RowMap{2, pl.j0, pl.j1 - pl.j0, F};
            nrows = 2 * (pl.j1 - pl.j0);
          } else if (sg == SG_DOWN) {
            W = reinterpret_cast<const char*>(lptr[l].wdownT);
            map = RowMap{0, pl.j0, 0, F};
            nrows = pl.j1 - pl.j0;
          } else {
            W = reinterpret_cast<const char*>(P.head);
            map = RowMap{0, pl.v0, 0, F};
            nrows = pl.v1 - pl.v0;
          }
        }
        const bool full = (rowb & 1023) == 0;
        const int base = n;  // stream index of the segment's first slot
        for (int k = (lw - base % kLoaders + kLoaders) % kLoaders; k < nsl; k += kLoaders) {
          const int m = base + k, pos = m % S;
          // Wait for a free ring position; first mark everything in flight
          // landed, so compute waves never wait on slots held back here.
          if (*(volatile int HH_LDS*)&syp->consumed[pos] < m - S) {
            const unsigned long long t0s = wall_clock64();
            if (lw == 0 && P.trace && lane == 0 && stall == 0) P.trace[((size_t)wg * (L + 1) + l) * 32 + 23] = t0s;
            HH_STEP_VMWAIT(0);
            compiler_fence();
            publish_upto(m - kLoaders);
            unsigned spins = 0;
            unsigned long long t0 = 0;
            while (*(volatile int HH_LDS*)&syp->consumed[pos] < m - S) {
              __builtin_amdgcn_s_sleep(1);
              if (give_up(spins, t0, syp, (int HH_GLB*)P.err)) break;
            }
            compiler_fence();
            stall += wall_clock64() - t0s;
          }
          // Optionally keep HBM quiet while this workgroup's compute waves wait
          // for other workgroups (shorter exchange latency, less prefetch).
          // quiet 1: stop issuing; quiet 2: keep at most one slot in flight.
          if (P.quiet == 1 && *(volatile int HH_LDS*)&syp->quiet) {
            HH_STEP_VMWAIT(0);
            compiler_fence();
            publish_upto(m - kLoaders);
            unsigned spins = 0;
            unsigned long long t0 = 0;
            while (*(volatile int HH_LDS*)&syp->quiet) {
              __builtin_amdgcn_s_sleep(1);
              if (give_up(spins, t0, syp, (int HH_GLB*)P.err)) break;
            }
            compiler_fence();
          } else if (P.quiet == 2 && *(volatile int HH_LDS*)&syp->quiet) {
            HH_STEP_VMWAIT(0);
            compiler_fence();
            publish_upto(m - kLoaders);
          }
          char* dst = ring + (size_t)pos * kSlot;
          if (sg == SG_KV) {
            // K/V pages of the item: fp16 tiles swizzled (2 pages per slot:
            // [K a][V a][K b][V b]), fp32 tiles plain (1 page: [K][V]).
            const int pg_a = pl.it_pg0 + k * pl.pps;
#pragma unroll
            for (int q = 0; q < 8; ++q) {
              const char* src;
              if constexpr (sizeof(TKV) == 2) {
                const int pg = pg_a + (q >> 2);
                const int pgv = pg < pl.it_pg1 ? pg : pg_a;  // a missing page b repeats page a
                const int phys = item_pages[pgv - pl.it_pg0];
                const int kind = (q >> 1) & 1;
                src = reinterpret_cast<const char*>(P.kvc + P.kv.head_tile(l, phys, kind, pl.it_g)) + kvoff[q & 1];
              } else {
                const int phys = item_pages[pg_a - pl.it_pg0];
                const int kind = q >> 2;
                const int key = (q & 3) * 4 + (lane >> 4);
                src = reinterpret_cast<const char*>(P.kvc + P.kv.head_tile(l, phys, kind, pl.it_g)) + key * 256 +
                      (lane & 15) * 16;
              }
              __builtin_amdgcn_global_load_lds(src, dst + q * 1024, 16, 0, 0);
            }
          } else if constexpr (std::is_same<TW, Q4Row>::value) {
            issue_q4_slot(dst, W, map, nrows, k);
          } else {
            issue_row_slot<NPD>(dst, W, map, rowb, nrows, k, full);
          }
          // Keep at most `depth` of this wave's slots in flight.
          switch (depth) {
            case 1: HH_STEP_VMWAIT(0); break;
            case 2: HH_STEP_VMWAIT(8); break;
            case 3: HH_STEP_VMWAIT(16); break;
            case 4: HH_STEP_VMWAIT(24); break;
            case 5: HH_STEP_VMWAIT(32); break;
            case 6: HH_STEP_VMWAIT(40); break;
            default: HH_STEP_VMWAIT(48); break;
          }
          compiler_fence();
          publish_upto(m - kLoaders * (depth - 1));
        }
        n = base + nsl;
      }
      if (lw == 0 && P.trace && lane == 0) {
        P.trace[((size_t)wg * (L + 1) + l) * 32 + 21] = stall;
        P.trace[((size_t)wg * (L + 1) + l) * 32 + 22] = wall_clock64();
      }
    }
    HH_STEP_VMWAIT(0);
    compiler_fence();
    publish_upto(n - 1);
    return;
  }

  // ================================================================ compute waves
  const int cw = wave - kLoaders;
  int gen = 0;  // compute-wave barrier generation
  int HH_GLB* err = (int HH_GLB*)P.err;

  // Stage x (words at epoch ep, or the embedding row when src is null) times
  // the RMSNorm gain into xa; returns 1 / rms after a compute-wave barrier.
  // Optional delay before a phase's first poll (ticks of the 100 MHz clock):
  // a poll issued before the last producer's words are visible costs a full
  // extra round trip.
  auto poll_delay = [&](int ticks) {
    if (ticks > 0) {
      const unsigned long long t_end = wall_clock64() + (unsigned)ticks;
      while (wall_clock64() < t_end) __builtin_amdgcn_s_sleep(1);
    }
  };
  auto quiet = [&](int on) {
    if (cw == 0 && lane == 0) *(volatile int HH_LDS*)&syp->quiet = on;
  };
  auto tr = [&](int l, int ev) {
    return PollTrace{P.trace ? P.trace + ((size_t)wg * (L + 1) + l) * 32 + ev : nullptr};
  };
  auto stage_norm = [&](const unsigned long long* src, unsigned ep, const float* gain, PollTrace pt) -> float {
    quiet(1);
    if (src) poll_delay(P.poll_delay);
    float ss = 0.f;
    const int tc = tid - 64 * kLoaders;
    if (src) {
      // The gains are loaded before the words are polled, so they never
      // cost a round trip of their own after the words arrive.
      for (int base = tc; base < d; base += kNC * 64 * kPollX) {
        float gr[kPollX];
#pragma unroll
        for (int u = 0; u < kPollX; ++u) {
          const int i = base + u * kNC * 64;
          gr[u] = i < d ? ((const float HH_GLB*)gain)[i] : 0.f;
        }
        poll_words<kPollX>([=](int i) { return src + base - tc + i; }, d - (base - tc), ep, syp, err,
                           [&](int i, float v) {
                             const int u = (i - tc) / (kNC * 64);
                             float g = 0.f;
#pragma unroll
                             for (int q = 0; q < kPollX; ++q) g = q == u ? gr[q] : g;
                             xa[base - tc + i] = v * g;
                             ss = fmaf(v, v, ss);
                           },
                           pt);
      }
    } else {
      for (int i = tc; i < d; i += kNC * 64) {
        const float v = (float)erow[i];
        xa[i] = v * ((const float HH_GLB*)gain)[i];
        ss = fmaf(v, v, ss);
      }
    }
    ss = wave_sum_u(ss);
    if (lane == 0) syp->ss[cw] = ss;
    cbar(syp, gen, err);
    quiet(0);
    float tot = 0.f;
#pragma unroll
    for (int w = 0; w < kNC; ++w) tot += syp->ss[w];
    return rsqrtf(tot / (float)d + P.eps);
  };

  // Consume this wave's slots of a row segment (global slot index base);
  auto run_rows = [&](int base, int nsl, const float* xs, int K, int nrows) {
    if constexpr (std::is_same<TW, Q4Row>::value) {
      // This lane's 32 inputs (elements 512 c + 8 l + e) in the layout of the
      // biased code pairs serve every slot of the phase.
      h2x xh[16];
      float xb[4];
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const float4 a = *reinterpret_cast<const float4*>(xs + 512 * c + 8 * lane);
        const float4 b = *reinterpret_cast<const float4*>(xs + 512 * c + 8 * lane + 4);
        xh[4 * c] = h2x{(_Float16)a.x, (_Float16)b.x};
        xh[4 * c + 1] = h2x{(_Float16)(a.y * 0.0625f), (_Float16)(b.y * 0.0625f)};
        xh[4 * c + 2] = h2x{(_Float16)a.z, (_Float16)b.z};
        xh[4 * c + 3] = h2x{(_Float16)(a.w * 0.0625f), (_Float16)(b.w * 0.0625f)};
        const float s02 = ((float)xh[4 * c].x + (float)xh[4 * c].y) + ((float)xh[4 * c + 2].x + (float)xh[4 * c + 2].y);
        const float s13 =
            ((float)xh[4 * c + 1].x + (float)xh[4 * c + 1].y) + ((float)xh[4 * c + 3].x + (float)xh[4 * c + 3].y);
        xb[c] = -fmaf(1032.f, s02, 1152.f * s13);
      }
      auto rows = [&](auto RC) {
        constexpr int R = decltype(RC)::value;
        for (int k = cw; k < nsl; k += kNC) {
          const int n = base + k, pos = n % S;
          wait_landed(syp, n, pos, err);
          q4_slot_rows<R>(ring + (size_t)pos * kSlot, xh, xb, k, nrows, res);
          release_slot(syp, pos, n);
        }
      };
      const int R = q4_rows(nrows);
      if (R == 2) rows(std::integral_constant<int, 2>{});
      else if (R == 3) rows(std::integral_constant<int, 3>{});
      else rows(std::integral_constant<int, kQ4Rows>{});
    } else {
      for (int k = cw; k < nsl; k += kNC) {
        const int n = base + k, pos = n % S;
        wait_landed(syp, n, pos, err);
        slot_rows<TW, NPD, FD>(ring + (size_t)pos * kSlot, xs, K, k, nrows, res);
        release_slot(syp, pos, n);
      }
    }
  };

  float inv = 1.f;
  for (int l = 0; l < L; ++l) {
    const int lbase = l * pl.per_layer;

    // ---------------------------------------------------- RMSNorm + QKV + RoPE
    STEP_MARK(l, 0);
    inv = stage_norm(l == 0 ? nullptr : P.ll_xb, ep_of(E0, l - 1, 5), lptr[l].attn_norm, tr(l, 24));
    STEP_MARK(l, 1);
    run_rows(lbase + pl.o_qkv, pl.n_qkv, xa, d, 2 * (pl.pq1 - pl.pq0));
    cbar(syp, gen, err);
    STEP_MARK(l, 2);
    if (cw == 0) {
      const unsigned e = ep_of(E0, l, 0);
      for (int lp = lane; lp < pl.pq1 - pl.pq0; lp += 64) {
        const int gp = pl.pq0 + lp, head = gp >> 5, i = gp & 31;
        const float y0 = res[2 * lp] * (inv * ws), y1 = res[2 * lp + 1] * (inv * ws);
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
    }
    STEP_MARK(l, 3);

    // ---------------------------------------------------- attention item
    if (pl.has_item) {
      STEP_MARK(l, 4);
      const int g = pl.it_g, j0 = g * G;
      const unsigned e0 = ep_of(E0, l, 0);
      const float qscale = 0.125f * 1.4426950408889634f;  // 1/sqrt(64) * log2(e)
      {
        // One poll over the item's query heads, then the key and value of
        // the current position (offsets from ll_q: a select among three
        // pointers would be lowered to a table in scratch memory).
        const unsigned long long* qb = P.ll_q;
        const int oq = j0 * 64, ok = (int)(P.ll_kn - P.ll_q) + g * 64 - G * 64,
                  ov = (int)(P.ll_vn - P.ll_q) + g * 64 - G * 64 - 64;
        quiet(1);
        poll_words<2>(
            [=](int i) { return qb + i + oq + (i >= G * 64 ? ok - oq : 0) + (i >= G * 64 + 64 ? ov - ok : 0); }, G * 64 + 128, e0,
            syp, err, [&](int i, float v) {
              if (i < G * 64) qs[i] = v * qscale;
              else if (i < G * 64 + 64) kn[i - G * 64] = v;
              else vn[i - G * 64 - 64] = v;
            });
      }
      cbar(syp, gen, err);
      quiet(0);
      STEP_MARK(l, 5);
      const int kbase = lbase + pl.o_kv;
      const int nsl = pl.n_kv;
      const int key_base = pl.it_pg0 * kPage;
      const int kend = t < pl.it_pg1 * kPage ? t : pl.it_pg1 * kPage;  // keys of this item: [key_base, kend)
      float* stw = st + (size_t)cw * G * kStRow;
      if constexpr (sizeof(TKV) == 2) {
        // ---- fp16 K/V: 16x16x32 MFMAs.  S^T[key][head] = K Q^T, lane l:
        // head l % 16, keys 4 (l / 16) + r of each 16-key tile; then
        // O^T[dim][head] += V^T P^T with the contraction's key order chosen
        // so P goes from the score accumulators straight into the B operand.
        const int hcol = lane & 15, grp = lane >> 4;
        f16x8v qh[2], ql[2];
#pragma unroll
        for (int hh = 0; hh < 2; ++hh)
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float v = hcol < G ? qs[hcol * 64 + 32 * hh + 8 * grp + e] : 0.f;
            const _Float16 hi = (_Float16)v;
            qh[hh][e] = hi;
            ql[hh][e] = (_Float16)(v - (float)hi);
          }
        float m = -INFINITY, lsum = 0.f;
        f32x4 oacc[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) oacc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
        for (int k = cw; k < nsl; k += kNC) {
          const int n = kbase + k, pos = n % S;
          const int key0 = key_base + k * 32;  // position of the slot's first key
          wait_landed(syp, n, pos, err);
          char* slot = ring + (size_t)pos * kSlot;
          // The slot holding this step's position gets the exchanged key and
          // value (its cache row may not have been written yet when it was
          // streamed) -- also when that position is the slot's last row;
          // rows past the item's last key get zero values (stale or foreign
          // slots: weight 0, and 0 * NaN would be NaN).
          if (p >= key0 && p < key0 + 32 && p < kend) {
            const int kk = p - key0, tt = kk >> 4, key = kk & 15;
            const int off = tt * 4096 + key * 128 + ((((lane >> 3) ^ ((key >> 1) & 7))) << 4) + (lane & 7) * 2;
            *reinterpret_cast<_Float16*>(slot + off) = (_Float16)kn[lane];
            *reinterpret_cast<_Float16*>(slot + off + 2048) = (_Float16)vn[lane];
          }
          if (key0 + 32 > kend) {
            for (int r = kend - key0 + (lane >> 3); r < 32; r += 8)
              *reinterpret_cast<u32x4*>(slot + (r >> 4) * 4096 + 2048 + (r & 15) * 128 + (lane & 7) * 16) =
                  u32x4{0u, 0u, 0u, 0u};
          }
          f32x4 sc[2];
#pragma unroll
          for (int tt = 0; tt < 2; ++tt) {
            sc[tt] = f32x4{0.f, 0.f, 0.f, 0.f};
            const int key = lane & 15;
            const char* Kt = slot + tt * 4096;
#pragma unroll
            for (int hh = 0; hh < 2; ++hh) {
              const int c = 4 * hh + grp;
              const f16x8v a = *reinterpret_cast<const f16x8v*>(Kt + key * 128 + ((c ^ ((key >> 1) & 7)) << 4));
              sc[tt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, qh[hh], sc[tt], 0, 0, 0);
              sc[tt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, ql[hh], sc[tt], 0, 0, 0);
            }
          }
          float bm = -INFINITY;
#pragma unroll
          for (int tt = 0; tt < 2; ++tt)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const int kp = key0 + 16 * tt + 4 * grp + r;
              const float v = kp < kend ? sc[tt][r] : -INFINITY;
              sc[tt][r] = v;
              bm = fmaxf(bm, v);
            }
          bm = fmaxf(bm, __shfl_xor(bm, 16, 64));
          bm = fmaxf(bm, __shfl_xor(bm, 32, 64));
          const float mn = fmaxf(m, bm);  // finite: the slot's first key is in the item
          const float alpha = exp2f(m - mn);
          f16x8v pb;
          float ls = 0.f;
#pragma unroll
          for (int tt = 0; tt < 2; ++tt)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const float pv = exp2f(sc[tt][r] - mn);
              ls += pv;
              pb[4 * tt + r] = (_Float16)pv;
            }
          lsum = lsum * alpha + ls;
#pragma unroll
          for (int i = 0; i < 4; ++i) oacc[i] *= alpha;
#pragma unroll
          for (int dt = 0; dt < 4; ++dt) {
            const int dim = 16 * dt + hcol;
            f16x8v a;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              const int tt = e >> 2, kk = 4 * grp + (e & 3);
              a[e] = *reinterpret_cast<const _Float16*>(slot + tt * 4096 + 2048 + kk * 128 +
                                                        ((((dim >> 3) ^ ((kk >> 1) & 7))) << 4) + (dim & 7) * 2);
            }
            oacc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, pb, oacc[dt], 0, 0, 0);
          }
          m = mn;
          release_slot(syp, pos, n);
        }
        lsum += __shfl_xor(lsum, 16, 64);
        lsum += __shfl_xor(lsum, 32, 64);
        if (hcol < G) {
          float* sh = stw + hcol * kStRow;
          if (grp == 0) {
            sh[0] = m;
            sh[1] = lsum;
          }
#pragma unroll
          for (int dt = 0; dt < 4; ++dt)
#pragma unroll
            for (int r = 0; r < 4; ++r) sh[2 + 16 * dt + 4 * grp + r] = oacc[dt][r];
        }
      } else {
        // ---- fp32 K/V (one page per slot): VALU.  Lane l: key l / 4,
        // dims 16 (l % 4) .. + 16; G query heads at once.
        const int key = lane >> 2, quarter = lane & 3;
        float m[kMaxGroupF32], lsum[kMaxGroupF32], o[kMaxGroupF32][16];
#pragma unroll
        for (int h = 0; h < kMaxGroupF32; ++h) {
          m[h] = -INFINITY;
          lsum[h] = 0.f;
#pragma unroll
          for (int e = 0; e < 16; ++e) o[h][e] = 0.f;
        }
        for (int k = cw; k < nsl; k += kNC) {
          const int n = kbase + k, pos = n % S;
          const int kp = key_base + k * kPage + key;
          wait_landed(syp, n, pos, err);
          const float* Kt = reinterpret_cast<const float*>(ring + (size_t)pos * kSlot) + key * 64 + quarter * 16;
          const float* Vt = Kt + kPage * 64;
          float kf[16], vf[16];
#pragma unroll
          for (int e = 0; e < 16; e += 4) {
            const float4 a = *reinterpret_cast<const float4*>(Kt + e);
            const float4 b = *reinterpret_cast<const float4*>(Vt + e);
            kf[e] = a.x; kf[e + 1] = a.y; kf[e + 2] = a.z; kf[e + 3] = a.w;
            vf[e] = b.x; vf[e + 1] = b.y; vf[e + 2] = b.z; vf[e + 3] = b.w;
          }
          if (kp == p) {
#pragma unroll
            for (int e = 0; e < 16; ++e) {
              kf[e] = kn[quarter * 16 + e];
              vf[e] = vn[quarter * 16 + e];
            }
          }
          if (kp >= kend) {
#pragma unroll
            for (int e = 0; e < 16; ++e) vf[e] = 0.f;
          }
          release_slot(syp, pos, n);
#pragma unroll
          for (int h = 0; h < kMaxGroupF32; ++h) {
            if (h < G) {
              float sc = 0.f;
#pragma unroll
              for (int e = 0; e < 16; ++e) sc = fmaf(qs[h * 64 + quarter * 16 + e], kf[e], sc);
              sc += dpp<0xB1>(sc);
              sc += dpp<0x4E>(sc);
              if (kp >= kend) sc = -INFINITY;
              const float mn = fmaxf(m[h], wave_max_u(sc));
              const float alpha = exp2f(m[h] - mn);
              const float pk = exp2f(sc - mn);
              lsum[h] = lsum[h] * alpha + (quarter == 0 ? pk : 0.f);
#pragma unroll
              for (int e = 0; e < 16; ++e) o[h][e] = fmaf(pk, vf[e], o[h][e] * alpha);
              m[h] = mn;
            }
          }
        }
#pragma unroll
        for (int h = 0; h < kMaxGroupF32; ++h) {
          if (h < G) {
            const float lt = wave_sum_u(lsum[h]);
            float* sh = stw + h * kStRow;
#pragma unroll
            for (int e = 0; e < 16; ++e) {
              float v = o[h][e];
              v += dpp<0x124>(v);  // keys of a 16-lane row with this quarter
              v += dpp<0x128>(v);
              v += __shfl_xor(v, 16, 64);
              v += __shfl_xor(v, 32, 64);
              if (key == 0) sh[2 + quarter * 16 + e] = v;
            }
            if (lane == 0) {
              sh[0] = m[h];
              sh[1] = lt;
            }
          }
        }
      }
      cbar(syp, gen, err);
      STEP_MARK(l, 6);
      // Merge the compute waves' states into this item's partial of each
      // query head (wave h % 7 takes head h; lane = head dimension) and
      // publish it.  With more splits than the O-phase consumers merge,
      // split 0 then combines all splits of the head (its own included, read
      // back like the others) into the final output.
      {
        const unsigned e1 = ep_of(E0, l, 1);
        for (int h = cw; h < G; h += kNC) {
          float M = -INFINITY;
          for (int w = 0; w < kNC; ++w) M = fmaxf(M, st[((size_t)w * G + h) * kStRow]);
          float Ls = 0.f, O = 0.f;
          for (int w = 0; w < kNC; ++w) {
            const float* sh = st + ((size_t)w * G + h) * kStRow;
            const float f = exp2f(sh[0] - M);
            Ls = fmaf(sh[1], f, Ls);
            O = fmaf(sh[2 + lane], f, O);
          }
          O /= Ls;
          const int j = j0 + h;
          unsigned long long* pp = P.ll_part + ((size_t)j * s_cap + pl.it_sp) * 66;
          // Partial = (log2 weight lambda = M + log2 Ls, normalised o): the
          // splits of a head combine as a softmax over lambda.
          if (lane == 0) ll_put(pp, M + log2f(Ls), e1);
          ll_put(pp + 2 + lane, O, e1);
          if (!pl.consumer_comb && pl.it_sp == 0) {
            const unsigned long long* pj = P.ll_part + (size_t)j * s_cap * 66;
            float Lm = -INFINITY, Ws = 0.f, Oc = 0.f;
            for (int r0 = 0; r0 < pl.nspl; r0 += 8) {
              unsigned long long w[8][2];
              unsigned stale = 0;
#pragma unroll
              for (int u = 0; u < 8; ++u) {
                const int i = r0 + u;
                w[u][0] = w[u][1] = (unsigned long long)e1 << 32;
                if (i < pl.nspl) {
                  const unsigned long long* q0 = pj + (size_t)i * 66;
                  w[u][0] = ll_get(q0);
                  w[u][1] = ll_get(q0 + 2 + lane);
                }
                stale |= ((unsigned)(w[u][0] >> 32) != e1 || (unsigned)(w[u][1] >> 32) != e1 ? 1u : 0u) << u;
              }
              unsigned spins = 0;
              unsigned long long t0 = 0;
              while (stale) {
                __builtin_amdgcn_s_sleep(1);
#pragma unroll
                for (int u = 0; u < 8; ++u)
                  if (stale & (1u << u)) {
                    const unsigned long long* q0 = pj + (size_t)(r0 + u) * 66;
                    w[u][0] = ll_get(q0);
                    w[u][1] = ll_get(q0 + 2 + lane);
                    if ((unsigned)(w[u][0] >> 32) == e1 && (unsigned)(w[u][1] >> 32) == e1) stale &= ~(1u << u);
                  }
                if (stale && give_up(spins, t0, syp, err)) break;
              }
#pragma unroll
              for (int u = 0; u < 8; ++u) {
                if (r0 + u < pl.nspl) {
                  const float lam = __uint_as_float((unsigned)w[u][0]);
                  const float oi = __uint_as_float((unsigned)w[u][1]);
                  const float Mn = fmaxf(Lm, lam);
                  const float fa = exp2f(Lm - Mn), fb = exp2f(lam - Mn);
                  Oc = Oc * fa + oi * fb;
                  Ws = Ws * fa + fb;
                  Lm = Mn;
                }
              }
            }
            Oc /= Ws;
            ll_put(P.ll_o + j * 64 + lane, Oc, ep_of(E0, l, 2));
          }
        }
      }
      STEP_MARK(l, 7);
    }

    // ---------------------------------------------------- O projection + residual
    STEP_MARK(l, 8);
    quiet(1);
    poll_delay(P.poll_delay);
    if (pl.consumer_comb) {
      // o[j] = softmax over the splits i of head j of lambda_i, applied to
      // the splits' o_i.  Wave cw takes heads cw + kNC u; all of a wave's
      // loads are issued before any wait.
      constexpr int HPW = kHeadsPerWave;  // heads per wave and round
      const unsigned e1 = ep_of(E0, l, 1);
      const int nsp = pl.nspl;
      for (int jr = cw; jr < hq; jr += kNC * HPW) {
        unsigned long long w[HPW][kMaxConsumerSplits][2];
        unsigned stale = 0;
#pragma unroll
        for (int u = 0; u < HPW; ++u)
#pragma unroll
          for (int i = 0; i < kMaxConsumerSplits; ++i) {
            const int j = jr + u * kNC;
            w[u][i][0] = w[u][i][1] = (unsigned long long)e1 << 32;
            if (j < hq && i < nsp) {
              const unsigned long long* q0 = P.ll_part + ((size_t)j * s_cap + i) * 66;
              w[u][i][0] = ll_get(q0);
              w[u][i][1] = ll_get(q0 + 2 + lane);
            }
            stale |= ((unsigned)(w[u][i][0] >> 32) != e1 || (unsigned)(w[u][i][1] >> 32) != e1 ? 1u : 0u)
                     << (u * kMaxConsumerSplits + i);
          }
        unsigned spins = 0;
        unsigned long long t0 = 0;
        while (stale) {
          __builtin_amdgcn_s_sleep(1);
#pragma unroll
          for (int u = 0; u < HPW; ++u)
#pragma unroll
            for (int i = 0; i < kMaxConsumerSplits; ++i) {
              const unsigned bit = 1u << (u * kMaxConsumerSplits + i);
              if (stale & bit) {
                const unsigned long long* q0 = P.ll_part + ((size_t)(jr + u * kNC) * s_cap + i) * 66;
                w[u][i][0] = ll_get(q0);
                w[u][i][1] = ll_get(q0 + 2 + lane);
                if ((unsigned)(w[u][i][0] >> 32) == e1 && (unsigned)(w[u][i][1] >> 32) == e1) stale &= ~bit;
              }
            }
          if (stale && give_up(spins, t0, syp, err)) break;
        }
#pragma unroll
        for (int u = 0; u < HPW; ++u) {
          const int j = jr + u * kNC;
          if (j < hq) {
            float M = -INFINITY;
#pragma unroll
            for (int i = 0; i < kMaxConsumerSplits; ++i)
              if (i < nsp) M = fmaxf(M, __uint_as_float((unsigned)w[u][i][0]));
            float Ws = 0.f, O = 0.f;
#pragma unroll
            for (int i = 0; i < kMaxConsumerSplits; ++i)
              if (i < nsp) {
                const float f = exp2f(__uint_as_float((unsigned)w[u][i][0]) - M);
                Ws += f;
                O = fmaf(f, __uint_as_float((unsigned)w[u][i][1]), O);
              }
            xc[j * 64 + lane] = O / Ws;
          }
        }
      }
    } else {
      poll_span<kPollX>(P.ll_o, hq * 64, ep_of(E0, l, 2), syp, err, [&](int i, float v) { xc[i] = v; });
    }
    cbar(syp, gen, err);
    quiet(0);
    STEP_MARK(l, 9);
    run_rows(lbase + pl.o_o, pl.n_o, xc, hq * 64, nd);
    cbar(syp, gen, err);
    STEP_MARK(l, 10);
    if (cw == 0) {
      const unsigned e = ep_of(E0, l, 3);
      for (int i = lane; i < nd; i += 64) {
        const float xn = xown[i] + res[i] * ws;
        xown[i] = xn;
        ll_put(P.ll_xa + pl.rd0 + i, xn, e);
      }
    }
    STEP_MARK(l, 11);

    // ---------------------------------------------------- RMSNorm + gate/up + SwiGLU
    STEP_MARK(l, 12);
    inv = stage_norm(P.ll_xa, ep_of(E0, l, 3), lptr[l].mlp_norm, tr(l, 26));
    STEP_MARK(l, 13);
    const int nj = pl.j1 - pl.j0;
    run_rows(lbase + pl.o_gu, pl.n_gu, xa, d, 2 * nj);
    cbar(syp, gen, err);
    STEP_MARK(l, 14);
    // ---------------------------------------------------- down projection (split-K) + residual
    // This workgroup owns SwiGLU outputs j0 .. j1 - 1, so it multiplies them
    // by the same columns of Wdown (rows of Wdown^T): a partial of the whole
    // output, no exchange of the SwiGLU vector.  Partials are summed per
    // output row, in workgroup order, by the row's owner.
    {
      float* red = xa;  // [kNC][d] over the staging buffers, idle once the slots are done
      const int dbase = lbase + pl.o_down;
      if constexpr (std::is_same<TW, Q4Row>::value) {
        // 4-bit Wdown^T rows: lane l accumulates outputs 512 c + 8 l + e (as
        // the 16-bit rows do): sum_j c_j q_je with c_j = m_j s_j,(16c + l/4).
        float acc[32];
#pragma unroll
        for (int i = 0; i < 32; ++i) acc[i] = 0.f;
        auto rows = [&](auto RC) {
          constexpr int R = decltype(RC)::value;
          for (int k = cw; k < pl.n_down; k += kNC) {
            const int n = dbase + k, pos = n % S;
            wait_landed(syp, n, pos, err);
            const char* slot = ring + (size_t)pos * kSlot;
            // Words and scales first (the LDS reads overlap), then the FMAs.
            unsigned wds[R][4];
            float scs[R][4];
#pragma unroll
            for (int r = 0; r < R; ++r)
#pragma unroll
              for (int c = 0; c < 4; ++c) {
                wds[r][c] = *reinterpret_cast<const unsigned*>(slot + r * 1024 + 256 * c + 4 * lane);
                scs[r][c] = (float)*reinterpret_cast<const __bf16*>(slot + kQ4ScaleOff + r * 128 +
                                                                     2 * (16 * c + (lane >> 2)));
              }
            // Lane r < R forms the SwiGLU output of the slot's row r (rows
            // missing from the slot repeat its first row: weight 0).
            const int jv = k * R + lane;
            const float mv =
                lane < R && jv < nj ? silu(res[jv] * (inv * ws)) * (res[nj + jv] * (inv * ws)) : 0.f;
#pragma unroll
            for (int r = 0; r < R; ++r) {
              const float mj = lane_read(mv, r);
#pragma unroll
              for (int c = 0; c < 4; ++c) {
                const float cj = mj * scs[r][c];
                h2x q[4];
                q4_codes(wds[r][c], q);
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                  acc[8 * c + j] = fmaf(cj, (float)q[j].x, acc[8 * c + j]);
                  acc[8 * c + j + 4] = fmaf(cj, (float)q[j].y, acc[8 * c + j + 4]);
                }
              }
            }
            release_slot(syp, pos, n);
          }
        };
        const int R = q4_rows(nj);
        if (R == 2) rows(std::integral_constant<int, 2>{});
        else if (R == 3) rows(std::integral_constant<int, 3>{});
        else rows(std::integral_constant<int, kQ4Rows>{});
        // Sum the compute waves' partials (fixed order) and publish them.
#pragma unroll
        for (int c = 0; c < 4; ++c)
#pragma unroll
          for (int e = 0; e < 8; e += 4)
            *reinterpret_cast<float4*>(red + (size_t)cw * d + 512 * c + 8 * lane + e) =
                make_float4(acc[8 * c + e], acc[8 * c + e + 1], acc[8 * c + e + 2], acc[8 * c + e + 3]);
      } else {
        constexpr int E = 16 / (int)sizeof(TW), PE = 1024 / (int)sizeof(TW);
        constexpr int RPS = rows_per_slot(NPD);
        float acc[NPD * E];
#pragma unroll
        for (int i = 0; i < NPD * E; ++i) acc[i] = 0.f;
        for (int k = cw; k < pl.n_down; k += kNC) {
          const int n = dbase + k, pos = n % S;
          wait_landed(syp, n, pos, err);
          const char* slot = ring + (size_t)pos * kSlot;
#pragma unroll
          for (int r = 0; r < RPS; ++r) {
            const int jl = k * RPS + r;
            // Rows missing from the slot repeat its first row: weight 0.
            const float mj = jl < nj ? silu(res[jl] * (inv * ws)) * (res[nj + jl] * (inv * ws)) : 0.f;
#pragma unroll
            for (int c = 0; c < NPD; ++c) {
              const u32x4 w = *reinterpret_cast<const u32x4*>(slot + (r * NPD + c) * 1024 + lane * 16);
              float wf[E];
              widen16(w, wf, TW());
#pragma unroll
              for (int e = 0; e < E; ++e) acc[c * E + e] = fmaf(mj, wf[e], acc[c * E + e]);
            }
          }
          release_slot(syp, pos, n);
        }
        // Sum the compute waves' partials (fixed order) and publish them.
#pragma unroll
        for (int c = 0; c < NPD; ++c)
#pragma unroll
          for (int e = 0; e < E; e += 4)
            *reinterpret_cast<float4*>(red + (size_t)cw * d + c * PE + lane * E + e) =
                make_float4(acc[c * E + e], acc[c * E + e + 1], acc[c * E + e + 2], acc[c * E + e + 3]);
      }
      cbar(syp, gen, err);
      STEP_MARK(l, 15);
      {
        const unsigned e4 = ep_of(E0, l, 4);
        for (int i = tid - 64 * kLoaders; i < d; i += kNC * 64) {
          float v = 0.f;
#pragma unroll
          for (int w = 0; w < kNC; ++w) v += red[(size_t)w * d + i];
          ll_put(P.ll_dp + (size_t)wg * d + i, v * ws, e4);
        }
      }
      cbar(syp, gen, err);  // red is reused below
      STEP_MARK(l, 16);
      // Gather the partials of this workgroup's rows from every workgroup.
      quiet(1);
      poll_delay(P.poll_delay);
      {
        const unsigned long long* dp = P.ll_dp + pl.rd0;
        const int ndd = nd > 0 ? nd : 1;
        poll_words<kPollX>([=](int i) { return dp + (size_t)(i / ndd) * d + (i % ndd); }, nwg * nd,
                           ep_of(E0, l, 4), syp, err, [&](int i, float v) { red[i] = v; }, tr(l, 28));
      }
      cbar(syp, gen, err);
      quiet(0);
      STEP_MARK(l, 17);
      // Row r of this workgroup: 32 lanes sum workgroups q, q + 32, ...;
      // then the 32 lanes combine (a fixed reduction tree).
      {
        const unsigned e5 = ep_of(E0, l, 5);
        for (int t0 = 0; t0 < nd * 32; t0 += kNC * 64) {
          const int t = t0 + tid - 64 * kLoaders, r = t >> 5, q = t & 31;
          float v = 0.f;
          if (r < nd)
            for (int w = q; w < nwg; w += 32) v += red[w * nd + r];
          v = row_sum16(v);
          v += __shfl_xor(v, 16, 64);
          if (q == 0 && r < nd) {
            const float xn = xown[r] + v;
            xown[r] = xn;
            ll_put(P.ll_xb + pl.rd0 + r, xn, e5);
          }
        }
      }
      STEP_MARK(l, 19);
    }
  }

  // ---------------------------------------------------- final RMSNorm + LM head + argmax
  STEP_MARK(L, 0);
  inv = stage_norm(L == 0 ? nullptr : P.ll_xb, ep_of(E0, L - 1, 5), P.final_norm, tr(L, 24));
  STEP_MARK(L, 1);
  const int nv = pl.v1 - pl.v0;
  run_rows(L * pl.per_layer, pl.head_slots, xa, d, nv);
  cbar(syp, gen, err);
  STEP_MARK(L, 2);
  if (cw == 0) {
    unsigned long long best = 0ull;
    for (int i = lane; i < nv; i += 64) {
      const float v = res[i] * (inv * ws);
      if (P.logits) P.logits[pl.v0 + i] = v;
      const unsigned long long k = argmax_key(v, (uint32_t)(pl.v0 + i));
      best = k > best ? k : best;
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      const unsigned long long o2 = __shfl_xor(best, off, 64);
      best = o2 > best ? o2 : best;
    }
    const unsigned e6 = ep_of(E0, L, 6);
    if (lane == 0) {
      ll_put_u(P.ll_keys + 2 * wg, (unsigned)(best >> 32), e6);
      ll_put_u(P.ll_keys + 2 * wg + 1, (unsigned)best, e6);
    }
    if (wg == 0) {
      // fail_wait (a test of the failure path, set from the host): wait for
      // an epoch no workgroup publishes, so this wait runs into its limit.
      const unsigned e6w = P.fail_wait ? E0 + 511u : e6;
      unsigned long long b = 0ull;
      for (int i0 = 0; i0 < nwg; i0 += 64) {
        const int i = i0 + lane;
        unsigned long long hi = (unsigned long long)e6w << 32, lo = hi;
        if (i < nwg) {
          hi = ll_get(P.ll_keys + 2 * i);
          lo = ll_get(P.ll_keys + 2 * i + 1);
        }
        unsigned spins = 0;
        unsigned long long t0 = 0;
        while (__any((unsigned)(hi >> 32) != e6w || (unsigned)(lo >> 32) != e6w)) {
          __builtin_amdgcn_s_sleep(1);
          if ((unsigned)(hi >> 32) != e6w) hi = ll_get(P.ll_keys + 2 * i);
          if ((unsigned)(lo >> 32) != e6w) lo = ll_get(P.ll_keys + 2 * i + 1);
          if (give_up(spins, t0, syp, err)) break;
        }
        if (i < nwg) {
          const unsigned long long k = ((unsigned long long)(unsigned)hi << 32) | (unsigned)lo;
          b = k > b ? k : b;
        }
      }
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) {
        const unsigned long long o2 = __shfl_xor(b, off, 64);
        b = o2 > b ? o2 : b;
      }
      if (lane == 0) {
        // A wait of this step gave up: its argmax is not a result.
        const bool gave_up = __hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0;
        const int nt = gave_up ? -1 : argmax_index(b);
        P.pending[s] = nt;
        P.hist[(size_t)s * P.max_ctx + p] = nt;
        P.pos[s] = p + 1;
      }
    }
    STEP_MARK(L, 3);
  }
  (void)kred;
}

// ---------------------------------------------------------------- launcher

template <typename TW, typename TKV>
int StepKernel<TW, TKV>::xc_floats(int d, int F, int hq, int hkv) {
  return step_xc_floats(d, hq, hkv);
}

template <typename TW, typename TKV>
size_t StepKernel<TW, TKV>::lds_bytes(int d, int F, int hq, int hkv, int ring_slots) {
  return (size_t)ring_slots * kSlot + (size_t)(d + xc_floats(d, F, hq, hkv) + 2 * kStepResFloats) * sizeof(float);
}

// Pieces (1 KiB) per weight row for the row lengths d and F.
template <typename TW>
constexpr int pieces(int k) {
  return (k * (int)sizeof(TW) + 1023) / 1024;
}

template <typename TW, typename TKV, int NPD, bool FD>
static hipError_t launch_step(const StepParams<TW, TKV>& P, int nwg, hipStream_t st) {
  const size_t lds = StepKernel<TW, TKV>::lds_bytes(P.d, P.F, P.hq, P.hkv, P.ring_slots);
  auto kern = k_decode_step<TW, TKV, NPD, FD>;
  if (lds > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  kern<<<nwg, kStepThreads, lds, st>>>(P);
  return hipGetLastError();
}

// Instantiated row shapes (every streamed row has d elements): bf16 rows of
// exactly 4 pieces (d = 2048), fp32 rows of exactly 1 piece (d = 256), 4-bit
// rows of 1152 bytes (d = 2048; their slots are laid out separately).
template <typename TW>
static bool shape_ok(int d, int F) {
  (void)F;
  if constexpr (std::is_same<TW, Q4Row>::value) return d == 2048;  // 64 groups: one per lane
  if (sizeof(TW) == 2) return d * 2 == 4 * 1024;
  return d * 4 == 1024;
}

template <typename TW, typename TKV>
bool StepKernel<TW, TKV>::supports(int d, int F, int hq, int hkv, int V, int n_layers, int nwg) {
  if (!shape_ok<TW>(d, F)) return false;
  const int G = hq / hkv;
  if (hq * 64 != d || hq % hkv || G > kMaxGroup || nwg / hkv < 1 || n_layers > kStepMaxLayers) return false;
  if (sizeof(TKV) == 4 && G > kMaxGroupF32) return false;
  const int pairs = (hq + 2 * hkv) * 32;
  // Row results per phase (gate/up shares grow by at most the item rebalancing).
  if ((V + nwg - 1) / nwg > kStepResFloats || 2 * ((F + nwg - 1) / nwg) + 64 > kStepResFloats ||
      2 * ((pairs + nwg - 1) / nwg) > kStepResFloats || 2 * ((d + nwg - 1) / nwg) > kStepResFloats)
    return false;
  if (lds_bytes(d, F, hq, hkv, kStepRingSlots) > 148 * 1024) return false;  // plus the static LDS
  return true;
}

template <typename TW, typename TKV>
hipError_t StepKernel<TW, TKV>::launch(const StepParams<TW, TKV>& P, int nwg, hipStream_t st) {
  if constexpr (sizeof(TW) == 2) return launch_step<TW, TKV, 4, true>(P, nwg, st);
  else return launch_step<TW, TKV, 1, true>(P, nwg, st);
}

template <typename TW, typename TKV>
int StepKernel<TW, TKV>::max_blocks_per_cu(int d, int F, int hq, int hkv) {
  const size_t lds = lds_bytes(d, F, hq, hkv, kStepRingSlots);
  int nb = 0;
  hipError_t e;
  if constexpr (sizeof(TW) == 2)
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, k_decode_step<TW, TKV, 4, true>, kStepThreads, lds);
  else
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, k_decode_step<TW, TKV, 1, true>, kStepThreads, lds);
  return e == hipSuccess ? nb : 0;
}

template struct StepKernel<_Float16, _Float16>;
template struct StepKernel<float, float>;
template struct StepKernel<Q4Row, _Float16>;

}  // namespace hh
