// Decode-side kernels for gfx950: embedding gather, the batch-1 weight-streaming
// GEMVs with fused prologues/epilogues (RMSNorm, RoPE + KV append, SwiGLU,
// residual add, LM head + argmax), split-K paged GQA attention and its
// log-sum-exp combine, row RMSNorm, and the per-step bookkeeping.
//
// Batch-1 decode is bound by streaming the weights from HBM once per token, so
// every GEMV reads its matrix with coalesced 16-byte non-temporal loads (a
// wavefront reads 1 KiB contiguous per instruction), keeps the fp32 activation
// vector in LDS, accumulates in fp32 registers and reduces with wave64
// shuffles.  Each workgroup owns whole output rows, so results are written
// without atomics and are bitwise reproducible.
#include "hh_kernels.h"

namespace hh {

// ---------------------------------------------------------------- step setup

// Row bookkeeping + embedding gather (x[r] = E[token_r] widened to fp32).
// Decode: row r belongs to stream row_stream[r] at position pos[stream].
// Prefill: all rows belong to `prefill_stream`, row r at position pos + r.
// The token is feed[r] if feed != nullptr, else the stream's pending argmax.
template <typename TW>
__global__ __launch_bounds__(256) void k_prep_embed(int prefill_stream, const int* __restrict__ feed,
                                                    int* __restrict__ row_stream, int* __restrict__ row_pos,
                                                    const int* __restrict__ pos, const int* __restrict__ pending,
                                                    unsigned long long* __restrict__ slot,
                                                    const TW* __restrict__ embed, float* __restrict__ x, int d) {
  // prefill_stream >= 0: rows r of that stream at positions pos + r; -1: one
  // row per listed stream at its position; -2: row_stream and row_pos given.
  const int r = blockIdx.x;
  const int s = prefill_stream >= 0 ? prefill_stream : row_stream[r];
  const int p = prefill_stream == -2 ? row_pos[r] : pos[s] + (prefill_stream >= 0 ? r : 0);
  int tok = feed ? feed[r] : pending[s];
  if (threadIdx.x == 0 && prefill_stream != -2) {
    row_pos[r] = p;
    if (prefill_stream >= 0) row_stream[r] = s;
  }
  // A negative pending token marks a stream whose earlier decode step gave
  // up (see k_finalize): the row gathers row 0 and its argmax slot is pinned
  // to the all-ones key, which k_finalize turns back into -1.
  if (tok < 0) {
    tok = 0;
    if (threadIdx.x == 0) slot[s] = ~0ull;
  }
  const TW* e = embed + (size_t)tok * d;
  for (int i = threadIdx.x; i < d; i += blockDim.x) x[(size_t)r * d + i] = (float)e[i];
}

// Consume the argmax slots of rows [r0, r0 + n): pending token, history and
// stream position advance to row_pos + 1.  With slot == nullptr only the
// positions advance (an intermediate prefill pass).
__global__ void k_finalize(int r0, int n, const int* __restrict__ row_stream, const int* __restrict__ row_pos,
                           unsigned long long* __restrict__ slot, int* __restrict__ pending,
                           int* __restrict__ hist, int* __restrict__ pos, int max_ctx) {
  for (int i = threadIdx.x; i < n; i += blockDim.x) {
    const int r = r0 + i;
    const int s = row_stream[r];
    const int p = row_pos[r];
    if (slot) {
      const unsigned long long key = slot[s];
      const int tok = key == ~0ull ? -1 : argmax_index(key);
      pending[s] = tok;
      hist[(size_t)s * max_ctx + p] = tok;
      slot[s] = 0ull;
    }
    pos[s] = p + 1;
  }
}

// ---------------------------------------------------------------- GEMV core

// Stage the fp32 input vector into LDS, optionally RMS-normalised:
// xs = x * rsqrt(mean(x^2) + eps) * gain.
__device__ __forceinline__ void stage_vector(const float* __restrict__ x, const float* __restrict__ gain,
                                             float eps, int K, float* xs, float* red) {
  float ss = 0.f;
  for (int i = threadIdx.x; i < K; i += 256) {
    const float v = x[i];
    xs[i] = v;
    ss += v * v;
  }
  if (gain) {
    const float tot = block_sum256(ss, red);
    const float inv = rsqrtf(tot / (float)K + eps);
    for (int i = threadIdx.x; i < K; i += 256) xs[i] = xs[i] * inv * gain[i];
  }
  __syncthreads();
}

// out[r] = dot(W[rows[r], :], xs) for R rows; rows[r] < 0 contributes 0.
// Each thread owns 16-byte chunks c = tid, tid + 256, ... of the K axis and
// issues all R row loads of a chunk before using them.
template <typename TW, int R>
__device__ __forceinline__ void gemv_rows(const TW* __restrict__ W, const int* rows, int K,
                                          const float* xs, float* out, float* red) {
  constexpr int V = Vec16<TW>::n;
  const int nch = K / V;
  float acc[R];
#pragma unroll
  for (int r = 0; r < R; ++r) acc[r] = 0.f;
  for (int c = threadIdx.x; c < nch; c += 256) {
    float w[R][V];
#pragma unroll
    for (int r = 0; r < R; ++r) {
      if (rows[r] >= 0) load16<TW, true>(W + (size_t)rows[r] * K + (size_t)c * V, w[r]);
      else {
#pragma unroll
        for (int i = 0; i < V; ++i) w[r][i] = 0.f;
      }
    }
    float xv[V];
#pragma unroll
    for (int i = 0; i < V; ++i) xv[i] = xs[c * V + i];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int i = 0; i < V; ++i) acc[r] = fmaf(w[r][i], xv[i], acc[r]);
  }
  const int wv = threadIdx.x >> 6, lane = threadIdx.x & 63;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const float s = wave_sum(acc[r]);
    if (lane == 0) red[wv * R + r] = s;
  }
  __syncthreads();
  if (threadIdx.x < R) {
    const int r = threadIdx.x;
    out[r] = red[r] + red[R + r] + red[2 * R + r] + red[3 * R + r];
  }
  __syncthreads();
}

// ---------------------------------------------------------------- GEMV kernels

// Fused RMSNorm + QKV projection + RoPE + KV append for one decode row.
// Block b handles 4 rotary pairs: pair gp = 4b + p is (head gp / 32, i = gp % 32),
// i.e. rows head*64 + i and head*64 + i + 32 of W_qkv = [Wq; Wk; Wv].  Query
// heads are rotated into q; key heads rotated and value heads copied into the
// row's KV page slot.
template <typename TW, typename TKV>
__global__ __launch_bounds__(256) void k_qkv_gemv(const TW* __restrict__ W, const float* __restrict__ x,
                                                  const float* __restrict__ gain, float eps, int d, int hq, int hkv,
                                                  const int* __restrict__ row_stream, const int* __restrict__ row_pos,
                                                  const float2* __restrict__ rope, float* __restrict__ q,
                                                  TKV* __restrict__ kv, KvLayout L, int layer,
                                                  const int* __restrict__ page_table) {
  extern __shared__ float xs[];
  __shared__ float red[4 * 8];
  __shared__ float res[8];
  stage_vector(x, gain, eps, d, xs, red);
  int rows[8];
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    const int gp = blockIdx.x * 4 + p;
    rows[2 * p] = (gp / 32) * 64 + gp % 32;
    rows[2 * p + 1] = rows[2 * p] + 32;
  }
  gemv_rows<TW, 8>(W, rows, d, xs, res, red);
  if (threadIdx.x < 4) {
    const int gp = blockIdx.x * 4 + threadIdx.x;
    const int head = gp / 32, i = gp % 32;
    const float y0 = res[2 * threadIdx.x], y1 = res[2 * threadIdx.x + 1];
    const int s = row_stream[0], p = row_pos[0];
    if (head < hq + hkv) {
      const float2 cs = rope[(size_t)p * 32 + i];
      const float r0 = y0 * cs.x - y1 * cs.y, r1 = y1 * cs.x + y0 * cs.y;
      if (head < hq) {
        q[head * 64 + i] = r0;
        q[head * 64 + i + 32] = r1;
      } else {
        const int page = page_table[(size_t)s * L.max_pages + p / kPage];
        TKV* dst = kv + L.head_tile(layer, page, 0, head - hq) + (p % kPage) * 64;
        dst[i] = from_f32<TKV>(r0);
        dst[i + 32] = from_f32<TKV>(r1);
      }
    } else {
      const int page = page_table[(size_t)s * L.max_pages + p / kPage];
      TKV* dst = kv + L.head_tile(layer, page, 1, head - hq - hkv) + (p % kPage) * 64;
      dst[i] = from_f32<TKV>(y0);
      dst[i + 32] = from_f32<TKV>(y1);
    }
  }
}

// xres[row] += dot(W[row, :], in) for rows [8b, 8b + 8) < N (O and down projections).
template <typename TW>
__global__ __launch_bounds__(256) void k_resid_gemv(const TW* __restrict__ W, const float* __restrict__ in, int K,
                                                    int N, float* __restrict__ xres) {
  extern __shared__ float xs[];
  __shared__ float red[4 * 8];
  __shared__ float res[8];
  stage_vector(in, nullptr, 0.f, K, xs, red);
  int rows[8];
#pragma unroll
  for (int r = 0; r < 8; ++r) rows[r] = blockIdx.x * 8 + r < N ? blockIdx.x * 8 + r : -1;
  gemv_rows<TW, 8>(W, rows, K, xs, res, red);
  if (threadIdx.x < 8 && rows[threadIdx.x] >= 0) xres[rows[threadIdx.x]] += res[threadIdx.x];
}

// Fused RMSNorm + gate/up projection + SwiGLU: m[j] = silu(Wg_j . h) * (Wu_j . h)
// for j in [4b, 4b + 4); W = [Wg; Wu] so up row j is row F + j.
template <typename TW>
__global__ __launch_bounds__(256) void k_gateup_gemv(const TW* __restrict__ W, const float* __restrict__ x,
                                                     const float* __restrict__ gain, float eps, int d, int F,
                                                     float* __restrict__ m) {
  extern __shared__ float xs[];
  __shared__ float red[4 * 8];
  __shared__ float res[8];
  stage_vector(x, gain, eps, d, xs, red);
  int rows[8];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int j = blockIdx.x * 4 + r;
    rows[r] = j < F ? j : -1;
    rows[4 + r] = j < F ? F + j : -1;
  }
  gemv_rows<TW, 8>(W, rows, d, xs, res, red);
  if (threadIdx.x < 4 && rows[threadIdx.x] >= 0)
    m[blockIdx.x * 4 + threadIdx.x] = silu(res[threadIdx.x]) * res[4 + threadIdx.x];
}

// Final RMSNorm + LM head for one row `row` of x, streaming: two blocks per
// CU each stage the normalised vector once and take an equal share of the
// rows, each wave one row at a time (lane l: 16-byte chunks l, l + 64,
// l + 128, l + 192) with its next two rows' loads in flight in two more
// register sets (strict rotation: no register copy, so the compiler waits for
// exactly the oldest set).  Writes optional fp32 logits and a packed
// (value, index) atomicMax into the stream's argmax slot.  Rows need at most
// 4 chunks per lane (d * sizeof(TW) <= 4096).
template <typename TW>
__device__ __forceinline__ void head_row_loads(u32x4* w, const TW* __restrict__ W, int row, int nch) {
  const u32x4* src = reinterpret_cast<const u32x4*>(W + (size_t)row * nch * Vec16<TW>::n);
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int c = 0; c < 4; ++c) w[c] = __builtin_nontemporal_load(src + min(lane + 64 * c, nch - 1));
}

template <typename TW>
__device__ __forceinline__ float head_row_dot(const u32x4* w, const float* xs, int nch) {
  constexpr int V = Vec16<TW>::n;
  const int lane = threadIdx.x & 63;
  float acc = 0.f;
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const int ch = lane + 64 * c;
    const bool in = ch < nch;
    const float4* xc = reinterpret_cast<const float4*>(xs + (in ? ch : nch - 1) * V);
    float wf[V], xv[V];
    widen16(w[c], wf, TW());
#pragma unroll
    for (int e = 0; e < V / 4; ++e) {  // 16-byte LDS reads; the select acts on the values
      const float4 t = xc[e];
      xv[4 * e] = in ? t.x : 0.f;
      xv[4 * e + 1] = in ? t.y : 0.f;
      xv[4 * e + 2] = in ? t.z : 0.f;
      xv[4 * e + 3] = in ? t.w : 0.f;
    }
#pragma unroll
    for (int e = 0; e < V; ++e) acc = fmaf(wf[e], xv[e], acc);
  }
  return wave_sum(acc);
}

template <typename TW>
__global__ __launch_bounds__(256) void k_head_stream(const TW* __restrict__ W, const float* __restrict__ x,
                                                     const float* __restrict__ gain, float eps, int d, int V, int row,
                                                     const int* __restrict__ row_stream, float* __restrict__ logits,
                                                     unsigned long long* __restrict__ slot) {
  extern __shared__ float xs[];
  __shared__ float red[4];
  __shared__ unsigned long long kred[4];
  stage_vector(x + (size_t)row * d, gain, eps, d, xs, red);
  const int r0 = (int)(((long long)V * blockIdx.x) / gridDim.x), r1 = (int)(((long long)V * (blockIdx.x + 1)) / gridDim.x);
  if (r0 >= r1) return;
  const int nch = d / Vec16<TW>::n;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  unsigned long long best = 0ull;
  auto take = [&](const u32x4* w, int r) {
    const float v = head_row_dot<TW>(w, xs, nch);
    if (lane == 0) {
      if (logits) logits[r] = v;
      const unsigned long long k = argmax_key(v, (uint32_t)r);
      best = k > best ? k : best;
    }
  };
  // Rows r0 + wave, + 4, ...; loads past r1 re-read the block's last row.
  u32x4 a[4], b[4], c[4];
  head_row_loads<TW>(a, W, min(r0 + wave, r1 - 1), nch);
  head_row_loads<TW>(b, W, min(r0 + wave + 4, r1 - 1), nch);
  for (int r = r0 + wave; r < r1; r += 12) {
    head_row_loads<TW>(c, W, min(r + 8, r1 - 1), nch);
    take(a, r);
    if (r + 4 >= r1) break;
    head_row_loads<TW>(a, W, min(r + 12, r1 - 1), nch);
    take(b, r + 4);
    if (r + 8 >= r1) break;
    head_row_loads<TW>(b, W, min(r + 16, r1 - 1), nch);
    take(c, r + 8);
  }
  if (lane == 0) kred[wave] = best;
  __syncthreads();
  if (threadIdx.x == 0 && slot) {
    for (int w = 1; w < 4; ++w) best = kred[w] > best ? kred[w] : best;
    atomicMax(slot + row_stream[row], best);
  }
}

// Compute units of the current device (cached per device).
static int device_cus() {
  static int cus[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cus[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cus[dev] = n;
  }
  return cus[dev];
}

// Final RMSNorm + LM head rows [8b, 8b + 8) < V for decode row `row`:
// optional fp32 logits, and a packed (value, index) atomicMax into the
// stream's argmax slot (slot == nullptr: logits only).
template <typename TW>
__global__ __launch_bounds__(256) void k_head_gemv(const TW* __restrict__ W, const float* __restrict__ x,
                                                   const float* __restrict__ gain, float eps, int d, int V, int row,
                                                   const int* __restrict__ row_stream, float* __restrict__ logits,
                                                   unsigned long long* __restrict__ slot) {
  extern __shared__ float xs[];
  __shared__ float red[4 * 8];
  __shared__ float res[8];
  stage_vector(x + (size_t)row * d, gain, eps, d, xs, red);
  int rows[8];
#pragma unroll
  for (int r = 0; r < 8; ++r) rows[r] = blockIdx.x * 8 + r < V ? blockIdx.x * 8 + r : -1;
  gemv_rows<TW, 8>(W, rows, d, xs, res, red);
  if (threadIdx.x == 0) {
    unsigned long long best = 0ull;
    for (int r = 0; r < 8; ++r) {
      if (rows[r] < 0) continue;
      if (logits) logits[rows[r]] = res[r];
      const unsigned long long k = argmax_key(res[r], (uint32_t)rows[r]);
      best = k > best ? k : best;
    }
    if (slot) atomicMax(slot + row_stream[row], best);
  }
}

// ---------------------------------------------------------------- attention

// Split count and pages per split for a row attending over t keys.
__device__ __forceinline__ void split_plan(int t, int s_max, int& nspl, int& pps) {
  const int npg = (t + kPage - 1) / kPage;
  nspl = npg < s_max ? npg : s_max;
  pps = (npg + nspl - 1) / nspl;
  nspl = (npg + pps - 1) / pps;
}

// Paged GQA attention of row r (blockIdx.z) for kv head g (blockIdx.y), pages
// of split blockIdx.x.  Wave w serves query heads g*G + w, g*G + w + 4, ...
// Scores use exp2 with log2(e)/sqrt(64) folded into q; online softmax.
// s_max > 1: writes (m, l, o[64]) partials for k_attn_combine;
// s_max == 1: writes the normalised output directly (o32 fp32 and oM).
template <typename TKV, typename TM>
__global__ __launch_bounds__(256) void k_attn(const float* __restrict__ q, const TKV* __restrict__ kv, KvLayout L,
                                              int layer, const int* __restrict__ page_table,
                                              const int* __restrict__ row_stream, const int* __restrict__ row_pos,
                                              int hq, int hkv, int s_max, float* __restrict__ part,
                                              float* __restrict__ o32, TM* __restrict__ oM) {
  const int r = blockIdx.z, g = blockIdx.y, sp = blockIdx.x;
  const int s = row_stream[r];
  const int t = row_pos[r] + 1;
  int nspl, pps;
  split_plan(t, s_max, nspl, pps);
  if (sp >= nspl) return;
  const int npg = (t + kPage - 1) / kPage;
  const int pg0 = sp * pps, pg1 = min(npg, pg0 + pps);
  const int G = hq / hkv;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int key = lane >> 2, quarter = lane & 3;
  const float qscale = 0.125f * 1.4426950408889634f;  // 1/sqrt(64) * log2(e)
  for (int jj = w; jj < G; jj += 4) {
    const int j = g * G + jj;
    const float* qj = q + ((size_t)r * hq + j) * 64 + quarter * 16;
    float qv[16];
#pragma unroll
    for (int e = 0; e < 16; ++e) qv[e] = qj[e] * qscale;
    float m = -INFINITY, l = 0.f, o = 0.f;
    for (int pg = pg0; pg < pg1; ++pg) {
      const int page = page_table[(size_t)s * L.max_pages + pg];
      const TKV* Kp = kv + L.head_tile(layer, page, 0, g);
      const TKV* Vp = kv + L.head_tile(layer, page, 1, g);
      float kf[16];
      load16<TKV>(Kp + key * 64 + quarter * 16, kf);
      load16<TKV>(Kp + key * 64 + quarter * 16 + Vec16<TKV>::n, kf + Vec16<TKV>::n);
      if constexpr (Vec16<TKV>::n == 4) {
        load16<TKV>(Kp + key * 64 + quarter * 16 + 8, kf + 8);
        load16<TKV>(Kp + key * 64 + quarter * 16 + 12, kf + 12);
      }
      float sc = 0.f;
#pragma unroll
      for (int e = 0; e < 16; ++e) sc = fmaf(qv[e], kf[e], sc);
      sc += __shfl_xor(sc, 1, kWave);
      sc += __shfl_xor(sc, 2, kWave);
      if (pg * kPage + key >= t) sc = -INFINITY;
      const float mn = fmaxf(m, wave_max(sc));
      const float alpha = exp2f(m - mn);
      const float p = exp2f(sc - mn);
      l = l * alpha + wave_sum(quarter == 0 ? p : 0.f);
      o *= alpha;
#pragma unroll
      for (int kk = 0; kk < kPage; ++kk) {
        // Slots past the stream's length hold stale data (possibly non-finite
        // bit patterns): their weight is 0, and 0 * NaN would be NaN.
        const float v = pg * kPage + kk < t ? (float)Vp[kk * 64 + lane] : 0.f;
        o = fmaf(__shfl(p, kk * 4, kWave), v, o);
      }
      m = mn;
    }
    if (s_max == 1) {
      const float out = o / l;
      o32[((size_t)r * hq + j) * 64 + lane] = out;
      if (oM) oM[((size_t)r * hq + j) * 64 + lane] = (TM)out;
    } else {
      float* pp = part + (((size_t)r * hq + j) * s_max + sp) * 66;
      if (lane == 0) {
        pp[0] = m;
        pp[1] = l;
      }
      pp[2 + lane] = o;
    }
  }
}

// Log-sum-exp combine of the split partials of row blockIdx.y, query head
// blockIdx.x (one lane per head dimension).
template <typename TM>
__global__ __launch_bounds__(64) void k_attn_combine(const float* __restrict__ part,
                                                     const int* __restrict__ row_pos, int hq, int s_max,
                                                     float* __restrict__ o32, TM* __restrict__ oM) {
  const int j = blockIdx.x, r = blockIdx.y, lane = threadIdx.x;
  int nspl, pps;
  split_plan(row_pos[r] + 1, s_max, nspl, pps);
  const float* pp = part + ((size_t)r * hq + j) * s_max * 66;
  float M = -INFINITY;
  for (int i = 0; i < nspl; ++i) M = fmaxf(M, pp[i * 66]);
  float Lsum = 0.f, O = 0.f;
  for (int i = 0; i < nspl; ++i) {
    const float f = exp2f(pp[i * 66] - M);
    Lsum = fmaf(pp[i * 66 + 1], f, Lsum);
    O = fmaf(pp[i * 66 + 2 + lane], f, O);
  }
  const float out = O / Lsum;
  o32[((size_t)r * hq + j) * 64 + lane] = out;
  if (oM) oM[((size_t)r * hq + j) * 64 + lane] = (TM)out;
}

// Paged GQA attention for decode rows: one 512-thread workgroup per (row,
// kv head) serves the G query heads of that kv head, so each K/V page is
// read once.  The row's page list is staged in LDS; wave w takes pages w,
// w + 8, ..., its first four (three for fp32 caches or eight query heads)
// all issued at the start, later ones with the next two pages' K/V in flight
// in two more register sets (strict rotation, no register copies).  Lane
// (key = lane / 4, quarter =
// lane % 4) holds 16 dims of one key; scores use exp2 with 1/sqrt(64)*log2(e)
// folded into q; each head keeps its own online softmax state.  The waves'
// states are merged in LDS, one wave per head.
constexpr int kRowsMaxPages = 2048;  // pages of one row kept in LDS (32768 positions); later ones are read from the table

template <typename TKV>
struct KvPage {
  u32x4 k[sizeof(TKV)], v[sizeof(TKV)];  // 16 elements of a key: 2 chunks (fp16) or 4 (fp32)
};

template <typename TKV>
__device__ __forceinline__ void kv_page_load(KvPage<TKV>& P, const TKV* kv, const KvLayout& L, int layer,
                                             int page, int g, int key, int quarter) {
  const u32x4* Kp = reinterpret_cast<const u32x4*>(kv + L.head_tile(layer, page, 0, g) + key * 64 + quarter * 16);
  const u32x4* Vp = reinterpret_cast<const u32x4*>(kv + L.head_tile(layer, page, 1, g) + key * 64 + quarter * 16);
#pragma unroll
  for (int c = 0; c < (int)sizeof(TKV); ++c) {
    P.k[c] = Kp[c];
    P.v[c] = Vp[c];
  }
}

// kv is not __restrict__: with the QKV fold the kernel also writes the cache
// (through fold.kv) at each row's position.
template <typename TKV, typename TM, int G>
__global__ __launch_bounds__(512) void k_attn_rows(const float* __restrict__ q, const TKV* kv, KvLayout L,
                                                   int layer, const int* __restrict__ page_table,
                                                   const int* __restrict__ row_stream, const int* __restrict__ row_pos,
                                                   int hq, float* __restrict__ o32, TM* __restrict__ oM,
                                                   QkvFold<TKV> fold) {
  constexpr int NW = 8, NT = NW * 64;
  constexpr int SLOT = 66;  // m, l, o[64]
  __shared__ float st[NW * G * 4 * SLOT];
  __shared__ int pts[kRowsMaxPages];
  // Folded QKV: this row's q heads g G .. g G + G - 1, then k and v of head
  // g (64 values each), and the new key and value as the cache stores them.
  __shared__ float qkv_s[(G + 2) * 64];
  __shared__ __attribute__((aligned(16))) TKV new_kv[2][64];
  const int g = blockIdx.x, r = blockIdx.y;
  const bool folded = fold.part != nullptr;
  const int hkv = hq / G;
  // Folded QKV: column c < (G + 2) 64 of this row's slice (q heads, then k,
  // then v of head g); thread t takes columns t + NT i.
  constexpr int CPT = ((G + 2) * 64 + NT - 1) / NT;
  auto fold_col = [&](int c) {
    return c < G * 64 ? g * G * 64 + c
                      : (c < (G + 1) * 64 ? (hq + g) * 64 + (c - G * 64) : (hq + hkv + g) * 64 + (c - (G + 1) * 64));
  };
  // The first eight split partials of those columns load before anything
  // else: they depend on nothing, and the row's position and page list are
  // two dependent round trips away.  Clamped indices; extras unused.
  float fp[CPT][8];
  if (folded) {
    const size_t stride = (size_t)gridDim.y * fold.ncols;
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int c = min(threadIdx.x + NT * i, (G + 2) * 64 - 1);
      const float* pp = fold.part + (size_t)r * fold.ncols + fold_col(c);
#pragma unroll
      for (int j = 0; j < 8; ++j) fp[i][j] = pp[min(j, fold.splits - 1) * stride];
    }
  }
  const int s = row_stream[r], p = row_pos[r], t = p + 1, npg = (t + kPage - 1) / kPage;
  // The wave index is uniform: taken into a scalar register, page choices and
  // the last-page test below become scalar branches.
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63, key = lane >> 2,
            quarter = lane & 3;
  const float qscale = 0.125f * 1.4426950408889634f;  // 1/sqrt(64) * log2(e)
  // Rotation of the pair (e, e + 32) this thread applies below (q heads and k).
  float2 cs = make_float2(1.f, 0.f);
  if (folded && threadIdx.x < (G + 1) * 32) cs = fold.rope[(size_t)p * 32 + (threadIdx.x & 31)];
  // Pages wave, wave + 8, ...: the wave's first PU pages are all issued here,
  // before the folded QKV reduction, whose loads they overlap (the row's own
  // key, which the reduction writes, is taken from LDS, not from these
  // loads); their page ids (and the new key's page) come straight from the
  // table, one round trip after the row's position.  Waves with fewer pages
  // re-read the row's last page, so that every wave issues the same loads
  // and the waits stay exact (spreading those re-reads over the row's pages
  // measured the same).  The LDS copy of the page list serves rows
  // longer than PU * 8 pages, which continue below with three register sets
  // in rotation.
  constexpr int PU = sizeof(TKV) == 2 && G <= 4 ? 4 : 3;
  const int* prow = page_table + (size_t)s * L.max_pages;
  int pid[PU];
#pragma unroll
  for (int k = 0; k < PU; ++k) pid[k] = prow[min(wave + NW * k, npg - 1)];
  const int new_page = folded ? prow[p / kPage] : 0;
  const bool long_row = npg > PU * NW;
  if (long_row)
    for (int i = threadIdx.x; i < npg && i < kRowsMaxPages; i += NT) pts[i] = prow[i];
  auto page_of = [&](int pg) { return pg < kRowsMaxPages ? pts[pg] : prow[pg]; };
  KvPage<TKV> P[PU];
#pragma unroll
  for (int k = 0; k < PU; ++k) kv_page_load(P[k], kv, L, layer, pid[k], g, key, quarter);
  float qv[G][16];
  if (!folded) {
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
      for (int e = 0; e < 16; ++e) qv[h][e] = q[((size_t)r * hq + g * G + h) * 64 + quarter * 16 + e] * qscale;
  } else {
    // Sum the split partials of the row's columns in split order and scale
    // them (the reduction the QKV epilogue would otherwise run).
    const size_t stride = (size_t)gridDim.y * fold.ncols;
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int c = threadIdx.x + NT * i;
      if (c < (G + 2) * 64) {
        float v = 0.f;
#pragma unroll
        for (int j = 0; j < 8; ++j)
          if (j < fold.splits) v += fp[i][j];
        // More than eight splits: the rest eight at a time.
        const float* pp = fold.part + (size_t)r * fold.ncols + fold_col(c);
        for (int s0 = 8; s0 < fold.splits; s0 += 8) {
          float u[8];
#pragma unroll
          for (int j = 0; j < 8; ++j) u[j] = pp[min(s0 + j, fold.splits - 1) * stride];
#pragma unroll
          for (int j = 0; j < 8; ++j)
            if (s0 + j < fold.splits) v += u[j];
        }
        qkv_s[c] = v * fold.scale;
      }
    }
    __syncthreads();  // pts, qkv_s

    // Rotary pairs (i, i + 32) of the q heads and of k; k and v go to the
    // cache at position p and, as stored, to new_kv for this row's own key.
    for (int i = threadIdx.x; i < (G + 2) * 32; i += NT) {
      const int hh = i >> 5, e = i & 31;
      float y0 = qkv_s[hh * 64 + e], y1 = qkv_s[hh * 64 + e + 32];
      if (hh <= G) {
        const float2 c2 = i == (int)threadIdx.x ? cs : fold.rope[(size_t)p * 32 + e];
        const float r0 = y0 * c2.x - y1 * c2.y, r1 = y1 * c2.x + y0 * c2.y;
        y0 = r0;
        y1 = r1;
      }
      if (hh < G) {
        qkv_s[hh * 64 + e] = y0;
        qkv_s[hh * 64 + e + 32] = y1;
      } else {
        const int kind = hh - G;
        const TKV a = (TKV)y0, b = (TKV)y1;
        new_kv[kind][e] = a;
        new_kv[kind][e + 32] = b;
        TKV* dst = fold.kv + L.head_tile(layer, new_page, kind, g) + (p % kPage) * 64;
        dst[e] = a;
        dst[e + 32] = b;
      }
    }
    __syncthreads();
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
      for (int e = 0; e < 16; ++e) qv[h][e] = qkv_s[h * 64 + quarter * 16 + e] * qscale;
  }

  // Softmax state per head: running max m (log2 units), sum and output.
  float m[G], lsum[G], o[G][16];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    lsum[h] = 0.f;
#pragma unroll
    for (int e = 0; e < 16; ++e) o[h][e] = 0.f;
  }
  // Only the row's last page holds keys past the stream's length (stale
  // slots, possibly non-finite bit patterns: their V becomes 0, since
  // 0 * NaN would be NaN, and their score -inf) and, with the QKV fold, the
  // row's own key and value, which come from LDS (the cache write above may
  // not be visible to this wave's loads yet).  Returns the lane's validity.
  auto patch_last = [&](KvPage<TKV>& P, int pg) {
    const bool valid = pg * kPage + key < t;
    if (folded && pg * kPage + key == p) {
      const u32x4* nk = reinterpret_cast<const u32x4*>(&new_kv[0][quarter * 16]);
      const u32x4* nv = reinterpret_cast<const u32x4*>(&new_kv[1][quarter * 16]);
#pragma unroll
      for (int c = 0; c < (int)sizeof(TKV); ++c) {
        P.k[c] = nk[c];
        P.v[c] = nv[c];
      }
    }
#pragma unroll
    for (int c = 0; c < (int)sizeof(TKV); ++c) P.v[c] = valid ? P.v[c] : u32x4{0u, 0u, 0u, 0u};
    return valid;
  };
  // Scores of the G heads for this lane's key (all four lanes of a key get
  // the full dot product).
  auto scores = [&](const KvPage<TKV>& P, float* sc) {
    float kf[16];
#pragma unroll
    for (int c = 0; c < (int)sizeof(TKV); ++c) widen16(P.k[c], kf + c * Vec16<TKV>::n, TKV());
#pragma unroll
    for (int h = 0; h < G; ++h) {
      float a0 = 0.f, a1 = 0.f;
#pragma unroll
      for (int e = 0; e < 16; e += 2) {
        a0 = fmaf(qv[h][e], kf[e], a0);
        a1 = fmaf(qv[h][e + 1], kf[e + 1], a1);
      }
      float x = a0 + a1;
      x += dpp<0xB1>(x);  // the 4 lanes of a key hold quarters of its dot product
      x += dpp<0x4E>(x);
      sc[h] = x;
    }
  };
  // Weights exp2(score - m) into the sums; lsum runs on all four lanes of a
  // key, so its total is taken a quarter below.
  auto accumulate = [&](const KvPage<TKV>& P, const float* sc) {
    float vf[16];
#pragma unroll
    for (int c = 0; c < (int)sizeof(TKV); ++c) widen16(P.v[c], vf + c * Vec16<TKV>::n, TKV());
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float pk = __builtin_amdgcn_exp2f(sc[h] - m[h]);
      lsum[h] += pk;
#pragma unroll
      for (int e = 0; e < 16; ++e) o[h][e] = fmaf(pk, vf[e], o[h][e]);
    }
  };
  // The wave's first PU pages are in registers together: scores of all of
  // them first, one max per head over the wave, then the weighted sums (no
  // rescaling).  Pages past the row's end (re-read copies) score -inf.
  {
    float sc[PU][G];
#pragma unroll
    for (int k = 0; k < PU; ++k) {
      const int pg = wave + NW * k;
      bool valid = pg < npg;
      if (pg == npg - 1) valid = patch_last(P[k], pg);
      scores(P[k], sc[k]);
#pragma unroll
      for (int h = 0; h < G; ++h) sc[k][h] = valid ? sc[k][h] : -INFINITY;
    }
#pragma unroll
    for (int h = 0; h < G; ++h) {
      float mx = sc[0][h];
#pragma unroll
      for (int k = 1; k < PU; ++k) mx = fmaxf(mx, sc[k][h]);
      m[h] = wave_max_u(mx);  // -inf for a wave without pages
    }
#pragma unroll
    for (int k = 0; k < PU; ++k)
      if (wave + NW * k < npg) accumulate(P[k], sc[k]);
  }
  // Longer rows: later pages one at a time with an online update (the max
  // is finite here: the wave took PU pages above); the next two pages' K/V
  // are in flight while one is taken; loads past the end re-read the row's
  // last page.
  auto take = [&](KvPage<TKV>& P, int pg) {
    bool valid = true;
    if (pg == npg - 1) valid = patch_last(P, pg);
    float sc[G];
    scores(P, sc);
#pragma unroll
    for (int h = 0; h < G; ++h) {
      sc[h] = valid ? sc[h] : -INFINITY;
      const float mn = fmaxf(m[h], wave_max_u(sc[h]));
      const float alpha = __builtin_amdgcn_exp2f(m[h] - mn);
      lsum[h] *= alpha;
#pragma unroll
      for (int e = 0; e < 16; ++e) o[h][e] *= alpha;
      m[h] = mn;
    }
    accumulate(P, sc);
  };
  if (long_row) __syncthreads();  // pts (the folded path's barriers came earlier)
  if (wave + NW * PU < npg) {
    KvPage<TKV>&A = P[0], &B = P[1], &C = P[2];
    const int pg0 = wave + NW * PU;
    kv_page_load(A, kv, L, layer, page_of(pg0), g, key, quarter);
    kv_page_load(B, kv, L, layer, page_of(min(pg0 + NW, npg - 1)), g, key, quarter);
    for (int pg = pg0; pg < npg; pg += 3 * NW) {
      kv_page_load(C, kv, L, layer, page_of(min(pg + 2 * NW, npg - 1)), g, key, quarter);
      take(A, pg);
      if (pg + NW >= npg) break;
      kv_page_load(A, kv, L, layer, page_of(min(pg + 3 * NW, npg - 1)), g, key, quarter);
      take(B, pg + NW);
      if (pg + 2 * NW >= npg) break;
      kv_page_load(B, kv, L, layer, page_of(min(pg + 4 * NW, npg - 1)), g, key, quarter);
      take(C, pg + 2 * NW);
    }
  }
  // Per head: reduce over the keys of each row of 16 lanes (lanes sharing
  // `quarter`; row_ror by 4 and 8 keeps lane bits 0-1), leave row partials in
  // the wave's slots; waves without pages leave m = -inf, l = 0, o = 0.
#pragma unroll
  for (int h = 0; h < G; ++h) {
    const float ls = wave_sum_u(lsum[h]) * 0.25f;
    float* sw = st + ((wave * G + h) * 4 + (lane >> 4)) * SLOT;
    if ((lane & 15) == 0) {
      sw[0] = m[h];
      sw[1] = ls;
    }
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      float v = o[h][e];
      v += dpp<0x124>(v);
      v += dpp<0x128>(v);
      if ((lane & 15) < 4) sw[2 + quarter * 16 + e] = v;
    }
  }
  __syncthreads();
  if (wave < G) {
    const int h = wave, j = g * G + h;
    float Mg[NW], Lg[NW], Og[NW];
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const float* sv = st + (w * G + h) * 4 * SLOT;
      Mg[w] = sv[0];
      Lg[w] = sv[1];
      Og[w] = (sv[2 + lane] + sv[SLOT + 2 + lane]) + (sv[2 * SLOT + 2 + lane] + sv[3 * SLOT + 2 + lane]);
    }
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < NW; ++w) M = fmaxf(M, Mg[w]);
    float Ls = 0.f, O = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const float f = Mg[w] > -INFINITY ? exp2f(Mg[w] - M) : 0.f;
      Ls = fmaf(Lg[w], f, Ls);
      O = fmaf(Og[w], f, O);
    }
    const float out = O / Ls;
    o32[((size_t)r * hq + j) * 64 + lane] = out;
    if (oM) oM[((size_t)r * hq + j) * 64 + lane] = (TM)out;
  }
}

// ---------------------------------------------------------------- rows RMSNorm

// h[r] = x[r] * rsqrt(mean(x[r]^2) + eps) * gain, stored as the MFMA operand type.
template <typename TM>
__global__ __launch_bounds__(256) void k_rmsnorm_rows(const float* __restrict__ x, const float* __restrict__ gain,
                                                      float eps, int d, TM* __restrict__ h) {
  __shared__ float red[4];
  const float* xr = x + (size_t)blockIdx.x * d;
  float ss = 0.f;
  for (int i = threadIdx.x; i < d; i += 256) ss += xr[i] * xr[i];
  const float inv = rsqrtf(block_sum256(ss, red) / (float)d + eps);
  for (int i = threadIdx.x; i < d; i += 256) h[(size_t)blockIdx.x * d + i] = (TM)(xr[i] * inv * gain[i]);
}

// ---------------------------------------------------------------- launchers

template <typename TW, typename TKV, typename TM>
void DecodeKernels<TW, TKV, TM>::prep_embed(hipStream_t st, int n_rows, int prefill_stream, const int* feed,
                                            int* row_stream, int* row_pos, const int* pos, const int* pending,
                                            unsigned long long* slot, const TW* embed, float* x, int d) {
  k_prep_embed<TW><<<n_rows, 256, 0, st>>>(prefill_stream, feed, row_stream, row_pos, pos, pending, slot, embed, x,
                                           d);
}

template <typename TW, typename TKV, typename TM>
void DecodeKernels<TW, TKV, TM>::qkv_gemv(hipStream_t st, const TW* W, const float* x, const float* gain, float eps,
                                          int d, int hq, int hkv, const int* row_stream, const int* row_pos,
                                          const float2* rope, float* q, TKV* kv, KvLayout L, int layer,
                                          const int* page_table) {
  const int blocks = (hq + 2 * hkv) * 8;  // 32 pairs per head, 4 pairs per block
  k_qkv_gemv<TW, TKV><<<blocks, 256, d * sizeof(float), st>>>(W, x, gain, eps, d, hq, hkv, row_stream, row_pos,
                                                               rope, q, kv, L, layer, page_table);
}

template <typename TW, typename TKV, typename TM>
void DecodeKernels<TW, TKV, TM>::resid_gemv(hipStream_t st, const TW* W, const float* in, int K, int N,
                                            float* xres) {
  k_resid_gemv<TW><<<(N + 7) / 8, 256, K * sizeof(float), st>>>(W, in, K, N, xres);
}

template <typename TW, typename TKV, typename TM>
void DecodeKernels<TW, TKV, TM>::gateup_gemv(hipStream_t st, const TW* W, const float* x, const float* gain,
                                             float eps, int d, int F, float* m) {
  k_gateup_gemv<TW><<<(F + 3) / 4, 256, d * sizeof(float), st>>>(W, x, gain, eps, d, F, m);
}

template <typename TW, typename TKV, typename TM>
void DecodeKernels<TW, TKV, TM>::head_gemv(hipStream_t st, const TW* W, const float* x, const float* gain, float eps,
                                           int d, int V, int row, const int* row_stream, float* logits,
                                           unsigned long long* slot) {
  if (d / Vec16<TW>::n <= 256)
    k_head_stream<TW><<<2 * device_cus(), 256, d * sizeof(float), st>>>(W, x, gain, eps, d, V, row, row_stream,
                                                                        logits, slot);
  else
    k_head_gemv<TW><<<(V + 7) / 8, 256, d * sizeof(float), st>>>(W, x, gain, eps, d, V, row, row_stream, logits,
                                                                  slot);
}

template <typename TW, typename TKV, typename TM>
void DecodeKernels<TW, TKV, TM>::attention(hipStream_t st, int n_rows, const float* q, const TKV* kv, KvLayout L,
                                           int layer, const int* page_table, const int* row_stream,
                                           const int* row_pos, int hq, int hkv, int s_max, float* part, float* o32,
                                           TM* oM) {
  dim3 grid(s_max, hkv, n_rows);
  k_attn<TKV, TM><<<grid, 256, 0, st>>>(q, kv, L, layer, page_table, row_stream, row_pos, hq, hkv, s_max, part, o32,
                                        oM);
  if (s_max > 1)
    k_attn_combine<TM><<<dim3(hq, n_rows), 64, 0, st>>>(part, row_pos, hq, s_max, o32, oM);
}

template <typename TW, typename TKV, typename TM>
void DecodeKernels<TW, TKV, TM>::attention_rows(hipStream_t st, int n_rows, const float* q, const TKV* kv,
                                                KvLayout L, int layer, const int* page_table, const int* row_stream,
                                                const int* row_pos, int hq, int hkv, float* o32, TM* oM,
                                                const QkvFold<TKV>& fold) {
  const dim3 grid(hkv, n_rows);
  switch (hq / hkv) {
    case 1: k_attn_rows<TKV, TM, 1><<<grid, 512, 0, st>>>(q, kv, L, layer, page_table, row_stream, row_pos, hq, o32, oM, fold); break;
    case 2: k_attn_rows<TKV, TM, 2><<<grid, 512, 0, st>>>(q, kv, L, layer, page_table, row_stream, row_pos, hq, o32, oM, fold); break;
    case 4: k_attn_rows<TKV, TM, 4><<<grid, 512, 0, st>>>(q, kv, L, layer, page_table, row_stream, row_pos, hq, o32, oM, fold); break;
    default: k_attn_rows<TKV, TM, 8><<<grid, 512, 0, st>>>(q, kv, L, layer, page_table, row_stream, row_pos, hq, o32, oM, fold); break;
  }
}

template <typename TW, typename TKV, typename TM>
void DecodeKernels<TW, TKV, TM>::rmsnorm_rows(hipStream_t st, int n_rows, const float* x, const float* gain,
                                              float eps, int d, TM* h) {
  k_rmsnorm_rows<TM><<<n_rows, 256, 0, st>>>(x, gain, eps, d, h);
}

// Small host integer arrays (page ids, stream lists, teacher-forced tokens)
// reach the device as kernel arguments, not as copies from pageable memory.
struct IntArgs {
  int n;
  int v[kPutInts];
};
__global__ void k_put_ints(int* __restrict__ dst, IntArgs a) {
  if ((int)threadIdx.x < a.n) dst[threadIdx.x] = a.v[threadIdx.x];
}

void put_ints(hipStream_t st, int* dst, const int* src, int n) {
  for (int o = 0; o < n; o += kPutInts) {
    IntArgs a;
    a.n = n - o < kPutInts ? n - o : kPutInts;
    for (int i = 0; i < a.n; ++i) a.v[i] = src[o + i];
    k_put_ints<<<1, 64, 0, st>>>(dst + o, a);
  }
}

void finalize(hipStream_t st, int r0, int n, const int* row_stream, const int* row_pos, unsigned long long* slot,
              int* pending, int* hist, int* pos, int max_ctx) {
  k_finalize<<<1, 64, 0, st>>>(r0, n, row_stream, row_pos, slot, pending, hist, pos, max_ctx);
}

template struct DecodeKernels<float, float, float>;
template struct DecodeKernels<__bf16, _Float16, _Float16>;

}  // namespace hh
