// Host-callable launchers of the gfx950 kernels (internal to the library).
// Template parameters: TW = weight storage type of the weight-streaming GEMVs
// (float or __bf16), TKV = KV-cache element type (float or _Float16), TM =
// MFMA operand type of the dense GEMM path (float or _Float16).
#pragma once

#include "hh_device.h"

namespace hh {

// Lockstep decode rows (one row per stream) whose QKV product was left as
// K-split partials: the attention kernel sums them, scales, rotates q and k,
// appends k and v to the cache and attends with them.  part == nullptr: q is
// already rotated in q[] and the cache holds the row's key and value.
template <typename TKV>
struct QkvFold {
  const float* part = nullptr;  // [splits][rows][ncols] fp32, ncols = (hq + 2 hkv) * 64
  int splits = 0, ncols = 0;
  float scale = 1.f;            // factor of the summed products (weight scale)
  const float2* rope = nullptr; // (cos, sin) at [position][pair]
  TKV* kv = nullptr;            // the cache (written at each row's position)
};

template <typename TW, typename TKV, typename TM>
struct DecodeKernels {
  static void prep_embed(hipStream_t st, int n_rows, int prefill_stream, const int* feed, int* row_stream,
                         int* row_pos, const int* pos, const int* pending, unsigned long long* slot, const TW* embed,
                         float* x, int d);
  static void qkv_gemv(hipStream_t st, const TW* W, const float* x, const float* gain, float eps, int d, int hq,
                       int hkv, const int* row_stream, const int* row_pos, const float2* rope, float* q, TKV* kv,
                       KvLayout L, int layer, const int* page_table);
  static void resid_gemv(hipStream_t st, const TW* W, const float* in, int K, int N, float* xres);
  static void gateup_gemv(hipStream_t st, const TW* W, const float* x, const float* gain, float eps, int d, int F,
                          float* m);
  static void head_gemv(hipStream_t st, const TW* W, const float* x, const float* gain, float eps, int d, int V,
                        int row, const int* row_stream, float* logits, unsigned long long* slot);
  static void attention(hipStream_t st, int n_rows, const float* q, const TKV* kv, KvLayout L, int layer,
                        const int* page_table, const int* row_stream, const int* row_pos, int hq, int hkv, int s_max,
                        float* part, float* o32, TM* oM);
  static void attention_rows(hipStream_t st, int n_rows, const float* q, const TKV* kv, KvLayout L, int layer,
                             const int* page_table, const int* row_stream, const int* row_pos, int hq, int hkv,
                             float* o32, TM* oM, const QkvFold<TKV>& fold = QkvFold<TKV>());
  static void rmsnorm_rows(hipStream_t st, int n_rows, const float* x, const float* gain, float eps, int d, TM* h);
};

void finalize(hipStream_t st, int r0, int n, const int* row_stream, const int* row_pos, unsigned long long* slot,
              int* pending, int* hist, int* pos, int max_ctx);

// dst[0 .. n) = src[0 .. n) (host ints) through kernel arguments, kPutInts per launch.
constexpr int kPutInts = 62;
void put_ints(hipStream_t st, int* dst, const int* src, int n);

// fp32 scratch (in the context's arena) for split-K partial tiles of the
// MFMA GEMM; splits are reduced until the partials fit.
struct GemmWorkspace {
  float* ptr;
  size_t bytes;
};

// RMSNorm split across a residual product and the product that reads its
// output, for the <= 32-row GEMMs: a row's norm factor is one scalar, so it
// can scale the consumer's output rows instead of its input.
//  * producer (a residual product whose K is split): the last split of each
//    64-column block to finish adds the split sum (in split order) into x,
//    writes y = x * gain (elementwise) as fp16 and the block's per-row sums
//    of squares to ss_out[row * (N / 64) + block]; cnt holds one counter per
//    column block (ncnt of them), zero before and after every launch;
//  * consumer: row r of A is such a y (nss <= 32 block sums per row, a
//    multiple of 4); the product's row r is scaled by rsqrt(sum over blocks
//    of ss_in[r * nss + j] / n + eps) before its split partials or
//    epilogue.
struct RowNorm {
  const float* ss_in = nullptr;
  int nss = 0;
  float n = 1.f, eps = 0.f;
  int* cnt = nullptr;
  int ncnt = 0;
  const float* gain = nullptr;
  _Float16* y = nullptr;
  float* ss_out = nullptr;
};

template <typename TM, typename TKV>
struct GemmKernels {
  // Wt (optional): the same matrix as 16 x 32 operand tiles (tile16), used
  // for M <= 32 rows.
  static void qkv(hipStream_t st, GemmWorkspace ws, const TM* A, int M, const TM* W, int d, int hq, int hkv, float scale,
                  const int* row_stream, const int* row_pos, const float2* rope, float* q, TM* qM, TKV* kv,
                  KvLayout L, int layer, const int* page_table, const TM* Wt = nullptr);
  // The same product for lockstep decode rows with the split-K reduction
  // left to the attention kernel: returns the K splits (partials in ws.ptr
  // when > 1, nothing written yet); 1: the epilogue ran as in qkv().
  static int qkv_deferred(hipStream_t st, GemmWorkspace ws, const TM* A, int M, const TM* W, int d, int hq, int hkv,
                          float scale, const int* row_stream, const int* row_pos, const float2* rope, float* q, TKV* kv,
                          KvLayout L, int layer, const int* page_table, const TM* Wt = nullptr,
                          const RowNorm& rn = RowNorm());
  // x += A W^T * scale; with gain, then h = rmsnorm(x) * gain (fused into the
  // split-K reduction when K is split).  Requires norm_fusable(N) with gain.
  // With ss and cnt (RowNorm's producer buffers, ncnt counters) the 32-row
  // GEMM may instead leave h = x * gain and the row sums of squares in ss:
  // returns true then, and the product reading h takes
  // RowNorm{ss, N / 64, N, eps}.
  static bool resid(hipStream_t st, GemmWorkspace ws, const TM* A, int M, const TM* W, int K, int N, float scale, float* x,
                    const float* gain = nullptr, float eps = 0.f, TM* h = nullptr, const TM* Wt = nullptr,
                    float* ss = nullptr, int* cnt = nullptr, int ncnt = 0);
  static bool norm_fusable(int N);
  // h = rmsnorm(x) * gain, one row per workgroup (norm_fusable(N)).
  static void rmsnorm(hipStream_t st, int M, float* x, int N, const float* gain, float eps, TM* h);
  static void gateup(hipStream_t st, GemmWorkspace ws, const TM* A, int M, const TM* W, int d, int F, float scale, TM* m,
                     const TM* Wt = nullptr, const RowNorm& rn = RowNorm());
  static void logits(hipStream_t st, GemmWorkspace ws, const TM* A, int M, const TM* W, int d, int V, float scale, float* logits,
                     unsigned long long* slot, const int* row_stream, const TM* Wt = nullptr,
                     const RowNorm& rn = RowNorm());
};

// ---- causal flash attention for prefill rows of one stream (k_attn_prefill.hip)
// layer_kv_elems: K and V elements of one layer's cache (the kernel's
// offsets are 32-bit).
bool flash_prefill_supported(int G, int max_context, size_t layer_kv_elems);
void flash_prefill(hipStream_t st, const _Float16* qM, const _Float16* kv, KvLayout L, int layer,
                   const int* page_table, int s, int p0, int n_rows, int hq, int hkv, _Float16* oM);

// ---- batch-1 decode step as one persistent kernel (k_step.hip)
constexpr int kStepThreads = 512;     // threads per workgroup (8 waves)
constexpr int kStepResFloats = 1024;  // LDS row results per workgroup and phase
constexpr int kStepMaxLayers = 63;    // layers the persistent kernel supports
constexpr int kStepRingSlots = 12;    // 8 KiB slots of the per-workgroup LDS weight ring
constexpr int kStepLoadDepth = 2;    // ring slots each streaming wave keeps in flight (1 .. 7)

template <typename TW>
struct LayerPtrs {
  const TW* wqkv;   // [(Hq + 2 Hkv) * 64, d]
  const TW* wo;     // [d, Hq * 64]
  const TW* wgu;    // [2F, d] = [Wgate; Wup]
  const TW* wdown;  // [d, F]
  const TW* wdownT; // [F, d] = Wdown^T (the batch-1 decode kernel's split-K down projection)
  const float* attn_norm;
  const float* mlp_norm;
};

// The batch-1 decode kernel streams the fp16 (x 2^s) copies of bf16 models'
// matrices (one v_fma_mix per weight, no widening); the token embedding it
// looks up stays in the model's own type.
template <typename TW> struct StepEmbed { using type = TW; };
template <> struct StepEmbed<_Float16> { using type = __bf16; };
// Element tag of the 4-bit rows (HH_WF_Q4G32, d_model 2048: 1024 bytes of
// codes and 64 bf16 scales per row) the batch-1 kernel streams for 4-bit
// models; their embedding table stays bf16.
struct Q4Row {};
template <> struct StepEmbed<Q4Row> { using type = __bf16; };

template <typename TW, typename TKV>
struct StepParams {
  int d, F, hq, hkv, V, n_layers, max_ctx, stream;
  int ring_slots;              // LDS ring slots per workgroup (<= 16)
  int load_depth;              // ring slots each streaming wave keeps in flight (1 .. 7)
  int quiet;                   // 1: streaming pauses while compute waves wait for other workgroups
  int poll_delay;              // ticks (10 ns) to wait before a phase's first exchange poll
  unsigned long long wait_ticks;  // ticks (10 ns) after which a wait gives up (0: 1 s)
  int fail_wait;               // tests of the failure path: the final argmax wait expects an epoch never published
  float eps;
  unsigned epoch;              // base epoch of this step (distinct for every step)
  const LayerPtrs<TW>* layer;  // device array [n_layers]
  float wscale_inv;            // 1 / the power-of-two scale of the streamed matrices
  const typename StepEmbed<TW>::type* embed;
  const TW* head;
  const float* final_norm;
  const float2* rope;
  TKV* kvc;
  KvLayout kv;
  const int* page_table;
  int* pos;
  int* pending;
  int* hist;
  const int* feed;  // nullptr: consume the pending token
  float* logits;    // nullptr or [V]
  // Epoch-tagged exchange words (fp32 bits | epoch << 32) between workgroups.
  unsigned long long* ll_xa;    // [d] x after the O projection
  unsigned long long* ll_xb;    // [d] x after the down projection
  unsigned long long* ll_q;     // [Hq * 64] rotated queries
  unsigned long long* ll_kn;    // [Hkv * 64] rotated key of the current position
  unsigned long long* ll_vn;    // [Hkv * 64] value of the current position
  unsigned long long* ll_part;  // [Hq][nwg / Hkv][66] attention split partials
  unsigned long long* ll_o;     // [Hq * 64] attention output
  unsigned long long* ll_dp;    // [nwg][d] each workgroup's partial down projection
  unsigned long long* ll_keys;  // [2 * nwg] per-workgroup argmax keys
  int* err;                     // set to 1 if a wait timed out
  unsigned long long* trace;    // nullptr, or [nwg][n_layers + 1][32] phase timestamps
};

template <typename TW, typename TKV>
struct StepKernel {
  static bool supports(int d, int F, int hq, int hkv, int V, int n_layers, int nwg);
  static hipError_t launch(const StepParams<TW, TKV>& P, int nwg, hipStream_t st);
  static int max_blocks_per_cu(int d, int F, int hq, int hkv);
  static size_t lds_bytes(int d, int F, int hq, int hkv, int ring_slots);
  static int xc_floats(int d, int F, int hq, int hkv);
};

// Load-time weight preparation.
void widen_bf16(hipStream_t st, const __bf16* src, float* dst, size_t n);
void absmax_bf16(hipStream_t st, const __bf16* src, size_t n, unsigned int* out_bits);
void bf16_to_f16_scaled(hipStream_t st, const __bf16* src, _Float16* dst, size_t n, float scale);
// 4-bit group format of rows x K bf16 values (K % 32 == 0): stored rows into
// q4 (K / 2 + K / 16 bytes each) and/or q * s * scale as fp16 into deq
// (either may be null; deq may equal src).
void q4g32(hipStream_t st, const __bf16* src, size_t rows, int K, unsigned char* q4, _Float16* deq, float scale);
// 16 x 32 operand tiles of a [rows][K] fp16 matrix taken as logical_rows rows
// (see k_tile16); dst holds ceil(logical_rows / 16) * 16 * K elements.
void tile16(hipStream_t st, const _Float16* src, _Float16* dst, int rows, int K, int logical_rows, int interleave_f);
// dst = src^T for a row-major rows x cols matrix.
template <typename T>
void transpose(hipStream_t st, const T* src, T* dst, int rows, int cols);

}  // namespace hh
