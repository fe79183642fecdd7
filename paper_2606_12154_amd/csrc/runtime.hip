// Host runtime behind the C ABI in include/hh.h: arena carve-up, weight
// upload and repack, per-stream KV page allocation, and the enqueue order of
// one prefill pass / one decode step (decode steps are captured once per
// shape into a HIP graph and replayed; positions live in device memory, so a
// graph does not depend on where in the sequence a stream is).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <tuple>
#include <type_traits>
#include <vector>

#include "hh.h"
#include "hh_kernels.h"

using namespace hh;

namespace {

constexpr int kSplitMax = 64;   // attention splits per (row, kv head) in decode
constexpr int kLogitRows = 64;  // rows of the logits staging buffer (prefill ALL)
constexpr int kMaxStepWG = 1024; // upper bound on persistent decode-step workgroups

size_t al(size_t x) { return (x + 255) & ~size_t(255); }

struct Layout {
  // element sizes
  size_t ew, ekv, em;
  int nqkv, max_pages, n_pages, rows_cap, logit_rows;
  // byte offsets into the arena
  size_t embed, lm_head, embedM, lm_headM;
  std::vector<size_t> wqkv, wo, wgu, wdown, wdownT, wqkvM, woM, wguM, wdownM, attn_norm, mlp_norm;
  // 16 x 32 operand tiles of the fp16 copies for <= 32-row GEMMs (multi-stream
  // contexts of bf16 models only; empty otherwise).
  std::vector<size_t> wqkvT16, woT16, wguT16, wdownT16;
  size_t lm_headT16;
  // Stored 4-bit rows (HH_WF_Q4G32 only; empty otherwise): [Wq; Wk; Wv],
  // Wo, [Wgate; Wup], Wdown^T and the LM head, K / 2 + K / 16 bytes per row.
  std::vector<size_t> wqkvQ, woQ, wguQ, wdownTQ;
  size_t lm_headQ;
  size_t final_norm, rope, kv, page_table, pos, pending, slot, hist, ll, ll_words, layer_tab, trace;
  size_t row_stream, row_pos, feed, x, h, q, qM, o32, oM, m32, mM, part, logits, gemm_ws, gemm_ws_bytes, scratch_u32;
  // RowNorm buffers of the lockstep decode rows: column-block counters (zero
  // between launches; in the zero-initialised range) and row sums of squares.
  size_t nrm_cnt, nrm_ss;
  int nrm_ncnt;
  size_t total;
};

bool config_supported(const hh_config& c, std::string& why) {
  if (c.n_layers < 0 || c.d_model <= 0 || c.n_heads <= 0 || c.n_kv_heads <= 0 || c.ffn_dim <= 0 || c.vocab < 2 ||
      c.max_streams < 1 || c.max_context < 1 || c.max_prefill < 0) {
    why = "non-positive dimension in config";
    return false;
  }
  if (c.head_dim != 64) { why = "head_dim must be 64"; return false; }
  if (c.page_size != kPage) { why = "page_size must be 16"; return false; }
  const int grp = c.n_heads / c.n_kv_heads;
  if (c.n_heads % c.n_kv_heads != 0 || (grp != 1 && grp != 2 && grp != 4 && grp != 8)) {
    why = "n_heads / n_kv_heads must be 1, 2, 4 or 8";
    return false;
  }
  if (c.max_context > 131072) { why = "max_context must be at most 131072"; return false; }
  if (c.d_model % 64 != 0) { why = "d_model must be a multiple of 64"; return false; }
  if (c.ffn_dim % 8 != 0) { why = "ffn_dim must be a multiple of 8"; return false; }
  if (c.d_model > 16384 || c.ffn_dim > 65536 || c.n_heads * 64 > 16384) { why = "dimension too large"; return false; }
  if (c.dtype != HH_F32 && c.dtype != HH_BF16) { why = "dtype must be HH_F32 or HH_BF16"; return false; }
  if (!(c.rms_eps >= 0.f) || !(c.rope_theta > 0.f)) { why = "bad rms_eps / rope_theta"; return false; }
  if (c.weight_format != HH_WF_DTYPE && c.weight_format != HH_WF_Q4G32) {
    why = "weight_format must be HH_WF_DTYPE or HH_WF_Q4G32";
    return false;
  }
  if (c.weight_format == HH_WF_Q4G32 && c.dtype != HH_BF16) {
    why = "HH_WF_Q4G32 needs bf16 weights";
    return false;
  }
  return true;
}

// Where the decode-step kernel's exchange words live: the context's arena
// (hh_decode_step) or the fixed device array (hh_decode_step_noalloc).
// Layout for up to `cap` workgroups: xa, xb [d], q [Hq*64], kn, vn
// [Hkv*64], attention partials [Hq][cap][66], o [Hq*64], down partials
// [cap][d], argmax keys [2*cap], then the error word.
struct StepWords {
  unsigned long long* base;
  size_t cap;
  unsigned epoch;  // first epoch of this step (a multiple of 512, never 0)
};

size_t step_words(const hh_config& g, size_t cap) {
  const size_t d = g.d_model, hq = g.n_heads, hkv = g.n_kv_heads;
  return 2 * d + 2 * hq * 64 + 2 * hkv * 64 + hq * cap * 66 + cap * d + 2 * cap + 8;
}

int* step_err_word(const hh_config& g, const StepWords& w) {
  return reinterpret_cast<int*>(w.base + step_words(g, w.cap) - 8);
}

Layout make_layout(const hh_config& c) {
  Layout L{};
  const bool bf = c.dtype == HH_BF16;
  L.ew = bf ? 2 : 4;
  L.ekv = bf ? 2 : 4;
  L.em = bf ? 2 : 0;  // fp32 models use their weights directly as MFMA operands
  const size_t d = c.d_model, F = c.ffn_dim, V = c.vocab, hq = c.n_heads;
  L.nqkv = (c.n_heads + 2 * c.n_kv_heads) * 64;
  L.max_pages = (c.max_context + kPage - 1) / kPage;
  L.n_pages = c.max_streams * L.max_pages;
  const int mp = c.max_prefill > 0 ? std::min(c.max_prefill, c.max_context) : c.max_context;
  L.rows_cap = std::max(c.max_streams, mp);
  L.logit_rows = std::max(c.max_streams, kLogitRows);
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t o = off; off += al(bytes); return o; };
  L.embed = take(V * d * L.ew);
  L.lm_head = c.tied_embeddings ? L.embed : take(V * d * L.ew);
  for (int l = 0; l < c.n_layers; ++l) {
    L.wqkv.push_back(take((size_t)L.nqkv * d * L.ew));
    L.wo.push_back(take(d * hq * 64 * L.ew));
    L.wgu.push_back(take(2 * F * d * L.ew));
    L.wdown.push_back(take(d * F * L.ew));
    L.wdownT.push_back(take(d * F * L.ew));
  }
  if (bf) {
    L.embedM = take(V * d * L.em);
    L.lm_headM = c.tied_embeddings ? L.embedM : take(V * d * L.em);
    for (int l = 0; l < c.n_layers; ++l) {
      L.wqkvM.push_back(take((size_t)L.nqkv * d * L.em));
      L.woM.push_back(take(d * hq * 64 * L.em));
      L.wguM.push_back(take(2 * F * d * L.em));
      L.wdownM.push_back(take(d * F * L.em));
    }
    if (c.max_streams > 1) {
      auto tiles = [&](size_t logical_rows, size_t K) { return take((logical_rows + 15) / 16 * 16 * K * 2); };
      L.lm_headT16 = tiles(V, d);
      for (int l = 0; l < c.n_layers; ++l) {
        L.wqkvT16.push_back(tiles(L.nqkv, d));
        L.woT16.push_back(tiles(d, hq * 64));
        L.wguT16.push_back(tiles((F + 31) / 32 * 64, d));
        L.wdownT16.push_back(tiles(d, F));
      }
    }
  } else {
    L.embedM = L.embed;
    L.lm_headM = L.lm_head;
    L.wqkvM = L.wqkv;
    L.woM = L.wo;
    L.wguM = L.wgu;
    L.wdownM = L.wdown;
  }
  if (c.weight_format == HH_WF_Q4G32) {
    auto q4 = [&](size_t rows, size_t K) { return take(rows * (K / 2 + K / 16)); };
    L.lm_headQ = q4(V, d);
    for (int l = 0; l < c.n_layers; ++l) {
      L.wqkvQ.push_back(q4(L.nqkv, d));
      L.woQ.push_back(q4(d, hq * 64));
      L.wguQ.push_back(q4(2 * F, d));
      L.wdownTQ.push_back(q4(F, d));
    }
  }
  for (int l = 0; l < c.n_layers; ++l) {
    L.attn_norm.push_back(take(d * 4));
    L.mlp_norm.push_back(take(d * 4));
  }
  L.final_norm = take(d * 4);
  L.rope = take((size_t)c.max_context * 32 * sizeof(float2));
  L.kv = take((size_t)c.n_layers * L.n_pages * 2 * c.n_kv_heads * kPage * 64 * L.ekv);
  L.page_table = take((size_t)c.max_streams * L.max_pages * 4);
  L.pos = take((size_t)c.max_streams * 4);
  L.pending = take((size_t)c.max_streams * 4);
  L.slot = take((size_t)c.max_streams * 8);
  L.hist = take((size_t)c.max_streams * c.max_context * 4);
  // Epoch-tagged exchange words of the persistent decode kernel (see k_step.hip):
  // xa, xb [d], q [Hq*64], kn, vn [Hkv*64], partials [Hq][kMaxStepWG][66],
  // o [Hq*64], down partials [kMaxStepWG][d], keys [2*kMaxStepWG], then the
  // error flag.
  L.ll_words = step_words(c, kMaxStepWG);
  L.ll = take(L.ll_words * 8);
  L.layer_tab = take((size_t)c.n_layers * sizeof(LayerPtrs<float>));
  L.trace = take((size_t)kMaxStepWG * (c.n_layers + 1) * 32 * 8);  // optional phase timestamps
  // One counter per 64-column block of a residual product.
  L.nrm_ncnt = (int)(d / 64 + 1);
  L.nrm_cnt = take((size_t)L.nrm_ncnt * 4);
  const size_t R = L.rows_cap, tm = bf ? 2 : 4;
  L.row_stream = take(R * 4);
  L.row_pos = take(R * 4);
  L.feed = take(R * 4);
  L.x = take(R * d * 4);
  L.h = take(R * std::max(d, (size_t)hq * 64) * tm);
  L.q = take(R * hq * 64 * 4);
  L.qM = take(R * hq * 64 * tm);
  L.o32 = take(R * hq * 64 * 4);
  L.oM = take(R * hq * 64 * tm);
  L.m32 = take(F * 4);
  L.mM = take(R * F * tm);
  L.part = take((size_t)c.max_streams * hq * kSplitMax * 66 * 4);
  L.logits = take((size_t)L.logit_rows * V * 4);
  // Split-K partials: up to 4 splits of the widest non-head product at R rows, at most 256 MiB.
  L.gemm_ws_bytes = std::min<size_t>((size_t)4 * R * std::max((size_t)2 * F, (size_t)L.nqkv) * 4, (size_t)256 << 20);
  L.gemm_ws = take(L.gemm_ws_bytes);
  L.scratch_u32 = take(256);
  L.nrm_ss = take((size_t)32 * (d / 64) * 4);
  L.total = off;
  return L;
}

bool is_device_ptr(const void* p) {
  hipPointerAttribute_t a;
  if (hipPointerGetAttributes(&a, p) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  return a.type == hipMemoryTypeDevice || a.type == hipMemoryTypeManaged;
}

}  // namespace

struct hh_ctx {
  hh_config cfg{};
  Layout L;
  char* arena = nullptr;
  hipStream_t stream = nullptr;
  bool loaded = false;
  bool use_graphs = true;
  bool row_norm = true;  // HH_ROWNORM=0: every RMSNorm as a pass of its own (for comparison)
  float wscale = 1.f;  // MFMA weights hold w * wscale (fp16 repack); epilogues multiply by 1/wscale
  int step_wg = 0;     // workgroups of the persistent batch-1 decode kernel (0: not usable)
  bool step_q4 = false;  // the persistent kernel streams the stored 4-bit rows
  unsigned step_count = 0;  // persistent-kernel launches so far (names each step's epochs)
  int device = 0;           // HIP device current at hh_create
  int step_depth = kStepLoadDepth;  // HH_LOAD_DEPTH: ring slots in flight per streaming wave
  // HH_STEP_QUIET: pause streaming during exchange waits (1, the default:
  // 0.657 -> 0.650 ms per token on the bench request; 0 streams through).
  int step_quiet = 1;
  int step_ring = kStepRingSlots;   // HH_RING_SLOTS: LDS ring slots used (at most kStepRingSlots)
  int step_poll_delay = 60;         // HH_POLL_DELAY: 10 ns ticks before a phase's first exchange poll
  unsigned long long step_wait_ticks = 0;  // HH_STEP_WAIT_TICKS: wait limit (10 ns ticks; 0: 1 s), and
  int step_fail_wait = 0;                  // HH_STEP_FAIL_WAIT: one wait that never completes -- both for
                                           // tests of the failure path
  std::string trace_path;   // HH_STEP_TRACE: file receiving the last traced step's phase timestamps
  std::string err;
  // host mirror of the device bookkeeping
  std::vector<int> len;
  std::vector<std::vector<int>> pages;
  std::vector<int> free_pages;
  std::vector<int> uploaded_streams;  // row_stream contents last uploaded for decode
  std::map<std::tuple<int, int, int>, hipGraphExec_t> graphs;

  template <typename T> T* at(size_t off) const { return reinterpret_cast<T*>(arena + off); }
  hh_status fail(hh_status s, const std::string& m) {
    err = m;
    return s;
  }
  hh_status hip_fail(hipError_t e, const char* what) {
    err = std::string(what) + ": " + hipGetErrorString(e);
    return HH_ERR_HIP;
  }
};

#define HIPCHK(ctx, expr)                                      \
  do {                                                         \
    hipError_t e_ = (expr);                                    \
    if (e_ != hipSuccess) return (ctx)->hip_fail(e_, #expr);   \
  } while (0)

namespace {

KvLayout kv_layout(const hh_ctx* c) { return KvLayout{c->L.n_pages, c->cfg.n_kv_heads, c->L.max_pages}; }

// Enqueue the transformer layers + head for n rows whose bookkeeping
// (row_stream, row_pos, x) has been prepared.  decode_gemv: batch-1 weight
// streaming path; otherwise the MFMA GEMM path.  s_max: attention splits
// (1 = direct output).  head_row >= 0: LM head + argmax of that row only;
// head_row == -1: LM head + argmax of every row (multi-stream decode);
// head_row == -2: no head.
template <typename TW, typename TKV, typename TM>
void enqueue_layers(hh_ctx* c, int n, bool decode_gemv, int s_max, int head_row, float* logits,
                    int prefill_stream = -1, int prefill_pos = 0) {
  using DK = DecodeKernels<TW, TKV, TM>;
  using GK = GemmKernels<TM, TKV>;
  const hh_config& g = c->cfg;
  const Layout& L = c->L;
  hipStream_t st = c->stream;
  const int d = g.d_model, hq = g.n_heads, hkv = g.n_kv_heads, F = g.ffn_dim, V = g.vocab;
  const float eps = g.rms_eps, ws = 1.f / c->wscale;
  const KvLayout kl = kv_layout(c);
  const GemmWorkspace gws{c->at<float>(L.gemm_ws), L.gemm_ws_bytes};
  int* rs = c->at<int>(L.row_stream);
  int* rp = c->at<int>(L.row_pos);
  float* x = c->at<float>(L.x);
  float* q = c->at<float>(L.q);
  float* o32 = c->at<float>(L.o32);
  TKV* kv = c->at<TKV>(L.kv);
  const int* pt = c->at<int>(L.page_table);
  const float2* rope = c->at<float2>(L.rope);
  unsigned long long* slot = c->at<unsigned long long>(L.slot);
  // Lockstep decode rows on fp16 operands with tiled weights split each
  // RMSNorm across the residual product that feeds it and the product that
  // reads it (RowNorm); `pending`: h holds x * gain and the row sums of
  // squares are in nrm_ss, not yet applied.  (For prompt rows the large-tile
  // kernels' arrival chain cost as much as the norm pass it replaced.)
  const bool rnorm = sizeof(TM) == 2 && !decode_gemv && prefill_stream < 0 && head_row == -1 &&
                     !L.wqkvT16.empty() && GK::norm_fusable(d) && d % 256 == 0 && d <= 2048 && c->row_norm;
  float* nss = rnorm ? c->at<float>(L.nrm_ss) : nullptr;
  int* ncnt = rnorm ? c->at<int>(L.nrm_cnt) : nullptr;
  RowNorm rn_use;
  rn_use.ss_in = nss;
  rn_use.nss = d / 64;
  rn_use.n = (float)d;
  rn_use.eps = eps;
  bool pending = false, final_normed = false;
  for (int l = 0; l < g.n_layers; ++l) {
    const float* an = c->at<float>(L.attn_norm[l]);
    const float* mn = c->at<float>(L.mlp_norm[l]);
    if (decode_gemv) {
      DK::qkv_gemv(st, c->at<TW>(L.wqkv[l]), x, an, eps, d, hq, hkv, rs, rp, rope, q, kv, kl, l, pt);
      DK::attention_rows(st, n, q, kv, kl, l, pt, rs, rp, hq, hkv, o32, nullptr);
      DK::resid_gemv(st, c->at<TW>(L.wo[l]), o32, hq * 64, d, x);
      DK::gateup_gemv(st, c->at<TW>(L.wgu[l]), x, mn, eps, d, F, c->at<float>(L.m32));
      DK::resid_gemv(st, c->at<TW>(L.wdown[l]), c->at<float>(L.m32), F, d, x);
    } else {
      TM* h = c->at<TM>(L.h);
      TM* oM = c->at<TM>(L.oM);
      TM* mM = c->at<TM>(L.mM);
      // The attention norm of layer l > 0 was fused into layer l - 1's down
      // projection (its split-K reduction when K is split).
      const bool fuse = GK::norm_fusable(d);
      if (!fuse) DK::rmsnorm_rows(st, n, x, an, eps, d, h);
      else if (l == 0) GK::rmsnorm(st, n, x, d, an, eps, h);
      // Prefill rows of one stream with an fp16 cache use MFMA flash attention.
      const bool flash = prefill_stream >= 0 && sizeof(TKV) == 2 &&
                         flash_prefill_supported(hq / hkv, c->cfg.max_context,
                                                 (size_t)kl.n_pages * 2 * hkv * kPage * kHeadDim);
      // Flash attention reads only the fp16 queries.
      const bool tiled = !L.wqkvT16.empty();
      // Lockstep decode rows (one per stream): the attention kernel takes
      // over the QKV split-K reduction, rotation and KV append.
      const bool fold = prefill_stream < 0 && head_row == -1;
      QkvFold<TKV> qf;
      if (fold) {
        const int sp = GK::qkv_deferred(st, gws, h, n, c->at<TM>(L.wqkvM[l]), d, hq, hkv, ws, rs, rp, rope, q, kv, kl, l,
                                        pt, tiled ? c->at<TM>(L.wqkvT16[l]) : nullptr,
                                        pending ? rn_use : RowNorm());
        if (sp > 1) qf = QkvFold<TKV>{gws.ptr, sp, (hq + 2 * hkv) * 64, ws, rope, kv};
      } else {
        GK::qkv(st, gws, h, n, c->at<TM>(L.wqkvM[l]), d, hq, hkv, ws, rs, rp, rope, flash ? nullptr : q,
                flash ? c->at<TM>(L.qM) : nullptr, kv, kl, l, pt, tiled ? c->at<TM>(L.wqkvT16[l]) : nullptr);
      }
      if (flash) {
        if constexpr (sizeof(TKV) == 2)
          flash_prefill(st, reinterpret_cast<const _Float16*>(c->at<TM>(L.qM)), reinterpret_cast<const _Float16*>(kv),
                        kl, l, pt, prefill_stream, prefill_pos, n, hq, hkv, reinterpret_cast<_Float16*>(oM));
      } else if (prefill_stream >= 0) {
        DK::attention(st, n, q, kv, kl, l, pt, rs, rp, hq, hkv, 1, c->at<float>(L.part), o32, oM);
      } else {
        DK::attention_rows(st, n, q, kv, kl, l, pt, rs, rp, hq, hkv, o32, oM, qf);
      }
      const TM* wo_t = tiled ? c->at<TM>(L.woT16[l]) : nullptr;
      if (fuse) {
        pending = GK::resid(st, gws, oM, n, c->at<TM>(L.woM[l]), hq * 64, d, ws, x, mn, eps, h, wo_t,
                            nss, ncnt, L.nrm_ncnt);
      } else {
        GK::resid(st, gws, oM, n, c->at<TM>(L.woM[l]), hq * 64, d, ws, x, nullptr, 0.f, nullptr, wo_t);
        DK::rmsnorm_rows(st, n, x, mn, eps, d, h);
      }
      GK::gateup(st, gws, h, n, c->at<TM>(L.wguM[l]), d, F, ws, mM, tiled ? c->at<TM>(L.wguT16[l]) : nullptr,
                 pending ? rn_use : RowNorm());
      // The last layer's down projection takes the final norm along under
      // RowNorm (the head reads h next).
      const float* next_an = (fuse && l + 1 < g.n_layers) ? c->at<float>(L.attn_norm[l + 1])
                             : (rnorm && l + 1 == g.n_layers) ? c->at<float>(L.final_norm)
                                                              : nullptr;
      pending = GK::resid(st, gws, mM, n, c->at<TM>(L.wdownM[l]), F, d, ws, x, next_an, eps, h,
                          tiled ? c->at<TM>(L.wdownT16[l]) : nullptr, next_an ? nss : nullptr, ncnt, L.nrm_ncnt);
      if (rnorm && l + 1 == g.n_layers) final_normed = true;
    }
  }
  const float* fn = c->at<float>(L.final_norm);
  if (head_row >= 0) {
    DK::head_gemv(st, c->at<TW>(L.lm_head), x, fn, eps, d, V, head_row, rs, logits, slot);
  } else if (head_row == -1) {
    if (decode_gemv) {
      DK::head_gemv(st, c->at<TW>(L.lm_head), x, fn, eps, d, V, 0, rs, logits, slot);
    } else {
      TM* h = c->at<TM>(L.h);
      if (!final_normed) {
        if (GK::norm_fusable(d)) GK::rmsnorm(st, n, x, d, fn, eps, h);
        else DK::rmsnorm_rows(st, n, x, fn, eps, d, h);
      }
      GK::logits(st, gws, h, n, c->at<TM>(L.lm_headM), d, V, ws, logits, slot, rs,
                 L.wqkvT16.empty() ? nullptr : c->at<TM>(L.lm_headT16), pending ? rn_use : RowNorm());
    }
  }
}

// One decode step for n rows (row_stream already on the device).
template <typename TW, typename TKV, typename TM>
void enqueue_decode(hh_ctx* c, int n, bool feed, bool want_logits) {
  const Layout& L = c->L;
  using DK = DecodeKernels<TW, TKV, TM>;
  DK::prep_embed(c->stream, n, -1, feed ? c->at<int>(L.feed) : nullptr, c->at<int>(L.row_stream),
                 c->at<int>(L.row_pos), c->at<int>(L.pos), c->at<int>(L.pending),
                 c->at<unsigned long long>(L.slot), c->at<TW>(L.embed), c->at<float>(L.x), c->cfg.d_model);
  // The batch-1 GEMV kernels read the model's own (bf16) matrices, which a
  // 4-bit model does not compute with: it takes the MFMA path at one row.
  const bool gemv = n == 1 && c->cfg.weight_format == HH_WF_DTYPE;
  enqueue_layers<TW, TKV, TM>(c, n, gemv, kSplitMax, -1, want_logits ? c->at<float>(L.logits) : nullptr);
  finalize(c->stream, 0, n, c->at<int>(L.row_stream), c->at<int>(L.row_pos), c->at<unsigned long long>(L.slot),
           c->at<int>(L.pending), c->at<int>(L.hist), c->at<int>(L.pos), c->cfg.max_context);
}

// Size the persistent decode kernel to one workgroup per CU (all co-resident)
// and upload the per-layer weight pointer table it reads.
template <typename TW>
hipError_t setup_step_tables(hh_ctx* c) {
  const hh_config& g = c->cfg;
  const Layout& L = c->L;
  std::vector<LayerPtrs<TW>> tab(g.n_layers);
  for (int l = 0; l < g.n_layers; ++l)
    tab[l] = LayerPtrs<TW>{c->at<TW>(L.wqkvM[l]),     c->at<TW>(L.woM[l]),
                           c->at<TW>(L.wguM[l]),      c->at<TW>(L.wdownM[l]),
                           c->at<TW>(L.wdownT[l]),    c->at<float>(L.attn_norm[l]),
                           c->at<float>(L.mlp_norm[l])};
  if (g.n_layers == 0) return hipSuccess;
  hipError_t e = hipMemcpyAsync(c->arena + L.layer_tab, tab.data(), tab.size() * sizeof(LayerPtrs<TW>),
                                hipMemcpyHostToDevice, c->stream);
  if (e == hipSuccess) e = hipStreamSynchronize(c->stream);
  return e;
}

template <typename TW, typename TKV>
int step_workgroups(const hh_config& g) {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  const char* env = std::getenv("HH_STEP_KERNEL");
  if (env && env[0] == '0') return 0;
  const int nwg = std::min(cus, kMaxStepWG);
  if (!StepKernel<TW, TKV>::supports(g.d_model, g.ffn_dim, g.n_heads, g.n_kv_heads, g.vocab, g.n_layers, nwg))
    return 0;
  // An attention item covers at most 256 pages (its page list sits in LDS).
  if ((g.max_context + kPage - 1) / kPage > 256 * (nwg / g.n_kv_heads)) return 0;
  if (StepKernel<TW, TKV>::max_blocks_per_cu(g.d_model, g.ffn_dim, g.n_heads, g.n_kv_heads) < 1) return 0;
  return nwg;
}

// 4-bit models: the stored rows of every streamed matrix (Wdown^T for the
// split-K down projection; the unused Wdown slot repeats it).
hipError_t setup_step_tables_q4(hh_ctx* c) {
  const hh_config& g = c->cfg;
  const Layout& L = c->L;
  std::vector<LayerPtrs<Q4Row>> tab(g.n_layers);
  for (int l = 0; l < g.n_layers; ++l)
    tab[l] = LayerPtrs<Q4Row>{c->at<Q4Row>(L.wqkvQ[l]),   c->at<Q4Row>(L.woQ[l]),
                              c->at<Q4Row>(L.wguQ[l]),    c->at<Q4Row>(L.wdownTQ[l]),
                              c->at<Q4Row>(L.wdownTQ[l]), c->at<float>(L.attn_norm[l]),
                              c->at<float>(L.mlp_norm[l])};
  if (g.n_layers == 0) return hipSuccess;
  hipError_t e = hipMemcpyAsync(c->arena + L.layer_tab, tab.data(), tab.size() * sizeof(LayerPtrs<Q4Row>),
                                hipMemcpyHostToDevice, c->stream);
  if (e == hipSuccess) e = hipStreamSynchronize(c->stream);
  return e;
}

hipError_t setup_step_kernel(hh_ctx* c) {
  if (c->cfg.dtype == HH_BF16) {
    if (c->cfg.weight_format == HH_WF_Q4G32) {
      // Without the 4-bit kernel (other shapes) the fp16 one streams the
      // fp16 copies, which hold the same values.
      c->step_wg = step_workgroups<Q4Row, _Float16>(c->cfg);
      c->step_q4 = c->step_wg > 0;
      if (c->step_q4) return setup_step_tables_q4(c);
    }
    c->step_wg = step_workgroups<_Float16, _Float16>(c->cfg);
    return setup_step_tables<_Float16>(c);
  }
  c->step_wg = step_workgroups<float, float>(c->cfg);
  return setup_step_tables<float>(c);
}

template <typename TW, typename TKV>
hh_status launch_step(hh_ctx* c, int s, bool feed, bool want_logits, const StepWords& words) {
  const hh_config& g = c->cfg;
  const Layout& L = c->L;
  StepParams<TW, TKV> P{};
  P.d = g.d_model;
  P.F = g.ffn_dim;
  P.hq = g.n_heads;
  P.hkv = g.n_kv_heads;
  P.V = g.vocab;
  P.n_layers = g.n_layers;
  P.max_ctx = g.max_context;
  P.stream = s;
  P.ring_slots = c->step_ring;
  P.load_depth = c->step_depth;
  P.quiet = c->step_quiet;
  P.poll_delay = c->step_poll_delay;
  P.wait_ticks = c->step_wait_ticks;
  P.fail_wait = c->step_fail_wait;
  P.eps = g.rms_eps;
  P.epoch = words.epoch;
  P.layer = c->at<LayerPtrs<TW>>(L.layer_tab);
  P.embed = c->at<typename StepEmbed<TW>::type>(L.embed);
  // 4-bit rows carry their own scales (no power-of-two factor).
  constexpr bool q4 = std::is_same<TW, Q4Row>::value;
  P.head = c->at<TW>(q4 ? L.lm_headQ : L.lm_headM);
  P.wscale_inv = q4 ? 1.0f : 1.0f / c->wscale;
  P.final_norm = c->at<float>(L.final_norm);
  P.rope = c->at<float2>(L.rope);
  P.kvc = c->at<TKV>(L.kv);
  P.kv = kv_layout(c);
  P.page_table = c->at<int>(L.page_table);
  P.pos = c->at<int>(L.pos);
  P.pending = c->at<int>(L.pending);
  P.hist = c->at<int>(L.hist);
  P.feed = feed ? c->at<int>(L.feed) : nullptr;
  P.logits = want_logits ? c->at<float>(L.logits) : nullptr;
  unsigned long long* w = words.base;
  const size_t d = g.d_model, hq = g.n_heads, hkv = g.n_kv_heads, cap = words.cap;
  P.ll_xa = w;
  P.ll_xb = P.ll_xa + d;
  P.ll_q = P.ll_xb + d;
  P.ll_kn = P.ll_q + hq * 64;
  P.ll_vn = P.ll_kn + hkv * 64;
  P.ll_part = P.ll_vn + hkv * 64;
  P.ll_o = P.ll_part + hq * cap * 66;
  P.ll_dp = P.ll_o + hq * 64;
  P.ll_keys = P.ll_dp + cap * d;
  P.err = reinterpret_cast<int*>(P.ll_keys + 2 * cap);
  P.trace = c->trace_path.empty() ? nullptr : c->at<unsigned long long>(L.trace);
  const hipError_t e = StepKernel<TW, TKV>::launch(P, c->step_wg, c->stream);
  if (e != hipSuccess) return c->hip_fail(e, "decode-step kernel launch");
  return HH_OK;
}

// Make sure stream s owns pages for positions [0, new_len); upload new entries.
hh_status ensure_pages(hh_ctx* c, int s, int new_len) {
  const int need = (new_len + kPage - 1) / kPage;
  std::vector<int>& pg = c->pages[s];
  const int first_new = (int)pg.size();
  if (need <= first_new) return HH_OK;
  if ((int)c->free_pages.size() < need - first_new) return c->fail(HH_ERR_CONTEXT_FULL, "KV page pool exhausted");
  for (int i = first_new; i < need; ++i) {
    pg.push_back(c->free_pages.back());
    c->free_pages.pop_back();
  }
  int* dst = c->at<int>(c->L.page_table) + (size_t)s * c->L.max_pages + first_new;
  put_ints(c->stream, dst, pg.data() + first_new, need - first_new);
  HIPCHK(c, hipGetLastError());
  return HH_OK;
}

// LM head + greedy key of row `row` of x into logits (optional) and the
// row's stream slot.  A 4-bit model's head values live only in the fp16
// copy: RMSNorm of the row, then a one-row MFMA product.
template <typename TW, typename TKV, typename TM>
void enqueue_head_row(hh_ctx* c, int row, float* logits, unsigned long long* slot) {
  const Layout& L = c->L;
  const hh_config& g = c->cfg;
  hipStream_t st = c->stream;
  if constexpr (sizeof(TM) == 2) {
    if (g.weight_format == HH_WF_Q4G32) {
      using GK = GemmKernels<TM, TKV>;
      const GemmWorkspace gws{c->at<float>(L.gemm_ws), L.gemm_ws_bytes};
      TM* h = c->at<TM>(L.h);
      GK::rmsnorm(st, 1, c->at<float>(L.x) + (size_t)row * g.d_model, g.d_model, c->at<float>(L.final_norm),
                  g.rms_eps, h);
      GK::logits(st, gws, h, 1, c->at<TM>(L.lm_headM), g.d_model, g.vocab, 1.f / c->wscale, logits, slot,
                 c->at<int>(L.row_stream) + row, L.wqkvT16.empty() ? nullptr : c->at<TM>(L.lm_headT16));
      return;
    }
  }
  using DK = DecodeKernels<TW, TKV, TM>;
  DK::head_gemv(st, c->at<TW>(L.lm_head), c->at<float>(L.x), c->at<float>(L.final_norm), g.rms_eps, g.d_model,
                g.vocab, row, c->at<int>(L.row_stream), logits, slot);
}

template <typename TW, typename TKV, typename TM>
hh_status do_prefill(hh_ctx* c, int s, const int32_t* tokens, int n, int mode, float* logits, int32_t* next) {
  const Layout& L = c->L;
  using DK = DecodeKernels<TW, TKV, TM>;
  hipStream_t st = c->stream;
  const int V = c->cfg.vocab;
  hh_status rc = ensure_pages(c, s, c->len[s] + n);
  if (rc != HH_OK) return rc;
  const int chunk = L.rows_cap;
  float* lbuf = c->at<float>(L.logits);
  // The prefill rows overwrite row_stream: the next decode uploads its ids.
  c->uploaded_streams.clear();
  for (int r0 = 0; r0 < n; r0 += chunk) {
    const int P = std::min(chunk, n - r0);
    const bool last = r0 + P == n;
    HIPCHK(c, hipMemcpyAsync(c->at<int>(L.feed), tokens + r0, P * sizeof(int), hipMemcpyHostToDevice, st));
    DK::prep_embed(st, P, s, c->at<int>(L.feed), c->at<int>(L.row_stream), c->at<int>(L.row_pos), c->at<int>(L.pos),
                   c->at<int>(L.pending), c->at<unsigned long long>(L.slot), c->at<TW>(L.embed), c->at<float>(L.x),
                   c->cfg.d_model);
    enqueue_layers<TW, TKV, TM>(c, P, false, 1, -2, nullptr, s, c->len[s] + r0);
    unsigned long long* slot = c->at<unsigned long long>(L.slot);
    if (mode == HH_LOGITS_ALL) {
      for (int b0 = 0; b0 < P; b0 += kLogitRows) {
        const int nb = std::min(kLogitRows, P - b0);
        for (int i = 0; i < nb; ++i)
          enqueue_head_row<TW, TKV, TM>(c, b0 + i, lbuf + (size_t)i * V, (last && b0 + i == P - 1) ? slot : nullptr);
        HIPCHK(c, hipMemcpyAsync(logits + (size_t)(r0 + b0) * V, lbuf, (size_t)nb * V * sizeof(float),
                                 hipMemcpyDefault, st));
      }
    } else if (last) {
      enqueue_head_row<TW, TKV, TM>(c, P - 1, mode == HH_LOGITS_LAST ? lbuf : nullptr, slot);
      if (mode == HH_LOGITS_LAST)
        HIPCHK(c, hipMemcpyAsync(logits, lbuf, (size_t)V * sizeof(float), hipMemcpyDefault, st));
    }
    finalize(st, P - 1, 1, c->at<int>(L.row_stream), c->at<int>(L.row_pos), last ? slot : nullptr,
             c->at<int>(L.pending), c->at<int>(L.hist), c->at<int>(L.pos), c->cfg.max_context);
    HIPCHK(c, hipGetLastError());
  }
  if (next) HIPCHK(c, hipMemcpyAsync(next, c->at<int>(L.pending) + s, sizeof(int), hipMemcpyDefault, st));
  c->len[s] += n;
  return HH_OK;
}

// Prompts of several streams: their rows go through every layer together
// (each row attends to its own stream's keys), in passes of at most rows_cap
// rows; a prompt longer than what is left of a pass continues in the next
// one (its later rows attend to the keys the earlier pass wrote).  After each
// pass, the streams whose last row it held get their next token from the
// n-row head on those rows.
template <typename TW, typename TKV, typename TM>
hh_status do_prefill_batch(hh_ctx* c, int n, const int32_t* ids, const int32_t* lens, const int32_t* tokens,
                           int32_t* next) {
  const Layout& L = c->L;
  using DK = DecodeKernels<TW, TKV, TM>;
  using GK = GemmKernels<TM, TKV>;
  hipStream_t st = c->stream;
  const hh_config& g = c->cfg;
  const int d = g.d_model;
  for (int i = 0; i < n; ++i) {
    hh_status rc = ensure_pages(c, ids[i], c->len[ids[i]] + lens[i]);
    if (rc != HH_OK) return rc;
  }
  c->uploaded_streams.clear();
  int* row_stream = c->at<int>(L.row_stream);
  int* row_pos = c->at<int>(L.row_pos);
  float* x = c->at<float>(L.x);
  const float* fn = c->at<float>(L.final_norm);
  unsigned long long* slot = c->at<unsigned long long>(L.slot);
  TM* h = c->at<TM>(L.h);
  const GemmWorkspace gws{c->at<float>(L.gemm_ws), L.gemm_ws_bytes};
  std::vector<int> base(n), done(n, 0), offset(n + 1, 0);
  for (int i = 0; i < n; ++i) {
    base[i] = c->len[ids[i]];
    offset[i + 1] = offset[i] + lens[i];
  }
  int cur = 0;  // first stream with rows left
  while (cur < n) {
    std::vector<int> rs, rp, tk, last_s, last_p, last_r;
    while (cur < n && (int)rs.size() < L.rows_cap) {
      const int take = std::min(lens[cur] - done[cur], L.rows_cap - (int)rs.size());
      for (int j = 0; j < take; ++j) {
        rs.push_back(ids[cur]);
        rp.push_back(base[cur] + done[cur] + j);
        tk.push_back(tokens[offset[cur] + done[cur] + j]);
      }
      done[cur] += take;
      if (done[cur] == lens[cur]) {
        last_r.push_back((int)rs.size() - 1);
        last_s.push_back(ids[cur]);
        last_p.push_back(rp.back());
        ++cur;
      }
    }
    const int R = (int)rs.size(), ne = (int)last_r.size();
    HIPCHK(c, hipMemcpyAsync(row_stream, rs.data(), R * sizeof(int), hipMemcpyHostToDevice, st));
    HIPCHK(c, hipMemcpyAsync(row_pos, rp.data(), R * sizeof(int), hipMemcpyHostToDevice, st));
    HIPCHK(c, hipMemcpyAsync(c->at<int>(L.feed), tk.data(), R * sizeof(int), hipMemcpyHostToDevice, st));
    DK::prep_embed(st, R, -2, c->at<int>(L.feed), row_stream, row_pos, c->at<int>(L.pos), c->at<int>(L.pending),
                   slot, c->at<TW>(L.embed), x, d);
    enqueue_layers<TW, TKV, TM>(c, R, false, 1, -2, nullptr);
    if (ne > 0) {
      // Last rows to rows 0 .. ne-1 (row i's source lies at or after row i
      // and after every earlier destination), then the head and argmax.
      for (int i = 0; i < ne; ++i)
        if (last_r[i] != i)
          HIPCHK(c, hipMemcpyAsync(x + (size_t)i * d, x + (size_t)last_r[i] * d, d * sizeof(float),
                                   hipMemcpyDeviceToDevice, st));
      HIPCHK(c, hipMemcpyAsync(row_stream, last_s.data(), ne * sizeof(int), hipMemcpyHostToDevice, st));
      HIPCHK(c, hipMemcpyAsync(row_pos, last_p.data(), ne * sizeof(int), hipMemcpyHostToDevice, st));
      if (GK::norm_fusable(d)) GK::rmsnorm(st, ne, x, d, fn, g.rms_eps, h);
      else DK::rmsnorm_rows(st, ne, x, fn, g.rms_eps, d, h);
      GK::logits(st, gws, h, ne, c->at<TM>(L.lm_headM), d, g.vocab, 1.f / c->wscale, nullptr, slot, row_stream,
                 L.wqkvT16.empty() ? nullptr : c->at<TM>(L.lm_headT16));
      finalize(st, 0, ne, row_stream, row_pos, slot, c->at<int>(L.pending), c->at<int>(L.hist), c->at<int>(L.pos),
               g.max_context);
    }
    HIPCHK(c, hipGetLastError());
    // The host arrays above are read by the copies: wait for them.
    HIPCHK(c, hipStreamSynchronize(st));
  }
  if (next)
    for (int i = 0; i < n; ++i)
      HIPCHK(c, hipMemcpyAsync(next + i, c->at<int>(L.pending) + ids[i], sizeof(int), hipMemcpyDefault, st));
  for (int i = 0; i < n; ++i) c->len[ids[i]] += lens[i];
  return HH_OK;
}

// words: null for the context's own exchange words, else the fixed array of
// the allocation-free entry point (batch-1 single-kernel steps only).
template <typename TW, typename TKV, typename TM>
hh_status do_decode(hh_ctx* c, int n, const std::vector<int>& ids, const int32_t* tokens, float* logits,
                    int32_t* next, const StepWords* words = nullptr) {
  const Layout& L = c->L;
  hipStream_t st = c->stream;
  for (int i = 0; i < n; ++i) {
    hh_status rc = ensure_pages(c, ids[i], c->len[ids[i]] + 1);
    if (rc != HH_OK) return rc;
  }
  if (c->uploaded_streams != ids) {
    put_ints(st, c->at<int>(L.row_stream), ids.data(), n);
    HIPCHK(c, hipGetLastError());
    c->uploaded_streams = ids;
  }
  if (tokens) {
    put_ints(st, c->at<int>(L.feed), tokens, n);
    HIPCHK(c, hipGetLastError());
  }
  const bool want_logits = logits != nullptr;
  if (n == 1 && (c->step_wg > 0 || words)) {
    // Each step owns 512 epochs (8 phases x 64 layers); epoch 0 is never
    // used, so zero-initialised exchange words never look current.
    StepWords w{c->at<unsigned long long>(L.ll), (size_t)kMaxStepWG, 0};
    if (words) {
      w = *words;
    } else {
      c->step_count += 1;
      w.epoch = c->step_count * 512u;
    }
    hh_status rc;
    if constexpr (sizeof(TM) == 2)
      rc = c->step_q4 ? launch_step<Q4Row, TKV>(c, ids[0], tokens != nullptr, want_logits, w)
                      : launch_step<TM, TKV>(c, ids[0], tokens != nullptr, want_logits, w);
    else
      rc = launch_step<TM, TKV>(c, ids[0], tokens != nullptr, want_logits, w);
    if (rc != HH_OK) return rc;
  } else if (c->use_graphs) {
    auto key = std::make_tuple(n, tokens != nullptr ? 1 : 0, want_logits ? 1 : 0);
    auto it = c->graphs.find(key);
    if (it == c->graphs.end()) {
      hipGraph_t graph;
      HIPCHK(c, hipStreamBeginCapture(st, hipStreamCaptureModeRelaxed));
      enqueue_decode<TW, TKV, TM>(c, n, tokens != nullptr, want_logits);
      hipError_t e = hipStreamEndCapture(st, &graph);
      if (e != hipSuccess) return c->hip_fail(e, "hipStreamEndCapture");
      hipGraphExec_t exec;
      e = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
      (void)hipGraphDestroy(graph);
      if (e != hipSuccess) return c->hip_fail(e, "hipGraphInstantiate");
      it = c->graphs.emplace(key, exec).first;
    }
    HIPCHK(c, hipGraphLaunch(it->second, st));
  } else {
    enqueue_decode<TW, TKV, TM>(c, n, tokens != nullptr, want_logits);
    HIPCHK(c, hipGetLastError());
  }
  if (logits)
    HIPCHK(c, hipMemcpyAsync(logits, c->at<float>(L.logits), (size_t)n * c->cfg.vocab * sizeof(float),
                             hipMemcpyDefault, st));
  if (next) {
    // pending[] is indexed by stream id; gather the listed streams' tokens.
    bool contiguous = true;
    for (int i = 0; i < n; ++i) contiguous = contiguous && ids[i] == ids[0] + i;
    if (contiguous) {
      HIPCHK(c, hipMemcpyAsync(next, c->at<int>(L.pending) + ids[0], n * sizeof(int), hipMemcpyDefault, st));
    } else {
      for (int i = 0; i < n; ++i)
        HIPCHK(c, hipMemcpyAsync(next + i, c->at<int>(L.pending) + ids[i], sizeof(int), hipMemcpyDefault, st));
    }
  }
  for (int i = 0; i < n; ++i) c->len[ids[i]] += 1;
  return HH_OK;
}

hh_status reset_stream(hh_ctx* c, int s) {
  for (int p : c->pages[s]) c->free_pages.push_back(p);
  c->pages[s].clear();
  c->len[s] = 0;
  HIPCHK(c, hipMemsetAsync(c->at<int>(c->L.pos) + s, 0, sizeof(int), c->stream));
  HIPCHK(c, hipMemsetAsync(c->at<int>(c->L.pending) + s, 0, sizeof(int), c->stream));
  HIPCHK(c, hipMemsetAsync(c->at<unsigned long long>(c->L.slot) + s, 0, sizeof(unsigned long long), c->stream));
  return HH_OK;
}

// Synchronize when outputs live in host memory; report a timed-out grid
// barrier of the persistent decode kernel at that point.
hh_status finish(hh_ctx* c, bool host_out, const int* err_word = nullptr) {
  if (!host_out) return HH_OK;
  int err = 0;
  if (!err_word && c->step_wg > 0)
    err_word = reinterpret_cast<const int*>(c->at<unsigned long long>(c->L.ll) + c->L.ll_words - 8);
  if (err_word) HIPCHK(c, hipMemcpyAsync(&err, err_word, sizeof(int), hipMemcpyDeviceToHost, c->stream));
  HIPCHK(c, hipStreamSynchronize(c->stream));
  if (err)
    return c->fail(HH_ERR_HIP, "decode-step exchange wait timed out (workgroups not co-resident); "
                               "steps record -1 until hh_reset");
  return HH_OK;
}

// ---------------------------------------------------------------- allocation-free decode step

// Exchange words of hh_decode_step_noalloc: a fixed array in every device's
// memory (each GPU the library runs on holds its own copy until the process
// ends).  In host code `scratch` names a host-side stand-in, not device
// memory: only the address hipGetSymbolAddress returns for the current
// device is ever passed to kernels or copies.
constexpr size_t kScratchWords = (size_t)9 << 17;  // 9 MiB of 8-byte words
static __device__ __align__(256) unsigned long long scratch[kScratchWords];

constexpr int kMaxDevices = 64;
struct ScratchTable {
  std::mutex mu;
  unsigned long long* ptr[kMaxDevices] = {};
  hipError_t rc[kMaxDevices] = {};
  unsigned steps[kMaxDevices] = {};  // noalloc steps launched on the device (names their epochs)
};
ScratchTable& scratch_table() {
  static ScratchTable t;
  return t;
}

// Once per device, with that device current: the device address of its copy.
void scratch_setup(int dev) {
  if (dev < 0 || dev >= kMaxDevices) return;
  ScratchTable& t = scratch_table();
  std::lock_guard<std::mutex> lk(t.mu);
  if (t.ptr[dev] || t.rc[dev] != hipSuccess) return;
  void* p = nullptr;
  const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
  if (e == hipSuccess && p) t.ptr[dev] = static_cast<unsigned long long*>(p);
  else t.rc[dev] = e != hipSuccess ? e : hipErrorInvalidSymbol;
}

__global__ void k_zero_words(unsigned long long* p, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0ull;
}

}  // namespace

extern "C" {

hh_status hh_workspace_size(const hh_config* cfg, size_t* bytes) {
  if (!cfg || !bytes) return HH_ERR_INVALID_ARG;
  std::string why;
  if (!config_supported(*cfg, why)) return HH_ERR_UNSUPPORTED;
  *bytes = make_layout(*cfg).total;
  return HH_OK;
}

hh_status hh_create(const hh_config* cfg, void* arena, size_t arena_bytes, void* hip_stream, hh_ctx** out) {
  if (!cfg || !out || !arena || !hip_stream || (reinterpret_cast<uintptr_t>(arena) & 255)) return HH_ERR_INVALID_ARG;
  std::string why;
  if (!config_supported(*cfg, why)) return HH_ERR_UNSUPPORTED;
  Layout L = make_layout(*cfg);
  if (arena_bytes < L.total) return HH_ERR_OOM;
  hh_ctx* c = new hh_ctx();
  c->cfg = *cfg;
  c->L = L;
  c->arena = static_cast<char*>(arena);
  c->stream = static_cast<hipStream_t>(hip_stream);
  if (hipGetDevice(&c->device) != hipSuccess) c->device = -1;
  scratch_setup(c->device);
  const char* tp = std::getenv("HH_STEP_TRACE");
  if (tp) c->trace_path = tp;
  if (const char* q = std::getenv("HH_STEP_QUIET")) c->step_quiet = std::atoi(q);
  if (const char* pd = std::getenv("HH_POLL_DELAY")) c->step_poll_delay = std::max(0, std::atoi(pd));
  if (const char* r = std::getenv("HH_RING_SLOTS")) c->step_ring = std::min(kStepRingSlots, std::max(6, std::atoi(r)));
  if (const char* ld = std::getenv("HH_LOAD_DEPTH")) c->step_depth = std::min(7, std::max(1, std::atoi(ld)));
  if (const char* wt = std::getenv("HH_STEP_WAIT_TICKS")) c->step_wait_ticks = std::max(1LL, std::atoll(wt));
  if (const char* fw = std::getenv("HH_STEP_FAIL_WAIT")) c->step_fail_wait = std::atoi(fw) != 0;
  const char* ge = std::getenv("HH_GRAPHS");
  c->use_graphs = !(ge && ge[0] == '0');
  const char* rne = std::getenv("HH_ROWNORM");
  c->row_norm = !(rne && rne[0] == '0');
  c->len.assign(cfg->max_streams, 0);
  c->pages.assign(cfg->max_streams, {});
  for (int p = L.n_pages - 1; p >= 0; --p) c->free_pages.push_back(p);
  // RoPE table: angle p * theta^(-2i/64) in fp64, cos/sin rounded to fp32.
  std::vector<float2> rope((size_t)cfg->max_context * 32);
  for (int p = 0; p < cfg->max_context; ++p)
    for (int i = 0; i < 32; ++i) {
      const double a = (double)p * std::pow((double)cfg->rope_theta, -2.0 * i / 64.0);
      rope[(size_t)p * 32 + i] = make_float2((float)std::cos(a), (float)std::sin(a));
    }
  hipError_t e = hipMemcpyAsync(c->at<float2>(L.rope), rope.data(), rope.size() * sizeof(float2),
                                hipMemcpyHostToDevice, c->stream);
  if (e == hipSuccess) e = hipMemsetAsync(c->arena + L.page_table, 0, L.row_stream - L.page_table, c->stream);
  if (e == hipSuccess) e = setup_step_kernel(c);
  if (e == hipSuccess) e = hipStreamSynchronize(c->stream);
  if (e != hipSuccess) {
    delete c;
    return HH_ERR_HIP;
  }
  *out = c;
  return HH_OK;
}

hh_status hh_load_weights(hh_ctx* c, const void* const* tensors, int32_t n_tensors) {
  if (!c) return HH_ERR_INVALID_ARG;
  const hh_config& g = c->cfg;
  const int expect = 1 + 9 * g.n_layers + 1 + (g.tied_embeddings ? 0 : 1);
  if (!tensors || n_tensors != expect)
    return c->fail(HH_ERR_INVALID_ARG, "expected " + std::to_string(expect) + " weight tensors");
  for (int i = 0; i < n_tensors; ++i)
    if (!tensors[i]) return c->fail(HH_ERR_INVALID_ARG, "NULL weight tensor " + std::to_string(i));
  const Layout& L = c->L;
  hipStream_t st = c->stream;
  const size_t d = g.d_model, F = g.ffn_dim, V = g.vocab, hq = g.n_heads, hkv = g.n_kv_heads;
  const bool bf = g.dtype == HH_BF16;
  auto copy = [&](size_t off, const void* src, size_t bytes) {
    return hipMemcpyAsync(c->arena + off, src, bytes, hipMemcpyDefault, st);
  };
  // Norm gains arrive in the weight dtype; they are kept as fp32.
  char* tmp = c->arena + L.mM;  // scratch (prefill activations) while loading
  auto gain = [&](size_t off, const void* src) {
    if (!bf) return copy(off, src, d * 4);
    hipError_t e = hipMemcpyAsync(tmp, src, d * 2, hipMemcpyDefault, st);
    if (e == hipSuccess) {
      widen_bf16(st, reinterpret_cast<const __bf16*>(tmp), c->at<float>(off), d);
      e = hipStreamSynchronize(st);
    }
    return e;
  };
  int t = 0;
  HIPCHK(c, copy(L.embed, tensors[t++], V * d * L.ew));
  for (int l = 0; l < g.n_layers; ++l) {
    HIPCHK(c, gain(L.attn_norm[l], tensors[t++]));
    HIPCHK(c, copy(L.wqkv[l], tensors[t++], hq * 64 * d * L.ew));
    HIPCHK(c, copy(L.wqkv[l] + hq * 64 * d * L.ew, tensors[t++], hkv * 64 * d * L.ew));
    HIPCHK(c, copy(L.wqkv[l] + (hq + hkv) * 64 * d * L.ew, tensors[t++], hkv * 64 * d * L.ew));
    HIPCHK(c, copy(L.wo[l], tensors[t++], d * hq * 64 * L.ew));
    HIPCHK(c, gain(L.mlp_norm[l], tensors[t++]));
    HIPCHK(c, copy(L.wgu[l], tensors[t++], F * d * L.ew));
    HIPCHK(c, copy(L.wgu[l] + F * d * L.ew, tensors[t++], F * d * L.ew));
    HIPCHK(c, copy(L.wdown[l], tensors[t++], d * F * L.ew));
    if (!bf) transpose(st, c->at<float>(L.wdown[l]), c->at<float>(L.wdownT[l]), (int)d, (int)F);
  }
  HIPCHK(c, gain(L.final_norm, tensors[t++]));
  if (!g.tied_embeddings) HIPCHK(c, copy(L.lm_head, tensors[t++], V * d * L.ew));
  if (bf) {
    // fp16 operands for the MFMA path: one power-of-two scale for all matrices.
    std::vector<std::tuple<size_t, size_t, size_t>> list;
    list.emplace_back(L.embed, L.embedM, V * d);
    if (!g.tied_embeddings) list.emplace_back(L.lm_head, L.lm_headM, V * d);
    for (int l = 0; l < g.n_layers; ++l) {
      list.emplace_back(L.wqkv[l], L.wqkvM[l], (size_t)L.nqkv * d);
      list.emplace_back(L.wo[l], L.woM[l], d * hq * 64);
      list.emplace_back(L.wgu[l], L.wguM[l], 2 * F * d);
      list.emplace_back(L.wdown[l], L.wdownM[l], d * F);
    }
    unsigned int* amax = c->at<unsigned int>(L.scratch_u32);
    HIPCHK(c, hipMemsetAsync(amax, 0, 4, st));
    for (auto& m : list) absmax_bf16(st, c->at<__bf16>(std::get<0>(m)), std::get<2>(m), amax);
    unsigned int bits = 0;
    HIPCHK(c, hipMemcpyAsync(&bits, amax, 4, hipMemcpyDeviceToHost, st));
    HIPCHK(c, hipStreamSynchronize(st));
    float mx;
    std::memcpy(&mx, &bits, 4);
    if (!(mx < 3.0e38f)) return c->fail(HH_ERR_INVALID_ARG, "non-finite weight");
    const int e = mx > 0.f ? (int)std::ceil(std::log2((double)mx)) : 0;
    const int sexp = std::max(-20, std::min(40, 14 - e));  // largest |w| * 2^s <= 2^14
    c->wscale = std::ldexp(1.0f, sexp);
    if (g.weight_format == HH_WF_Q4G32) {
      // 4-bit rows for the streaming decode kernel; the fp16 copies hold their
      // values q * s (times 2^s, exactly), so every path computes with them.
      auto quant = [&](size_t src, size_t rows, size_t K, size_t q4, size_t dst) {
        q4g32(st, c->at<__bf16>(src), rows, (int)K, c->at<unsigned char>(q4), c->at<_Float16>(dst), c->wscale);
      };
      if (g.tied_embeddings) {
        quant(L.embed, V, d, L.lm_headQ, L.embedM);
      } else {
        bf16_to_f16_scaled(st, c->at<__bf16>(L.embed), c->at<_Float16>(L.embedM), V * d, c->wscale);
        quant(L.lm_head, V, d, L.lm_headQ, L.lm_headM);
      }
      for (int l = 0; l < g.n_layers; ++l) {
        quant(L.wqkv[l], L.nqkv, d, L.wqkvQ[l], L.wqkvM[l]);
        quant(L.wo[l], d, hq * 64, L.woQ[l], L.woM[l]);
        quant(L.wgu[l], 2 * F, d, L.wguQ[l], L.wguM[l]);
        // W_down is grouped along its output rows: quantize the rows of its
        // transpose (in place: bf16 in, fp16 values out), then transpose back.
        transpose(st, c->at<__bf16>(L.wdown[l]), c->at<__bf16>(L.wdownT[l]), (int)d, (int)F);
        quant(L.wdownT[l], F, d, L.wdownTQ[l], L.wdownT[l]);
        transpose(st, c->at<_Float16>(L.wdownT[l]), c->at<_Float16>(L.wdownM[l]), (int)F, (int)d);
      }
    } else {
      for (auto& m : list)
        bf16_to_f16_scaled(st, c->at<__bf16>(std::get<0>(m)), c->at<_Float16>(std::get<1>(m)), std::get<2>(m),
                           c->wscale);
      // Wdown^T of the fp16 copy, for the batch-1 decode kernel's split-K down projection.
      for (int l = 0; l < g.n_layers; ++l)
        transpose(st, c->at<_Float16>(L.wdownM[l]), c->at<_Float16>(L.wdownT[l]), (int)d, (int)F);
    }
    if (!L.wqkvT16.empty()) {
      tile16(st, c->at<_Float16>(L.lm_headM), c->at<_Float16>(L.lm_headT16), (int)V, (int)d, (int)V, 0);
      for (int l = 0; l < g.n_layers; ++l) {
        tile16(st, c->at<_Float16>(L.wqkvM[l]), c->at<_Float16>(L.wqkvT16[l]), L.nqkv, (int)d, L.nqkv, 0);
        tile16(st, c->at<_Float16>(L.woM[l]), c->at<_Float16>(L.woT16[l]), (int)d, (int)(hq * 64), (int)d, 0);
        tile16(st, c->at<_Float16>(L.wguM[l]), c->at<_Float16>(L.wguT16[l]), (int)(2 * F), (int)d,
               (int)((F + 31) / 32 * 64), (int)F);
        tile16(st, c->at<_Float16>(L.wdownM[l]), c->at<_Float16>(L.wdownT16[l]), (int)d, (int)F, (int)d, 0);
      }
    }
  } else {
    c->wscale = 1.f;
  }
  HIPCHK(c, hipGetLastError());
  HIPCHK(c, hipStreamSynchronize(st));
  for (int s = 0; s < g.max_streams; ++s) {
    hh_status rc = reset_stream(c, s);
    if (rc != HH_OK) return rc;
  }
  HIPCHK(c, hipStreamSynchronize(st));
  c->loaded = true;
  c->err.clear();
  return HH_OK;
}

hh_status hh_prefill(hh_ctx* c, int32_t s, const int32_t* tokens, int32_t n, int32_t mode, float* logits,
                     int32_t* next) {
  if (!c) return HH_ERR_INVALID_ARG;
  if (!c->loaded) return c->fail(HH_ERR_NOT_LOADED, "weights not loaded");
  const hh_config& g = c->cfg;
  if (s < 0 || s >= g.max_streams) return c->fail(HH_ERR_INVALID_ARG, "stream id out of range");
  if (!tokens || n <= 0) return c->fail(HH_ERR_INVALID_ARG, "need at least one token");
  if (mode < HH_LOGITS_NONE || mode > HH_LOGITS_ALL) return c->fail(HH_ERR_INVALID_ARG, "bad logits mode");
  if (mode != HH_LOGITS_NONE && !logits) return c->fail(HH_ERR_INVALID_ARG, "logits buffer required");
  for (int i = 0; i < n; ++i)
    if (tokens[i] < 0 || tokens[i] >= g.vocab) return c->fail(HH_ERR_INVALID_ARG, "token id out of range");
  if ((long long)c->len[s] + n > g.max_context) return c->fail(HH_ERR_CONTEXT_FULL, "prompt exceeds max_context");
  hh_status rc = g.dtype == HH_BF16 ? do_prefill<__bf16, _Float16, _Float16>(c, s, tokens, n, mode, logits, next)
                                    : do_prefill<float, float, float>(c, s, tokens, n, mode, logits, next);
  if (rc != HH_OK) return rc;
  return finish(c, (logits && !is_device_ptr(logits)) || (next && !is_device_ptr(next)));
}

hh_status hh_prefill_batch(hh_ctx* c, int32_t n, const int32_t* stream_ids, const int32_t* lengths,
                           const int32_t* tokens, int32_t* next_tokens) {
  if (!c) return HH_ERR_INVALID_ARG;
  if (!c->loaded) return c->fail(HH_ERR_NOT_LOADED, "weights not loaded");
  const hh_config& g = c->cfg;
  if (n < 1 || n > g.max_streams || !stream_ids || !lengths || !tokens)
    return c->fail(HH_ERR_INVALID_ARG, "need 1..max_streams streams, their lengths and tokens");
  std::vector<char> seen(g.max_streams, 0);
  long long total = 0;
  for (int i = 0; i < n; ++i) {
    const int s = stream_ids[i];
    if (s < 0 || s >= g.max_streams) return c->fail(HH_ERR_INVALID_ARG, "stream id out of range");
    if (seen[s]) return c->fail(HH_ERR_INVALID_ARG, "stream listed twice");
    seen[s] = 1;
    if (lengths[i] < 1) return c->fail(HH_ERR_INVALID_ARG, "every prompt needs at least one token");
    if ((long long)c->len[s] + lengths[i] > g.max_context)
      return c->fail(HH_ERR_CONTEXT_FULL, "prompt exceeds max_context");
    total += lengths[i];
  }
  for (long long i = 0; i < total; ++i)
    if (tokens[i] < 0 || tokens[i] >= g.vocab) return c->fail(HH_ERR_INVALID_ARG, "token id out of range");
  hh_status rc = g.dtype == HH_BF16
                     ? do_prefill_batch<__bf16, _Float16, _Float16>(c, n, stream_ids, lengths, tokens, next_tokens)
                     : do_prefill_batch<float, float, float>(c, n, stream_ids, lengths, tokens, next_tokens);
  if (rc != HH_OK) return rc;
  return finish(c, next_tokens && !is_device_ptr(next_tokens));
}

hh_status hh_decode_step(hh_ctx* c, int32_t n, const int32_t* stream_ids, const int32_t* tokens, float* logits,
                         int32_t* next) {
  if (!c) return HH_ERR_INVALID_ARG;
  if (!c->loaded) return c->fail(HH_ERR_NOT_LOADED, "weights not loaded");
  const hh_config& g = c->cfg;
  if (n < 1 || n > g.max_streams) return c->fail(HH_ERR_INVALID_ARG, "n_streams out of range");
  std::vector<int> ids(n);
  std::vector<char> seen(g.max_streams, 0);
  for (int i = 0; i < n; ++i) {
    ids[i] = stream_ids ? stream_ids[i] : i;
    if (ids[i] < 0 || ids[i] >= g.max_streams) return c->fail(HH_ERR_INVALID_ARG, "stream id out of range");
    if (seen[ids[i]]) return c->fail(HH_ERR_INVALID_ARG, "duplicate stream id");
    seen[ids[i]] = 1;
    if (c->len[ids[i]] + 1 > g.max_context) return c->fail(HH_ERR_CONTEXT_FULL, "stream at max_context");
    if (!tokens && c->len[ids[i]] == 0) return c->fail(HH_ERR_INVALID_ARG, "empty stream needs an explicit token");
    if (tokens && (tokens[i] < 0 || tokens[i] >= g.vocab))
      return c->fail(HH_ERR_INVALID_ARG, "token id out of range");
  }
  // Page availability is checked before any state changes.
  int need = 0;
  for (int i = 0; i < n; ++i) {
    const int have = (int)c->pages[ids[i]].size();
    need += std::max(0, (c->len[ids[i]] + 1 + kPage - 1) / kPage - have);
  }
  if (need > (int)c->free_pages.size()) return c->fail(HH_ERR_CONTEXT_FULL, "KV page pool exhausted");
  hh_status rc = g.dtype == HH_BF16 ? do_decode<__bf16, _Float16, _Float16>(c, n, ids, tokens, logits, next)
                                    : do_decode<float, float, float>(c, n, ids, tokens, logits, next);
  if (rc != HH_OK) return rc;
  return finish(c, (logits && !is_device_ptr(logits)) || (next && !is_device_ptr(next)));
}

hh_status hh_decode_step_noalloc(hh_ctx* c, int32_t s, const int32_t* token, float* logits, int32_t* next) {
  if (!c) return HH_ERR_INVALID_ARG;
  if (!c->loaded) return c->fail(HH_ERR_NOT_LOADED, "weights not loaded");
  const hh_config& g = c->cfg;
  if (s < 0 || s >= g.max_streams) return c->fail(HH_ERR_INVALID_ARG, "stream id out of range");
  if (c->step_wg <= 0)
    return c->fail(HH_ERR_UNSUPPORTED, "the single-kernel decode step is not available for this configuration");
  const size_t need = step_words(g, (size_t)c->step_wg);
  if (need > kScratchWords)
    return c->fail(HH_ERR_UNSUPPORTED, "exchange words exceed the fixed array (" + std::to_string(need) + " > " +
                                           std::to_string(kScratchWords) + " words)");
  if (c->device < 0 || c->device >= kMaxDevices) return c->fail(HH_ERR_HIP, "no HIP device recorded for the context");
  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess || cur != c->device)
    return c->fail(HH_ERR_INVALID_ARG, "the context's device is not the current device");
  if (c->len[s] + 1 > g.max_context) return c->fail(HH_ERR_CONTEXT_FULL, "stream at max_context");
  if (!token && c->len[s] == 0) return c->fail(HH_ERR_INVALID_ARG, "empty stream needs an explicit token");
  if (token && (*token < 0 || *token >= g.vocab)) return c->fail(HH_ERR_INVALID_ARG, "token id out of range");
  const int have = (int)c->pages[s].size();
  if ((c->len[s] + 1 + kPage - 1) / kPage > have && c->free_pages.empty())
    return c->fail(HH_ERR_CONTEXT_FULL, "KV page pool exhausted");
  ScratchTable& t = scratch_table();
  StepWords w{nullptr, (size_t)c->step_wg, 0};
  {
    std::lock_guard<std::mutex> lk(t.mu);
    if (!t.ptr[c->device]) {
      c->err = std::string("fixed exchange array: hipGetSymbolAddress: ") + hipGetErrorString(t.rc[c->device]);
      return HH_ERR_HIP;
    }
    w.base = t.ptr[c->device];
    // Epochs are counted per device, across contexts, so the words another
    // context left in the array never look current to this step.
    t.steps[c->device] += 1;
    w.epoch = t.steps[c->device] * 512u;
  }
  // The error word must start at zero (a fill kernel: capture-safe).
  const int n_err = 8;
  k_zero_words<<<1, 64, 0, c->stream>>>(w.base + need - n_err, n_err);
  HIPCHK(c, hipGetLastError());
  const std::vector<int> ids{s};
  hh_status rc = g.dtype == HH_BF16 ? do_decode<__bf16, _Float16, _Float16>(c, 1, ids, token, logits, next, &w)
                                    : do_decode<float, float, float>(c, 1, ids, token, logits, next, &w);
  if (rc != HH_OK) return rc;
  return finish(c, (logits && !is_device_ptr(logits)) || (next && !is_device_ptr(next)), step_err_word(g, w));
}

hh_status hh_reset(hh_ctx* c, int32_t s) {
  if (!c) return HH_ERR_INVALID_ARG;
  if (s < -1 || s >= c->cfg.max_streams) return c->fail(HH_ERR_INVALID_ARG, "stream id out of range");
  for (int i = 0; i < c->cfg.max_streams; ++i)
    if (s == -1 || s == i) {
      hh_status rc = reset_stream(c, i);
      if (rc != HH_OK) return rc;
    }
  // Clear the decode-step kernel's error word: later steps run again (a
  // stream that recorded -1 keeps it as its pending token until reset).
  if (c->step_wg > 0)
    HIPCHK(c, hipMemsetAsync(c->at<unsigned long long>(c->L.ll) + c->L.ll_words - 8, 0, sizeof(int), c->stream));
  return HH_OK;
}

hh_status hh_stream_length(const hh_ctx* c, int32_t s, int32_t* length) {
  if (!c || !length || s < 0 || s >= c->cfg.max_streams) return HH_ERR_INVALID_ARG;
  *length = c->len[s];
  return HH_OK;
}

hh_status hh_read_argmax(hh_ctx* c, int32_t s, int32_t first, int32_t n, int32_t* out) {
  if (!c) return HH_ERR_INVALID_ARG;
  if (s < 0 || s >= c->cfg.max_streams || !out || n < 0 || first < 0 || first + n > c->len[s])
    return c->fail(HH_ERR_INVALID_ARG, "argmax range outside the stream");
  if (n == 0) return HH_OK;
  HIPCHK(c, hipMemcpyAsync(out, c->at<int>(c->L.hist) + (size_t)s * c->cfg.max_context + first, n * sizeof(int),
                           hipMemcpyDeviceToHost, c->stream));
  HIPCHK(c, hipStreamSynchronize(c->stream));
  return HH_OK;
}

void hh_destroy(hh_ctx* c) {
  if (!c) return;
  if (!c->trace_path.empty() && c->step_wg > 0 && c->step_count > 0) {
    // Diagnostic dump: binary [nwg][n_layers + 1][32] uint64 timestamps of the last step.
    const size_t n = (size_t)c->step_wg * (c->cfg.n_layers + 1) * 32;
    std::vector<unsigned long long> h(n);
    if (hipMemcpyAsync(h.data(), c->at<unsigned long long>(c->L.trace), n * 8, hipMemcpyDeviceToHost, c->stream) ==
            hipSuccess &&
        hipStreamSynchronize(c->stream) == hipSuccess) {
      if (FILE* f = std::fopen(c->trace_path.c_str(), "wb")) {
        std::fwrite(h.data(), 8, n, f);
        std::fclose(f);
      }
    }
  }
  for (auto& kv : c->graphs) (void)hipGraphExecDestroy(kv.second);
  delete c;
}

const char* hh_last_error(const hh_ctx* c) { return c ? c->err.c_str() : "NULL context"; }

hh_status hh_q4g32_quantize(const uint16_t* src, int64_t rows, int32_t K, uint8_t* dst, void* hip_stream) {
  if (!src || !dst || rows < 1 || K < 32 || K % 32 != 0) return HH_ERR_INVALID_ARG;
  q4g32(static_cast<hipStream_t>(hip_stream), reinterpret_cast<const __bf16*>(src), (size_t)rows, K,
        reinterpret_cast<unsigned char*>(dst), nullptr, 1.f);
  return hipGetLastError() == hipSuccess ? HH_OK : HH_ERR_HIP;
}

}  // extern "C"

namespace hh {
void read_probe(hipStream_t st, const void* src, size_t bytes);  // k_load.hip
}

extern "C" {

hh_status hh_read_probe(const void* src, size_t bytes, void* hip_stream) {
  if (!src || bytes < 16 || bytes % 16 != 0 || reinterpret_cast<uintptr_t>(src) % 16 != 0) return HH_ERR_INVALID_ARG;
  if (!is_device_ptr(src)) return HH_ERR_INVALID_ARG;
  read_probe(static_cast<hipStream_t>(hip_stream), src, bytes);
  return hipGetLastError() == hipSuccess ? HH_OK : HH_ERR_HIP;
}

}  // extern "C"
