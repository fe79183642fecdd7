// Host-callable launchers of the gfx950 kernels (internal to the library).
// Template parameters: TW = weight storage type of the weight-streaming GEMVs
// (float or __bf16), TKV = KV-cache element type (float or _Float16), TM =
// MFMA operand type of the dense GEMM path (float or _Float16).
#pragma once

#include "hh_device.h"

namespace hh {

template <typename TW, typename TKV, typename TM>
struct DecodeKernels {
  static void prep_embed(hipStream_t st, int n_rows, int prefill_stream, const int* feed, int* row_stream,
                         int* row_pos, const int* pos, const int* pending, const TW* embed, float* x, int d);
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
  static void rmsnorm_rows(hipStream_t st, int n_rows, const float* x, const float* gain, float eps, int d, TM* h);
};

void finalize(hipStream_t st, int r0, int n, const int* row_stream, const int* row_pos, unsigned long long* slot,
              int* pending, int* hist, int* pos, int max_ctx);

template <typename TM, typename TKV>
struct GemmKernels {
  static void qkv(hipStream_t st, const TM* A, int M, const TM* W, int d, int hq, int hkv, float scale,
                  const int* row_stream, const int* row_pos, const float2* rope, float* q, TKV* kv, KvLayout L,
                  int layer, const int* page_table);
  static void resid(hipStream_t st, const TM* A, int M, const TM* W, int K, int N, float scale, float* x);
  static void gateup(hipStream_t st, const TM* A, int M, const TM* W, int d, int F, float scale, TM* m);
  static void logits(hipStream_t st, const TM* A, int M, const TM* W, int d, int V, float scale, float* logits,
                     unsigned long long* slot, const int* row_stream);
};

// Load-time weight preparation.
void widen_bf16(hipStream_t st, const __bf16* src, float* dst, size_t n);
void absmax_bf16(hipStream_t st, const __bf16* src, size_t n, unsigned int* out_bits);
void bf16_to_f16_scaled(hipStream_t st, const __bf16* src, _Float16* dst, size_t n, float scale);

}  // namespace hh
