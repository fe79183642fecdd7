/*
 * hh.h -- C ABI of the MI355X (gfx950) decoder runtime for the "mouth" model
 * of the Horsehair runtime path.
 *
 * The paper's runtime phase ends with a 1B-class decoder-only model that
 * streams a rendered answer (Sec. 4, "Runtime phase"): one prompt evaluation,
 * whose latency is the time to first token, followed by token-by-token
 * streaming decode (the three speed quantities are defined in Sec. 6.2; the
 * KV cache's memory grows with the context window, Sec. 6.6).  The paper does
 * not describe the model's internals, so the library implements the standard
 * Llama-style decoder: RMSNorm, rotary embeddings (rotate-half pairing), grouped
 * query attention, SwiGLU MLP, tied or untied LM head, greedy argmax.
 *
 * Conventions for every call:
 *  - Every function returns an hh_status; HH_OK is 0, errors are negative.
 *    On any error the context's state (stream lengths, KV contents, pending
 *    tokens, loaded weights) is unchanged and hh_last_error() describes it.
 *  - A context is not thread-safe: use it from one host thread at a time.
 *  - All GPU work of a context is enqueued on the HIP stream given to
 *    hh_create.  Calls whose outputs are host memory synchronize that stream
 *    before returning; calls whose outputs are device memory (or absent) only
 *    enqueue.
 *  - Pointer arguments documented "host or device" are classified with
 *    hipPointerGetAttributes; "host" arguments must be host memory.
 */
#ifndef HH_H_
#define HH_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t hh_status;

enum {
  HH_OK = 0,
  HH_ERR_INVALID_ARG = -1,   /* bad pointer, id, size or tensor count        */
  HH_ERR_OOM = -2,           /* arena smaller than hh_workspace_size()       */
  HH_ERR_CONTEXT_FULL = -3,  /* a stream would exceed max_context            */
  HH_ERR_NOT_LOADED = -4,    /* prefill/decode before hh_load_weights        */
  HH_ERR_HIP = -5,           /* a HIP runtime call failed                    */
  HH_ERR_UNSUPPORTED = -6    /* configuration outside what the kernels cover */
};

enum { HH_F32 = 0, HH_BF16 = 1 };                       /* weight / KV element type */
/*
 * Weight formats.  HH_WF_DTYPE: the weights are used as loaded (cfg.dtype).
 * HH_WF_Q4G32 (bf16 models only): the paper's mouth model runs 4-bit weights
 * (Sec. 4 "Runtime phase", Sec. 5) without naming the format; this library's
 * 4-bit format is symmetric per group of 32 consecutive elements of a row:
 * scale s = bf16(max|w| / 7) (fp32 division, round to nearest even), codes
 * q = clamp(rint(w / s), -8, 7) (fp32 division, ties to even), value q * s.
 * At load the bf16 matrices are quantized row by row (W_q, W_k, W_v, W_o,
 * W_gate, W_up along their input dimension, W_down along its output
 * dimension, i.e. the rows of W_down^T, and the LM head's copy of the
 * embedding); the token-embedding table stays bf16.  Every kernel then
 * computes with the values q * s.
 */
enum { HH_WF_DTYPE = 0, HH_WF_Q4G32 = 1 };
enum { HH_LOGITS_NONE = 0, HH_LOGITS_LAST = 1, HH_LOGITS_ALL = 2 };

/*
 * Model and capacity description.  Supported: head_dim == 64, page_size == 16,
 * n_heads / n_kv_heads in {1, 2, 4, 8}, d_model % 64 == 0, ffn_dim % 8 == 0,
 * vocab >= 2, max_context <= 131072; anything else gives HH_ERR_UNSUPPORTED.  rms_eps is added to the mean square inside the root;
 * rope_theta is the rotary base (frequencies theta^(-2i/head_dim)).
 */
typedef struct {
  int32_t n_layers, d_model, n_heads, n_kv_heads, head_dim, ffn_dim, vocab;
  float rms_eps, rope_theta;
  int32_t tied_embeddings;   /* 1: LM head is the embedding matrix           */
  int32_t dtype;             /* HH_F32 or HH_BF16: weights and KV cache      */
  int32_t max_streams;       /* independent sequences held at once (>= 1)    */
  int32_t max_context;       /* positions per stream (prompt + generated)    */
  int32_t page_size;         /* KV page length in tokens; must be 16         */
  int32_t max_prefill;       /* rows per prefill pass; 0 means max_context.
                                Longer prompts are processed in passes.      */
  int32_t weight_format;     /* HH_WF_DTYPE or HH_WF_Q4G32 (dtype HH_BF16,
                                d_model % 32 == 0)                           */
} hh_config;

typedef struct hh_ctx hh_ctx;

/* Bytes of device memory hh_create needs for this configuration. */
hh_status hh_workspace_size(const hh_config* cfg, size_t* bytes);

/*
 * Create a context inside a caller-owned device arena.
 *  arena       device pointer, 256-byte aligned, at least hh_workspace_size()
 *              bytes; it holds weights, KV pages, RoPE tables and scratch and
 *              must outlive hh_destroy.  The library never allocates device
 *              memory of its own.
 *  hip_stream  hipStream_t to enqueue on; must not be the legacy NULL stream
 *              (decode steps are replayed as HIP graphs captured on it).
 *  out         receives the context (host object owned by the library).
 * Errors: INVALID_ARG (NULL/unaligned arena, NULL stream), UNSUPPORTED, OOM.
 */
hh_status hh_create(const hh_config* cfg, void* arena, size_t arena_bytes, void* hip_stream,
                    hh_ctx** out);

/*
 * Copy the model weights into the arena (repacking them for the kernels).
 *  tensors    n_tensors pointers, host or device, element type cfg.dtype
 *             (float or bf16 bits), row-major [out, in] as in nn.Linear:
 *               embed[vocab, d];
 *               per layer: attn_norm[d], wq[Hq*64, d], wk[Hkv*64, d],
 *                          wv[Hkv*64, d], wo[d, Hq*64], mlp_norm[d],
 *                          w_gate[F, d], w_up[F, d], w_down[d, F];
 *               final_norm[d]; lm_head[vocab, d] only if untied.
 *  n_tensors  must be 1 + 9 * n_layers + 1 (+1 if untied).
 * The caller may free the sources after return (the call synchronizes).
 * Loading resets every stream.  Errors: INVALID_ARG, HIP.
 */
hh_status hh_load_weights(hh_ctx* ctx, const void* const* tensors, int32_t n_tensors);

/*
 * Prompt evaluation (the TTFT step): append n_tokens tokens to stream
 * stream_id, starting at its current length, and compute the greedy next
 * token from the last row.
 *  tokens       host, n_tokens ids in [0, vocab).
 *  logits_mode  HH_LOGITS_NONE, _LAST (logits = [vocab]) or _ALL
 *               (logits = [n_tokens, vocab]); fp32, host or device.
 *  next_token   NULL or one int32 (host or device): argmax of the last row,
 *               lowest index among ties.  The same token is kept on the
 *               device as the stream's pending token for hh_decode_step.
 * Errors: INVALID_ARG (id out of range, n_tokens <= 0, NULL logits with a
 * logits mode), CONTEXT_FULL, NOT_LOADED, HIP.
 */
hh_status hh_prefill(hh_ctx* ctx, int32_t stream_id, const int32_t* tokens, int32_t n_tokens,
                     int32_t logits_mode, float* logits, int32_t* next_token);

/*
 * Prompt evaluation for several streams together (several requests
 * arriving together, the paper's runtime phase at more than one user): the
 * prompts of n distinct streams are appended as one set of rows, every layer
 * runs over all of them (each row attends to its own stream's keys up to its
 * position), and the greedy next token of each stream comes from its last
 * row, as hh_prefill would give it.  Rows go through in passes of at most
 * max_prefill rows (max_context when 0, and at least max_streams), in
 * stream_ids order; a prompt that does not fit in what is left of a pass
 * continues in the next one.
 *  stream_ids   host, n distinct ids; lengths host, n counts >= 1.
 *  tokens       host, the prompts concatenated in stream_ids order
 *               (sum of lengths ids in [0, vocab)).
 *  next_tokens  NULL or n int32 (host or device), in stream_ids order.
 * The call waits for its passes to finish.  Errors: INVALID_ARG (n outside
 * 1..max_streams, an id out of range or repeated, a length < 1, a token out
 * of range), CONTEXT_FULL, NOT_LOADED, HIP.
 */
hh_status hh_prefill_batch(hh_ctx* ctx, int32_t n, const int32_t* stream_ids, const int32_t* lengths,
                           const int32_t* tokens, int32_t* next_tokens);

/*
 * One greedy decode step of n_streams streams in lockstep: each listed stream
 * consumes one token at its current length and advances by one.
 *  stream_ids   host, n_streams distinct ids; NULL means 0..n_streams-1.
 *  tokens       host, n_streams ids to consume (teacher forcing), or NULL to
 *               consume each stream's pending token (the previous argmax,
 *               kept on the device: no host round trip).
 *  logits       NULL or [n_streams, vocab] fp32, host or device.
 *  next_tokens  NULL or [n_streams] int32, host or device.
 * A stream with no tokens yet decodes at position 0 (its pending token must
 * then be given through tokens).  Errors: INVALID_ARG, CONTEXT_FULL,
 * NOT_LOADED, HIP.
 * Failure of a batch-1 step: every cross-workgroup wait of the single-kernel
 * step is bounded (about 1 s).  When one gives up, the step's token is -1
 * (pending token, next_tokens, and the history hh_read_argmax returns), and
 * so is the token of every later step of that stream, and of every step of
 * any stream until hh_reset; the first call with host outputs after the
 * failure returns HH_ERR_HIP.  Device-fed loops detect it by the -1.
 */
hh_status hh_decode_step(hh_ctx* ctx, int32_t n_streams, const int32_t* stream_ids,
                         const int32_t* tokens, float* logits, int32_t* next_tokens);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): one greedy
 * batch-1 decode step of stream_id, as hh_decode_step with n_streams == 1,
 * whose cross-workgroup exchange words live in a fixed array the library
 * keeps in each device's memory (9 MiB per device, held until the process
 * ends) instead of the context's arena.  The call allocates nothing and
 * captures no graph: it enqueues a small fill of the array's error word and
 * the single-kernel step on the context's stream.
 *  token        host, one id to consume, or NULL for the stream's pending
 *               token.
 *  logits       NULL or [vocab] fp32, host or device.
 *  next_token   NULL or one int32, host or device.
 * Every context on a device shares that device's array, and it keeps the
 * last step's contents: steps of different contexts that overlap in time on
 * one device (different streams, no ordering between them) race and give
 * wrong results.  Steps in one stream's order are safe.
 * Errors: as hh_decode_step; UNSUPPORTED when the configuration has no
 * single-kernel step or needs more exchange words than the array holds
 * (d_model 2048 with 32 query heads fits up to 256 workgroups); INVALID_ARG
 * when the context's device is not the current one.
 */
hh_status hh_decode_step_noalloc(hh_ctx* ctx, int32_t stream_id, const int32_t* token, float* logits,
                                 int32_t* next_token);

/* Drop a stream's KV pages and set its length to 0 (stream_id -1: all).
 * Also clears the context's record of a failed decode step (see
 * hh_decode_step). */
hh_status hh_reset(hh_ctx* ctx, int32_t stream_id);

/* Current length (positions held in the KV cache) of a stream. */
hh_status hh_stream_length(const hh_ctx* ctx, int32_t stream_id, int32_t* length);

/*
 * Read back greedy outputs recorded on the device: out[i] is the argmax
 * computed at position first_pos + i of stream_id (i.e. the prediction of the
 * token at position first_pos + i + 1).  Positions must be < the stream's
 * length and must have been the last row of a prefill or a decode step.
 *  out  host, n int32.  Synchronizes the stream.
 */
hh_status hh_read_argmax(hh_ctx* ctx, int32_t stream_id, int32_t first_pos, int32_t n,
                         int32_t* out);

/*
 * The HH_WF_Q4G32 quantizer the loader runs, on its own: quantize rows of
 * bf16 values into the stored row format -- for each row, K / 2 bytes of
 * codes (n = q + 8; element 2k in the low nibble of byte k, 2k + 1 in the
 * high nibble) followed by the K / 32 scales as little-endian bf16, i.e.
 * K / 2 + K / 16 bytes per row.
 *  src         device, rows x K bf16 bits, row-major; finite values.
 *  K           a positive multiple of 32.
 *  dst         device, rows x (K / 2 + K / 16) bytes.
 *  hip_stream  hipStream_t the kernel is enqueued on (not synchronized).
 * Errors: INVALID_ARG (NULL pointer, rows < 1, K not a multiple of 32), HIP.
 */
hh_status hh_q4g32_quantize(const uint16_t* src, int64_t rows, int32_t K, uint8_t* dst, void* hip_stream);

/* Destroy the host context (the arena stays the caller's). NULL is a no-op. */
void hh_destroy(hh_ctx* ctx);

/* Measurement aid, not a step of the decoder: enqueue on hip_stream one pass
 * that reads `bytes` of device memory at src once (16-byte vector loads from
 * every CU) and computes nothing visible.  Timed by the caller with events,
 * it gives the read bandwidth a kernel can reach on the device, the
 * reference the decode kernel's HBM fraction is also reported against.
 * src must be device memory, 16-byte aligned, bytes a positive multiple of
 * 16; otherwise HH_ERR_INVALID_ARG. */
hh_status hh_read_probe(const void* src, size_t bytes, void* hip_stream);

/* Message of the last error on this context ("" if none); never NULL. */
const char* hh_last_error(const hh_ctx* ctx);

#ifdef __cplusplus
}
#endif

#endif /* HH_H_ */
