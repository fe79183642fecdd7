// Host-side checks of the library's C ABI, built with AddressSanitizer and
// UndefinedBehaviorSanitizer by tests/test_host_sanitize.py.  Everything here
// runs without a GPU: configuration validation and workspace sizing (layout
// arithmetic for the largest supported shapes), the argument checks every
// entry point makes before it touches HIP, and the router / renderer.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "hh.h"
#include "hh_router.h"

static int failures = 0;
#define CHECK(cond)                                                    \
  do {                                                                 \
    if (!(cond)) {                                                     \
      std::fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #cond); \
      ++failures;                                                      \
    }                                                                  \
  } while (0)

static hh_config tiny() {
  hh_config c{};
  c.n_layers = 2; c.d_model = 256; c.n_heads = 4; c.n_kv_heads = 2; c.head_dim = 64; c.ffn_dim = 688; c.vocab = 4096;
  c.rms_eps = 1e-5f; c.rope_theta = 10000.f; c.tied_embeddings = 1; c.dtype = HH_F32;
  c.max_streams = 2; c.max_context = 128; c.page_size = 16; c.max_prefill = 0; c.weight_format = HH_WF_DTYPE;
  return c;
}

static hh_config one_b() {
  hh_config c = tiny();
  c.n_layers = 16; c.d_model = 2048; c.n_heads = 32; c.n_kv_heads = 8; c.ffn_dim = 8192; c.vocab = 128256;
  c.rope_theta = 500000.f; c.dtype = HH_BF16; c.max_context = 8704; c.max_streams = 1;
  return c;
}

static void check_configs() {
  size_t b = 0, b2 = 0;
  hh_config c = tiny();
  CHECK(hh_workspace_size(&c, &b) == HH_OK && b > 0);
  CHECK(hh_workspace_size(nullptr, &b) == HH_ERR_INVALID_ARG);
  CHECK(hh_workspace_size(&c, nullptr) == HH_ERR_INVALID_ARG);
  // Every unsupported field is rejected, not mis-sized.
  struct Bad { int32_t hh_config::*f; int32_t v; } bad[] = {
    {&hh_config::head_dim, 128}, {&hh_config::page_size, 32}, {&hh_config::n_kv_heads, 3}, {&hh_config::d_model, 200},
    {&hh_config::ffn_dim, 690}, {&hh_config::dtype, 7}, {&hh_config::max_streams, 0}, {&hh_config::max_context, 131073},
    {&hh_config::weight_format, 2}, {&hh_config::weight_format, HH_WF_Q4G32}, {&hh_config::n_layers, -1},
    {&hh_config::vocab, 1}, {&hh_config::max_context, 0}, {&hh_config::n_heads, -4}, {&hh_config::max_prefill, -1},
  };
  for (const Bad& x : bad) {
    hh_config d = tiny();
    d.*(x.f) = x.v;
    const hh_status s = hh_workspace_size(&d, &b);
    CHECK(s == HH_ERR_UNSUPPORTED || s == HH_ERR_INVALID_ARG);
  }
  // The size grows with the window; the largest windows and many streams
  // exercise the layout arithmetic far past 32-bit ranges.
  hh_config o = one_b();
  CHECK(hh_workspace_size(&o, &b) == HH_OK);
  o.max_context = 131072;
  CHECK(hh_workspace_size(&o, &b2) == HH_OK && b2 > b);
  o.max_streams = 64;
  CHECK(hh_workspace_size(&o, &b) == HH_OK && b > b2 && b > ((size_t)64 * 131072 * 32768));
  o.max_streams = 1; o.max_context = 8704; o.max_prefill = 8192;
  CHECK(hh_workspace_size(&o, &b) == HH_OK);
  o.weight_format = HH_WF_Q4G32;
  CHECK(hh_workspace_size(&o, &b2) == HH_OK && b2 > 0);
}

static void check_entry_points() {
  // Argument checks run before any HIP call, so none of these touches a GPU.
  hh_config c = tiny();
  hh_ctx* ctx = reinterpret_cast<hh_ctx*>(0x1);
  CHECK(hh_create(nullptr, reinterpret_cast<void*>(256), 1 << 30, reinterpret_cast<void*>(1), &ctx) == HH_ERR_INVALID_ARG);
  CHECK(hh_create(&c, nullptr, 1 << 30, reinterpret_cast<void*>(1), &ctx) == HH_ERR_INVALID_ARG);
  CHECK(hh_create(&c, reinterpret_cast<void*>(4096 + 8), 1 << 30, reinterpret_cast<void*>(1), &ctx) == HH_ERR_INVALID_ARG);
  CHECK(hh_create(&c, reinterpret_cast<void*>(4096), 1 << 30, nullptr, &ctx) == HH_ERR_INVALID_ARG);
  CHECK(hh_create(&c, reinterpret_cast<void*>(4096), 1 << 30, reinterpret_cast<void*>(1), nullptr) == HH_ERR_INVALID_ARG);
  CHECK(ctx == reinterpret_cast<hh_ctx*>(0x1));  // untouched on error
  const int32_t tok[2] = {1, 2}, sid[1] = {0}, len[1] = {2};
  int32_t nxt[2] = {0, 0}, n = 0;
  CHECK(hh_load_weights(nullptr, nullptr, 0) == HH_ERR_INVALID_ARG);
  CHECK(hh_prefill(nullptr, 0, tok, 2, HH_LOGITS_NONE, nullptr, nxt) == HH_ERR_INVALID_ARG);
  CHECK(hh_prefill_batch(nullptr, 1, sid, len, tok, nxt) == HH_ERR_INVALID_ARG);
  CHECK(hh_decode_step(nullptr, 1, sid, tok, nullptr, nxt) == HH_ERR_INVALID_ARG);
  CHECK(hh_decode_step_noalloc(nullptr, 0, tok, nullptr, nxt) == HH_ERR_INVALID_ARG);
  CHECK(hh_reset(nullptr, 0) == HH_ERR_INVALID_ARG);
  CHECK(hh_stream_length(nullptr, 0, &n) == HH_ERR_INVALID_ARG);
  CHECK(hh_read_argmax(nullptr, 0, 0, 1, nxt) == HH_ERR_INVALID_ARG);
  uint16_t src[64] = {};
  uint8_t dst[64] = {};
  CHECK(hh_q4g32_quantize(nullptr, 1, 32, dst, nullptr) == HH_ERR_INVALID_ARG);
  CHECK(hh_q4g32_quantize(src, 1, 48, dst, nullptr) == HH_ERR_INVALID_ARG);
  CHECK(hh_q4g32_quantize(src, 0, 32, dst, nullptr) == HH_ERR_INVALID_ARG);
  CHECK(hh_read_probe(nullptr, 64, nullptr) == HH_ERR_INVALID_ARG);
  CHECK(hh_read_probe(src, 15, nullptr) == HH_ERR_INVALID_ARG);
  hh_destroy(nullptr);
}

static void check_router() {
  const char* store[] = {
    "The capital of France is Paris.",
    "Paris is also a city in Texas",
    "",                                  // an entry without terms
    "!!! ??? ...",                       // separators only
    "Caf\xc3\xa9 au lait, na\xc3\xafve r\xc3\xa9sum\xc3\xa9",  // UTF-8 words stay whole
    "tea tea tea tea tea tea tea tea tea tea tea tea tea",
  };
  const int n = (int)(sizeof(store) / sizeof(store[0]));
  hh_router* r = nullptr;
  CHECK(hh_router_create(nullptr, n, 1.2f, 0.75f, &r) == HH_ERR_INVALID_ARG);
  CHECK(hh_router_create(store, 0, 1.2f, 0.75f, &r) == HH_ERR_INVALID_ARG);
  CHECK(hh_router_create(store, n, -1.f, 0.75f, &r) == HH_ERR_INVALID_ARG);
  CHECK(hh_router_create(store, n, 1.2f, 1.5f, &r) == HH_ERR_INVALID_ARG);
  CHECK(hh_router_create(store, n, 1.2f, 0.75f, nullptr) == HH_ERR_INVALID_ARG);
  const char* empty_store[] = {"", "--"};
  CHECK(hh_router_create(empty_store, 2, 1.2f, 0.75f, &r) == HH_ERR_INVALID_ARG && r == nullptr);
  CHECK(hh_router_create(store, n, 1.2f, 0.75f, &r) == HH_OK && r != nullptr);
  int32_t ne = 0, nt = 0;
  CHECK(hh_router_size(r, &ne, &nt) == HH_OK && ne == n && nt > 10);
  std::vector<int32_t> ids(16, -1);
  std::vector<double> sc(16, -1.0);
  int32_t got = 0;
  CHECK(hh_router_query(r, "capital of France", 2, ids.data(), sc.data(), &got) == HH_OK && got == 2 && ids[0] == 0);
  CHECK(sc[0] >= sc[1]);
  CHECK(hh_router_query(r, "paris", 16, ids.data(), sc.data(), &got) == HH_OK && got == n);
  for (int i = 1; i < got; ++i) CHECK(sc[i - 1] > sc[i] || (sc[i - 1] == sc[i] && ids[i - 1] < ids[i]));
  CHECK(hh_router_query(r, "", 3, ids.data(), sc.data(), &got) == HH_OK && got == 3 && sc[0] == 0.0);
  CHECK(hh_router_query(r, "r\xc3\xa9sum\xc3\xa9", 1, ids.data(), sc.data(), &got) == HH_OK && ids[0] == 4);
  CHECK(hh_router_query(r, "paris", 0, ids.data(), sc.data(), &got) == HH_ERR_INVALID_ARG);
  CHECK(hh_router_query(r, nullptr, 1, ids.data(), sc.data(), &got) == HH_ERR_INVALID_ARG);
  std::string longq;
  for (int i = 0; i < 20000; ++i) longq += (i % 7 == 0) ? " tea" : " x" + std::to_string(i % 97);
  CHECK(hh_router_query(r, longq.c_str(), 4, ids.data(), sc.data(), &got) == HH_OK && ids[0] == 5);
  int32_t entry = -1, esc = -1;
  double margin = -1.0;
  CHECK(hh_router_route(r, "capital of France", 0.05f, &entry, &margin, &esc) == HH_OK && entry == 0 && esc == 0);
  CHECK(margin > 0.05 && margin <= 1.0);
  CHECK(hh_router_route(r, "zzz unknown", 0.05f, &entry, &margin, &esc) == HH_OK && margin == 0.0 && esc == 1);
  CHECK(hh_router_route(r, "paris", std::nanf(""), &entry, &margin, &esc) == HH_ERR_INVALID_ARG);
  CHECK(hh_router_route(r, "paris", 0.05f, nullptr, &margin, &esc) == HH_ERR_INVALID_ARG);
  hh_router_destroy(r);
  hh_router_destroy(nullptr);

  int64_t need = 0;
  CHECK(hh_render_marker("line one\r\nline two", nullptr, 0, &need) == HH_ERR_INVALID_ARG && need > 0);
  std::vector<char> out((size_t)need, '\0');
  int64_t wrote = 0;
  CHECK(hh_render_marker("line one\r\nline two", out.data(), need, &wrote) == HH_OK && wrote == need);
  const std::string s(out.data(), (size_t)wrote);
  CHECK(s.find("line one  line two\n") != std::string::npos);
  CHECK(s.find('\r') == std::string::npos);
  CHECK(hh_render_marker("x", out.data(), 1, &wrote) == HH_ERR_INVALID_ARG);
  CHECK(hh_render_marker(nullptr, out.data(), need, &wrote) == HH_ERR_INVALID_ARG);
  CHECK(hh_render_marker("x", out.data(), need, nullptr) == HH_ERR_INVALID_ARG);
}

int main() {
  check_configs();
  check_entry_points();
  check_router();
  if (failures) {
    std::fprintf(stderr, "%d host checks failed\n", failures);
    return 1;
  }
  std::printf("host checks passed\n");
  return 0;
}
