// Host-side router and renderer: Okapi BM25 over the store's entries with the
// margin gate, and the marker-line answer envelope (declared in hh_router.h).
#include "hh_router.h"

#include <algorithm>
#include <cmath>
#include <cstring>
#include <new>
#include <string>
#include <unordered_map>
#include <utility>
#include <vector>

struct hh_router {
  int32_t n_docs = 0;
  double k1 = 0.0, b = 0.0, avgdl = 0.0;
  std::unordered_map<std::string, int32_t> vocab;
  std::vector<double> idf;                                  // per term
  std::vector<std::vector<std::pair<int32_t, int32_t>>> postings;  // per term: (entry, tf), entries ascending
  std::vector<double> norm;                                 // per entry: k1 (1 - b + b |d| / avgdl)
};

namespace {

// Calls f(term) for each term of s (see hh_router.h for the rule).
template <class F>
void for_each_term(const char* s, F&& f) {
  std::string cur;
  for (const unsigned char* p = reinterpret_cast<const unsigned char*>(s);; ++p) {
    const unsigned char c = *p;
    const bool word = (c >= 'a' && c <= 'z') || (c >= '0' && c <= '9') || (c >= 'A' && c <= 'Z') || c >= 0x80;
    if (word) {
      cur.push_back(c >= 'A' && c <= 'Z' ? static_cast<char>(c - 'A' + 'a') : static_cast<char>(c));
    } else if (!cur.empty()) {
      f(cur);
      cur.clear();
    }
    if (c == 0) break;
  }
}

// BM25 scores of every entry for `query`, summed in query-term order.
void score_all(const hh_router* r, const char* query, std::vector<double>& sc) {
  sc.assign(r->n_docs, 0.0);
  const double k1p = r->k1 + 1.0;
  for_each_term(query, [&](const std::string& t) {
    const auto it = r->vocab.find(t);
    if (it == r->vocab.end()) return;
    const double w = r->idf[it->second];
    for (const auto& [d, tf] : r->postings[it->second]) sc[d] += w * (tf * k1p) / (tf + r->norm[d]);
  });
}

bool better(const std::vector<double>& sc, int32_t i, int32_t j) {
  return sc[i] > sc[j] || (sc[i] == sc[j] && i < j);
}

}  // namespace

extern "C" {

hh_status hh_router_create(const char* const* entries, int32_t n_entries, float k1, float b, hh_router** out) {
  if (!entries || !out || n_entries < 1 || !(k1 >= 0.f) || !(b >= 0.f && b <= 1.f)) return HH_ERR_INVALID_ARG;
  for (int32_t i = 0; i < n_entries; ++i)
    if (!entries[i]) return HH_ERR_INVALID_ARG;
  hh_router* r = new (std::nothrow) hh_router;
  if (!r) return HH_ERR_OOM;
  try {
    r->n_docs = n_entries;
    r->k1 = k1;
    r->b = b;
    std::vector<int64_t> len(n_entries, 0);
    int64_t total = 0;
    for (int32_t d = 0; d < n_entries; ++d) {
      std::unordered_map<int32_t, int32_t> tf;
      for_each_term(entries[d], [&](const std::string& t) {
        auto it = r->vocab.find(t);
        if (it == r->vocab.end()) {
          it = r->vocab.emplace(t, static_cast<int32_t>(r->postings.size())).first;
          r->postings.emplace_back();
        }
        ++tf[it->second];
        ++len[d];
      });
      for (const auto& [t, c] : tf) r->postings[t].emplace_back(d, c);
      total += len[d];
    }
    if (total == 0) {
      delete r;
      return HH_ERR_INVALID_ARG;
    }
    r->avgdl = static_cast<double>(total) / n_entries;
    const double N = n_entries;
    r->idf.resize(r->postings.size());
    for (size_t t = 0; t < r->postings.size(); ++t) {
      const double n = static_cast<double>(r->postings[t].size());
      r->idf[t] = std::log(1.0 + (N - n + 0.5) / (n + 0.5));
    }
    r->norm.resize(n_entries);
    for (int32_t d = 0; d < n_entries; ++d)
      r->norm[d] = r->k1 * (1.0 - r->b + r->b * static_cast<double>(len[d]) / r->avgdl);
  } catch (const std::bad_alloc&) {
    delete r;
    return HH_ERR_OOM;
  }
  *out = r;
  return HH_OK;
}

hh_status hh_router_query(const hh_router* r, const char* query, int32_t k, int32_t* ids, double* scores,
                          int32_t* n_out) {
  if (!r || !query || !ids || !scores || !n_out || k < 1) return HH_ERR_INVALID_ARG;
  std::vector<double> sc;
  std::vector<int32_t> order(r->n_docs);
  try {
    score_all(r, query, sc);
    for (int32_t i = 0; i < r->n_docs; ++i) order[i] = i;
  } catch (const std::bad_alloc&) {
    return HH_ERR_OOM;
  }
  const int32_t m = std::min(k, r->n_docs);
  std::partial_sort(order.begin(), order.begin() + m, order.end(),
                    [&](int32_t i, int32_t j) { return better(sc, i, j); });
  for (int32_t i = 0; i < m; ++i) {
    ids[i] = order[i];
    scores[i] = sc[order[i]];
  }
  *n_out = m;
  return HH_OK;
}

hh_status hh_router_route(const hh_router* r, const char* query, float tau, int32_t* entry, double* margin,
                          int32_t* escalate) {
  if (!r || !query || !entry || !margin || !escalate || std::isnan(tau)) return HH_ERR_INVALID_ARG;
  int32_t ids[2];
  double s[2] = {0.0, 0.0};
  int32_t n = 0;
  const hh_status st = hh_router_query(r, query, 2, ids, s, &n);
  if (st != HH_OK) return st;
  const double s1 = s[0], s2 = n > 1 ? s[1] : 0.0;
  const double m = s1 > 0.0 ? (s1 - s2) / s1 : 0.0;
  *entry = ids[0];
  *margin = m;
  *escalate = m < static_cast<double>(tau) ? 1 : 0;
  return HH_OK;
}

hh_status hh_router_size(const hh_router* r, int32_t* n_entries, int32_t* n_terms) {
  if (!r || !n_entries || !n_terms) return HH_ERR_INVALID_ARG;
  *n_entries = r->n_docs;
  *n_terms = static_cast<int32_t>(r->postings.size());
  return HH_OK;
}

void hh_router_destroy(hh_router* r) { delete r; }

hh_status hh_render_marker(const char* answer, char* out, int64_t cap, int64_t* n_out) {
  static const char kHead[] = "Repeat the line after the marker exactly.\n### ANSWER\n";
  if (!answer || !n_out) return HH_ERR_INVALID_ARG;
  const int64_t head = static_cast<int64_t>(sizeof(kHead) - 1);
  const int64_t body = static_cast<int64_t>(std::strlen(answer));
  const int64_t need = head + body + 1;
  *n_out = need;
  if (!out || cap < need) return HH_ERR_INVALID_ARG;
  std::memcpy(out, kHead, head);
  for (int64_t i = 0; i < body; ++i) out[head + i] = (answer[i] == '\n' || answer[i] == '\r') ? ' ' : answer[i];
  out[head + body] = '\n';
  return HH_OK;
}

}  // extern "C"
