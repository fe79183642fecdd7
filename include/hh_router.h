/* hh_router.h — host-side serving steps either side of the decoder.
 *
 * The paper's runtime phase (§4 "Runtime phase") maps a question to a stored
 * entry with a lexical router, renders the entry's answer deterministically,
 * and has the small decoder speak it.  §6.3 measures BM25 routing over a
 * naive scan of the store and gates low-confidence routes on the score
 * margin over the runner-up (threshold tau = 0.05); §6.4 finds that a bare
 * answer line after a structural marker is the envelope the small model
 * repeats verbatim.  These calls implement those steps on the host CPU; they
 * touch no GPU and need no hh_ctx.
 *
 * Conventions: every function returns an hh_status (include/hh.h); on an
 * error nothing is written to the outputs except where stated, and a router
 * is unchanged.  Strings are NUL-terminated byte strings (UTF-8 or ASCII).
 * A router is immutable after hh_router_create: queries from several host
 * threads at once are safe.
 */
#ifndef HH_ROUTER_H_
#define HH_ROUTER_H_

#include <stdint.h>

#include "hh.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct hh_router hh_router;

/* Terms of a text: maximal runs of ASCII letters and digits, or bytes >= 0x80
 * (so UTF-8 words stay whole), with ASCII letters lower-cased; everything
 * else separates terms.  The same rule splits entries and queries. */

/* Index n_entries texts (host strings, copied; entry i is id i) for Okapi
 * BM25 with parameters k1 >= 0 and 0 <= b <= 1 (§6.3 names BM25; the paper
 * gives no parameters, the usual choice is k1 = 1.2, b = 0.75).
 *   score(q, d) = sum over query terms t (repeats counted) of
 *                 idf(t) * tf(t,d) (k1 + 1) / (tf(t,d) + k1 (1 - b + b |d| / avgdl))
 *   idf(t)      = ln(1 + (N - n(t) + 0.5) / (n(t) + 0.5))
 * with N entries, n(t) entries containing t, |d| the term count of entry d
 * and avgdl its mean.  Terms absent from every entry score 0.
 * Errors: HH_ERR_INVALID_ARG for n_entries < 1, a NULL pointer, k1 < 0,
 * b outside [0, 1], or a store with no terms at all.  *out is set only on
 * success; free it with hh_router_destroy. */
hh_status hh_router_create(const char* const* entries, int32_t n_entries, float k1, float b, hh_router** out);

/* Score every entry against `query` (a linear pass over the store's term
 * postings) and return the k best: ids[0..*n_out) and their scores in
 * descending score order, ties to the lower id; *n_out = min(k, n_entries).
 * ids and scores are host arrays of at least k elements.
 * Errors: HH_ERR_INVALID_ARG for a NULL pointer or k < 1. */
hh_status hh_router_query(const hh_router* r, const char* query, int32_t k, int32_t* ids, double* scores,
                          int32_t* n_out);

/* Route with the margin gate: *entry = the best entry, *margin =
 * (s1 - s2) / s1 for the best and runner-up scores (s2 = 0 with a single
 * entry; margin 0 when s1 <= 0, i.e. no query term matched), *escalate = 1
 * when margin < tau (the route is not trusted and the query goes elsewhere),
 * else 0.  The paper's threshold is tau = 0.05 (§6.3).
 * Errors: HH_ERR_INVALID_ARG for a NULL pointer or tau that is NaN. */
hh_status hh_router_route(const hh_router* r, const char* query, float tau, int32_t* entry, double* margin,
                          int32_t* escalate);

/* Number of entries and of distinct terms indexed. */
hh_status hh_router_size(const hh_router* r, int32_t* n_entries, int32_t* n_terms);

void hh_router_destroy(hh_router* r);

/* Marker-line envelope (§6.4): the decoder's prompt for a locked answer is
 *   "Repeat the line after the marker exactly.\n### ANSWER\n" + line + "\n"
 * where line is `answer` with every CR or LF replaced by a space, so the
 * answer is one bare line after the marker.  Writes the prompt (without a
 * NUL) to out[0..*n_out) when it fits in cap bytes; otherwise writes nothing,
 * sets *n_out to the size needed and returns HH_ERR_INVALID_ARG, as it does
 * for NULL answer or n_out (out may be NULL when cap is 0). */
hh_status hh_render_marker(const char* answer, char* out, int64_t cap, int64_t* n_out);

#ifdef __cplusplus
}
#endif

#endif /* HH_ROUTER_H_ */
