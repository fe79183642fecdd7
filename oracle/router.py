"""Oracle for the serving steps around the decoder.  TEST INFRASTRUCTURE ONLY.

Plain fp64 Python for the lexical router and the answer envelope of the
paper's runtime phase (Sec. 4 "Runtime phase"): BM25 routing over a naive
scan of the store, the score-margin confidence gate with threshold 0.05
(Sec. 6.3), and the marker-line envelope, a bare answer line after a
structural marker (Sec. 6.4).  Only ``tests/`` may import it.

BM25 is the Okapi weighting of Robertson et al. (TREC-3, 1994) with the
non-negative inverse document frequency ln(1 + (N - n + 0.5) / (n + 0.5))
used by Lucene; the paper names BM25 but gives no parameters, so k1 and b
are arguments (1.2 and 0.75 by default).  Readings where the paper is
silent: terms are runs of ASCII letters/digits (lower-cased) or of bytes
>= 0x80; a query's repeated terms count once per occurrence; ties rank the
lower entry first; the margin is relative, (s1 - s2) / s1, 0 when nothing
matched; the envelope's wording is fixed here.

Pins (``tests/test_router.py``): worked examples computed by hand, the
single-entry closed form, saturation in term frequency, b = 0 (no length
normalisation), k1 = 0 (binary matching), a term present everywhere, query
repeats, unseen terms, permutation of the store, and the tokenizer on
mixed text.
"""
from __future__ import annotations

import math
from typing import Dict, List, Sequence, Tuple


def terms(text) -> List[str]:
    """Terms of a text (bytes or str, str taken as UTF-8)."""
    raw = text.encode() if isinstance(text, str) else bytes(text)
    out: List[str] = []
    cur = bytearray()
    for c in raw:
        if 0x30 <= c <= 0x39 or 0x61 <= c <= 0x7A or c >= 0x80:
            cur.append(c)
        elif 0x41 <= c <= 0x5A:
            cur.append(c + 0x20)
        elif cur:
            out.append(cur.decode("utf-8", "replace"))
            cur = bytearray()
    if cur:
        out.append(cur.decode("utf-8", "replace"))
    return out


def bm25_scores(entries: Sequence, query, k1: float = 1.2, b: float = 0.75) -> List[float]:
    """BM25 score of every entry for the query, in entry order."""
    docs = [terms(e) for e in entries]
    N = len(docs)
    avgdl = sum(len(d) for d in docs) / N
    df: Dict[str, int] = {}
    for d in docs:
        for t in set(d):
            df[t] = df.get(t, 0) + 1
    scores = []
    for d in docs:
        tf: Dict[str, int] = {}
        for t in d:
            tf[t] = tf.get(t, 0) + 1
        s = 0.0
        for t in terms(query):
            f = tf.get(t, 0)
            if f == 0:  # a term absent from the entry adds nothing
                continue
            idf = math.log(1.0 + (N - df[t] + 0.5) / (df[t] + 0.5))
            s += idf * (f * (k1 + 1.0)) / (f + k1 * (1.0 - b + b * len(d) / avgdl))
        scores.append(s)
    return scores


def rank(scores: Sequence[float], k: int) -> List[int]:
    """The k best entry ids, descending score, ties to the lower id."""
    order = sorted(range(len(scores)), key=lambda i: (-scores[i], i))
    return order[:k]


def route(entries: Sequence, query, tau: float = 0.05, k1: float = 1.2, b: float = 0.75) -> Tuple[int, float, bool]:
    """(best entry, relative margin over the runner-up, escalate?)."""
    s = bm25_scores(entries, query, k1, b)
    top = rank(s, 2)
    s1 = s[top[0]]
    s2 = s[top[1]] if len(top) > 1 else 0.0
    margin = (s1 - s2) / s1 if s1 > 0 else 0.0
    return top[0], margin, margin < tau


def render_marker(answer: str) -> str:
    """The marker-line prompt for a locked answer: one bare line after the marker."""
    line = answer.replace("\r", " ").replace("\n", " ")
    return "Repeat the line after the marker exactly.\n### ANSWER\n" + line + "\n"
