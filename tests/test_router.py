"""Router and renderer around the decoder (CPU only): the fp64 oracle against
worked examples and properties of BM25, then the native library against the
oracle on a synthetic store, and the marker-line envelope."""
import math

import numpy as np
import pytest

import synth
from oracle import router as orc
from paper_2606_12154_amd import hh, serve


# ---------------------------------------------------------------- oracle pins

def test_tokenizer_rule():
    assert orc.terms("Hello, WORLD! x2 café-au_lait") == ["hello", "world", "x2", "café", "au", "lait"]
    assert orc.terms("  --  ") == []


def test_worked_example_three_entries():
    # N = 3, |d| = 6, 5, 4, avgdl = 5.  "cat" is in two entries:
    # idf = ln(1 + 1.5 / 2.5) = ln 1.6; "mat" in one: ln(1 + 2.5 / 1.5) = ln(8/3).
    # Entry 0: K = 1.2 (0.25 + 0.75 * 6/5) = 1.38, each term tf 1: 2.2 / 2.38.
    # Entry 1: K = 1.2, so "cat" scores its idf exactly.
    store = ["the cat sat on the mat", "a dog and a cat", "fish swim in water"]
    s = orc.bm25_scores(store, "cat mat")
    assert s[0] == pytest.approx((math.log(1.6) + math.log(8 / 3)) * 2.2 / 2.38, rel=1e-14)
    assert s[1] == pytest.approx(math.log(1.6), rel=1e-14)
    assert s[2] == 0.0
    assert s[0] == pytest.approx(1.3411060, abs=1e-7)


def test_worked_example_saturation_without_length_norm():
    # b = 0, k1 = 2: "x" twice in entry 0, idf ln 2, score 2 * 3 / (2 + 2) * ln 2.
    s = orc.bm25_scores(["x x y", "y z"], "x", k1=2.0, b=0.0)
    assert s == [pytest.approx(1.5 * math.log(2), rel=1e-14), 0.0]


def test_single_entry_closed_form():
    # N = n = 1: idf = ln(4/3); tf = 1 and |d| = avgdl, so the tf factor is 1.
    assert orc.bm25_scores(["a b"], "a") == [pytest.approx(math.log(4 / 3), rel=1e-14)]


def test_term_frequency_saturates():
    k1 = 1.2
    store = [" ".join(["t"] * n + ["pad"] * (60 - n)) for n in range(1, 51)] + ["other words only"]
    s = orc.bm25_scores(store, "t", k1=k1, b=0.0)
    idf = orc.bm25_scores(["t", "u"], "t", k1=0.0, b=0.0)[0]  # k1 = 0: the idf of a term in 1 of 2
    assert all(a < c for a, c in zip(s[:49], s[1:50]))
    n_t = 50
    bound = math.log(1 + (51 - n_t + 0.5) / (n_t + 0.5)) * (k1 + 1)
    assert s[49] < bound and s[49] > 0.9 * bound
    assert idf == pytest.approx(math.log(1 + 1.5 / 1.5), rel=1e-14)


def test_b_zero_ignores_length_and_b_one_penalises_it():
    store = ["k filler", "k " + "filler " * 30, "none here"]
    s0 = orc.bm25_scores(store, "k", b=0.0)
    assert s0[0] == pytest.approx(s0[1], rel=1e-14)
    s1 = orc.bm25_scores(store, "k", b=1.0)
    assert s1[0] > s1[1] > 0


def test_k1_zero_is_binary_matching():
    store = ["p p p q", "p r", "s t", "q"]
    s = orc.bm25_scores(store, "p q", k1=0.0)
    idf_p = math.log(1 + (4 - 2 + 0.5) / 2.5)
    idf_q = math.log(1 + (4 - 2 + 0.5) / 2.5)
    assert s == [pytest.approx(idf_p + idf_q), pytest.approx(idf_p), 0.0, pytest.approx(idf_q)]


def test_common_term_weighs_least_and_stays_positive():
    store = ["common rare1", "common rare2 x", "common y z"]
    s_common = orc.bm25_scores(store, "common")
    s_rare = orc.bm25_scores(store, "rare1")
    assert all(v > 0 for v in s_common)
    assert s_rare[0] > s_common[0]


def test_query_repeats_and_unseen_terms():
    store = ["alpha beta", "beta gamma delta", "alpha alpha"]
    one = orc.bm25_scores(store, "alpha")
    two = orc.bm25_scores(store, "alpha ALPHA")
    assert two == [pytest.approx(2 * v, rel=1e-14) for v in one]
    assert orc.bm25_scores(store, "unseen words") == [0.0, 0.0, 0.0]
    assert orc.bm25_scores(store, "alpha unseen") == one


def test_store_permutation_permutes_scores():
    store = [t for t, _ in synth.make_store(40, 4, seed=3)]
    q = " ".join(store[7].split()[:5])
    s = orc.bm25_scores(store, q)
    perm = np.random.default_rng(0).permutation(len(store))
    sp = orc.bm25_scores([store[i] for i in perm], q)
    assert sp == [pytest.approx(s[i], rel=1e-12) for i in perm]


def test_margin_gate_cases():
    # Two identical entries tie: margin 0, escalated, lower id first.
    assert orc.route(["same words", "same words", "else"], "same") == (0, 0.0, True)
    e, m, esc = orc.route(["cat sat", "dog ran", "bird flew"], "cat")
    assert (e, esc) == (0, False) and m == pytest.approx(1.0)
    assert orc.route(["a b", "c d"], "zzz") == (0, 0.0, True)


# ---------------------------------------------------------------- native vs oracle

@pytest.mark.parametrize("k1,b", [(1.2, 0.75), (0.9, 0.4), (2.0, 1.0)])
def test_native_scores_and_ranks_match_oracle(k1, b):
    store = synth.make_store(150, 6, seed=11)
    texts = [t for t, _ in store]
    queries = synth.make_queries(store, 1, seed=12)[::3]
    r = hh.hh_router_create(texts, k1, b)
    k1, b = float(np.float32(k1)), float(np.float32(b))  # the library takes k1 and b as fp32
    try:
        assert hh.hh_router_size(r)[0] == 150
        for q, _ in queries:
            ref = orc.bm25_scores(texts, q, k1, b)
            ids, sc = hh.hh_router_query(r, q, 5)
            assert list(ids) == orc.rank(ref, 5)
            np.testing.assert_allclose(sc, [ref[i] for i in ids], rtol=1e-12, atol=0)
            e, m, esc = hh.hh_router_route(r, q, 0.05)
            oe, om, oesc = orc.route(texts, q, 0.05, k1, b)
            assert (e, esc) == (oe, oesc) and m == pytest.approx(om, rel=1e-10, abs=1e-14)
    finally:
        hh.hh_router_destroy(r)


def test_native_ties_empty_matches_and_utf8():
    r = hh.hh_router_create(["same words", "same words", "Café au lait"])
    try:
        ids, sc = hh.hh_router_query(r, "same", 3)
        assert list(ids) == [0, 1, 2] and sc[0] == sc[1] and sc[2] == 0.0
        assert hh.hh_router_route(r, "nothing matches") == (0, 0.0, True)
        ids, sc = hh.hh_router_query(r, "CAFÉ", 1)  # non-ASCII bytes are not case-folded
        assert sc[0] == 0.0
        ids, sc = hh.hh_router_query(r, "café", 1)
        assert ids[0] == 2 and sc[0] > 0
        ids, _ = hh.hh_router_query(r, "same", 10)
        assert len(ids) == 3
    finally:
        hh.hh_router_destroy(r)


def test_native_rejects_bad_arguments():
    for entries, k1, b in [([], 1.2, 0.75), (["a"], -1.0, 0.75), (["a"], 1.2, 1.5), (["a"], 1.2, float("nan")),
                           (["--", "!!"], 1.2, 0.75)]:
        with pytest.raises(hh.HHError) as e:
            hh.hh_router_create(entries, k1, b)
        assert e.value.status == hh.HH_ERR_INVALID_ARG
    r = hh.hh_router_create(["a b"])
    try:
        with pytest.raises(hh.HHError):
            hh.hh_router_query(r, "a", 0)
        with pytest.raises(hh.HHError):
            hh.hh_router_route(r, "a", float("nan"))
    finally:
        hh.hh_router_destroy(r)


# ---------------------------------------------------------------- envelope

def test_marker_envelope_golden_and_native():
    got = hh.hh_render_marker("Tais vean is 8979\nas of 1990.\r")
    want = b"Repeat the line after the marker exactly.\n### ANSWER\nTais vean is 8979 as of 1990. \n"
    assert got == want
    assert orc.render_marker("Tais vean is 8979\nas of 1990.\r").encode() == want
    for _, ans in synth.make_store(30, 3, seed=5):
        assert hh.hh_render_marker(ans) == orc.render_marker(ans).encode()


def test_byte_tokens_round_trip():
    p = hh.hh_render_marker("x")
    ids = serve.byte_tokens(p)
    assert ids.dtype == np.int32 and ids.min() >= 3 and ids.max() <= 258
    assert bytes((ids - 3).astype(np.uint8)) == p
