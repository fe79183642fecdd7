"""The serving path on the GPU (tiny fp32 decoder): route, render, stream.
The streamed ids are the device's greedy sequence (its argmax history), the
oracle's greedy continuation of the rendered prompt up to the first near-tie,
and an escalated query decodes nothing."""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import new_context, top2_margin
from oracle import router as orc
from paper_2606_12154_amd import hh, serve

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def tiny_server():
    shape = synth.TINY
    tensors = synth.make_weights(shape, 0, gain_std=0.1)
    model = oracle.Decoder(shape, synth.weights_as_f64(shape, tensors))
    store = synth.make_store(60, 4, seed=21)
    ctx = new_context(shape, tensors, streams=5, context=256)
    router = serve.Router([t for t, _ in store])
    srv = serve.Server(ctx, router, [a for _, a in store], max_tokens=32, stream_id=4, max_batch=4)
    yield shape, model, store, ctx, srv
    router.close()
    ctx.close()


def check_greedy(model, prompt, tokens, what):
    """The oracle's greedy continuation, compared up to its first near-tie."""
    logits, cache = model.prefill(prompt, rows="last")
    row = logits[0]
    for i, tok in enumerate(tokens):
        if top2_margin(row) <= 1e-2:
            break
        assert tok == int(np.argmax(row)), f"token {i} of {what!r}"
        row = model.decode(cache, tok)


def test_streamed_tokens_are_the_greedy_sequence(tiny_server):
    shape, model, store, ctx, srv = tiny_server
    queries = synth.make_queries(store, 1, seed=22)
    served = 0
    for q, want in queries[:12]:
        e, m, esc = orc.route([t for t, _ in store], q)
        a = srv.answer(q, 24)
        assert (a.entry, a.escalated) == (e, esc)
        if esc:
            assert a.tokens == []
            continue
        served += 1
        prompt = serve.byte_tokens(orc.render_marker(store[e][1]).encode())
        assert a.prompt_tokens == len(prompt)
        assert len(a.tokens) == 24
        hist = ctx.read_argmax(4, len(prompt) - 1, 24)
        assert list(hist) == a.tokens
        assert 0 < a.t_route <= a.t_render <= a.t_first <= a.t_last
        check_greedy(model, prompt, a.tokens, q)
    assert served >= 8
    print(f"served {served} of 12 queries")


def test_escalated_query_decodes_nothing(tiny_server):
    shape, model, store, ctx, srv = tiny_server
    before = ctx.length(4)
    a = srv.answer("zzzz qqqq", 8)
    assert a.escalated and a.margin == 0.0 and a.tokens == []
    assert ctx.length(4) == before
    with pytest.raises(ValueError):
        srv.answer(synth.make_queries(store, 1, seed=22)[0][0], 33)


def test_batch_of_requests_in_lockstep(tiny_server):
    shape, model, store, ctx, srv = tiny_server
    texts = [t for t, _ in store]
    queries = [q for q, _ in synth.make_queries(store, 2, seed=23) if not orc.route(texts, q)[2]][:4]
    queries.insert(2, "zzzz qqqq")  # escalated: takes no stream
    answers = srv.answer_batch(queries[:4], 16, streams=[0, 1, 2, 3])
    assert [a.escalated for a in answers] == [False, False, True, False]
    for s, (q, a) in enumerate(zip(queries[:4], answers)):
        if a.escalated:
            assert a.tokens == []
            continue
        prompt = serve.byte_tokens(orc.render_marker(store[a.entry][1]).encode())
        assert a.entry == orc.route(texts, q)[0] and a.prompt_tokens == len(prompt)
        assert len(a.tokens) == 16
        assert list(ctx.read_argmax(s, len(prompt) - 1, 16)) == a.tokens
        check_greedy(model, prompt, a.tokens, q)
        assert 0 < a.t_first <= a.t_last
    with pytest.raises(ValueError):
        srv.answer_batch(queries[:2], 4, streams=[0])


def test_batch_prompts_longer_than_a_pass(tiny_server):
    """Rendered prompts longer than one prefill pass (max_prefill 32 rows):
    the batch prefill continues each prompt in the next pass, and every
    stream still decodes the oracle's greedy continuation."""
    shape, model, store, _, _ = tiny_server
    tensors = synth.make_weights(shape, 0, gain_std=0.1)
    ctx = new_context(shape, tensors, streams=4, context=256, max_prefill=32)
    router = serve.Router([t for t, _ in store])
    try:
        srv = serve.Server(ctx, router, [a for _, a in store], max_tokens=12, max_batch=3)
        texts = [t for t, _ in store]
        queries = [q for q, _ in synth.make_queries(store, 2, seed=24) if not orc.route(texts, q)[2]][:3]
        answers = srv.answer_batch(queries, 12, streams=[2, 0, 3])
        for s, (q, a) in zip([2, 0, 3], zip(queries, answers)):
            prompt = serve.byte_tokens(orc.render_marker(store[a.entry][1]).encode())
            assert len(prompt) > 32
            assert len(a.tokens) == 12
            assert list(ctx.read_argmax(s, len(prompt) - 1, 12)) == a.tokens
            check_greedy(model, prompt, a.tokens, q)
    finally:
        router.close()
        ctx.close()
