"""GPU parity on the tiny fp32 decoder (2 layers, d 256, 4/2 heads, FFN 688,
vocab 4096): every path against the fp64 oracle at max-abs 1e-4, argmax equal
where the oracle's top-2 margin exceeds 1e-2.  Sizes span several GEMM tiles,
ragged tails (FFN 688 is not a multiple of 64), several KV pages and
attention splits."""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import check_logits, new_context, top2_margin

pytestmark = pytest.mark.gpu
TOL = 1e-4


@pytest.fixture(scope="module")
def tiny():
    shape = synth.TINY
    # Random RMSNorm gains catch a dropped or mis-indexed gain multiply.
    tensors = synth.make_weights(shape, 0, gain_std=0.1)
    model = oracle.Decoder(shape, synth.weights_as_f64(shape, tensors))
    return shape, tensors, model


def oracle_greedy(model, prompt, steps):
    """Oracle greedy continuation: (tokens, logits per step incl. prompt-last)."""
    logits, cache = model.prefill(prompt, rows="last")
    rows = [logits[0]]
    toks = [int(np.argmax(logits[0]))]
    for _ in range(steps):
        rows.append(model.decode(cache, toks[-1]))
        toks.append(int(np.argmax(rows[-1])))
    return np.array(toks), np.array(rows)


def test_prefill_all_logits(tiny):
    shape, tensors, model = tiny
    toks = synth.make_tokens(shape.vocab, 64, 1)
    ref, _ = model.prefill(toks)
    ctx = new_context(shape, tensors)
    nxt, got = ctx.prefill(0, toks, logits="all")
    check_logits(got, ref, TOL, what="prefill all")
    assert nxt == int(np.argmax(ref[-1]))
    assert ctx.length(0) == 64


def test_decode_teacher_forced(tiny):
    shape, tensors, model = tiny
    prompt = synth.make_tokens(shape.vocab, 64, 1)
    toks, ref = oracle_greedy(model, prompt, 32)
    ctx = new_context(shape, tensors)
    nxt, last = ctx.prefill(0, prompt, logits="last")
    check_logits(last, ref[0], TOL, what="prefill last")
    for i in range(32):
        nxt, lg = ctx.decode_step([0], [int(toks[i])], logits=True)
        check_logits(lg[0], ref[i + 1], TOL, what=f"decode step {i}")
        assert nxt[0] == int(np.argmax(lg[0]))
    assert ctx.length(0) == 96


def test_decode_free_running_device_feedback(tiny):
    shape, tensors, model = tiny
    prompt = synth.make_tokens(shape.vocab, 64, 1)
    toks, ref = oracle_greedy(model, prompt, 32)
    margins = np.sort(ref, axis=-1)
    margins = margins[:, -1] - margins[:, -2]
    ctx = new_context(shape, tensors)
    ctx.prefill(0, prompt)
    for _ in range(32):
        ctx.decode_step([0], None, host_next=False)
    got = ctx.read_argmax(0, 63, 33)
    # Free-running sequences may part after a near-tie; compare up to the first.
    n_cmp = 33
    near = np.nonzero(margins < 1e-3)[0]
    if near.size:
        n_cmp = int(near[0]) + 1
    assert np.array_equal(got[:n_cmp], toks[:n_cmp])


def test_multistream_lockstep(tiny):
    """Streams of different lengths decoded together (the MFMA GEMM path)
    equal each stream run alone through the oracle."""
    shape, tensors, model = tiny
    lens = [5, 17, 40, 64]
    prompts = [synth.make_tokens(shape.vocab, n, 100 + i) for i, n in enumerate(lens)]
    ctx = new_context(shape, tensors, streams=6)
    caches = []
    for i, p in enumerate(prompts):
        ctx.prefill(i + 1, p)  # streams 1..4
        caches.append(model.prefill(p, rows="last")[1])
    rng = np.random.default_rng(7)
    ids = [3, 1, 4, 2]
    for step in range(6):
        feed = rng.integers(0, shape.vocab, size=4).astype(np.int32)
        nxt, lg = ctx.decode_step(ids, feed, logits=True)
        for k, s in enumerate(ids):
            ref = model.decode(caches[s - 1], int(feed[k]))
            check_logits(lg[k], ref, TOL, what=f"step {step} stream {s}")
    for s, n in zip(range(1, 5), lens):
        assert ctx.length(s) == n + 6


def test_prefill_between_lockstep_steps(tiny):
    """A prefill into another stream between two decode steps over the same
    stream list: the prefill's rows reuse the row-stream table, so the second
    step must not take the table for still uploaded (regression)."""
    shape, tensors, model = tiny
    ctx = new_context(shape, tensors, streams=6)
    ids = [0, 1, 2]
    caches = []
    for s in ids:
        p = synth.make_tokens(shape.vocab, 9 + 5 * s, 200 + s)
        ctx.prefill(s, p)
        caches.append(model.prefill(p, rows="last")[1])
    rng = np.random.default_rng(8)
    for step in range(3):
        if step == 1:
            ctx.prefill(5, synth.make_tokens(shape.vocab, 12, 299))  # rows 0..11 name stream 5
        feed = rng.integers(0, shape.vocab, size=3).astype(np.int32)
        _, lg = ctx.decode_step(ids, feed, logits=True)
        for k, s in enumerate(ids):
            check_logits(lg[k], model.decode(caches[s], int(feed[k])), TOL, what=f"step {step} stream {s}")
    assert [ctx.length(s) for s in ids] == [9 + 5 * s + 3 for s in ids]
    assert ctx.length(5) == 12


def test_prefill_batch_matches_oracle(tiny):
    """Several streams' prompts in one call (ragged, one of a single token,
    one appended to a stream that already holds tokens, one of 230 tokens
    whose rows attend over 15 pages; 331 rows, so the 256-row passes split
    the last prompt): each stream's next token and the KV it leaves (checked
    by a lockstep decode step) equal the oracle's run of that stream alone."""
    shape, tensors, model = tiny
    ctx = new_context(shape, tensors, streams=6)
    head = synth.make_tokens(shape.vocab, 10, 310)
    ctx.prefill(2, head)
    lens = {0: 1, 2: 7, 3: 93, 5: 230}
    prompts = {s: synth.make_tokens(shape.vocab, n, 320 + s) for s, n in lens.items()}
    ids = [3, 0, 5, 2]
    nxt = ctx.prefill_batch(ids, [prompts[s] for s in ids])
    caches, rows = {}, {}
    for s in ids:
        full = np.concatenate([head, prompts[s]]) if s == 2 else prompts[s]
        logits, caches[s] = model.prefill(full, rows="last")
        rows[s] = logits[0]
    for k, s in enumerate(ids):
        if top2_margin(rows[s]) > 1e-2:
            assert int(nxt[k]) == int(np.argmax(rows[s])), f"stream {s}"
        assert ctx.length(s) == lens[s] + (10 if s == 2 else 0)
    feed = np.array([11, 22, 33, 44], dtype=np.int32)
    _, lg = ctx.decode_step(ids, feed, logits=True)
    for k, s in enumerate(ids):
        check_logits(lg[k], model.decode(caches[s], int(feed[k])), TOL, what=f"after batch prefill, stream {s}")
    from paper_2606_12154_amd import hh
    for bad_ids, bad_prompts in [([1, 1], [[5], [6]]), ([1], [[]]), ([1, 4], [[1] * 3, [4096]])]:
        with pytest.raises(hh.HHError) as e:
            ctx.prefill_batch(bad_ids, bad_prompts)
        assert e.value.status == hh.HH_ERR_INVALID_ARG
    assert ctx.length(1) == 0 and ctx.length(4) == 0


def test_long_rows_lockstep_and_batch(tiny):
    """Rows longer than the pages the row attention keeps in registers up
    front (three per wave for an fp32 cache: 24 pages, 384 positions) take
    its online page loop: a 450-token stream decoded in lockstep with a short
    one, and a 420-token prompt in a batch prefill (rows past 384 attend
    with the same loop), against the oracle run of each stream alone."""
    shape, tensors, model = tiny
    ctx = new_context(shape, tensors, streams=3, context=640)
    try:
        lens = [450, 20]
        prompts = [synth.make_tokens(shape.vocab, n, 500 + i) for i, n in enumerate(lens)]
        caches = []
        for i, p in enumerate(prompts):
            ctx.prefill(i, p)
            caches.append(model.prefill(p, rows="last")[1])
        rng = np.random.default_rng(9)
        for step in range(3):
            feed = rng.integers(0, shape.vocab, size=2).astype(np.int32)
            _, lg = ctx.decode_step([0, 1], feed, logits=True)
            for k in range(2):
                check_logits(lg[k], model.decode(caches[k], int(feed[k])), TOL, what=f"long rows step {step} row {k}")
        long_prompt = synth.make_tokens(shape.vocab, 420, 510)
        nxt = ctx.prefill_batch([2], [long_prompt])
        ref, cache2 = model.prefill(long_prompt, rows="last")
        if top2_margin(ref[0]) > 1e-2:
            assert int(nxt[0]) == int(np.argmax(ref[0]))
        _, lg = ctx.decode_step([2], [7], logits=True)
        check_logits(lg[0], model.decode(cache2, 7), TOL, what="after a 420-token batch prefill")
    finally:
        ctx.close()


def test_chunked_and_appended_prefill(tiny):
    shape, tensors, model = tiny
    toks = synth.make_tokens(shape.vocab, 70, 3)
    ref, _ = model.prefill(toks)
    ctx = new_context(shape, tensors, max_prefill=16)   # 70 rows in 5 passes
    _, got = ctx.prefill(0, toks, logits="all")
    check_logits(got, ref, TOL, what="chunked")
    ctx2 = new_context(shape, tensors)
    _, a = ctx2.prefill(2, toks[:29], logits="all")
    _, b = ctx2.prefill(2, toks[29:], logits="all")
    check_logits(np.concatenate([a, b]), ref, TOL, what="appended")


def test_long_context_many_splits(tiny):
    """A prompt of 1500 positions: decode attention over 94 pages uses the
    maximum split count with several pages per split."""
    shape, tensors, model = tiny
    toks = synth.make_tokens(shape.vocab, 1500, 4)
    ctx = new_context(shape, tensors, streams=1, context=1600, max_prefill=512)
    _, cache = model.prefill(toks[:-4], rows="last")
    ctx.prefill(0, toks[:-4])
    for t in toks[-4:]:
        _, lg = ctx.decode_step([0], [int(t)], logits=True)
        check_logits(lg[0], model.decode(cache, int(t)), TOL, what="long decode")


def test_reset_and_errors(tiny):
    from paper_2606_12154_amd import hh
    shape, tensors, model = tiny
    ctx = new_context(shape, tensors, streams=2, context=40)
    toks = synth.make_tokens(shape.vocab, 30, 5)
    ctx.prefill(0, toks)
    with pytest.raises(hh.HHError) as e:
        ctx.prefill(0, toks)          # 60 > 40 positions
    assert e.value.status == hh.HH_ERR_CONTEXT_FULL
    assert ctx.length(0) == 30        # unchanged by the failed call
    with pytest.raises(hh.HHError) as e:
        ctx.prefill(1, np.array([1, 4096], np.int32))
    assert e.value.status == hh.HH_ERR_INVALID_ARG
    with pytest.raises(hh.HHError) as e:
        ctx.decode_step([1], None)    # empty stream, no token given
    assert e.value.status == hh.HH_ERR_INVALID_ARG
    with pytest.raises(hh.HHError) as e:
        ctx.decode_step([0, 0], [1, 2])
    assert e.value.status == hh.HH_ERR_INVALID_ARG
    ctx.reset(0)
    assert ctx.length(0) == 0
    ref, _ = model.prefill(toks[:10])
    _, got = ctx.prefill(0, toks[:10], logits="all")
    check_logits(got, ref, TOL, what="after reset")


def test_stale_arena_contents(tiny):
    """The arena is caller memory with arbitrary contents: KV slots past a
    stream's length (the rest of its last page) must not leak into the
    result even when they hold non-finite bit patterns.  An allocation of
    the arena's size is filled with 0xFF bytes (NaN in fp16 and fp32) and
    released, so torch's caching allocator hands that block to the next
    context."""
    import torch
    from paper_2606_12154_amd import hh
    shape, tensors, model = tiny
    cfg = hh.make_config(shape, 4, 96)
    junk = torch.full((hh.hh_workspace_size(cfg),), 0xFF, dtype=torch.uint8, device="cuda:0")
    torch.cuda.synchronize()
    del junk
    ctx = hh.Context(cfg)
    try:
        ctx.load_weights(tensors)
        lens = [5, 17, 1, 30]  # partial last pages
        prompts = [synth.make_tokens(shape.vocab, n, 40 + i) for i, n in enumerate(lens)]
        caches = []
        for i, p in enumerate(prompts):
            _, lg = ctx.prefill(i, p, logits="last")
            ref, cache = model.prefill(p, rows="last")
            check_logits(lg, ref[0], TOL, what=f"prefill {i}")
            caches.append(cache)
        feed = np.array([3, 1000, 2047, 7], np.int32)
        _, lg = ctx.decode_step([0, 1, 2, 3], feed, logits=True)
        check_logits(lg, model.decode_batch(caches, feed), TOL, what="multi decode")
        _, lg = ctx.decode_step([2], [11], logits=True)  # batch-1 kernel on the 1-token stream
        check_logits(lg[0], model.decode(caches[2], 11), TOL, what="single decode")
    finally:
        ctx.close()


@pytest.mark.parametrize("var,value", [("HH_RING_SLOTS", "6"), ("HH_LOAD_DEPTH", "1"), ("HH_LOAD_DEPTH", "7"),
                                       ("HH_STEP_QUIET", "0"), ("HH_STEP_QUIET", "2"), ("HH_POLL_DELAY", "0"),
                                       ("HH_POLL_DELAY", "400")])
def test_step_schedule_variants(tiny, var, value):
    """The single-kernel decode step's schedule settings (ring slots, loads
    in flight per streaming wave, pausing the streams during exchange waits,
    delay before the first poll) change timing only: teacher-forced logits
    still match the oracle."""
    import os
    shape, tensors, model = tiny
    prompt = synth.make_tokens(shape.vocab, 64, 1)
    toks, ref = oracle_greedy(model, prompt, 8)
    os.environ[var] = value
    try:
        ctx = new_context(shape, tensors, streams=1, context=96)
    finally:
        del os.environ[var]
    try:
        ctx.prefill(0, prompt)
        for i in range(8):
            _, lg = ctx.decode_step([0], [int(toks[i])], logits=True)
            check_logits(lg[0], ref[i + 1], TOL, what=f"{var}={value} step {i}")
    finally:
        ctx.close()


def test_failed_step_is_reported(tiny):
    """A decode step whose bounded wait gives up (forced from the host: the
    final argmax wait expects an epoch no workgroup publishes, with a 10 us
    limit; every wave still runs to its end) leaves -1 as its token, later
    device-fed steps of the stream and multi-stream steps including it keep
    -1, the first call with host outputs returns HH_ERR_HIP, and hh_reset
    brings the stream back."""
    import os
    from paper_2606_12154_amd import hh
    shape, tensors, model = tiny
    p0 = synth.make_tokens(shape.vocab, 40, 61)
    p1 = synth.make_tokens(shape.vocab, 24, 62)
    os.environ["HH_STEP_WAIT_TICKS"] = "1000"
    os.environ["HH_STEP_FAIL_WAIT"] = "1"
    try:
        ctx = new_context(shape, tensors, streams=2, context=96)
    finally:
        del os.environ["HH_STEP_WAIT_TICKS"]
        del os.environ["HH_STEP_FAIL_WAIT"]
    try:
        ctx.prefill(0, p0)
        ctx.prefill(1, p1)
        for _ in range(3):
            ctx.decode_step([0], None, host_next=False)
        assert list(ctx.read_argmax(0, 40, 3)) == [-1, -1, -1]
        ref1, cache1 = model.prefill(p1, rows="last")
        ctx.decode_step([0, 1], None, host_next=False)  # the multi-row path
        assert int(ctx.read_argmax(0, 43, 1)[0]) == -1
        ref = model.decode(cache1, int(np.argmax(ref1[0])))
        if top2_margin(ref) > 1e-2:
            assert int(ctx.read_argmax(1, 24, 1)[0]) == int(np.argmax(ref))
        with pytest.raises(hh.HHError) as e:
            ctx.decode_step([0], [5], logits=True)
        assert e.value.status == hh.HH_ERR_HIP
        ctx.reset()
        nxt, last = ctx.prefill(0, p0, logits="last")
        ref0, _ = model.prefill(p0, rows="last")
        check_logits(last, ref0[0], TOL, what="prefill after reset")
        assert nxt == int(np.argmax(ref0[0]))
    finally:
        ctx.close()
