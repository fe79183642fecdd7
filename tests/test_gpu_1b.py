"""GPU parity on the 1B-class bf16 decoder (16 layers, d 2048, 32/8 heads,
FFN 8192, vocab 128256): teacher-forced logits within max-abs 2e-2 of the fp64
oracle over the whole vocabulary, argmax equal wherever the oracle's top-2
margin exceeds 1e-2.  The oracle consumes the same bf16 weights widened to
fp64; the GPU keeps the KV cache in fp16 and feeds its MFMA path fp16
operands, the only sources of difference beyond summation order."""
import os

import numpy as np
import pytest

import oracle
import synth
from gpu_util import check_logits, new_context, top2_margin

pytestmark = pytest.mark.gpu
TOL = 2e-2


@pytest.fixture(scope="module")
def one_b():
    shape = synth.ONE_B
    tensors = synth.make_weights(shape, 1)
    model = oracle.Decoder(shape, synth.weights_as_f64(shape, tensors))
    return shape, tensors, model


@pytest.fixture(scope="module")
def ctx(one_b):
    shape, tensors, _ = one_b
    c = new_context(shape, tensors, streams=5, context=512, max_prefill=256)
    yield c
    c.close()


@pytest.fixture(scope="module")
def prompt_ref(one_b):
    """Oracle logits of every row of the 256-token prompt (by causality, the
    first n rows are also the logits of the prompt's first n tokens)."""
    shape, _, model = one_b
    toks = synth.make_tokens(shape.vocab, 256, 2)
    ref, _ = model.prefill(toks)
    return toks, ref


def test_prefill_256_all_logits(one_b, ctx, prompt_ref):
    toks, ref = prompt_ref
    ctx.reset()
    nxt, got = ctx.prefill(0, toks, logits="all")
    worst = check_logits(got, ref, TOL, what="1B prefill all")
    print(f"1B prefill 256 rows: max-abs {worst:.4g}")
    assert nxt == int(np.argmax(got[-1]))


@pytest.mark.parametrize("cut", [72, 129])
def test_prefill_appended_chunk(one_b, ctx, prompt_ref, cut):
    """A prompt fed in two calls: the second chunk's queries start mid key
    block, so some key-split groups of the flash kernel see no visible key for
    some queries."""
    toks, ref = prompt_ref
    ctx.reset()
    ctx.prefill(0, toks[:cut])
    nxt, got = ctx.prefill(0, toks[cut:200], logits="all")
    worst = check_logits(got, ref[cut:200], TOL, what=f"1B appended chunk {cut}:200")
    print(f"1B appended chunk {cut}:200: max-abs {worst:.4g}")
    assert nxt == int(np.argmax(got[-1]))


GEMM_KINDS = ("HH_GEMM_QKV", "HH_GEMM_RESID", "HH_GEMM_DOWN", "HH_GEMM_GATEUP")


@pytest.mark.parametrize("tile", ["256x256x1", "256x128x1", "128x256x1", "128x128x1", "256x256x4", "128x128x2",
                                  "256x256x1x8", "256x128x2x8", "128x256x1x8", "128x128x1x8", "128x128x2x8"])
@pytest.mark.parametrize("n", [256, 200])
def test_prefill_wide_tiles(one_b, ctx, prompt_ref, tile, n):
    """Every large-tile GEMM shape (and split-K; four or eight waves per
    workgroup) of the prompt path, forced for the QKV, residual and gate/up
    GEMMs, on a whole and a ragged row count."""
    toks, ref = prompt_ref
    saved = {k: os.environ.get(k) for k in GEMM_KINDS}
    try:
        for k in GEMM_KINDS:
            os.environ[k] = tile
        ctx.reset()
        nxt, got = ctx.prefill(0, toks[:n], logits="all")
    finally:
        for k, v in saved.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v
    worst = check_logits(got, ref[:n], TOL, what=f"1B prefill {n} rows, tiles {tile}")
    print(f"1B prefill {n} rows, tiles {tile}: max-abs {worst:.4g}")
    assert nxt == int(np.argmax(got[-1]))


@pytest.mark.parametrize("plen,steps", [(256, 40), (140, 6), (100, 4)], ids=["p256", "p140", "p100"])
def test_decode_teacher_forced(one_b, ctx, plen, steps):
    """The batch-1 kernel against the oracle.  With attention items of at
    most 8 pages: 256 + 40 positions take three splits per kv head (combined
    at the producer), 140 + 6 two (combined by the O-phase consumers) and
    100 + 4 one."""
    shape, _, model = one_b
    prompt = synth.make_tokens(shape.vocab, plen, 2)
    ref_last, cache = model.prefill(prompt, rows="last")
    ctx.reset()
    nxt, last = ctx.prefill(0, prompt, logits="last")
    worst = check_logits(last, ref_last[0], TOL, what="prefill last")
    tok = int(np.argmax(ref_last[0]))
    # With 256 + 40: attended lengths 257 .. 296 include item lengths that
    # are whole 32-key slots (t = 272, 288), where the step's own key and
    # value sit in the last row of a streamed slot.
    for i in range(steps):
        ref = model.decode(cache, tok)
        _, lg = ctx.decode_step([0], [tok], logits=True)
        worst = max(worst, check_logits(lg[0], ref, TOL, what=f"decode step {i}"))
        tok = int(np.argmax(ref))
    print(f"1B teacher-forced decode ({plen} + {steps}): max-abs {worst:.4g}")


def multistream_lockstep(model, shape, ctx, what):
    lens = [16, 33, 7, 48]
    prompts = [synth.make_tokens(shape.vocab, n, 100 + i) for i, n in enumerate(lens)]
    ctx.reset()
    caches = []
    for i, p in enumerate(prompts):
        ctx.prefill(i, p)
        caches.append(model.prefill(p, rows="last")[1])
    rng = np.random.default_rng(11)
    worst = 0.0
    for step in range(3):
        feed = rng.integers(0, shape.vocab, size=4).astype(np.int32)
        _, lg = ctx.decode_step([0, 1, 2, 3], feed, logits=True)
        ref = model.decode_batch(caches, feed)
        worst = max(worst, check_logits(lg, ref, TOL, what=f"{what} step {step}"))
    print(f"{what}: max-abs {worst:.4g}")


def test_multistream_lockstep(one_b, ctx):
    """Four ragged streams in lockstep (prompts of up to 48 tokens run through
    the skinny GEMMs too), activation-resident skinny kernel."""
    shape, _, model = one_b
    multistream_lockstep(model, shape, ctx, "1B 4-stream decode")


@pytest.mark.parametrize("env", [{"HH_SKINNY_RES": "0"}, {"HH_ROWNORM": "0"}], ids=["batched_skinny", "separate_norms"])
def test_multistream_lockstep_variants(one_b, env):
    """The same with the batched skinny kernel (HH_SKINNY_RES=0, which serves
    grids or K ranges the resident one does not take, and norms as passes of
    their own), and with the resident kernel but every RMSNorm as a pass of
    its own (HH_ROWNORM=0); a context of its own, run eagerly, so that no
    graph captured under the default is replayed."""
    shape, tensors, model = one_b
    saved = {k: os.environ.get(k) for k in list(env) + ["HH_GRAPHS"]}
    os.environ.update(env)
    os.environ["HH_GRAPHS"] = "0"
    c = None
    try:
        c = new_context(shape, tensors, streams=5, context=512, max_prefill=256)
        multistream_lockstep(model, shape, c, f"1B 4-stream decode, {env}")
    finally:
        if c is not None:
            c.close()
        for k, v in saved.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v


def test_multistream_long_row(one_b):
    """A stream longer than the 32 pages (512 positions) the fp16 row
    attention keeps in registers up front, decoded in lockstep with a short
    one: the online loop over its later pages against the oracle."""
    shape, tensors, model = one_b
    c = None
    try:
        c = new_context(shape, tensors, streams=2, context=600, max_prefill=256)
        lens = [530, 20]
        prompts = [synth.make_tokens(shape.vocab, n, 600 + i) for i, n in enumerate(lens)]
        caches = []
        for i, p in enumerate(prompts):
            c.prefill(i, p)
            caches.append(model.prefill(p, rows="last")[1])
        feed = np.array([17, 29], dtype=np.int32)
        _, lg = c.decode_step([0, 1], feed, logits=True)
        worst = max(check_logits(lg[k], model.decode(caches[k], int(feed[k])), TOL, what=f"long row {k}")
                    for k in range(2))
        print(f"1B lockstep with a 531-position row: max-abs {worst:.4g}")
    finally:
        if c is not None:
            c.close()


@pytest.fixture(scope="module")
def forced_256(one_b):
    """The bench prompt (256 tokens, seed 2) and 8 teacher-forced steps of the
    oracle: (prompt, fed tokens, reference logits of the prompt's last row
    and of each step)."""
    shape, _, model = one_b
    prompt = synth.make_tokens(shape.vocab, 256, 2)
    ref, cache = model.prefill(prompt, rows="last")
    rows, fed = [ref[0]], []
    for _ in range(8):
        fed.append(int(np.argmax(rows[-1])))
        rows.append(model.decode(cache, fed[-1]))
    return prompt, fed, rows


def forced_run(ctx, forced, what):
    prompt, fed, rows = forced
    ctx.reset()
    _, last = ctx.prefill(0, prompt, logits="last")
    worst = check_logits(last, rows[0], TOL, what=f"{what} prompt last row")
    for i, tok in enumerate(fed):
        _, lg = ctx.decode_step([0], [tok], logits=True)
        worst = max(worst, check_logits(lg[0], rows[i + 1], TOL, what=f"{what} step {i}"))
    return worst


def test_gemv_graph_path(one_b, forced_256):
    """The batch-1 path of separate GEMV / attention kernels replayed as a
    graph (taken when the single-kernel step is switched off, and the side
    the long-context consistency checks compare with) against the oracle."""
    shape, tensors, _ = one_b
    os.environ["HH_STEP_KERNEL"] = "0"
    try:
        c = new_context(shape, tensors, streams=1, context=512, max_prefill=256)
    finally:
        del os.environ["HH_STEP_KERNEL"]
    try:
        worst = forced_run(c, forced_256, "GEMV graph path")
    finally:
        c.close()
    print(f"1B GEMV graph path, 256 prompt + 8 steps: max-abs {worst:.4g}")


def test_window_131072_short_use(one_b, forced_256):
    """The paper's window sweep as stated (a large allocated context, short
    use): a 131072-position context serving the bench request's prompt and
    8 decode steps."""
    shape, tensors, _ = one_b
    c = new_context(shape, tensors, streams=1, context=131072, max_prefill=256)
    try:
        worst = forced_run(c, forced_256, "131072-position window")
    finally:
        c.close()
    print(f"1B in a 131072-position window, 256 prompt + 8 steps: max-abs {worst:.4g}")


def test_prefill_batch_1b(one_b, ctx, forced_256):
    """Ragged prompts in one hh_prefill_batch call on the 1B bf16 model (MFMA
    GEMMs over the packed rows, per-row attention, n-row head): the bench
    prompt of 256 tokens (16 pages per row) plus 5 and 40 tokens, 301 rows in
    two 256-row passes.  Next tokens and the KV each stream is left with,
    checked by a lockstep decode step, against the oracle's run of each
    stream alone."""
    shape, _, model = one_b
    prompt, fed, rows = forced_256
    ctx.reset()
    ids = [4, 1, 2]
    prompts = [prompt] + [synth.make_tokens(shape.vocab, n, 400 + n) for n in (5, 40)]
    nxt = ctx.prefill_batch(ids, prompts)
    refs, caches, worst = [rows[0]], [None], 0.0
    for p in prompts[1:]:
        logits, cache = model.prefill(p, rows="last")
        refs.append(logits[0])
        caches.append(cache)
    for k in range(3):
        if top2_margin(refs[k]) > 1e-2:
            assert int(nxt[k]) == int(np.argmax(refs[k])), f"stream {ids[k]}"
    feed = np.array([fed[0], 202, 303], dtype=np.int32)
    _, lg = ctx.decode_step(ids, feed, logits=True)
    worst = check_logits(lg[0], rows[1], TOL, what="1B batch prefill stream 4")
    for k in (1, 2):
        worst = max(worst, check_logits(lg[k], model.decode(caches[k], int(feed[k])), TOL,
                                        what=f"1B batch prefill stream {ids[k]}"))
    print(f"1B batch prefill (256, 5, 40 rows) then lockstep step: max-abs {worst:.4g}")
