"""GPU parity with the fp64 oracle at the 1B workload sizes whose prompts the
oracle cannot evaluate within a test run: the stored oracle values of
``tests/golden/oracle_1b.npz`` (written by ``tests/golden/make_oracle_1b.py``,
which calls only the oracle and the seeded generators) hold the residual
stream after the last block of every compared row, and the oracle's own LM
head (``Decoder.logits``) turns them into logits here.

Every compared row: max-abs over the whole vocabulary within 2e-2, argmax
equal wherever the oracle's top-2 margin exceeds 1e-2.  The token fed to
each decode step is the oracle's greedy token of the row before (teacher
forcing), for the GPU and the oracle alike.

* long context (8192-token prompt, the long-context workload) in the context
  configuration the benchmark times (32 streams, 8192 + 513 positions, one
  8192-row prefill pass), and again prefilled in 2048-row passes: the
  prompt's last row and 4 batch-1 decode steps (the single-kernel step,
  attention split over 8 items per kv head, partials combined by the
  producers);
* an 1100-token prompt in 512-row passes and 6 decode steps (more than two
  attention items per kv head from the first step);
* 32 streams with 256-token prompts (the multi-stream workload), prefilled one
  stream at a time, and again all 32 in one ``hh_prefill_batch`` call: every
  stream's last prompt row and 2 lockstep decode steps (the multi-row path,
  17 pages per row).
"""
import os

import numpy as np
import pytest

import oracle
import synth
from gpu_util import check_logits, new_context

pytestmark = pytest.mark.gpu
TOL = 2e-2
GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "oracle_1b.npz")


@pytest.fixture(scope="module")
def one_b():
    shape = synth.ONE_B
    tensors = synth.make_weights(shape, 1)
    # The oracle's head needs only the embedding (tied) and the final gain.
    names = [n for n, _ in shape.tensor_specs()]
    head = {"embed": synth.bf16_bits_to_f32(tensors[0]).reshape(shape.vocab, shape.d_model).astype(np.float64),
            "final_norm": synth.bf16_bits_to_f32(tensors[names.index("final_norm")]).astype(np.float64)}
    model = oracle.Decoder(shape, head)
    gold = dict(np.load(GOLDEN))
    return shape, tensors, model, gold


@pytest.fixture(scope="module")
def bench_ctx(one_b):
    """The context configuration the benchmark times."""
    shape, tensors, _, _ = one_b
    ctx = new_context(shape, tensors, streams=32, context=8192 + 513, max_prefill=8192)
    yield ctx
    ctx.close()


def teacher_forced(ctx, model, prompt, fed, hidden, what):
    ctx.reset(0)
    _, last = ctx.prefill(0, prompt, logits="last")
    worst = check_logits(last, model.logits(hidden[0]), TOL, what=f"{what} prompt last row")
    for i, tok in enumerate(fed):
        _, lg = ctx.decode_step([0], [int(tok)], logits=True)
        worst = max(worst, check_logits(lg[0], model.logits(hidden[i + 1]), TOL, what=f"{what} decode step {i}"))
    assert ctx.length(0) == len(prompt) + len(fed)
    return worst


def test_long_context_single_pass(one_b, bench_ctx):
    shape, _, model, g = one_b
    prompt = synth.make_tokens(shape.vocab, int(g["long_prompt"]), int(g["long_seed"]))
    worst = teacher_forced(bench_ctx, model, prompt, g["long_fed"], g["long_hidden"], "8192 one pass")
    print(f"1B 8192-token prompt (one pass) + 4 steps: max-abs {worst:.4g}")


def test_long_context_chunked(one_b):
    shape, tensors, model, g = one_b
    prompt = synth.make_tokens(shape.vocab, int(g["long_prompt"]), int(g["long_seed"]))
    ctx = new_context(shape, tensors, streams=1, context=8192 + 8, max_prefill=2048)
    try:
        worst = teacher_forced(ctx, model, prompt, g["long_fed"], g["long_hidden"], "8192 in 2048-row passes")
    finally:
        ctx.close()
    print(f"1B 8192-token prompt (2048-row passes) + 4 steps: max-abs {worst:.4g}")


def test_1100_positions(one_b):
    shape, tensors, model, g = one_b
    prompt = synth.make_tokens(shape.vocab, int(g["mid_prompt"]), int(g["mid_seed"]))
    ctx = new_context(shape, tensors, streams=1, context=1200, max_prefill=512)
    try:
        worst = teacher_forced(ctx, model, prompt, g["mid_fed"], g["mid_hidden"], "1100 positions")
    finally:
        ctx.close()
    print(f"1B 1100-token prompt (512-row passes) + 6 steps: max-abs {worst:.4g}")


def multi_prompts(shape, g):
    n, P, s0 = 32, int(g["multi_prompt"]), int(g["multi_seed0"])
    return [synth.make_tokens(shape.vocab, P, s0 + s) for s in range(n)]


def lockstep_steps(ctx, model, g, what):
    worst = 0.0
    ids = list(range(32))
    for step, (fed, hid) in enumerate([(g["multi_fed1"], g["multi_hidden1"]), (g["multi_fed2"], g["multi_hidden2"])]):
        _, lg = ctx.decode_step(ids, fed, logits=True)
        worst = max(worst, check_logits(lg, model.logits(hid), TOL, what=f"{what} lockstep step {step}"))
    return worst


def test_32_streams_per_stream_prefill(one_b, bench_ctx):
    shape, _, model, g = one_b
    ctx = bench_ctx
    ctx.reset(-1)
    worst = 0.0
    ref0 = model.logits(g["multi_hidden0"])
    for s, p in enumerate(multi_prompts(shape, g)):
        _, last = ctx.prefill(s, p, logits="last")
        worst = max(worst, check_logits(last, ref0[s], TOL, what=f"stream {s} prompt last row"))
    worst = max(worst, lockstep_steps(ctx, model, g, "32 streams"))
    print(f"1B 32 streams x 256-token prompts + 2 lockstep steps: max-abs {worst:.4g}")


def test_32_streams_batch_prefill(one_b, bench_ctx):
    shape, _, model, g = one_b
    ctx = bench_ctx
    ctx.reset(-1)
    nxt = ctx.prefill_batch(list(range(32)), multi_prompts(shape, g))
    # The oracle's greedy tokens of the prompts' last rows (the tokens the
    # first lockstep step is fed) wherever their margin is clear.
    ref0 = model.logits(g["multi_hidden0"])
    srt = np.sort(ref0, axis=-1)
    sure = srt[:, -1] - srt[:, -2] > 1e-2
    assert np.array_equal(nxt[sure], g["multi_fed1"][sure])
    worst = lockstep_steps(ctx, model, g, "32 streams, batch prefill")
    print(f"1B 32 x 256 tokens in one hh_prefill_batch call + 2 lockstep steps: max-abs {worst:.4g}")
