"""hh_decode_step_noalloc (the allocation-free batch-1 step, exchange words in
the library's fixed device array) against hh_decode_step (the same step with
the context's own exchange words), through the C ABI: two contexts on the
same weights and prompt, teacher-forced steps, then device-fed steps, for two
requests in a row, the second with a shorter prompt.  Bar: the oracle bar of
each model (max-abs 1e-4 fp32, 2e-2 bf16, argmax equal); the two run the same
kernel with the same summation order, so their logits are expected to be
identical."""
import numpy as np
import pytest

import synth
from gpu_util import new_context
from paper_2606_12154_amd import hh

pytestmark = pytest.mark.gpu


def compare(shape, tensors, prompts, tol, context):
    V = shape.vocab
    ref = new_context(shape, tensors, streams=2, context=context)
    new = new_context(shape, tensors, streams=2, context=context)
    worst, same = 0.0, True
    try:
        for prompt in prompts:
            ref.reset()
            new.reset()
            ref.prefill(1, prompt)
            new.prefill(1, prompt)
            tok = 7
            for i in range(4):
                nr, lr = ref.decode_step([1], [tok], logits=True)
                ln = np.empty(V, dtype=np.float32)
                nn = np.zeros(1, dtype=np.int32)
                hh.hh_decode_step_noalloc(new.ctx, 1, tok, ln.ctypes.data, nn.ctypes.data)
                err = float(np.abs(ln.astype(np.float64) - lr[0]).max())
                worst = max(worst, err)
                same = same and np.array_equal(ln, lr[0])
                assert np.isfinite(ln).all()
                assert err <= tol, f"prompt {len(prompt)}, step {i}: max-abs {err:.3g}"
                assert int(nn[0]) == int(nr[0]) == int(np.argmax(lr[0]))
                tok = int(nr[0])
            # Device-fed steps (pending token, no host outputs), then the
            # recorded argmax history of both.
            for _ in range(5):
                ref.decode_step([1], None, host_next=False)
                hh.hh_decode_step_noalloc(new.ctx, 1, None, None, None)
            n = len(prompt) + 9
            assert ref.length(1) == new.length(1) == n
            assert np.array_equal(ref.read_argmax(1, len(prompt), 9), new.read_argmax(1, len(prompt), 9))
    finally:
        ref.close()
        new.close()
    return worst, same


def test_noalloc_step_tiny():
    shape = synth.TINY
    tensors = synth.make_weights(shape, 0, gain_std=0.1)
    prompts = [synth.make_tokens(shape.vocab, 64, 1), synth.make_tokens(shape.vocab, 20, 2)]
    worst, same = compare(shape, tensors, prompts, 1e-4, 128)
    print(f"tiny: noalloc vs hh_decode_step max-abs {worst:.3g}, identical {same}")


def test_noalloc_step_1b():
    shape = synth.ONE_B
    tensors = synth.make_weights(shape, 1)
    prompts = [synth.make_tokens(shape.vocab, 256, 2), synth.make_tokens(shape.vocab, 40, 3)]
    worst, same = compare(shape, tensors, prompts, 2e-2, 320)
    print(f"1B: noalloc vs hh_decode_step max-abs {worst:.3g}, identical {same}")


def test_noalloc_rejects_bad_calls():
    shape = synth.TINY
    tensors = synth.make_weights(shape, 0)
    ctx = new_context(shape, tensors, streams=1, context=16)
    try:
        with pytest.raises(hh.HHError) as e:
            hh.hh_decode_step_noalloc(ctx.ctx, 0, None, None, None)  # empty stream, no token
        assert e.value.status == hh.HH_ERR_INVALID_ARG
        with pytest.raises(hh.HHError) as e:
            hh.hh_decode_step_noalloc(ctx.ctx, 1, 5, None, None)  # no such stream
        assert e.value.status == hh.HH_ERR_INVALID_ARG
        with pytest.raises(hh.HHError) as e:
            hh.hh_decode_step_noalloc(ctx.ctx, 0, shape.vocab, None, None)
        assert e.value.status == hh.HH_ERR_INVALID_ARG
        ctx.prefill(0, synth.make_tokens(shape.vocab, 16, 3))
        with pytest.raises(hh.HHError) as e:
            hh.hh_decode_step_noalloc(ctx.ctx, 0, 5, None, None)  # context full
        assert e.value.status == hh.HH_ERR_CONTEXT_FULL
        assert ctx.length(0) == 16
    finally:
        ctx.close()
