"""Shared helpers of the GPU parity tests (no oracle arithmetic here)."""
import numpy as np

from paper_2606_12154_amd import hh


def new_context(shape, tensors, streams=4, context=256, max_prefill=0):
    ctx = hh.Context(hh.make_config(shape, streams, context, max_prefill))
    ctx.load_weights(tensors)
    return ctx


def top2_margin(ref):
    srt = np.sort(ref, axis=-1)
    return srt[..., -1] - srt[..., -2]


def check_logits(got, ref, tol, margin=1e-2, what=""):
    """max-abs within tol, and identical argmax wherever the reference's
    top-2 margin exceeds `margin`."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    err = np.abs(got - ref)
    worst = float(err.max())
    assert np.isfinite(got).all(), f"{what}: non-finite logits"
    assert worst <= tol, f"{what}: max-abs {worst:.3g} > {tol} at {np.unravel_index(err.argmax(), err.shape)}"
    sure = top2_margin(ref) > margin
    ga, ra = np.argmax(got, axis=-1), np.argmax(ref, axis=-1)
    bad = np.argwhere(sure & (ga != ra))
    assert bad.size == 0, f"{what}: argmax differs at {bad[:5].tolist()}"
    return worst
