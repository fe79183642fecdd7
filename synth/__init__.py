"""Seeded synthetic inputs shared by the HIP path's tests/bench and by the oracle.

This module holds model shapes and random-number draws only: no step of the
decoder's arithmetic lives here.  Both sides receive the same arrays from it.

Workloads (the mouth model of the runtime path, paper Sec. 4 "Runtime phase";
its trained weights and corpus are unavailable, so weights are seeded random
draws and prompts are uniform random token ids -- a dense decoder's cost
depends only on lengths, not on token values):

* ``tiny``  : 2 layers, d 256, 4 q heads / 2 kv heads of dim 64, FFN 688,
              vocab 4096, RMSNorm eps 1e-5, RoPE theta 1e4, tied, fp32.
* ``1b``    : 16 layers, d 2048, 32 q heads / 8 kv heads of dim 64, FFN 8192,
              vocab 128256, eps 1e-5, RoPE theta 5e5, tied, bf16.

Weight recipe: every matrix is i.i.d. N(0, 0.02^2), drawn in fp32 with
``numpy.random.Generator(PCG64(SeedSequence([seed, i]))).standard_normal``
where i is the tensor's index in the C-ABI load order (one generator per
tensor, so tensors can be drawn in parallel); bf16 models round each fp32 draw
to nearest-even bf16.  RMSNorm gains are 1.0 unless ``gain_std`` > 0, in which
case they are 1 + N(0, gain_std^2) from the generator of
SeedSequence([seed, i, 1]), so the matrices are the same either way.
"""
from __future__ import annotations

import concurrent.futures as cf
import dataclasses
import os
from typing import Dict, List

import numpy as np

F32 = 0
BF16 = 1


@dataclasses.dataclass(frozen=True)
class ModelShape:
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    ffn_dim: int
    vocab: int
    rms_eps: float
    rope_theta: float
    tied: bool
    dtype: int  # F32 or BF16: the element type of every weight tensor

    @property
    def q_dim(self) -> int:
        return self.n_heads * self.head_dim

    @property
    def kv_dim(self) -> int:
        return self.n_kv_heads * self.head_dim

    def tensor_specs(self):
        """(name, shape) of every weight tensor, in C-ABI load order."""
        d, F = self.d_model, self.ffn_dim
        specs = [("embed", (self.vocab, d))]
        for l in range(self.n_layers):
            specs += [
                (f"l{l}.attn_norm", (d,)),
                (f"l{l}.wq", (self.q_dim, d)),
                (f"l{l}.wk", (self.kv_dim, d)),
                (f"l{l}.wv", (self.kv_dim, d)),
                (f"l{l}.wo", (d, self.q_dim)),
                (f"l{l}.mlp_norm", (d,)),
                (f"l{l}.w_gate", (F, d)),
                (f"l{l}.w_up", (F, d)),
                (f"l{l}.w_down", (d, F)),
            ]
        specs.append(("final_norm", (d,)))
        if not self.tied:
            specs.append(("lm_head", (self.vocab, d)))
        return specs

    def n_params(self) -> int:
        return int(sum(int(np.prod(s)) for _, s in self.tensor_specs()))


TINY = ModelShape(2, 256, 4, 2, 64, 688, 4096, 1e-5, 1e4, True, F32)
ONE_B = ModelShape(16, 2048, 32, 8, 64, 8192, 128256, 1e-5, 5e5, True, BF16)

# Workloads: (shape, weight seed, prompt length, prompt seed(s), decode steps, streams)
WORKLOADS = {
    "tiny": dict(shape=TINY, wseed=0, prompt=64, tseed=1, steps=32, streams=1),
    "1b_decode": dict(shape=ONE_B, wseed=1, prompt=256, tseed=2, steps=256, streams=1),
    "1b_prefill": dict(shape=ONE_B, wseed=1, prompt=1024, tseed=3, steps=64, streams=1),
    "1b_long": dict(shape=ONE_B, wseed=1, prompt=8192, tseed=4, steps=512, streams=1),
    "1b_multi": dict(shape=ONE_B, wseed=1, prompt=256, tseed=100, steps=256, streams=32),
}


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round fp32 values to the nearest bf16 (ties to even); returns uint16 bits.

    Storage-format conversion of the seeded draws (finite inputs only)."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    bias = ((u >> 16) & 1) + np.uint32(0x7FFF)
    return ((u + bias) >> 16).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to fp32."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _draw_tensor(shape: "ModelShape", seed: int, i: int, shp, gain_std: float) -> np.ndarray:
    if len(shp) == 1:
        if gain_std > 0:
            g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, i, 1])))
            w = (1.0 + gain_std * g.standard_normal(shp)).astype(np.float32)
        else:
            w = np.ones(shp, dtype=np.float32)
    else:
        g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, i])))
        w = g.standard_normal(shp, dtype=np.float32)
        w *= np.float32(0.02)
    return f32_to_bf16_bits(w) if shape.dtype == BF16 else w


def make_weights(shape: ModelShape, seed: int, gain_std: float = 0.0) -> List[np.ndarray]:
    """Seeded weights in C-ABI tensor order and storage format.

    fp32 models give float32 arrays; bf16 models give uint16 arrays of bf16
    bits.  Matrices are N(0, 0.02^2); gains are ones (or 1 + N(0, gain_std^2))."""
    specs = shape.tensor_specs()
    workers = max(1, min(16, os.cpu_count() or 1))
    with cf.ThreadPoolExecutor(max_workers=workers) as ex:
        futs = [ex.submit(_draw_tensor, shape, seed, i, shp, gain_std) for i, (_, shp) in enumerate(specs)]
        return [f.result() for f in futs]


def weights_as_f64(shape: ModelShape, tensors: List[np.ndarray]) -> Dict[str, np.ndarray]:
    """Exact fp64 view of the stored weights, keyed by tensor name."""
    res = {}
    for (name, shp), t in zip(shape.tensor_specs(), tensors):
        v = bf16_bits_to_f32(t) if shape.dtype == BF16 else np.asarray(t, dtype=np.float32)
        res[name] = v.reshape(shp).astype(np.float64)
    return res


def make_tokens(vocab: int, n: int, seed: int) -> np.ndarray:
    """n uniform random token ids in [0, vocab) from PCG64(seed), int32."""
    rng = np.random.Generator(np.random.PCG64(seed))
    return rng.integers(0, vocab, size=n, dtype=np.int32)


# ---------------------------------------------------------------- synthetic knowledge store

_SYLLABLES = ["ka", "lo", "mi", "ne", "su", "ta", "ri", "po", "ve", "du", "an", "el", "or", "is", "um",
              "bra", "cle", "dro", "fin", "gal", "hem", "jor", "kel", "mon", "nar", "pel", "quo", "ser",
              "tin", "vor", "wex", "yal", "zer"]


def _word(rng: np.random.Generator) -> str:
    return "".join(rng.choice(_SYLLABLES, size=int(rng.integers(2, 5))))


def make_store(n_entries: int = 563, n_documents: int = 17, seed: int = 0):
    """A seeded synthetic store in the shape of the paper's routing study
    (563 entries harvested from 17 documents): entries of one document share
    its topic words, each entry has its own distinctive words, and every text
    mixes in common words drawn Zipf-like from a shared vocabulary.  Returns
    a list of (indexed text, answer line) pairs.  Plain text generation: no
    scoring arithmetic."""
    rng = np.random.default_rng(np.random.SeedSequence([seed, 9001]))
    common = sorted({_word(rng) for _ in range(400)})
    zipf = 1.0 / np.arange(1, len(common) + 1)
    zipf /= zipf.sum()
    topics = [[_word(rng) for _ in range(30)] for _ in range(n_documents)]
    doc_of = np.sort(rng.integers(0, n_documents, size=n_entries))
    store = []
    for i in range(n_entries):
        own = [_word(rng) for _ in range(int(rng.integers(4, 9)))]
        topic = list(rng.choice(topics[doc_of[i]], size=8, replace=False))
        filler = list(rng.choice(common, size=int(rng.integers(20, 50)), p=zipf))
        words = own + topic + filler
        rng.shuffle(words)
        text = " ".join(words)
        answer = f"{own[0].capitalize()} {topic[0]} is {int(rng.integers(1, 10000))} {own[1]} as of {1990 + i % 35}."
        store.append((text, answer))
    return store


def make_queries(store, per_entry: int = 2, seed: int = 1):
    """Queries generated from each entry's own vocabulary (as the paper's
    1,126 queries for 563 entries were): 3 to 6 of the entry's words, one
    or two of them possibly shared with other entries.  Returns a list of
    (query text, entry id)."""
    rng = np.random.default_rng(np.random.SeedSequence([seed, 9002]))
    out = []
    for i, (text, _) in enumerate(store):
        words = text.split()
        for _ in range(per_entry):
            k = int(rng.integers(3, 7))
            q = list(rng.choice(words, size=k, replace=False))
            out.append((" ".join(q), i))
    return out
