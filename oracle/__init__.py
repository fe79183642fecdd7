"""Oracle for the mouth model's prefill + greedy decode.  TEST INFRASTRUCTURE ONLY.

A plain, slow, fp64 numpy implementation of the decoder-only forward pass the
HIP library computes.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import it; the product path never
does, and this package imports nothing from the product package.

What it follows.  The paper fixes the role and the measured quantities: a
1B-class model streams the rendered answer after one prompt evaluation (Sec. 4
"Runtime phase"); TTFT, decode rate and end-to-end throughput are separate
quantities (Sec. 6.2); the KV cache grows with the context window (Sec. 6.6).
It names the model (MiniCPM5-1B, 4-bit; Sec. 4, Sec. 5) but not its
architecture, so the decoder here is the textbook Llama-style definition:
RMSNorm (Zhang & Sennrich 2019), rotary position embedding in rotate-half
pairing (Su et al. 2021), grouped-query attention (Ainslie et al. 2023),
SwiGLU MLP (Shazeer 2020), tied embedding/LM head, greedy argmax with ties to
the lowest index.  Every function is written as that definition; there is no
blocking, fusion or reordering beyond chunking attention over query rows.

Pins (``tests/test_oracle.py``): closed-form RMSNorm/RoPE/SiLU values, fp64
brute-force attention on tiny shapes, GQA == MHA with repeated KV heads, the
HuggingFace transformers Llama implementation on the tiny model, causality,
KV-cached decode == full recompute, chunked == one-shot prefill, and the
zero-layer echo model; for the 4-bit group format (``quant.py``): a worked
example, exact round trips of representable groups, the half-step error
bound, ties to even, zero groups and the nibble layout.  Matching the paper's
own model outputs is parity unpinned: its weights and printed outputs do not
exist, and neither does its 4-bit format's definition.

``router.py`` is the oracle of the serving steps around the decoder (BM25
routing with the margin gate, the marker-line envelope), pinned in
``tests/test_router.py``; it is imported as ``oracle.router``.
"""
from .decoder import (Decoder, KVCache, apply_rope, attention, greedy, rms_norm,
                      rope_angles, silu)
from .quant import q4_dequantize, q4_model_weights, q4_pack_rows, q4_quantize_rows

__all__ = ["Decoder", "KVCache", "apply_rope", "attention", "greedy", "rms_norm",
           "rope_angles", "silu", "q4_quantize_rows", "q4_dequantize", "q4_pack_rows",
           "q4_model_weights"]
