"""Group-wise 4-bit weights (test infrastructure only, like the rest of oracle/).

The paper's mouth model runs with 4-bit weights (Sec. 4 "Runtime phase",
Sec. 5) but does not name the format, so this is the reading taken here, a
plain symmetric group format ("Q4G32"):

* every streamed matrix row w[0..K) is cut into groups of 32 consecutive
  elements; group g holds w[32 g .. 32 g + 32);
* its scale is s = bf16(a / 7) with a = max |w_i| over the group, the
  division in fp32 and the bf16 rounding to nearest even (a = 0 gives s = 0);
* each element becomes q_i = clamp(rint(w_i / s), -8, 7): fp32 division,
  rounding half to even (q_i = 0 when s = 0);
* the value the model computes with is q_i * s, exact in fp32 (a 4-bit
  integer times an 8-bit significand).

Rows are the rows of W_q, W_k, W_v, W_o, W_gate, W_up and of the LM head
(groups along each matrix's input dimension), and the rows of W_down^T
(groups of 32 consecutive output rows of W_down for each of its columns).
The token-embedding lookup keeps the bf16 table; only the LM head's copy of
the tied embedding is quantized.

Storage of one row (what the library's kernels read): K / 2 bytes of
nibbles, n_i = q_i + 8, element 2k in the low nibble of byte k and 2k + 1 in
the high nibble, followed by the K / 32 scales as little-endian bf16.
"""
from __future__ import annotations

import numpy as np

GROUP = 32


def _bf16_round(a: np.ndarray) -> np.ndarray:
    """fp32 -> nearest bf16 (ties to even), returned as fp32 values."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    r = (u + (((u >> 16) & 1) + np.uint32(0x7FFF))) & np.uint32(0xFFFF0000)
    return r.view(np.float32)


def q4_quantize_rows(w: np.ndarray):
    """Quantize rows [R, K] (K a multiple of 32; finite values) to codes
    q int8 [R, K] in [-8, 7] and scales s float32 [R, K / 32] (bf16 values)."""
    w = np.asarray(w, dtype=np.float32)
    R, K = w.shape
    assert K % GROUP == 0
    g = w.reshape(R, K // GROUP, GROUP)
    a = np.max(np.abs(g), axis=-1)
    s = _bf16_round(a / np.float32(7.0))
    with np.errstate(divide="ignore", invalid="ignore"):
        r = g / s[..., None]
    r = np.where(s[..., None] > 0, r, np.float32(0.0))
    q = np.clip(np.rint(r), -8, 7).astype(np.int8)
    return q.reshape(R, K), s


def q4_dequantize(q: np.ndarray, s: np.ndarray) -> np.ndarray:
    """Values q * s of the group format, fp64 [R, K]."""
    R, K = q.shape
    v = q.reshape(R, K // GROUP, GROUP).astype(np.float64) * s.astype(np.float64)[..., None]
    return v.reshape(R, K)


def q4_pack_rows(q: np.ndarray, s: np.ndarray) -> np.ndarray:
    """The stored rows, uint8 [R, K / 2 + 2 K / 32]."""
    n = (q.astype(np.int16) + 8).astype(np.uint8)
    nib = n[:, 0::2] | (n[:, 1::2] << 4)
    sb = (np.ascontiguousarray(s, dtype=np.float32).view(np.uint32) >> 16).astype("<u2")
    return np.concatenate([nib, sb.view(np.uint8).reshape(q.shape[0], -1)], axis=1)


def q4_model_weights(cfg, w: dict) -> dict:
    """The weights a Q4G32 model computes with, from the fp64 view of its
    bf16 tensors (keys as in Decoder): quantized-then-dequantized matrices,
    W_down through its transpose, an untied head holding Q4G32(embed); the
    embedding table and the norm gains unchanged."""
    out = dict(w)

    def qd(m):
        q, s = q4_quantize_rows(m.astype(np.float32))
        return q4_dequantize(q, s)

    for l in range(cfg.n_layers):
        p = f"l{l}."
        for k in ("wq", "wk", "wv", "wo", "w_gate", "w_up"):
            out[p + k] = qd(w[p + k])
        out[p + "w_down"] = qd(w[p + "w_down"].T).T
    out["lm_head"] = qd(w.get("lm_head", w["embed"]))
    return out
