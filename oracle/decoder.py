"""fp64 reference decoder (test infrastructure only; see the package docstring).

Shapes: ``d`` model width, ``Hq``/``Hkv`` query/key-value heads, ``hd`` head
dim, ``F`` MLP width, ``V`` vocab.  Weight matrices are ``[out, in]`` as in
``nn.Linear``.  The configuration object only needs attributes n_layers,
d_model, n_heads, n_kv_heads, head_dim, ffn_dim, vocab, rms_eps, rope_theta.
"""
from __future__ import annotations

import numpy as np

# Queries per attention block: bounds the [rows, keys] score matrix in memory.
_Q_CHUNK = 256


def rms_norm(x: np.ndarray, gain: np.ndarray, eps: float, dtype=np.float64) -> np.ndarray:
    """RMSNorm: x / sqrt(mean(x^2) + eps) * gain over the last axis (Zhang &
    Sennrich 2019; eps added to the mean square inside the root)."""
    x = np.asarray(x, dtype=dtype)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * gain


def silu(z: np.ndarray) -> np.ndarray:
    """SiLU / swish: z * sigmoid(z)."""
    return z / (1.0 + np.exp(-z))


def rope_angles(positions: np.ndarray, head_dim: int, theta: float) -> np.ndarray:
    """Rotation angles p * theta^(-2i/hd) for i < hd/2, fp64, shape [T, hd/2]."""
    i = np.arange(head_dim // 2, dtype=np.float64)
    omega = theta ** (-2.0 * i / head_dim)
    return np.outer(np.asarray(positions, dtype=np.float64), omega)


def apply_rope(u: np.ndarray, positions: np.ndarray, theta: float, dtype=np.float64) -> np.ndarray:
    """Rotary embedding of u [T, H, hd] at absolute positions [T].

    Rotate-half pairing: component i is rotated together with i + hd/2,
    y_i = u_i cos a - u_{i+hd/2} sin a and y_{i+hd/2} = u_{i+hd/2} cos a +
    u_i sin a, with a = p * theta^(-2i/hd)."""
    hd = u.shape[-1]
    half = hd // 2
    a = rope_angles(positions, hd, theta)[:, None, :]
    c, s = np.cos(a).astype(dtype), np.sin(a).astype(dtype)
    lo, hi = u[..., :half], u[..., half:]
    return np.concatenate([lo * c - hi * s, hi * c + lo * s], axis=-1)


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, q_pos: np.ndarray) -> np.ndarray:
    """Causal grouped-query attention.

    q [Tq, Hq, hd] are queries at absolute positions q_pos [Tq]; k, v
    [Tk, Hkv, hd] hold keys/values of positions 0..Tk-1.  Query head j reads
    kv head j // (Hq / Hkv); query at position p sees keys 0..p (itself
    included); scores are scaled by 1/sqrt(hd); softmax subtracts the row max.
    """
    Tq, Hq, hd = q.shape
    Tk, Hkv, _ = k.shape
    group = Hq // Hkv
    scale = float(1.0 / np.sqrt(hd))
    out = np.zeros((Tq, Hq, hd), dtype=q.dtype)
    key_pos = np.arange(Tk)
    for j in range(Hq):
        g = j // group
        for r0 in range(0, Tq, _Q_CHUNK):
            r1 = min(Tq, r0 + _Q_CHUNK)
            s = (q[r0:r1, j, :] @ k[:, g, :].T) * scale
            s = np.where(key_pos[None, :] > q_pos[r0:r1, None], -np.inf, s)
            s = s - s.max(axis=1, keepdims=True)
            w = np.exp(s)
            w /= w.sum(axis=1, keepdims=True)
            out[r0:r1, j, :] = w @ v[:, g, :]
    return out


def greedy(logits: np.ndarray) -> np.ndarray:
    """Greedy next token: argmax over the vocab, lowest index among ties."""
    return np.argmax(logits, axis=-1)


class KVCache:
    """Per-stream contiguous cache of rotated keys and values, per layer [T, Hkv, hd]."""

    def __init__(self, n_layers: int, n_kv_heads: int, head_dim: int, dtype=np.float64):
        empty = np.zeros((0, n_kv_heads, head_dim), dtype=dtype)
        self.k = [empty.copy() for _ in range(n_layers)]
        self.v = [empty.copy() for _ in range(n_layers)]

    @property
    def length(self) -> int:
        return self.k[0].shape[0]


class Decoder:
    """Llama-style decoder over fp64 weights keyed as in the C-ABI load order:
    embed, l{i}.{attn_norm,wq,wk,wv,wo,mlp_norm,w_gate,w_up,w_down},
    final_norm and (untied models only) lm_head."""

    def __init__(self, cfg, weights: dict, dtype=np.float64):
        """dtype: the working precision of every step (fp64 unless a caller
        asks for another; the weights are taken in that type)."""
        self.cfg = cfg
        self.dtype = dtype
        self.w = {k: np.asarray(v, dtype=dtype) for k, v in weights.items()}
        self.head = self.w.get("lm_head", self.w["embed"])  # tied unless given

    def new_cache(self) -> KVCache:
        c = self.cfg
        return KVCache(c.n_layers, c.n_kv_heads, c.head_dim, self.dtype)

    def _block(self, l: int, x: np.ndarray, segments) -> np.ndarray:
        """One transformer block on rows x [T, d]; ``segments`` lists
        (cache, first_row, n_rows): rows first_row.. belong to that stream and
        sit at positions cache.length, cache.length+1, ... ."""
        c, w = self.cfg, self.w
        p = f"l{l}."
        T = x.shape[0]
        h = rms_norm(x, w[p + "attn_norm"], c.rms_eps, self.dtype)
        q = (h @ w[p + "wq"].T).reshape(T, c.n_heads, c.head_dim)
        k = (h @ w[p + "wk"].T).reshape(T, c.n_kv_heads, c.head_dim)
        v = (h @ w[p + "wv"].T).reshape(T, c.n_kv_heads, c.head_dim)
        o = np.zeros_like(q)
        for cache, r0, n in segments:
            positions = cache.k[l].shape[0] + np.arange(n)  # layer l not yet appended
            qr = apply_rope(q[r0:r0 + n], positions, c.rope_theta, self.dtype)
            kr = apply_rope(k[r0:r0 + n], positions, c.rope_theta, self.dtype)
            cache.k[l] = np.concatenate([cache.k[l], kr], axis=0)
            cache.v[l] = np.concatenate([cache.v[l], v[r0:r0 + n]], axis=0)
            o[r0:r0 + n] = attention(qr, cache.k[l], cache.v[l], positions)
        x = x + o.reshape(T, -1) @ w[p + "wo"].T
        h2 = rms_norm(x, w[p + "mlp_norm"], c.rms_eps, self.dtype)
        m = silu(h2 @ w[p + "w_gate"].T) * (h2 @ w[p + "w_up"].T)
        return x + m @ w[p + "w_down"].T

    def logits(self, x: np.ndarray) -> np.ndarray:
        """LM head of residual-stream rows x [..., d]: final RMSNorm, then the
        (tied or untied) head matrix."""
        xf = rms_norm(x, self.w["final_norm"], self.cfg.rms_eps, self.dtype)
        return xf @ self.head.T

    def _hidden(self, tokens: np.ndarray, segments, rows: str) -> np.ndarray:
        """Residual stream after the last block (before the final norm) of
        every new row, or of each segment's last row."""
        x = self.w["embed"][np.asarray(tokens, dtype=np.int64)]
        for l in range(self.cfg.n_layers):
            x = self._block(l, x, segments)
        if rows == "all":
            return x
        return x[[r0 + n - 1 for _, r0, n in segments]]

    def _run(self, tokens: np.ndarray, segments, rows: str) -> np.ndarray:
        return self.logits(self._hidden(tokens, segments, rows))

    def forward_hidden(self, tokens, cache: KVCache, rows: str = "all") -> np.ndarray:
        """As ``forward``, but returns the residual-stream rows that the LM
        head (``logits``) maps to logits, [T, d] or [1, d]."""
        return self._hidden(np.asarray(tokens), [(cache, 0, len(tokens))], rows)

    def decode_batch_hidden(self, caches, tokens) -> np.ndarray:
        """As ``decode_batch``, but returns the residual-stream rows [n, d]."""
        segs = [(cache, i, 1) for i, cache in enumerate(caches)]
        return self._hidden(np.asarray(tokens), segs, rows="all")

    def forward(self, tokens, cache: KVCache | None = None, rows: str = "all") -> np.ndarray:
        """Append ``tokens`` to one stream's cache (a fresh one if None) and
        return logits of every new row (rows='all', [T, V]) or of the last
        row only (rows='last', [1, V])."""
        tokens = np.asarray(tokens)
        if cache is None:
            cache = self.new_cache()
        return self._run(tokens, [(cache, 0, len(tokens))], rows)

    def prefill(self, tokens, rows: str = "all"):
        """Prompt evaluation from an empty cache; returns (logits, cache)."""
        cache = self.new_cache()
        return self.forward(tokens, cache, rows), cache

    def decode(self, cache: KVCache, token: int) -> np.ndarray:
        """One decode step of one stream: logits [V] of the new position."""
        return self.forward(np.array([token]), cache, rows="all")[0]

    def decode_batch(self, caches, tokens) -> np.ndarray:
        """One lockstep decode step of several independent streams (batched
        linear layers, per-stream attention); logits [n, V]."""
        segs = [(cache, i, 1) for i, cache in enumerate(caches)]
        return self._run(np.asarray(tokens), segs, rows="all")
