"""ctypes binding of the C ABI in include/hh.h (argument marshalling only).

The module-level functions carry the C names and signatures one to one; the
``Context`` class strings them together for tests and benchmarks, allocating
the device arena and the HIP stream through PyTorch.  Every step of the
decoder runs in the HIP library: if ``libhh.so`` is missing or cannot be
loaded, ``load_library`` raises, and nothing falls back to another
implementation.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, byref, c_float, c_int32, c_size_t, c_void_p

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libhh.so")

HH_OK, HH_ERR_INVALID_ARG, HH_ERR_OOM, HH_ERR_CONTEXT_FULL = 0, -1, -2, -3
HH_ERR_NOT_LOADED, HH_ERR_HIP, HH_ERR_UNSUPPORTED = -4, -5, -6
HH_F32, HH_BF16 = 0, 1
HH_LOGITS_NONE, HH_LOGITS_LAST, HH_LOGITS_ALL = 0, 1, 2
HH_WF_DTYPE, HH_WF_Q4G32 = 0, 1

EXPORTED = ["hh_workspace_size", "hh_create", "hh_load_weights", "hh_prefill", "hh_prefill_batch", "hh_decode_step",
            "hh_decode_step_noalloc", "hh_reset", "hh_stream_length", "hh_read_argmax", "hh_destroy", "hh_last_error",
            "hh_q4g32_quantize", "hh_router_create", "hh_router_query", "hh_router_route",
            "hh_router_size", "hh_router_destroy", "hh_render_marker", "hh_read_probe"]


class hh_config(ctypes.Structure):
    _fields_ = [(n, c_int32) for n in ("n_layers", "d_model", "n_heads", "n_kv_heads", "head_dim",
                                        "ffn_dim", "vocab")] + [
        ("rms_eps", c_float), ("rope_theta", c_float),
        ("tied_embeddings", c_int32), ("dtype", c_int32), ("max_streams", c_int32),
        ("max_context", c_int32), ("page_size", c_int32), ("max_prefill", c_int32),
        ("weight_format", c_int32)]


class HHError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"hh status {status}: {msg}")
        self.status = status


_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libhh.so (built by paper_2606_12154_amd/build.py); raises if absent."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"HIP library not built: {path} (run paper_2606_12154_amd/build.py)")
    lib = ctypes.CDLL(path)
    i32p = POINTER(c_int32)
    sig = {
        "hh_workspace_size": ([POINTER(hh_config), POINTER(c_size_t)], c_int32),
        "hh_create": ([POINTER(hh_config), c_void_p, c_size_t, c_void_p, POINTER(c_void_p)], c_int32),
        "hh_load_weights": ([c_void_p, POINTER(c_void_p), c_int32], c_int32),
        "hh_prefill": ([c_void_p, c_int32, i32p, c_int32, c_int32, c_void_p, c_void_p], c_int32),
        "hh_decode_step": ([c_void_p, c_int32, i32p, i32p, c_void_p, c_void_p], c_int32),
        "hh_prefill_batch": ([c_void_p, c_int32, i32p, i32p, i32p, c_void_p], c_int32),
        "hh_decode_step_noalloc": ([c_void_p, c_int32, i32p, c_void_p, c_void_p], c_int32),
        "hh_reset": ([c_void_p, c_int32], c_int32),
        "hh_stream_length": ([c_void_p, c_int32, i32p], c_int32),
        "hh_read_argmax": ([c_void_p, c_int32, c_int32, c_int32, i32p], c_int32),
        "hh_destroy": ([c_void_p], None),
        "hh_last_error": ([c_void_p], ctypes.c_char_p),
        "hh_q4g32_quantize": ([c_void_p, ctypes.c_int64, c_int32, c_void_p, c_void_p], c_int32),
        "hh_router_create": ([POINTER(ctypes.c_char_p), c_int32, c_float, c_float, POINTER(c_void_p)], c_int32),
        "hh_router_query": ([c_void_p, ctypes.c_char_p, c_int32, i32p, POINTER(ctypes.c_double), i32p], c_int32),
        "hh_router_route": ([c_void_p, ctypes.c_char_p, c_float, i32p, POINTER(ctypes.c_double), i32p], c_int32),
        "hh_router_size": ([c_void_p, i32p, i32p], c_int32),
        "hh_router_destroy": ([c_void_p], None),
        "hh_render_marker": ([ctypes.c_char_p, c_void_p, ctypes.c_int64, POINTER(ctypes.c_int64)], c_int32),
        "hh_read_probe": ([c_void_p, c_size_t, c_void_p], c_int32),
    }
    for name, (args, res) in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = res
    _lib = lib
    return lib


# ------------------------------------------------------------ C names, 1:1

def hh_workspace_size(cfg: hh_config) -> int:
    n = c_size_t()
    _check(None, load_library().hh_workspace_size(byref(cfg), byref(n)))
    return n.value


def hh_create(cfg: hh_config, arena_ptr: int, arena_bytes: int, hip_stream: int) -> int:
    ctx = c_void_p()
    _check(None, load_library().hh_create(byref(cfg), c_void_p(arena_ptr), arena_bytes,
                                          c_void_p(hip_stream), byref(ctx)))
    return ctx.value


def hh_load_weights(ctx: int, ptrs) -> None:
    arr = (c_void_p * len(ptrs))(*ptrs)
    _check(ctx, load_library().hh_load_weights(ctx, arr, len(ptrs)))


def hh_prefill(ctx: int, stream_id: int, tokens: np.ndarray, logits_mode: int, logits_ptr, next_ptr) -> None:
    tokens = np.ascontiguousarray(tokens, dtype=np.int32)
    _check(ctx, load_library().hh_prefill(ctx, stream_id, tokens.ctypes.data_as(POINTER(c_int32)), len(tokens),
                                          logits_mode, logits_ptr, next_ptr))


def hh_prefill_batch(ctx: int, stream_ids, prompts, next_ptr) -> None:
    ids = np.ascontiguousarray(stream_ids, dtype=np.int32)
    lens = np.array([len(p) for p in prompts], dtype=np.int32)
    toks = np.ascontiguousarray(np.concatenate([np.asarray(p, dtype=np.int32) for p in prompts])
                                if len(prompts) else np.zeros(0, np.int32), dtype=np.int32)
    _check(ctx, load_library().hh_prefill_batch(ctx, len(ids), ids.ctypes.data_as(POINTER(c_int32)),
                                                lens.ctypes.data_as(POINTER(c_int32)),
                                                toks.ctypes.data_as(POINTER(c_int32)), next_ptr))


def hh_decode_step(ctx: int, n_streams: int, stream_ids, tokens, logits_ptr, next_ptr) -> None:
    ids = None if stream_ids is None else np.ascontiguousarray(stream_ids, dtype=np.int32)
    tok = None if tokens is None else np.ascontiguousarray(tokens, dtype=np.int32)
    _check(ctx, load_library().hh_decode_step(
        ctx, n_streams, None if ids is None else ids.ctypes.data_as(POINTER(c_int32)),
        None if tok is None else tok.ctypes.data_as(POINTER(c_int32)), logits_ptr, next_ptr))


def hh_decode_step_noalloc(ctx: int, stream_id: int, token, logits_ptr, next_ptr) -> None:
    tok = None if token is None else np.array([token], dtype=np.int32)
    _check(ctx, load_library().hh_decode_step_noalloc(
        ctx, stream_id, None if tok is None else tok.ctypes.data_as(POINTER(c_int32)), logits_ptr, next_ptr))


def hh_reset(ctx: int, stream_id: int) -> None:
    _check(ctx, load_library().hh_reset(ctx, stream_id))


def hh_stream_length(ctx: int, stream_id: int) -> int:
    n = c_int32()
    _check(ctx, load_library().hh_stream_length(ctx, stream_id, byref(n)))
    return n.value


def hh_read_argmax(ctx: int, stream_id: int, first_pos: int, n: int) -> np.ndarray:
    out = np.zeros(n, dtype=np.int32)
    _check(ctx, load_library().hh_read_argmax(ctx, stream_id, first_pos, n, out.ctypes.data_as(POINTER(c_int32))))
    return out


def hh_destroy(ctx: int) -> None:
    load_library().hh_destroy(ctx)


def hh_last_error(ctx: int) -> str:
    return load_library().hh_last_error(ctx).decode()


def hh_q4g32_quantize(src_ptr: int, rows: int, K: int, dst_ptr: int, hip_stream: int) -> None:
    _check(None, load_library().hh_q4g32_quantize(c_void_p(src_ptr), rows, K, c_void_p(dst_ptr),
                                                  c_void_p(hip_stream)))


def hh_read_probe(src_ptr: int, nbytes: int, hip_stream: int) -> None:
    _check(None, load_library().hh_read_probe(c_void_p(src_ptr), nbytes, c_void_p(hip_stream)))


def _text(s) -> bytes:
    return s.encode() if isinstance(s, str) else bytes(s)


def hh_router_create(entries, k1: float = 1.2, b: float = 0.75) -> int:
    raw = [_text(e) for e in entries]
    arr = (ctypes.c_char_p * len(raw))(*raw)
    r = c_void_p()
    _check(None, load_library().hh_router_create(arr, len(raw), k1, b, byref(r)))
    return r.value


def hh_router_query(router: int, query, k: int):
    """Returns (ids int32 array, scores float64 array), best first."""
    ids = np.zeros(max(k, 1), dtype=np.int32)
    sc = np.zeros(max(k, 1), dtype=np.float64)
    n = c_int32()
    _check(None, load_library().hh_router_query(router, _text(query), k, ids.ctypes.data_as(POINTER(c_int32)),
                                                sc.ctypes.data_as(POINTER(ctypes.c_double)), byref(n)))
    return ids[:n.value], sc[:n.value]


def hh_router_route(router: int, query, tau: float = 0.05):
    """Returns (entry, margin, escalate)."""
    e, m, x = c_int32(), ctypes.c_double(), c_int32()
    _check(None, load_library().hh_router_route(router, _text(query), tau, byref(e), byref(m), byref(x)))
    return e.value, m.value, bool(x.value)


def hh_router_size(router: int):
    n, t = c_int32(), c_int32()
    _check(None, load_library().hh_router_size(router, byref(n), byref(t)))
    return n.value, t.value


def hh_router_destroy(router: int) -> None:
    load_library().hh_router_destroy(router)


def hh_render_marker(answer) -> bytes:
    need = ctypes.c_int64()
    lib = load_library()
    a = _text(answer)
    lib.hh_render_marker(a, None, 0, byref(need))
    buf = ctypes.create_string_buffer(max(need.value, 1))
    _check(None, lib.hh_render_marker(a, buf, need.value, byref(need)))
    return buf.raw[:need.value]


def _check(ctx, status: int) -> None:
    if status != HH_OK:
        raise HHError(status, hh_last_error(ctx) if ctx else "")


# ------------------------------------------------------------ convenience

def make_config(shape, max_streams: int, max_context: int, max_prefill: int = 0,
                weight_format: int = 0) -> hh_config:
    """hh_config from a model-shape object (attributes as in synth.ModelShape)."""
    return hh_config(shape.n_layers, shape.d_model, shape.n_heads, shape.n_kv_heads, shape.head_dim,
                     shape.ffn_dim, shape.vocab, shape.rms_eps, shape.rope_theta, int(shape.tied),
                     int(shape.dtype), max_streams, max_context, 16, max_prefill, weight_format)


class Context:
    """One library context inside a torch-allocated device arena and stream."""

    def __init__(self, cfg: hh_config, device: str = "cuda:0"):
        import torch
        self.torch = torch
        self.cfg = cfg
        self.device = torch.device(device)
        self.bytes = hh_workspace_size(cfg)
        self.arena = torch.empty(self.bytes, dtype=torch.uint8, device=self.device)
        self.stream = torch.cuda.Stream(device=self.device)  # default priority
        self.ctx = hh_create(cfg, self.arena.data_ptr(), self.bytes, self.stream.cuda_stream)

    def load_weights(self, tensors) -> None:
        """tensors: numpy arrays (host) or torch tensors (any device), C-ABI order."""
        keep = [t if not isinstance(t, np.ndarray) else np.ascontiguousarray(t) for t in tensors]
        ptrs = [t.ctypes.data if isinstance(t, np.ndarray) else t.data_ptr() for t in keep]
        hh_load_weights(self.ctx, ptrs)

    def prefill(self, stream_id: int, tokens, logits: str = "none"):
        """Returns (next_token, logits ndarray or None) in host memory."""
        n = len(tokens)
        V = self.cfg.vocab
        mode = {"none": HH_LOGITS_NONE, "last": HH_LOGITS_LAST, "all": HH_LOGITS_ALL}[logits]
        buf = None
        if mode == HH_LOGITS_LAST:
            buf = np.empty(V, dtype=np.float32)
        elif mode == HH_LOGITS_ALL:
            buf = np.empty((n, V), dtype=np.float32)
        nxt = np.zeros(1, dtype=np.int32)
        hh_prefill(self.ctx, stream_id, tokens, mode, None if buf is None else buf.ctypes.data,
                   nxt.ctypes.data)
        return int(nxt[0]), buf

    def prefill_batch(self, stream_ids, prompts) -> np.ndarray:
        """Prompts of several streams in one pass; returns their next tokens."""
        nxt = np.zeros(len(stream_ids), dtype=np.int32)
        hh_prefill_batch(self.ctx, stream_ids, prompts, nxt.ctypes.data)
        return nxt

    def decode_step(self, stream_ids=None, tokens=None, logits: bool = False, n_streams: int | None = None,
                    host_next: bool = True):
        """One lockstep step; returns (next tokens or None, logits or None)."""
        n = n_streams if n_streams is not None else (len(stream_ids) if stream_ids is not None else 1)
        buf = np.empty((n, self.cfg.vocab), dtype=np.float32) if logits else None
        nxt = np.zeros(n, dtype=np.int32) if host_next else None
        hh_decode_step(self.ctx, n, stream_ids, tokens, None if buf is None else buf.ctypes.data,
                       None if nxt is None else nxt.ctypes.data)
        return nxt, buf

    def reset(self, stream_id: int = -1) -> None:
        hh_reset(self.ctx, stream_id)

    def length(self, stream_id: int) -> int:
        return hh_stream_length(self.ctx, stream_id)

    def read_argmax(self, stream_id: int, first_pos: int, n: int) -> np.ndarray:
        return hh_read_argmax(self.ctx, stream_id, first_pos, n)

    def synchronize(self) -> None:
        self.stream.synchronize()

    def close(self) -> None:
        if self.ctx:
            hh_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
