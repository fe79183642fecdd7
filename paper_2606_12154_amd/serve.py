"""The serving path around the decoder (the paper's runtime phase, §4):
route the question to a stored entry (native BM25 with the margin gate,
§6.3), render the entry's answer in the marker-line envelope (§6.4), and
stream the decoder's greedy continuation token by token, timing the
quantities §6.2 keeps apart: time to first token, decode rate, end-to-end
throughput.

Routing and rendering run in the native library (``include/hh_router.h``);
this module strings the calls together.  The prompt's token ids come from a
byte-level stand-in tokenizer (id = 3 + byte): the decoder's weights are
seeded random tensors with no trained vocabulary, so only the lengths and the
timing of the streamed tokens are meaningful, not their text.
"""
from __future__ import annotations

import time
from dataclasses import dataclass, field
from typing import Iterator, List, Optional, Sequence

import numpy as np

from . import hh

TAU = 0.05  # margin threshold of the confidence gate (§6.3)


def _token(tok: int) -> int:
    """A streamed id; -1 is the library's mark of a decode step that gave up
    waiting (the context yields -1 until it is reset)."""
    if tok < 0:
        raise RuntimeError("decode step failed (a bounded wait timed out); reset the context")
    return tok


def byte_tokens(prompt: bytes) -> np.ndarray:
    """Stand-in tokenizer: one id per byte, ids 3..258 (0..2 stay free)."""
    return np.frombuffer(prompt, dtype=np.uint8).astype(np.int32) + 3


class Router:
    """A native BM25 index over the store's entry texts."""

    def __init__(self, texts: Sequence[str], k1: float = 1.2, b: float = 0.75):
        self.handle = hh.hh_router_create(texts, k1, b)

    def top(self, query: str, k: int = 3):
        return hh.hh_router_query(self.handle, query, k)

    def route(self, query: str, tau: float = TAU):
        return hh.hh_router_route(self.handle, query, tau)

    def close(self) -> None:
        if self.handle:
            hh.hh_router_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


@dataclass
class Answer:
    """One served query: the route, the streamed token ids and the clocks
    (seconds, host wall time from the query's arrival)."""
    entry: int
    margin: float
    escalated: bool
    tokens: List[int] = field(default_factory=list)
    t_route: float = 0.0
    t_render: float = 0.0
    t_first: float = 0.0
    t_last: float = 0.0
    prompt_tokens: int = 0

    @property
    def ttft_ms(self) -> float:
        return self.t_first * 1e3

    @property
    def decode_tok_s(self) -> float:
        n = len(self.tokens) - 1
        return n / (self.t_last - self.t_first) if n > 0 and self.t_last > self.t_first else 0.0

    @property
    def e2e_tok_s(self) -> float:
        return len(self.tokens) / self.t_last if self.t_last > 0 else 0.0


class Server:
    """Route, render and stream on one decoder stream of a library context.

    Decode steps are device-fed (each consumes the previous step's argmax on
    the GPU); every step's token is copied into pinned host memory behind an
    event, and ``stream`` yields tokens in order as their events complete, so
    the host sees each token as soon as its step ends while later steps are
    already queued."""

    def __init__(self, ctx: "hh.Context", router: Router, answers: Sequence[str], max_tokens: int,
                 stream_id: int = 0, tau: float = TAU, max_batch: int = 1):
        import torch
        self.torch = torch
        self.ctx, self.router, self.answers = ctx, router, list(answers)
        self.stream_id, self.tau, self.max_tokens = stream_id, tau, max_tokens
        self.max_batch = max_batch
        # Token slots [step][request]; one event per step.
        self.dev = torch.zeros((max_tokens, max_batch), dtype=torch.int32, device=ctx.device)
        self.host = torch.zeros((max_tokens, max_batch), dtype=torch.int32, pin_memory=True)
        self.events = [torch.cuda.Event() for _ in range(max_tokens)]
        self.ids = np.array([stream_id], dtype=np.int32)

    def stream(self, query: str, n_tokens: int, ans: Optional[Answer] = None) -> Iterator[int]:
        """Yields the answer's token ids as they reach host memory; fills
        ``ans`` (route, clocks) on the way.  An escalated query yields nothing."""
        if not 1 <= n_tokens <= self.max_tokens:
            raise ValueError(f"n_tokens must be in 1..{self.max_tokens}")
        torch = self.torch
        t0 = time.perf_counter()
        entry, margin, esc = self.router.route(query, self.tau)
        a = ans if ans is not None else Answer(entry, margin, esc)
        a.entry, a.margin, a.escalated = entry, margin, esc
        a.t_route = time.perf_counter() - t0
        if esc:
            return
        ids = byte_tokens(hh.hh_render_marker(self.answers[entry]))
        a.prompt_tokens = len(ids)
        a.t_render = time.perf_counter() - t0
        self.ctx.reset(self.stream_id)
        first, _ = self.ctx.prefill(self.stream_id, ids)  # returns once the first token is on the host
        first = _token(first)
        a.t_first = time.perf_counter() - t0
        a.tokens.append(first)
        yield first
        st = self.ctx.stream
        with torch.cuda.stream(st):
            for i in range(1, n_tokens):
                hh.hh_decode_step(self.ctx.ctx, 1, self.ids, None, None, self.dev[i].data_ptr())
                self.host[i, 0:1].copy_(self.dev[i, 0:1], non_blocking=True)
                self.events[i].record(st)
        for i in range(1, n_tokens):
            self.events[i].synchronize()
            tok = _token(int(self.host[i, 0]))
            a.tokens.append(tok)
            a.t_last = time.perf_counter() - t0
            yield tok
        if n_tokens == 1:
            a.t_last = a.t_first

    def answer(self, query: str, n_tokens: int) -> Answer:
        a = Answer(-1, 0.0, False)
        for _ in self.stream(query, n_tokens, a):
            pass
        return a

    def answer_batch(self, queries: Sequence[str], n_tokens: int, streams: Sequence[int]) -> List[Answer]:
        """Serve several queries at once: each routed query is rendered into
        its own decoder stream (``streams[i]`` for query i), the prompts are
        prefilled together (passes of the library's multi-stream prefill),
        then all of them decode in lockstep (one multi-stream step per token,
        device-fed), every step's tokens copied behind one event.  Escalated
        queries take no stream time.  Clocks run from the batch's arrival."""
        if not 1 <= n_tokens <= self.max_tokens:
            raise ValueError(f"n_tokens must be in 1..{self.max_tokens}")
        if len(queries) != len(streams) or len(queries) > self.max_batch:
            raise ValueError(f"need one stream per query and at most {self.max_batch} queries")
        torch = self.torch
        t0 = time.perf_counter()
        out: List[Answer] = []
        live: List[int] = []
        for i, q in enumerate(queries):
            entry, margin, esc = self.router.route(q, self.tau)
            a = Answer(entry, margin, esc)
            a.t_route = time.perf_counter() - t0
            out.append(a)
            if not esc:
                live.append(i)
        prompts = {}
        for i in live:
            a = out[i]
            prompts[i] = byte_tokens(hh.hh_render_marker(self.answers[a.entry]))
            a.prompt_tokens = len(prompts[i])
            a.t_render = time.perf_counter() - t0
            self.ctx.reset(streams[i])
        # One call for all prompts; the library runs as many passes as the
        # rows need (a prompt longer than a pass continues in the next one).
        if live:
            firsts = self.ctx.prefill_batch([streams[i] for i in live], [prompts[i] for i in live])
            now = time.perf_counter() - t0
            for i, f in zip(live, firsts):
                out[i].t_first = now
                out[i].tokens.append(_token(int(f)))
        n = len(live)
        if n == 0 or n_tokens == 1:
            for i in live:
                out[i].t_last = out[i].t_first
            return out
        sids = np.array([streams[i] for i in live], dtype=np.int32)
        st = self.ctx.stream
        with torch.cuda.stream(st):
            for k in range(1, n_tokens):
                hh.hh_decode_step(self.ctx.ctx, n, sids, None, None, self.dev[k].data_ptr())
                self.host[k, :n].copy_(self.dev[k, :n], non_blocking=True)
                self.events[k].record(st)
        for k in range(1, n_tokens):
            self.events[k].synchronize()
            now = time.perf_counter() - t0
            row = self.host[k, :n].tolist()
            for j, i in enumerate(live):
                out[i].tokens.append(_token(int(row[j])))
                out[i].t_last = now
        return out
