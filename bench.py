"""Benchmark of the mouth model's hot path on one MI355X.

One step = one request of the 1B-class bf16 decoder (16 layers, d 2048,
32/8 heads, FFN 8192, vocab 128256): prefill of a 256-token uniform-random
prompt (time to first token), then 256 greedy decode steps whose tokens are
fed back on the device.  Weights are seeded N(0, 0.02^2) random draws rounded
to bf16 (no trained checkpoint exists here); the prompt is uniform random ids.

Prints ONE JSON line: decode tok/s (value), TTFT, the HBM roofline of the
decode step, and the fp64 CPU oracle timed on a bounded sample.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
METRIC = "batch-1 decode tok/s + % HBM roofline; TTFT (ms) for 1B bf16 model"


def decode_bytes_per_token(shape, t_avg: float, kv_elem: int) -> float:
    """Algorithmic HBM bytes of one batch-1 decode token: every weight once
    (bf16) plus the K and V of t positions in every layer."""
    w = shape.n_params() * 2
    kv = shape.n_layers * 2 * shape.n_kv_heads * shape.head_dim * kv_elem * t_avg
    return w + kv


def cpu_baseline(shape, wseed, prompt, n_decode):
    """The fp64 oracle on the host: prefill of the prompt, then n_decode
    cached decode steps; returns decode tok/s, prefill seconds and threads."""
    import oracle
    import synth
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:
        cores = os.cpu_count() or 1
    tensors = synth.make_weights(shape, wseed)
    model = oracle.Decoder(shape, synth.weights_as_f64(shape, tensors))
    del tensors
    t0 = time.perf_counter()
    logits, cache = model.prefill(prompt, rows="last")
    t1 = time.perf_counter()
    tok = int(np.argmax(logits[0]))
    for _ in range(n_decode):
        tok = int(np.argmax(model.decode(cache, tok)))
    t2 = time.perf_counter()
    return n_decode / (t2 - t1), t1 - t0, cores


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-decode-steps", type=int, default=4)
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only: the decoder runs on a single MI355X "
              f"(--gpus {args.gpus} is not supported)", file=sys.stderr)
        sys.exit(2)

    import torch

    import synth
    from paper_2606_12154_amd import hh

    wl = synth.WORKLOADS["1b_decode"]
    shape, P, N = wl["shape"], wl["prompt"], wl["steps"]
    prompt = synth.make_tokens(shape.vocab, P, wl["tseed"])
    tensors = synth.make_weights(shape, wl["wseed"])
    ctx = hh.Context(hh.make_config(shape, 1, P + N + 1, max_prefill=P))
    ctx.load_weights(tensors)
    del tensors
    st = ctx.stream

    def one_step():
        ctx.reset(0)
        t0 = time.perf_counter()
        nxt, _ = ctx.prefill(0, prompt)            # host ids in, host token out
        ttft = time.perf_counter() - t0
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(st)
        for _ in range(N):
            hh.hh_decode_step(ctx.ctx, 1, None, None, None, None)
        e1.record(st)
        e1.synchronize()
        return ttft, e0.elapsed_time(e1) / 1e3

    for _ in range(args.warmup):
        one_step()
    torch.cuda.synchronize()
    ttfts, decs = [], []
    t_start = time.perf_counter()
    for _ in range(args.steps):
        a, b = one_step()
        ttfts.append(a)
        decs.append(b)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    gen = ctx.read_argmax(0, P - 1, N + 1)
    assert gen.min() >= 0 and gen.max() < shape.vocab

    dec_s = float(np.sum(decs))
    tok_s = args.steps * N / dec_s
    t_avg = P + (N + 1) / 2.0
    bpt = decode_bytes_per_token(shape, t_avg, 2)
    achieved = bpt * tok_s / 1e9
    out = {
        "metric": METRIC,
        "value": round(tok_s, 2),
        "unit": "tok/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall / args.steps * 1e3, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"1B bf16 decoder, batch 1, {P}-token uniform-random prompt, "
                               f"{N} greedy decode steps (device-fed)",
                   "prompt": P, "decode_steps": N, "batch": 1},
        "ttft_ms": round(float(np.mean(ttfts)) * 1e3, 3),
        "ttft_ms_min": round(float(np.min(ttfts)) * 1e3, 3),
        "ttft_ms_max": round(float(np.max(ttfts)) * 1e3, 3),
        "decode_ms_per_token": round(dec_s / (args.steps * N) * 1e3, 4),
        "roofline": {"bound": "hbm", "kernel": "decode step (graph)", "achieved": round(achieved, 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": None, "bytes_per_token": int(bpt)},
    }
    ctx.close()
    del ctx
    torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        rate, pre_s, cores = cpu_baseline(shape, wl["wseed"], prompt, args.cpu_decode_steps)
        out["cpu_baseline"] = {"value": round(rate, 4), "unit": "tok/s", "cores": cores, "kind": "oracle",
                               "sample": f"fp64 oracle: prefill {P} tokens ({pre_s:.2f} s, untimed for the value) "
                                         f"then {args.cpu_decode_steps} cached decode steps"}
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
