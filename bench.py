"""Benchmark of the mouth model's hot path on one MI355X.

Headline workload (one "step" = one request): the 1B-class bf16 decoder (16
layers, d 2048, 32/8 heads, FFN 8192, vocab 128256) prefills a 256-token
uniform-random prompt (time to first token) and then runs 256 greedy decode
steps whose tokens are fed back on the device.  Weights are seeded N(0, 0.02^2)
draws rounded to bf16 (no trained checkpoint exists here); prompts are uniform
random ids, which stand in exactly for the paper's rendered-answer prompts
because a dense decoder's cost depends only on lengths.

Printed: ONE JSON line with decode tok/s (value), TTFT, the HBM roofline of
the persistent decode-step kernel (one launch per token, timed with HIP events
on the library's stream) and the fp64 CPU oracle timed on a bounded sample.
The same line carries the three other 1B workloads, measured on the same
context: the 1024-token prompt's TTFT and its MFMA fraction (device time of
the prefill against the dense fp16 peak), decode over 8192 cached positions
and 32 lockstep streams, each with its HBM fraction.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
MFMA_PEAK_FLOPS = 2.5166e15  # dense fp16/bf16: 256 CUs x 2.4 GHz x 4096 FLOP per clock
METRIC = "batch-1 decode tok/s + % HBM roofline; TTFT (ms) for 1B bf16 model"
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "decode_step_1b_traffic.json")
STEP_SOURCES = ["paper_2606_12154_amd/csrc/k_step.hip", "paper_2606_12154_amd/csrc/hh_device.h",
                "paper_2606_12154_amd/csrc/hh_kernels.h"]


def step_source_hash() -> str:
    h = hashlib.sha256()
    for p in STEP_SOURCES:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def kv_bytes_per_position(shape) -> int:
    """fp16 K and V of one position in every layer (the cache's element type)."""
    return shape.n_layers * 2 * shape.n_kv_heads * shape.head_dim * 2


def decode_step_bytes(shape, t: float) -> float:
    """Algorithmic HBM bytes of one batch-1 decode launch attending t
    positions: every bf16 weight once, the K/V of t positions, and the new
    position's K/V write."""
    return shape.n_params() * 2 + kv_bytes_per_position(shape) * (t + 1)


def measured_traffic(launch_bytes: float):
    """HBM bytes per decode-step launch from the committed counter profile,
    or None when absent or taken on a different version of the kernel."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("source_sha256") != step_source_hash():
        return None
    return rec.get("bytes_per_launch")


def cpu_baseline(shape, wseed, prompt, n_decode):
    """The oracle on the host, in its fp64 working precision and again in
    fp32: prefill of the prompt, then n_decode cached decode steps.  Returns
    {precision: (decode tok/s, prefill seconds)} and the threads used."""
    import oracle
    import synth
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:
        cores = os.cpu_count() or 1
    w64 = synth.weights_as_f64(shape, synth.make_weights(shape, wseed))
    out = {}
    for name, dt in (("fp64", np.float64), ("fp32", np.float32)):
        model = oracle.Decoder(shape, w64, dtype=dt)
        t0 = time.perf_counter()
        logits, cache = model.prefill(prompt, rows="last")
        t1 = time.perf_counter()
        tok = int(np.argmax(logits[0]))
        for _ in range(n_decode):
            tok = int(np.argmax(model.decode(cache, tok)))
        t2 = time.perf_counter()
        out[name] = (n_decode / (t2 - t1), t1 - t0)
        del model, cache
    return out, cores


def prefill_flops(shape, P: int) -> float:
    """Algorithmic FLOPs of a P-token prompt evaluation: every projection of
    every row (2 per weight), causal attention (Q K^T and P V over the
    P (P + 1) / 2 visible pairs of every head) and the LM head of the last row."""
    d, hd = shape.d_model, shape.head_dim
    lin = shape.n_layers * (d * (shape.q_dim + 2 * shape.kv_dim) + shape.q_dim * d + 3 * d * shape.ffn_dim)
    attn = shape.n_layers * shape.n_heads * 4 * hd * P * (P + 1) / 2
    return 2.0 * lin * P + attn + 2.0 * shape.vocab * d


def measure_others(ctx, shape, st, names):
    """The other workloads on the same context: 1024-token TTFT, decode over
    8192 cached positions, 32-stream lockstep decode."""
    import torch

    import synth
    from paper_2606_12154_amd import hh
    other = {}
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    if "prompt1024" in names:
        # 1024-token prompt: TTFT (the prefill-dominated workload), then 64
        # steps.  TTFT is host to host (token ids in, first id out); the
        # MFMA fraction uses the prefill's device time (events on the
        # library's stream around the same call).
        w3 = synth.WORKLOADS["1b_prefill"]
        p3 = synth.make_tokens(shape.vocab, w3["prompt"], w3["tseed"])
        tt, dev = [], []
        for i in range(6):
            ctx.reset(0)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            e0.record(st)
            ctx.prefill(0, p3)
            e1.record(st)
            t1 = time.perf_counter()
            e1.synchronize()
            if i:
                tt.append(t1 - t0)
                dev.append(e0.elapsed_time(e1) / 1e3)
        e0.record(st)
        for _ in range(w3["steps"]):
            hh.hh_decode_step(ctx.ctx, 1, None, None, None, None)
        e1.record(st)
        e1.synchronize()
        fl = prefill_flops(shape, w3["prompt"])
        other["prompt1024"] = {"ttft_ms": round(float(np.mean(tt)) * 1e3, 3),
                               "ttft_ms_min": round(float(np.min(tt)) * 1e3, 3),
                               "prefill_device_ms": round(float(np.mean(dev)) * 1e3, 3),
                               "prefill_flop": fl,
                               "prefill_tflops": round(fl / float(np.mean(dev)) / 1e12, 1),
                               "mfma_frac": round(fl / float(np.mean(dev)) / MFMA_PEAK_FLOPS, 4),
                               "decode_tok_s": round(w3["steps"] / (e0.elapsed_time(e1) / 1e3), 1)}

    if "cache8192" in names:
        # 8192 positions already cached (untimed prefill), then 512 decode steps.
        w4 = synth.WORKLOADS["1b_long"]
        ctx.reset(0)
        ctx.prefill(0, synth.make_tokens(shape.vocab, w4["prompt"], w4["tseed"]))
        e0.record(st)
        for _ in range(w4["steps"]):
            hh.hh_decode_step(ctx.ctx, 1, None, None, None, None)
        e1.record(st)
        e1.synchronize()
        s4 = e0.elapsed_time(e1) / 1e3
        t4 = w4["prompt"] + (w4["steps"] - 1) / 2.0 + 1
        b4 = decode_step_bytes(shape, t4)
        other["cache8192"] = {"decode_tok_s": round(w4["steps"] / s4, 1),
                              "ms_per_token": round(s4 / w4["steps"] * 1e3, 4),
                              "bytes_per_token": int(b4),
                              "hbm_frac": round(b4 * w4["steps"] / s4 / 1e9 / HBM_PEAK_GBS, 4)}

    if "streams32" in names:
        # 32 independent streams, 256-token prompts, lockstep decode.
        w5 = synth.WORKLOADS["1b_multi"]
        ctx.reset(-1)
        ns = w5["streams"]
        for s_ in range(ns):
            ctx.prefill(s_, synth.make_tokens(shape.vocab, w5["prompt"], w5["tseed"] + s_))
        hh.hh_decode_step(ctx.ctx, ns, None, None, None, None)  # first step captures the graph
        e0.record(st)
        n5 = w5["steps"] - 1
        for _ in range(n5):
            hh.hh_decode_step(ctx.ctx, ns, None, None, None, None)
        e1.record(st)
        e1.synchronize()
        s5 = e0.elapsed_time(e1) / 1e3
        t5 = w5["prompt"] + 1 + n5 / 2.0 + 1
        b5 = shape.n_params() * 2 + ns * kv_bytes_per_position(shape) * (t5 + 1)
        other["streams32"] = {"aggregate_tok_s": round(ns * n5 / s5, 1), "step_ms": round(s5 / n5 * 1e3, 3),
                              "bytes_per_step": int(b5),
                              "hbm_frac": round(b5 * n5 / s5 / 1e9 / HBM_PEAK_GBS, 4)}
    return other


def q4_step_bytes(shape, t: float) -> float:
    """Algorithmic HBM bytes of one batch-1 decode launch of the 4-bit model:
    every streamed matrix's stored rows (K / 2 bytes of codes + K / 16 of
    bf16 scales per row of K = d_model), the K/V of t positions, the new
    position's K/V write and the embedding row read."""
    d = shape.d_model
    rows = shape.vocab + shape.n_layers * (shape.q_dim + 2 * shape.kv_dim + d + 3 * shape.ffn_dim)
    return rows * (d // 2 + d // 16) + kv_bytes_per_position(shape) * (t + 1) + 2 * d


def measure_q4_decode(shape):
    """The bench workload (256-token prompt, 256 device-fed greedy steps) on
    the 4-bit model (HH_WF_Q4G32, quantized at load from the same seeded
    bf16 weights): TTFT and decode rate, and the HBM fraction of the
    4-bit stream."""
    import torch

    import synth
    from paper_2606_12154_amd import hh
    wl = synth.WORKLOADS["1b_decode"]
    P, N = wl["prompt"], wl["steps"]
    tensors = synth.make_weights(shape, wl["wseed"])
    ctx = hh.Context(hh.make_config(shape, 1, P + N + 8, P, weight_format=hh.HH_WF_Q4G32))
    ctx.load_weights(tensors)
    del tensors
    st = ctx.stream
    prompt = synth.make_tokens(shape.vocab, P, wl["tseed"])
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    tt, ms = [], []
    for rep in range(4):
        ctx.reset(0)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        ctx.prefill(0, prompt)
        tt.append(time.perf_counter() - t0)
        e0.record(st)
        for _ in range(N):
            hh.hh_decode_step(ctx.ctx, 1, None, None, None, None)
        e1.record(st)
        e1.synchronize()
        ms.append(e0.elapsed_time(e1) / N)
    ctx.close()
    tt, ms = tt[1:], ms[1:]
    sec = float(np.mean(ms)) / 1e3
    b = q4_step_bytes(shape, P + (N - 1) / 2.0 + 1)
    return {"decode_tok_s": round(1.0 / sec, 1), "ms_per_token": round(sec * 1e3, 4),
            "ttft_ms": round(float(np.mean(tt)) * 1e3, 3), "bytes_per_token": int(b),
            "hbm_frac": round(b / sec / 1e9 / HBM_PEAK_GBS, 4)}


def measure_ctx_sweep(shape):
    """Decode rate against the number of cached positions (the paper's window
    sweep, here over positions actually attended): a 1-stream context of
    131072 positions; for each length a seeded prompt fills the cache
    (untimed), then 64 device-fed decode steps are timed."""
    import torch

    import synth
    from paper_2606_12154_amd import hh
    steps = 64
    tensors = synth.make_weights(shape, synth.WORKLOADS["1b_decode"]["wseed"])
    ctx = hh.Context(hh.make_config(shape, 1, 131072, 8192))
    ctx.load_weights(tensors)
    del tensors
    st = ctx.stream
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    rows = []
    for n in (1024, 2048, 4096, 8192, 16384, 32768, 65536, 131072 - steps):
        ctx.reset(0)
        ctx.prefill(0, synth.make_tokens(shape.vocab, n, 500 + n))
        hh.hh_decode_step(ctx.ctx, 1, None, None, None, None)
        e0.record(st)
        for _ in range(steps - 1):
            hh.hh_decode_step(ctx.ctx, 1, None, None, None, None)
        e1.record(st)
        e1.synchronize()
        sec = e0.elapsed_time(e1) / 1e3
        t = n + 1 + (steps - 2) / 2.0 + 1
        b = decode_step_bytes(shape, t)
        rows.append({"cached": n, "decode_tok_s": round((steps - 1) / sec, 1),
                     "ms_per_token": round(sec / (steps - 1) * 1e3, 4),
                     "hbm_frac": round(b * (steps - 1) / sec / 1e9 / HBM_PEAK_GBS, 4)})
        print(json.dumps(rows[-1]), file=sys.stderr, flush=True)
    ctx.close()
    return rows


def measure_windows(shape):
    """The paper's window sweep as stated (allocated context, short use): for
    windows of 4K..128K positions, the arena the library asks for and the
    decode rate of the bench request (256-token prompt, 256 device-fed
    steps) in a context of that window.  The bf16 weights are uploaded once
    and loaded from device memory into each context."""
    import torch

    import synth
    from paper_2606_12154_amd import hh
    wl = synth.WORKLOADS["1b_decode"]
    P, N = wl["prompt"], wl["steps"]
    tensors = [torch.from_numpy(np.ascontiguousarray(t).view(np.int16) if t.dtype == np.uint16 else np.ascontiguousarray(t))
               for t in synth.make_weights(shape, wl["wseed"])]
    dev = [t.to("cuda") for t in tensors]
    del tensors
    prompt = synth.make_tokens(shape.vocab, P, wl["tseed"])
    rows = []
    for w in (4096, 8192, 16384, 32768, 65536, 131072):
        cfg = hh.make_config(shape, 1, w, P)
        ctx = hh.Context(cfg)
        ctx.load_weights(dev)
        st = ctx.stream
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        ms = []
        for rep in range(3):
            ctx.reset(0)
            ctx.prefill(0, prompt)
            e0.record(st)
            for _ in range(N):
                hh.hh_decode_step(ctx.ctx, 1, None, None, None, None)
            e1.record(st)
            e1.synchronize()
            ms.append(e0.elapsed_time(e1) / N)
        ctx.close()
        del ctx
        sec = float(np.mean(ms[1:])) / 1e3
        rows.append({"window": w, "arena_bytes": int(hh.hh_workspace_size(cfg)),
                     "decode_tok_s": round(1.0 / sec, 1), "ms_per_token": round(sec * 1e3, 4)})
        print(json.dumps(rows[-1]), file=sys.stderr, flush=True)
    return rows


def measure_e2e(shape):
    """The serving path around the decoder (route, render, stream) on a
    synthetic store shaped like the paper's routing study (563 entries from
    17 documents, 1,126 queries drawn from entry vocabulary): routing
    accuracy, gate rate and route latency over all queries (native BM25 on
    the host), then 16 routed queries served end to end by the 1B bf16
    decoder, 64 streamed tokens each: TTFT (query to first token on the
    host), decode rate and end-to-end throughput, medians; then 32 routed
    queries served at once (lockstep decode over 32 streams)."""
    import synth
    from paper_2606_12154_amd import hh, serve
    store = synth.make_store()
    queries = synth.make_queries(store)
    router = serve.Router([t for t, _ in store])
    hit1 = hit3 = esc = ok = 0
    lat = []
    for q, want in queries:
        ids, _ = router.top(q, 3)
        hit1 += int(ids[0] == want)
        hit3 += int(want in ids)
        t0 = time.perf_counter()
        e, m, x = router.route(q)
        lat.append(time.perf_counter() - t0)
        esc += int(x)
        ok += int((not x) and e == want)
    nq = len(queries)
    routing = {"entries": len(store), "queries": nq, "top1": round(hit1 / nq, 4), "top3": round(hit3 / nq, 4),
               "escalated": round(esc / nq, 4), "top1_of_answered": round(ok / max(1, nq - esc), 4),
               "route_us_p50": round(float(np.median(lat)) * 1e6, 2)}
    wl = synth.WORKLOADS["1b_decode"]
    tensors = synth.make_weights(shape, wl["wseed"])
    ctx = hh.Context(hh.make_config(shape, 32, 4096, 4096))
    ctx.load_weights(tensors)
    del tensors
    srv = serve.Server(ctx, router, [a for _, a in store], max_tokens=64, max_batch=32)
    answered = [q for q, _ in queries if not router.route(q)[2]]
    runs = []
    for i, q in enumerate(answered[:17]):
        a = srv.answer(q, 64)
        if i > 0:  # the first request warms up
            runs.append(a)
    # 32 requests at once: their prompts prefilled together (one pass over
    # all rows), then decoded in lockstep (the second batch is timed).
    for rep in range(2):
        batch = srv.answer_batch(answered[32 * rep:32 * rep + 32], 64, list(range(32)))
    ctx.close()
    router.close()
    t_end = max(a.t_last for a in batch)
    batched = {"requests": len(batch), "tokens_each": 64,
               "ttft_ms_p50": round(float(np.median([a.ttft_ms for a in batch])), 3),
               "ttft_ms_max": round(max(a.ttft_ms for a in batch), 3),
               "e2e_ms": round(t_end * 1e3, 3),
               "aggregate_tok_s": round(sum(len(a.tokens) for a in batch) / t_end, 1),
               "lockstep_decode_tok_s": round(sum(len(a.tokens) - 1 for a in batch) /
                                              (t_end - max(a.t_first for a in batch)), 1)}
    med = lambda f: round(float(np.median([f(a) for a in runs])), 3)
    serving = {"requests": len(runs), "tokens_each": 64,
               "prompt_tokens_p50": med(lambda a: a.prompt_tokens),
               "route_render_ms_p50": med(lambda a: a.t_render * 1e3),
               "ttft_ms_p50": med(lambda a: a.ttft_ms), "decode_tok_s_p50": med(lambda a: a.decode_tok_s),
               "e2e_ms_p50": med(lambda a: a.t_last * 1e3), "e2e_tok_s_p50": med(lambda a: a.e2e_tok_s)}
    return {"routing": routing, "serving": serving, "serving_32_at_once": batched}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-other-configs", action="store_true",
                    help="skip the 1024-token prompt, 8192-token cache and 32-stream workloads")
    ap.add_argument("--only", choices=["prompt1024", "cache8192", "streams32", "ctxsweep", "windows", "q4decode",
                                       "e2e"],
                    help="measure just this one of the other workloads (for a kernel trace of it); "
                         "prints its figures instead of the decode line")
    ap.add_argument("--cpu-decode-steps", type=int, default=256)
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="also run one plain 1 GiB device copy (reference for HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: the decoder runs on a single MI355X; "
              f"--gpus {args.gpus} is not supported", file=sys.stderr)
        sys.exit(2)

    import torch

    import synth
    from paper_2606_12154_amd import hh

    wl = synth.WORKLOADS["1b_decode"]
    shape, P, N = wl["shape"], wl["prompt"], wl["steps"]
    if args.only == "q4decode":
        print(json.dumps({"metric": METRIC, "workload": "q4decode", "data": "synthetic", "n_gpus": 1,
                          **measure_q4_decode(shape)}), flush=True)
        return
    if args.only == "e2e":
        print(json.dumps({"metric": METRIC, "workload": "e2e", "data": "synthetic", "n_gpus": 1,
                          **measure_e2e(shape)}), flush=True)
        return
    if args.only == "windows":
        rows = measure_windows(shape)
        print(json.dumps({"metric": METRIC, "workload": "windows", "data": "synthetic", "n_gpus": 1,
                          "decode_vs_allocated_window": rows}), flush=True)
        return
    if args.only == "ctxsweep":
        rows = measure_ctx_sweep(shape)
        print(json.dumps({"metric": METRIC, "workload": "ctxsweep", "data": "synthetic", "n_gpus": 1,
                          "decode_vs_cached_positions": rows}), flush=True)
        return
    prompt = synth.make_tokens(shape.vocab, P, wl["tseed"])
    tensors = synth.make_weights(shape, wl["wseed"])
    # One context serves every 1B workload: 32 streams, 8192 + 512 positions.
    ctx = hh.Context(hh.make_config(shape, 32, 8192 + 513, 8192))
    ctx.load_weights(tensors)
    del tensors
    st = ctx.stream

    if args.calibrate_copy:
        a = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
        b = torch.empty_like(a)
        b.copy_(a)
        torch.cuda.synchronize()
        del a, b

    def one_step():
        ctx.reset(0)
        t0 = time.perf_counter()
        nxt, _ = ctx.prefill(0, prompt)        # host ids in, host token out
        ttft = time.perf_counter() - t0
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(st)
        for _ in range(N):
            hh.hh_decode_step(ctx.ctx, 1, None, None, None, None)
        e1.record(st)
        e1.synchronize()
        return ttft, e0.elapsed_time(e1) / 1e3

    if args.only:
        other = measure_others(ctx, shape, st, [args.only])
        print(json.dumps({"metric": METRIC, "workload": args.only, "data": "synthetic", "n_gpus": 1,
                          **other[args.only]}), flush=True)
        ctx.close()
        return
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

    # Achievable read bandwidth on this device: a plain streaming read of
    # 4 GiB (the library's read probe), 10 timed passes after 2 warm ones.
    probe = torch.empty(4 << 30, dtype=torch.uint8, device="cuda")
    p0 = torch.cuda.Event(enable_timing=True)
    p1 = torch.cuda.Event(enable_timing=True)
    for _ in range(2):
        hh.hh_read_probe(probe.data_ptr(), probe.numel(), st.cuda_stream)
    p0.record(st)
    for _ in range(10):
        hh.hh_read_probe(probe.data_ptr(), probe.numel(), st.cuda_stream)
    p1.record(st)
    p1.synchronize()
    read_gbs = 10 * probe.numel() / (p0.elapsed_time(p1) / 1e3) / 1e9
    del probe

    dec_s = float(np.sum(decs))
    tok_s = args.steps * N / dec_s
    launch_s = dec_s / (args.steps * N)          # one persistent-kernel launch per token
    t_mean = P + (N - 1) / 2.0 + 1                # positions attended, averaged over the steps
    launch_bytes = decode_step_bytes(shape, t_mean)
    achieved = launch_bytes / launch_s / 1e9
    traffic = measured_traffic(launch_bytes)
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
        "config": {"workload": f"1B bf16 decoder (16 layers, d 2048, 32/8 heads, FFN 8192, vocab 128256), "
                               f"batch 1: prefill of a {P}-token uniform-random prompt, then {N} greedy "
                               f"decode steps fed back on the device",
                   "prompt": P, "decode_steps": N, "batch": 1, "kv_cache": "fp16, 16-token pages"},
        "ttft_ms": round(float(np.mean(ttfts)) * 1e3, 3),
        "ttft_ms_min": round(float(np.min(ttfts)) * 1e3, 3),
        "ttft_ms_max": round(float(np.max(ttfts)) * 1e3, 3),
        "decode_ms_per_token": round(launch_s * 1e3, 4),
        "decode_tok_s_min": round(N / max(decs), 2),
        "decode_tok_s_max": round(N / min(decs), 2),
        "e2e_tok_s": round(args.steps * (N + 1) / wall, 2),
        "roofline": {"bound": "hbm", "kernel": "k_decode_step (one launch per token)",
                     "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
                     "bytes_per_launch": int(launch_bytes), "launch_us": round(launch_s * 1e6, 2),
                     "measured_read_gbs": round(read_gbs, 1),
                     "frac_of_measured_read": round(achieved / read_gbs, 4)},
    }

    if not args.no_other_configs:
        # The other workloads on the same context, as keys of the same line.
        oth = measure_others(ctx, shape, st, ["prompt1024", "cache8192", "streams32"])
        a, b, c = oth["prompt1024"], oth["cache8192"], oth["streams32"]
        out.update({
            "ttft_ms_p1024": a["ttft_ms"], "ttft_ms_p1024_min": a["ttft_ms_min"],
            "prefill_p1024_device_ms": a["prefill_device_ms"], "prefill_p1024_tflops": a["prefill_tflops"],
            "prefill_mfma_frac": a["mfma_frac"], "decode_tok_s_p1024": a["decode_tok_s"],
            "cache8192_decode_tok_s": b["decode_tok_s"], "cache8192_ms_per_token": b["ms_per_token"],
            "cache8192_hbm_frac": b["hbm_frac"],
            "streams32_tok_s": c["aggregate_tok_s"], "streams32_step_ms": c["step_ms"],
            "streams32_hbm_frac": c["hbm_frac"],
        })

    ctx.close()
    del ctx
    torch.cuda.empty_cache()
    if not args.no_other_configs:
        # The same request on the 4-bit model (weights quantized at load).
        q4 = measure_q4_decode(shape)
        out.update({"q4_decode_tok_s": q4["decode_tok_s"], "q4_ms_per_token": q4["ms_per_token"],
                    "q4_hbm_frac": q4["hbm_frac"], "q4_ttft_ms": q4["ttft_ms"]})
        torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        res, cores = cpu_baseline(shape, wl["wseed"], prompt, args.cpu_decode_steps)
        (rate, pre_s), (rate32, pre32) = res["fp64"], res["fp32"]
        out["cpu_baseline"] = {"value": round(rate, 4), "unit": "tok/s", "cores": cores, "kind": "oracle",
                               "sample": f"the numpy oracle (fp64) on the same weights: prefill of the {P}-token "
                                         f"prompt ({pre_s:.1f} s, not in the rate), then {args.cpu_decode_steps} "
                                         f"cached decode steps (rate = steps / their wall time)",
                               "fp32": {"value": round(rate32, 4), "unit": "tok/s", "prefill_s": round(pre32, 2),
                                        "sample": "the same oracle and request in fp32 working precision"}}
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
