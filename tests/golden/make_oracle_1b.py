"""Write the stored oracle values of the 1B parity tests whose prompts the fp64
oracle cannot evaluate within a test's time (tests/golden/oracle_1b.npz).

Calls only the oracle and the seeded input generators.  For each case it
stores the teacher-forced token sequence and the oracle's residual stream
after the last block (the rows the LM head maps to logits) in fp64; the tests
rebuild the logits from these rows with the oracle's own head
(``Decoder.logits``), so the file stays small (16 KiB per row).

Cases (1B bf16 model, weight seed 1):
* ``long``: the long-context workload, an 8192-token prompt (seed 4); the
  prompt's last row, then 4 greedy decode steps (attended lengths
  8193..8196), each fed the oracle's argmax of the row before.
* ``mid``: an 1100-token prompt (seed 5, lengths 1101..1106 attended by the 6
  decode steps): a context split into more than two attention items.
* ``multi``: the multi-stream workload, 32 streams with 256-token prompts
  (seeds 100 + s); each stream's last prompt row, then 2 lockstep decode
  steps, each fed the oracle's argmax of the stream's row before.

Run: python tests/golden/make_oracle_1b.py  (about 15 minutes on 8 cores,
12 GB of memory).
"""
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
import synth  # noqa: E402

OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "oracle_1b.npz")


def greedy_rows(model, prompt, steps):
    """Prompt's last hidden row, then `steps` teacher-forced decode rows."""
    cache = model.new_cache()
    rows = [model.forward_hidden(prompt, cache, rows="last")[0]]
    fed = []
    for _ in range(steps):
        tok = int(oracle.greedy(model.logits(rows[-1])))
        fed.append(tok)
        rows.append(model.forward_hidden(np.array([tok]), cache, rows="all")[0])
    return np.array(fed, dtype=np.int32), np.stack(rows)


def main():
    shape = synth.ONE_B
    t0 = time.time()
    model = oracle.Decoder(shape, synth.weights_as_f64(shape, synth.make_weights(shape, 1)))
    print(f"weights {time.time() - t0:.0f} s", flush=True)
    out = {}

    t0 = time.time()
    fed, rows = greedy_rows(model, synth.make_tokens(shape.vocab, 8192, 4), 4)
    out.update(long_seed=np.int32(4), long_prompt=np.int32(8192), long_fed=fed, long_hidden=rows)
    print(f"long: {time.time() - t0:.0f} s", flush=True)

    t0 = time.time()
    fed, rows = greedy_rows(model, synth.make_tokens(shape.vocab, 1100, 5), 6)
    out.update(mid_seed=np.int32(5), mid_prompt=np.int32(1100), mid_fed=fed, mid_hidden=rows)
    print(f"mid: {time.time() - t0:.0f} s", flush=True)

    t0 = time.time()
    n, P = 32, 256
    caches, h0 = [], []
    for s in range(n):
        c = model.new_cache()
        h0.append(model.forward_hidden(synth.make_tokens(shape.vocab, P, 100 + s), c, rows="last")[0])
        caches.append(c)
    h0 = np.stack(h0)
    fed1 = oracle.greedy(model.logits(h0)).astype(np.int32)
    h1 = model.decode_batch_hidden(caches, fed1)
    fed2 = oracle.greedy(model.logits(h1)).astype(np.int32)
    h2 = model.decode_batch_hidden(caches, fed2)
    out.update(multi_seed0=np.int32(100), multi_prompt=np.int32(P), multi_hidden0=h0, multi_fed1=fed1,
               multi_hidden1=h1, multi_fed2=fed2, multi_hidden2=h2)
    print(f"multi: {time.time() - t0:.0f} s", flush=True)

    np.savez_compressed(OUT, **out)
    print(f"wrote {OUT}", flush=True)


if __name__ == "__main__":
    main()
