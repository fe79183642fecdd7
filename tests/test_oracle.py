"""Pins of the fp64 oracle against things other than itself (CPU only).

Each test is chosen so that a plausible mistake in the oracle -- a dropped
gain, interleaved instead of rotate-half RoPE pairing, a wrong frequency
exponent, a wrong GQA head map, a missing 1/sqrt(hd), an off-by-one causal
mask, a cache that forgets positions, an untied head read from the embedding
-- fails at least one of them.
"""
import dataclasses
import math

import numpy as np
import pytest

import oracle
import synth


def small_shape(**kw):
    base = dict(n_layers=2, d_model=64, n_heads=4, n_kv_heads=2, head_dim=16,
                ffn_dim=88, vocab=97, rms_eps=1e-5, rope_theta=1e4, tied=True,
                dtype=synth.F32)
    base.update(kw)
    return synth.ModelShape(**base)


def model_for(shape, seed=5, gain_std=0.1):
    t = synth.make_weights(shape, seed, gain_std=gain_std)
    return oracle.Decoder(shape, synth.weights_as_f64(shape, t))


# ---------------------------------------------------------------- closed forms

def test_rmsnorm_worked_values():
    # (3, 4): mean square 12.5 -> 3/sqrt(12.50001), 4/sqrt(12.50001)
    y = oracle.rms_norm(np.array([3.0, 4.0]), np.ones(2), 1e-5)
    np.testing.assert_allclose(y, [0.8485278, 1.1313704], atol=1e-6)
    y = oracle.rms_norm(np.array([3.0, 4.0]), np.array([2.0, 0.5]), 1e-5)
    np.testing.assert_allclose(y, [1.6970556, 0.5656852], atol=1e-6)


def test_rmsnorm_invariants():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((5, 32)) * 3.0
    y = oracle.rms_norm(x, np.ones(32), 0.0)
    np.testing.assert_allclose(np.sqrt(np.mean(y * y, axis=-1)), 1.0, rtol=1e-12)
    np.testing.assert_allclose(oracle.rms_norm(7.5 * x, np.ones(32), 0.0), y, rtol=1e-12)


def test_rope_worked_values_pin_pairing_and_frequency():
    # hd = 4, theta = 1e4: omega_0 = 1, omega_1 = 1e4^(-1/2) = 0.01.
    q = np.array([[[1.0, 0.0, 0.0, 0.0]]])
    y = oracle.apply_rope(q, np.array([1]), 1e4)[0, 0]
    # rotate-half pairs (0, 2): interleaved pairing would give (c, s, 0, 0)
    np.testing.assert_allclose(y, [0.5403023, 0.0, 0.8414710, 0.0], atol=1e-7)
    q = np.array([[[0.0, 1.0, 0.0, 0.0]]])
    y = oracle.apply_rope(q, np.array([1]), 1e4)[0, 0]
    np.testing.assert_allclose(y, [0.0, 0.9999500, 0.0, 0.0099998], atol=1e-7)


def test_rope_invariants():
    rng = np.random.default_rng(1)
    u = rng.standard_normal((3, 2, 64))
    np.testing.assert_allclose(oracle.apply_rope(u, np.zeros(3), 5e5), u, atol=0)
    y = oracle.apply_rope(u, np.array([3, 100, 8191]), 5e5)
    half = 32
    np.testing.assert_allclose(u[..., :half] ** 2 + u[..., half:] ** 2,
                               y[..., :half] ** 2 + y[..., half:] ** 2, rtol=1e-12)
    # relative-position property: <R_{p+D} q, R_{s+D} k> = <R_p q, R_s k>
    q, k = rng.standard_normal((1, 1, 64)), rng.standard_normal((1, 1, 64))
    a = np.sum(oracle.apply_rope(q, [7], 1e4) * oracle.apply_rope(k, [3], 1e4))
    b = np.sum(oracle.apply_rope(q, [7 + 500], 1e4) * oracle.apply_rope(k, [3 + 500], 1e4))
    assert abs(a - b) < 1e-10


def test_silu_values():
    np.testing.assert_allclose(oracle.silu(np.array([1.0, -1.0, 0.0])),
                               [0.7310586, -0.2689414, 0.0], atol=1e-7)


# ---------------------------------------------------------------- attention

def brute_attention(q, k, v, q_pos):
    """Scalar-loop causal GQA attention in fp64 (independent restatement)."""
    Tq, Hq, hd = q.shape
    Hkv = k.shape[1]
    out = np.zeros_like(q)
    for i in range(Tq):
        for j in range(Hq):
            g = j * Hkv // Hq
            scores = []
            for t in range(int(q_pos[i]) + 1):
                scores.append(sum(q[i, j, e] * k[t, g, e] for e in range(hd)) / math.sqrt(hd))
            mx = max(scores)
            ws = [math.exp(s - mx) for s in scores]
            z = sum(ws)
            for e in range(hd):
                out[i, j, e] = sum(ws[t] * v[t, g, e] for t in range(len(ws))) / z
    return out


def test_attention_brute_force():
    rng = np.random.default_rng(2)
    q = rng.standard_normal((5, 4, 8))
    k = rng.standard_normal((7, 2, 8))
    v = rng.standard_normal((7, 2, 8))
    q_pos = np.array([2, 3, 4, 5, 6])
    np.testing.assert_allclose(oracle.attention(q, k, v, q_pos),
                               brute_attention(q, k, v, q_pos), rtol=1e-12, atol=1e-12)


def test_attention_special_cases():
    rng = np.random.default_rng(3)
    q = rng.standard_normal((1, 4, 8))
    k = rng.standard_normal((6, 2, 8))
    v = rng.standard_normal((6, 2, 8))
    o = oracle.attention(q, k, v, np.array([0]))       # one visible key -> its value
    np.testing.assert_allclose(o[0, :2], v[[0, 0], [0, 0]], atol=1e-15)
    np.testing.assert_allclose(o[0, 2:], v[[0, 0], [1, 1]], atol=1e-15)
    o = oracle.attention(np.zeros_like(q), k, v, np.array([3]))  # uniform weights -> mean
    np.testing.assert_allclose(o[0, 0], v[:4, 0].mean(0), atol=1e-14)
    np.testing.assert_allclose(o[0, 3], v[:4, 1].mean(0), atol=1e-14)


def test_gqa_equals_mha_with_repeated_heads():
    rng = np.random.default_rng(4)
    q = rng.standard_normal((6, 8, 16))
    k = rng.standard_normal((6, 2, 16))
    v = rng.standard_normal((6, 2, 16))
    pos = np.arange(6)
    a = oracle.attention(q, k, v, pos)
    b = oracle.attention(q, np.repeat(k, 4, axis=1), np.repeat(v, 4, axis=1), pos)
    np.testing.assert_allclose(a, b, rtol=1e-13, atol=1e-13)


def test_attention_matches_torch_sdpa():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(5)
    T = 19
    q = rng.standard_normal((T, 8, 64))
    k = rng.standard_normal((T, 2, 64))
    v = rng.standard_normal((T, 2, 64))
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.tensor(q).transpose(0, 1), torch.tensor(np.repeat(k, 4, 1)).transpose(0, 1),
        torch.tensor(np.repeat(v, 4, 1)).transpose(0, 1), is_causal=True)
    np.testing.assert_allclose(oracle.attention(q, k, v, np.arange(T)),
                               ref.transpose(0, 1).numpy(), rtol=1e-10, atol=1e-10)


# ---------------------------------------------------------------- whole model

def hf_logits(shape, tensors, tokens):
    torch = pytest.importorskip("torch")
    tf = pytest.importorskip("transformers")
    cfg = tf.LlamaConfig(
        vocab_size=shape.vocab, hidden_size=shape.d_model, intermediate_size=shape.ffn_dim,
        num_hidden_layers=shape.n_layers, num_attention_heads=shape.n_heads,
        num_key_value_heads=shape.n_kv_heads, head_dim=shape.head_dim,
        rms_norm_eps=shape.rms_eps, rope_theta=shape.rope_theta,
        tie_word_embeddings=shape.tied, max_position_embeddings=4096,
        attention_bias=False, mlp_bias=False)
    model = tf.LlamaForCausalLM(cfg).double().eval()
    w = synth.weights_as_f64(shape, tensors)
    sd = {"model.embed_tokens.weight": w["embed"], "model.norm.weight": w["final_norm"]}
    for l in range(shape.n_layers):
        p = f"model.layers.{l}."
        sd[p + "input_layernorm.weight"] = w[f"l{l}.attn_norm"]
        sd[p + "post_attention_layernorm.weight"] = w[f"l{l}.mlp_norm"]
        for a, b in (("q_proj", "wq"), ("k_proj", "wk"), ("v_proj", "wv"), ("o_proj", "wo")):
            sd[p + f"self_attn.{a}.weight"] = w[f"l{l}.{b}"]
        for a, b in (("gate_proj", "w_gate"), ("up_proj", "w_up"), ("down_proj", "w_down")):
            sd[p + f"mlp.{a}.weight"] = w[f"l{l}.{b}"]
    sd["lm_head.weight"] = w.get("lm_head", w["embed"])
    model.load_state_dict({k_: torch.tensor(v_) for k_, v_ in sd.items()}, strict=False)
    with torch.no_grad():
        return model(torch.tensor(tokens[None].astype(np.int64))).logits[0].numpy()


@pytest.mark.parametrize("tied", [True, False])
def test_model_matches_transformers_llama(tied):
    shape = dataclasses.replace(synth.TINY, tied=tied)
    tensors = synth.make_weights(shape, 11, gain_std=0.1)
    tokens = synth.make_tokens(shape.vocab, 24, 12)
    ours, _ = oracle.Decoder(shape, synth.weights_as_f64(shape, tensors)).prefill(tokens)
    ref = hf_logits(shape, tensors, tokens)
    # transformers computes RMSNorm and RoPE tables in fp32: ~1e-7 relative.
    np.testing.assert_allclose(ours, ref, atol=2e-5, rtol=0)
    assert np.array_equal(oracle.greedy(ours), oracle.greedy(ref))


def test_causality_future_tokens_do_not_matter():
    shape = small_shape()
    m = model_for(shape)
    a = synth.make_tokens(shape.vocab, 20, 1)
    b = a.copy()
    b[12:] = synth.make_tokens(shape.vocab, 8, 2)
    la, _ = m.prefill(a)
    lb, _ = m.prefill(b)
    np.testing.assert_allclose(la[:12], lb[:12], atol=1e-12, rtol=0)
    assert np.abs(la[12:] - lb[12:]).max() > 1e-3


def test_kv_cached_decode_equals_recompute():
    shape = small_shape()
    m = model_for(shape)
    toks = synth.make_tokens(shape.vocab, 30, 3)
    full, _ = m.prefill(toks)
    _, cache = m.prefill(toks[:17])
    rows = [m.decode(cache, int(t)) for t in toks[17:]]
    np.testing.assert_allclose(np.array(rows), full[17:], atol=1e-12, rtol=0)
    assert cache.length == 30


def test_chunked_prefill_equals_one_shot():
    shape = small_shape()
    m = model_for(shape)
    toks = synth.make_tokens(shape.vocab, 40, 4)
    full, _ = m.prefill(toks)
    cache = m.new_cache()
    parts = [m.forward(toks[a:b], cache) for a, b in ((0, 9), (9, 25), (25, 40))]
    np.testing.assert_allclose(np.concatenate(parts), full, atol=1e-12, rtol=0)
    last = m.forward(toks, None, rows="last")
    np.testing.assert_allclose(last[0], full[-1], atol=1e-12, rtol=0)


def test_batched_decode_equals_single_streams():
    shape = small_shape()
    m = model_for(shape)
    prompts = [synth.make_tokens(shape.vocab, n, 10 + n) for n in (5, 9, 13)]
    caches = [m.prefill(p)[1] for p in prompts]
    nxt = np.array([3, 50, 96])
    got = m.decode_batch(caches, nxt)
    for i, p in enumerate(prompts):
        ref, _ = m.prefill(np.concatenate([p, nxt[i:i + 1]]))
        np.testing.assert_allclose(got[i], ref[-1], atol=1e-12, rtol=0)


def test_zero_layer_model_echoes_its_input():
    shape = dataclasses.replace(synth.TINY, n_layers=0)
    tensors = synth.make_weights(shape, 0)
    m = oracle.Decoder(shape, synth.weights_as_f64(shape, tensors))
    toks = synth.make_tokens(shape.vocab, 50, 9)
    logits, _ = m.prefill(toks)
    assert np.array_equal(oracle.greedy(logits), toks)
    # logit of the input token = |E_t|^2 / rms(E_t) ~= d * 0.02 = 5.12
    own = logits[np.arange(50), toks]
    np.testing.assert_allclose(own.mean(), 5.12, rtol=0.05)
    others = np.delete(logits[0], toks[0])
    assert abs(others.std() - 0.32) < 0.03


def test_greedy_ties_take_lowest_index():
    assert oracle.greedy(np.array([1.0, 3.0, 2.0, 3.0])) == 1


# ---------------------------------------------------------------- 4-bit group format (oracle/quant.py)

def test_q4_worked_example():
    """Hand-computed: a = 0.7, a / 7 = 0.1 in fp32 (0x3DCCCCCD) rounds up to the
    bf16 0x3DCD = 0.10009765625; 0.7 / s = 6.993 -> 7, -0.35 / s = -3.497 -> -3,
    0.1 / s = 0.999 -> 1."""
    w = np.zeros((1, 32), np.float32)
    w[0, :3] = [0.7, -0.35, 0.1]
    q, s = oracle.q4_quantize_rows(w)
    assert s.shape == (1, 1) and s[0, 0] == np.float32(0.10009765625)
    assert q[0, :4].tolist() == [7, -3, 1, 0] and not q[0, 4:].any()
    d = oracle.q4_dequantize(q, s)
    assert d[0, :3].tolist() == [0.70068359375, -0.30029296875, 0.10009765625]


def test_q4_representable_groups_round_trip():
    rng = np.random.default_rng(3)
    k = rng.integers(-7, 8, size=(5, 64))
    k[:, 0] = 7          # every group reaches |k| = 7 ...
    k[:, 32] = -7        # ... so its scale is exactly s
    s = np.float32(2.0 ** -6)
    w = (k * s).astype(np.float32)
    q, sc = oracle.q4_quantize_rows(w)
    assert np.all(sc == s)
    assert np.array_equal(q, k)
    assert np.array_equal(oracle.q4_dequantize(q, sc), w.astype(np.float64))


def test_q4_error_bound_and_range():
    rng = np.random.default_rng(4)
    w = (0.02 * rng.standard_normal((64, 256))).astype(np.float32)
    w[3, 32:64] *= 1e-6     # a group of tiny values
    q, s = oracle.q4_quantize_rows(w)
    assert q.min() >= -7 and q.max() <= 7     # the scale never lets a value reach -8
    err = np.abs(oracle.q4_dequantize(q, s) - w.astype(np.float64))
    bound = np.repeat(s.astype(np.float64), 32, axis=1) / 2 * (1 + 1e-6)
    assert np.all(err <= bound)
    # Each group's largest magnitude maps to +-7 (to +-6 only if the bf16
    # scale rounded up past a / 6.5, which cannot happen: a / 7 < a / 6.5).
    g = np.abs(q.reshape(64, -1, 32)).max(axis=-1)
    assert np.all(g == 7)


def test_q4_ties_to_even_and_zero_group():
    w = np.zeros((2, 32), np.float32)
    w[0, :5] = [2.5, 3.5, -2.5, -0.5, 7.0]     # a = 7 -> s = 1 exactly
    q, s = oracle.q4_quantize_rows(w)
    assert s[0, 0] == 1.0 and q[0, :5].tolist() == [2, 4, -2, 0, 7]
    assert s[1, 0] == 0.0 and not q[1].any()
    assert not oracle.q4_dequantize(q, s)[1].any()


def test_q4_pack_layout():
    q = np.zeros((1, 64), np.int8)
    q[0, :4] = [-8, 7, 0, 1]
    s = np.array([[1.0, 0.10009765625]], np.float32)
    b = oracle.q4_pack_rows(q, s)
    assert b.shape == (1, 32 + 4)
    assert b[0, :2].tolist() == [0xF0, 0x98]             # (0 | 15 << 4), (8 | 9 << 4)
    assert np.all(b[0, 2:32] == 0x88)                    # zeros are nibble 8
    assert b[0, 32:].tolist() == [0x80, 0x3F, 0xCD, 0x3D]  # bf16 1.0 = 0x3F80, 0.1000977 = 0x3DCD


def test_q4_model_weights_groups():
    """W_down is grouped along its output rows (the rows of W_down^T), the other
    matrices along their input columns; the head is Q4(embed), the embedding
    table and gains untouched."""
    shape = synth.TINY
    w = synth.weights_as_f64(shape, synth.make_weights(shape, 0, gain_std=0.1))
    qw = oracle.q4_model_weights(shape, w)
    assert np.array_equal(qw["embed"], w["embed"]) and np.array_equal(qw["l0.attn_norm"], w["l0.attn_norm"])
    q, s = oracle.q4_quantize_rows(w["embed"].astype(np.float32))
    assert np.array_equal(qw["lm_head"], oracle.q4_dequantize(q, s))
    q, s = oracle.q4_quantize_rows(w["l1.w_down"].T.astype(np.float32))
    assert np.array_equal(qw["l1.w_down"], oracle.q4_dequantize(q, s).T)
    q, s = oracle.q4_quantize_rows(w["l1.wo"].astype(np.float32))
    assert np.array_equal(qw["l1.wo"], oracle.q4_dequantize(q, s))
    # A W_down whose columns are representable per 32 output rows is kept
    # exactly; the same matrix grouped along its rows would not be.
    k = np.random.default_rng(5).integers(-7, 8, size=(256, 688))
    k[::32, :] = 7
    wd = k * 2.0 ** -7
    w2 = dict(w)
    w2["l0.w_down"] = wd
    assert np.array_equal(oracle.q4_model_weights(shape, w2)["l0.w_down"], wd)
    qr, sr = oracle.q4_quantize_rows(wd[:, :672].astype(np.float32))
    assert not np.array_equal(oracle.q4_dequantize(qr, sr), wd[:, :672])
