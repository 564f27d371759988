"""Pins of the synthetic decoder oracle (oracle/decoder_oracle.py) against
closed forms, invariants and special cases, independent of the GPU path."""
import numpy as np
import pytest

from oracle import decoder_oracle as D
import oracle as O


# ---------------------------------------------------------------- RMSNorm
def test_rms_norm_closed_forms():
    # [3, 4]: rms = sqrt((9 + 16) / 2) = 5 / sqrt(2)
    out = D.rms_norm(np.array([3.0, 4.0]), np.ones(2), 0.0)
    assert np.allclose(out, np.array([3.0, 4.0]) * np.sqrt(2) / 5, rtol=1e-15)
    # a constant row c: c / sqrt(c^2 + eps) times the gain
    c, eps = -0.75, 1e-5
    g = np.array([1.0, 2.0, -0.5, 3.0])
    assert np.allclose(D.rms_norm(np.full(4, c), g, eps), c / np.sqrt(c * c + eps) * g, rtol=1e-15)
    # the gain multiplies elementwise; a zero row stays zero
    assert np.all(D.rms_norm(np.zeros(8), np.ones(8), 1e-5) == 0)


def test_rms_norm_invariants():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((5, 64))
    g = rng.standard_normal(64)
    y = D.rms_norm(x, np.ones(64), 0.0)
    assert np.allclose(np.mean(y * y, axis=1), 1.0, rtol=1e-13)          # unit mean square
    assert np.allclose(D.rms_norm(3.7 * x, g, 0.0), D.rms_norm(x, g, 0.0), rtol=1e-13)  # scale-free
    assert np.allclose(D.rms_norm(-x, g, 0.0), -D.rms_norm(x, g, 0.0), rtol=1e-15)     # odd


# ---------------------------------------------------------------- rotary positions
def test_rope_two_dimensional_case_is_a_rotation_by_the_position():
    # head_dim 2: one pair, frequency base^0 = 1, so position p rotates by p radians
    x = np.zeros((3, 1, 2))
    x[:, 0, 0] = 1.0
    out = D.rope(x, [0, 1, 2], 10000.0)
    for p in range(3):
        assert np.allclose(out[p, 0], [np.cos(p), np.sin(p)], rtol=1e-15, atol=1e-15)


def test_rope_invariants():
    rng = np.random.default_rng(1)
    q = rng.standard_normal((1, 3, 16))
    k = rng.standard_normal((1, 3, 16))
    assert np.allclose(D.rope(q, [0], 10000.0), q, rtol=0, atol=0)       # position 0 = identity
    r = D.rope(q, [37], 10000.0)
    half = 8
    assert np.allclose(r[..., :half] ** 2 + r[..., half:] ** 2,
                       q[..., :half] ** 2 + q[..., half:] ** 2, rtol=1e-13)  # pairs keep their norm
    # scores depend only on the position difference
    def score(pq, pk):
        return np.sum(D.rope(q, [pq], 10000.0) * D.rope(k, [pk], 10000.0), axis=-1)
    assert np.allclose(score(5, 2), score(105, 102), rtol=1e-10)
    assert not np.allclose(score(5, 2), score(5, 3), rtol=1e-6)
    # the pairing is (i, i + Dh/2): element 1 of a position-1 rotation of e_1 moves into i + Dh/2
    e = np.zeros((1, 1, 16))
    e[0, 0, 1] = 1.0
    out = D.rope(e, [1], 10000.0)
    theta = 10000.0 ** (-2.0 / 16)
    assert np.isclose(out[0, 0, 1], np.cos(theta)) and np.isclose(out[0, 0, 9], np.sin(theta))


# ---------------------------------------------------------------- attention
def test_attention_special_cases():
    rng = np.random.default_rng(2)
    v = rng.standard_normal((6, 2, 8))
    k = rng.standard_normal((6, 2, 8))
    q = rng.standard_normal((6, 2, 8))
    out = D.causal_attention(q, k, v, range(6))
    assert np.allclose(out[0], v[0], rtol=1e-15)                          # one visible key
    zero_q = np.zeros_like(q)
    mean = D.causal_attention(zero_q, k, v, range(6))                      # equal scores
    for t in range(6):
        assert np.allclose(mean[t], v[:t + 1].mean(axis=0), rtol=1e-13)
    # a dominant key takes (almost) all the weight
    k2 = k.copy()
    k2[3] = 400.0 * q[5]
    out2 = D.causal_attention(q, k2, v, [5])
    assert np.allclose(out2[0], v[3], atol=1e-8)


def test_attention_is_causal():
    rng = np.random.default_rng(3)
    q, k, v = (rng.standard_normal((7, 2, 8)) for _ in range(3))
    base = D.causal_attention(q, k, v, range(7))
    k2, v2 = k.copy(), v.copy()
    k2[5:] += 3.0
    v2[5:] -= 2.0
    out = D.causal_attention(q, k2, v2, range(7))
    assert np.array_equal(out[:5], base[:5]) and not np.allclose(out[5:], base[5:])


# ---------------------------------------------------------------- decoder
def _tiny(seed=4, layers=2):
    shape = D.DecoderShape(n_layers=layers, d_model=256, n_heads=2, head_dim=128, vocab=97,
                           d_ff=128, n_experts=4, top_k=2)
    rng = np.random.default_rng(seed)
    f32 = lambda *s, scale=0.02: (rng.standard_normal(s) * scale).astype(np.float32)
    d, e, f, v = shape.d_model, shape.n_experts, shape.d_ff, shape.vocab
    experts = []
    for _ in range(layers):
        experts.append({x: O.quantize_expert(f32(f, d), f32(f, d), f32(d, f)) for x in range(e)})
    w = D.DecoderWeights(embed=f32(v, d, scale=1.0), lm_head=f32(v, d), final_norm=1 + f32(d, scale=0.1),
                         attn_norm=[1 + f32(d, scale=0.1) for _ in range(layers)],
                         wq=[f32(d, d) for _ in range(layers)], wk=[f32(d, d) for _ in range(layers)],
                         wv=[f32(d, d) for _ in range(layers)], wo=[f32(d, d) for _ in range(layers)],
                         moe_norm=[1 + f32(d, scale=0.1) for _ in range(layers)],
                         w_router=[f32(e, d) for _ in range(layers)], experts=experts)
    return shape, w


def test_decoder_with_silent_blocks_is_embedding_then_head():
    """Zero attention output and zero experts: the residual stream is the
    embedding, so the logits are W_lm RMSNorm(embed[token])."""
    shape, w = _tiny()
    z = np.zeros_like(w.wo[0])
    w.wo = [z for _ in w.wo]
    zq = O.quantize_expert(np.zeros((128, 256), np.float32), np.zeros((128, 256), np.float32),
                           np.zeros((256, 128), np.float32))
    w.experts = [{x: zq for x in range(4)} for _ in range(shape.n_layers)]
    toks = [3, 50, 7]
    x, logits, nxt = D.decoder_forward(shape, w, toks, D.KVState())
    assert np.array_equal(x, w.embed[toks].astype(np.float64))
    ref = w.lm_head.astype(np.float64) @ D.rms_norm(w.embed[7], w.final_norm, shape.rms_eps)
    assert np.allclose(logits, ref, rtol=1e-13) and nxt == int(np.argmax(ref))


def test_decoder_incremental_cache_equals_full_prefill():
    """Prefill of the prompt, then one token at a time through the cache,
    equals one prefill of the whole sequence (causality + the cache)."""
    shape, w = _tiny(seed=5)
    seq = [11, 2, 60, 33, 8]
    x_full, logits_full, _ = D.decoder_forward(shape, w, seq, D.KVState())
    kv = D.KVState()
    D.decoder_forward(shape, w, seq[:3], kv)
    D.decoder_forward(shape, w, seq[3:4], kv)
    x_last, logits_last, _ = D.decoder_forward(shape, w, seq[4:], kv)
    assert kv.k[0].shape[0] == 5
    assert np.allclose(x_last[-1], x_full[-1], rtol=1e-10, atol=1e-12)
    assert np.allclose(logits_last, logits_full, rtol=1e-10, atol=1e-12)


def test_decoder_first_position_attention_is_the_value():
    """At position 0 the only visible key is its own, so the attention output
    is Wo (Wv n) exactly: check one layer with silent experts by hand."""
    shape, w = _tiny(seed=6, layers=1)
    zq = O.quantize_expert(np.zeros((128, 256), np.float32), np.zeros((128, 256), np.float32),
                           np.zeros((256, 128), np.float32))
    w.experts = [{x: zq for x in range(4)}]
    x, _, _ = D.decoder_forward(shape, w, [9], D.KVState())
    e = w.embed[9].astype(np.float64)
    n = D.rms_norm(e, w.attn_norm[0], shape.rms_eps)
    ref = e + w.wo[0].astype(np.float64) @ (w.wv[0].astype(np.float64) @ n)
    assert np.allclose(x[0], ref, rtol=1e-12, atol=1e-14)
