"""Plain CPU oracle of a synthetic OLMoE-shaped decoder around the MoE layer.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this module; only the test-suite and the benchmark's CPU-baseline leg
use it.  It shares no code with the HIP library.

The paper evaluates an OLMoE decoder whose router, attention, embeddings,
normalization layers and language-model head stay in BF16 while the routed
experts use the W4A16 layer (abstract; Sec. 4.1: 16 sparse layers, 64
experts, top-8, hidden size 2048, expert size 1024, SDPA attention, greedy
decoding).  The paper gives no further architecture, so this decoder is the
textbook pre-norm transformer with those sizes (readings, each stated where
it is used):

    x_0 = Embed[token]
    per layer:  x += Wo Attn(RoPE(Wq n), RoPE(Wk n), Wv n),  n = RMSNorm(x; g_attn)
                x += MoE(RMSNorm(x; g_moe))          (the W4A16 layer, Eq. 1-2)
    logits = W_lm RMSNorm(x; g_final);  next token = argmax (greedy)

Everything is fp64 on the dequantized expert weights (Eq. 3); bf16 tensors
are passed as float32 arrays holding the bf16 values exactly.  Every function
is pinned by tests/test_decoder_oracle_pins.py; none is "parity unpinned".
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from . import exactmoe_oracle as O


def rms_norm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """RMSNorm over the last axis: x / sqrt(mean(x^2) + eps) * g (textbook definition)."""
    x = np.asarray(x, np.float64)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * np.asarray(g, np.float64)


def rope(x: np.ndarray, positions, base: float) -> np.ndarray:
    """Rotary position embedding of x [T][H][Dh] at the given token positions.

    Reading (the paper names no position encoding): the rotate-half form, in
    which element i < Dh/2 of a head is paired with element i + Dh/2 and the
    pair is rotated by the angle p * base^(-2i/Dh) for position p.
    """
    x = np.asarray(x, np.float64)
    dh = x.shape[-1]
    half = dh // 2
    inv = base ** (-2.0 * np.arange(half) / dh)                  # [half]
    ang = np.asarray(positions, np.float64)[:, None] * inv[None]  # [T][half]
    c, s = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
    a, b = x[..., :half], x[..., half:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def causal_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, q_positions) -> np.ndarray:
    """Scaled dot-product attention of queries q [T][H][Dh] (at absolute
    positions q_positions) over keys/values k, v [L][H][Dh] at positions
    0 .. L-1: query at position p sees keys 0 .. p, softmax(q.k / sqrt(Dh))."""
    q, k, v = (np.asarray(a, np.float64) for a in (q, k, v))
    t, h, dh = q.shape
    out = np.zeros((t, h, dh))
    for i, p in enumerate(q_positions):
        n = int(p) + 1
        s = np.einsum("hd,lhd->hl", q[i], k[:n]) / np.sqrt(dh)   # [H][n]
        s -= s.max(axis=1, keepdims=True)
        w = np.exp(s)
        w /= w.sum(axis=1, keepdims=True)
        out[i] = np.einsum("hl,lhd->hd", w, v[:n])
    return out


@dataclass
class DecoderShape:
    n_layers: int
    d_model: int
    n_heads: int
    head_dim: int
    vocab: int
    d_ff: int
    n_experts: int
    top_k: int
    rope_base: float = 10000.0
    rms_eps: float = 1e-5


@dataclass
class DecoderWeights:
    """All as float32 arrays holding bf16 values; expert weights quantized lazily."""
    embed: np.ndarray        # [V][d]
    lm_head: np.ndarray      # [V][d]
    final_norm: np.ndarray   # [d]
    attn_norm: list          # [L] of [d]
    wq: list                 # [L] of [d][d]  (nn.Linear order: [out][in])
    wk: list
    wv: list
    wo: list
    moe_norm: list           # [L] of [d]
    w_router: list           # [L] of [E][d]
    experts: list            # [L] of {e: QuantizedExpert} (or a mapping-like object)


@dataclass
class KVState:
    """Keys (after RoPE) and values of every layer for positions 0 .. len-1."""
    k: list = field(default_factory=list)   # [L] of [len][H][Dh]
    v: list = field(default_factory=list)


def decoder_forward(shape: DecoderShape, w: DecoderWeights, tokens, kv: KVState,
                    renormalize: bool = True):
    """Run tokens (positions len(kv) .. len(kv)+T-1) through the decoder,
    appending their keys/values to kv.  Returns (hidden states x [T][d] after
    the last layer, logits [V] of the last token, greedy next token)."""
    d, hn, dh = shape.d_model, shape.n_heads, shape.head_dim
    tokens = [int(t) for t in tokens]
    pos0 = 0 if not kv.k else kv.k[0].shape[0]
    positions = np.arange(pos0, pos0 + len(tokens))
    x = np.asarray(w.embed, np.float64)[tokens]                  # [T][d]
    for layer in range(shape.n_layers):
        n = rms_norm(x, w.attn_norm[layer], shape.rms_eps)
        q = (n @ np.asarray(w.wq[layer], np.float64).T).reshape(-1, hn, dh)
        k = (n @ np.asarray(w.wk[layer], np.float64).T).reshape(-1, hn, dh)
        v = (n @ np.asarray(w.wv[layer], np.float64).T).reshape(-1, hn, dh)
        q, k = rope(q, positions, shape.rope_base), rope(k, positions, shape.rope_base)
        if len(kv.k) <= layer:
            kv.k.append(np.zeros((0, hn, dh)))
            kv.v.append(np.zeros((0, hn, dh)))
        kv.k[layer] = np.concatenate([kv.k[layer], k])
        kv.v[layer] = np.concatenate([kv.v[layer], v])
        a = causal_attention(q, kv.k[layer], kv.v[layer], positions).reshape(-1, d)
        x = x + a @ np.asarray(w.wo[layer], np.float64).T
        m = rms_norm(x, w.moe_norm[layer], shape.rms_eps)
        r = O.route(m, np.asarray(w.w_router[layer], np.float64), shape.top_k, renormalize)
        x = x + O.moe_forward(m, w.experts[layer], r)
    last = rms_norm(x[-1], w.final_norm, shape.rms_eps)
    logits = np.asarray(w.lm_head, np.float64) @ last
    return x, logits, int(np.argmax(logits))
