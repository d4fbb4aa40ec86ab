"""The masked diffusion LM forward pass in fp64 (Definition 3 of the paper).

Given a partially observed sequence S~ over Sigma + {[MASK]}, one forward pass
gives a distribution over Sigma at every masked position.  Predictions are
not prefix conditioned: every position attends to every position (the
bidirectional-conditioning remark that follows Definition 3), so attention
here has no causal mask and [MASK] positions are keys like any other.

Architecture readings (the paper uses LLaDA-8B through Hugging Face and
describes no layer; the shapes come from the workload description):
pre-norm blocks ``x += Attn(Norm(x)); x += FFN(Norm(x))``, a final norm,
an untied head; no biases; norm gains are 1; multi-head attention with scale
1/sqrt(d_head); rotary position embedding (rotate-half pairing of dims i and
i + d_head/2, base theta) on queries and keys; FFN either exact-erf GELU or
SwiGLU ``(silu(x Wg^T) * x Wu^T) Wd^T``.
"""
from __future__ import annotations

import math

import numpy as np
from scipy.special import erf


def layer_norm(x: np.ndarray, eps: float) -> np.ndarray:
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps)


def rms_norm(x: np.ndarray, eps: float) -> np.ndarray:
    return x / np.sqrt((x * x).mean(axis=-1, keepdims=True) + eps)


def norm(shape, x: np.ndarray) -> np.ndarray:
    if shape.norm == "layernorm":
        return layer_norm(x, shape.norm_eps)
    return rms_norm(x, shape.norm_eps)


def rope_cos_sin(T: int, d_head: int, theta: float):
    """Angles pos * theta**(-2i/d_head) for pair index i in [0, d_head/2)."""
    half = d_head // 2
    inv = theta ** (-2.0 * np.arange(half, dtype=np.float64) / d_head)
    ang = np.arange(T, dtype=np.float64)[:, None] * inv[None, :]
    return np.cos(ang), np.sin(ang)


def apply_rope(x: np.ndarray, cos: np.ndarray, sin: np.ndarray) -> np.ndarray:
    """Rotate each (i, i + d_head/2) pair of x [T, H, d_head] by its angle."""
    half = x.shape[-1] // 2
    x1, x2 = x[..., :half], x[..., half:]
    c, s = cos[:, None, :], sin[:, None, :]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def softmax(s: np.ndarray, axis: int = -1) -> np.ndarray:
    m = s.max(axis=axis, keepdims=True)
    e = np.exp(s - m)
    return e / e.sum(axis=axis, keepdims=True)


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, want_probs: bool = False):
    """Full (non-causal) softmax attention; q, k, v are [T, H, d_head].  With
    want_probs also the probabilities [H, Tq, Tk].  Heads are independent and
    are computed one at a time, so a long chunk needs one [T, T] score matrix
    at a time."""
    T, H, d_head = q.shape
    o = np.empty((T, H, d_head), dtype=np.result_type(q, k, v))
    probs = []
    for h in range(H):
        p = softmax((q[:, h, :] @ k[:, h, :].T) / math.sqrt(d_head), axis=-1)   # [Tq, Tk]
        o[:, h, :] = p @ v[:, h, :]
        if want_probs:
            probs.append(p)
    return (o, np.stack(probs)) if want_probs else o


def gelu(x: np.ndarray) -> np.ndarray:
    return 0.5 * x * (1.0 + erf(x / math.sqrt(2.0)))


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def block(shape, w: dict, x: np.ndarray, cos, sin, rope: bool = True, probs_out=None) -> np.ndarray:
    """One pre-norm transformer block on the residual stream x [T, d].  If
    probs_out is a list, the head-averaged attention probabilities [Tq, Tk]
    of the block are appended to it."""
    T, d = x.shape
    H, dh = shape.n_heads, shape.d_head
    h = norm(shape, x)
    q = (h @ w["q"].T).reshape(T, H, dh)
    k = (h @ w["k"].T).reshape(T, H, dh)
    v = (h @ w["v"].T).reshape(T, H, dh)
    if rope:
        q, k = apply_rope(q, cos, sin), apply_rope(k, cos, sin)
    if probs_out is None:
        o = attention(q, k, v).reshape(T, d)
    else:
        o, p = attention(q, k, v, want_probs=True)
        o = o.reshape(T, d)
        probs_out.append(p.mean(axis=0))
    x = x + o @ w["o"].T
    h = norm(shape, x)
    if shape.ffn == "gelu":
        f = gelu(h @ w["ffn_in"].T)
    else:
        f = silu(h @ w["ffn_in"].T) * (h @ w["ffn_up"].T)
    return x + f @ w["ffn_out"].T


def hidden(shape, W, state: np.ndarray, rope: bool = True) -> np.ndarray:
    """Final-norm hidden states [T, d] of one chunk ``state`` [T]."""
    state = np.asarray(state, dtype=np.int64)
    T = state.shape[0]
    x = W.embed_rows(state)
    cos, sin = rope_cos_sin(T, shape.d_head, shape.rope_theta)
    for l in range(shape.n_layers):
        x = block(shape, W.layer(l), x, cos, sin, rope=rope)
    return norm(shape, x)


def masked_positions(shape, state: np.ndarray) -> np.ndarray:
    """The masked set M = {x : s~_x = [MASK]} in ascending order."""
    return np.nonzero(np.asarray(state) == shape.mask_id)[0]


def logits(shape, W, state: np.ndarray, rope: bool = True, vocab_rows=None):
    """Logits over Sigma at the masked positions of one chunk: ([|M|, V], M)."""
    pos = masked_positions(shape, state)
    h = hidden(shape, W, state, rope=rope)[pos]
    head = W.head() if vocab_rows is None else W.head_rows(vocab_rows)
    return h @ head.T, pos
