"""Pins of the oracle forward pass (Definition 3) against library routines,
special cases and invariants."""
import dataclasses
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import workloads as wl
from oracle import model as OM
from oracle import weights as OW


def small_shape(**kw):
    base = dict(name="t", n_layers=2, d_model=64, n_heads=4, d_ffn=96, vocab=50,
                ffn="gelu", norm="layernorm", dtype="f32", embed_exp=0, attn_exp=3,
                ffn_in_exp=3, ffn_out_exp=3, head_exp=3, seed=5)
    base.update(kw)
    return wl.ModelShape(**base)


def torch_forward(shape, W, state):
    """The same network written with torch's own fp64 routines:
    F.layer_norm / F.rms_norm, F.scaled_dot_product_attention (non-causal),
    F.gelu(exact) / F.silu, and RoPE as multiplication by a unit complex
    number on the (i, i + d_head/2) pairs."""
    T = len(state)
    d, H, dh = shape.d_model, shape.n_heads, shape.d_head
    x = torch.from_numpy(W.embed_rows(state))

    def nrm(t):
        if shape.norm == "layernorm":
            return F.layer_norm(t, (d,), eps=shape.norm_eps)
        return F.rms_norm(t, (d,), eps=shape.norm_eps)

    half = dh // 2
    inv = shape.rope_theta ** (-torch.arange(half, dtype=torch.float64) * 2.0 / dh)
    ang = torch.arange(T, dtype=torch.float64)[:, None] * inv[None, :]
    rot = torch.polar(torch.ones_like(ang), ang)          # e^{i angle}

    def rope(t):  # t [T, H, dh]
        z = torch.complex(t[..., :half], t[..., half:]) * rot[:, None, :]
        return torch.cat([z.real, z.imag], dim=-1)

    for l in range(shape.n_layers):
        w = {k: torch.from_numpy(v) for k, v in W.layer(l).items()}
        h = nrm(x)
        q = rope((h @ w["q"].T).view(T, H, dh)).transpose(0, 1)
        k = rope((h @ w["k"].T).view(T, H, dh)).transpose(0, 1)
        v = (h @ w["v"].T).view(T, H, dh).transpose(0, 1)
        o = F.scaled_dot_product_attention(q[None], k[None], v[None], is_causal=False)[0]
        x = x + o.transpose(0, 1).reshape(T, d) @ w["o"].T
        h = nrm(x)
        if shape.ffn == "gelu":
            f = F.gelu(h @ w["ffn_in"].T, approximate="none")
        else:
            f = F.silu(h @ w["ffn_in"].T) * (h @ w["ffn_up"].T)
        x = x + f @ w["ffn_out"].T
    h = nrm(x)
    pos = np.nonzero(np.asarray(state) == shape.mask_id)[0]
    return (h[pos] @ torch.from_numpy(W.head()).T).numpy()


@pytest.mark.parametrize("ffn,norm", [("gelu", "layernorm"), ("swiglu", "rmsnorm")])
@pytest.mark.parametrize("T", [1, 7, 40])
def test_forward_matches_torch_routines(ffn, norm, T):
    shape = small_shape(ffn=ffn, norm=norm, dtype="bf16" if ffn == "swiglu" else "f32")
    W = OW.Weights(shape)
    state = wl.random_state(11 + T, 1, T, shape.vocab, 0.5)[0]
    state[0] = shape.mask_id
    ours, pos = OM.logits(shape, W, state)
    ref = torch_forward(shape, W, state)
    assert ours.shape == ref.shape == (len(pos), shape.vocab)
    assert np.max(np.abs(ours - ref)) <= 1e-11 * max(1.0, np.max(np.abs(ref)))


def test_zero_layers_is_norm_embed_head():
    shape = small_shape(n_layers=0)
    W = OW.Weights(shape)
    state = np.array([3, shape.mask_id, 7, shape.mask_id])
    ours, pos = OM.logits(shape, W, state)
    e = W.embed_rows(state[pos])
    mu = e.mean(1, keepdims=True)
    sd = np.sqrt(((e - mu) ** 2).mean(1, keepdims=True) + shape.norm_eps)
    assert np.allclose(ours, ((e - mu) / sd) @ W.head().T, rtol=0, atol=1e-12)


def test_single_position_attention_returns_values():
    rng = np.random.default_rng(1)
    q, k, v = (rng.standard_normal((1, 3, 8)) for _ in range(3))
    assert np.allclose(OM.attention(q, k, v), v, atol=1e-15)


def test_rope_position_zero_is_identity_and_rotation_is_isometric():
    cos, sin = OM.rope_cos_sin(5, 16, 10000.0)
    rng = np.random.default_rng(2)
    x = rng.standard_normal((5, 2, 16))
    y = OM.apply_rope(x, cos, sin)
    assert np.allclose(y[0], x[0], atol=0)
    assert np.allclose(np.linalg.norm(y, axis=-1), np.linalg.norm(x, axis=-1), atol=1e-12)


def test_rope_scores_depend_only_on_offset():
    # q.k after rotation depends on the position difference only.
    dh, T = 16, 12
    cos, sin = OM.rope_cos_sin(T, dh, 10000.0)
    rng = np.random.default_rng(3)
    q = rng.standard_normal((1, 1, dh)).repeat(T, 0)
    k = rng.standard_normal((1, 1, dh)).repeat(T, 0)
    qr, kr = OM.apply_rope(q, cos, sin)[:, 0], OM.apply_rope(k, cos, sin)[:, 0]
    s = qr @ kr.T
    for off in range(-3, 4):
        d = np.diagonal(s, offset=off)
        assert np.allclose(d, d[0], atol=1e-12)


def test_rope_first_pair_rotates_by_position():
    # rotate-half pairing: dims (0, dh/2) form the plane of the lowest-index
    # (fastest) frequency theta**0 = 1, so e_0 at position p becomes
    # cos(p) e_0 + sin(p) e_{dh/2}.
    dh = 8
    cos, sin = OM.rope_cos_sin(4, dh, 10000.0)
    x = np.zeros((4, 1, dh))
    x[:, 0, 0] = 1.0
    y = OM.apply_rope(x, cos, sin)[:, 0]
    p = np.arange(4)
    assert np.allclose(y[:, 0], np.cos(p)) and np.allclose(y[:, dh // 2], np.sin(p))
    assert np.allclose(np.delete(y, [0, dh // 2], axis=1), 0.0)


def test_permutation_equivariance_without_rope():
    shape = small_shape()
    W = OW.Weights(shape)
    state = wl.random_state(4, 1, 16, shape.vocab, 0.6)[0]
    state[:3] = shape.mask_id
    h = OM.hidden(shape, W, state, rope=False)
    perm = np.random.default_rng(0).permutation(16)
    h2 = OM.hidden(shape, W, state[perm], rope=False)
    assert np.allclose(h2, h[perm], atol=1e-12)


def test_all_mask_rows_identical():
    # with nothing revealed every position has the same input, the same
    # value vectors, hence the same hidden state: a property of the method.
    shape = small_shape()
    W = OW.Weights(shape)
    lg, _ = OM.logits(shape, W, np.full(9, shape.mask_id))
    assert np.allclose(lg, lg[0], atol=1e-12)
