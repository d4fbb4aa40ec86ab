"""Pins of the oracle's attention-based initial context: the vector chain
against the explicit rollout product, flow conservation, the captured
attention against the block's own output, and the selection rule."""
import dataclasses

import numpy as np
import pytest

import workloads as wl
from oracle import context as OX
from oracle import driver as OD
from oracle import model as OM
from oracle import weights as OW


def small():
    sh = dataclasses.replace(wl.TINY, n_layers=3, name="ctx")
    return sh, OW.Weights(sh)


def test_vector_chain_equals_explicit_rollout():
    sh, W = small()
    toks = wl.markov2_bytes(24, 3)
    masked = np.arange(24) % 2 == 0
    state = np.where(masked, sh.mask_id, toks)
    maps = OX.attention_maps(sh, W, state)
    assert len(maps) == 3
    # the rollout of the paper's reference: R = A~_L ... A~_1, A~ = (A + I) / 2
    R = np.eye(24)
    for A in maps:
        R = (0.5 * A + 0.5 * np.eye(24)) @ R
    np.testing.assert_allclose(OX.rollout_flow(maps, masked), masked.astype(float) @ R, rtol=1e-12)


def test_attention_rows_and_flow_conservation():
    sh, W = small()
    toks = wl.markov2_bytes(30, 5)
    masked = np.arange(30) % 2 == 1
    maps = OX.attention_maps(sh, W, np.where(masked, sh.mask_id, toks))
    for A in maps:                       # softmax rows are distributions
        np.testing.assert_allclose(A.sum(axis=1), 1.0, rtol=1e-12)
        assert np.all(A >= 0)
    # every rollout row sums to one, so the flow out of the masked rows is |M|
    assert OX.rollout_flow(maps, masked).sum() == pytest.approx(masked.sum(), rel=1e-12)


def test_captured_attention_matches_block_output():
    sh, W = small()
    st = np.where(np.arange(16) % 3 == 0, sh.mask_id, wl.markov2_bytes(16, 8))
    x = W.embed_rows(st)
    cos, sin = OM.rope_cos_sin(16, sh.d_head, sh.rope_theta)
    probs = []
    y = OM.block(sh, W.layer(0), x, cos, sin, probs_out=probs)
    np.testing.assert_array_equal(y, OM.block(sh, W.layer(0), x, cos, sin))
    assert probs[0].shape == (16, 16)


def test_no_layers_scores_nothing():
    sh = dataclasses.replace(wl.TINY, n_layers=0, name="ctx0")
    W = OW.Weights(sh)
    # without layers the rollout is the identity: no visible position gets flow,
    # so the selection falls back to the lowest positions
    assert np.all(OX.context_scores(sh, W, wl.markov2_bytes(10, 1)) == 0.0)
    assert OX.attention_context(sh, W, wl.markov2_bytes(10, 1), 3).tolist() == [0, 1, 2]


def test_attention_context_roundtrip():
    w = wl.WORKLOADS["tiny"]
    codec = dataclasses.replace(w.codec, chunk_len=32, m_min=4, m_max=4, context=5,
                                context_kind="attention")
    W = OW.Weights(w.model)
    toks = wl.markov2_bytes(40, 2)
    res = OD.encode(w.model, W, toks, codec)
    sc = OX.context_scores(w.model, W, toks[:32])
    ctx = np.frombuffer(res[0].payload[:10], dtype="<u2").astype(int)
    top = sorted(range(32), key=lambda j: (-sc[j], j))[:5]
    assert sorted(top) == ctx.tolist()
    assert np.array_equal(OD.decode(w.model, W, [r.payload for r in res], 40, codec), toks)
