"""GPU parity of the left-to-right block schedules (uniform block,
progressive), the rANS coder and the initial context, through the C ABI.

Block schedules fix their positions in advance, so the GPU and the oracle
follow the same trajectory: selections and stored contexts are compared
exactly, and the information content of the coded symbols (sum -log2 q, q
= f / 2^P) within 0.5% of the oracle's along the GPU's trajectory, with no
additive slack.
"""
import dataclasses
import math

import numpy as np
import pytest

import workloads as wl
from oracle import driver as OD
from oracle import weights as OW

from gpu_common import codec, log, payloads, shape

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

import paper_2608_11249_amd as dl  # noqa: E402


TINY_CASES = [
    dict(schedule="uniform", blocks=16, m_min=16, m_max=16),
    dict(schedule="progressive", u1=2, growth=1.5, m_min=1, m_max=128),
    dict(schedule="uniform", blocks=12, m_min=1, m_max=32, coder="rans", context=8,
         context_kind="random", context_seed=5),
    dict(m_min=4, m_max=4, coder="rans", context=3, context_kind="contiguous"),
    dict(schedule="uniform", blocks=256, m_min=1, m_max=1, coder="rans"),   # autoregressive
]


@pytest.mark.parametrize("kw", TINY_CASES)
def test_tiny_against_oracle(kw):
    """fp32 tiny model, two 256-byte chunks: same selections and contexts as
    the oracle; along the GPU's trajectory the coded symbols' information
    content sum -log2 (f / 2^P) is within 0.5% of the oracle's (no additive
    slack); exact round trip."""
    w = wl.WORKLOADS["tiny"]
    cd = dataclasses.replace(w.codec, batch=2, **kw)
    toks = wl.make_tokens(w, 512)
    log("tiny vs oracle", kw)
    sel, coded = {}, {}

    def tr(d, chunk, pas, pos, ent, iv, h):
        if d == 0:
            sel[(chunk, pas)] = tuple(pos)
            coded[(chunk, pas)] = tuple(iv)

    with dl.Model(w.model, max_chunk=256, max_batch=2) as m:
        m.set_trace(tr, coded=True)
        data = m.encode(toks, cd)
        m.set_trace(None)
        assert np.array_equal(m.decode(data, batch=1), toks)
    W = OW.Weights(w.model)
    res = OD.encode(w.model, W, toks, cd)
    P = cd.cdf_bits
    for c, (r, gp) in enumerate(zip(res, payloads(data))):
        ctx = min(cd.context, 256)
        assert gp[: 6 * ctx] == r.payload[: 6 * ctx]            # stored context, bit-exact
        n_pass = sum(1 for (cc, _) in sel if cc == c)
        if cd.schedule != "entropy":
            assert [sel[(c, p)] for p in range(r.passes)] == [tuple(s.tolist()) for s in r.selections]
            assert n_pass == r.passes
        forced = [np.array(sel[(c, p)], dtype=np.int64) for p in range(n_pass)]
        along = OD.encode_chunk(w.model, W, toks[c * 256:(c + 1) * 256], cd, forced=forced, chunk_index=c)
        gpu_bits = sum(P - math.log2(f) for p in range(n_pass) for _, f in coded[(c, p)])
        rel = abs(gpu_bits - along.ideal_bits) / along.ideal_bits
        log(f"chunk {c}: {gpu_bits:.3f} vs oracle {along.ideal_bits:.3f} bits, rel {rel:.2e}")
        assert rel <= 0.005


@pytest.mark.parametrize("kw", [
    dict(schedule="uniform", blocks=7, mmin=1, mmax=16, coder="rans", context=5,
         context_kind="random", context_seed=3),
    dict(schedule="progressive", u1=1, growth=1.4, mmin=1, mmax=64, context=2),
    dict(tau=2.0, mmin=1, mmax=8, coder="rans", context=4, context_kind="random", context_seed=9),
])
def test_bf16_batch_invariance_and_roundtrip(kw):
    sh = shape(ffn="swiglu", norm="rmsnorm")
    cd = codec(64, P=24, W=64, batch=4, **kw)
    toks = wl.markov1_tokens(64 * 5 + 23, sh.vocab, 21)
    log("bf16 batch invariance", kw)
    with dl.Model(sh, max_chunk=64, max_batch=4) as m:
        a = m.encode(toks, cd, crc=True)
        b = m.encode(toks, cd, batch=1, crc=True)
        assert payloads(a) == payloads(b)
        assert np.array_equal(m.decode(a, batch=3), toks)


def test_schedule_errors():
    sh = shape()
    toks = wl.markov1_tokens(100, sh.vocab, 1)
    with dl.Model(sh, max_chunk=64) as m:
        with pytest.raises(dl.DlmcError) as e:      # a 64-symbol block exceeds m_max = 8
            m.encode(toks, codec(64, mmin=1, mmax=8, schedule="uniform", blocks=1))
        assert e.value.code == -1
        cd = codec(64, mmin=1, mmax=16, schedule="uniform", blocks=8, coder="rans", context=3)
        data = bytearray(m.encode(toks, cd))
        hdr = int.from_bytes(data[8:12], "little")
        data[hdr] = 0xFF                               # first context position out of range
        data[hdr + 1] = 0xFF
        with pytest.raises(dl.DlmcError) as e:
            m.decode(bytes(data))
        assert e.value.code == -5


# ---------------------------------------------------------------- attention-based context
from oracle import context as OX  # noqa: E402


@pytest.mark.parametrize("T", [64, 256])
def test_context_scores_against_oracle_fp32(T):
    w = wl.WORKLOADS["tiny"]
    toks = wl.make_tokens(w, T)
    log("context scores fp32", T)
    with dl.Model(w.model, max_chunk=T) as m:
        got = m.context_scores(toks).astype(np.float64)
    ref = OX.context_scores(w.model, OW.Weights(w.model), toks)
    assert np.max(np.abs(got - ref)) <= 1e-4 * np.max(np.abs(ref)) + 1e-6
    # the selection wherever the c-th boundary is clear of the numeric error
    order = sorted(range(T), key=lambda j: (-ref[j], j))
    for c in (1, 5, T // 4):
        if ref[order[c - 1]] - ref[order[c]] > 1e-3 * np.max(np.abs(ref)):
            sel = sorted(range(T), key=lambda j: (-got[j], j))[:c]
            assert sorted(sel) == sorted(order[:c]), c


def test_attention_context_roundtrip_and_stored_positions_bf16():
    sh = shape(ffn="swiglu", norm="rmsnorm")
    cd = codec(64, P=24, W=64, batch=2, mmin=4, mmax=4, coder="rans", context=6,
               context_kind="attention")
    toks = wl.markov1_tokens(64 * 2 + 20, sh.vocab, 31)
    log("attention context bf16")
    with dl.Model(sh, max_chunk=64, max_batch=2) as m:
        data = m.encode(toks, cd)
        assert np.array_equal(m.decode(data, batch=1), toks)
        for c, p in enumerate(payloads(data)):
            seg = toks[64 * c: 64 * (c + 1)]
            sc = m.context_scores(seg)
            top = sorted(sorted(range(len(seg)), key=lambda j: (-sc[j], j))[:min(6, len(seg))])
            assert np.frombuffer(p[: 2 * len(top)], dtype="<u2").tolist() == top
        ref = OX.context_scores(sh, OW.Weights(sh), toks[:64])
        got = m.context_scores(toks[:64]).astype(np.float64)
    assert np.max(np.abs(got - ref)) <= 3e-2 * np.max(np.abs(ref))
