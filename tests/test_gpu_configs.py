"""GPU checks of the five workload configurations at their real model shapes.

Round trips use a prefix of each workload's seeded stream (whole chunks, in
the workload's chunk length and schedule).  The small workload runs its full
batch of 64 chunks; the 8B-shaped ones run reduced batches (8 of 32 chunks
under the 0.5-bit rule, 1 of 4 long chunks), where a full batch would not fit
a test's time budget -- the kernels are batch invariant, which test_gpu_parity
checks separately.  Logits of the 8B-shaped
model are compared with the oracle at full width with one layer (the launch
shapes of every kernel are those of the 32-layer model), on a sample of
vocabulary columns.
"""
import dataclasses
import time

import numpy as np
import pytest

import workloads as wl
from oracle import model as OM
from oracle import weights as OW

from gpu_common import log, payloads, rel_err_rows, shape

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

import paper_2608_11249_amd as dl  # noqa: E402


def dev_state(st):
    return torch.from_numpy(np.ascontiguousarray(st, dtype=np.int32)).cuda()


def roundtrip_workload(name, n_chunks, batch=None, trace=False):
    """Round trip of the first n_chunks chunks of a workload.  With trace, the
    per-pass decisions of encode and decode (positions, entropies, coded
    intervals, CDF hashes) must be identical."""
    w = wl.WORKLOADS[name]
    cd = w.codec if batch is None else dataclasses.replace(w.codec, batch=batch)
    toks = wl.make_tokens(w, n_chunks * cd.chunk_len)
    log("round trip", name, f"{n_chunks} chunks x {cd.chunk_len}, batch {cd.batch}")
    traces = {0: {}, 1: {}}

    def tr(d, chunk, pas, pos, ent, coded, h):
        traces[d][(chunk, pas)] = (tuple(pos), tuple(ent), tuple(coded), h)

    with dl.Model(w.model, max_chunk=cd.chunk_len, max_batch=cd.batch) as m:
        if trace:
            m.set_trace(tr, coded=True)
        t0 = time.time()
        data = m.encode(toks, cd)
        t1 = time.time()
        back = m.decode(data)
        t2 = time.time()
        m.set_trace(None)
    assert np.array_equal(back, toks)
    if trace:
        assert len(traces[0]) > 0 and traces[0] == traces[1]
        log(f"{name}: encode and decode traces identical over {len(traces[0])} (chunk, pass) records")
    log(f"{name}: {len(toks)} tokens -> {len(data)} bytes "
        f"({8 * len(data) / (len(toks) * w.token_bytes):.3f} bits/input byte), "
        f"encode {t1 - t0:.1f}s decode {t2 - t1:.1f}s")
    return data


def test_roundtrip_small_config():
    # the full batch: 64 chunks of 1024 tokens per forward, one batch
    roundtrip_workload("small", 64, trace=True)


def test_roundtrip_8b_config():
    roundtrip_workload("8b", 1, trace=True)


def test_roundtrip_8b_threshold_schedule():
    # tau = 0.5 bits, 1..64 positions per pass; report the pass count
    w = wl.WORKLOADS["8b-throughput"]
    nb = 8
    cd = dataclasses.replace(w.codec, batch=nb)
    toks = wl.make_tokens(w, nb * cd.chunk_len)
    log("8b-throughput round trip", f"{nb} chunks x {cd.chunk_len}, batch {nb}")
    traces = {0: {}, 1: {}}

    def tr(d, chunk, pas, pos, ent, coded, h):
        traces[d][(chunk, pas)] = (tuple(pos), tuple(ent), tuple(coded), h)

    with dl.Model(w.model, max_chunk=cd.chunk_len, max_batch=nb) as m:
        m.set_trace(tr, coded=True)
        data = m.encode(toks, cd)
        back = m.decode(data)
        m.set_trace(None)
    assert np.array_equal(back, toks)
    # encode and decode took bit-identical decisions under the 0.5-bit rule
    assert traces[0] == traces[1]
    counts = [(c, len(t[0])) for (c, _), t in traces[0].items()]
    per_chunk = [sum(1 for c, _ in counts if c == k) for k in range(nb)]
    assert all(1 <= n <= 64 for _, n in counts)
    # every pass commits all positions at or under 0.5 bits (capped at 64),
    # at least one
    for t in traces[0].values():
        ent = t[1]
        assert sum(h <= 0.5 for h in ent) == len(ent) or len(ent) == 1 or len(ent) == 64
    log("8b-throughput passes per chunk", per_chunk)


def test_roundtrip_8b_long_chunk():
    roundtrip_workload("8b-long", 1, batch=1)


def test_logits_8b_full_width_one_layer():
    sh = wl.with_layers(wl.DLM8B, 1)
    T = 2048
    st = wl.random_state(21, 1, T, sh.vocab, 0.5)
    st[0, 0] = sh.mask_id
    cols = np.sort(np.random.default_rng(0).choice(sh.vocab, 4096, replace=False))
    log("8b full width L=1 logits", T)
    with dl.Model(sh, max_chunk=T, max_batch=1) as m:
        lg, rows = m.forward_logits(dev_state(st))
        gpu = lg[:, torch.from_numpy(cols).cuda()].cpu().numpy()
        rows = rows.cpu().numpy()
    W = OW.Weights(sh)
    ref, pos = OM.logits(sh, W, st[0], vocab_rows=cols)
    assert np.array_equal(rows, pos)
    err = rel_err_rows(gpu, ref)
    log("max rel err", err)
    assert err <= 2e-2


@pytest.mark.timeout(400)  # the fp64 oracle takes about a minute at T = 8192
def test_logits_8b_long_attention_launch():
    """The long-chunk workload's attention launch: d_model 4096, 32 heads of
    128, one chunk of 8192 (with four chunks the workload runs the same
    blocks): (8192 / 256) x 32 = 1024 blocks, so attention runs 256-query
    blocks.  One layer, a small FFN and vocabulary keep the fp64 oracle
    affordable; QKV, attention and O-proj run at the workload's shape."""
    sh = dataclasses.replace(wl.with_layers(wl.DLM8B, 1), d_ffn=512, vocab=384,
                             ffn_out_exp=wl.fan_in_exp(512))
    T = 8192
    st = wl.random_state(23, 1, T, sh.vocab, 0.3)
    log("8b-long attention launch: L=1 d=4096 32x128 T=8192")
    with dl.Model(sh, max_chunk=T, max_batch=1) as m:
        lg, rows = m.forward_logits(dev_state(st))
        lg, rows = lg.cpu().numpy(), rows.cpu().numpy()
    log("oracle (fp64) forward at T=8192")
    ref, pos = OM.logits(sh, OW.Weights(sh), st[0])
    assert np.array_equal(rows, pos)
    err = rel_err_rows(lg, ref)
    log("max rel err", err)
    assert err <= 2e-2


def test_logits_long_chunk_attention():
    # T = 8192 non-causal attention with head dim 128 (one head)
    sh = shape(d_model=128, n_heads=1, d_ffn=128, n_layers=1, vocab=300, ffn="swiglu",
               norm="rmsnorm")
    T = 8192
    st = wl.random_state(5, 1, T, sh.vocab, 0.3)
    log("attention T=8192")
    with dl.Model(sh, max_chunk=T, max_batch=1) as m:
        lg, rows = m.forward_logits(dev_state(st))
        lg, rows = lg.cpu().numpy(), rows.cpu().numpy()
    ref, pos = OM.logits(sh, OW.Weights(sh), st[0])
    assert np.array_equal(rows, pos)
    err = rel_err_rows(lg, ref)
    log("max rel err", err)
    assert err <= 2e-2


def test_roundtrip_8b_uniform_blocks_rans_context():
    """The paper's best trade-off family at the 8B shape: uniform blocks of 16
    (K = 128 on a 2048-token chunk), rANS, two random context symbols."""
    w = wl.WORKLOADS["8b"]
    cd = dataclasses.replace(w.codec, schedule="uniform", blocks=128, m_min=1, m_max=160,
                             coder="rans", context=2, context_kind="random", context_seed=1)
    toks = wl.make_tokens(w, cd.chunk_len)
    log("round trip 8b uniform/rANS/context", cd)
    sizes = []

    def tr(d, chunk, pas, pos, ent, h):
        if d == 0:
            sizes.append(len(pos))

    with dl.Model(w.model, max_chunk=cd.chunk_len, max_batch=1) as m:
        m.set_trace(tr)
        t0 = time.time()
        data = m.encode(toks, cd)
        t1 = time.time()
        m.set_trace(None)
        back = m.decode(data)
        t2 = time.time()
    assert np.array_equal(back, toks)
    # 2046 masked positions in 128 blocks: 127 of 15, the last 15 + 141
    assert sizes == [15] * 127 + [15 + 2046 - 15 * 128]
    log(f"8b uniform: {len(data)} bytes, encode {t1 - t0:.1f}s decode {t2 - t1:.1f}s")


def test_roundtrip_8b_attention_context():
    """Attention-based context at the 8B shape: two extra passes store and read
    32 head-averaged 2048 x 2048 maps; the stored context is the top of the
    GPU's own scores."""
    w = wl.WORKLOADS["8b"]
    cd = dataclasses.replace(w.codec, schedule="uniform", blocks=128, m_min=1, m_max=160,
                             coder="rans", context=8, context_kind="attention")
    toks = wl.make_tokens(w, cd.chunk_len)
    log("round trip 8b attention context", cd)
    with dl.Model(w.model, max_chunk=cd.chunk_len, max_batch=1) as m:
        t0 = time.time()
        data = m.encode(toks, cd)
        t1 = time.time()
        back = m.decode(data)
        sc = m.context_scores(toks)
    assert np.array_equal(back, toks)
    top = sorted(sorted(range(len(toks)), key=lambda j: (-sc[j], j))[:8])
    (p,) = payloads(data)
    assert np.frombuffer(p[:16], dtype="<u2").tolist() == top
    log(f"8b attention context: encode {t1 - t0:.1f}s, context {top}")
