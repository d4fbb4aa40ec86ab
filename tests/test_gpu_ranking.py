"""GPU parity of the symbol ranking back end, through the C ABI.

The rank and select-by-rank kernels are compared exactly with the oracle's
rank definition applied to the same fp32 logits (the comparisons that decide
an integer are taken in the kernel's precision on both sides).  Round trips
cover every compressor, schedules and contexts; on the fp32 tiny model the
ranks stored by the GPU are compared with the oracle's fp64 ranks along the
same (block-schedule) trajectory.
"""
import dataclasses

import numpy as np
import pytest

import workloads as wl
from oracle import driver as OD
from oracle import ranking as R
from oracle import weights as OW

from gpu_common import FIXED_HEADER, codec, log, shape

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

import paper_2608_11249_amd as dl  # noqa: E402


@pytest.mark.parametrize("V", [3, 256, 1001, 32768, 126464])
def test_rank_and_select_kernels_exact(V):
    log("rank kernels", V)
    rng = np.random.default_rng(V)
    rows = 12
    lg = wl.random_logits(V, rows, V, 4.0)
    lg[1] = 0.0                                              # uniform: ranks are ids
    lg[2] = rng.integers(-2, 3, size=V).astype(np.float32)   # heavy ties
    lg[3, : V // 2] = -0.0                                   # signed zeros tie
    lg[3, V // 2:] = 0.0
    lg[4] = -np.inf
    lg[4, V - 1] = 1.0
    sym = rng.integers(0, V, size=rows).astype(np.int32)
    sym[4] = V - 1
    rk = rng.integers(0, V, size=rows).astype(np.int32)
    with dl.Model(shape(vocab=V, n_layers=0), max_chunk=8) as m:
        dlg = torch.from_numpy(lg).cuda()
        got_r = m.rank_rows(dlg, torch.from_numpy(sym).cuda()).cpu().numpy()
        got_s = m.select_rank_rows(dlg, torch.from_numpy(rk).cuda()).cpu().numpy()
        back = m.select_rank_rows(dlg, torch.from_numpy(got_r).cuda()).cpu().numpy()
    for i in range(rows):
        assert got_r[i] == R.rank_of(lg[i], int(sym[i])), i
        assert got_s[i] == R.symbol_at(lg[i], int(rk[i])), i
    assert np.array_equal(back, sym)


def section(container: bytes, kind: str):
    hdr = int.from_bytes(container[8:12], "little")
    nc = int.from_bytes(container[136:144], "little")
    offs = [int.from_bytes(container[FIXED_HEADER + 8 * c: FIXED_HEADER + 8 + 8 * c], "little")
            for c in range(nc + 1)]
    body = R.decompress(container[hdr:], kind)
    return [body[offs[c]: offs[c + 1]] for c in range(nc)]


@pytest.mark.parametrize("kw", [
    dict(schedule="uniform", blocks=32, m_min=1, m_max=8, rank_compressor="lzma", rank_level=9),
    dict(schedule="uniform", blocks=16, m_min=1, m_max=64, rank_compressor="zlib", rank_level=9,
         context=2, context_kind="random", context_seed=4),
    dict(schedule="uniform", blocks=8, m_min=1, m_max=32, rank_compressor="zstd", rank_level=3),
])
def test_tiny_ranks_against_oracle(kw):
    w = wl.WORKLOADS["tiny"]
    cd = dataclasses.replace(w.codec, batch=2, coder="rank", **kw)
    toks = wl.make_tokens(w, 512)
    log("tiny ranks vs oracle", kw)
    with dl.Model(w.model, max_chunk=256, max_batch=2) as m:
        data = m.encode(toks, cd)
        assert np.array_equal(m.decode(data, batch=1), toks)
    res = OD.encode(w.model, OW.Weights(w.model), toks, cd)
    ours = section(data, cd.rank_compressor)
    same = total = 0
    for r, g in zip(res, ours):
        c = min(cd.context, 256)
        assert g[: 6 * c] == r.payload[: 6 * c]
        n = 256 - c
        a, _ = R.varint_decode(g, n, 6 * c)
        b, _ = R.varint_decode(r.payload, n, 6 * c)
        same += sum(x == y for x, y in zip(a, b))
        total += n
    log(f"ranks equal to the oracle's fp64 ranks: {same}/{total}")
    assert same >= 0.99 * total


@pytest.mark.parametrize("comp,level", [("none", 0), ("zlib", 6), ("lzma", 6), ("zstd", 19)])
@pytest.mark.parametrize("sched", [dict(mmin=4, mmax=4),
                                   dict(schedule="progressive", u1=1, growth=1.5, mmin=1, mmax=64,
                                        context=3, context_kind="random", context_seed=2)])
def test_bf16_rank_roundtrip_and_batch_invariance(comp, level, sched):
    sh = shape(ffn="swiglu", norm="rmsnorm", vocab=5000)
    cd = codec(64, batch=4, coder="rank", rank_compressor=comp, rank_level=level, **sched)
    toks = wl.markov1_tokens(64 * 3 + 29, sh.vocab, 8)
    log("bf16 rank round trip", comp, sched)
    with dl.Model(sh, max_chunk=64, max_batch=4) as m:
        a = m.encode(toks, cd, crc=True)
        b = m.encode(toks, cd, batch=1, crc=True)
        # identical apart from the header's default decode batch (bytes 72..75)
        assert a[:72] == b[:72] and a[76:] == b[76:]
        assert np.array_equal(m.decode(a, batch=2), toks)
        if comp in ("zlib", "lzma", "zstd"):
            assert section(a, comp)  # the section is a valid stream of that compressor


def test_rank_container_errors():
    sh = shape()
    toks = wl.markov1_tokens(100, sh.vocab, 3)
    cd = codec(50, k=5, coder="rank", rank_compressor="zlib", rank_level=9)
    with dl.Model(sh, max_chunk=64) as m:
        data = bytearray(m.encode(toks, cd))
        data[-2] ^= 0x55                               # damage the compressed section
        with pytest.raises(dl.DlmcError) as e:
            m.decode(bytes(data))
        assert e.value.code in (-4, -5)
        with pytest.raises(dl.DlmcError) as e:         # zlib level out of range
            m.encode(toks, dataclasses.replace(cd, rank_level=12))
        assert e.value.code == -1
