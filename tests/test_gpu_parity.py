"""GPU parity of the HIP path against the CPU oracle, through the C ABI.

Tolerances (logits, per row max |gpu - oracle| / max |oracle|): 1e-5 for the
fp32 model, 2e-2 for bf16 models.  Integer work (selection, CDFs given the
GPU's own g, round trips) is compared bit-exactly.
"""
import math

import numpy as np
import pytest

import workloads as wl
from oracle import cdf as OC
from oracle import driver as OD
from oracle import model as OM
from oracle import schedule as OS
from oracle import weights as OW

from gpu_common import codec, log, payloads, rel_err_rows, shape

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

import paper_2608_11249_amd as dl  # noqa: E402


def dev_state(state):
    return torch.from_numpy(np.ascontiguousarray(state, dtype=np.int32)).cuda()


# ---------------------------------------------------------------- weights
@pytest.mark.parametrize("sh", [
    shape(dtype="f32", d_model=64, n_heads=2, d_ffn=96),
    shape(dtype="bf16", ffn="swiglu", norm="rmsnorm"),
    shape(dtype="bf16", d_model=256, n_heads=2, d_ffn=256, ffn="swiglu", norm="rmsnorm", n_layers=1),
])
def test_weights_bit_identical_to_oracle(sh):
    log("weights", sh)
    W = OW.Weights(sh)
    with dl.Model(sh, max_chunk=8) as m:
        d, F, V = sh.d_model, sh.d_ffn, sh.vocab
        cases = [(1, V + 1, d, sh.embed_exp), (2, V, d, sh.head_exp)]
        for l in range(sh.n_layers):
            b = 16 + 16 * l
            cases += [(b, d, d, sh.attn_exp), (b + 1, d, d, sh.attn_exp), (b + 2, d, d, sh.attn_exp),
                      (b + 3, d, d, sh.attn_exp), (b + 4, F, d, sh.ffn_in_exp),
                      (b + 6, d, F, sh.ffn_out_exp)]
            if sh.ffn == "swiglu":
                cases.append((b + 5, F, d, sh.ffn_in_exp))
        for tid, rows, cols, e in cases:
            got = m.weight(tid, rows, cols)
            ref = OW.gen_tensor(sh.seed, tid, (rows, cols), e, sh.dtype)
            if sh.dtype == "bf16":
                assert np.array_equal(got, OW.bf16_bits(ref)), tid
            else:
                assert np.array_equal(got, ref.astype(np.float32)), tid


# ---------------------------------------------------------------- forward
def check_logits(sh, B, T, mask_frac, tol, seed=0):
    log("logits", sh.name, sh.dtype, f"L={sh.n_layers} d={sh.d_model} B={B} T={T}")
    W = OW.Weights(sh)
    st = wl.random_state(seed, B, T, sh.vocab, mask_frac)
    st[:, 0] = sh.mask_id
    with dl.Model(sh, max_chunk=T, max_batch=B) as m:
        lg, rows = m.forward_logits(dev_state(st))
        lg, rows = lg.cpu().numpy(), rows.cpu().numpy()
    ref_rows, errs = [], []
    for b in range(B):
        ref, pos = OM.logits(sh, W, st[b])
        ref_rows.extend(b * T + pos)
        sel = (rows >= b * T) & (rows < (b + 1) * T)
        errs.append(rel_err_rows(lg[sel], ref))
    assert np.array_equal(rows, np.array(ref_rows))
    err = max(errs)
    log("max rel err", err)
    assert err <= tol, err
    return lg, rows


@pytest.mark.parametrize("B,T", [(3, 256), (2, 100), (1, 1), (1, 77)])
def test_logits_fp32_tiny(B, T):
    check_logits(wl.TINY, B, T, 0.5, 1e-5)


@pytest.mark.parametrize("kw,B,T", [
    (dict(), 2, 100),
    (dict(ffn="swiglu", norm="rmsnorm"), 3, 130),
    (dict(d_model=256, n_heads=2, ffn="swiglu", norm="rmsnorm", vocab=1000), 2, 257),
    (dict(d_model=256, n_heads=4, d_ffn=512, vocab=333), 1, 64),
])
def test_logits_bf16_small_shapes(kw, B, T):
    check_logits(shape(**kw), B, T, 0.6, 2e-2)


@pytest.mark.parametrize("kw", [dict(ffn="swiglu", norm="rmsnorm"), dict(ffn="gelu", norm="layernorm")])
def test_logits_bf16_wide_rows(kw):
    """d_model = 1024 takes the 16-byte-load norm kernel (both norm kinds)."""
    sh = shape(d_model=1024, n_heads=8, d_ffn=1024, n_layers=1, vocab=300, **kw)
    check_logits(sh, 2, 96, 0.6, 2e-2)


def test_logits_bf16_256_tile_ragged_rows():
    """A wide SwiGLU FFN (2F = 98304 columns) puts the FFN-in GEMM on the
    4-wave 256 x 256 kernel; 300 rows leave its second row tile ragged (44
    live rows), whose loads clamp the row index."""
    sh = shape(d_model=128, n_heads=1, d_ffn=49152, ffn="swiglu", norm="rmsnorm", n_layers=1,
               vocab=300)
    check_logits(sh, 1, 300, 0.6, 2e-2)
    check_logits(sh, 2, 256, 0.6, 2e-2, seed=1)


@pytest.mark.parametrize("kw", [dict(ffn="swiglu", norm="rmsnorm"), dict(ffn="gelu", norm="layernorm")])
@pytest.mark.parametrize("B,T", [(1, 300), (2, 256)])
def test_logits_bf16_256x128_tiles(kw, B, T):
    """At 300 or 512 rows, d_model 512, FFN 1024 and vocabulary 384, the tile
    choice puts QKV (rotary epilogue), O-proj and FFN-out (residual), FFN-in
    (SwiGLU or GELU) and the LM head (fp32 store) on the 4-wave 256 x 128
    kernel; 300 rows leave its second row tile ragged."""
    sh = shape(d_model=512, n_heads=4, d_ffn=1024, n_layers=1, vocab=384, **kw)
    check_logits(sh, B, T, 0.6, 2e-2)


def test_logits_bf16_256x256_tiles_head_dim_64():
    """The small model's layer shape (d_model 768, 12 heads of 64, GELU FFN
    3072) at 4 x 1024 rows: QKV and FFN-in take the 4-wave 256 x 256 kernel,
    with the rotary pairs of 64-wide heads inside its 128-column wave tiles."""
    sh = shape(d_model=768, n_heads=12, d_ffn=3072, n_layers=1, vocab=384)
    check_logits(sh, 4, 1024, 0.6, 2e-2)


@pytest.mark.parametrize("B,T", [(4, 1024), (3, 1300)])
def test_logits_bf16_column_split_tiles(B, T):
    """GELU FFN of 4352 at 4096 or 3900 rows: FFN-in splits its columns
    between a 256 x 256 launch (columns 0..2303, 9 x 16 tiles) and a 256 x 128
    launch (the other 2048, 16 x 16 tiles), each filling whole waves of tiles;
    at 3900 rows the last row tile of both launches holds 60 live rows."""
    sh = shape(d_model=256, n_heads=4, d_ffn=4352, n_layers=1, vocab=384)
    check_logits(sh, B, T, 0.6, 2e-2)


def test_logits_qkv_no_wide_tiles_across_q_k_v():
    """d_model 1408 (11 heads of 128) at 4 x 1024 rows: a column split of QKV
    would put a 256-wide tile across the Q / K boundary (column 1408), so QKV
    stays on 256 x 128 tiles, each inside one of Q, K and V."""
    sh = shape(d_model=1408, n_heads=11, d_ffn=512, n_layers=1, vocab=384)
    check_logits(sh, 4, 1024, 0.6, 2e-2)


@pytest.mark.parametrize("d_model,n_heads,B,T", [(2048, 32, 1, 2000), (1024, 8, 4, 1999)])
def test_logits_attention_256_query_blocks(d_model, n_heads, B, T):
    """With at least one 256-query block per CU ((Tp / 256) x heads x batch >=
    256) attention runs 8-wave blocks of 256 queries; a ragged T leaves
    queries and keys past T in the last block (head dims 64 and 128)."""
    sh = shape(d_model=d_model, n_heads=n_heads, d_ffn=512, n_layers=1, vocab=384)
    check_logits(sh, B, T, 0.6, 2e-2)


def test_logits_bf16_small_config():
    sh = wl.WORKLOADS["small"].model
    check_logits(sh, 1, 1024, 0.7, 2e-2)


def test_logits_batch_invariant():
    sh = shape(ffn="swiglu", norm="rmsnorm")
    st = wl.random_state(5, 4, 96, sh.vocab, 0.5)
    with dl.Model(sh, max_chunk=96, max_batch=4) as m:
        lg, rows = m.forward_logits(dev_state(st))
        lg = lg.cpu().numpy()
        rows = rows.cpu().numpy()
        for b in (0, 3):
            one, r1 = m.forward_logits(dev_state(st[b:b + 1]))
            sel = (rows >= b * 96) & (rows < (b + 1) * 96)
            assert np.array_equal(one.cpu().numpy(), lg[sel])


def test_logits_batch_invariant_across_tile_choices():
    """Four chunks of 1024 put FFN-in (4352 columns) on the two-launch column
    split; one chunk alone puts it on a single launch of other tiles.  Every
    chunk's logits must still be bit-identical: each output is the same
    sequential sum over k-tiles whatever tile computes it."""
    sh = shape(d_model=256, n_heads=4, d_ffn=4352, n_layers=1, vocab=384)
    st = wl.random_state(11, 4, 1024, sh.vocab, 0.6)
    with dl.Model(sh, max_chunk=1024, max_batch=4) as m:
        lg, rows = m.forward_logits(dev_state(st))
        lg, rows = lg.cpu().numpy(), rows.cpu().numpy()
        for b in (0, 3):
            one, r1 = m.forward_logits(dev_state(st[b:b + 1]))
            sel = (rows >= b * 1024) & (rows < (b + 1) * 1024)
            assert np.array_equal(r1.cpu().numpy() + b * 1024, rows[sel])
            assert np.array_equal(one.cpu().numpy(), lg[sel])


# ---------------------------------------------------------------- entropy / CDF
@pytest.mark.parametrize("V,P,scale", [(256, 16, 3.0), (1001, 16, 8.0), (32768, 24, 2.0),
                                       (126464, 24, 9.0)])
def test_entropy_and_cdf_kernels(V, P, scale):
    log("entropy/cdf", V, P)
    sh = shape(vocab=V, n_layers=0)
    lg = wl.random_logits(V + 1, 24, V, scale)
    lg[3] = 0.0                     # uniform row
    lg[4] = -50.0
    lg[4, 7] = 10.0                 # one dominant symbol
    with dl.Model(sh, max_chunk=8) as m:
        H, mx, g, cdf = m.entropy_cdf(torch.from_numpy(lg).cuda(), P)
        H, mx, g, cdf = (t.cpu().numpy() for t in (H, mx, g, cdf))
    g = g.view(np.uint32).astype(np.int64)
    cdf = cdf.view(np.uint32).astype(np.int64)
    Href = OS.entropy_bits(lg.astype(np.float64))
    assert np.max(np.abs(H - Href)) <= 1e-3, np.max(np.abs(H - Href))
    assert np.array_equal(mx, lg.max(axis=1))
    for i in range(len(lg)):
        gref = OC.quantise_g(lg[i])
        assert np.max(np.abs(g[i] - gref)) <= 2
        # the integer stage is bit-exact given the GPU's own g
        assert np.array_equal(cdf[i], OC.integer_cdf(g[i], P)), i


# ---------------------------------------------------------------- selection
@pytest.mark.parametrize("tau,mmin,mmax", [(float("-inf"), 4, 4), (0.5, 1, 64), (3.0, 2, 5),
                                           (100.0, 1, 16), (float("-inf"), 64, 64)])
def test_select_kernel_exact(tau, mmin, mmax):
    log("select", tau, mmin, mmax)
    B, T = 5, 300
    rng = np.random.default_rng(mmax)
    st = wl.random_state(9, B, T, 10, 0.6)
    st[3] = 0                       # a chunk with nothing masked
    st[4] = 10                      # fully masked
    rows = np.nonzero(st.reshape(-1) == 10)[0].astype(np.int32)
    H = np.round(rng.uniform(0, 6, len(rows)), 1).astype(np.float32)   # many ties
    sh = shape(vocab=10, n_layers=0)
    with dl.Model(sh, max_chunk=T, max_batch=B) as m:
        sp, sr, ns = m.select(torch.from_numpy(H).cuda(), torch.from_numpy(rows).cuda(), B, T,
                              tau, mmin, mmax)
        sp, sr, ns = sp.cpu().numpy(), sr.cpu().numpy(), ns.cpu().numpy()
    for b in range(B):
        seg = (rows >= b * T) & (rows < (b + 1) * T)
        pos = rows[seg] - b * T
        ref = OS.select(H[seg].astype(np.float64), pos, tau, mmin, mmax)
        assert ns[b] == len(ref)
        assert np.array_equal(sp[b, : ns[b]], ref)
        assert np.array_equal(rows[sr[b, : ns[b]]] - b * T, ref)


# ---------------------------------------------------------------- round trips
def roundtrip(m, toks, cd, batch_dec=0, crc=False):
    data = m.encode(toks, cd, crc=crc)
    back = m.decode(data, batch=batch_dec)
    assert np.array_equal(back, toks)
    return data


def coded_bits(pairs, P):
    """sum -log2(f / 2^P) over coded (start, f) pairs: the information content
    of the symbols under the quantised distributions actually coded."""
    return float(sum(P - math.log2(f) for _, f in pairs))


def trace_recorder():
    traces = {0: {}, 1: {}}

    def tr(d, chunk, pas, pos, ent, coded, h):
        traces[d][(chunk, pas)] = (tuple(pos), tuple(ent), tuple(coded), h)

    return traces, tr


def test_roundtrip_tiny_workload_full_with_trace_and_code_length():
    """fp32 tiny model, the whole 4 KiB input: encode and decode take
    bit-identical decisions; along the GPU's own trajectory the code length
    sum -log2 q of the coded symbols is within 0.5% of the oracle's (no
    additive slack); and the GPU payload is exactly what the oracle's range
    coder writes for the GPU's coded intervals."""
    from oracle import coder as ORC
    w = wl.WORKLOADS["tiny"]
    toks = wl.make_tokens(w)
    log("tiny round trip", len(toks))
    traces, tr = trace_recorder()
    with dl.Model(w.model, max_chunk=w.codec.chunk_len, max_batch=w.codec.batch) as m:
        m.set_trace(tr, coded=True)
        data = roundtrip(m, toks, w.codec)
        m.set_trace(None)
    # encode and decode made bit-identical decisions, CDFs and coded intervals
    assert traces[0] == traces[1] and len(traces[0]) == 16 * 64
    W = OW.Weights(w.model)
    P, Wc = w.codec.cdf_bits, w.codec.coder_bits
    gpu_payloads = payloads(data)
    for c in (0, 7):
        passes = [traces[0][(c, p)] for p in range(64)]
        pairs = [iv for t in passes for iv in t[2]]
        enc = ORC.RangeEncoder(Wc, P)
        for st, f in pairs:
            enc.encode(st, f)
        assert enc.finish() == gpu_payloads[c]
        forced = [np.array(t[0]) for t in passes]
        seg = toks[c * 256:(c + 1) * 256]
        r = OD.encode_chunk(w.model, W, seg, w.codec, forced=forced)
        gpu_bits = coded_bits(pairs, P)
        rel = abs(gpu_bits - r.ideal_bits) / r.ideal_bits
        log(f"tiny chunk {c}: code length {gpu_bits:.3f} vs oracle {r.ideal_bits:.3f} bits, rel {rel:.2e}")
        assert rel <= 0.005


def oracle_bits_along(sh, W, toks, enc_passes, P, sample):
    """sum -log2 q under the oracle's fp64 CDFs of the symbols the GPU coded in
    the sampled passes, each pass evaluated at the state the GPU's earlier
    selections leave (the GPU's trajectory)."""
    from oracle import cdf as OCdf
    T = len(toks)
    bits = 0.0
    for p in sample:
        state = np.full(T, sh.mask_id, dtype=np.int64)
        for q in range(p):
            sel = np.array(enc_passes[q][0], dtype=np.int64)
            state[sel] = toks[sel]
        lg, pos = OM.logits(sh, W, state)
        row_of = {int(x): i for i, x in enumerate(pos)}
        for x in enc_passes[p][0]:
            cdf = OCdf.cdf_row(lg[row_of[int(x)]], P)
            s_ = int(toks[x])
            bits += P - math.log2(int(cdf[s_ + 1] - cdf[s_]))
    return bits


def test_code_length_bf16_small_shape_two_layers():
    """The small model's shape (d 768, 12 heads, GELU 3072, vocabulary 32768)
    with 2 layers, bf16, one 1024-token chunk, k = 8, P = 24, W = 64: encode
    and decode traces are identical, and over every eighth pass (16 passes,
    128 symbols) the GPU's sum -log2 q is within 0.5% of the oracle's fp64
    value along the GPU's trajectory, with no additive slack."""
    w = wl.WORKLOADS["small"]
    sh = wl.with_layers(w.model, 2)
    cd = w.codec
    toks = wl.make_tokens(w, cd.chunk_len)
    log("bf16 code length", sh.name, cd)
    traces, tr = trace_recorder()
    with dl.Model(sh, max_chunk=cd.chunk_len, max_batch=1) as m:
        m.set_trace(tr, coded=True)
        data = m.encode(toks, cd, batch=1)
        back = m.decode(data)
        m.set_trace(None)
    assert np.array_equal(back, toks)
    assert traces[0] == traces[1] and len(traces[0]) == cd.chunk_len // cd.m_max
    enc = [traces[0][(0, p)] for p in range(len(traces[0]))]
    sample = list(range(0, len(enc), 8))
    gpu_bits = sum(coded_bits(enc[p][2], cd.cdf_bits) for p in sample)
    ref_bits = oracle_bits_along(sh, OW.Weights(sh), toks, enc, cd.cdf_bits, sample)
    rel = abs(gpu_bits - ref_bits) / ref_bits
    log(f"bf16 small L=2: code length {gpu_bits:.2f} vs oracle {ref_bits:.2f} bits, rel {rel:.2e}")
    assert rel <= 0.005


@pytest.mark.parametrize("dec_batch", [1, 3])
def test_roundtrip_batch_invariance(dec_batch):
    sh = shape(ffn="swiglu", norm="rmsnorm")
    cd = codec(64, k=5, batch=4)
    toks = wl.markov1_tokens(64 * 5 + 17, sh.vocab, 12)
    log("batch invariance", dec_batch)
    with dl.Model(sh, max_chunk=64, max_batch=4) as m:
        a = roundtrip(m, toks, cd, batch_dec=dec_batch)
        b = m.encode(toks, cd, batch=1)
    assert payloads(a) == payloads(b)


def test_roundtrip_batch_invariance_8b_layer_shape():
    """One layer of the 8B shape, two chunks of 2048: with batch 2 (4096 rows)
    QKV runs on 256 x 256 tiles and O-proj / FFN-out on 256 x 256; with
    batch 1 (2048 rows) QKV runs the column-split kernel and the residual
    GEMMs 256 x 128 tiles.  The payloads must still be byte-identical, and
    the batch-2 container must decode with batch 1."""
    sh = shape(d_model=4096, n_heads=32, d_ffn=12288, ffn="swiglu", norm="rmsnorm", n_layers=1,
               vocab=384)
    cd = codec(2048, k=64, batch=2)
    toks = wl.markov1_tokens(2 * 2048, sh.vocab, 13)
    with dl.Model(sh, max_chunk=2048, max_batch=2) as m:
        a = roundtrip(m, toks, cd, batch_dec=1)
        b = m.encode(toks, cd, batch=1)
    assert payloads(a) == payloads(b)


def test_roundtrip_batch_invariance_attention_block_size():
    """One layer of the small model's shape (12 heads of 64), eight chunks of
    1024: with batch 8 attention runs 256-query blocks ((1024 / 256) x 12 x 8
    >= 256), with batch 1 128-query blocks.  The payloads must not change."""
    sh = shape(d_model=768, n_heads=12, d_ffn=3072, n_layers=1, vocab=384)
    cd = codec(1024, k=64, batch=8)
    toks = wl.markov1_tokens(8 * 1024, sh.vocab, 14)
    with dl.Model(sh, max_chunk=1024, max_batch=8) as m:
        a = roundtrip(m, toks, cd, batch_dec=1)
        b = m.encode(toks, cd, batch=1)
    assert payloads(a) == payloads(b)


def test_roundtrip_batch_invariance_192_row_tiles():
    """One layer of the small model's shape, 32 chunks of 1024: with batch 32
    (32768 rows) QKV and the GELU FFN-in run on 192 x 128 tiles, two blocks
    per CU, whose row tiles straddle chunk boundaries; with batch 1 (1024
    rows) they run on 128 x 128 tiles.  The payloads must not change."""
    sh = shape(d_model=768, n_heads=12, d_ffn=3072, n_layers=1, vocab=384)
    cd = codec(1024, k=64, batch=32)
    toks = wl.markov1_tokens(32 * 1024, sh.vocab, 15)
    log("batch invariance, 192 x 128 tiles")
    with dl.Model(sh, max_chunk=1024, max_batch=32) as m:
        a = roundtrip(m, toks, cd, batch_dec=1)
        b = m.encode(toks, cd, batch=1)
    assert payloads(a) == payloads(b)


@pytest.mark.parametrize("kw,cd,n", [
    (dict(), codec(100, tau=4.0, mmin=1, mmax=8, batch=3), 350),
    (dict(ffn="swiglu", norm="rmsnorm", vocab=70000), codec(128, k=16, P=24, W=64, batch=2), 300),
    (dict(dtype="f32", d_model=64, n_heads=4, d_ffn=64, vocab=256), codec(50, k=7, batch=2), 123),
])
def test_roundtrip_schedules_and_coders(kw, cd, n):
    sh = shape(**kw)
    toks = wl.markov1_tokens(n, sh.vocab, 4)
    log("roundtrip", kw, cd)
    with dl.Model(sh, max_chunk=cd.chunk_len, max_batch=cd.batch) as m:
        roundtrip(m, toks, cd, crc=True)


def test_errors_on_gpu_model():
    sh = shape()
    cd = codec(32, k=4)
    toks = wl.markov1_tokens(70, sh.vocab, 1)
    with dl.Model(sh, max_chunk=32) as m:
        data = m.encode(toks, cd, crc=True)
        bad = bytearray(data)
        bad[-3] ^= 0x5A
        with pytest.raises(dl.DlmcError) as e:
            m.decode(bytes(bad))
        assert e.value.code in (-5,)
        with pytest.raises(dl.DlmcError) as e:
            m.encode(np.array([0, 1, sh.vocab]), cd)
        assert e.value.code == -1
    other = shape(seed=4)
    with dl.Model(other, max_chunk=32) as m2:
        with pytest.raises(dl.DlmcError) as e:
            m2.decode(data)
        assert e.value.code == -4


@pytest.mark.parametrize("coder,W", [("range", 32), ("range", 64), ("rans", 32)])
def test_device_decoder_corrupt_streams(coder, W):
    """The device decoders on damaged coded bytes (bf16 model, two chunks
    decoded side by side).  A range stream whose first W/8 bytes are all ones
    gives a first target of 2^P (code - low >= range) and is refused with
    E_CORRUPT; so is an rANS stream whose final state is changed.  Random
    single-byte damage in the payload section is refused with E_CORRUPT or
    decodes: with the per-chunk CRC only to the original tokens, without it to
    any tokens.  The same model then decodes the intact container."""
    sh = shape()
    cd = codec(32, k=4, batch=2, W=W, coder=coder)
    toks = wl.markov1_tokens(100, sh.vocab, 5)
    with dl.Model(sh, max_chunk=32, max_batch=2) as m:
        for crc in (True, False):
            data = m.encode(toks, cd, crc=crc)
            hdr = int.from_bytes(data[8:12], "little")
            offs = [int.from_bytes(data[144 + 8 * c: 152 + 8 * c], "little") for c in range(5)]
            bad = bytearray(data)
            s1 = hdr + offs[1]  # chunk 1's stream (no initial context)
            if coder == "range":
                bad[s1: s1 + W // 8] = b"\xff" * (W // 8)
            else:
                bad[s1 + 3] ^= 0x10  # a bit of the final state below 2^31
            log("corrupt head of chunk 1", coder, W, crc)
            with pytest.raises(dl.DlmcError) as e:
                m.decode(bytes(bad))
            assert e.value.code == -5
            rng = np.random.default_rng(7 + W)
            for trial in range(6):
                bad = bytearray(data)
                pos = int(rng.integers(hdr, len(data)))
                bad[pos] ^= int(rng.integers(1, 256))
                log("corrupt byte", coder, W, crc, pos)
                try:
                    back = m.decode(bytes(bad))
                except dl.DlmcError as err:
                    assert err.code == -5
                else:
                    assert len(back) == len(toks)
                    if crc:
                        assert np.array_equal(back, toks)
            log("intact", coder, W, crc)
            assert np.array_equal(m.decode(data), toks)


def test_decode_damaged_containers():
    """Seeded random damage anywhere in a container -- the header's codec
    fields and chunk offsets included -- through the GPU decoder (range coder
    and rANS, bf16 model, batch 2).  Every launch size comes from fields that
    the header checks bound by the model (chunk length, batch, m_max, CDF
    bits, context), so each decode returns some tokens or raises a format,
    corrupt, buffer or argument error (codec fields out of range), never a
    device error; the intact container still decodes."""
    sh = shape()
    toks = wl.markov1_tokens(90, sh.vocab, 12)
    rng = np.random.default_rng(5)
    with dl.Model(sh, max_chunk=32, max_batch=2) as m:
        for coder in ("range", "rans"):
            cd = codec(32, k=4, batch=2, coder=coder)
            data = m.encode(toks, cd)
            for trial in range(30):
                bad = bytearray(data)
                if trial % 3 == 2:
                    bad = bad[: int(rng.integers(1, len(bad)))]
                else:
                    for _ in range(int(rng.integers(1, 4))):
                        bad[int(rng.integers(0, len(bad)))] ^= int(rng.integers(1, 256))
                log("damaged container", coder, trial)
                try:
                    m.decode(bytes(bad))
                except dl.DlmcError as e:
                    # never E_DEVICE: no launch may fail
                    assert e.code in (-1, -4, -5, -6), (coder, trial, e)
            log("intact", coder)
            assert np.array_equal(m.decode(data), toks)


def test_stage_profile_mask():
    """Only the stages named in the profile mask are timed; the CDF stage's
    work is filled in only when it is itself timed."""
    sh = shape(ffn="swiglu", norm="rmsnorm")
    cd = codec(64, k=8)
    toks = wl.markov1_tokens(64, sh.vocab, 2)
    log("profile mask", sh, cd)
    with dl.Model(sh, max_chunk=64) as m:
        enc = m.encoder(cd, toks)
        m.profile(True, stages=["ffn_in", "reveal"])
        enc.step()
        p = m.profile_read()
        assert p["ffn_in"][1] == sh.n_layers and p["ffn_in"][2] > 0
        assert p["reveal"][1] == 1
        for name, (ms, n, work) in p.items():
            if name not in ("ffn_in", "reveal"):
                assert n == 0 and ms == 0.0 and work == 0.0, name
        m.profile(True)
        enc.step()
        p = m.profile_read()
        assert all(p[s][1] > 0 for s in ("qkv", "attn", "oproj", "ffn_in", "ffn_out", "head", "cdf"))
        assert p["cdf"][2] == 8 * (8.0 * sh.vocab + 4.0)
        # one layer per forward: one FFN-in launch per pass, the head as usual
        m.profile(True, stages=["ffn_in", "head"], one_layer=True)
        for _ in range(3):
            enc.step()
        p = m.profile_read()
        assert p["ffn_in"][1] == 3 and p["head"][1] == 3 and p["qkv"][1] == 0
        m.profile(False)


# ---------------------------------------------------------------- error codes
def test_numeric_errors():
    """E_NUMERIC: the schedule refuses non-finite entropies, and the encoder
    refuses a pass whose model output holds a NaN (forced by the test hook);
    the model keeps working afterwards."""
    sh = shape(vocab=10, n_layers=0)
    rows = np.arange(8, dtype=np.int32)
    H = np.linspace(0.5, 3.0, 8).astype(np.float32)
    H[5] = np.nan
    with dl.Model(sh, max_chunk=16) as m:
        with pytest.raises(dl.DlmcError) as e:
            m.select(torch.from_numpy(H).cuda(), torch.from_numpy(rows).cuda(), 1, 16,
                     float("-inf"), 2, 2)
        assert e.value.code == -7
        H[5] = np.inf
        with pytest.raises(dl.DlmcError) as e:
            m.select(torch.from_numpy(H).cuda(), torch.from_numpy(rows).cuda(), 1, 16, 1.0, 1, 4)
        assert e.value.code == -7
    sh = shape()
    cd = codec(32, k=4)
    toks = wl.markov1_tokens(70, sh.vocab, 3)
    with dl.Model(sh, max_chunk=32) as m:
        m.inject_nonfinite(True)
        with pytest.raises(dl.DlmcError) as e:
            m.encode(toks, cd)
        assert e.value.code == -7
        m.inject_nonfinite(False)
        assert np.array_equal(m.decode(m.encode(toks, cd)), toks)


def test_out_of_memory_is_reported():
    """E_NOMEM: a workspace for 128 chunks of 8192 tokens over a 126464-symbol
    vocabulary needs 530 GB of fp32 logits; the model is refused before any
    kernel runs, and the GPU stays usable."""
    big = shape(n_layers=0, vocab=126464)
    with pytest.raises(dl.DlmcError) as e:
        dl.Model(big, max_chunk=8192, max_batch=128)
    assert e.value.code == -2
    sh = shape()
    toks = wl.markov1_tokens(40, sh.vocab, 5)
    with dl.Model(sh, max_chunk=32) as m:
        assert np.array_equal(m.decode(m.encode(toks, codec(32, k=4))), toks)


# ---------------------------------------------------------------- chunk ranges
@pytest.mark.parametrize("kw", [
    dict(k=5),
    dict(mmin=1, mmax=16, schedule="uniform", blocks=8, coder="rank", rank_compressor="zlib",
         rank_level=6),
    dict(k=4, coder="rans", context=3, context_kind="random", context_seed=2),
])
def test_encode_range_and_merge_byte_identical(kw):
    """Chunks [0, 2) coded by one model handle and [2, 6) by another (the last
    chunk partial), merged: byte-identical to one encode of the whole input
    (windows are independent), and the merged container decodes.  A partial
    container does not decode on its own."""
    sh = shape(ffn="swiglu", norm="rmsnorm")
    cd = codec(64, P=24, W=64, batch=2, **kw)
    toks = wl.markov1_tokens(64 * 5 + 23, sh.vocab, 17)
    log("encode range + merge", kw)
    with dl.Model(sh, max_chunk=64, max_batch=2) as m1, dl.Model(sh, max_chunk=64, max_batch=2) as m2:
        full = m1.encode(toks, cd, crc=True)
        a = m1.encode_range(toks, cd, 0, 2, crc=True)
        b = m2.encode_range(toks, cd, 2, 4, crc=True)
        assert dl.merge([b, a]) == full
        c = m2.encode_range(toks, cd, 3, 2 ** 64 - 1, crc=True)           # to the last chunk
        mid = m1.encode_range(toks, cd, 2, 1, crc=True)
        assert dl.merge([a, mid, c]) == full
        assert np.array_equal(m2.decode(dl.merge([a, b]), batch=1), toks)
        with pytest.raises(dl.DlmcError) as e:
            m1.decode(a)
        assert e.value.code == -4
        with pytest.raises(dl.DlmcError) as e:
            m1.encode_range(toks, cd, 5, 2)
        assert e.value.code == -1


@pytest.mark.parametrize("kw,T,V", [
    (dict(ffn="swiglu", norm="rmsnorm"), 96, 500),       # 128 x 128 head tiles, ragged group
    (dict(d_model=512, n_heads=4, d_ffn=1024), 300, 384),  # 256 x 128 head tiles
    (dict(d_model=128, n_heads=1, d_ffn=256), 600, 98304),  # 256 x 256 head tiles
])
def test_fused_head_statistics_equal_standalone(kw, T, V):
    """The entropies the encoder uses come from softmax statistics fused into
    the LM head's epilogue; at every pass they must equal, bit for bit, the
    standalone statistics kernel on the stored logits of the same state (one
    128-column partition for both, whatever the head's tile shape)."""
    sh = shape(vocab=V, **kw)
    k = T // 8
    cd = codec(T, k=k, P=24, W=64)
    toks = wl.markov1_tokens(T, V, 8)
    log("fused head statistics", kw, T, V)
    recs = {}

    def tr(d, chunk, pas, pos, ent, h):
        if d == 0:
            recs[pas] = (pos, ent)

    with dl.Model(sh, max_chunk=T) as m:
        m.set_trace(tr)
        m.encode(toks, cd)
        m.set_trace(None)
        state = np.full(T, sh.mask_id, dtype=np.int64)
        for p in sorted(recs):
            pos, ent = recs[p]
            lg, rows = m.forward_logits(dev_state(state[None, :]))
            H, mx, _, _ = m.entropy_cdf(lg, 24, want_cdf=False)
            H, rows = H.cpu().numpy(), rows.cpu().numpy()
            row_of = {int(r): i for i, r in enumerate(rows)}
            got = np.array([H[row_of[q]] for q in pos], dtype=np.float32)
            assert np.array_equal(got, np.array(ent, dtype=np.float32)), p
            state[pos] = toks[pos]


@pytest.mark.parametrize("kw,cd,n", [
    # 256 x 256 head tiles over the masked rows, 128 x 128 for the few slots
    (dict(d_model=128, n_heads=1, d_ffn=256, vocab=98304), codec(600, k=16, P=24, W=64, batch=2), 1500),
    # 0.5-bit threshold rule (1 to 64 per pass), three chunks per forward
    (dict(ffn="swiglu", norm="rmsnorm"), codec(200, tau=0.5, mmin=1, mmax=64, P=24, W=64, batch=3), 700),
    # symbol ranking reads the logits by slot too
    (dict(vocab=3000), codec(128, k=8, batch=2, coder="rank"), 400),
])
def test_deferred_head_logits_same_containers(kw, cd, n):
    """The LM head may store only the entropy statistics and leave the logits
    of the committed rows to a second, smaller product after the selection.
    Forcing that path on every pass, or forcing the full store, must give
    byte-identical containers and identical traces (positions, entropies,
    coded intervals, CDF hashes), and each container must decode under the
    other mode."""
    sh = shape(**kw)
    toks = wl.markov1_tokens(n, sh.vocab, 21)
    log("deferred head logits", kw, cd)
    out = {}
    with dl.Model(sh, max_chunk=cd.chunk_len, max_batch=cd.batch) as m:
        for mode in (1, 2):
            traces, tr = trace_recorder()
            m.head_logits_mode(mode)
            m.set_trace(tr, coded=True)
            data = m.encode(toks, cd)
            m.head_logits_mode(3 - mode)
            back = m.decode(data)
            m.set_trace(None)
            assert np.array_equal(back, toks)
            assert traces[0] == traces[1]
            out[mode] = (data, traces[0])
        m.head_logits_mode(0)
    assert out[1][0] == out[2][0]
    assert out[1][1] == out[2][1]


@pytest.mark.parametrize("n", [0, 1, 2, 31, 32, 33, 95])
def test_roundtrip_edge_lengths(n):
    """Inputs of 0, 1 and 2 tokens, one less than, exactly and one more than a
    chunk, and a ragged tail after whole chunks (bf16 model, fixed k, batch
    2): each round-trips bit-exactly, the empty input through an empty
    container, and the decoder reports the stored length."""
    sh = shape()
    cd = codec(32, k=5, batch=2)
    toks = wl.markov1_tokens(n, sh.vocab, 9)[:n] if n else np.zeros(0, dtype=np.int64)
    log("edge length", n)
    with dl.Model(sh, max_chunk=32, max_batch=2) as m:
        data = m.encode(toks, cd)
        assert dl.decode_size(data) == n
        back = m.decode(data)
    assert len(back) == n and np.array_equal(back, toks)


def test_roundtrip_degenerate_inputs():
    """A constant stream of the largest token id under fixed k, with every
    masked position committed in the first pass (k above the chunk length),
    and under the 0.5-bit rule; and a stream that alternates the smallest
    and the largest ids.  All round-trip bit-exactly."""
    sh = shape()
    const = np.full(70, sh.vocab - 1, dtype=np.int64)
    alt = np.where(np.arange(70) % 2 == 0, 0, sh.vocab - 1).astype(np.int64)
    log("degenerate inputs")
    with dl.Model(sh, max_chunk=32, max_batch=2) as m:
        for toks in (const, alt):
            for cd in (codec(32, k=4, batch=2), codec(32, k=64, batch=2),
                       codec(32, tau=0.5, mmin=1, mmax=64, batch=2)):
                data = m.encode(toks, cd)
                assert np.array_equal(m.decode(data), toks), cd
