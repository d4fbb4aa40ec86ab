"""Seeded synthetic workloads shared by the HIP path's tests/bench and the oracle.

This module holds *inputs only*: model shapes, codec parameters and seeded token
sources.  It contains none of the compression method's arithmetic (no forward
pass, no entropy, no CDF, no coder), so both the product binding and the CPU
oracle may import it without sharing any of the method's code.

The paper evaluates on the first 1 MB / 10 MB of enwik8 tokenised by the LLaDA
tokenizer (Experimental Methodology).  Neither is available here, so the
sources below are seeded Markov/Zipf stand-ins with the shapes of those
workloads: byte streams for the tiny model, and token-id streams over a 32768
or 126464-symbol vocabulary for the larger models.

Randomness is counter based: ``u64(seed, k) = splitmix64(splitmix64(seed) + k)``
(splitmix64 as published by Steele, Lea and Flood, "Fast splittable
pseudorandom number generators", OOPSLA 2014), uniforms are
``(u64 >> 11) * 2**-53``.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, Optional

import numpy as np

MASK64 = (1 << 64) - 1
GOLDEN = 0x9E3779B97F4A7C15


# --------------------------------------------------------------------------
# model / codec descriptions
# --------------------------------------------------------------------------
@dataclasses.dataclass(frozen=True)
class ModelShape:
    """A masked-diffusion transformer shape (Definition 3 of the paper).

    ``vocab`` is |Sigma|; the input-only [MASK] id equals ``vocab`` so the
    embedding table has ``vocab + 1`` rows and the head has ``vocab`` rows.
    ``*_exp`` are the random-init scale exponents: a tensor's entries are
    uniform on [-2**-exp, 2**-exp).
    """
    name: str
    n_layers: int
    d_model: int
    n_heads: int
    d_ffn: int
    vocab: int
    ffn: str            # "gelu" | "swiglu"
    norm: str           # "layernorm" | "rmsnorm"
    dtype: str          # "f32" | "bf16"
    rope_theta: float = 10000.0
    norm_eps: float = 1e-5
    embed_exp: int = 0
    attn_exp: int = 0
    ffn_in_exp: int = 0
    ffn_out_exp: int = 0
    head_exp: int = 0
    seed: int = 0

    @property
    def d_head(self) -> int:
        return self.d_model // self.n_heads

    @property
    def mask_id(self) -> int:
        return self.vocab


@dataclasses.dataclass(frozen=True)
class CodecParams:
    """Commitment-schedule and coder parameters stored in the container header.

    schedule (Symbol Commitment Schedules):
      "entropy"     item 3: commit every masked position with H <= tau_bits; if
                    fewer than m_min qualify commit the m_min lowest-entropy
                    ones; m_max caps the count.  tau_bits = -inf gives the
                    fixed-k rule (m_min = m_max = k).
      "uniform"     item 1: ``blocks`` = K left-to-right blocks per chunk.
      "progressive" item 2: left-to-right blocks of round(u1 * growth^(k-1)).
    coder: "range" (W = coder_bits), "rans" (64-bit state, 32-bit words) or
    "rank" (symbol ranking: varint ranks, the container's payloads compressed
    with rank_compressor at rank_level).
    context / context_kind (Initial Context Strategies): c symbols per chunk
    left visible and stored in the container, the first c ("contiguous"), c
    seeded-random positions ("random", seed context_seed + chunk index), or
    the c positions with the highest attention-rollout scores ("attention").
    """
    chunk_len: int
    tau_bits: float
    m_min: int
    m_max: int
    cdf_bits: int
    coder_bits: int
    batch: int = 1
    schedule: str = "entropy"
    blocks: int = 0
    u1: int = 0
    growth: float = 1.0
    coder: str = "range"
    context: int = 0
    context_kind: str = "contiguous"
    context_seed: int = 0
    rank_compressor: str = "none"
    rank_level: int = 0


def fan_in_exp(fan_in: int) -> int:
    """Exponent e with 2**-e closest (in log scale) to sqrt(3/fan_in)."""
    return int(round(0.5 * math.log2(fan_in / 3.0)))


def _shape(name, L, d, H, F, V, ffn, norm, dtype, head_exp=None, attn_exp=None, seed=0):
    return ModelShape(
        name=name, n_layers=L, d_model=d, n_heads=H, d_ffn=F, vocab=V, ffn=ffn,
        norm=norm, dtype=dtype, embed_exp=0,
        attn_exp=fan_in_exp(d) if attn_exp is None else attn_exp,
        ffn_in_exp=fan_in_exp(d), ffn_out_exp=fan_in_exp(F),
        head_exp=fan_in_exp(d) if head_exp is None else head_exp, seed=seed)


TINY = _shape("tiny-f32", 2, 128, 4, 512, 256, "gelu", "layernorm", "f32")
SMALL = _shape("small-bf16", 12, 768, 12, 3072, 32768, "gelu", "layernorm", "bf16")
# The 8B-shaped model.  Its head uses 2**-2 (logit std ~9) and its attention
# projections twice the fan-in scale: with fan-in attention a random-init
# model attends almost uniformly, every masked position gets nearly the same
# prediction and the 0.5-bit threshold schedule never fires; sharper attention
# makes predictions position specific, with roughly a fifth of the positions
# under 0.5 bits, as a trained model would have some confident positions.
DLM8B = _shape("8b-bf16", 32, 4096, 32, 12288, 126464, "swiglu", "rmsnorm", "bf16",
               head_exp=2, attn_exp=fan_in_exp(4096) - 1)


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    model: ModelShape
    codec: CodecParams
    source: str
    n_tokens: int
    token_bytes: int       # little-endian width of one input symbol
    data_seed: int


NEG_INF = float("-inf")

WORKLOADS: Dict[str, Workload] = {
    "tiny": Workload("tiny", TINY, CodecParams(256, NEG_INF, 4, 4, 16, 32, batch=16),
                     "markov2_bytes", 4096, 1, 1),
    "small": Workload("small", SMALL, CodecParams(1024, NEG_INF, 8, 8, 24, 64, batch=64),
                      "markov1_tokens", 524288, 2, 2),
    "8b": Workload("8b", DLM8B, CodecParams(2048, NEG_INF, 16, 16, 24, 64, batch=1),
                   "markov1_tokens", 2097152, 4, 3),
    "8b-throughput": Workload("8b-throughput", DLM8B,
                              CodecParams(2048, 0.5, 1, 64, 24, 64, batch=32),
                              "markov1_tokens", 16777216, 4, 4),
    "8b-long": Workload("8b-long", DLM8B, CodecParams(8192, NEG_INF, 64, 64, 24, 64, batch=4),
                        "mixed_spans", 262144, 4, 5),
}


def with_layers(shape: ModelShape, n_layers: int, **kw) -> ModelShape:
    """Same shape with another depth (the launch shapes of every kernel are kept)."""
    return dataclasses.replace(shape, n_layers=n_layers, name=f"{shape.name}-L{n_layers}", **kw)


# --------------------------------------------------------------------------
# counter-based randomness
# --------------------------------------------------------------------------
def _mix_inplace(z: np.ndarray) -> np.ndarray:
    z ^= z >> np.uint64(30)
    z *= np.uint64(0xBF58476D1CE4E5B9)
    z ^= z >> np.uint64(27)
    z *= np.uint64(0x94D049BB133111EB)
    z ^= z >> np.uint64(31)
    return z


def _splitmix_scalar(x: int) -> int:
    z = (x + GOLDEN) & MASK64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
    return z ^ (z >> 31)


def u64_stream(seed: int, start: int, n: int) -> np.ndarray:
    base = _splitmix_scalar(seed & MASK64)
    k = np.arange(start, start + n, dtype=np.uint64)
    k += np.uint64(base)
    k += np.uint64(GOLDEN)
    return _mix_inplace(k)


def uniform_stream(seed: int, start: int, n: int) -> np.ndarray:
    return (u64_stream(seed, start, n) >> np.uint64(11)).astype(np.float64) * (2.0 ** -53)


def seeded_permutation(seed: int, n: int) -> np.ndarray:
    keys = u64_stream(seed, 0, n)
    return np.argsort(keys, kind="stable").astype(np.int64)


def zipf_table(n: int, s: float) -> np.ndarray:
    w = np.arange(1, n + 1, dtype=np.float64) ** (-s)
    c = np.cumsum(w)
    return c / c[-1]


def zipf_ranks(u: np.ndarray, table: np.ndarray) -> np.ndarray:
    """0-based Zipf ranks by inverse CDF."""
    r = np.searchsorted(table, u, side="right")
    return np.minimum(r, len(table) - 1).astype(np.int64)


# --------------------------------------------------------------------------
# sources
# --------------------------------------------------------------------------
def markov2_bytes(n: int, seed: int, s: float = 1.1) -> np.ndarray:
    """Order-2 byte Markov chain: context (a, b) picks a Zipf(s) rank over its
    own seeded permutation of 0..255."""
    tab = zipf_table(256, s)
    ranks = zipf_ranks(uniform_stream(seed, 0, n), tab).tolist()
    perms: Dict[int, list] = {}
    out = [0] * n
    a = b = 0
    for t in range(n):
        ctx = (a << 8) | b
        p = perms.get(ctx)
        if p is None:
            p = seeded_permutation((seed * 0x10001 + ctx + 1) & MASK64, 256).tolist()
            perms[ctx] = p
        x = p[ranks[t]]
        out[t] = x
        a, b = b, x
    return np.asarray(out, dtype=np.int64)


def markov1_tokens(n: int, vocab: int, seed: int, s: float = 1.05) -> np.ndarray:
    """Order-1 token chain x' = pi[(rho + h(x)) mod V] with rho ~ Zipf(s):
    every row is a rotated Zipf distribution, with no V x V table."""
    tab = zipf_table(vocab, s)
    pi = seeded_permutation(seed ^ 0x5EED, vocab).tolist()
    h = (u64_stream(seed ^ 0xA5A5, 0, vocab) % np.uint64(vocab)).astype(np.int64).tolist()
    rho = zipf_ranks(uniform_stream(seed, 0, n), tab).tolist()
    out = [0] * n
    x = pi[0]
    for t in range(n):
        x = pi[(rho[t] + h[x]) % vocab]
        out[t] = x
    return np.asarray(out, dtype=np.int64)


def mixed_spans(n: int, vocab: int, seed_a: int, seed_b: int, span: int = 512,
                s: float = 1.05) -> np.ndarray:
    """Alternating spans: A = a period-64 Zipf motif with 1/64 Zipf substitutions
    (low entropy), B = uniform over the 4096 most Zipf-probable ids (high entropy)."""
    tab = zipf_table(vocab, s)
    pi = seeded_permutation(seed_a ^ 0x5EED, vocab)
    motif = pi[zipf_ranks(uniform_stream(seed_a ^ 0x3117, 0, 64), tab)]
    ua = uniform_stream(seed_a, 0, 2 * n)
    sub = ua[:n] < (1.0 / 64.0)
    subs = pi[zipf_ranks(ua[n:], tab)]
    ub = u64_stream(seed_b, 0, n)
    uni = pi[(ub % np.uint64(4096)).astype(np.int64)]
    t = np.arange(n)
    in_a = ((t // span) % 2) == 0
    a_tok = np.where(sub, subs, motif[t % 64])
    return np.where(in_a, a_tok, uni).astype(np.int64)


def make_tokens(w: Workload, n: Optional[int] = None) -> np.ndarray:
    """The first ``n`` tokens (default: all) of a workload's seeded stream."""
    n = w.n_tokens if n is None else int(n)
    V = w.model.vocab
    if w.source == "markov2_bytes":
        return markov2_bytes(n, w.data_seed)
    if w.source == "markov1_tokens":
        return markov1_tokens(n, V, w.data_seed)
    if w.source == "mixed_spans":
        return mixed_spans(n, V, w.data_seed, w.data_seed + 1)
    raise ValueError(w.source)


def random_state(rng_seed: int, B: int, T: int, vocab: int, mask_frac: float) -> np.ndarray:
    """A partially masked state [B, T] (tokens in [0, V), MASK = V) for forward tests."""
    u = uniform_stream(rng_seed, 0, 2 * B * T)
    tok = (u64_stream(rng_seed ^ 0x77, 0, B * T) % np.uint64(vocab)).astype(np.int64)
    st = np.where(u[: B * T] < mask_frac, vocab, tok)
    return st.reshape(B, T).astype(np.int64)


def random_logits(rng_seed: int, rows: int, vocab: int, scale: float) -> np.ndarray:
    """Gaussian-like fp32 logits (sum of 4 uniforms) for entropy/CDF kernel tests."""
    u = uniform_stream(rng_seed, 0, 4 * rows * vocab).reshape(4, rows, vocab)
    g = (u.sum(axis=0) - 2.0) * math.sqrt(3.0)
    return (g * scale).astype(np.float32)
