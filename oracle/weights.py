"""Random-init weights of the masked diffusion LM, generated on the CPU.

The paper runs a pretrained LLaDA; no weights are available here, so every
tensor is random.  The init is counter based and free of transcendentals so
that an independent implementation in any language produces identical bits:

    c   = splitmix64(seed XOR (tensor_id * 0x9E3779B97F4A7C15 mod 2**64))
    u_i = splitmix64(c + i)                      (i = row-major flat index)
    w_i = ((u_i >> 40) - 2**23) * 2**(-23 - e)   (exact in fp32)

then round-to-nearest-even to bf16 for bf16 models.  splitmix64 is the
published generator of Steele, Lea and Flood (OOPSLA 2014).

Tensor ids: embedding 1, head 2, layer l / kind k -> 16 + 16*l + k with kinds
q=0, k=1, v=2, o=3, ffn_in (GELU W1 or SwiGLU gate)=4, SwiGLU up=5,
ffn_out=6.  All tensors are [out_features, in_features]; the embedding is
[vocab + 1, d] (the last row is the [MASK] id).
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

MASK64 = (1 << 64) - 1
GOLDEN = 0x9E3779B97F4A7C15

EMBED, HEAD = 1, 2
Q, K, V, O, FFN_IN, FFN_UP, FFN_OUT = range(7)


def layer_tensor_id(layer: int, kind: int) -> int:
    return 16 + 16 * layer + kind


def splitmix64_int(x: int) -> int:
    """One splitmix64 output for state ``x`` (Python ints, mod 2**64)."""
    z = (x + GOLDEN) & MASK64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
    return z ^ (z >> 31)


def splitmix64_array(x: np.ndarray) -> np.ndarray:
    """splitmix64 applied elementwise to a uint64 array (wrapping arithmetic)."""
    z = x + np.uint64(GOLDEN)
    z ^= z >> np.uint64(30)
    z *= np.uint64(0xBF58476D1CE4E5B9)
    z ^= z >> np.uint64(27)
    z *= np.uint64(0x94D049BB133111EB)
    z ^= z >> np.uint64(31)
    return z


def tensor_key(seed: int, tensor_id: int) -> int:
    return splitmix64_int((seed ^ ((tensor_id * GOLDEN) & MASK64)) & MASK64)


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to the nearest bf16 (ties to even); returns fp32."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + np.uint64(0x7FFF) + ((u >> np.uint64(16)) & np.uint64(1))) >> np.uint64(16)
    return (u << np.uint64(16)).astype(np.uint32).view(np.float32)


def gen_rows(seed: int, tensor_id: int, n_cols: int, rows: np.ndarray, exp: int,
             dtype: str) -> np.ndarray:
    """Rows ``rows`` of tensor ``tensor_id`` (``n_cols`` columns) as fp64."""
    key = tensor_key(seed, tensor_id)
    rows = np.asarray(rows, dtype=np.uint64)
    idx = rows[:, None] * np.uint64(n_cols) + np.arange(n_cols, dtype=np.uint64)[None, :]
    idx += np.uint64(key)
    u = splitmix64_array(idx)
    q = (u >> np.uint64(40)).astype(np.int64) - (1 << 23)
    w = q.astype(np.float32) * np.float32(2.0 ** (-23 - exp))
    if dtype == "bf16":
        w = round_to_bf16(w)
    return w.astype(np.float64)


def gen_tensor(seed: int, tensor_id: int, shape, exp: int, dtype: str,
               block_rows: int = 512) -> np.ndarray:
    """A whole [out, in] tensor, generated in row blocks (bounded memory) on a
    thread pool; every block is the same pure function of its row indices."""
    n_out, n_in = shape
    out = np.empty((n_out, n_in), dtype=np.float64)

    def fill(r0):
        r1 = min(n_out, r0 + block_rows)
        out[r0:r1] = gen_rows(seed, tensor_id, n_in, np.arange(r0, r1), exp, dtype)

    starts = range(0, n_out, block_rows)
    if n_out * n_in < (1 << 20):
        for r0 in starts:
            fill(r0)
    else:
        with ThreadPoolExecutor(min(16, os.cpu_count() or 1)) as ex:
            list(ex.map(fill, starts))
    return out


class Weights:
    """Lazily generated fp64 weights of a ``workloads.ModelShape``.

    ``layer(l)`` returns the seven (or six) matrices of one layer; embedding
    rows are generated on demand, so a full-width model can be evaluated one
    layer at a time without holding every tensor.
    """

    def __init__(self, shape, cache_layers: bool = True):
        self.s = shape
        self.cache = {} if cache_layers else None
        self._embed_rows = {}
        self._head = None

    def _gen(self, tid, shape, exp):
        return gen_tensor(self.s.seed, tid, shape, exp, self.s.dtype)

    def embed_rows(self, ids: np.ndarray) -> np.ndarray:
        ids = np.asarray(ids, dtype=np.int64)
        uniq = np.unique(ids)
        need = [int(i) for i in uniq if int(i) not in self._embed_rows]
        if need:
            block = gen_rows(self.s.seed, EMBED, self.s.d_model, np.asarray(need),
                             self.s.embed_exp, self.s.dtype)
            for i, r in zip(need, block):
                self._embed_rows[i] = r
        table = np.stack([self._embed_rows[int(i)] for i in uniq])
        pos = np.searchsorted(uniq, ids)
        return table[pos]

    def head(self) -> np.ndarray:
        if self._head is None:
            self._head = self._gen(HEAD, (self.s.vocab, self.s.d_model), self.s.head_exp)
        return self._head

    def head_rows(self, rows: np.ndarray) -> np.ndarray:
        return gen_rows(self.s.seed, HEAD, self.s.d_model, rows, self.s.head_exp, self.s.dtype)

    def layer(self, l: int) -> dict:
        if self.cache is not None and l in self.cache:
            return self.cache[l]
        s = self.s
        d, F = s.d_model, s.d_ffn
        t = lambda k: layer_tensor_id(l, k)
        w = {
            "q": self._gen(t(Q), (d, d), s.attn_exp),
            "k": self._gen(t(K), (d, d), s.attn_exp),
            "v": self._gen(t(V), (d, d), s.attn_exp),
            "o": self._gen(t(O), (d, d), s.attn_exp),
            "ffn_in": self._gen(t(FFN_IN), (F, d), s.ffn_in_exp),
            "ffn_out": self._gen(t(FFN_OUT), (d, F), s.ffn_out_exp),
        }
        if s.ffn == "swiglu":
            w["ffn_up"] = self._gen(t(FFN_UP), (F, d), s.ffn_in_exp)
        if self.cache is not None:
            self.cache[l] = w
        return w


def bf16_bits(w: np.ndarray) -> np.ndarray:
    """The 16-bit patterns of bf16-exact values held in fp64."""
    return (w.astype(np.float32).view(np.uint32) >> np.uint32(16)).astype(np.uint16)
