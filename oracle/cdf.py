"""Quantisation of a predicted distribution into an integer CDF.

The paper entropy-codes each committed symbol with the distribution the DLM
predicts for it (Implementation Details: statistical coding with rANS).  It
gives no quantisation rule, so this one is a reading, chosen so that
everything after the exponential is exact integer arithmetic:

    e_v = exp(l_v - max_u l_u)                 in (0, 1]
    g_v = floor(e_v * 2**24)                   (the argmax gets exactly 2**24)
    G   = sum_v g_v
    f_v = 1 + floor(g_v * (2**P - V) / G)      every symbol keeps f_v >= 1
    R   = 2**P - sum_v f_v                     in [0, V)
    f_a += R   with a the lowest index of maximal g
    cdf[0] = 0, cdf[v+1] = cdf[v] + f_v        so cdf[V] = 2**P

The oracle takes the exponential in fp64.  ``integer_cdf`` is the integer
stage alone; given the same g it is bit-identical on any implementation.
"""
from __future__ import annotations

import numpy as np

G_ONE = 1 << 24


def quantise_g(logits_row: np.ndarray) -> np.ndarray:
    l = np.asarray(logits_row, dtype=np.float64)
    e = np.exp(l - l.max())
    return np.floor(e * float(G_ONE)).astype(np.int64)


def integer_cdf(g: np.ndarray, P: int) -> np.ndarray:
    g = np.asarray(g, dtype=np.int64)
    V = g.shape[0]
    if V >= (1 << P):
        raise ValueError("alphabet does not fit the CDF precision")
    G = int(g.sum())
    f = 1 + (g * ((1 << P) - V)) // G
    R = (1 << P) - int(f.sum())
    a = int(np.argmax(g))          # first index of the maximum
    f[a] += R
    cdf = np.zeros(V + 1, dtype=np.int64)
    np.cumsum(f, out=cdf[1:])
    return cdf


def cdf_row(logits_row: np.ndarray, P: int) -> np.ndarray:
    return integer_cdf(quantise_g(logits_row), P)
