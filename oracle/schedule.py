"""Per-position entropy and the entropy-based commitment schedule.

Entropy (Symbol Commitment Schedules, item 3): for every masked position j,
H_j = -sum_v p_j(v) log p_j(v), here in bits (the log base is not printed; the
threshold of the workloads is stated in bits), with 0 log 0 = 0.

Schedule: commit every masked position with H_j <= tau; if fewer than m_min
qualify, commit the m_min lowest-entropy positions.  Readings where the paper
is silent: entropy ties go to the lower position; at most m_max positions are
committed (the m_max lowest); if fewer than m_min positions are still masked,
all of them are committed; committed positions are coded in ascending position
order.  The fixed-k rule is tau = -inf, m_min = m_max = k.

Left-to-right block schedules (items 1 and 2) commit the next u_k still-masked
positions in ascending order at pass k; they need no entropies.
- Uniform block: u = floor(n / K) per pass over the n masked positions.  Where
  the paper is silent: the remainder n mod K goes to the last block, and
  K > n is read as K = n (one symbol per pass, the autoregressive order).
- Progressive: u_k = round(u_1 r^(k-1)), rounding half up, with r^(k-1) formed
  by repeated multiplication in fp64; every block holds at least one symbol
  and the last one is cut to what remains.  With r = 1 and u_1 = n / K (K
  dividing n) it is the uniform block schedule.
"""
from __future__ import annotations

import math

import numpy as np

from .model import softmax


def entropy_bits(logits: np.ndarray) -> np.ndarray:
    """H = -sum p log2 p per row of ``logits`` [R, V], p = softmax(logits)."""
    p = softmax(np.asarray(logits, dtype=np.float64), axis=-1)
    with np.errstate(divide="ignore", invalid="ignore"):
        plogp = np.where(p > 0.0, p * np.log2(p), 0.0)
    return -plogp.sum(axis=-1)


def commit_count(H: np.ndarray, tau: float, m_min: int, m_max: int) -> int:
    """How many positions the schedule commits from the masked set with entropies H."""
    n_thr = int(np.count_nonzero(np.asarray(H) <= tau))
    return min(len(H), max(m_min, min(m_max, n_thr)))


def select(H: np.ndarray, pos: np.ndarray, tau: float, m_min: int, m_max: int) -> np.ndarray:
    """Committed positions (ascending) among masked positions ``pos`` with entropies ``H``."""
    H = np.asarray(H, dtype=np.float64)
    pos = np.asarray(pos, dtype=np.int64)
    n = commit_count(H, tau, m_min, m_max)
    order = sorted(range(len(pos)), key=lambda i: (H[i], pos[i]))
    return np.sort(pos[order[:n]])


def uniform_blocks(n: int, K: int) -> list:
    """Block sizes u_1..u_K of the uniform block schedule over n positions."""
    if n <= 0:
        return []
    K = max(1, min(K, n))
    u = n // K
    sizes = [u] * K
    sizes[-1] += n - u * K
    return sizes


def progressive_blocks(n: int, u1: int, r: float) -> list:
    """Block sizes of the progressive schedule over n positions."""
    sizes, left, g = [], n, float(u1)
    while left > 0:
        u = max(1, int(math.floor(g + 0.5)))
        u = min(u, left)
        sizes.append(u)
        left -= u
        g = g * float(r)
    return sizes


def block_sizes(codec, n: int) -> list:
    """Per-pass commit counts of a left-to-right block schedule."""
    if codec.schedule == "uniform":
        return uniform_blocks(n, codec.blocks)
    if codec.schedule == "progressive":
        return progressive_blocks(n, codec.u1, codec.growth)
    raise ValueError(codec.schedule)
