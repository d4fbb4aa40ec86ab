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
"""
from __future__ import annotations

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
