"""Attention-based initial context (Initial Context Strategies, item 4).

Two extra forward passes over the chunk -- one with the even positions masked,
one with the odd positions masked -- score every position by the attention it
receives from the masked positions, aggregated over layers with Attention
Rollout (Abnar and Zuidema, 2020): per layer the head-averaged attention A_l
mixed with the residual path, A~_l = (A_l + I) / 2, and the rollout
R = A~_L ... A~_1, whose entry (i, j) is the flow from input position j to
output position i.  The score of a position visible in a pass is the flow it
sends to that pass's masked positions, (1_M^T R)_j; each position is scored
in the pass where it is visible.  The c highest scores are the context (where
the paper is silent: ties by position, the lower first).

1_M^T R is evaluated right to left as a chain of vector-matrix products,
v <- A~_l^T v from the last layer down to the first, which is the same
product reassociated (a test compares it with the explicit matrix product).
"""
from __future__ import annotations

import numpy as np

from . import model as M


def attention_maps(shape, W, state: np.ndarray) -> list:
    """Head-averaged attention probabilities [T, T] of every layer."""
    state = np.asarray(state, dtype=np.int64)
    T = state.shape[0]
    x = W.embed_rows(state)
    cos, sin = M.rope_cos_sin(T, shape.d_head, shape.rope_theta)
    maps = []
    for l in range(shape.n_layers):
        x = M.block(shape, W.layer(l), x, cos, sin, probs_out=maps)
    return maps


def rollout_flow(maps: list, masked: np.ndarray) -> np.ndarray:
    """1_M^T R for the indicator 1_M of the masked positions."""
    v = np.asarray(masked, dtype=np.float64).copy()
    for A in reversed(maps):
        v = 0.5 * (A.T @ v) + 0.5 * v
    return v


def context_scores(shape, W, tokens: np.ndarray) -> np.ndarray:
    """Score of every position of a chunk (even positions from the pass with
    the odd positions masked, odd positions from the other pass)."""
    tokens = np.asarray(tokens, dtype=np.int64)
    T = tokens.shape[0]
    idx = np.arange(T)
    score = np.zeros(T, dtype=np.float64)
    for masked_parity in (0, 1):
        masked = (idx % 2) == masked_parity
        state = np.where(masked, shape.mask_id, tokens)
        flow = rollout_flow(attention_maps(shape, W, state), masked)
        score[~masked] = flow[~masked]
    return score


def attention_context(shape, W, tokens: np.ndarray, c: int) -> np.ndarray:
    """The c highest-scoring positions (ties by position), ascending."""
    score = context_scores(shape, W, tokens)
    c = min(int(c), len(score))
    order = sorted(range(len(score)), key=lambda j: (-score[j], j))
    return np.sort(np.asarray(order[:c], dtype=np.int64))
