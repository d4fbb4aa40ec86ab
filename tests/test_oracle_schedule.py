"""Pins of the oracle's entropy and entropy-based schedule, including brute
force over subsets and over every single-position coding order on 8-token
chunks."""
import itertools
import math

import numpy as np
import pytest
import scipy.stats

import workloads as wl
from oracle import cdf as OC
from oracle import coder as ORC
from oracle import model as OM
from oracle import schedule as OS
from oracle import weights as OW


def test_entropy_closed_forms():
    V = 1000
    assert OS.entropy_bits(np.zeros((1, V)))[0] == pytest.approx(math.log2(V), abs=1e-12)
    two = np.full((1, V), -np.inf)
    two[0, [3, 700]] = 5.0
    assert OS.entropy_bits(two)[0] == pytest.approx(1.0, abs=1e-12)
    one = np.full((1, V), -np.inf)
    one[0, 9] = 0.0
    assert OS.entropy_bits(one)[0] == 0.0


def test_entropy_matches_scipy_and_identity():
    rng = np.random.default_rng(0)
    lg = rng.standard_normal((20, 3000)) * rng.uniform(0.1, 12, (20, 1))
    H = OS.entropy_bits(lg)
    p = OM.softmax(lg)
    assert np.allclose(H, scipy.stats.entropy(p, base=2, axis=1), atol=1e-10)
    # H = log2 Z - sum e (l - m) / (Z ln 2) with e = exp(l - m)
    m = lg.max(1, keepdims=True)
    e = np.exp(lg - m)
    Z = e.sum(1)
    ident = np.log2(Z) - (e * (lg - m)).sum(1) / (Z * math.log(2))
    assert np.allclose(H, ident, atol=1e-12)


def test_commit_count_rule():
    H = np.array([0.1, 0.9, 0.4, 2.0, 0.5])
    assert OS.commit_count(H, 0.5, 1, 64) == 3          # H <= tau, inclusive
    assert OS.commit_count(H, 0.05, 2, 64) == 2         # fewer than m_min qualify
    assert OS.commit_count(H, 10.0, 1, 4) == 4          # capped by m_max
    assert OS.commit_count(H[:2], -np.inf, 4, 4) == 2   # fewer masked than k
    assert OS.commit_count(H, -np.inf, 3, 3) == 3       # fixed k


def tiny8():
    w = wl.WORKLOADS["tiny"]
    return w.model, OW.Weights(w.model)


def lex_key(H, pos, subset):
    return sorted((H[i], pos[i]) for i in subset)


@pytest.mark.parametrize("seed", [0, 1])
def test_selection_is_lexicographic_minimum_bruteforce(seed):
    shape, W = tiny8()
    toks = wl.markov2_bytes(8, 100 + seed)
    state = np.full(8, shape.mask_id)
    rng = np.random.default_rng(seed)
    while np.any(state == shape.mask_id):
        lg, pos = OM.logits(shape, W, state)
        H = OS.entropy_bits(lg)
        # ties at the all-mask pass: add nothing, the rule must break them by position
        for k in range(1, 5):
            sel = OS.select(H, pos, -np.inf, k, k)
            n = min(k, len(pos))
            best = min(itertools.combinations(range(len(pos)), n), key=lambda s: lex_key(H, pos, s))
            assert list(sel) == sorted(pos[list(best)])
        for tau in (-1.0, float(np.median(H)), 100.0):
            for mmin, mmax in ((1, 8), (2, 3), (3, 3)):
                sel = OS.select(H, pos, tau, mmin, mmax)
                n = OS.commit_count(H, tau, mmin, mmax)
                best = min(itertools.combinations(range(len(pos)), n), key=lambda s: lex_key(H, pos, s))
                assert list(sel) == sorted(pos[list(best)])
                if n > mmin:                  # every committed position qualifies
                    assert np.all(H[np.isin(pos, sel)] <= tau)
        k = int(rng.integers(1, 4))
        sel = OS.select(H, pos, -np.inf, k, k)
        state[sel] = toks[sel]


def test_every_single_position_order_roundtrips_bruteforce():
    """All 8! one-position-per-pass orders of an 8-token chunk: each order's
    code length from the table of per-(state, position) CDFs equals what the
    range coder produces, and every order decodes back exactly.  The greedy
    lowest-entropy order (k = 1) is one of them."""
    shape, W = tiny8()
    T, P, Wb = 8, 16, 32
    toks = wl.markov2_bytes(T, 7)
    # one forward per revealed subset (2**8 states)
    table = {}
    for mask in range(1 << T):
        state = np.array([toks[i] if (mask >> i) & 1 else shape.mask_id for i in range(T)])
        if mask == (1 << T) - 1:
            continue
        lg, pos = OM.logits(shape, W, state)
        table[mask] = ({int(p): OC.cdf_row(lg[i], P) for i, p in enumerate(pos)},
                       OS.entropy_bits(lg), pos)
    # greedy order under the k=1 schedule
    greedy, mask = [], 0
    while mask != (1 << T) - 1:
        cdfs, H, pos = table[mask]
        p = int(OS.select(H, pos, -np.inf, 1, 1)[0])
        greedy.append(p)
        mask |= 1 << p
    seen_greedy = False
    for order in itertools.permutations(range(T)):
        enc = ORC.RangeEncoder(Wb, P)
        bits, mask = 0.0, 0
        for p in order:
            cdf = table[mask][0][p]
            s = int(toks[p])
            f = int(cdf[s + 1] - cdf[s])
            bits += -math.log2(f / 2.0 ** P)
            enc.encode(int(cdf[s]), f)
            mask |= 1 << p
        assert enc.code_length_bits() - bits < T * math.log2(1 + 2.0 ** -8) + 1e-9
        payload = enc.finish()
        dec = ORC.RangeDecoder(payload, Wb, P)
        mask = 0
        for p in order:
            assert dec.decode(table[mask][0][p]) == toks[p]
            mask |= 1 << p
        if list(order) == greedy:
            seen_greedy = True
    assert seen_greedy


# ---------------------------------------------------------------- block schedules
from oracle.schedule import progressive_blocks, uniform_blocks  # noqa: E402


@pytest.mark.parametrize("n,K", [(10, 3), (2048, 16), (2048, 2048), (7, 1), (5, 9), (1, 1), (100, 7)])
def test_uniform_blocks_cover_left_to_right(n, K):
    sizes = uniform_blocks(n, K)
    Ke = min(K, n)
    assert sum(sizes) == n and len(sizes) == Ke
    # floor(n / K) per pass, the remainder n mod K on the last block
    assert all(u == n // Ke for u in sizes[:-1]) and sizes[-1] == n // Ke + n % Ke


def test_uniform_blocks_special_cases():
    assert uniform_blocks(0, 4) == []
    assert uniform_blocks(9, 1) == [9]           # one-shot
    assert uniform_blocks(6, 6) == [1] * 6       # autoregressive: one symbol per pass
    assert uniform_blocks(3, 50) == [1, 1, 1]    # K > n read as K = n


def test_progressive_blocks_hand_example():
    # u1 = 2, r = 1.5: 2, 3 (2 * 1.5), round(4.5) = 5 (half up), round(6.75) = 7,
    # then 10.125 is cut to the 3 positions left (20 = 2 + 3 + 5 + 7 + 3)
    assert progressive_blocks(20, 2, 1.5) == [2, 3, 5, 7, 3]
    # shrinking budgets never commit fewer than one symbol: 4, 2, 1, round(0.5) = 1, ...
    assert progressive_blocks(10, 4, 0.5) == [4, 2, 1, 1, 1, 1]


@pytest.mark.parametrize("n,K", [(12, 4), (2048, 16), (64, 64), (30, 1)])
def test_progressive_with_unit_growth_is_uniform(n, K):
    # Schedules, item 2: r = 1 reduces to the uniform block schedule
    assert progressive_blocks(n, n // K, 1.0) == uniform_blocks(n, K)
