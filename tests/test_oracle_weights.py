"""Pins of the oracle's counter-based weight init."""
import numpy as np
import pytest
import torch

from oracle import weights as OW


def test_splitmix64_published_sequence():
    # splitmix64 seeded with 0 (state advances by the golden gamma before each
    # output): the first outputs of the reference generator of Steele, Lea and
    # Flood / Vigna's splitmix64.c.
    golden = read_golden("splitmix64_seed0.txt")
    got = [OW.splitmix64_int((i * OW.GOLDEN) & OW.MASK64) for i in range(len(golden))]
    assert got == golden


def read_golden(name):
    import os
    path = os.path.join(os.path.dirname(__file__), "golden", name)
    vals = []
    for line in open(path):
        line = line.strip()
        if line and not line.startswith("#"):
            vals.append(int(line, 16))
    return vals


def test_array_matches_scalar():
    x = np.arange(1000, dtype=np.uint64) * np.uint64(0x1234567) + np.uint64(99)
    a = OW.splitmix64_array(x.copy())
    b = [OW.splitmix64_int(int(v)) for v in x]
    assert [int(v) for v in a] == b


@pytest.mark.parametrize("exp", [0, 3, 6])
def test_values_are_exact_uniform_grid(exp):
    w = OW.gen_rows(7, 33, 512, np.arange(64), exp, "f32")
    scaled = w * 2.0 ** (23 + exp)
    assert np.all(scaled == np.round(scaled))                  # 24-bit integers
    assert w.min() >= -(2.0 ** -exp) and w.max() < 2.0 ** -exp
    assert abs(w.mean()) < 0.02 * 2.0 ** -exp                   # centred
    assert abs(w.std() - 2.0 ** -exp / np.sqrt(3.0)) < 0.02 * 2.0 ** -exp


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    x = (rng.standard_normal(100000) * 10.0 ** rng.uniform(-6, 6, 100000)).astype(np.float32)
    ours = OW.round_to_bf16(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(ours.view(np.uint32), ref.view(np.uint32))


def test_row_subsets_are_consistent():
    full = OW.gen_tensor(3, 17, (300, 40), 2, "bf16", block_rows=64)
    rows = np.array([0, 5, 299, 64, 63])
    assert np.array_equal(OW.gen_rows(3, 17, 40, rows, 2, "bf16"), full[rows])


def test_distinct_tensors_and_seeds_differ():
    a = OW.gen_rows(0, 16, 64, np.arange(4), 0, "f32")
    b = OW.gen_rows(0, 17, 64, np.arange(4), 0, "f32")
    c = OW.gen_rows(1, 16, 64, np.arange(4), 0, "f32")
    assert not np.array_equal(a, b) and not np.array_equal(a, c)
