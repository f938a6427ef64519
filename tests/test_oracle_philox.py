"""Pins of the oracle's counter-based generator and the draws derived from it."""

import os
import random
from fractions import Fraction

import numpy as np
import pytest

from oracle import philox


def _kat_rows(golden_dir):
    rows = []
    with open(os.path.join(golden_dir, "philox4x64_10_kat.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            w = [int(x, 16) for x in line.split()]
            rows.append((tuple(w[0:4]), tuple(w[4:6]), tuple(w[6:10])))
    return rows


def test_published_known_answer_vectors(golden_dir):
    rows = _kat_rows(golden_dir)
    assert len(rows) == 3
    for ctr, key, expect in rows:
        assert philox.philox4x64(ctr, key) == expect


def _numpy_block(ctr, key):
    """Philox4x64-10 block from numpy's independent implementation.

    numpy increments its 256-bit counter before generating a block, so the
    state is set one below the wanted counter."""
    c = list(ctr)
    for i in range(4):
        c[i] = (c[i] - 1) % (1 << 64)
        if c[i] != (1 << 64) - 1:
            break
    bg = np.random.Philox(key=np.array(key, dtype=np.uint64))
    st = bg.state
    st["state"]["counter"] = np.array(c, dtype=np.uint64)
    st["buffer_pos"] = 4
    bg.state = st
    return tuple(int(x) for x in bg.random_raw(4))


def test_matches_numpy_philox_on_random_blocks():
    rng = random.Random(2604)
    for _ in range(300):
        ctr = tuple(rng.getrandbits(64) for _ in range(4))
        key = tuple(rng.getrandbits(64) for _ in range(2))
        assert philox.philox4x64(ctr, key) == _numpy_block(ctr, key)


def test_draw_block_counter_layout():
    # draw j of step s under seed k reads counter (j, s, 0, 0), key (k, 0)
    assert philox.draw_block(7, 3, 5) == _numpy_block((5, 3, 0, 0), (7, 0))


@pytest.mark.parametrize("n", [1, 2, 3, 7, 64, 1000, 1 << 20, (1 << 31) - 1])
def test_uniform_index_is_floor_of_scaled_word(n):
    rng = random.Random(n)
    xs = [0, 1, (1 << 64) - 1, 1 << 63] + [rng.getrandbits(64) for _ in range(200)]
    for x in xs:
        exact = Fraction(x * n, 1 << 64)
        got = philox.uniform_index(x, n)
        assert got == int(exact)  # floor for nonnegative values
        assert 0 <= got < n


def test_uniform_index_preimage_sizes_differ_by_at_most_one():
    # every bucket of [0, n) receives floor or ceil of 2^64/n words
    for n in [3, 5, 6, 1000, 151936]:
        lo = (1 << 64) // n
        for i in [0, 1, n // 2, n - 1]:
            first = -(-(i << 64) // n)      # smallest x with floor(x n/2^64) >= i
            nxt = -(-((i + 1) << 64) // n)
            assert nxt - first in (lo, lo + 1)
            assert philox.uniform_index(first, n) == i
            if first > 0:
                assert philox.uniform_index(first - 1, n) == i - 1


def test_coin_threshold():
    assert not philox.coin((1 << 64) - 1, 0)
    assert not philox.coin(0, 0)
    assert philox.coin((1 << 64) - 1, 1 << 32)
    assert philox.coin(5 << 32, 6)
    assert not philox.coin(6 << 32, 6)
    assert philox.p_to_q32(0.0) == 0
    assert philox.p_to_q32(1.0) == 1 << 32
    assert philox.p_to_q32(0.5) == 1 << 31
