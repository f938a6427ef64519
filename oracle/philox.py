"""Philox4x64-10 counter-based generator and the draws derived from it.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).

The paper does not say which random generator its sampler uses (App. B,
"BufferStructure.sample" calls a library sampler).  For a sampler whose draws
must be identical on the CPU and on the GPU we fix a counter-based generator:
Philox4x64 with 10 rounds, as defined in J. K. Salmon, M. A. Moraes,
R. O. Dror, D. E. Shaw, "Parallel random numbers: as easy as 1, 2, 3", SC'11.
Written here from that definition in exact Python integer arithmetic.

Pinned by: the published known-answer vector for counter = key = 0, and by
numpy's independent implementation (``numpy.random.Philox`` is Philox4x64-10)
on random keys and counters (tests/test_oracle_philox.py).

Derived draws (defined here; the paper fixes none of it):

* draw ``j`` of sampling step ``step`` under ``seed`` reads the block
  ``philox(counter=(j, step, 0, 0), key=(seed, 0))`` -> four 64-bit words
  ``x0..x3``;
* an index uniform over ``[0, n)`` is ``floor(x0 * n / 2**64)`` (the high word
  of the 128-bit product; bias at most ``n / 2**64``);
* the stratum coin with threshold ``p_q32`` (``floor(p * 2**32)``, in
  ``[0, 2**32]``) is ``(x1 >> 32) < p_q32``.
"""

MASK64 = (1 << 64) - 1

# Multipliers and Weyl key increments of Philox4x64 (Salmon et al., SC'11).
PHILOX_M0 = 0xD2E7470EE14C6C93
PHILOX_M1 = 0xCA5A826395121157
PHILOX_W0 = 0x9E3779B97F4A7C15  # golden ratio
PHILOX_W1 = 0xBB67AE8584CAA73B  # sqrt(3) - 1

ROUNDS = 10


def mulhilo64(a, b):
    """Return (high, low) 64-bit words of the exact 128-bit product a*b."""
    p = (a & MASK64) * (b & MASK64)
    return p >> 64, p & MASK64


def philox4x64(counter, key, rounds=ROUNDS):
    """One Philox4x64 block: 4 x u64 counter, 2 x u64 key -> 4 x u64 output.

    Each round multiplies words 0 and 2 by the two round constants; the high
    halves are XOR-ed with the other two words and the round key, and the words
    are permuted.  The key advances by the Weyl increments between rounds.
    """
    x0, x1, x2, x3 = (int(c) & MASK64 for c in counter)
    k0, k1 = (int(k) & MASK64 for k in key)
    for r in range(rounds):
        if r > 0:
            k0 = (k0 + PHILOX_W0) & MASK64
            k1 = (k1 + PHILOX_W1) & MASK64
        hi0, lo0 = mulhilo64(PHILOX_M0, x0)
        hi1, lo1 = mulhilo64(PHILOX_M1, x2)
        x0, x1, x2, x3 = hi1 ^ x1 ^ k0, lo1, hi0 ^ x3 ^ k1, lo0
    return x0, x1, x2, x3


def draw_block(seed, step, j):
    """The four words read by draw ``j`` of sampling step ``step``."""
    return philox4x64((j, step, 0, 0), (seed, 0))


def uniform_index(x, n):
    """floor(x * n / 2**64): a 64-bit word mapped onto [0, n)."""
    if n <= 0:
        raise ValueError("uniform_index needs n >= 1")
    return ((int(x) & MASK64) * int(n)) >> 64


def coin(x, p_q32):
    """True with probability p_q32 / 2**32, from the high 32 bits of x."""
    return ((int(x) & MASK64) >> 32) < int(p_q32)


def p_to_q32(p):
    """Host-side threshold for a stratum probability p in [0, 1]."""
    if not (0.0 <= p <= 1.0):
        raise ValueError("probability outside [0, 1]")
    return min(int(p * 4294967296.0), 1 << 32)
