"""Pins the oracle's Philox4x64-10 to numpy's independent implementation.

numpy.random.Philox is run as a black box (a known-answer source). Its
bit generator advances the 256-bit counter by one before producing each block,
so its first block for counter c is the Philox function at c + 1.
"""
import numpy as np
import pytest

import oracle

M64 = (1 << 64) - 1


def numpy_block(ctr, key):
    """Philox4x64-10 at counter `ctr` via numpy (counter - 1, then one block)."""
    c = list(ctr)
    # subtract one with borrow over the 4 x 64-bit counter
    for i in range(4):
        if c[i] > 0:
            c[i] -= 1
            break
        c[i] = M64  # borrow (the all-zero counter wraps to all ones)
    bg = np.random.Philox(key=np.array(key, dtype=np.uint64),
                          counter=np.array(c, dtype=np.uint64))
    return [int(x) for x in bg.random_raw(4)]


@pytest.mark.parametrize("ctr,key", [
    ([0, 0, 0, 0], [0, 0]),
    ([1, 0, 0, 0], [0, 0]),
    ([123456789, 3, 7, 0], [42, 0]),
    ([M64, 0, 0, 0], [1, 0]),            # counter word 0 all ones
    ([0, 1, 0, 0], [1, 0]),              # carry target of the previous case
    ([999_999_999, 0, 2, 0], [2**63 + 5, 0]),
    ([5, 6, 7, 8], [M64, M64]),
])
def test_block_matches_numpy(ctr, key):
    assert [int(x) for x in oracle.philox4x64_10(ctr, key)] == numpy_block(ctr, key)


def test_random_blocks_match_numpy():
    rng = np.random.default_rng(11)
    for _ in range(200):
        ctr = [int(x) for x in rng.integers(0, 2**63, size=4, dtype=np.int64)]
        ctr[0] += 1  # keep the numpy helper's borrow in word 0
        key = [int(x) for x in rng.integers(0, 2**63, size=2, dtype=np.int64)]
        assert [int(x) for x in oracle.philox4x64_10(ctr, key)] == numpy_block(ctr, key)


def test_draw_word_order():
    """u32 word j of (p, e): block j // 8 of counter (p, e, block, 0), key
    (seed, 0); output o_m gives words 2m (low half) and 2m + 1 (high half)."""
    seed, p, e = 77, 1234567, 3
    for block in range(3):
        raw = numpy_block([p, e, block, 0], [seed, 0])
        for j in range(8):
            v = raw[j // 2]
            want = (v & 0xFFFFFFFF) if j % 2 == 0 else (v >> 32)
            assert oracle.draw_u32(seed, p, e, 8 * block + j) == want


def test_draws_are_uniform():
    """Coarse uniformity of keep/window words over many positions."""
    vals = np.array([oracle.draw_u32(5, p, 0, 0) for p in range(20000)],
                    dtype=np.float64) / 2**32
    hist, _ = np.histogram(vals, bins=10, range=(0, 1))
    expected = len(vals) / 10
    chi2 = ((hist - expected) ** 2 / expected).sum()
    assert chi2 < 33.7  # chi-square, 9 dof, p = 1e-4
