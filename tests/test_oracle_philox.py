"""Pins for the oracle's Philox4x64-10 and fire mask.

The generator is pinned to numpy's independent Philox4x64-10 bit generator:
``numpy.random.Philox(counter=c, key=k).random_raw(4)`` returns the block for
counter c + 1 (numpy increments before generating), so the oracle's block at
counter c equals numpy's first block when numpy is seeded with c - 1 (a
256-bit decrement with borrow).
"""
import numpy as np
import pytest

from oracle import philox4x64, mulhilo64, fire_bits, fire_mask, fire_threshold, linear_index

MASK64 = (1 << 64) - 1


def numpy_block(counter, key):
    c = sum(int(v) << (64 * i) for i, v in enumerate(counter))
    c = (c - 1) % (1 << 256)
    words = [(c >> (64 * i)) & MASK64 for i in range(4)]
    g = np.random.Philox(counter=np.array(words, dtype=np.uint64),
                         key=np.array(key, dtype=np.uint64))
    return [int(v) for v in g.random_raw(4)]


CASES = [
    ((0, 0, 0, 0), (0, 0)),
    ((1, 0, 0, 0), (0, 0)),
    ((5, 7, 9, 0), (123, 0)),
    ((0, 3, 2, 0), (0, 0)),                 # borrow across words in numpy's form
    ((0, 0, 0, 0), (MASK64, MASK64)),
    ((MASK64, MASK64, MASK64, MASK64), (0xDEADBEEF, 42)),
    ((46117, 19, 5, 0), (2024, 0)),          # a typical (cell block, step, level, 0)
]


@pytest.mark.parametrize("counter,key", CASES)
def test_philox_matches_numpy(counter, key):
    got = [int(np.asarray(w)) for w in philox4x64(counter, key)]
    assert got == numpy_block(counter, key)


def test_philox_vectorised_matches_numpy():
    rng = np.random.default_rng(7)
    ctr = rng.integers(0, 1 << 63, size=(64, 4), dtype=np.uint64) * np.uint64(2) + np.uint64(1)
    key = (np.uint64(991), np.uint64(3))
    words = philox4x64(tuple(ctr[:, i] for i in range(4)), key)
    for r in range(ctr.shape[0]):
        want = numpy_block(tuple(int(v) for v in ctr[r]), (991, 3))
        assert [int(words[i][r]) for i in range(4)] == want


def test_mulhilo64_against_python_integers():
    rng = np.random.default_rng(3)
    a = rng.integers(0, 1 << 64, size=1000, dtype=np.uint64, endpoint=False)
    a[:4] = [0, 1, MASK64, 1 << 63]
    for b in (0, 1, MASK64, 0xD2E7470EE14C6C93, 0xCA5A826395121157):
        hi, lo = mulhilo64(a, np.uint64(b))
        for x, h, l in zip(a, hi, lo):
            p = int(x) * b
            assert int(h) == p >> 64 and int(l) == p & MASK64


def test_fire_threshold_values():
    assert fire_threshold(0.0) == 0
    assert fire_threshold(1.0) == 1 << 32
    assert fire_threshold(0.5) == 1 << 31
    assert fire_threshold(0.25) == 1 << 30
    with pytest.raises(ValueError):
        fire_threshold(1.5)
    with pytest.raises(ValueError):
        fire_threshold(-0.1)


def test_fire_extremes():
    assert not fire_mask(0, 0, 0, (2, 17, 33), 0.0).any()
    assert fire_mask(0, 0, 0, (2, 17, 33), 1.0).all()


def test_fire_bits_are_the_32_bit_halves_of_the_block():
    """Cell idx uses block (idx >> 3, t, l, 0), word (idx >> 1) & 3, upper half
    for odd idx and lower half for even idx: the 8 cells of a block use all
    256 bits of one Philox call."""
    seed, lvl, t = 11, 2, 5
    m = fire_mask(seed, lvl, t, (1, 4, 16), 0.5).reshape(-1)
    for idx in range(64):
        block = numpy_block((idx >> 3, t, lvl, 0), (seed, 0))
        word = block[(idx >> 1) & 3]
        draw = (word >> 32) if idx & 1 else (word & 0xFFFFFFFF)
        assert m[idx] == (draw < (1 << 31))


def test_fire_bits_of_one_block_use_distinct_bits():
    """The 8 draws of one block are the 8 distinct 32-bit halves (no draw is
    reused for two cells)."""
    seed, lvl, t = 3, 0, 1
    block = numpy_block((5, t, lvl, 0), (seed, 0))
    halves = sorted([w & 0xFFFFFFFF for w in block] + [w >> 32 for w in block])
    for p in (0.2, 0.5, 0.8):
        thr = fire_threshold(p)
        idx = np.arange(40, 48, dtype=np.uint64)
        got = fire_bits(seed, lvl, t, idx, p)
        assert int(got.sum()) == sum(h < thr for h in halves)


def test_batch_index_is_counter_word_3():
    """Image b of a batch draws from counter (idx >> 3, t, l, b); b = 0 is the
    single-image mask."""
    seed, lvl, t = 4, 1, 2
    for b in (0, 1, 7):
        m = fire_mask(seed, lvl, t, (1, 2, 16), 0.5, batch=b).reshape(-1)
        for idx in range(32):
            block = numpy_block((idx >> 3, t, lvl, b), (seed, 0))
            word = block[(idx >> 1) & 3]
            draw = (word >> 32) if idx & 1 else (word & 0xFFFFFFFF)
            assert m[idx] == (draw < (1 << 31))
    np.testing.assert_array_equal(fire_mask(seed, lvl, t, (2, 9, 13), 0.5),
                                  fire_mask(seed, lvl, t, (2, 9, 13), 0.5, batch=0))


def test_batch_masks_are_independent():
    base = fire_mask(0, 0, 0, (1, 64, 64), 0.5)
    for b in (1, 2):
        agree = (base == fire_mask(0, 0, 0, (1, 64, 64), 0.5, batch=b)).mean()
        assert 0.45 < agree < 0.55


def test_fire_rate_is_binomial():
    n = 1 << 18
    for p in (0.5, 0.1, 0.9):
        frac = fire_mask(0, 1, 3, (1, 1, n), p).mean()
        sd = np.sqrt(p * (1 - p) / n)
        assert abs(frac - p) < 6 * sd


def test_masks_differ_across_step_level_seed():
    base = fire_mask(0, 0, 0, (1, 64, 64), 0.5)
    for other in (fire_mask(0, 0, 1, (1, 64, 64), 0.5), fire_mask(0, 1, 0, (1, 64, 64), 0.5),
                  fire_mask(1, 0, 0, (1, 64, 64), 0.5)):
        agree = (base == other).mean()
        assert 0.45 < agree < 0.55


def test_window_indices_match_full_grid():
    grid = (3, 10, 14)
    full = fire_mask(9, 1, 2, grid, 0.5)
    origin, shape = (1, 2, 5), (2, 7, 6)
    idx = linear_index(origin, shape, grid)
    win = fire_bits(9, 1, 2, idx, 0.5)
    np.testing.assert_array_equal(win, full[1:3, 2:9, 5:11])
