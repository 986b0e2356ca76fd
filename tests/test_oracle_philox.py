"""Pins of the oracle's counter-based generator (Philox4x32-10) and of the dropout masks drawn from it.

The generator is pinned by the known-answer vectors published with it (the Random123 distribution of
Salmon et al., SC 2011: counter and key all zero, all ones, and the hexadecimal digits of pi), so a wrong
multiplier, Weyl constant, word order or round count fails here.  The mask is pinned by what the
definition fixes: p = 0 keeps everything at 1, the values are 0 or 1 / (1 - p), the dropped fraction
matches p, the four units of a 4-unit block are the four words of one generator call, and the step and
seed move the draw."""
import numpy as np
import pytest

from oracle import philox as PX


@pytest.mark.parametrize("ctr,key,want", [
    ((0, 0, 0, 0), (0, 0), (0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8)),
    ((0xFFFFFFFF,) * 4, (0xFFFFFFFF, 0xFFFFFFFF), (0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD)),
    ((0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344), (0xA4093822, 0x299F31D0),
     (0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1)),
])
def test_known_answer_vectors(ctr, key, want):
    assert tuple(int(x) for x in PX.philox4x32_10(np.array([ctr]), key)[0]) == want


def test_vectorised_rows_are_independent_calls():
    ctr = np.array([(0, 0, 0, 0), (0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344), (0, 0, 0, 0)])
    out = PX.philox4x32_10(ctr, (0, 0))
    assert np.array_equal(out[0], out[2]) and not np.array_equal(out[0], out[1])


def test_threshold():
    assert PX.dropout_threshold(0.0) == 0
    assert PX.dropout_threshold(0.5) == 2 ** 31
    assert PX.dropout_threshold(0.25) == 2 ** 30
    assert PX.dropout_threshold(1.0 - 2.0 ** -20) == 2 ** 32 - 2 ** 12
    assert PX.dropout_threshold(1.0 - 1e-12) == 2 ** 32 - 1  # floor((1 - 1e-12) 2^32) = 2^32 - 1
    for bad in (-0.1, 1.0, float("nan")):
        with pytest.raises(ValueError):
            PX.dropout_threshold(bad)


def test_zero_probability_keeps_every_unit():
    m = PX.dropout_mask(37, 13, 0.0, seed=5, step=1)
    assert m.shape == (37, 13) and m.dtype == np.float32 and np.all(m == 1.0)


@pytest.mark.parametrize("p", [0.1, 0.25, 0.5])
def test_values_and_dropped_fraction(p):
    m = PX.dropout_mask(400, 300, p, seed=123456789012345, step=7)
    s = np.float32(1.0 / (1.0 - p))
    assert set(np.unique(m).tolist()) == {0.0, float(s)}
    frac = float((m == 0).mean())
    sd = np.sqrt(p * (1 - p) / m.size)
    assert abs(frac - p) < 5 * sd
    # inverted dropout: the mean multiplier is 1 up to sampling noise
    assert abs(float(m.astype(np.float64).mean()) - 1.0) < 5 * sd * float(s)


def test_unit_blocks_are_the_words_of_one_call():
    seed, step, p = (7 << 32) | 3, (2 << 32) | 9, 0.5
    m = PX.dropout_mask(5, 11, p, seed, step)
    t = PX.dropout_threshold(p)
    for v in range(5):
        for jb in range(3):
            words = PX.philox4x32_10(np.array([(v, jb, 9, 2)]), (3, 7))[0]
            for i in range(4):
                j = 4 * jb + i
                if j < 11:
                    assert m[v, j] == (0.0 if words[i] < t else 2.0)


def test_step_and_seed_move_the_draw():
    a = PX.dropout_mask(64, 64, 0.5, seed=1, step=1)
    assert not np.array_equal(a, PX.dropout_mask(64, 64, 0.5, seed=1, step=2))
    assert not np.array_equal(a, PX.dropout_mask(64, 64, 0.5, seed=2, step=1))
    assert not np.array_equal(a, PX.dropout_mask(64, 64, 0.5, seed=1, step=1 + (1 << 32)))
    assert np.array_equal(a, PX.dropout_mask(64, 64, 0.5, seed=1, step=1))
    # a node's row does not depend on how many nodes are drawn
    assert np.array_equal(a[:10], PX.dropout_mask(10, 64, 0.5, seed=1, step=1))
