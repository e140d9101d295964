"""Pins of the oracle's candidate stream (Philox4x64-10 and its decoding).

Philox is pinned against numpy.random.Philox, an independent implementation
of the same published generator; numpy encrypts counter+1 for a stored counter
(established here: a stored all-ones counter yields the block of counter 0).
Integer maps are pinned with exact rational arithmetic; uniformity with a
chi-square test.
"""
from fractions import Fraction

import numpy as np
import pytest

from oracle.philox import (MASK64, Candidate, decode, draw, locate, mulhi64,
                           philox4x64, ternary_next, unit_r)


def numpy_block(ctr, key):
    """numpy's Philox block for counter `ctr` (numpy increments before encrypting)."""
    c = sum(int(v) << (64 * n) for n, v in enumerate(ctr)) - 1
    c %= 1 << 256
    words = [(c >> (64 * n)) & MASK64 for n in range(4)]
    bg = np.random.Philox(key=np.array([int(key[0]), int(key[1])], dtype=np.uint64),
                          counter=np.array(words, dtype=np.uint64))
    return tuple(int(v) for v in bg.random_raw(4))


def test_numpy_counter_convention():
    bg = np.random.Philox(key=[0, 0], counter=[MASK64] * 4)
    assert tuple(int(v) for v in bg.random_raw(4)) == philox4x64((0, 0, 0, 0), (0, 0))


@pytest.mark.parametrize("seed", [0, 1, 4002, 2 ** 64 - 1])
def test_philox_matches_numpy(seed):
    rng = np.random.Generator(np.random.PCG64(seed % 1000))
    for _ in range(50):
        ctr = [int(v) for v in rng.integers(0, 2 ** 63, size=4, dtype=np.uint64)]
        ctr[0] |= 1  # avoid the borrow-free special case only
        key = (seed, int(rng.integers(0, 2 ** 63)))
        assert philox4x64(ctr, key) == numpy_block(ctr, key)
    for t, k in [(0, 0), (1, 0), (0, 1), (19999, 0), (5000, 63), (2 ** 40, 7)]:
        assert draw(seed, 3, t, k) == numpy_block((t, k, 0, 0), (seed, 3))


def test_rounds_parameter_changes_output():
    assert philox4x64((1, 2, 3, 4), (5, 6), rounds=7) != philox4x64((1, 2, 3, 4), (5, 6))


def test_mulhi64_exact():
    rng = np.random.Generator(np.random.PCG64(7))
    for _ in range(2000):
        a = int(rng.integers(0, 2 ** 63)) * 2 + int(rng.integers(0, 2))
        n = int(rng.integers(1, 2 ** 40))
        q = mulhi64(a, n)
        assert Fraction(q) <= Fraction(a * n, 2 ** 64) < Fraction(q + 1)
        assert 0 <= q < n
    assert mulhi64(MASK64, 13008896) == 13008895
    assert mulhi64(0, 13008896) == 0


def test_unit_r_exact_grid():
    for m in [0, 1, 2 ** 23 - 1, 2 ** 23, 2 ** 23 + 1, 2 ** 24 - 1, 12345]:
        r = unit_r(m << 40 | 0xFFFFFFFFFF)
        assert r.dtype == np.float32
        assert Fraction(float(r)) == Fraction(m, 2 ** 23) - 1
    assert unit_r(0) == np.float32(-1.0)
    assert unit_r(MASK64) == np.float32(1.0 - 2.0 ** -23)


def test_increment_rounding_is_single_precision():
    """d = fl32(delta * r) and w' = fl32(w + d): one IEEE single rounding each."""
    delta = 0.05
    rng = np.random.Generator(np.random.PCG64(11))
    for _ in range(500):
        w2 = int(rng.integers(0, 2 ** 63)) * 2
        r = unit_r(w2)
        d = np.float32(np.float32(delta) * r)
        exact = Fraction(float(np.float32(delta))) * Fraction(float(r))
        # the nearest fp32 to the exact product, checked against its neighbours
        up = np.nextafter(d, np.float32(np.inf))
        dn = np.nextafter(d, np.float32(-np.inf))
        err = abs(Fraction(float(d)) - exact)
        assert err <= abs(Fraction(float(up)) - exact)
        assert err <= abs(Fraction(float(dn)) - exact)


def test_flat_index_uniformity_chi2():
    """Flat indices over 10 equal bins are uniform (chi-square, 9 dof)."""
    P = 13008896
    n = 200000
    counts = np.zeros(10)
    for k in range(n):
        counts[mulhi64(draw(1, 2, k // 64, k % 64)[0], P) * 10 // P] += 1
    chi2 = float(((counts - n / 10) ** 2 / (n / 10)).sum())
    assert chi2 < 27.9  # p = 0.001 for 9 dof


def test_r_uniformity_chi2():
    n = 100000
    counts = np.zeros(16)
    for k in range(n):
        r = float(unit_r(draw(9, 9, k, 0)[2]))
        counts[min(int((r + 1.0) * 8), 15)] += 1
    chi2 = float(((counts - n / 16) ** 2 / (n / 16)).sum())
    assert chi2 < 37.7  # p = 0.001 for 15 dof


def test_decode_round_trip_weight_mode():
    shapes = [(16384, 784), (10, 16384)]
    sizes = [s[0] * s[1] for s in shapes]
    for t in range(300):
        c = decode(draw(4002, 2, t, 5), shapes, 0.05, "weight")
        assert 0 <= c.flat < sum(sizes)
        off = c.flat - sum(sizes[:c.layer])
        assert off == c.j * shapes[c.layer][1] + c.i
        assert locate(c.flat, sizes) == (c.layer, off)
        assert abs(float(c.d)) <= 0.05


def test_decode_layer_mode():
    shapes = [(256, 784)] + [(256, 256)] * 23 + [(10, 256)]
    seen = set()
    for t in range(2000):
        w = draw(4003, 3, t, 0)
        c = decode(w, shapes, 0.01, "layer")
        assert c.layer == mulhi64(w[1], 25)
        seen.add(c.layer)
        assert 0 <= c.j < shapes[c.layer][0] and 0 <= c.i < shapes[c.layer][1]
    assert seen == set(range(25))


def test_decode_one_dimensional_tensor():
    shapes = [(65, 128), (128,), (3, 4)]
    for t in range(500):
        c = decode(draw(1, 1, t, 0), shapes, 0.02, "weight")
        if c.layer == 1:
            assert c.i == 0 and 0 <= c.j < 128
            return
    pytest.fail("no draw landed in the 1-D tensor")


def test_ternary_moves():
    assert [ternary_next(-1, b) for b in (0, 1)] == [0, 1]
    assert [ternary_next(0, b) for b in (0, 1)] == [-1, 1]
    assert [ternary_next(1, b) for b in (0, 1)] == [-1, 0]
    codes = [np.array([[1, 0], [-1, 0]], dtype=np.int8)]
    scales = [np.float32(1 / np.sqrt(2))]
    for t in range(100):
        w = draw(5, 5, t, 0)
        c = decode(w, [(2, 2)], 0.0, "weight", codes, scales)
        cur = int(codes[0][c.j, c.i])
        assert c.code != cur and c.code in (-1, 0, 1)
        assert c.code == ternary_next(cur, w[3] >> 63)
        assert Fraction(float(c.d)) == (c.code - cur) * Fraction(float(scales[0]))


@pytest.mark.parametrize("delta", [0.05, 0.01, 0.1])
def test_decode_increment_from_numpy_words(delta):
    """The continuous increment of Eq. 1 rebuilt from numpy's raw Philox words
    and exact rationals: r = (w2 >> 40) / 2^23 - 1 (word w2, top 24 bits) and
    d = the fp32 nearest to fl32(delta) * r.  Decoding r from any other word,
    or other bits, fails here."""
    shapes = [(16384, 784), (10, 16384)]
    df = Fraction(float(np.float32(delta)))
    for t in range(200):
        w = numpy_block((t, 3, 0, 0), (4002, 2))
        c = decode(draw(4002, 2, t, 3), shapes, delta, "weight")
        r = Fraction(w[2] >> 40, 2 ** 23) - 1
        exact = df * r  # <= 48 significant bits: exact in fp64
        assert Fraction(float(exact)) == exact
        want = np.float32(float(exact))  # one rounding to single precision
        assert np.float32(c.d).tobytes() == want.tobytes(), (t, c.d, want)
        P = sum(a * b for a, b in shapes)
        assert c.flat == (w[0] * P) >> 64


def test_accept_uniform_from_numpy_words():
    """The Metropolis uniform (Eq. 7): word w0 of the block at counter
    (t, k, 1, 0), U = (w0 >> 11) / 2^53, exact in fp64."""
    from oracle.philox import accept_uniform
    for t, k in [(0, 0), (7, 3), (19999, 63), (2 ** 33, 1)]:
        w = numpy_block((t, k, 1, 0), (4001, 1))
        u = accept_uniform(4001, 1, t, k)
        assert Fraction(u) == Fraction(w[0] >> 11, 2 ** 53)
        assert 0.0 <= u < 1.0
        assert u != float(Fraction(draw(4001, 1, t, k)[0] >> 11, 2 ** 53))  # not stream 0
