"""Pins of the oracle's channel mutation (Sec. 2.3) and ReLU transfer (Sec. 2).

* The channel draw against numpy's Philox words and exact rational
  arithmetic: units by integer mulhi, re-drawn weights as the fp32 rounding
  of fl32(sqrt(8 / n)) times the grid value r.
* The incremental channel loss change (field changes layer to layer plus
  each path weight's point change) against the definition: the loss of the
  net with all path weights replaced, recomputed by PyTorch's fp64 ops.
* Special cases: a channel that leaves every weight as it is changes
  nothing, exactly; a one-layer channel is a single-weight change.
* Commits keep every cached field equal to a fresh forward pass.
* ReLU's field-change rule against its three cases, and the ReLU forward
  pass against torch.relu.
"""
import math
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle.mlp import FullMLP, IncrementalMLP, MLPState, dphi, forward_fields, mean_ce, phi
from oracle.philox import (Candidate, Channel, channel_words, decode_channel, he_amplitude,
                           philox4x64, unit_r)
from test_oracle_philox import numpy_block

MASK64 = (1 << 64) - 1


def fp32_round(q: Fraction) -> Fraction:
    """Round-to-nearest-even of a rational to fp32 (normal range)."""
    if q == 0:
        return Fraction(0)
    sign = -1 if q < 0 else 1
    a = abs(q)
    e = math.floor(math.log2(a))
    while Fraction(2) ** e > a:
        e -= 1
    while Fraction(2) ** (e + 1) <= a:
        e += 1
    ulp = Fraction(2) ** (e - 23)
    n = a / ulp
    fl = math.floor(n)
    rem = n - fl
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and fl % 2 == 1):
        fl += 1
    return sign * fl * ulp


def small_net(widths, seed=0, scale=None):
    rng = np.random.default_rng(seed)
    Ws = []
    for l in range(len(widths) - 1):
        a = math.sqrt(8.0 / widths[l]) if scale is None else scale
        Ws.append(rng.uniform(-a, a, (widths[l + 1], widths[l])).astype(np.float32))
    return Ws


def small_data(n0, N, C, seed=1):
    rng = np.random.default_rng(seed)
    X = (rng.uniform(0, 1, (N, n0)) * (rng.uniform(size=(N, n0)) < 0.4)).astype(np.float32)
    y = rng.integers(0, C, N)
    return X, y


def torch_loss(Ws, X, y, act, gamma):
    """The loss by PyTorch's fp64 ops (the definition, an independent library)."""
    a = torch.from_numpy(X.astype(np.float64))
    for l, W in enumerate(Ws):
        z = a @ torch.from_numpy(W.astype(np.float64)).T
        if l < len(Ws) - 1:
            if act == "relu":
                a = torch.relu(z)
            elif act == "tanh":
                a = torch.tanh(z)
            else:
                a = torch.exp(-gamma * z * z)
    return float(torch.nn.functional.cross_entropy(z, torch.from_numpy(y)))


# --------------------------------------------------------------------------
# the draw
# --------------------------------------------------------------------------

@pytest.mark.parametrize("widths", [(784, 256, 256, 256, 10), (784, 1024, 10), (5, 3)])
def test_channel_draw_from_numpy_words_and_exact_fractions(widths):
    L = len(widths) - 1
    seed, tag = 4021, 21
    for t, k in [(0, 0), (3, 5), (1000, 15), (2 ** 33, 63)]:
        n = 2 * L + 1
        words = []
        for b in range((n + 3) // 4):
            words += list(numpy_block((t, k, 2 + b, 0), (seed, tag)))
        words = words[:n]
        assert words == channel_words(seed, tag, t, k, n)
        ch = decode_channel(words, widths, "redraw")
        for m in range(L + 1):
            assert ch.units[m] == (words[m] * widths[m]) >> 64
            assert 0 <= ch.units[m] < widths[m]
        for m in range(L):
            # r on the 2^-23 grid of [-1, 1); the amplitude is fl32(sqrt(8 / n))
            r = Fraction(words[L + 1 + m] >> 40, 2 ** 23) - 1
            assert Fraction(float(unit_r(words[L + 1 + m]))) == r
            amp = fp32_round(Fraction(math.sqrt(8.0 / widths[m])))
            assert Fraction(float(he_amplitude(widths[m]))) == amp
            exp = fp32_round(amp * r) if r != 0 else Fraction(0)
            assert Fraction(float(ch.w_new[m])) == exp
            assert abs(float(ch.w_new[m])) <= float(amp)
        z = decode_channel(words, widths, "zero")
        assert z.units == ch.units and all(float(v) == 0.0 for v in z.w_new)


def test_channel_words_are_not_the_single_parameter_block():
    """Channel words come from counters (t, k, 2 + b, 0): never the draw's
    block (t, k, 0, 0) nor the Metropolis block (t, k, 1, 0)."""
    w = channel_words(9, 3, 11, 2, 12)
    assert tuple(w[:4]) == philox4x64((11, 2, 2, 0), (9, 3))
    assert tuple(w[4:8]) == philox4x64((11, 2, 3, 0), (9, 3))
    assert tuple(w[:4]) != philox4x64((11, 2, 0, 0), (9, 3))
    assert tuple(w[:4]) != philox4x64((11, 2, 1, 0), (9, 3))


# --------------------------------------------------------------------------
# the loss change
# --------------------------------------------------------------------------

@pytest.mark.parametrize("act", ["relu", "tanh", "gauss"])
@pytest.mark.parametrize("widths", [(12, 3), (12, 8, 3), (12, 8, 6, 3), (12, 8, 8, 8, 3)])
def test_channel_delta_matches_the_definition(act, widths):
    Ws = small_net(widths)
    X, y = small_data(widths[0], 60, widths[-1])
    inc = IncrementalMLP(MLPState(Ws), X, y, act, 0.4)
    L0 = torch_loss(Ws, X, y, act, 0.4)
    assert abs(inc.loss() - L0) <= 1e-12 * L0
    for scheme in ("channel_redraw", "channel_zero"):
        for k in range(12):
            ch = inc.candidate(7, 1, 0, k, 0.0, scheme)
            assert isinstance(ch, Channel) and len(ch.units) == len(widths)
            dl, mag = inc.delta(ch)
            ws = MLPState(Ws).with_channel(ch)
            exact = torch_loss(ws, X, y, act, 0.4) - L0
            # fp64 recomputation keeps ~1e-16 of the loss: the bar is that, or
            # 1e-10 of the change
            assert abs(dl - exact) <= 1e-10 * abs(exact) + 1e-14, (scheme, k, dl, exact)
            assert mag >= abs(dl) * 0.0  # sizes are non-negative
            full_dl, _ = FullMLP(MLPState(Ws), X, y, act, 0.4).delta(ch)
            assert abs(full_dl - exact) <= 1e-13


def test_channel_that_changes_nothing_is_exactly_zero():
    widths = (12, 8, 8, 3)
    Ws = small_net(widths)
    X, y = small_data(12, 40, 3)
    inc = IncrementalMLP(MLPState(Ws), X, y, "relu")
    u = (3, 2, 5, 1)
    same = Channel(u, tuple(np.float32(Ws[m][u[m + 1], u[m]]) for m in range(3)))
    assert inc.delta(same) == (0.0, 0.0)
    # zeroing a path that is already zero
    Wz = [w.copy() for w in Ws]
    for m in range(3):
        Wz[m][u[m + 1], u[m]] = 0.0
    incz = IncrementalMLP(MLPState(Wz), X, y, "relu")
    assert incz.delta(Channel(u, (np.float32(0),) * 3))[0] == 0.0


def test_one_layer_channel_is_a_single_weight_change():
    Ws = small_net((12, 3))
    X, y = small_data(12, 40, 3)
    inc = IncrementalMLP(MLPState(Ws), X, y, "relu")
    ch = Channel((4, 2), (np.float32(0.3),))
    c = Candidate(2 * 12 + 4, 0, 2, 4, np.float32(np.float32(0.3) - Ws[0][2, 4]))
    assert MLPState(Ws).new_value(c) == np.float32(0.3)
    a, _ = inc.delta(ch)
    b, _ = inc.delta(c)
    assert abs(a - b) <= 1e-15 * max(abs(b), 1e-300)


@pytest.mark.parametrize("act", ["relu", "tanh"])
def test_channel_commits_keep_the_caches_exact(act):
    widths = (12, 8, 8, 8, 3)
    Ws = small_net(widths)
    X, y = small_data(12, 50, 3)
    inc = IncrementalMLP(MLPState(Ws), X, y, act)
    full = FullMLP(MLPState(Ws), X, y, act)
    for t in range(6):
        ch = inc.candidate(3, 2, t, 0, 0.0, "channel_redraw" if t % 2 else "channel_zero")
        dl, _ = inc.delta(ch)
        inc.commit(ch, inc.loss() + dl)
        full.commit(ch, 0.0)
    for a, b in zip(inc.state.weights, full.state.weights):
        assert a.tobytes() == b.tobytes()
    Z = forward_fields([w.astype(np.float64) for w in inc.state.weights], inc.X, act, 1.0)
    for a, b in zip(inc.Z, Z):
        np.testing.assert_allclose(a, b, rtol=0, atol=1e-12)
    assert abs(inc.loss() - mean_ce(Z[-1], y)) <= 1e-12


# --------------------------------------------------------------------------
# ReLU
# --------------------------------------------------------------------------

def test_relu_field_change_cases():
    z = np.array([1.0, -1.0, 0.5, -0.5, 0.0, 0.0, 2.0])
    dz = np.array([0.25, 0.25, -1.0, 1.0, 0.0, -1.0, 1e-300])
    got = dphi(z, dz, "relu")
    exp = [0.25, 0.0, -0.5, 0.5, 0.0, 0.0, 1e-300]
    assert got.tolist() == exp
    # where both fields are positive the change is dz itself, whatever the size of z
    assert dphi(np.array([1e10]), np.array([1e-5]), "relu")[0] == 1e-5
    assert phi(np.array([-2.0, 0.0, 3.0]), "relu").tolist() == [0.0, 0.0, 3.0]


def test_relu_forward_matches_torch():
    widths = (20, 16, 16, 4)
    Ws = small_net(widths)
    X, y = small_data(20, 64, 4)
    L = mean_ce(forward_fields([w.astype(np.float64) for w in Ws], X.astype(np.float64), "relu",
                               1.0)[-1], y)
    assert abs(L - torch_loss(Ws, X, y, "relu", 1.0)) <= 1e-13
