"""Pins of the oracle's difference form of the loss change.

The incremental oracle carries the changes of the local fields from layer to
layer and forms each sample's loss change from its logit change, with
  phi(z + dz) - phi(z) = sinh(dz) / (cosh z cosh(z + dz))          (tanh),
                       = exp(-g z^2) expm1(-g dz (2 z + dz))         (Gaussian),
  l(z + dz) - l(z)     = log1p(sum_c softmax(z)_c expm1(dz_c)) - dz_y.
These are exact identities, so the only question is rounding:

* against long-double (64-bit mantissa) direct differences of the library
  functions, over many scales of z and dz;
* against the definition L(W') - L(W) in fp64 where the change is large
  (the nets of the incremental-vs-full test);
* against the definition in long double on a deep, narrow tanh net with
  small initial weights (the deep workload's shape at a reduced sample
  count), where |dL| ~ 1e-11 and the fp64 definition itself keeps only four
  or five digits;
* a zero increment gives a zero change exactly.
"""
import numpy as np
import pytest

from oracle.mlp import (FullMLP, IncrementalMLP, MLPState, ce_change, dphi, phi, softmax)
from oracle.philox import Candidate, decode, draw
from workloads import CONFIGS, mlp_workload

from test_oracle_mlp import random_net

LD = np.longdouble


def _grid():
    rng = np.random.Generator(np.random.PCG64(41))
    z = np.concatenate([rng.uniform(-4, 4, 400), rng.normal(scale=1e-5, size=200),
                        rng.uniform(-20, 20, 50)])
    dz = np.concatenate([rng.uniform(-1, 1, 400) * 10.0 ** rng.uniform(-9, 0, 400),
                         rng.normal(scale=1e-6, size=200), rng.uniform(-1, 1, 50)])
    return z, dz


def test_dphi_tanh_against_long_double():
    z, dz = _grid()
    ref = np.tanh(z.astype(LD) + dz.astype(LD)) - np.tanh(z.astype(LD))
    got = dphi(z, dz, "tanh")
    ref = ref.astype(np.float64)
    # the long-double direct difference rounds two values of size <= 1 and
    # the argument z + dz: absolute error ~2^-64 (1 + |z|)
    tol = 1e-14 * np.abs(ref) + 4.0 * 2.0 ** -64 * (1 + np.abs(z))
    assert np.all(np.abs(got - ref) <= tol)
    assert np.all(dphi(z, np.zeros_like(z), "tanh") == 0.0)


@pytest.mark.parametrize("gamma", [1.0, 0.04])
def test_dphi_gauss_against_long_double(gamma):
    z, dz = _grid()
    zl, dzl = z.astype(LD), dz.astype(LD)
    ref = np.exp(-LD(gamma) * (zl + dzl) ** 2) - np.exp(-LD(gamma) * zl * zl)
    got = dphi(z, dz, "gauss", gamma)
    ref = ref.astype(np.float64)
    # two exponentials of size <= 1 and their rounded arguments g (z + dz)^2
    tol = 1e-13 * np.abs(ref) + 8.0 * 2.0 ** -64 * (1 + gamma * (np.abs(z) + np.abs(dz)) ** 2)
    assert np.all(np.abs(got - ref) <= tol)
    assert np.all(dphi(z, np.zeros_like(z), "gauss", gamma) == 0.0)


def test_ce_change_against_long_double():
    rng = np.random.Generator(np.random.PCG64(42))
    for C, scale in [(10, 1e-6), (10, 1.0), (65, 3.0), (2, 1e-3)]:
        z = rng.normal(scale=scale, size=(300, C))
        dz = rng.normal(size=(300, C)) * 10.0 ** rng.uniform(-10, -1, size=(300, 1))
        y = rng.integers(0, C, 300)
        zl, dzl = z.astype(LD), dz.astype(LD)

        def ce(v):
            m = v.max(axis=1, keepdims=True)
            return m[:, 0] + np.log(np.exp(v - m).sum(axis=1)) - v[np.arange(300), y]
        ref = (ce(zl + dzl) - ce(zl)).astype(np.float64)
        got, mag = ce_change(softmax(z), dz, y)
        # long double keeps 2^-64 of the loss (~ln C) in each of its two terms
        tol = 1e-13 * mag + 8.0 * 2.0 ** -64 * (np.log(C) + 2 * np.abs(z).max(axis=1))
        assert np.all(np.abs(got - ref) <= tol)
        assert np.all(ce_change(softmax(z), np.zeros_like(dz), y)[0] == 0.0)


@pytest.mark.parametrize("act", ["tanh", "gauss"])
@pytest.mark.parametrize("widths", [(7, 5, 3), (6, 5, 4, 3), (8, 6, 6, 5, 4)])
def test_delta_equals_definition_where_large(act, widths):
    X, y, Ws = random_net(widths, 53, 4, scale=1.5)
    full = FullMLP(MLPState(Ws), X, y, act, 0.8)
    inc = IncrementalMLP(MLPState(Ws), X, y, act, 0.8)
    n = 0
    for l in range(len(widths) - 1):
        for j in range(widths[l + 1]):
            for i in range(widths[l]):
                c = Candidate(0, l, j, i, np.float32(0.173))
                a, ma = full.delta(c)
                b, mb = inc.delta(c)
                # the fp64 definition rounds L' and L (~2) to 2^-53 each
                assert abs(a - b) <= 1e-9 * abs(a) + 2e-15, (c, a, b)
                # the sizes: of the logit change (full), of its terms (incremental)
                assert mb >= ma * (1 - 1e-9)
                n += abs(a) > 1e-6
    assert n > 10


def _long_double_loss(weights, X, y):
    a = X.astype(LD)
    for l, W in enumerate(weights):
        z = a @ W.astype(LD).T
        if l < len(weights) - 1:
            a = np.tanh(z)
    m = z.max(axis=1, keepdims=True)
    return np.mean(m[:, 0] + np.log(np.exp(z - m).sum(axis=1)) - z[np.arange(len(y)), y])


def test_delta_on_deep_narrow_net_against_long_double():
    """The deep workload's net (784 -> 24 x 256 -> 10 tanh, U(+-1/sqrt(fan_in)))
    on 48 of its samples: the logits are ~1e-7 and |dL| ~ 1e-11.  The
    difference form agrees with the long-double definition to 1e-6 relative
    (long double keeps ~2^-64 * 2.3 / 1e-11 ~ 1e-8 of dL)."""
    cfg = CONFIGS["deep"]
    w = mlp_workload(cfg.scaled(n_samples=48))
    X, y, Ws = w["X"], w["y"], w["weights"]
    inc = IncrementalMLP(MLPState(Ws), X, y, "tanh")
    L0 = _long_double_loss(Ws, X, y)
    shapes = [W.shape for W in Ws]
    worst_fp64 = 0.0
    for k in range(4):
        c = decode(draw(cfg.seed_stream, cfg.stream_tag, 0, k), shapes, cfg.delta, "layer")
        W2 = [W.copy() for W in Ws]
        W2[c.layer][c.j, c.i] = np.float32(Ws[c.layer][c.j, c.i] + c.d)
        ref = float(_long_double_loss(W2, X, y) - L0)
        got, _ = inc.delta(c)
        assert 0 < abs(ref) < 1e-8
        assert abs(got - ref) <= 1e-6 * abs(ref), (c, got, ref)
        fp64 = FullMLP(MLPState(Ws), X, y, "tanh").delta(c)[0]
        worst_fp64 = max(worst_fp64, abs(fp64 - ref) / abs(ref))
    # the reason the oracle uses the difference form: the fp64 definition is
    # far from the long-double value here
    assert worst_fp64 > 1e-6


def test_zero_increment_zero_change():
    X, y, Ws = random_net((10, 8, 6, 4), 33, 6)
    inc = IncrementalMLP(MLPState(Ws), X, y, "tanh")
    for l, (a, b) in enumerate([(8, 10), (6, 8), (4, 6)]):
        for j in range(a):
            c = Candidate(0, l, j, 1, np.float32(0.0))
            assert inc.delta(c) == (0.0, 0.0)


def test_commit_moves_caches_by_the_changes():
    X, y, Ws = random_net((9, 7, 6, 5), 61, 8, scale=1.3)
    inc = IncrementalMLP(MLPState(Ws), X, y, "gauss", 0.6)
    for t in range(40):
        c = inc.candidate(3, 4, t, 0, 0.3)
        dL, _ = inc.delta(c)
        L = inc.loss()
        inc.commit(c, L + dL)
        assert inc.loss() == L + dL
    fresh = IncrementalMLP(MLPState(inc.state.weights), X, y, "gauss", 0.6)
    for a, b in zip(inc.Z, fresh.Z):
        np.testing.assert_allclose(a, b, rtol=0, atol=1e-12)
    assert abs(inc.loss() - fresh.loss()) <= 1e-12
