"""Pins of the oracle's deep MLPs with biases and layer normalization (Sec. 2.1).

* The forward pass and loss against PyTorch's fp64 linear (with bias),
  layer_norm (no affine parameters) and transfer functions.
* Each candidate's loss change against the definition recomputed by
  PyTorch on the whole net, for weights and biases of every layer, with and
  without normalization and biases, for ReLU, tanh and the Gaussian.
* The layer-sticky schedule against numpy's Philox words; every candidate of
  a block in the block's layer; bias entries drawn.
* A bias candidate moves every sample; commits keep the caches exact.
"""
import numpy as np
import pytest
import torch

from oracle.normmlp import NormMLP, layer_norm, sticky_layer
from oracle.philox import Candidate
from test_oracle_philox import numpy_block


def net(widths, bias=True, seed=0, a=None):
    rng = np.random.default_rng(seed)
    ws = []
    for l in range(len(widths) - 1):
        amp = np.sqrt(8.0 / widths[l]) if a is None else a
        w = rng.uniform(-amp, amp, (widths[l + 1], widths[l] + (1 if bias else 0)))
        ws.append(w.astype(np.float32))
    return ws


def data(n0, N, C, seed=1):
    rng = np.random.default_rng(seed)
    X = (rng.uniform(0, 1, (N, n0)) * (rng.uniform(size=(N, n0)) < 0.5)).astype(np.float32)
    return X, rng.integers(0, C, N)


def torch_loss(ws, X, y, act, gamma, bias, ln, eps):
    a = torch.from_numpy(X.astype(np.float64))
    L = len(ws)
    for l, w in enumerate(ws):
        W = torch.from_numpy(w.astype(np.float64))
        z = torch.nn.functional.linear(a, W[:, :-1], W[:, -1]) if bias else a @ W.T
        if l < L - 1:
            h = torch.nn.functional.layer_norm(z, (z.shape[1],), eps=eps) if ln else z
            a = {"relu": torch.relu, "tanh": torch.tanh,
                 "gauss": lambda v: torch.exp(-gamma * v * v)}[act](h)
    return float(torch.nn.functional.cross_entropy(z, torch.from_numpy(y)))


def test_layer_norm_matches_torch():
    z = np.random.default_rng(3).standard_normal((7, 33)) * 5 + 2
    ref = torch.nn.functional.layer_norm(torch.from_numpy(z), (33,), eps=1e-5).numpy()
    np.testing.assert_allclose(layer_norm(z, 1e-5), ref, rtol=0, atol=1e-13)


@pytest.mark.parametrize("act", ["relu", "tanh", "gauss"])
@pytest.mark.parametrize("bias,ln", [(True, True), (True, False), (False, True)])
def test_forward_and_delta_match_torch(act, bias, ln):
    widths = (20, 16, 16, 16, 4)
    ws = net(widths, bias)
    X, y = data(20, 48, 4)
    m = NormMLP(ws, X, y, act, 0.4, bias=bias, ln=ln, eps=1e-5)
    L0 = torch_loss(ws, X, y, act, 0.4, bias, ln, 1e-5)
    assert abs(m.loss() - L0) <= 1e-13
    rng = np.random.default_rng(5)
    for l in range(len(ws)):
        rows, cols = ws[l].shape
        for j, i in [(int(rng.integers(rows)), int(rng.integers(cols - 1))), (rows - 1, cols - 1)]:
            c = Candidate(0, l, j, i, np.float32(0.05))
            dl, mag = m.delta(c)
            exact = torch_loss(m.with_candidate(c), X, y, act, 0.4, bias, ln, 1e-5) - L0
            assert abs(dl - exact) <= 1e-9 * abs(exact) + 1e-14, (l, j, i, dl, exact)
            assert mag > 0 or exact == 0.0


def test_bias_moves_every_sample_and_commit_keeps_caches():
    widths = (12, 8, 8, 3)
    ws = net(widths, True)
    X, y = data(12, 30, 3)
    X[:, 5] = 0.0  # an input that is zero on every sample
    m = NormMLP(ws, X, y, "relu", bias=True, ln=True)
    # a weight on an always-zero input changes nothing; the bias of its row does
    assert m.delta(Candidate(0, 0, 2, 5, np.float32(0.1)))[0] == 0.0
    dl, _ = m.sample_changes(Candidate(0, 0, 2, 12, np.float32(0.1)))
    assert np.count_nonzero(dl) == len(y)
    for t in range(5):
        c = m.candidate(1, 2, t, 0, 0.05, "weight")
        d, _ = m.delta(c)
        m.commit(c, m.loss() + d)
    assert abs(m.loss() - torch_loss(m.weights, X, y, "relu", 1.0, True, True, 1e-5)) <= 1e-13


def test_sticky_schedule():
    widths = (30, 16, 16, 16, 5)
    ws = net(widths, True)
    X, y = data(30, 10, 5)
    m = NormMLP(ws, X, y, "relu", sticky=8)
    seed, tag = 77, 9
    for e in range(6):
        w0 = numpy_block((e, 0, 0, 1), (seed, tag))[0]
        assert sticky_layer(seed, tag, e, 4) == (w0 * 4) >> 64
    layers = set()
    bias_hits = 0
    for t in range(0, 48):
        lt = sticky_layer(seed, tag, t // 8, 4)
        layers.add(lt)
        for k in range(6):
            c = m.candidate(seed, tag, t, k, 0.01, "sticky")
            assert c.layer == lt
            rows, cols = ws[lt].shape
            assert 0 <= c.j < rows and 0 <= c.i < cols
            w = numpy_block((t, k, 0, 0), (seed, tag))
            assert c.j * cols + c.i == (w[0] * rows * cols) >> 64
            bias_hits += c.i == cols - 1
    assert len(layers) >= 3 and bias_hits > 0
