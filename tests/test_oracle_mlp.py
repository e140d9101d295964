"""Pins of the fp64 MLP oracle.

* The loss (Eq. 2) against PyTorch's CPU fp64 ``tanh``/``exp``/``cross_entropy``
  (an independent library implementation), and the closed form L = ln C when
  the output layer is zero.
* Weight indexing against the local limit of Eq. 8: dL/d -> dL/dW[l][j, i]
  from PyTorch autograd; a transposed index fails.
* The incremental evaluator of Sec. 2.4 against full recomputation.
* The size convention against the parameter counts the paper prints.
"""
import math
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle.mlp import (FullMLP, IncrementalMLP, MLPState, forward_fields, mean_ce,
                        per_sample_ce, phi)
from oracle.philox import Candidate

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def torch_loss(weights, X, y, act, gamma=1.0, requires_grad=False):
    Ws = [torch.tensor(np.asarray(w, dtype=np.float64), requires_grad=requires_grad) for w in weights]
    a = torch.tensor(np.asarray(X, dtype=np.float64))
    for l, W in enumerate(Ws):
        z = a @ W.T
        if l < len(Ws) - 1:
            a = torch.tanh(z) if act == "tanh" else torch.exp(-gamma * z * z)
    L = F.cross_entropy(z, torch.tensor(np.asarray(y, dtype=np.int64)))
    return L, Ws


def random_net(widths, N, seed, scale=1.0, density=0.3):
    rng = np.random.Generator(np.random.PCG64(seed))
    X = (rng.uniform(size=(N, widths[0])) * (rng.uniform(size=(N, widths[0])) < density)).astype(np.float32)
    y = rng.integers(0, widths[-1], size=N).astype(np.int32)
    Ws = [rng.uniform(-scale, scale, size=(widths[l + 1], widths[l])).astype(np.float32)
          / np.float32(math.sqrt(widths[l])) for l in range(len(widths) - 1)]
    return X, y, Ws


@pytest.mark.parametrize("act", ["tanh", "gauss"])
@pytest.mark.parametrize("widths", [(5, 7, 3), (64, 32, 10), (20, 16, 12, 8, 6)])
def test_loss_matches_torch(act, widths):
    X, y, Ws = random_net(widths, 97, 1, scale=2.0)
    ours = FullMLP(MLPState(Ws), X, y, act, 0.7).loss()
    ref, _ = torch_loss(Ws, X, y, act, 0.7)
    assert abs(ours - ref.item()) <= 1e-12 * abs(ref.item())


def test_per_sample_ce_matches_torch_with_large_logits():
    rng = np.random.Generator(np.random.PCG64(3))
    z = rng.normal(scale=300.0, size=(50, 65))
    y = rng.integers(0, 65, size=50)
    ref = F.cross_entropy(torch.tensor(z), torch.tensor(y), reduction="none").numpy()
    np.testing.assert_allclose(per_sample_ce(z, y), ref, rtol=1e-13, atol=1e-10)


@pytest.mark.parametrize("C", [2, 10, 65])
def test_zero_output_layer_gives_log_C(C):
    X, y, Ws = random_net((12, 9, C), 40, 5)
    Ws[-1][:] = 0
    L = FullMLP(MLPState(Ws), X, y, "tanh").loss()
    assert abs(L - math.log(C)) <= 4e-16 * math.log(C)


def test_paper_parameter_counts():
    rows = [l.split() for l in open(os.path.join(GOLDEN, "paper_param_counts.txt"))
            if l.strip() and not l.startswith("#")]
    for kind, nl, value in rows:
        widths = [784] + [256] * (int(nl) - 2) + [10]
        shapes = [(widths[l + 1], widths[l]) for l in range(len(widths) - 1)]
        n_weights = sum(a * b for a, b in shapes)
        n_biases = sum(widths[1:])
        if kind == "weights_exact":
            assert n_weights == int(value)
        else:
            total = n_weights + n_biases
            assert float(f"{total:.3g}") == float(value), (nl, total)


@pytest.mark.parametrize("act", ["tanh", "gauss"])
def test_finite_difference_matches_autograd(act):
    """Eq. 8: dL = g . dW + O(|dW|^2); a transposed or shifted index fails."""
    widths = (6, 5, 4, 3)
    X, y, Ws = random_net(widths, 64, 8, scale=1.5, density=0.8)
    L, Wt = torch_loss(Ws, X, y, act, 1.0, requires_grad=True)
    L.backward()
    model = FullMLP(MLPState(Ws), X, y, act, 1.0)
    L0 = model.loss()
    rng = np.random.Generator(np.random.PCG64(2))
    checked = 0
    for _ in range(30):
        l = int(rng.integers(0, 3))
        j = int(rng.integers(0, widths[l + 1]))
        i = int(rng.integers(0, widths[l]))
        g = Wt[l].grad[j, i].item()
        if abs(g) < 1e-4:
            continue
        errs = []
        for d in (np.float32(1e-3), np.float32(1e-4)):
            c = Candidate(0, l, j, i, d)
            dw = float(model.state.new_value(c)) - float(Ws[l][j, i])
            fd = (model.eval(c) - L0) / dw
            errs.append(abs(fd - g))
        assert errs[1] <= 1e-3
        assert errs[1] <= 0.5 * errs[0] + 1e-10  # the error shrinks with d: O(d)
        if j < widths[l] and i < widths[l + 1]:
            gt = Wt[l].grad[i, j].item()
            if abs(gt - g) > 10 * errs[1]:
                assert abs(fd - gt) > abs(fd - g)
        checked += 1
    assert checked >= 10


def _all_candidates(widths, ternary=False):
    cands = []
    for l in range(len(widths) - 1):
        for j in range(widths[l + 1]):
            for i in range(widths[l]):
                if ternary:
                    cands.append(Candidate(0, l, j, i, np.float32(0), 1))
                else:
                    cands.append(Candidate(0, l, j, i, np.float32(0.173)))
                    cands.append(Candidate(0, l, j, i, np.float32(-0.031)))
    return cands


@pytest.mark.parametrize("act", ["tanh", "gauss"])
@pytest.mark.parametrize("widths", [(7, 5, 3), (6, 5, 4, 3), (8, 6, 6, 5, 4)])
def test_incremental_equals_full(act, widths):
    X, y, Ws = random_net(widths, 53, 4, scale=1.5)
    full = FullMLP(MLPState(Ws), X, y, act, 0.8)
    inc = IncrementalMLP(MLPState(Ws), X, y, act, 0.8)
    assert abs(full.loss() - inc.loss()) <= 1e-13
    cands = _all_candidates(widths)
    for n, c in enumerate(cands):
        a, b = full.eval(c), inc.eval(c)
        assert abs(a - b) <= 1e-12 * abs(a), (c, a, b)
        if n % 7 == 0:  # commit a few, the caches must stay consistent
            full.commit(c, a)
            inc.commit(c, b)
            assert abs(full.loss_of(full.state.weights) - inc.loss()) <= 1e-12


def test_incremental_equals_full_ternary():
    widths = (9, 6, 5, 4)
    rng = np.random.Generator(np.random.PCG64(12))
    X, y, _ = random_net(widths, 41, 12)
    codes = [rng.integers(-1, 2, size=(widths[l + 1], widths[l])).astype(np.int8) for l in range(3)]
    scales = [np.float32(1 / math.sqrt(widths[l])) for l in range(3)]
    Ws = [(c.astype(np.float32) * s).astype(np.float32) for c, s in zip(codes, scales)]
    full = FullMLP(MLPState(Ws, codes, scales), X, y, "gauss")
    inc = IncrementalMLP(MLPState(Ws, codes, scales), X, y, "gauss")
    for t in range(120):
        c = full.candidate(1, 1, t, 0, 0.0)
        assert c == inc.candidate(1, 1, t, 0, 0.0)
        a, b = full.eval(c), inc.eval(c)
        assert abs(a - b) <= 1e-12 * a
        if a < full.loss():
            full.commit(c, a)
            inc.commit(c, b)
    for l in range(3):
        np.testing.assert_array_equal(full.state.codes[l], inc.state.codes[l])
        np.testing.assert_array_equal(full.state.weights[l],
                                      full.state.codes[l].astype(np.float32) * scales[l])


def test_zero_delta_leaves_loss_bitwise():
    X, y, Ws = random_net((10, 8, 6, 4), 33, 6)
    full = FullMLP(MLPState(Ws), X, y, "tanh")
    L = full.loss()
    for c in _all_candidates((10, 8, 6, 4))[::5]:
        z = Candidate(0, c.layer, c.j, c.i, np.float32(0.0))
        assert full.eval(z) == L


def test_phi_values():
    z = np.array([0.0, 0.5, -2.0])
    np.testing.assert_allclose(phi(z, "gauss", 1.0), np.exp(-z * z), rtol=0, atol=0)
    assert phi(np.array([0.0]), "gauss", 0.4)[0] == 1.0
    np.testing.assert_allclose(phi(z, "tanh"), torch.tanh(torch.tensor(z)).numpy(), rtol=1e-15)
