"""Pins of the oracle's selection loop (Eq. 1, Eq. 6, Eq. 9, Eq. 12).

* Along the accepted trajectory the loss strictly decreases; on a rejected
  step it is unchanged (Eq. 6 with the strict reading).
* A zero increment leaves the loss unchanged bit for bit.
* Discrete weights (Eq. 12, W_ij in {-1, 0, 1}): on a 4-3-2 net all 36
  single-weight moves are enumerated with PyTorch fp64, every candidate's loss
  equals its table entry, and each step commits the first improving candidate
  of the table in stream order; the run ends in a one-flip local minimum after
  which nothing is accepted.  On a 2-2-2 net all 3^8 states are enumerated:
  the end state is a one-flip local minimum and no better than the global one.
* Eq. 9: for small increments, accepted moves go against the gradient.
* A K-candidate step equals the sequential scan of the same stream that drops
  the rest of a step after its first acceptance.
"""
import itertools
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import mca
from oracle.mlp import FullMLP, IncrementalMLP, MLPState
from oracle.philox import Candidate, ternary_next

from test_oracle_mlp import random_net, torch_loss


def test_trajectory_monotone_and_constant_on_reject():
    X, y, Ws = random_net((16, 12, 10, 5), 200, 21, scale=1.0)
    model = IncrementalMLP(MLPState(Ws), X, y, "tanh")
    recs = mca.run(model, 0, 600, 4, 77, 1, 0.2, scan_all=True)
    n_acc = 0
    for r in recs:
        if r.chosen >= 0:
            n_acc += 1
            assert r.L_after < r.L_before
            assert r.L_after == r.losses[r.chosen]
            assert all(Lk >= r.L_before for Lk in r.losses[:r.chosen])
        else:
            assert r.L_after == r.L_before
            assert all(Lk >= r.L_before for Lk in r.losses)
    assert 20 < n_acc < 600
    # the committed state really has the claimed loss
    fresh = FullMLP(MLPState(model.state.weights), X, y, "tanh")
    assert abs(fresh.loss() - recs[-1].L_after) < 1e-12


def test_ties_reading_accepts_zero_change():
    """With a dead input (always zero) every move on its weights has dL = 0:
    rejected under the strict rule, accepted when ties are accepted (Eq. 6)."""
    X, y, Ws = random_net((3, 2, 2), 30, 3)
    X[:, :] = 0
    X[:, 0] = 1.0
    model = FullMLP(MLPState(Ws), X, y, "tanh")
    L = model.loss()
    c = Candidate(0, 0, 1, 2, np.float32(0.05))
    assert model.eval(c) == L
    assert not mca.accepts(0.0, False) and mca.accepts(0.0, True)
    assert not mca.accepts(float("nan"), True) and not mca.accepts(float("inf"), True)


def ternary_torch_table(codes, scales, X, y, act):
    """L after every single-weight move of a ternary net, by PyTorch fp64."""
    base = [c.astype(np.float64) * float(s) for c, s in zip(codes, scales)]
    table = {}
    for l, c in enumerate(codes):
        for j, i in itertools.product(range(c.shape[0]), range(c.shape[1])):
            for new in (-1, 0, 1):
                if new == c[j, i]:
                    continue
                ws = [w.copy() for w in base]
                ws[l][j, i] = new * float(np.float32(scales[l]))
                L, _ = torch_loss(ws, X, y, act)
                table[(l, j, i, new)] = L.item()
    return table


def test_ternary_4_3_2_bruteforce():
    rng = np.random.Generator(np.random.PCG64(432))
    widths = (4, 3, 2)
    X = rng.uniform(size=(24, 4)).astype(np.float32)
    y = rng.integers(0, 2, size=24).astype(np.int32)
    codes = [rng.integers(-1, 2, size=(widths[l + 1], widths[l])).astype(np.int8) for l in range(2)]
    scales = [np.float32(1.0), np.float32(1.0 / math.sqrt(3))]
    Ws = [(c.astype(np.float32) * s) for c, s in zip(codes, scales)]
    model = FullMLP(MLPState(Ws, codes, scales), X, y, "gauss")
    K, steps_at_min = 4, 0
    for t in range(400):
        table = ternary_torch_table(model.state.codes, scales, X, y, "gauss")
        assert len(table) == 36
        L_t, _ = torch_loss([w.astype(np.float64) for w in model.state.weights], X, y, "gauss")
        L_t = L_t.item()
        assert abs(model.loss() - L_t) < 1e-12
        rec = mca.step(model, t, K, 9, 9, 0.0, scan_all=True)
        expect = -1
        for k, c in enumerate(rec.cands):
            ref = table[(c.layer, c.j, c.i, c.code)]
            assert abs(rec.losses[k] - ref) < 1e-12
            if expect < 0 and ref - L_t < -1e-12:
                expect = k
        assert rec.chosen == expect
        if min(table.values()) >= L_t - 1e-12:  # one-flip local minimum
            assert rec.chosen == -1
            steps_at_min += 1
            if steps_at_min > 60:
                break
    assert steps_at_min > 60, "never reached a one-flip local minimum"


def test_ternary_2_2_2_exhaustive():
    rng = np.random.Generator(np.random.PCG64(222))
    X = rng.uniform(-1, 1, size=(16, 2)).astype(np.float32)
    y = rng.integers(0, 2, size=16).astype(np.int32)
    scales = [np.float32(1 / math.sqrt(2))] * 2
    s = float(scales[0])
    states = np.array(list(itertools.product((-1, 0, 1), repeat=8)), dtype=np.float64)
    W1 = torch.tensor(states[:, :4].reshape(-1, 2, 2) * s)
    W2 = torch.tensor(states[:, 4:].reshape(-1, 2, 2) * s)
    xt = torch.tensor(X.astype(np.float64))
    z = torch.tanh(xt @ W1.transpose(1, 2)) @ W2.transpose(1, 2)
    yt = torch.tensor(y.astype(np.int64))
    all_L = torch.stack([F.cross_entropy(z[n], yt) for n in range(len(states))]).numpy()
    index = {tuple(int(v) for v in st): n for n, st in enumerate(states)}
    codes = [np.array([[1, 1], [1, 1]], dtype=np.int8), np.array([[-1, 1], [1, -1]], dtype=np.int8)]
    Ws = [(c.astype(np.float32) * sc) for c, sc in zip(codes, scales)]
    model = FullMLP(MLPState(Ws, codes, scales), X, y, "tanh")
    key = lambda: tuple(int(v) for v in np.concatenate([c.reshape(-1) for c in model.state.codes]))
    for t in range(300):
        before = all_L[index[key()]]
        assert abs(model.loss() - before) < 1e-12
        rec = mca.step(model, t, 2, 5, 5, 0.0, scan_all=True)
        after = all_L[index[key()]]
        if rec.chosen >= 0:
            assert after < before
    final = key()
    Lf = all_L[index[final]]
    for pos in range(8):  # every one-flip neighbour is no better
        for b in (0, 1):
            nb = list(final)
            nb[pos] = ternary_next(nb[pos], b)
            assert all_L[index[tuple(nb)]] >= Lf - 1e-12
    assert Lf >= all_L.min()


def test_accepted_moves_oppose_gradient():
    """Eq. 9 in the small-perturbation limit: an accepted increment has the
    sign of -dL/dw."""
    X, y, Ws = random_net((8, 6, 4), 80, 31, scale=1.5, density=0.9)
    L, Wt = torch_loss(Ws, X, y, "tanh", requires_grad=True)
    L.backward()
    model = FullMLP(MLPState(Ws), X, y, "tanh")
    L0 = model.loss()
    n_acc = 0
    for t in range(400):
        c = model.candidate(3, 3, t, 0, 1e-4)
        g = Wt[c.layer].grad[c.j, c.i].item()
        if abs(g) < 1e-3 or c.d == 0:
            continue
        if mca.accepts(model.eval(c) - L0, False):
            n_acc += 1
            assert np.sign(float(c.d)) == -np.sign(g)
    assert n_acc > 50


def test_batched_step_equals_sequential_scan_with_drop():
    X, y, Ws = random_net((10, 8, 4), 64, 41, scale=1.0)
    K, T, seed, tag, delta = 5, 80, 13, 2, 0.3
    batched = IncrementalMLP(MLPState(Ws), X, y, "tanh")
    mca.run(batched, 0, T, K, seed, tag, delta, scan_all=False)
    seq = FullMLP(MLPState(Ws), X, y, "tanh")
    for t in range(T):
        for k in range(K):
            c = seq.candidate(seed, tag, t, k, delta)
            Lk = seq.eval(c)
            if Lk < seq.loss():
                seq.commit(c, Lk)
                break  # the rest of step t is dropped
    for a, b in zip(batched.state.weights, seq.state.weights):
        np.testing.assert_array_equal(a, b)


def test_scan_all_and_first_improver_agree():
    X, y, Ws = random_net((10, 8, 4), 64, 43)
    a = IncrementalMLP(MLPState(Ws), X, y, "tanh")
    b = IncrementalMLP(MLPState(Ws), X, y, "tanh")
    ra = mca.run(a, 0, 50, 6, 1, 1, 0.2, scan_all=True)
    rb = mca.run(b, 0, 50, 6, 1, 1, 0.2, scan_all=False)
    assert [r.chosen for r in ra] == [r.chosen for r in rb]
    for u, v in zip(a.state.weights, b.state.weights):
        np.testing.assert_array_equal(u, v)


@pytest.mark.parametrize("beta,dL", [(50.0, 0.01), (200.0, 0.004), (10.0, 0.2), (1e3, 1e-3)])
def test_metropolis_acceptance_frequency(beta, dL):
    """Eq. 7: a candidate with change dL > 0 passes with probability
    exp(-beta dL); over 40,000 candidates of the stream the frequency is
    within 4.5 sigma of it."""
    n = 40000
    hits = 0
    for m in range(n):
        th = mca.thresholds(9, 1, m // 64, 64, beta)[m % 64] if m % 64 == 0 else None
        if th is None:
            from oracle.philox import accept_uniform
            th = mca.metropolis_threshold(accept_uniform(9, 1, m // 64, m % 64), beta)
        hits += mca.accepts(dL, False, th)
    p = math.exp(-beta * dL)
    sigma = math.sqrt(p * (1 - p) / n)
    assert abs(hits / n - p) <= 4.5 * sigma + 1e-12, (hits / n, p)


def test_metropolis_never_rejects_downhill_or_zero():
    from oracle.philox import accept_uniform
    for t in range(200):
        th = mca.metropolis_threshold(accept_uniform(3, 3, t, 0), 7.0)
        assert th > 0
        assert mca.accepts(0.0, False, th) and mca.accepts(-1e-9, False, th)
        assert not mca.accepts(float("nan"), False, th)


def test_metropolis_infinite_beta_is_greedy_with_ties():
    """beta -> infinity: Eq. 7 becomes the greedy rule that accepts dL <= 0
    (min{1, e^0} = 1), so the run equals the ties-accepting greedy run bit
    for bit; the net has dead inputs, so zero changes occur."""
    X, y, Ws = random_net((6, 5, 4), 80, 31, scale=1.0)
    X[:, 4:] = 0.0
    a = IncrementalMLP(MLPState(Ws), X, y, "tanh")
    b = IncrementalMLP(MLPState(Ws), X, y, "tanh")
    ra = mca.run(a, 0, 300, 3, 5, 6, 0.3, accept_ties=True, scan_all=True)
    rb = mca.run(b, 0, 300, 3, 5, 6, 0.3, scan_all=True, beta=1e300)
    zero_acc = 0
    for p, q in zip(ra, rb):
        assert p.chosen == q.chosen
        assert p.dls == q.dls
        zero_acc += p.chosen >= 0 and p.dls[p.chosen] == 0.0
    assert zero_acc > 0
    for u, v in zip(a.state.weights, b.state.weights):
        assert u.tobytes() == v.tobytes()


def test_metropolis_run_climbs_uphill_sometimes():
    """A finite beta accepts some moves with dL > 0, each with U < exp(-beta dL)."""
    from oracle.philox import accept_uniform
    X, y, Ws = random_net((8, 6, 4), 100, 32, scale=1.0)
    model = IncrementalMLP(MLPState(Ws), X, y, "tanh")
    beta = 300.0
    recs = mca.run(model, 0, 400, 2, 11, 12, 0.2, scan_all=True, beta=beta)
    up = 0
    for r in recs:
        if r.chosen >= 0 and r.dls[r.chosen] > 0:
            up += 1
            u = accept_uniform(11, 12, r.t, r.chosen)
            assert u < math.exp(-beta * r.dls[r.chosen])
        for k in range(r.chosen if r.chosen >= 0 else len(r.dls)):
            u = accept_uniform(11, 12, r.t, k)
            assert not (u < math.exp(-beta * r.dls[k]))
    assert up > 0


def test_pruning_moves_zero_the_weight_and_match_definition():
    """Sec. 2.2: a pruning move sets its weight to zero (d = -w); its loss
    change equals the definition; a pure-pruning run only ever zeroes
    weights, never lowers the loss count of zeros, and strictly lowers L on
    every accepted step."""
    X, y, Ws = random_net((9, 7, 5), 120, 41, scale=1.2)
    inc = IncrementalMLP(MLPState(Ws), X, y, "tanh")
    full = FullMLP(MLPState(Ws), X, y, "tanh")
    for t in range(30):
        c = inc.candidate(2, 3, t, 0, 0.1, prune=True)
        assert c.prune and c.d == -Ws[c.layer][c.j, c.i] and inc.state.new_value(c) == 0.0
        a, _ = full.delta(c)
        b, _ = inc.delta(c)
        assert abs(a - b) <= 1e-9 * abs(a) + 2e-15
    ratio0 = mca.remaining_weight_ratio(inc)
    recs = mca.run(inc, 0, 300, 4, 2, 3, 0.1, scan_all=True, n_prune=4)
    acc = [r for r in recs if r.chosen >= 0]
    assert acc and all(r.L_after < r.L_before for r in acc)
    assert all(r.cands[r.chosen].prune for r in acc)
    total = sum(w.size for w in Ws)
    assert round(mca.remaining_weight_ratio(inc) * total) == round(ratio0 * total) - len(acc)
    fresh = FullMLP(MLPState(inc.state.weights), X, y, "tanh")
    assert abs(fresh.loss() - inc.loss()) <= 1e-12


def test_mixed_pruning_puts_pruning_first():
    """n_prune < K: candidates 0 .. n_prune-1 prune, the rest mutate; the
    first passing candidate in that order wins (pruning preferred)."""
    X, y, Ws = random_net((9, 7, 5), 120, 43, scale=1.2)
    inc = IncrementalMLP(MLPState(Ws), X, y, "tanh")
    recs = mca.run(inc, 0, 200, 6, 4, 5, 0.2, scan_all=True, n_prune=2)
    kinds = set()
    for r in recs:
        assert [c.prune for c in r.cands] == [True, True, False, False, False, False]
        if r.chosen >= 0:
            kinds.add(r.cands[r.chosen].prune)
            assert all(d >= 0 for d in r.dls[:r.chosen])
    assert kinds == {True, False}


def test_minibatch_windows_and_means():
    """Sec. 2.2's minibatch: step t's window e = t // period covers samples
    (e size + m) mod N; a candidate's change is the mean over the window of
    its samples' changes; the committed loss stays the mean over all."""
    m = mca.minibatch(0, 10, 4, 3)
    assert list(np.flatnonzero(m)) == [0, 1, 2, 3]
    assert list(np.flatnonzero(mca.minibatch(2, 10, 4, 3))) == [0, 1, 2, 3]
    assert list(np.flatnonzero(mca.minibatch(3, 10, 4, 3))) == [4, 5, 6, 7]
    assert list(np.flatnonzero(mca.minibatch(6, 10, 4, 3))) == [0, 1, 8, 9]
    assert mca.minibatch(5, 10, 0, 1) is None
    X, y, Ws = random_net((9, 7, 5), 60, 47, scale=1.2)
    inc = IncrementalMLP(MLPState(Ws), X, y, "tanh")
    full = FullMLP(MLPState(Ws), X, y, "tanh")
    c = inc.candidate(1, 2, 0, 0, 0.3)
    rows, dl, _ = inc.sample_changes(c)
    per = np.zeros(60)
    per[rows] = dl
    inc.subset = mca.minibatch(4, 60, 25, 2)
    d, _ = inc.delta(c)
    inc.subset = None
    assert abs(d - per[mca.minibatch(4, 60, 25, 2)].mean()) <= 1e-15
    # a run with minibatches: decisions on the window, L over every sample
    recs = mca.run(inc, 0, 100, 4, 1, 2, 0.3, scan_all=True, subset=(25, 2))
    assert any(r.chosen >= 0 for r in recs)
    fresh = FullMLP(MLPState(inc.state.weights), X, y, "tanh")
    assert abs(fresh.loss() - inc.loss()) <= 1e-12
