"""fp64 oracle of the bias-free MLP and its loss.

Network (Sec. 3.6 notation): z_l = W_l a_{l-1}, a_l = phi(z_l) for hidden
layers, a_0 = x, and the last local field z_L is the logit vector.  phi is
tanh or the Gaussian exp(-gamma z^2) (Sec. 2).  The loss is the average
cross-entropy over the full sample set (Sec. 2; Eq. 2 with R(W) = 0).

Two evaluators of the loss after a single-weight mutation:

* ``FullMLP``: the definition -- rebuild the weights with the one entry
  replaced and run the whole forward pass again.
* ``IncrementalMLP``: the decomposition of Sec. 2.4 -- keep the local fields
  of every layer from the last accepted state; a change of W_l[j, i] moves
  only column j of z_l (by d * a_{l-1}[:, i]); that changes a_l[:, j], which
  moves z_{l+1} by a rank-1 term (the fan-out column W_{l+1}[:, j], the O(N)
  work per sample of Sec. 2.4); every later layer is recomputed densely.
  Pinned against ``FullMLP`` to rounding.

Arrays are sample-major (N x units) here; all arithmetic is float64.
"""
from __future__ import annotations

import numpy as np

from .philox import Candidate, decode, draw


def phi(z, act: str, gamma: float = 1.0):
    """Transfer function (Sec. 2): tanh, or the Gaussian exp(-gamma z^2)."""
    if act == "tanh":
        return np.tanh(z)
    if act == "gauss":
        return np.exp(-gamma * z * z)
    raise ValueError(act)


def per_sample_ce(logits, y):
    """Cross-entropy of each sample: logsumexp(z) - z[y] (max-shifted, natural log)."""
    m = logits.max(axis=1, keepdims=True)
    lse = m[:, 0] + np.log(np.exp(logits - m).sum(axis=1))
    return lse - logits[np.arange(logits.shape[0]), y]


def mean_ce(logits, y) -> float:
    """Average cross-entropy over all samples (Eq. 2, R = 0)."""
    return float(np.mean(per_sample_ce(logits, y)))


def forward_fields(weights64, X64, act, gamma):
    """All local fields [z_1, ..., z_L] of the forward pass (Sec. 3.6)."""
    Z = []
    a = X64
    for l, W in enumerate(weights64):
        z = a @ W.T
        Z.append(z)
        if l < len(weights64) - 1:
            a = phi(z, act, gamma)
    return Z


class MLPState:
    """Committed fp32 state: weights, and for discrete weights the int8 codes
    with per-layer fp32 scales (weight = code * scale)."""

    def __init__(self, weights, codes=None, scales=None):
        self.weights = [np.array(w, dtype=np.float32, copy=True) for w in weights]
        self.codes = None if codes is None else [np.array(c, dtype=np.int8, copy=True) for c in codes]
        self.scales = None if scales is None else [np.float32(s) for s in scales]

    @property
    def shapes(self):
        return [w.shape for w in self.weights]

    def new_value(self, c: Candidate) -> np.float32:
        """The proposed fp32 value: fl32(w + d) (Eq. 1) or code' * scale (Eq. 12)."""
        if self.codes is not None:
            return np.float32(np.float32(c.code) * self.scales[c.layer])
        return np.float32(self.weights[c.layer][c.j, c.i] + c.d)

    def apply(self, c: Candidate):
        w = self.new_value(c)
        self.weights[c.layer][c.j, c.i] = w
        if self.codes is not None:
            self.codes[c.layer][c.j, c.i] = c.code


class _Base:
    def __init__(self, state: MLPState, X, y, act: str, gamma: float = 1.0):
        self.state = state
        self.X = np.asarray(X, dtype=np.float32).astype(np.float64)
        self.y = np.asarray(y, dtype=np.int64)
        self.act = act
        self.gamma = float(gamma)

    def candidate(self, seed, tag, t, k, delta, mode="weight") -> Candidate:
        return decode(draw(seed, tag, t, k), self.state.shapes, delta, mode,
                      self.state.codes, self.state.scales)


class FullMLP(_Base):
    """Loss by full recomputation: the definition."""

    def loss_of(self, weights32) -> float:
        W64 = [w.astype(np.float64) for w in weights32]
        return mean_ce(forward_fields(W64, self.X, self.act, self.gamma)[-1], self.y)

    def loss(self) -> float:
        if getattr(self, "_L", None) is None:
            self._L = self.loss_of(self.state.weights)
        return self._L

    def eval(self, c: Candidate) -> float:
        """L(W') with W' = W except entry (layer, j, i) := its proposed value."""
        ws = list(self.state.weights)
        wl = ws[c.layer].copy()
        wl[c.j, c.i] = self.state.new_value(c)
        ws[c.layer] = wl
        return self.loss_of(ws)

    def commit(self, c: Candidate, loss_after: float):
        """Apply c; the loss of the new state is the one just evaluated for it
        (the same deterministic recomputation of the same weights)."""
        self.state.apply(c)
        self._L = float(loss_after)


class IncrementalMLP(_Base):
    """Loss after a mutation from cached local fields (Sec. 2.4)."""

    def __init__(self, state, X, y, act, gamma=1.0):
        super().__init__(state, X, y, act, gamma)
        self.refresh()

    def refresh(self):
        W64 = [w.astype(np.float64) for w in self.state.weights]
        self.Z = forward_fields(W64, self.X, self.act, self.gamma)
        self.L = mean_ce(self.Z[-1], self.y)

    def loss(self) -> float:
        return self.L

    def _act_in(self, l, i):
        """Column i of the input of layer l: x for the first layer, phi(z_{l-1}) otherwise."""
        if l == 0:
            return self.X[:, i]
        return phi(self.Z[l - 1][:, i], self.act, self.gamma)

    def _propagate(self, c: Candidate):
        """Fields that change under candidate c.

        Returns (new column j of z_l, {m: new z_m for every later layer m}).
        """
        l, j, i = c.layer, c.j, c.i
        nL = len(self.Z)
        d = np.float64(self.state.new_value(c)) - np.float64(self.state.weights[l][j, i])
        col = self.Z[l][:, j] + d * self._act_in(l, i)
        later = {}
        if l == nL - 1:
            return col, later
        da = phi(col, self.act, self.gamma) - phi(self.Z[l][:, j], self.act, self.gamma)
        Wn = self.state.weights[l + 1].astype(np.float64)
        z = self.Z[l + 1] + np.outer(da, Wn[:, j])
        later[l + 1] = z
        for m in range(l + 2, nL):
            z = phi(z, self.act, self.gamma) @ self.state.weights[m].astype(np.float64).T
            later[m] = z
        return col, later

    def _logits(self, c: Candidate, col, later):
        nL = len(self.Z)
        if c.layer == nL - 1:
            z = self.Z[-1].copy()
            z[:, c.j] = col
            return z
        return later[nL - 1]

    def eval(self, c: Candidate) -> float:
        col, later = self._propagate(c)
        return mean_ce(self._logits(c, col, later), self.y)

    def commit(self, c: Candidate, loss_after: float):
        col, later = self._propagate(c)
        self.Z[c.layer][:, c.j] = col
        for m, z in later.items():
            self.Z[m] = z
        self.state.apply(c)
        self.L = mean_ce(self.Z[-1], self.y)
