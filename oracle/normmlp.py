"""fp64 oracle of the deep MLPs of Sec. 2.1: biases, layer normalization and
the layer-sticky proposal schedule.

Network.  Each layer l has an augmented weight matrix [W_l | b_l] of shape
(n_{l+1}, n_l + 1): row j holds unit j's incoming weights and, in the last
column, its bias (a bias is a weight on a constant input 1).  The local field
is z_l = W_l a_{l-1} + b_l.  A hidden field is normalized over the units of
its layer, sample by sample, with no gain or bias of its own,
h = (z - mean(z)) / sqrt(var(z) + eps) (population variance), and
a_l = phi(h); without normalization h = z.  The logits z_L take no
normalization.  The loss is the average cross-entropy (Eq. 2).

Reading of the paper: it normalizes the hidden layers of its deep nets and
counts their parameters as weights plus one bias per unit (its parameter
totals for depths 5, 8, 11 and 21 at width 256 match that count and leave no
room for normalization gains), so the normalization carries no parameters;
it is placed on the summed input of each hidden unit, before the transfer
function.  The candidate's parameter index runs over the augmented matrices
in order (layer by layer, row by row, the bias last in each row).

Layer-sticky schedule (Sec. 2.1, current-layer caching): steps are grouped
in blocks of `sticky` consecutive steps; block e = floor(t / sticky) draws its
layer from word 0 of the Philox block at counter (e, 0, 0, 1),
l = floor(w0 L / 2^64), and every candidate of those steps mutates a
parameter of layer l, uniformly (its own block (t, k, 0, 0), word 0).

Evaluation of a candidate in layer l: the changed field column (or, for a
bias, the whole column: its input is 1) and every later layer are recomputed
from the cached input of layer l; each sample's loss change comes from the
logit change by the exact identity of ``mlp.ce_change``.  The commit
recomputes the caches.  This is the definition restricted to the part of
the net a change can reach; it is pinned against PyTorch's fp64 layer_norm
and linear ops on the whole net.

All arithmetic is float64 from fp32 parameters.
"""
from __future__ import annotations

import numpy as np

from .mlp import ce_change, mean_ce, phi, softmax
from .philox import Candidate, decode, draw, mulhi64, philox4x64


def layer_norm(z, eps: float):
    """(z - mean) / sqrt(var + eps) over the last axis (population variance)."""
    mu = z.mean(axis=1, keepdims=True)
    c = z - mu
    var = (c * c).mean(axis=1, keepdims=True)
    return c / np.sqrt(var + eps)


def sticky_layer(seed: int, tag: int, block: int, n_layers: int) -> int:
    """The layer of step block `block`: word 0 of counter (block, 0, 0, 1)."""
    return mulhi64(philox4x64((block, 0, 0, 1), (seed, tag))[0], n_layers)


class NormMLP:
    """Deep MLP with optional biases (augmented weights) and optional layer
    normalization of the hidden fields; caches every layer's input."""

    def __init__(self, weights, X, y, act: str, gamma: float = 1.0, bias: bool = True,
                 ln: bool = True, eps: float = 1e-5, sticky: int = 0):
        self.weights = [np.array(w, dtype=np.float32, copy=True) for w in weights]
        self.X = np.asarray(X, dtype=np.float32).astype(np.float64)
        self.y = np.asarray(y, dtype=np.int64)
        self.act, self.gamma = act, float(gamma)
        self.bias, self.ln, self.eps = bias, ln, float(eps)
        self.sticky = int(sticky)
        L = len(self.weights)
        for l, w in enumerate(self.weights):
            n_in = self.X.shape[1] if l == 0 else self.weights[l - 1].shape[0]
            assert w.shape[1] == n_in + (1 if bias else 0), (l, w.shape)
        self.L = L
        self.subset = None  # every sample
        self.refresh()

    # ---------------------------------------------------------------- forward
    @property
    def shapes(self):
        return [w.shape for w in self.weights]

    @property
    def widths(self):
        return (self.X.shape[1],) + tuple(w.shape[0] for w in self.weights)

    def _field(self, l, a, W64=None):
        W = self.weights[l].astype(np.float64) if W64 is None else W64
        if self.bias:
            return a @ W[:, :-1].T + W[:, -1]
        return a @ W.T

    def _act(self, z):
        return phi(layer_norm(z, self.eps) if self.ln else z, self.act, self.gamma)

    def forward_from(self, l, a_in, weights=None):
        """Fields of layers l .. L-1 from the input a_in of layer l."""
        ws = self.weights if weights is None else weights
        Z = []
        a = a_in
        for m in range(l, self.L):
            z = self._field(m, a, ws[m].astype(np.float64))
            Z.append(z)
            if m < self.L - 1:
                a = self._act(z)
        return Z

    def refresh(self):
        self.Z = self.forward_from(0, self.X)
        self.A = [self.X] + [self._act(z) for z in self.Z[:-1]]  # input of each layer
        self._P = softmax(self.Z[-1])
        self._L = mean_ce(self.Z[-1], self.y)

    def loss(self) -> float:
        return self._L

    # ------------------------------------------------------------- candidates
    def new_value(self, c: Candidate) -> np.float32:
        if c.prune:
            return np.float32(0.0)
        return np.float32(self.weights[c.layer][c.j, c.i] + c.d)

    def candidate(self, seed, tag, t, k, delta, mode="weight", prune=False) -> Candidate:
        """Candidate k of step t (Eq. 1) over the augmented matrices; mode
        "sticky" takes the layer of the step's block (Sec. 2.1)."""
        words = draw(seed, tag, t, k)
        if mode == "sticky":
            l = sticky_layer(seed, tag, t // self.sticky, self.L)
            size = int(np.prod(self.shapes[l]))
            off = mulhi64(words[0], size)
            j, i = divmod(off, self.shapes[l][1])
            flat = sum(int(np.prod(s)) for s in self.shapes[:l]) + off
            c = Candidate(flat, l, j, i, np.float32(np.float32(delta) * _unit_r(words[2])))
        else:
            c = decode(words, self.shapes, delta, mode)
        if prune:
            w = self.weights[c.layer][c.j, c.i]
            c = Candidate(c.flat, c.layer, c.j, c.i, np.float32(np.float32(0.0) - w), 0, True)
        return c

    def with_candidate(self, c):
        ws = list(self.weights)
        wl = ws[c.layer].copy()
        wl[c.j, c.i] = self.new_value(c)
        ws[c.layer] = wl
        return ws

    # ------------------------------------------------------------- evaluation
    def sample_changes(self, c: Candidate):
        """(per-sample loss changes, first-order sizes) on every sample: the
        layers from c.layer on are recomputed from the cached input."""
        l = c.layer
        ws = self.with_candidate(c)
        Z1 = self.forward_from(l, self.A[l], ws)
        dz = Z1[-1] - self.Z[-1]
        # the absolute terms of the logit changes: the last layer's input change
        # through |W_{L-1}| (and the changed weight itself when it is that layer's)
        if l == self.L - 1:
            a_in = self.A[l][:, c.i] if c.i < self.A[l].shape[1] else np.ones(len(dz))
            absz = np.abs(dz)
            absz[:, c.j] = np.abs(float(self.new_value(c)) - float(self.weights[l][c.j, c.i])) * np.abs(a_in)
        else:
            a1 = self._act(Z1[-2])
            da = a1 - self.A[-1]
            Wl = np.abs(ws[-1].astype(np.float64))
            absz = np.abs(da) @ (Wl[:, :-1] if self.bias else Wl).T
        return ce_change(self._P, dz, self.y, absz)

    def delta(self, c: Candidate):
        """(dL, A) of candidate c (Eq. 2 difference), over the minibatch when
        one is set."""
        dl, mag = self.sample_changes(c)
        if self.subset is not None:
            n = int(self.subset.sum())
            return float(dl[self.subset].sum()) / n, float(mag[self.subset].sum()) / n
        N = self.X.shape[0]
        return float(dl.sum()) / N, float(mag.sum()) / N

    def commit(self, c: Candidate, loss_after: float):
        self.weights[c.layer][c.j, c.i] = self.new_value(c)
        self.refresh()

    @property
    def state(self):
        return self

    def state_weights(self):
        return self.weights


def _unit_r(w2: int) -> np.float32:
    from .philox import unit_r
    return unit_r(w2)
