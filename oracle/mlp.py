"""fp64 oracle of the bias-free MLP and its loss.

Network (Sec. 3.6 notation): z_l = W_l a_{l-1}, a_l = phi(z_l) for hidden
layers, a_0 = x, and the last local field z_L is the logit vector.  phi is
tanh, ReLU max(0, z) or the Gaussian exp(-gamma z^2) (Sec. 2).  The loss is the average
cross-entropy over the full sample set (Sec. 2; Eq. 2 with R(W) = 0).

Two evaluators of the loss after a single-weight mutation:

* ``FullMLP``: the definition -- rebuild the weights with the one entry
  replaced and run the whole forward pass again.
* ``IncrementalMLP``: the decomposition of Sec. 2.4 -- keep the local fields
  of every layer from the last accepted state; a change of W_l[j, i] moves
  only column j of z_l (by d * a_{l-1}[:, i]); that changes a_l[:, j], which
  moves z_{l+1} by a rank-1 term (the fan-out column W_{l+1}[:, j], the O(N)
  work per sample of Sec. 2.4); every later layer changes densely.  It
  carries the *changes* of the fields from layer to layer and forms the
  loss change from them (``ce_change``), so that a loss change far below
  the loss itself keeps its relative precision: deep nets with small
  initial weights change the loss by 1e-11 per mutation, where L' - L of two
  fp64 totals near 2.3 would keep only four digits.  Pinned against
  ``FullMLP`` (where the change is large) and against a long-double full
  recomputation (where it is small).

Both also evaluate a channel mutation (Sec. 2.3): one weight per layer on an
input-to-output path changes at once.  The definition replaces all of them
and recomputes; the incremental form moves column units[1] of the first
field, then every later field by the dense change of its input plus the
point change of its own path weight (W'_m a'_m - W_m a_m =
W_m (a'_m - a_m) + (w'_m - w_m) a'_m[units[m]] at unit units[m + 1]).

Arrays are sample-major (N x units) here; all arithmetic is float64.
"""
from __future__ import annotations

import numpy as np

from .philox import Candidate, Channel, channel_words, decode, decode_channel, draw


def phi(z, act: str, gamma: float = 1.0):
    """Transfer function (Sec. 2): tanh, ReLU max(0, z), or the Gaussian exp(-gamma z^2)."""
    if act == "tanh":
        return np.tanh(z)
    if act == "relu":
        return np.maximum(z, 0.0)
    if act == "gauss":
        return np.exp(-gamma * z * z)
    raise ValueError(act)


def dphi(z, dz, act: str, gamma: float = 1.0):
    """phi(z + dz) - phi(z) without cancellation, from two textbook identities:
    tanh a - tanh b = sinh(a - b) / (cosh a cosh b), and
    exp(-g a^2) - exp(-g b^2) = exp(-g b^2) expm1(-g (a - b)(a + b)).
    For ReLU the change is dz itself where both fields are positive, zero
    where neither is, and the one non-zero activation where they straddle 0.
    Exactly zero where dz is zero."""
    if act == "tanh":
        return np.sinh(dz) / (np.cosh(z) * np.cosh(z + dz))
    if act == "relu":
        zn = z + dz
        return np.where((z > 0) & (zn > 0), dz, np.maximum(zn, 0.0) - np.maximum(z, 0.0))
    if act == "gauss":
        arg = -gamma * dz * (2.0 * z + dz)
        with np.errstate(over="ignore", invalid="ignore"):
            small = np.exp(-gamma * z * z) * np.expm1(arg)
        # a move far out of a saturated tail: no cancellation to avoid
        return np.where(arg > 30.0, phi(z + dz, act, gamma) - phi(z, act, gamma), small)
    raise ValueError(act)


def dphi_dz(z, act: str, gamma: float = 1.0):
    """phi'(z) (ReLU: the step function, 0 at z = 0)."""
    if act == "tanh":
        t = np.tanh(z)
        return 1.0 - t * t
    if act == "relu":
        return (np.asarray(z) > 0).astype(np.float64)
    return -2.0 * gamma * z * np.exp(-gamma * z * z)


def softmax(logits):
    """Row-wise softmax (max-shifted)."""
    e = np.exp(logits - logits.max(axis=1, keepdims=True))
    return e / e.sum(axis=1, keepdims=True)


def ce_change(p, dz, y, adz=None):
    """Change of each sample's cross-entropy when its logits move by dz (Eq. 2):
    l(z + dz) - l(z) = log(sum_c p_c e^{dz_c}) - dz_y
                     = log1p(sum_c p_c expm1(dz_c)) - dz_y,  p = softmax(z).
    Returns (per-sample change, per-sample size of its first-order terms
    sum_c p_c a_c + a_y, the scale of the rounding of any evaluation), with
    a = |dz|, or `adz` when given: the sums of the absolute terms each logit
    change is made of (a sum of many terms of both signs rounds in
    proportion to those, not to its result)."""
    rows = np.arange(dz.shape[0])
    dl = np.log1p((p * np.expm1(dz)).sum(axis=1)) - dz[rows, y]
    a = np.abs(dz) if adz is None else adz
    mag = (p * a).sum(axis=1) + a[rows, y]
    return dl, mag


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
        """The proposed fp32 value: fl32(w + d) (Eq. 1), code' * scale (Eq. 12),
        or zero for a pruning move (Sec. 2.2, d = -w)."""
        if c.prune:
            return np.float32(0.0)
        if self.codes is not None:
            return np.float32(np.float32(c.code) * self.scales[c.layer])
        return np.float32(self.weights[c.layer][c.j, c.i] + c.d)

    def apply_channel(self, ch: Channel):
        for m, w in enumerate(ch.w_new):
            self.weights[m][ch.units[m + 1], ch.units[m]] = np.float32(w)

    def with_channel(self, ch: Channel):
        """The weight list with the channel's entries replaced (copies of the
        changed layers only)."""
        ws = list(self.weights)
        for m, w in enumerate(ch.w_new):
            wl = ws[m].copy()
            wl[ch.units[m + 1], ch.units[m]] = np.float32(w)
            ws[m] = wl
        return ws

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

    @property
    def widths(self):
        ws = self.state.weights
        return (ws[0].shape[1],) + tuple(w.shape[0] for w in ws)

    def candidate(self, seed, tag, t, k, delta, mode="weight", prune=False):
        """Candidate k of step t; with prune, the same draw's weight is set to
        zero instead (d = -w, ternary code 0).  Modes "channel_redraw" and
        "channel_zero" draw a channel mutation (Sec. 2.3) instead."""
        if mode.startswith("channel_"):
            L = len(self.state.weights)
            return decode_channel(channel_words(seed, tag, t, k, 2 * L + 1), self.widths,
                                  mode[len("channel_"):])
        c = decode(draw(seed, tag, t, k), self.state.shapes, delta, mode,
                   self.state.codes, self.state.scales)
        if prune:
            w = self.state.weights[c.layer][c.j, c.i]
            c = Candidate(c.flat, c.layer, c.j, c.i, np.float32(np.float32(0.0) - w), 0, True)
        return c


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

    def delta(self, c):
        """(L(W') - L(W), A): the definition of the loss change, and the size
        A of its first-order terms over the logit change (see ce_change).
        c is a single-parameter Candidate or a Channel."""
        if isinstance(c, Channel):
            ws = self.state.with_channel(c)
        else:
            ws = list(self.state.weights)
            wl = ws[c.layer].copy()
            wl[c.j, c.i] = self.state.new_value(c)
            ws[c.layer] = wl
        if getattr(self, "_z0", None) is None:  # the committed logits, kept until a commit
            W0 = [w.astype(np.float64) for w in self.state.weights]
            self._z0 = forward_fields(W0, self.X, self.act, self.gamma)[-1]
        z0 = self._z0
        W1 = [w.astype(np.float64) for w in ws]
        z1 = forward_fields(W1, self.X, self.act, self.gamma)[-1]
        _, mag = ce_change(softmax(z0), z1 - z0, self.y)
        return mean_ce(z1, self.y) - mean_ce(z0, self.y), float(np.mean(mag))

    def commit(self, c: Candidate, loss_after: float):
        """Apply c; the loss of the new state is the one just evaluated for it
        (the same deterministic recomputation of the same weights)."""
        if isinstance(c, Channel):
            self.state.apply_channel(c)
        else:
            self.state.apply(c)
        self._L = float(loss_after)
        self._z0 = None


class IncrementalMLP(_Base):
    """Loss after a mutation from cached local fields (Sec. 2.4)."""

    def __init__(self, state, X, y, act, gamma=1.0):
        super().__init__(state, X, y, act, gamma)
        self.refresh()

    def refresh(self):
        W64 = [w.astype(np.float64) for w in self.state.weights]
        self.Z = forward_fields(W64, self.X, self.act, self.gamma)
        self.L = mean_ce(self.Z[-1], self.y)
        self._P = None

    def loss(self) -> float:
        return self.L

    def _act_in(self, l, i):
        """Column i of the input of layer l: x for the first layer, phi(z_{l-1}) otherwise."""
        if l == 0:
            return self.X[:, i]
        return phi(self.Z[l - 1][:, i], self.act, self.gamma)

    def _changes(self, c: Candidate):
        """The changes of the local fields under candidate c (Sec. 2.4), on the
        samples whose field moves (rows: every other sample has exactly zero
        change in every later layer, since dphi(z, 0) = 0):
        (rows, change of column j of z_l there, {m: change of z_m there})."""
        l, j, i = c.layer, c.j, c.i
        nL = len(self.Z)
        d = np.float64(self.state.new_value(c)) - np.float64(self.state.weights[l][j, i])
        dcol = d * self._act_in(l, i)
        rows = np.flatnonzero(dcol)
        dcol = dcol[rows]
        later = {}
        if l == nL - 1:
            return rows, dcol, later
        # the activation change of unit j, then the rank-1 term through the
        # fan-out column W_{l+1}[:, j]
        da = dphi(self.Z[l][rows, j], dcol, self.act, self.gamma)
        dz = np.outer(da, self.state.weights[l + 1][:, j].astype(np.float64))
        later[l + 1] = dz
        # every later layer: dz_m = (phi(z_{m-1} + dz_{m-1}) - phi(z_{m-1})) W_m^T
        for m in range(l + 2, nL):
            da = dphi(self.Z[m - 1][rows], dz, self.act, self.gamma)
            Wm = self.state.weights[m].astype(np.float64)
            dz = da @ Wm.T
            later[m] = dz
            if m == nL - 1:  # the absolute terms of the logit sums
                later["abs"] = np.abs(da) @ np.abs(Wm).T
        return rows, dcol, later

    def _logit_change(self, c: Candidate, rows, dcol, later):
        nL = len(self.Z)
        if c.layer == nL - 1:
            dz = np.zeros((len(rows), self.Z[-1].shape[1]))
            dz[:, c.j] = dcol
            return dz
        return later[nL - 1]

    def _softmax(self):
        """softmax of the cached logits (kept until the next commit)."""
        if getattr(self, "_P", None) is None:
            self._P = softmax(self.Z[-1])
        return self._P

    def _fwd_terms(self, l, unit, rows):
        """sum_k |W_l[unit, k] a_{l-1}[n, k]| on the given rows: the size of
        the terms of unit's local field, which an fp32 forward pass rounds in
        proportion to."""
        a = np.abs(self.X[rows]) if l == 0 else np.abs(phi(self.Z[l - 1][rows], self.act, self.gamma))
        return a @ np.abs(self.state.weights[l][unit].astype(np.float64))

    def _cache_sensitivity(self, c: Candidate, rows, dcol):
        """Per row, the relative change of the sample's loss change per unit
        of forward rounding (u * field-term size) in the two cached fields the
        candidate reads: its input a_{l-1}[n, i] = phi(z_{l-1}[n, i]) (the loss
        change is linear in it) and, for a hidden unit, its own field z_l[n, j]
        (through phi(z + dz) - phi(z))."""
        l, j, i = c.layer, c.j, c.i
        sens = np.zeros(len(rows))
        if l >= 1:
            z_in = self.Z[l - 1][rows, i]
            a_in = phi(z_in, self.act, self.gamma)
            sens += np.abs(dphi_dz(z_in, self.act, self.gamma)) * self._fwd_terms(l - 1, i, rows) / np.abs(a_in)
        if l < len(self.Z) - 1:
            z = self.Z[l][rows, j]
            da = dphi(z, dcol, self.act, self.gamma)
            slope = np.abs(dphi_dz(z + dcol, self.act, self.gamma) - dphi_dz(z, self.act, self.gamma))
            with np.errstate(divide="ignore", invalid="ignore"):
                own = np.where(da != 0, slope / np.abs(da), 0.0)
            sens += own * self._fwd_terms(l, j, rows)
        return sens

    def sample_changes(self, c: Candidate):
        """(rows, per-sample loss changes there, their first-order sizes there);
        every other sample's change is zero.  The sizes add to the terms of
        the change itself (ce_change) its sensitivity to the rounding of the
        cached fields it reads (_cache_sensitivity)."""
        rows, dcol, later = self._changes(c)
        dl, mag = ce_change(self._softmax()[rows], self._logit_change(c, rows, dcol, later),
                            self.y[rows], later.get("abs"))
        # an fp32 dot product rounds its result by about 2^-24 times the sum
        # of its terms' sizes: 1/16 of the size unit the evaluation's own
        # arithmetic is counted in (see ce_change's callers)
        mag = mag + np.abs(dl) * self._cache_sensitivity(c, rows, dcol) / 16.0
        return rows, dl, mag

    def _channel_changes(self, ch: Channel):
        """Field changes under channel ch on every sample (Sec. 2.3): {m: the
        change of z_m (for the first layer: of column units[1] only)}, and
        the absolute terms of the logit changes."""
        W = self.state.weights
        nL = len(self.Z)
        u = ch.units
        d = [np.float64(ch.w_new[m]) - np.float64(W[m][u[m + 1], u[m]]) for m in range(nL)]
        out = {}
        col = d[0] * self.X[:, u[0]]  # column u[1] of the first field
        out[0] = col
        if nL == 1:
            dz = np.zeros(self.Z[0].shape)
            dz[:, u[1]] = col
            out["logits"], out["abs"] = dz, np.abs(dz)
            return out
        # the first layer's new activation of the path unit and its change
        zc = self.Z[0][:, u[1]]
        a_path = phi(zc + col, self.act, self.gamma)
        da_col = dphi(zc, col, self.act, self.gamma)
        da = None  # dense activation change of the layer before (m >= 2)
        for m in range(1, nL):
            Wm = W[m].astype(np.float64)
            if m == 1:
                dz = np.outer(da_col, Wm[:, u[1]])
                absz = np.outer(np.abs(da_col), np.abs(Wm[:, u[1]]))
            else:
                dz = da @ Wm.T
                absz = np.abs(da) @ np.abs(Wm).T if m == nL - 1 else None
            point = d[m] * a_path
            dz[:, u[m + 1]] += point
            out[m] = dz
            if m == nL - 1:
                absz[:, u[m + 1]] += np.abs(point)
                out["logits"], out["abs"] = dz, absz
                return out
            z = self.Z[m]
            da = dphi(z, dz, self.act, self.gamma)
            a_path = phi(z[:, u[m + 1]] + dz[:, u[m + 1]], self.act, self.gamma)

    def channel_sample_changes(self, ch: Channel):
        """(per-sample loss changes, their first-order sizes) of channel ch."""
        out = self._channel_changes(ch)
        return ce_change(self._softmax(), out["logits"], self.y, out["abs"])

    # minibatch (Sec. 2.2): a boolean mask over the samples, or None for all
    subset = None

    def delta(self, c: Candidate):
        """(dL, A): the loss change of candidate c (Eq. 2 difference), from the
        field changes, and the mean size A of its first-order terms; over the
        current minibatch when one is set.  c may be a Channel (Sec. 2.3)."""
        if isinstance(c, Channel):
            assert self.subset is None, "channel mutations score every sample"
            dl, mag = self.channel_sample_changes(c)
            N = self.X.shape[0]
            return float(dl.sum()) / N, float(mag.sum()) / N
        rows, dl, mag = self.sample_changes(c)
        if self.subset is not None:
            keep = self.subset[rows]
            n = int(self.subset.sum())
            return float(dl[keep].sum()) / n, float(mag[keep].sum()) / n
        N = self.X.shape[0]
        return float(dl.sum()) / N, float(mag.sum()) / N

    def eval(self, c: Candidate) -> float:
        return self.L + self.delta(c)[0]

    def commit(self, c: Candidate, loss_after: float):
        """Apply c: every cached field moves by its change; the committed loss
        moves by the candidate's loss change (loss_after = L + dL)."""
        if isinstance(c, Channel):
            out = self._channel_changes(c)
            dl, _ = ce_change(self._softmax(), out["logits"], self.y)
            self.Z[0][:, c.units[1]] += out[0]
            for m in range(1, len(self.Z)):
                self.Z[m] += out[m]
            self._P = None
            self.state.apply_channel(c)
            self.L = self.L + float(dl.sum()) / self.X.shape[0]
            return
        rows, dcol, later = self._changes(c)
        dl, _ = ce_change(self._softmax()[rows], self._logit_change(c, rows, dcol, later),
                          self.y[rows])
        dL = float(dl.sum()) / self.X.shape[0]  # the loss over every sample
        self.Z[c.layer][rows, c.j] += dcol
        for m, dz in later.items():
            if m != "abs":
                self.Z[m][rows] += dz
        self._P = None
        self.state.apply(c)
        self.L = self.L + dL
