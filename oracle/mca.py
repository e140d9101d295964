"""Greedy mutation-selection loop of the oracle (Eq. 1, Eq. 5, Eq. 6).

One step t scores candidates k = 0..K-1 of the counter-based stream against the
same committed state W_t, in stream order.  The first candidate whose loss
change dL_k = L(W_t + dW_k) - L(W_t) passes the acceptance test is committed;
later candidates of the step are discarded.  With K = 1 this is the paper's
sequential rule (mutate one parameter, keep it if the loss does not increase,
otherwise retry).  Acceptance (Eq. 6 with the ties reading): dL < 0 by default,
dL <= 0 when ties are accepted.  A NaN or infinite dL is never accepted.

The Metropolis rule (Eq. 7) accepts with probability min{1, exp(-beta dL)}:
with the candidate's own uniform U (philox.accept_uniform), U < exp(-beta dL)
holds exactly when dL < theta = -ln(U) / beta, so it is the greedy test
against a per-candidate threshold theta > 0 (a zero change always passes).

Each candidate's loss change comes from the model's ``delta`` (the
difference form of the incremental oracle, the definition for the full
one); the decision is taken on dL itself, never on L + dL - L.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

from .philox import accept_uniform


def accepts(dL: float, accept_ties: bool, theta: float = 0.0) -> bool:
    """Selection test: Eq. 6 (strict unless ties are accepted) when theta is
    0, else the Metropolis test of Eq. 7 written as dL < theta."""
    if not math.isfinite(dL):
        return False
    if theta > 0.0:
        return dL < theta
    return dL <= 0.0 if accept_ties else dL < 0.0


def metropolis_threshold(u: float, beta: float) -> float:
    """theta with (U < exp(-beta dL)) == (dL < theta): -ln(U) / beta (+inf at U = 0)."""
    return math.inf if u == 0.0 else -math.log(u) / beta


def minibatch(t: int, N: int, size: int, period: int):
    """The samples whose loss changes step t averages (Sec. 2.2's minibatch;
    None = all): window e = floor(t / period) covers the `size` samples
    n = (e size + m) mod N, m < size -- consecutive windows of the sample
    order, wrapping around."""
    if not size:
        return None
    start = ((t // period) % N) * size % N
    mask = np.zeros(N, dtype=bool)
    mask[(start + np.arange(size)) % N] = True
    return mask


def thresholds(seed: int, tag: int, t: int, K: int, beta: float = 0.0):
    """Per-candidate thresholds of step t: 0 for the greedy rule (beta = 0)."""
    if not beta:
        return [0.0] * K
    return [metropolis_threshold(accept_uniform(seed, tag, t, k), beta) for k in range(K)]


@dataclass
class StepRecord:
    t: int
    L_before: float
    cands: list
    losses: List[float]          # L_k for every evaluated candidate
    chosen: int                  # index of the committed candidate or -1
    L_after: float
    dls: List[float] = field(default_factory=list)     # dL_k
    mags: List[float] = field(default_factory=list)    # size of dL_k's first-order terms
    thetas: List[float] = field(default_factory=list)  # acceptance thresholds (Eq. 7)


def _delta(model, c):
    if hasattr(model, "delta"):
        dL, mag = model.delta(c)
        return dL, mag
    L = model.loss()
    return model.eval(c) - L, None


def evaluate_all(model, t: int, K: int, seed: int, tag: int, delta: float,
                 mode: str = "weight", accept_ties: bool = False, scan_all: bool = True,
                 beta: float = 0.0, n_prune: int = 0, subset=(0, 1)):
    """Score candidates (t, 0..K-1) against the committed state without
    committing; candidates k < n_prune are pruning moves (Sec. 2.2: they come
    first in stream order, so pruning is preferred); subset = (size, period)
    averages each change over step t's minibatch.  Returns (L_t,
    candidates, dL list, sizes list, thresholds, index of the first that
    passes the test or -1)."""
    if subset[0]:
        model.subset = minibatch(t, model.X.shape[0], subset[0], subset[1])
    L_t = model.loss()
    th = thresholds(seed, tag, t, K, beta)
    cands, dls, mags = [], [], []
    chosen = -1
    for k in range(K):
        c = (model.candidate(seed, tag, t, k, delta, mode, prune=True) if k < n_prune
             else model.candidate(seed, tag, t, k, delta, mode))
        dL, mag = _delta(model, c)
        cands.append(c)
        dls.append(dL)
        mags.append(mag)
        if chosen < 0 and accepts(dL, accept_ties, th[k]):
            chosen = k
            if not scan_all:
                break
    if subset[0]:
        model.subset = None
    return L_t, cands, dls, mags, th[:len(dls)], chosen


def evaluate(model, t: int, K: int, seed: int, tag: int, delta: float,
             mode: str = "weight", accept_ties: bool = False, scan_all: bool = True,
             beta: float = 0.0):
    """Score candidates (t, 0..K-1) against the committed state without
    committing.  Returns (L_t, candidates, losses L_t + dL_k, index of the
    first that passes the test or -1).  scan_all=False stops at that first
    candidate."""
    L_t, cands, dls, _, _, chosen = evaluate_all(model, t, K, seed, tag, delta, mode,
                                                 accept_ties, scan_all, beta)
    return L_t, cands, [L_t + d for d in dls], chosen


def step(model, t: int, K: int, seed: int, tag: int, delta: float,
         mode: str = "weight", accept_ties: bool = False,
         scan_all: bool = True, force: Optional[int] = None,
         beta: float = 0.0, n_prune: int = 0, subset=(0, 1)) -> StepRecord:
    """One step of K candidates: evaluate, then commit the first that passes.

    scan_all=False stops at the first improving candidate (the sequential
    method); scan_all=True evaluates all K (the batched step, used for parity).
    `force` (None, -1 or k) overrides the decision; used only by parity tests
    where the decision lies inside the floating-point tie band.
    """
    L_t, cands, dls, mags, th, chosen = evaluate_all(model, t, K, seed, tag, delta, mode,
                                                     accept_ties, scan_all, beta, n_prune,
                                                     subset)
    losses = [L_t + d for d in dls]
    if force is not None:
        chosen = force
    if chosen >= 0:
        model.commit(cands[chosen], losses[chosen])
    return StepRecord(t, L_t, cands, losses, chosen, model.loss(), dls, mags, th)


def run(model, t0: int, n_steps: int, K: int, seed: int, tag: int, delta: float,
        mode: str = "weight", accept_ties: bool = False, scan_all: bool = False,
        beta: float = 0.0, n_prune: int = 0, subset=(0, 1)):
    """n_steps consecutive steps starting at step t0; returns the records."""
    return [step(model, t, K, seed, tag, delta, mode, accept_ties, scan_all, beta=beta,
                 n_prune=n_prune, subset=subset)
            for t in range(t0, t0 + n_steps)]


def remaining_weight_ratio(model) -> float:
    """Fraction of weights that are not zero (the pruning metric of Sec. 2.2)."""
    ws = model.state.weights
    return float(sum(np.count_nonzero(w) for w in ws)) / float(sum(w.size for w in ws))
