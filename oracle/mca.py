"""Greedy mutation-selection loop of the oracle (Eq. 1, Eq. 5, Eq. 6).

One step t scores candidates k = 0..K-1 of the counter-based stream against the
same committed state W_t, in stream order.  The first candidate whose loss
change dL_k = L(W_t + dW_k) - L(W_t) passes the acceptance test is committed;
later candidates of the step are discarded.  With K = 1 this is the paper's
sequential rule (mutate one parameter, keep it if the loss does not increase,
otherwise retry).  Acceptance (Eq. 6 with the ties reading): dL < 0 by default,
dL <= 0 when ties are accepted.  A NaN or infinite dL is never accepted.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np


def accepts(dL: float, accept_ties: bool) -> bool:
    """Greedy selection test of Eq. 6 (strict unless ties are accepted)."""
    if not math.isfinite(dL):
        return False
    return dL <= 0.0 if accept_ties else dL < 0.0


@dataclass
class StepRecord:
    t: int
    L_before: float
    cands: list
    losses: List[float]          # L_k for every evaluated candidate
    chosen: int                  # index of the committed candidate or -1
    L_after: float


def evaluate(model, t: int, K: int, seed: int, tag: int, delta: float,
             mode: str = "weight", accept_ties: bool = False, scan_all: bool = True):
    """Score candidates (t, 0..K-1) against the committed state without
    committing.  Returns (L_t, candidates, losses, index of the first that
    passes the test or -1).  scan_all=False stops at that first candidate."""
    L_t = model.loss()
    cands, losses = [], []
    chosen = -1
    for k in range(K):
        c = model.candidate(seed, tag, t, k, delta, mode)
        Lk = model.eval(c)
        cands.append(c)
        losses.append(Lk)
        if chosen < 0 and accepts(Lk - L_t, accept_ties):
            chosen = k
            if not scan_all:
                break
    return L_t, cands, losses, chosen


def step(model, t: int, K: int, seed: int, tag: int, delta: float,
         mode: str = "weight", accept_ties: bool = False,
         scan_all: bool = True, force: Optional[int] = None) -> StepRecord:
    """One step of K candidates: evaluate, then commit the first that passes.

    scan_all=False stops at the first improving candidate (the sequential
    method); scan_all=True evaluates all K (the batched step, used for parity).
    `force` (None, -1 or k) overrides the decision; used only by parity tests
    where the decision lies inside the floating-point tie band.
    """
    L_t, cands, losses, chosen = evaluate(model, t, K, seed, tag, delta, mode,
                                          accept_ties, scan_all)
    if force is not None:
        chosen = force
    if chosen >= 0:
        model.commit(cands[chosen], losses[chosen])
    return StepRecord(t, L_t, cands, losses, chosen, model.loss())


def run(model, t0: int, n_steps: int, K: int, seed: int, tag: int, delta: float,
        mode: str = "weight", accept_ties: bool = False, scan_all: bool = False):
    """n_steps consecutive steps starting at step t0; returns the records."""
    return [step(model, t, K, seed, tag, delta, mode, accept_ties, scan_all)
            for t in range(t0, t0 + n_steps)]
