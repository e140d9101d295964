"""Helpers shared by the GPU parity tests: build a context and an oracle from
the same seeded workload, compare candidate records bit for bit, and compare
per-candidate loss changes and accept decisions.

Parity bar (fp32 GPU vs fp64 oracle):

* every candidate's loss change dL_k within
      |dL_gpu - dL_orc| <= 1e-5 |dL_orc| + eps_k,
  eps_k = kappa_k 2^-24 A_k, where A_k = (1/N) sum_n (sum_c p_nc a_nc +
  a_n,y_n) is the size of the first-order terms of the change (the
  oracle's, ce_change: a = |dz|, or for a change that reaches the logits
  through a hidden layer the sum of the absolute terms of its logit sums),
  plus |dl_n| / 16 times the sensitivity of dl_n to the fp32 rounding of
  the two cached fields the candidate reads (its input activation, its
  unit's own field, each rounded by the forward pass to about 2^-24 times
  the sum of its terms' sizes: a field that is small by cancellation
  carries a large relative error, and dl_n is linear in the input; the 1/16
  makes that 8 ulp under kappa = 128), and kappa_k bounds the fp32 rounding
  of the method's arithmetic on them:
  a few ulp per sample for the transfer-function difference, the
  expm1/log1p terms and the C-term class sum, the in-order fp32 sum of up
  to 64 samples per tile, and for a change that passes through D dense
  layers their fp32 dot products (mlp_kappa);
* every decision equal, except where the oracle's margin |dL_k - theta_k|
  (theta_k = 0 for the greedy rule, the Metropolis threshold of Eq. 7
  otherwise) is within that tolerance: fp32 cannot resolve those;
* the tie band |dL_k| < 1e-6 of the decision-relevant candidates is counted
  and reported;
* candidate indices, increments and discrete codes bit-exact; continuous
  weights bit-exact (both sides apply the same fp32 w').
"""
import math

import numpy as np

from oracle import mca as omca
from oracle.mlp import FullMLP, IncrementalMLP, MLPState
from oracle.normmlp import NormMLP

REL_TOL = 1e-5
TIE = 1e-6
U32 = 2.0 ** -24


def cand_mode(cfg):
    """How the config's candidates are drawn: a channel scheme (Sec. 2.3) or
    the single-parameter pick."""
    m = getattr(cfg, "mutation", "single")
    return m if m.startswith("channel_") else getattr(cfg, "layer_pick", "weight")


def mlp_kappa(widths, layer):
    """Rounding budget of an MLP candidate in `layer` (units of 2^-24 A_k):
    128 for the column, rank-1 and cross-entropy work with its tile sums,
    plus 64 per dense layer the change then passes through."""
    L = len(widths) - 1
    dense = max(0, L - 3 - layer)
    return 128.0 + 64.0 * dense


def norm_kappa(widths, layer):
    """The same budget for a net with biases and normalized hidden fields:
    128 for the column and cross-entropy work, plus, for every layer the
    change then passes through, 256: its normalization pass (two row sums
    added in runs of 64 terms, up to 64 ulp of their terms' sizes each, and
    the difference form of the normalized field) and its dense product of W
    terms (64)."""
    L = len(widths) - 1
    return 128.0 + 256.0 * (L - 1 - layer)


def kappa_of(cfg, c):
    if getattr(cfg, "layer_norm", False) or getattr(cfg, "biases", False):
        return norm_kappa(cfg.widths, c.layer)
    return mlp_kappa(cfg.widths, getattr(c, "layer", 0))


REPORTS = []  # every ParityStats made in this session, printed in the terminal summary


class ParityStats:
    """Counts kept over a parity run (printed in the pytest terminal summary)."""

    def __init__(self, name=""):
        REPORTS.append(self)
        self.name = name
        self.n = 0             # candidates compared
        self.relevant = 0      # decision-relevant (up to the first acceptance)
        self.tie = 0           # decision-relevant with |dL| < 1e-6
        self.unresolved = 0    # margin within the fp32 tolerance
        self.flips = 0         # decisions that differed (only where unresolved)
        self.within_rel = 0    # |error| <= 1e-5 |dL| without the floor
        self.nonzero = 0
        self.worst = 0.0       # max |error| / tolerance
        self.worst_rel = 0.0   # max |error| / |dL| over nonzero dL

    def __str__(self):
        return (f"{self.name}: {self.n} candidates, worst error/tolerance {self.worst:.3f}, "
                f"worst relative error {self.worst_rel:.2e}, within 1e-5 relative "
                f"{self.within_rel}/{self.nonzero}, tie band {self.tie}/{self.relevant}, "
                f"unresolved {self.unresolved}, decision flips {self.flips}")


def make_pair(cfg, w, k_max, oracle="incremental", bound=0.0, beta=0.0, n_prune=0,
              subset=(0, 1)):
    from paper_2607_08406_amd import mca
    scales = w["scales"]
    desc = mca.mlp_desc(cfg.widths, cfg.act, gamma=cfg.gamma, delta=cfg.delta,
                        ternary_scales=scales, pick=cfg.layer_pick,
                        accept_ties=cfg.accept_ties, seed=cfg.seed_stream,
                        stream_tag=cfg.stream_tag, bound=bound, beta=beta, n_prune=n_prune,
                        subset_size=subset[0], subset_period=subset[1],
                        mutation=getattr(cfg, "mutation", "single"), biases=cfg.biases,
                        layer_norm=cfg.layer_norm, ln_eps=cfg.ln_eps,
                        sticky_steps=cfg.sticky_steps)
    ctx = mca.Context(desc, w["weights"], w["X"], w["y"], k_max=k_max, codes=w["codes"])
    if cfg.biases or cfg.layer_norm:
        ref = NormMLP(w["weights"], w["X"], w["y"], cfg.act, cfg.gamma, bias=cfg.biases,
                      ln=cfg.layer_norm, eps=cfg.ln_eps, sticky=cfg.sticky_steps)
        return ctx, ref
    cls = IncrementalMLP if oracle == "incremental" else FullMLP
    ref = cls(MLPState(w["weights"], w["codes"], scales), w["X"], w["y"], cfg.act, cfg.gamma)
    return ctx, ref


def assert_cands_equal(gpu, ref_cands):
    assert len(gpu) == len(ref_cands)
    for g, c in zip(gpu, ref_cands):
        got = (int(g["flat"]), int(g["layer"]), int(g["j"]), int(g["i"]), int(g["code"]))
        exp = (c.flat, c.layer, c.j, c.i, c.code)
        assert got == exp, (got, exp)
        assert np.float32(g["d"]).tobytes() == np.float32(c.d).tobytes(), (g["d"], c.d)


def check_batch(stats, gpu_dl, ref, cfg, t, K, kappa=None, beta=0.0):
    """One batch of explicit candidates of step t against the oracle's loss
    changes (no decision); returns the oracle's (L_t, candidates, dL)."""
    L_t, rc, dls, mags, th, chosen = omca.evaluate_all(
        ref, t, K, cfg.seed_stream, cfg.stream_tag, cfg.delta,
        getattr(cfg, "layer_pick", "weight"), cfg.accept_ties)
    kap = [kappa(c) if kappa else kappa_of(cfg, c) for c in rc]
    gch = next((k for k in range(K) if omca.accepts(float(gpu_dl[k]), cfg.accept_ties, th[k])), -1)
    check_step(stats, gpu_dl, dls, mags, kap, th, cfg.accept_ties, gch, chosen, tag=f"step {t}")
    return L_t, rc, dls, chosen


def _bounded(ref, c, bound):
    if bound <= 0:
        return False
    if hasattr(c, "units"):  # a channel: any path weight outside the bound
        return any(abs(float(w)) >= bound for w in c.w_new)
    return abs(float(ref.state.new_value(c))) >= bound


def check_step(stats, gpu_dl, ref_dl, mags, kappas, thetas, accept_ties, chosen_gpu,
               chosen_orc, bounded=None, tag=""):
    """Compare one step's loss changes and decision; returns the decision both
    sides follow (the oracle's, or the device's where only an unresolvable
    margin separates them)."""
    K = len(ref_dl)
    tols = []
    for k in range(K):
        g, r = float(gpu_dl[k]), float(ref_dl[k])
        if bounded is not None and bounded[k]:
            assert g == math.inf, (tag, k, g)  # rejected unevaluated (Eq. 1 bound)
            tols.append(0.0)
            continue
        eps = kappas[k] * U32 * (mags[k] if mags[k] is not None else 0.0)
        tol = REL_TOL * abs(r) + eps
        err = abs(g - r)
        assert err <= tol, (tag, k, g, r, err, tol, kappas[k])
        stats.n += 1
        stats.worst = max(stats.worst, err / tol if tol > 0 else 0.0)
        if r != 0.0:
            stats.nonzero += 1
            stats.worst_rel = max(stats.worst_rel, err / abs(r))
            stats.within_rel += err <= REL_TOL * abs(r)
        tols.append(tol)
    last = chosen_orc if chosen_orc >= 0 else K - 1
    for k in range(last + 1):
        if bounded is not None and bounded[k]:
            continue
        stats.relevant += 1
        stats.tie += abs(ref_dl[k]) < TIE
        if abs(ref_dl[k] - thetas[k]) <= tols[k]:
            stats.unresolved += 1
    if chosen_gpu == chosen_orc:
        return chosen_orc
    # the first candidate on which the two sides decide differently must
    # have a margin fp32 cannot resolve
    m = min(x if x >= 0 else K for x in (chosen_gpu, chosen_orc))
    assert abs(ref_dl[m] - thetas[m]) <= tols[m], (tag, m, chosen_gpu, chosen_orc, ref_dl[m])
    stats.flips += 1
    return chosen_gpu


def _oracle_step(ref, cfg, t, K, bound, beta, n_prune, subset=(0, 1)):
    """The oracle's view of step t: candidates, loss changes (+inf for those a
    weight bound rejects unevaluated, Eq. 1), sizes, thresholds, decision.
    `ref` is one oracle model or a pool of replicas (tests/oracle_pool.py)."""
    if hasattr(ref, "evaluate_all"):
        assert not subset[0]
        L_t, rc, dls, mags, th, chosen = ref.evaluate_all(
            t, K, cfg.seed_stream, cfg.stream_tag, cfg.delta, cand_mode(cfg), cfg.accept_ties,
            beta=beta, n_prune=n_prune)
    else:
        L_t, rc, dls, mags, th, chosen = omca.evaluate_all(
            ref, t, K, cfg.seed_stream, cfg.stream_tag, cfg.delta, cand_mode(cfg),
            cfg.accept_ties, beta=beta, n_prune=n_prune, subset=subset)
    bounded = [_bounded(ref, c, bound) for c in rc]
    if bound > 0:
        dls = [math.inf if b else d for b, d in zip(bounded, dls)]
        chosen = next((k for k in range(K) if not bounded[k]
                       and omca.accepts(dls[k], cfg.accept_ties, th[k])), -1)
    return L_t, rc, dls, mags, th, chosen, (bounded if bound > 0 else None)


def explicit_steps(ctx, ref, cfg, t0, n_steps, K, stats=None, bound=0.0, beta=0.0, n_prune=0,
                   subset=(0, 1)):
    """propose / eval_losses / commit-or-rollback on the GPU beside the oracle.
    Decisions follow the oracle's (the device's only inside the unresolvable
    margin, where both are valid).  With a minibatch, the device's next step
    is set to t first (the explicit evaluation scores its window)."""
    stats = stats if stats is not None else ParityStats()
    accepted = 0
    for t in range(t0, t0 + n_steps):
        cands = ctx.propose(t, K)
        L_t, rc, dls, mags, th, chosen, bounded = _oracle_step(ref, cfg, t, K, bound, beta,
                                                               n_prune, subset)
        assert_cands_equal(cands, rc)
        if subset[0]:
            ctx.set_step(t)
        _, gdl = ctx.eval_losses(cands)
        kap = [kappa_of(cfg, c) for c in rc]
        gch = next((k for k in range(K) if omca.accepts(float(gdl[k]), cfg.accept_ties, th[k])), -1)
        take = check_step(stats, gdl, dls, mags, kap, th, cfg.accept_ties, gch, chosen,
                          bounded, tag=f"step {t}")
        if take >= 0:
            ctx.commit(take)
            ref.commit(rc[take], L_t + dls[take])
            accepted += 1
        else:
            ctx.rollback()
    return stats, accepted


def replay_trace(ref, cfg, t0, chosen, dloss, K, stats=None, beta=0.0, kappa=None, bound=0.0,
                 n_prune=0, subset=(0, 1)):
    """Replay a device run's trace on the oracle: every traced loss change
    against the oracle's, every decision against the oracle's; where only an
    unresolvable margin separates them the oracle follows the device (both
    are valid)."""
    stats = stats if stats is not None else ParityStats()
    accepted = 0
    for n in range(len(chosen)):
        t = t0 + n
        L_t, rc, dls, mags, th, orc, bounded = _oracle_step(ref, cfg, t, K, bound, beta, n_prune,
                                                            subset)
        if kappa is None:
            kap = [kappa_of(cfg, c) for c in rc]
        else:
            kap = [kappa(c) for c in rc]
        g = int(chosen[n])
        if dloss is not None:
            take = check_step(stats, dloss[n], dls, mags, kap, th, cfg.accept_ties, g, orc,
                              bounded, tag=f"step {t}")
        else:
            if g != orc:
                m = min(x if x >= 0 else K for x in (g, orc))
                tol = REL_TOL * abs(dls[m]) + kap[m] * U32 * (mags[m] or 0.0)
                assert abs(dls[m] - th[m]) <= max(tol, TIE), (t, m, g, orc, dls[m])
                stats.flips += 1
            take = g
        if take >= 0:
            ref.commit(rc[take], L_t + dls[take])
            accepted += 1
    return stats, accepted


def assert_state_equal(ctx, ref):
    params, codes = ctx.params()
    weights = ref.state_weights() if hasattr(ref, "state_weights") else ref.state.weights
    for l, (a, b) in enumerate(zip(params, weights)):
        assert a.tobytes() == b.tobytes(), f"weights of layer {l} differ"
    if codes is not None:
        for l, (a, b) in enumerate(zip(codes, ref.state.codes)):
            np.testing.assert_array_equal(a, b)
