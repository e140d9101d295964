"""GPU parity of the selection rules and mutation kinds beyond the greedy
single-weight increment, against the fp64 oracle (through the C ABI):

* the Metropolis rule of Eq. 7 (accept with probability min{1, e^{-beta dL}}
  from a second counter-based word per candidate), explicit steps and both
  device loops, with uphill moves accepted; beta -> infinity equal to the
  ties-accepting greedy rule bit for bit;
* the greedy rule with ties accepted (Eq. 6 as printed: dL <= 0), on data
  with never-lit pixels, so zero changes occur and are committed;
* the weight bound |w'| < Delta of Eq. 1 at a level that rejects about half
  of each step's candidates unevaluated, and at one that rejects nearly all
  of a batch of 128, so that decisions fall past the first 64 candidates or
  find no winner;
* pruning moves (Sec. 2.2, w -> 0) alone and mixed with increments
  (pruning first in stream order), with the remaining-weight ratio.
"""
import math

import numpy as np
import pytest
import torch

from oracle import mca as omca
from parity_util import (ParityStats, assert_state_equal, explicit_steps, make_pair,
                         replay_trace)
from workloads import CONFIGS, mlp_workload

pytestmark = pytest.mark.gpu


def banner(msg):
    print(f"[gpu] {msg}", flush=True)


@pytest.fixture(scope="module")
def mca():
    from paper_2607_08406_amd import mca as m
    m.load_library()
    assert torch.cuda.is_available()
    return m


def small_wide(**kw):
    base = dict(name="wide_small", widths=(784, 512, 10), n_samples=1000)
    base.update(kw)
    return CONFIGS["wide"].scaled(**base)


def uphill(ref_run):
    return sum(1 for dl, ch in ref_run if ch >= 0 and dl[ch] > 0)


@pytest.mark.parametrize("persistent", [1, 0])
def test_metropolis_wide(mca, persistent):
    cfg = small_wide()
    beta = 2e5
    banner(f"Metropolis beta={beta} 784-512-10 persistent={persistent}")
    w = mlp_workload(cfg)
    ctx, ref = make_pair(cfg, w, k_max=16, beta=beta)
    ctx.set_option(mca.MCA_OPT_PERSISTENT_LOOP, persistent)
    ps = ParityStats(f"Metropolis beta={beta:g} 784-512-10 persistent={persistent}")
    _, acc = explicit_steps(ctx, ref, cfg, 0, 30, 16, ps, beta=beta)
    assert acc > 5
    assert_state_equal(ctx, ref)
    ctx.set_step(30)
    st, ch, dl = ctx.run_steps(120, 16, trace=True, trace_dloss=True)
    assert st.steps == 120
    replay_trace(ref, cfg, 30, ch, dl, 16, ps, beta=beta)
    assert_state_equal(ctx, ref)
    # the rule accepts moves that raise the loss
    ups = sum(1 for n in range(120) if ch[n] >= 0 and dl[n, ch[n]] > 0)
    assert ups > 0
    ctx.close()


def test_metropolis_infinite_beta_is_greedy_with_ties(mca):
    """beta = 1e300: every threshold is below 4e-299, so the device run
    equals the ties-accepting greedy run bit for bit."""
    cfg = small_wide(name="wide_ties", accept_ties=True)
    w = mlp_workload(cfg)
    a, _ = make_pair(cfg, w, k_max=16)
    b, _ = make_pair(cfg.scaled(accept_ties=False), w, k_max=16, beta=1e300)
    sa, ca, da = a.run_steps(150, 16, trace=True, trace_dloss=True)
    sb, cb, db = b.run_steps(150, 16, trace=True, trace_dloss=True)
    np.testing.assert_array_equal(ca, cb)
    assert da.tobytes() == db.tobytes()
    pa, _ = a.params()
    pb, _ = b.params()
    for x, y in zip(pa, pb):
        assert x.tobytes() == y.tobytes()
    a.close()
    b.close()


@pytest.mark.parametrize("persistent", [1, 0])
def test_accept_ties_on_device(mca, persistent):
    """Eq. 6 as printed (dL <= 0): the template images leave about 31 % of the
    pixels dark in every sample, so first-layer moves on them change nothing
    (dL = 0 exactly) and are committed under this rule."""
    cfg = small_wide(name="wide_ties", accept_ties=True)
    banner(f"accept ties 784-512-10 persistent={persistent}")
    w = mlp_workload(cfg)
    ctx, ref = make_pair(cfg, w, k_max=16)
    ctx.set_option(mca.MCA_OPT_PERSISTENT_LOOP, persistent)
    ps = ParityStats(f"accept ties 784-512-10 persistent={persistent}")
    _, acc = explicit_steps(ctx, ref, cfg, 0, 20, 16, ps)
    assert_state_equal(ctx, ref)
    ctx.set_step(20)
    st, ch, dl = ctx.run_steps(80, 16, trace=True, trace_dloss=True)
    replay_trace(ref, cfg, 20, ch, dl, 16, ps)
    assert_state_equal(ctx, ref)
    zeros = sum(1 for n in range(80) if ch[n] >= 0 and dl[n, ch[n]] == 0.0)
    assert zeros > 0
    ctx.close()


@pytest.mark.parametrize("persistent", [1, 0])
def test_bound_splits_batch(mca, persistent):
    """The weight bound of Eq. 1 at the median |w| of the first layer: about
    half of each step's candidates are rejected unevaluated (dL = +inf on
    both sides), the rest are scored and selected as usual."""
    cfg = small_wide(name="wide_bound")
    w = mlp_workload(cfg)
    bound = float(np.median(np.abs(w["weights"][0])))
    banner(f"bound {bound:.4f} 784-512-10 persistent={persistent}")
    ctx, ref = make_pair(cfg, w, k_max=32, bound=bound)
    ctx.set_option(mca.MCA_OPT_PERSISTENT_LOOP, persistent)
    ps = ParityStats(f"bound 784-512-10 persistent={persistent}")
    cands = ctx.propose(0, 32)
    _, dl0 = ctx.eval_losses(cands)
    ctx.rollback()
    rejected = int(np.isinf(dl0).sum())
    assert 4 <= rejected <= 28, rejected
    _, acc = explicit_steps(ctx, ref, cfg, 0, 20, 32, ps, bound=bound)
    assert acc > 3
    assert_state_equal(ctx, ref)
    ctx.set_step(20)
    st, ch, dl = ctx.run_steps(60, 32, trace=True, trace_dloss=True)
    replay_trace(ref, cfg, 20, ch, dl, 32, ps, bound=bound)
    assert_state_equal(ctx, ref)
    ctx.close()


def test_decision_beyond_one_chunk_of_64(mca):
    """K = 128 (the one-launch-per-phase loop; the persistent loop takes
    K <= 64) under a weight bound at the 3 % quantile of the first layer's
    magnitudes, so that most candidates are rejected unevaluated: the first
    passing candidate often lies past index 63, and some steps pass none.
    The selection's last block decides over chunks of 64 candidates; every
    traced loss change and decision against the oracle's."""
    cfg = small_wide(name="wide_k128")
    w = mlp_workload(cfg)
    K = 128
    bound = float(np.quantile(np.abs(w["weights"][0]), 0.03))
    banner(f"bound {bound:.6f} 784-512-10 K={K} device loop")
    ctx, ref = make_pair(cfg, w, k_max=K, bound=bound)
    ps = ParityStats(f"bound 784-512-10 K={K}")
    st, ch, dl = ctx.run_steps(60, K, trace=True, trace_dloss=True)
    assert st.next_step == 60
    replay_trace(ref, cfg, 0, ch, dl, K, ps, bound=bound)
    assert_state_equal(ctx, ref)
    ch = np.asarray(ch)
    late, none = int((ch >= 64).sum()), int((ch < 0).sum())
    print(f"[gpu] decisions past index 63: {late}, steps without a winner: {none}", flush=True)
    assert late >= 3 and none >= 3, (late, none)
    ctx.close()


def remaining(params):
    return sum(int(np.count_nonzero(p)) for p in params) / sum(p.size for p in params)


@pytest.mark.parametrize("persistent", [1, 0])
def test_pure_pruning_wide(mca, persistent):
    """Every candidate sets its weight to zero (Sec. 2.2); accepted when the
    loss falls (strict) -- the remaining-weight ratio falls by one weight per
    accepted step, on both sides."""
    cfg = small_wide(name="wide_prune", delta=0.0)
    banner(f"pure pruning 784-512-10 persistent={persistent}")
    w = mlp_workload(cfg)
    K = 16
    ctx, ref = make_pair(cfg, w, k_max=K, n_prune=K)
    ctx.set_option(mca.MCA_OPT_PERSISTENT_LOOP, persistent)
    ps = ParityStats(f"pure pruning 784-512-10 persistent={persistent}")
    r0 = remaining(w["weights"])
    _, acc = explicit_steps(ctx, ref, cfg, 0, 20, K, ps, n_prune=K)
    assert acc > 3
    assert_state_equal(ctx, ref)
    ctx.set_step(20)
    st, ch, dl = ctx.run_steps(100, K, trace=True, trace_dloss=True)
    _, acc2 = replay_trace(ref, cfg, 20, ch, dl, K, ps, n_prune=K)
    assert_state_equal(ctx, ref)
    total = sum(p.size for p in w["weights"])
    r1 = remaining(ctx.params()[0])
    assert round((r0 - r1) * total) == acc + acc2
    assert omca.remaining_weight_ratio(ref) == r1
    ctx.close()


def test_mixed_pruning_three_layer_ternary(mca):
    """Ternary 784-96-80-10 Gaussian net: candidates 0..7 of every step
    prune (code 0), 8..15 move to another code; pruning is preferred by
    stream order.  Explicit steps, then a device run replayed."""
    cfg = CONFIGS["ternary"].scaled(name="t3_prune", widths=(784, 96, 80, 10), n_samples=333,
                                    K=16)
    banner("mixed pruning ternary 784-96-80-10")
    w = mlp_workload(cfg)
    ctx, ref = make_pair(cfg, w, k_max=16, n_prune=8)
    ps = ParityStats("mixed pruning ternary 784-96-80-10")
    _, acc = explicit_steps(ctx, ref, cfg, 0, 30, 16, ps, n_prune=8)
    assert acc > 3
    assert_state_equal(ctx, ref)
    ctx.set_step(30)
    st, ch, dl = ctx.run_steps(40, 16, trace=True, trace_dloss=True)
    replay_trace(ref, cfg, 30, ch, dl, 16, ps, n_prune=8)
    assert_state_equal(ctx, ref)
    ctx.close()


def test_mixed_pruning_deep(mca):
    """784-256-256-256-10 tanh on 300 images, layer drawn first, candidates
    0..3 prune and 4..7 mutate: pruning through the dense chain, the slab
    and the column kernels."""
    cfg = CONFIGS["deep"].scaled(name="deep_prune", widths=(784, 256, 256, 256, 10),
                                 n_samples=300, K=8, delta=0.05)
    banner("mixed pruning deep 784-3x256-10")
    w = mlp_workload(cfg)
    ctx, ref = make_pair(cfg, w, k_max=8, n_prune=4)
    ps = ParityStats("mixed pruning deep 784-3x256-10")
    _, acc = explicit_steps(ctx, ref, cfg, 0, 30, 8, ps, n_prune=4)
    assert acc > 3
    assert_state_equal(ctx, ref)
    ctx.set_step(30)
    st, ch, dl = ctx.run_steps(30, 8, trace=True, trace_dloss=True)
    replay_trace(ref, cfg, 30, ch, dl, 8, ps, n_prune=4)
    assert_state_equal(ctx, ref)
    ctx.close()


@pytest.mark.parametrize("persistent", [1, 0])
def test_minibatch_wide(mca, persistent):
    """Sec. 2.2's minibatch: each step's loss changes average over a window of
    400 of the 1,000 samples (moving every 3 steps, wrapping around), pairs
    outside it are not scored; commits still move every sample, and the
    committed loss is the mean over all of them."""
    cfg = small_wide(name="wide_mb")
    sub = (400, 3)
    banner(f"minibatch {sub} 784-512-10 persistent={persistent}")
    w = mlp_workload(cfg)
    ctx, ref = make_pair(cfg, w, k_max=16, subset=sub)
    ctx.set_option(mca.MCA_OPT_PERSISTENT_LOOP, persistent)
    ps = ParityStats(f"minibatch 784-512-10 persistent={persistent}")
    _, acc = explicit_steps(ctx, ref, cfg, 0, 15, 16, ps, subset=sub)
    assert acc > 3
    assert_state_equal(ctx, ref)
    ctx.set_step(15)
    st, ch, dl = ctx.run_steps(60, 16, trace=True, trace_dloss=True)
    replay_trace(ref, cfg, 15, ch, dl, 16, ps, subset=sub)
    assert_state_equal(ctx, ref)
    L, t = ctx.loss()
    assert t == 75 and abs(L - ref.loss()) <= 1e-5 * ref.loss()
    ctx.close()


@pytest.mark.parametrize("kind", ["ternary3", "deep"])
def test_minibatch_other_paths(mca, kind):
    """The window on the three-layer slab and the deep chain paths, with
    pruning mixed in (Sec. 2.2's setting: pruning preferred, minibatches)."""
    if kind == "ternary3":
        cfg = CONFIGS["ternary"].scaled(name="t3_mb", widths=(784, 96, 80, 10), n_samples=333,
                                        K=16)
    else:
        cfg = CONFIGS["deep"].scaled(name="deep_mb", widths=(784, 256, 256, 256, 10),
                                     n_samples=300, K=16, delta=0.05)
    sub = (150, 2)
    banner(f"minibatch {sub} {cfg.name}")
    w = mlp_workload(cfg)
    ctx, ref = make_pair(cfg, w, k_max=16, n_prune=4, subset=sub)
    ps = ParityStats(f"minibatch + pruning {cfg.name}")
    explicit_steps(ctx, ref, cfg, 0, 20, 16, ps, n_prune=4, subset=sub)
    assert_state_equal(ctx, ref)
    ctx.set_step(20)
    st, ch, dl = ctx.run_steps(20, 16, trace=True, trace_dloss=True)
    replay_trace(ref, cfg, 20, ch, dl, 16, ps, n_prune=4, subset=sub)
    assert_state_equal(ctx, ref)
    L, _ = ctx.loss()
    assert abs(L - ref.loss()) <= 1e-5 * ref.loss()
    ctx.close()


def test_selection_options_validated(mca):
    cfg = small_wide()
    w = mlp_workload(cfg)
    for kw in [dict(beta=-1.0), dict(n_prune=-1), dict(subset_size=cfg.n_samples + 1),
               dict(subset_size=10, subset_period=0)]:
        d = mca.mlp_desc(cfg.widths, cfg.act, delta=cfg.delta, **kw)
        with pytest.raises(mca.MCAError, match="EINVAL"):
            mca.mca_plan(d, cfg.n_samples, 8)
    d = mca.mlp_desc(cfg.widths, cfg.act, delta=cfg.delta)
    d.accept_rule = 7
    with pytest.raises(mca.MCAError, match="EINVAL"):
        mca.mca_plan(d, cfg.n_samples, 8)
    ctx, _ = make_pair(cfg, w, k_max=4)
    c = ctx.propose(0, 4)
    c["flags"] = 4
    with pytest.raises(mca.MCAError, match="EINVAL"):
        ctx.eval_losses(c)
    ctx.close()
