"""GPU parity of three-layer MLPs against the fp64 oracle (through the C ABI).

A first-layer mutation moves one unit of the first hidden layer, every unit
of the second hidden layer for each affected sample (rank-1), and then the
logits; second- and third-layer mutations are the column cases of the
two-layer path.  Workloads: reduced ternary Gaussian and tanh nets whose
sample counts span several 24-sample tiles and a ragged tail, and the full
ternary 784-1024-1024-10 net on 8,192 samples at K = 64.
"""
import numpy as np
import pytest
import torch

from oracle import mca as omca
from oracle.mlp import FullMLP, MLPState, per_sample_ce
from parity_util import (REL_TOL, ParityStats, assert_cands_equal, assert_state_equal,
                         check_batch, explicit_steps, make_pair, replay_trace)
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


def assert_caches_match(ctx, ref, rel=1e-5):
    """The device's cached per-sample losses against the oracle's (recomputed
    from its own fp64 caches)."""
    got = ctx.sample_losses()
    exp = per_sample_ce(ref.Z[-1], ref.y)
    np.testing.assert_allclose(got, exp, rtol=rel, atol=1e-6)


def layer_counts(ref, cfg, t0, n, K):
    counts = np.zeros(cfg.n_layers, dtype=int)
    for t in range(t0, t0 + n):
        _, rc, _, _ = omca.evaluate(ref, t, K, cfg.seed_stream, cfg.stream_tag, cfg.delta,
                                    cfg.layer_pick, cfg.accept_ties)
        for c in rc:
            counts[c.layer] += 1
    return counts


def test_ternary_three_layer_small(mca):
    """784-96-80-10 Gaussian ternary net on 333 samples (13 full tiles of 24
    and a tail of 21): explicit steps, then a device run replayed."""
    cfg = CONFIGS["ternary"].scaled(name="t3_small", widths=(784, 96, 80, 10), n_samples=333,
                                    K=16)
    banner(f"{cfg.name} {cfg.widths} N={cfg.n_samples}")
    w = mlp_workload(cfg)
    ctx, ref = make_pair(cfg, w, k_max=16)
    L, _ = ctx.loss()
    assert abs(L - ref.loss()) <= REL_TOL * ref.loss()
    ps = ParityStats("ternary 784-96-80-10")
    _, acc = explicit_steps(ctx, ref, cfg, 0, 40, 16, ps)
    assert acc > 5
    assert_state_equal(ctx, ref)
    assert_caches_match(ctx, ref)
    ctx.set_step(40)
    st, ch, dl = ctx.run_steps(60, 16, trace=True, trace_dloss=True)
    assert st.steps == 60
    replay_trace(ref, cfg, 40, ch, dl, 16, ps)
    assert_state_equal(ctx, ref)
    assert_caches_match(ctx, ref)
    # first-layer candidates were drawn and some were committed
    first = [int(c) for n, c in enumerate(ch) if c >= 0]
    assert len(first) > 5
    ctx.close()


def test_three_layer_other_class_count(mca):
    """784-64-48-13 Gaussian ternary net on 250 template images: thirteen
    classes run the general variant of the layer-(L-3) kernel (12-sample
    tiles) and of the column kernels."""
    cfg = CONFIGS["ternary"].scaled(name="t3_c13", widths=(784, 64, 48, 13), n_samples=250, K=16)
    banner(f"{cfg.name} {cfg.widths} N={cfg.n_samples}")
    w = mlp_workload(cfg)
    ctx, ref = make_pair(cfg, w, k_max=16)
    L, _ = ctx.loss()
    assert abs(L - ref.loss()) <= REL_TOL * ref.loss()
    counts = layer_counts(ref, cfg, 0, 30, 16)
    assert counts[0] > 20  # the first layer is exercised
    ps = ParityStats("ternary 784-64-48-13")
    explicit_steps(ctx, ref, cfg, 0, 30, 16, ps)
    assert_state_equal(ctx, ref)
    assert_caches_match(ctx, ref)
    ctx.set_step(30)
    st, ch, dl = ctx.run_steps(30, 16, trace=True, trace_dloss=True)
    replay_trace(ref, cfg, 30, ch, dl, 16, ps)
    assert_state_equal(ctx, ref)
    assert_caches_match(ctx, ref)
    ctx.close()


def test_tanh_three_layer_continuous(mca):
    """64-48-40-10 tanh net with continuous weights on 500 samples, K = 8."""
    cfg = CONFIGS["tiny"].scaled(name="tanh3", widths=(64, 48, 40, 10), n_samples=500, K=8)
    banner(f"{cfg.name} {cfg.widths} N={cfg.n_samples}")
    w = mlp_workload(cfg)
    ctx, ref = make_pair(cfg, w, k_max=8)
    counts = layer_counts(ref, cfg, 0, 50, 8)
    assert counts[0] > 20  # the first layer is exercised
    ps = ParityStats("tanh 64-48-40-10")
    explicit_steps(ctx, ref, cfg, 0, 50, 8, ps)
    assert_state_equal(ctx, ref)
    assert_caches_match(ctx, ref)
    ctx.set_step(50)
    st, ch, dl = ctx.run_steps(150, 8, trace=True, trace_dloss=True)
    replay_trace(ref, cfg, 50, ch, dl, 8, ps)
    assert_state_equal(ctx, ref)
    assert_caches_match(ctx, ref)
    ctx.close()


@pytest.mark.parametrize("N", [1, 23, 24, 25, 49])
def test_three_layer_tile_edges(mca, N):
    cfg = CONFIGS["ternary"].scaled(name=f"t3_n{N}", widths=(784, 40, 36, 10), n_samples=N, K=8)
    w = mlp_workload(cfg)
    ctx, ref = make_pair(cfg, w, k_max=8)
    explicit_steps(ctx, ref, cfg, 0, 25, 8, ParityStats(f"ternary 784-40-36-10 N={N}"))
    assert_state_equal(ctx, ref)
    assert_caches_match(ctx, ref)
    ctx.close()


def test_rollback_three_layer_is_byte_identical(mca):
    cfg = CONFIGS["ternary"].scaled(name="t3_rb", widths=(784, 64, 48, 10), n_samples=200, K=16)
    w = mlp_workload(cfg)
    ctx, ref = make_pair(cfg, w, k_max=16)
    before_p, before_c = ctx.params()
    before_l = ctx.sample_losses()
    cands = ctx.propose(0, 16)
    ctx.eval_losses(cands)
    ctx.rollback()
    after_p, after_c = ctx.params()
    for a, b in zip(before_p, after_p):
        assert a.tobytes() == b.tobytes()
    for a, b in zip(before_c, after_c):
        assert a.tobytes() == b.tobytes()
    assert before_l.tobytes() == ctx.sample_losses().tobytes()
    ctx.close()


def test_full_ternary_workload(mca):
    """784-1024-1024-10 Gaussian ternary net on 8,192 samples, K = 64: init
    loss, one explicit step with every candidate against the incremental
    oracle and two first-layer candidates against full recomputation, then a
    short device run replayed."""
    cfg = CONFIGS["ternary"]
    banner("ternary 784-1024-1024-10 N=8192 K=64")
    w = mlp_workload(cfg)
    ctx, ref = make_pair(cfg, w, k_max=64)
    L, _ = ctx.loss()
    assert abs(L - ref.loss()) <= REL_TOL * ref.loss()
    ps = ParityStats("ternary 784-1024-1024-10 full")
    cands = ctx.propose(0, 64)
    losses, dl = ctx.eval_losses(cands)
    L_t, rc, dls, chosen = check_batch(ps, dl, ref, cfg, 0, 64)
    assert_cands_equal(cands, rc)
    full = FullMLP(MLPState(w["weights"], w["codes"], w["scales"]), w["X"], w["y"], cfg.act,
                   cfg.gamma)
    firsts = [k for k, c in enumerate(rc) if c.layer == 0][:2]
    assert firsts
    for k in firsts:
        assert abs(losses[k] - full.eval(rc[k])) <= REL_TOL * losses[k]
        d, _ = full.delta(rc[k])
        assert abs(dl[k] - d) <= 1e-5 * abs(d) + 1e-13, (k, dl[k], d)
    ctx.rollback()
    st, ch, dl = ctx.run_steps(50, 64, trace=True, trace_dloss=True)
    assert st.steps == 50
    replay_trace(ref, cfg, 0, ch, dl, 64, ps)
    assert_state_equal(ctx, ref)
    assert_caches_match(ctx, ref)
    ctx.close()
