"""GPU parity of deep MLPs against the fp64 oracle (through the C ABI).

A mutation in layers 0..L-4 moves one unit, every unit of the next layer for
each affected sample (rank-1), and then every later layer through dense
products on the matrix cores; layer L-3 and the last two layers take the
tile and column kernels.  Workloads: reduced tanh nets with 256-unit hidden
layers whose sample counts span several 64-sample tiles and a ragged tail,
sparse image inputs (sparse lists of affected samples), and the full
784-(24 x 256)-10 net on 4,096 samples at K = 32 with the layer drawn first.
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
    got = ctx.sample_losses()
    exp = per_sample_ce(ref.Z[-1], ref.y)
    np.testing.assert_allclose(got, exp, rtol=rel, atol=1e-6)


def layer_hist(ref, cfg, t0, n, K):
    h = np.zeros(cfg.n_layers, dtype=int)
    for t in range(t0, t0 + n):
        _, rc, _, _ = omca.evaluate(ref, t, K, cfg.seed_stream, cfg.stream_tag, cfg.delta,
                                    cfg.layer_pick, cfg.accept_ties)
        for c in rc:
            h[c.layer] += 1
    return h


def small_deep(**kw):
    base = dict(name="deep_small", widths=(64, 256, 256, 256, 256, 10), n_samples=200, K=8,
                delta=0.1)
    base.update(kw)
    return CONFIGS["deep"].scaled(data="sparse_uniform", **base)


def test_deep_small_every_layer_kind(mca):
    """64-256-256-256-256-10 tanh, 200 samples (3 tiles of 64 + 8), K = 8,
    layer drawn first: chain (layers 0, 1), tile (2) and column (3, 4)."""
    cfg = small_deep()
    banner(f"{cfg.name} {cfg.widths} N={cfg.n_samples}")
    w = mlp_workload(cfg)
    ctx, ref = make_pair(cfg, w, k_max=8)
    L, _ = ctx.loss()
    assert abs(L - ref.loss()) <= REL_TOL * ref.loss()
    h = layer_hist(ref, cfg, 0, 40, 8)
    assert (h > 0).all(), h
    ps = ParityStats("deep 64-4x256-10")
    _, acc = explicit_steps(ctx, ref, cfg, 0, 40, 8, ps)
    assert acc > 5
    assert_state_equal(ctx, ref)
    assert_caches_match(ctx, ref)
    ctx.set_step(40)
    st, ch, dl = ctx.run_steps(60, 8, trace=True, trace_dloss=True)
    assert st.steps == 60
    replay_trace(ref, cfg, 40, ch, dl, 8, ps)
    assert_state_equal(ctx, ref)
    assert_caches_match(ctx, ref)
    ctx.close()


def test_deep_other_class_count(mca):
    """64-256-256-256-12 tanh, 150 samples, K = 8, layer drawn first: twelve
    classes run the general variant of the dense chain and the other kernels."""
    cfg = small_deep(name="deep_c12", widths=(64, 256, 256, 256, 12), n_samples=150)
    banner(f"{cfg.name} {cfg.widths} N={cfg.n_samples}")
    w = mlp_workload(cfg)
    ctx, ref = make_pair(cfg, w, k_max=8)
    L, _ = ctx.loss()
    assert abs(L - ref.loss()) <= REL_TOL * ref.loss()
    ps = ParityStats("deep 64-3x256-12")
    explicit_steps(ctx, ref, cfg, 0, 30, 8, ps)
    assert_state_equal(ctx, ref)
    assert_caches_match(ctx, ref)
    ctx.set_step(30)
    st, ch, dl = ctx.run_steps(30, 8, trace=True, trace_dloss=True)
    replay_trace(ref, cfg, 30, ch, dl, 8, ps)
    assert_state_equal(ctx, ref)
    assert_caches_match(ctx, ref)
    ctx.close()


def test_deep_sparse_images(mca):
    """784-256-256-256-10 tanh on 300 template images (first-layer candidates
    change about 19 % of the samples, listed sparsely), K = 16."""
    cfg = CONFIGS["deep"].scaled(name="deep_img", widths=(784, 256, 256, 256, 10),
                                 n_samples=300, K=16, delta=0.05)
    banner(f"{cfg.name} {cfg.widths} N={cfg.n_samples}")
    w = mlp_workload(cfg)
    ctx, ref = make_pair(cfg, w, k_max=16)
    ps = ParityStats("deep 784-3x256-10 images")
    explicit_steps(ctx, ref, cfg, 0, 30, 16, ps)
    assert_state_equal(ctx, ref)
    assert_caches_match(ctx, ref)
    ctx.set_step(30)
    st, ch, dl = ctx.run_steps(30, 16, trace=True, trace_dloss=True)
    replay_trace(ref, cfg, 30, ch, dl, 16, ps)
    assert_state_equal(ctx, ref)
    assert_caches_match(ctx, ref)
    ctx.close()


@pytest.mark.parametrize("N", [1, 63, 64, 65])
def test_deep_tile_edges(mca, N):
    cfg = small_deep(name=f"deep_n{N}", widths=(64, 256, 256, 256, 10), n_samples=N, K=8)
    w = mlp_workload(cfg)
    ctx, ref = make_pair(cfg, w, k_max=8)
    explicit_steps(ctx, ref, cfg, 0, 20, 8, ParityStats(f"deep 64-3x256-10 N={N}"))
    assert_state_equal(ctx, ref)
    assert_caches_match(ctx, ref)
    ctx.close()


def test_deep_rollback_is_byte_identical(mca):
    cfg = small_deep(name="deep_rb", widths=(64, 256, 256, 256, 10), n_samples=130, K=8)
    w = mlp_workload(cfg)
    ctx, ref = make_pair(cfg, w, k_max=8)
    before_p, _ = ctx.params()
    before_l = ctx.sample_losses()
    for t in range(3):
        cands = ctx.propose(t, 8)
        ctx.eval_losses(cands)
        ctx.rollback()
    after_p, _ = ctx.params()
    for a, b in zip(before_p, after_p):
        assert a.tobytes() == b.tobytes()
    assert before_l.tobytes() == ctx.sample_losses().tobytes()
    ctx.close()


def test_full_deep_workload(mca):
    """784-(24 x 256)-10 tanh on 4,096 samples, K = 32, layer drawn first:
    init loss, one explicit step with every candidate against the incremental
    oracle and the deepest chain candidate against full recomputation, then a
    short device run replayed."""
    cfg = CONFIGS["deep"]
    banner("deep 784-(24x256)-10 N=4096 K=32")
    w = mlp_workload(cfg)
    ctx, ref = make_pair(cfg, w, k_max=32)
    L, _ = ctx.loss()
    assert abs(L - ref.loss()) <= REL_TOL * ref.loss()
    ps = ParityStats("deep 784-24x256-10 full")
    cands = ctx.propose(0, 32)
    losses, dl = ctx.eval_losses(cands)
    L_t, rc, dls, chosen = check_batch(ps, dl, ref, cfg, 0, 32)
    assert_cands_equal(cands, rc)
    # the changes are ~1e-11: resolvable only in difference form
    assert max(abs(d) for d in dls) < 1e-8
    k0 = min(range(32), key=lambda k: rc[k].layer)
    assert rc[k0].layer <= cfg.n_layers - 4
    full = FullMLP(MLPState(w["weights"]), w["X"], w["y"], cfg.act)
    assert abs(losses[k0] - full.eval(rc[k0])) <= REL_TOL * losses[k0]
    ctx.rollback()
    st, ch, dl = ctx.run_steps(3, 32, trace=True, trace_dloss=True)
    assert st.steps == 3
    replay_trace(ref, cfg, 0, ch, dl, 32, ps)
    assert_state_equal(ctx, ref)
    assert_caches_match(ctx, ref)
    ctx.close()
