"""GPU parity of the MLP hot path against the fp64 oracle (through the C ABI).

Workloads: the 64-32-10 tanh net (1,024 samples, K=1, the whole 20,000-step
window), a reduced wide net 784-512-10 (1,000 samples: three full 256-sample
tiles and a ragged tail of 232) and the full 784-16384-10 net on 10,000
samples at K=64, in the launch configuration the benchmark times.
"""
import math

import numpy as np
import pytest
import torch

from oracle import mca as omca
from oracle.mlp import FullMLP, IncrementalMLP, MLPState
from parity_util import (REL_TOL, TIE, ParityStats, assert_cands_equal, assert_state_equal,
                         check_batch, explicit_steps, make_pair, mlp_kappa, replay_trace)
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


def small_wide():
    return CONFIGS["wide"].scaled(name="wide_small", widths=(784, 512, 10), n_samples=1000)


def test_tiny_init_and_explicit_steps(mca):
    cfg = CONFIGS["tiny"]
    banner("tiny explicit steps")
    w = mlp_workload(cfg)
    ctx, ref = make_pair(cfg, w, k_max=4)
    L, t = ctx.loss()
    assert t == 0 and abs(L - ref.loss()) <= REL_TOL * ref.loss()
    full = FullMLP(MLPState(w["weights"]), w["X"], w["y"], cfg.act)
    assert abs(L - full.loss()) <= REL_TOL * full.loss()
    st, acc = explicit_steps(ctx, ref, cfg, 0, 300, 4, ParityStats("tiny explicit K=4"))
    assert acc > 50
    assert_state_equal(ctx, ref)
    ctx.close()


@pytest.mark.parametrize("persistent", [1, 0])
def test_tiny_device_loop_full_window(mca, persistent):
    """All 20,000 steps of the tiny workload (K=1) in the device loop, replayed
    on the oracle: every decision equal outside the tie band, weights bit-equal.
    Both the persistent cooperative loop and the one-launch-per-phase loop."""
    cfg = CONFIGS["tiny"]
    banner(f"tiny 20000-step device loop persistent={persistent}")
    w = mlp_workload(cfg)
    ctx, ref = make_pair(cfg, w, k_max=1)
    ctx.set_option(mca.MCA_OPT_PERSISTENT_LOOP, persistent)
    st, chosen, dloss = ctx.run_steps(cfg.steps, 1, trace=True, trace_dloss=True)
    assert st.steps == cfg.steps and st.evaluated == cfg.steps and st.next_step == cfg.steps
    ps, acc = replay_trace(ref, cfg, 0, chosen, dloss, 1,
                           ParityStats(f"tiny 20000 device steps persistent={persistent}"))
    assert acc == st.accepted
    assert ps.flips <= 20
    assert_state_equal(ctx, ref)
    L, _ = ctx.loss()
    assert abs(L - ref.loss()) <= REL_TOL * ref.loss()
    ctx.refresh()
    L2, _ = ctx.loss()
    assert abs(L2 - L) <= 1e-6 * L  # drift of the incremental caches
    ctx.close()


@pytest.mark.parametrize("persistent,tile", [(1, 64), (1, 40), (1, 16), (0, 64)])
def test_small_wide_explicit_and_loop(mca, persistent, tile):
    cfg = small_wide()
    banner(f"wide 784-512-10 N=1000 explicit + loop persistent={persistent} tile={tile}")
    w = mlp_workload(cfg)
    ctx, ref = make_pair(cfg, w, k_max=64)
    ctx.set_option(mca.MCA_OPT_PERSISTENT_LOOP, persistent)
    ctx.set_option(mca.MCA_OPT_LOOP_TILE, tile)
    ps = ParityStats(f"wide 784-512-10 persistent={persistent} tile={tile}")
    _, acc = explicit_steps(ctx, ref, cfg, 0, 40, 64, ps)
    assert acc > 10
    assert_state_equal(ctx, ref)
    assert ctx.loss()[1] == 0  # the explicit path leaves the step counter alone
    ctx.set_step(40)
    st, chosen, dloss = ctx.run_steps(60, 64, trace=True, trace_dloss=True)
    assert st.next_step == 100
    replay_trace(ref, cfg, 40, chosen, dloss, 64, ps)
    assert_state_equal(ctx, ref)
    ctx.close()


def test_ordinary_launch_of_the_loop(mca):
    """The persistent loop with an ordinary launch of its grid (the default)
    and a cooperative one: the same decisions and weights,
    over several calls (the counters of each call, the first step of each
    launch from device state)."""
    cfg = small_wide()
    w = mlp_workload(cfg)
    a, ref = make_pair(cfg, w, k_max=64)
    a.set_option(mca.MCA_OPT_LOOP_LAUNCH, 0)  # cooperative
    b, _ = make_pair(cfg, w, k_max=64)
    b.set_option(mca.MCA_OPT_LOOP_LAUNCH, 1)  # ordinary (the default)
    ps = ParityStats("wide 784-512-10 ordinary and cooperative launch")
    t = 0
    for n in (1, 7, 40):
        sa, ca, da = a.run_steps(n, 64, trace=True, trace_dloss=True)
        sb, cb, db = b.run_steps(n, 64, trace=True, trace_dloss=True)
        assert sa.steps == sb.steps == n and sa.next_step == sb.next_step == t + n
        assert sa.accepted == sb.accepted and sa.evaluated == n * 64
        np.testing.assert_array_equal(ca, cb)
        replay_trace(ref, cfg, t, cb, db, 64, ps)
        t += n
    pa, _ = a.params()
    pb, _ = b.params()
    for x, y in zip(pa, pb):
        assert x.tobytes() == y.tobytes()
    assert_state_equal(b, ref)
    for v in (2, -1):
        with pytest.raises(mca.MCAError, match="EINVAL"):
            b.set_option(mca.MCA_OPT_LOOP_LAUNCH, v)
    a.close()
    b.close()


def test_full_wide_workload(mca):
    """784-16384-10 on 10,000 samples, K=64: init loss, 20 device steps with
    every candidate's dL, replayed on the incremental oracle; two sampled
    candidates against full recomputation."""
    cfg = CONFIGS["wide"]
    banner("wide 784-16384-10 N=10000 K=64")
    w = mlp_workload(cfg)
    ctx, ref = make_pair(cfg, w, k_max=64)
    L, _ = ctx.loss()
    assert abs(L - ref.loss()) <= REL_TOL * ref.loss()
    ps = ParityStats("wide 784-16384-10 full")
    cands = ctx.propose(0, 64)
    losses, dl = ctx.eval_losses(cands)
    L_t, rc, dls, chosen = check_batch(ps, dl, ref, cfg, 0, 64)
    assert_cands_equal(cands, rc)
    full = FullMLP(MLPState(w["weights"]), w["X"], w["y"], cfg.act)
    for k in (0, 1):
        assert abs(losses[k] - full.eval(rc[k])) <= REL_TOL * losses[k]
        d, _ = full.delta(rc[k])
        assert abs(dl[k] - d) <= 1e-5 * abs(d) + 2e-15 * 64, (k, dl[k], d)
    ctx.rollback()
    st, ch, dloss = ctx.run_steps(20, 64, trace=True, trace_dloss=True)
    assert st.steps == 20
    replay_trace(ref, cfg, 0, ch, dloss, 64, ps)
    assert_state_equal(ctx, ref)
    ctx.close()


def test_wide_batched_evaluation(mca):
    """The batched evaluation at the size the benchmark's incremental-phase
    measurement uses: 1,000 candidates of one step of the 784-16384-10 stream
    (40 sample tiles of 256, the last holding 16 samples; 7 or 8 candidates per
    wave) scored in one launch against the committed state, every loss against
    the fp64 oracle, then the first improver committed."""
    cfg = CONFIGS["wide"]
    banner("wide 784-16384-10 N=10000 batched evaluation K=1000")
    w = mlp_workload(cfg)
    K = 1000
    ctx, ref = make_pair(cfg, w, k_max=K)
    cands = ctx.propose(7, K)
    assert sum(int(c["layer"]) == 1 for c in cands) > 0  # logit-layer weights too
    losses, dl = ctx.eval_losses(cands)
    L_t, rc, dls, chosen = check_batch(ParityStats("wide batched K=1000"), dl, ref, cfg, 7, K)
    assert_cands_equal(cands, rc)
    assert chosen >= 0
    ctx.commit(chosen)
    ref.commit(rc[chosen], L_t + dls[chosen])
    assert_state_equal(ctx, ref)
    L, _ = ctx.loss()
    assert abs(L - ref.loss()) <= REL_TOL * ref.loss()
    ctx.close()


@pytest.mark.parametrize("N", [16384, 16424])
def test_batched_evaluation_tile_masks(mca, N):
    """The batched evaluation skips the tiles where a first-layer candidate's
    pixel is zero in every sample, from per-feature masks of up to 64 tiles:
    at 16,384 samples every one of the 64 tiles has its bit (the last is bit
    63); at 16,424 (65 tiles, the last holding 40 samples) there are no masks
    and every tile is scored.  Both against the fp64 oracle."""
    cfg = CONFIGS["wide"].scaled(name="wide_tiles", widths=(784, 64, 10), n_samples=N)
    banner(f"wide 784-64-10 N={N} batched evaluation K=256")
    w = mlp_workload(cfg)
    X = w["X"].copy()
    # a lit pixel of these images is lit somewhere in every tile: blank every
    # third pixel on the odd tiles so that the masks select tiles per feature
    for t in range(1, (N + 255) // 256, 2):
        X[t * 256:(t + 1) * 256, 0::3] = 0.0
    w["X"] = X
    nz = np.array([[np.any(X[t * 256:(t + 1) * 256, i] != 0) for t in range(64)] for i in range(784)])
    assert (nz.any(axis=1) & ~nz.all(axis=1)).sum() > 100
    K = 256
    ctx, ref = make_pair(cfg, w, k_max=K)
    ps = ParityStats(f"wide 784-64-10 N={N} tile masks")
    for step in (0, 5):
        cands = ctx.propose(step, K)
        losses, dl = ctx.eval_losses(cands)
        L_t, rc, dls, chosen = check_batch(ps, dl, ref, cfg, step, K)
        assert_cands_equal(cands, rc)
        ctx.rollback()
    ctx.close()


def test_batched_evaluation_many_tiles(mca):
    """400,000 samples: 1,563 tiles, more than the blocks the GPU holds at
    once, so blocks walk several tiles, one block per tile, and there are no
    tile masks; 264 candidates, so each of a tile's four waves holds 66: two
    passes.  Sampled candidates (both passes, every wave) against the fp64
    oracle one by one."""
    cfg = CONFIGS["wide"].scaled(name="wide_long", widths=(16, 8, 10), n_samples=400_000,
                                 data="sparse_uniform")
    banner("16-8-10 N=400000 batched evaluation K=264")
    w = mlp_workload(cfg)
    K, t = 264, 3
    ctx, ref = make_pair(cfg, w, k_max=K)
    cands = ctx.propose(t, K)
    losses, dl = ctx.eval_losses(cands)
    sample = sorted(set(range(8)) | set(range(248, K)) | set(range(0, K, 17)))
    rc = [ref.candidate(cfg.seed_stream, cfg.stream_tag, t, k, cfg.delta) for k in sample]
    assert_cands_equal([cands[k] for k in sample], rc)
    ps = ParityStats("16-8-10 N=400000 sampled")
    for k, c in zip(sample, rc):
        d, mag = ref.delta(c)
        tol = REL_TOL * abs(d) + mlp_kappa(cfg.widths, c.layer) * 2.0 ** -24 * mag
        assert abs(dl[k] - d) <= tol, (k, dl[k], d)
        ps.n += 1
    ctx.rollback()
    ctx.close()


def test_single_layer_net(mca):
    """A net with no hidden layer (784-10): every candidate is a logit-layer
    weight fed straight by the pixels."""
    cfg = CONFIGS["wide"].scaled(name="linear", widths=(784, 10), n_samples=700, K=100)
    banner("784-10 N=700 explicit steps K=100 and device loop K=64")
    w = mlp_workload(cfg)
    ctx, ref = make_pair(cfg, w, k_max=100)
    ps = ParityStats("784-10 single layer")
    _, acc = explicit_steps(ctx, ref, cfg, 0, 10, 100, ps)
    assert acc > 3
    assert_state_equal(ctx, ref)
    ctx.set_step(10)
    st, ch, dl = ctx.run_steps(20, 64, trace=True, trace_dloss=True)
    replay_trace(ref, cfg, 10, ch, dl, 64, ps)
    assert_state_equal(ctx, ref)
    ctx.close()


@pytest.mark.parametrize("C", [7, 16])
def test_other_class_counts(mca, C):
    """Class counts other than 10 run the kernels' general variants: 784-256-C
    on 600 template images (C templates), explicit steps at K = 64 (batched
    evaluation), then the persistent device loop replayed on the oracle."""
    cfg = CONFIGS["wide"].scaled(name=f"wide_c{C}", widths=(784, 256, C), n_samples=600, K=64)
    banner(f"{cfg.name} {cfg.widths} N={cfg.n_samples}")
    w = mlp_workload(cfg)
    ctx, ref = make_pair(cfg, w, k_max=64)
    L, _ = ctx.loss()
    assert abs(L - ref.loss()) <= REL_TOL * ref.loss()
    ps = ParityStats(f"784-256-{C}")
    _, acc = explicit_steps(ctx, ref, cfg, 0, 20, 64, ps)
    assert acc > 5
    assert_state_equal(ctx, ref)
    ctx.set_step(20)
    st, ch, dl = ctx.run_steps(40, 64, trace=True, trace_dloss=True)
    assert st.steps == 40
    replay_trace(ref, cfg, 20, ch, dl, 64, ps)
    assert_state_equal(ctx, ref)
    L, _ = ctx.loss()
    assert abs(L - ref.loss()) <= REL_TOL * ref.loss()
    ctx.close()


def test_zero_increment_and_bound(mca):
    cfg = small_wide()
    w = mlp_workload(cfg)
    ctx, ref = make_pair(cfg, w, k_max=8)
    cands = ctx.propose(3, 8)
    cands["d"] = 0.0
    losses, dl = ctx.eval_losses(cands)
    assert np.all(dl == 0.0)
    L, _ = ctx.loss()
    assert np.all(losses == L)
    ctx.rollback()
    ctx.close()
    desc = mca.mlp_desc(cfg.widths, cfg.act, delta=cfg.delta, bound=1e-3, seed=cfg.seed_stream,
                        stream_tag=cfg.stream_tag)
    ctx = mca.Context(desc, w["weights"], w["X"], w["y"], k_max=8)
    losses, dl = ctx.eval_losses(ctx.propose(0, 8))
    assert np.all(np.isinf(dl))  # every init weight is far above the bound
    ctx.rollback()
    st, _, _ = ctx.run_steps(5, 8)
    assert st.accepted == 0
    ctx.close()


def test_rollback_is_byte_identical(mca):
    cfg = small_wide()
    w = mlp_workload(cfg)
    ctx, _ = make_pair(cfg, w, k_max=16)
    p0, _ = ctx.params()
    l0 = ctx.sample_losses()
    L0 = ctx.loss()
    ctx.eval_losses(ctx.propose(0, 16))
    ctx.rollback()
    p1, _ = ctx.params()
    for a, b in zip(p0, p1):
        assert a.tobytes() == b.tobytes()
    assert ctx.sample_losses().tobytes() == l0.tobytes()
    assert ctx.loss() == L0
    ctx.close()


def test_error_paths(mca):
    cfg = CONFIGS["tiny"]
    w = mlp_workload(cfg)
    ctx, _ = make_pair(cfg, w, k_max=4)
    with pytest.raises(mca.MCAError, match="ESTATE"):
        ctx.commit(0)
    with pytest.raises(mca.MCAError, match="ESTATE"):
        ctx.rollback()
    with pytest.raises(mca.MCAError, match="EINVAL"):
        ctx.propose(0, 5)
    cands = ctx.propose(0, 4)
    bad = cands.copy()
    bad[1]["j"] = 32
    with pytest.raises(mca.MCAError, match="EINVAL"):
        ctx.eval_losses(bad)
    ctx.eval_losses(cands)
    with pytest.raises(mca.MCAError, match="ESTATE"):
        ctx.eval_losses(cands)
    with pytest.raises(mca.MCAError, match="ESTATE"):
        ctx.run_steps(1, 4)
    with pytest.raises(mca.MCAError, match="EINVAL"):
        ctx.commit(4)
    ctx.commit(3)
    with pytest.raises(mca.MCAError, match="ESTATE"):
        ctx.commit(3)
    for opt, val in [(mca.MCA_OPT_LOOP_TILE, 15), (mca.MCA_OPT_LOOP_TILE, 65),
                     (mca.MCA_OPT_PERSISTENT_LOOP, 2), (99, 1)]:
        with pytest.raises(mca.MCAError, match="EINVAL"):
            ctx.set_option(opt, val)
    ctx.close()
    bad_y = w["y"].copy()
    bad_y[0] = 10
    desc = mca.mlp_desc(cfg.widths, cfg.act, delta=cfg.delta)
    with pytest.raises(mca.MCAError, match="EINVAL"):
        mca.Context(desc, w["weights"], w["X"], bad_y, k_max=1)


def test_resume_is_exact(mca):
    cfg = small_wide()
    w = mlp_workload(cfg)
    a, _ = make_pair(cfg, w, k_max=16)
    a.run_steps(60, 16)
    pa, _ = a.params()
    b, _ = make_pair(cfg, w, k_max=16)
    b.run_steps(30, 16)
    pb, _ = b.params()
    _, t = b.loss()
    c, _ = make_pair(cfg, w, k_max=16)
    c.set_state(pb, None, t)
    c.run_steps(30, 16)
    pc, _ = c.params()
    for x, y in zip(pa, pc):
        assert x.tobytes() == y.tobytes()
    for ctx in (a, b, c):
        ctx.close()


ONE_LOOP_CASES = {
    # name: (config overrides on the tiny family, K, steps, make_pair options)
    "tiny_k2": (dict(), 2, 300, {}),
    "micro_4_3_2": (dict(widths=(4, 3, 2), n_samples=200), 2, 400, {}),
    # 16 inputs: a hidden unit keeps several nonzero codes, so no move maps
    # its field exactly onto its mirror image (where the fp64 oracle's change
    # is exactly zero and fp32 history leaves a residue)
    "small_ternary": (dict(widths=(16, 4, 3), n_samples=300, act="gauss", init="ternary",
                           weight_mode="ternary"), 2, 400, {}),
    "linear_64_10": (dict(widths=(64, 10), n_samples=500), 2, 200, {}),
    "ragged_63": (dict(n_samples=63), 2, 200, {}),
    "single_sample": (dict(n_samples=1), 1, 60, {}),
    "classes_7": (dict(widths=(64, 32, 7), n_samples=700), 2, 200, {}),
    "metropolis": (dict(), 2, 300, dict(beta=3e4)),
    "pruning": (dict(), 2, 300, dict(n_prune=1)),
    "minibatch": (dict(), 2, 200, dict(subset=(256, 5))),
    # one candidate per step: passes of two steps scored against one state
    "tiny_k1": (dict(), 1, 400, {}),
    "micro_k1_odd": (dict(widths=(4, 3, 2), n_samples=200), 1, 401, {}),
    "ternary_k1": (dict(widths=(16, 4, 3), n_samples=300, act="gauss", init="ternary",
                        weight_mode="ternary"), 1, 400, {}),
    "linear_k1": (dict(widths=(64, 10), n_samples=500), 1, 301, {}),
    "metropolis_k1": (dict(), 1, 300, dict(beta=3e4)),
    "pruning_k1": (dict(), 1, 300, dict(n_prune=1)),
    "minibatch_k1": (dict(), 1, 203, dict(subset=(256, 5))),
    # the weight bound of Eq. 1 at half the init range: about half the draws
    # are rejected unevaluated (+inf), in either slot of a pass
    "bound_k1": (dict(), 1, 300, dict(bound=0.25)),
    "bound_k2": (dict(), 2, 200, dict(bound=0.25)),
    # Eq. 6 with <= on one sample: a first-layer draw on one of its zero
    # inputs changes nothing (dL exactly 0) and is accepted
    "ties_k1": (dict(n_samples=1, accept_ties=True), 1, 301, {}),
}


def speculative_waste(chosen, K):
    """Evaluations a run of two-step passes discards: with K = 1, a pass
    whose first step accepts has scored the step after it for nothing."""
    if K != 1:
        return 0
    n, t, waste = len(chosen), 0, 0
    while t < n:
        if chosen[t] >= 0:
            waste += int(t + 1 < n)
            t += 1
        else:
            t += 2
    return waste


@pytest.mark.parametrize("case", sorted(ONE_LOOP_CASES))
def test_one_workgroup_loop(mca, case):
    """Nets whose samples and weights fit one workgroup with at most two
    candidates per step run the one-workgroup loop (sample per thread,
    decision inside the workgroup; with one candidate, passes of two steps
    against one state).  Each case replays the device run on the oracle:
    ragged and single-sample sets, a net without a hidden layer, 7 classes,
    ternary codes on a 16-4-3 net, the Metropolis rule, pruning moves, a
    minibatch window, a weight bound, Eq. 6 with <= on one sample (zero
    changes accepted), and a 4-3-2 net where consecutive candidates share
    weights, units and columns all the time (the patches of a commit into
    the later steps' completed candidates)."""
    over, K, steps, opts = ONE_LOOP_CASES[case]
    cfg = CONFIGS["tiny"].scaled(name=f"one_{case}", K=K, **over)
    banner(f"one-workgroup loop {case}: {cfg.widths} N={cfg.n_samples} K={K} {opts}")
    w = mlp_workload(cfg)
    ctx, ref = make_pair(cfg, w, k_max=K, **opts)
    ps = ParityStats(f"one-workgroup loop {case}")
    st, ch, dl = ctx.run_steps(steps, K, trace=True, trace_dloss=True)
    assert st.steps == steps and st.next_step == steps
    _, acc = replay_trace(ref, cfg, 0, ch, dl, K, ps, **opts)
    assert acc == st.accepted
    assert st.wasted == speculative_waste(list(ch), K)
    if "bound" in opts:  # the bound rejected draws, and not all of them
        assert 0 < int(np.isinf(dl).sum()) < dl.size
    if cfg.accept_ties:  # zero changes occurred and were accepted
        assert any(dl[t, 0] == 0.0 and ch[t] == 0 for t in range(steps))
    assert_state_equal(ctx, ref)
    L, _ = ctx.loss()
    if "subset" not in opts:
        assert abs(L - ref.loss()) <= REL_TOL * ref.loss() + 1e-6
    ctx.close()


@pytest.mark.parametrize("N", [1, 63, 257])
def test_degenerate_sample_counts(mca, N):
    cfg = CONFIGS["tiny"].scaled(n_samples=N)
    w = mlp_workload(cfg)
    ctx, ref = make_pair(cfg, w, k_max=8)
    L, _ = ctx.loss()
    assert abs(L - ref.loss()) <= REL_TOL * ref.loss()
    explicit_steps(ctx, ref, cfg, 0, 20, 8, ParityStats(f"tiny N={N}"))
    assert_state_equal(ctx, ref)
    ctx.close()


def test_gauss_and_ternary_two_layer(mca):
    """Gaussian transfer and ternary codes (Eq. 12) on a two-layer net."""
    base = CONFIGS["ternary"]
    cfg = base.scaled(name="ternary2", widths=(784, 256, 10), n_samples=777, K=32)
    w = mlp_workload(cfg)
    ctx, ref = make_pair(cfg, w, k_max=32)
    ps = ParityStats("ternary 784-256-10 gauss")
    _, acc = explicit_steps(ctx, ref, cfg, 0, 30, 32, ps)
    assert acc > 5
    assert_state_equal(ctx, ref)
    ctx.set_step(30)
    st, ch, dl = ctx.run_steps(30, 32, trace=True, trace_dloss=True)
    replay_trace(ref, cfg, 30, ch, dl, 32, ps)
    assert_state_equal(ctx, ref)
    ctx.close()
