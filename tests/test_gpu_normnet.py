"""Deep nets of Sec. 2.1 on the GPU against the fp64 oracle, through the C ABI:
a bias per unit, hidden fields normalized over their layer, and the
layer-sticky schedule; widths 256, 512 and 1024 (tiles of 64, 32, 16 samples),
ReLU, tanh and the Gaussian; explicit propose / eval / commit / rollback
beside the oracle, device runs replayed on it, a candidate forced onto every
layer's bias, pruning candidates with a minibatch (Sec. 2.2's with-LN runs),
and the full-size 784-256-256-256-10 workload with pooled oracle replicas.

The bar (parity_util): candidate records bit-exact; each loss change within
1e-5 |dL| + kappa 2^-24 A with kappa = norm_kappa (128 per normalized layer
and dense product after the candidate's); decisions equal outside the band
fp32 cannot resolve; committed parameters (weights and biases) bit-exact.
"""
import numpy as np
import pytest
import torch

from oracle.philox import Candidate
from oracle_pool import OraclePool
from parity_util import (ParityStats, assert_state_equal, check_step, explicit_steps, make_pair,
                         norm_kappa, replay_trace)
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


def cfg_of(widths, act="relu", ln=True, bias=True, N=1000, K=16, pick="weight", sticky=0,
           seed=0, **kw):
    return CONFIGS["deepln"].scaled(name=f"normnet_{'-'.join(map(str, widths))}",
                                    widths=tuple(widths), act=act, layer_norm=ln, biases=bias,
                                    n_samples=N, K=K, layer_pick=pick, sticky_steps=sticky,
                                    seed_stream=4700 + seed, stream_tag=70 + seed,
                                    seed_init=3700 + seed, **kw)


CASES = [
    # widths, act, ln, bias, N, pick, sticky
    ((784, 256, 256, 256, 10), "relu", True, True, 1000, "weight", 0),
    ((784, 256, 256, 256, 10), "relu", True, True, 1000, "sticky", 4),
    ((784, 512, 512, 10), "relu", True, True, 700, "layer", 0),
    ((784, 1024, 1024, 10), "gauss", True, True, 500, "layer", 0),
    ((784, 256, 256, 10), "relu", False, True, 800, "layer", 0),
    ((784, 256, 256, 256, 10), "tanh", True, False, 600, "layer", 0),
    # plain deep nets (no biases, no normalization) 512 and 1024 wide take
    # the same dense per-layer path
    ((784, 512, 512, 512, 10), "tanh", False, False, 600, "layer", 0),
    ((784, 1024, 1024, 1024, 10), "relu", False, False, 400, "layer", 0),
]


@pytest.mark.parametrize("widths,act,ln,bias,N,pick,sticky", CASES)
def test_normnet_explicit_and_device(mca, widths, act, ln, bias, N, pick, sticky):
    cfg = cfg_of(widths, act, ln, bias, N, pick=pick, sticky=sticky,
                 gamma=0.4 if act == "gauss" else 1.0, delta=0.05)
    banner(f"normnet {widths} {act} ln={ln} bias={bias} N={N} pick={pick}")
    w = mlp_workload(cfg)
    ctx, ref = make_pair(cfg, w, k_max=cfg.K)
    L0, t = ctx.loss()
    assert t == 0 and abs(L0 - ref.loss()) <= 1e-5 * ref.loss()
    ps = ParityStats(f"normnet {'-'.join(map(str, widths))} {act} ln={int(ln)} bias={int(bias)} "
                     f"pick={pick}")
    _, acc = explicit_steps(ctx, ref, cfg, 0, 6, cfg.K, ps)
    assert_state_equal(ctx, ref)
    ctx.set_step(6)
    st, ch, dl = ctx.run_steps(8, cfg.K, trace=True, trace_dloss=True)
    assert st.steps == 8 and st.evaluated == 8 * cfg.K
    _, acc2 = replay_trace(ref, cfg, 6, ch, dl, cfg.K, ps)
    assert st.accepted == acc2
    assert acc + acc2 >= 1
    assert_state_equal(ctx, ref)
    L1, _ = ctx.loss()
    assert abs(L1 - ref.loss()) <= 1e-5 * ref.loss()
    # the caches after the commits equal a fresh forward pass's
    before = ctx.sample_losses()
    ctx.refresh()
    np.testing.assert_allclose(before, ctx.sample_losses(), rtol=3e-5, atol=3e-6)
    ctx.close()


def test_normnet_one_hidden_layer_keeps_the_per_phase_loop(mca):
    """A one-hidden-layer net with biases and normalization is run by the
    per-phase loop even when the persistent-loop option is set to 1 (neither
    device loop kernel takes biases): its device steps replay on the oracle."""
    cfg = cfg_of((784, 256, 10), "relu", True, True, 700, K=8, seed=6, delta=0.05)
    banner("normnet 784-256-10 with the persistent-loop option on")
    w = mlp_workload(cfg)
    ctx, ref = make_pair(cfg, w, k_max=8)
    ctx.set_option(mca.MCA_OPT_PERSISTENT_LOOP, 1)
    ps = ParityStats("normnet 784-256-10 loop option on")
    st, ch, dl = ctx.run_steps(10, 8, trace=True, trace_dloss=True)
    _, acc = replay_trace(ref, cfg, 0, ch, dl, 8, ps)
    assert st.accepted == acc
    assert_state_equal(ctx, ref)
    ctx.close()


def test_normnet_every_bias(mca):
    """A candidate forced onto a bias of every layer (column n_l), the logit
    layer's included, and onto a weight of every layer."""
    widths = (784, 256, 256, 256, 10)
    cfg = cfg_of(widths, "relu", True, True, 900, K=8, seed=2)
    w = mlp_workload(cfg)
    ctx, ref = make_pair(cfg, w, k_max=8)
    shapes = [np.shape(p) for p in w["weights"]]
    cands = []
    off = 0
    rng = np.random.default_rng(11)
    for l, (rows, cols) in enumerate(shapes):
        j = int(rng.integers(rows))
        for i in (cols - 1, int(rng.integers(cols - 1))):
            cands.append(Candidate(off + j * cols + i, l, j, i, np.float32(0.05)))
        off += rows * cols
    rec = np.zeros(len(cands), dtype=mca.CAND_DTYPE)
    for n, c in enumerate(cands):
        rec[n]["flat"], rec[n]["layer"], rec[n]["j"], rec[n]["i"] = c.flat, c.layer, c.j, c.i
        rec[n]["d"] = c.d
    _, gdl = ctx.eval_losses(rec)
    res = [ref.delta(c) for c in cands]
    ps = ParityStats("normnet bias of every layer")
    check_step(ps, gdl, [r[0] for r in res], [r[1] for r in res],
               [norm_kappa(widths, c.layer) for c in cands], [0.0] * len(cands), False, -1, -1,
               tag="every bias")
    # commit the first layer's bias: every sample moves
    ctx.commit(0)
    ref.commit(cands[0], ref.loss() + res[0][0])
    assert_state_equal(ctx, ref)
    ctx.close()


def test_normnet_pruning_with_minibatch(mca):
    """Pruning candidates first in every step and a sample window (Sec. 2.2's
    mixed pruning with normalization)."""
    widths = (784, 256, 256, 10)
    cfg = cfg_of(widths, "relu", True, True, 1000, K=16, seed=4, delta=0.05)
    w = mlp_workload(cfg)
    ctx, ref = make_pair(cfg, w, k_max=16, n_prune=6, subset=(400, 3))
    ps = ParityStats("normnet pruning + minibatch")
    _, acc = explicit_steps(ctx, ref, cfg, 0, 5, 16, ps, n_prune=6, subset=(400, 3))
    ctx.set_step(5)
    st, ch, dl = ctx.run_steps(6, 16, trace=True, trace_dloss=True)
    _, acc2 = replay_trace(ref, cfg, 5, ch, dl, 16, ps, n_prune=6, subset=(400, 3))
    assert st.accepted == acc2
    assert_state_equal(ctx, ref)
    L, _ = ctx.loss()
    assert abs(L - ref.loss()) <= 1e-5 * ref.loss()
    ctx.close()


def test_normnet_validation(mca):
    cfg = cfg_of((784, 256, 10), "relu", True, True, 300, K=4)
    w = mlp_workload(cfg)
    ctx, _ = make_pair(cfg, w, k_max=4)
    c = ctx.propose(0, 2)
    bad = c.copy()
    bad[0]["i"] = 786  # past the bias column
    with pytest.raises(mca.MCAError) as e:
        ctx.eval_losses(bad)
    assert "MCA_EINVAL" in str(e.value)
    with pytest.raises(mca.MCAError):
        mca.mca_eval_losses_noalloc(ctx.ctx, c)
    ctx.close()


def test_normnet_full_workload(mca):
    """784-256-256-256-10 ReLU with biases and normalization, N=8192, K=32,
    the sticky schedule: 2 explicit steps and 12 device steps against pooled
    oracle replicas."""
    cfg = CONFIGS["deepln"]
    banner("deepln 784-256-256-256-10 N=8192 K=32, pooled oracle")
    pool = OraclePool("mlp", cfg)
    try:
        w = mlp_workload(cfg)
        ctx, _ = make_pair(cfg, w, k_max=32)
        assert abs(ctx.loss()[0] - pool.loss()) <= 1e-5 * pool.loss()
        ps = ParityStats("deepln full 784-256-256-256-10")
        explicit_steps(ctx, pool, cfg, 0, 2, 32, ps)
        ctx.set_step(2)
        st, ch, dl = ctx.run_steps(12, 32, trace=True, trace_dloss=True)
        replay_trace(pool, cfg, 2, ch, dl, 32, ps)
        assert_state_equal(ctx, pool)
        ctx.close()
    finally:
        pool.close()
