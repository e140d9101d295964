"""Channel mutation (Sec. 2.3) on the GPU against the fp64 oracle, through the C ABI.

Every width the kernels take (256, 512, 1024: tiles of 64, 32, 16 samples),
nets of two to five layers (rank-1 only, rank-1 then logits, dense layers in
between), ReLU and the other transfer functions, both schemes (re-draw with
the He amplitude, zeroing), a ragged last tile, a weight bound that rejects
some channels, explicit propose / eval / commit / rollback beside the oracle,
device runs replayed on the oracle, and the full-size five-layer
784-1024-1024-1024-10 workload with pooled oracle replicas.

The bar: channel records bit-exact (units and fp32 weights); each loss change
within 1e-5 |dL| + kappa 2^-24 A (parity_util); decisions equal outside the
band fp32 cannot resolve; committed weights bit-exact.
"""
import math

import numpy as np
import pytest
import torch

from oracle.mlp import IncrementalMLP, MLPState
from oracle_pool import OraclePool
from parity_util import (ParityStats, _oracle_step, assert_state_equal, check_step, make_pair,
                         mlp_kappa, replay_trace)
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


def cfg_of(widths, act="relu", scheme="channel_redraw", N=1000, K=8, seed=0, **kw):
    return CONFIGS["channel"].scaled(name=f"channel_{'-'.join(map(str, widths))}",
                                     widths=tuple(widths), act=act, n_samples=N, K=K,
                                     mutation=scheme, seed_stream=4600 + seed, stream_tag=60 + seed,
                                     seed_init=3600 + seed, **kw)


def assert_channels_equal(got, ref, L):
    assert len(got) == len(ref)
    for g, c in zip(got, ref):
        assert tuple(int(u) for u in g["units"][:L + 1]) == tuple(c.units)
        for m in range(L):
            assert np.float32(g["w_new"][m]).tobytes() == np.float32(c.w_new[m]).tobytes()


def explicit_channel_steps(ctx, ref, cfg, t0, n, K, ps, bound=0.0):
    L = len(cfg.widths) - 1
    kap = mlp_kappa(cfg.widths, 0)
    acc = 0
    for t in range(t0, t0 + n):
        chans = ctx.propose_channels(t, K)
        L_t, rc, dls, mags, th, chosen, bounded = _oracle_step(ref, cfg, t, K, bound, 0.0, 0)
        assert_channels_equal(chans, rc, L)
        _, gdl = ctx.eval_channels(chans)
        gch = next((k for k in range(K) if math.isfinite(gdl[k]) and
                    (gdl[k] <= 0.0 if cfg.accept_ties else gdl[k] < 0.0)), -1)
        take = check_step(ps, gdl, dls, mags, [kap] * K, th, cfg.accept_ties, gch, chosen,
                          bounded, tag=f"step {t}")
        if take >= 0:
            ctx.commit(take)
            ref.commit(rc[take], L_t + dls[take])
            acc += 1
        else:
            ctx.rollback()
    return acc


CASES = [
    # widths, act, scheme, N
    ((784, 256, 256, 256, 10), "relu", "channel_redraw", 1000),
    ((784, 256, 256, 256, 10), "relu", "channel_zero", 1000),
    ((784, 512, 512, 512, 10), "relu", "channel_redraw", 700),
    ((784, 1024, 1024, 1024, 10), "relu", "channel_redraw", 600),
    ((784, 1024, 1024, 1024, 10), "relu", "channel_zero", 600),
    ((784, 512, 10), "relu", "channel_redraw", 1000),
    ((784, 256, 256, 10), "relu", "channel_redraw", 1000),
    ((784, 256, 256, 256, 256, 10), "tanh", "channel_redraw", 500),
    ((784, 512, 512, 10), "gauss", "channel_zero", 500),
]


@pytest.mark.parametrize("widths,act,scheme,N", CASES)
def test_channel_explicit_and_device(mca, widths, act, scheme, N):
    cfg = cfg_of(widths, act, scheme, N, gamma=0.4 if act == "gauss" else 1.0)
    banner(f"channel {widths} {act} {scheme} N={N}")
    w = mlp_workload(cfg)
    ctx, ref = make_pair(cfg, w, k_max=cfg.K)
    L0, t = ctx.loss()
    assert t == 0 and abs(L0 - ref.loss()) <= 1e-5 * ref.loss()
    ps = ParityStats(f"channel {'-'.join(map(str, widths))} {act} {scheme} N={N}")
    acc = explicit_channel_steps(ctx, ref, cfg, 0, 6, cfg.K, ps)
    assert_state_equal(ctx, ref)
    ctx.set_step(6)
    st, ch, dl = ctx.run_steps(6, cfg.K, trace=True, trace_dloss=True)
    assert st.steps == 6 and st.evaluated == 6 * cfg.K
    _, acc2 = replay_trace(ref, cfg, 6, ch, dl, cfg.K, ps)
    assert st.accepted == acc2
    assert_state_equal(ctx, ref)
    L1, _ = ctx.loss()
    assert abs(L1 - ref.loss()) <= 1e-5 * ref.loss() + 1e-6
    # the caches after the commits equal a fresh forward pass's
    before = ctx.sample_losses()
    ctx.refresh()
    after = ctx.sample_losses()
    np.testing.assert_allclose(before, after, rtol=2e-5, atol=2e-6)
    assert acc + acc2 >= 1 or scheme == "channel_zero"
    ctx.close()


def test_channel_bound_splits_a_batch(mca):
    """A weight bound (Eq. 1) that some re-drawn channels exceed: those get
    +inf unevaluated, the rest are scored as usual."""
    cfg = cfg_of((784, 256, 256, 10), "relu", "channel_redraw", 800, K=16, seed=3)
    w = mlp_workload(cfg)
    bound = 0.12  # between the He amplitudes sqrt(8/784) = 0.101 and sqrt(8/256) = 0.177
    ctx, ref = make_pair(cfg, w, k_max=16, bound=bound)
    ps = ParityStats("channel bound split")
    n_bounded = 0
    for t in range(4):
        chans = ctx.propose_channels(t, 16)
        _, gdl = ctx.eval_channels(chans)
        ctx.rollback()
        _, rc, dls, mags, th, chosen, bounded = _oracle_step(ref, cfg, t, 16, bound, 0.0, 0)
        n_bounded += sum(bounded)
        check_step(ps, gdl, dls, mags, [mlp_kappa(cfg.widths, 0)] * 16, th, True, -1, -1,
                   bounded, tag=f"bound step {t}")
    assert 0 < n_bounded < 64
    ctx.close()


def test_channel_validation(mca):
    cfg = cfg_of((784, 256, 10), "relu", "channel_redraw", 300, K=4)
    w = mlp_workload(cfg)
    ctx, _ = make_pair(cfg, w, k_max=4)
    chans = ctx.propose_channels(0, 2)
    bad = chans.copy()
    bad[0]["units"][1] = 256
    with pytest.raises(mca.MCAError) as e:
        ctx.eval_channels(bad)
    assert "MCA_EINVAL" in str(e.value)
    bad = chans.copy()
    bad[1]["w_new"][0] = np.inf
    with pytest.raises(mca.MCAError):
        ctx.eval_channels(bad)
    with pytest.raises(mca.MCAError):  # single-mutation calls on a channel context
        ctx.propose(0, 2)
    ctx.eval_channels(chans)
    with pytest.raises(mca.MCAError) as e:
        ctx.eval_channels(chans)
    assert "MCA_ESTATE" in str(e.value)
    ctx.rollback()
    ctx.close()


def test_channel_full_workload(mca):
    """The five-layer 784-1024-1024-1024-10 ReLU workload (N=8192, K=16): one
    explicit step and 4 device steps against pooled oracle replicas."""
    cfg = CONFIGS["channel"]
    banner("channel 784-1024-1024-1024-10 N=8192 K=16, pooled oracle")
    pool = OraclePool("mlp", cfg)
    try:
        w = mlp_workload(cfg)
        ctx, _ = make_pair(cfg, w, k_max=16)
        L0, _ = ctx.loss()
        assert abs(L0 - pool.loss()) <= 1e-5 * pool.loss()
        ps = ParityStats("channel full 784-1024-1024-1024-10")
        explicit_channel_steps(ctx, pool, cfg, 0, 1, 16, ps)
        ctx.set_step(1)
        st, ch, dl = ctx.run_steps(4, 16, trace=True, trace_dloss=True)
        replay_trace(pool, cfg, 1, ch, dl, 16, ps)
        assert_state_equal(ctx, pool)
        ctx.close()
    finally:
        pool.close()


@pytest.mark.parametrize("widths,loop", [((784, 512, 10), 1), ((784, 512, 10), 0),
                                         ((784, 256, 256, 10), 0), ((784, 256, 256, 256, 10), 0)])
def test_relu_single_mutations(mca, widths, loop):
    """ReLU (Sec. 2) through the single-mutation kernels: the persistent loop
    and the per-phase path of a one-hidden-layer net, the slab kernel of two
    hidden layers, the deep chain."""
    cfg = cfg_of(widths, "relu", "single", 900, K=16, seed=5, delta=0.05, layer_pick="layer")
    banner(f"relu single {widths} loop={loop}")
    w = mlp_workload(cfg)
    ctx, ref = make_pair(cfg, w, k_max=16)
    ctx.set_option(mca.MCA_OPT_PERSISTENT_LOOP, loop)
    ps = ParityStats(f"relu single {'-'.join(map(str, widths))} loop={loop}")
    st, ch, dl = ctx.run_steps(12, 16, trace=True, trace_dloss=True)
    _, acc = replay_trace(ref, cfg, 0, ch, dl, 16, ps)
    assert st.accepted == acc
    assert_state_equal(ctx, ref)
    ctx.close()
