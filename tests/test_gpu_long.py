"""Long parity windows on the full-size workloads (through the C ABI),
against the fp64 oracle: the wide net over 1,000 device steps (64,000
candidates), the deep net over 100 steps and the Transformer over 20 steps
(oracle replicas in worker processes, tests/oracle_pool.py), every traced
loss change compared element by element and every decision replayed; and one
explicit candidate in each of the Transformer's 38 tensors (every embedding,
LayerNorm gain and bias, projection weight and bias), on the reduced and the
full model.
"""
import numpy as np
import pytest
import torch

from oracle.philox import Candidate
from oracle.transformer import TransformerModel
from oracle_pool import OraclePool
from parity_util import ParityStats, assert_state_equal, check_step, make_pair, replay_trace
from workloads import CONFIGS, mlp_workload, transformer_workload

pytestmark = pytest.mark.gpu

KAPPA_TF = 8.0  # as in test_gpu_transformer


def banner(msg):
    print(f"[gpu] {msg}", flush=True)


@pytest.fixture(scope="module")
def mca():
    from paper_2607_08406_amd import mca as m
    m.load_library()
    assert torch.cuda.is_available()
    return m


def test_wide_1000_device_steps(mca):
    cfg = CONFIGS["wide"]
    banner("wide 784-16384-10 N=10000 K=64: 1000 device steps")
    w = mlp_workload(cfg)
    ctx, ref = make_pair(cfg, w, k_max=64)
    ps = ParityStats("wide 784-16384-10 1000 device steps")
    for t0 in range(0, 1000, 250):
        st, ch, dl = ctx.run_steps(250, 64, trace=True, trace_dloss=True)
        assert st.steps == 250
        replay_trace(ref, cfg, t0, ch, dl, 64, ps)
        banner(f"wide replayed to step {t0 + 250}")
    assert_state_equal(ctx, ref)
    L, _ = ctx.loss()
    assert abs(L - ref.loss()) <= 1e-5 * ref.loss()
    ctx.close()


def test_deep_100_device_steps(mca):
    cfg = CONFIGS["deep"]
    banner("deep 784-(24x256)-10 N=4096 K=32: 100 device steps, pooled oracle")
    pool = OraclePool("mlp", cfg)
    try:
        w = mlp_workload(cfg)
        ctx, _ = make_pair(cfg, w.copy(), k_max=32)
        ps = ParityStats("deep 784-24x256-10 100 device steps")
        for t0 in range(0, 100, 25):
            st, ch, dl = ctx.run_steps(25, 32, trace=True, trace_dloss=True)
            replay_trace(pool, cfg, t0, ch, dl, 32, ps)
            banner(f"deep replayed to step {t0 + 25}")
        assert_state_equal(ctx, pool)
        assert ps.n == 3200
        ctx.close()
    finally:
        pool.close()


def tf_pair(mca, cfg, k_max):
    w = transformer_workload(cfg)
    desc = mca.transformer_desc(cfg.vocab, cfg.ctx, cfg.d_model, cfg.n_layer, cfg.n_head,
                                cfg.d_mlp, delta=cfg.delta, ln_eps=cfg.ln_eps,
                                accept_ties=cfg.accept_ties, seed=cfg.seed_stream,
                                stream_tag=cfg.stream_tag)
    ctx = mca.TransformerContext(desc, w["params"], w["tokens"], w["targets"], k_max=k_max)
    return ctx, w


def test_transformer_20_device_steps(mca):
    cfg = CONFIGS["transformer"]
    banner("transformer char-LM 64x128 K=16: 20 device steps, pooled oracle")
    pool = OraclePool("transformer", cfg)
    try:
        ctx, _ = tf_pair(mca, cfg, 16)
        ps = ParityStats("transformer full 20 device steps")
        st, ch, dl = ctx.run_steps(20, 16, trace=True, trace_dloss=True)
        replay_trace(pool, cfg, 0, ch, dl, 16, ps, kappa=lambda c: KAPPA_TF)
        got, _ = ctx.params()
        for a, b in zip(got, pool.state_weights()):
            assert a.tobytes() == b.tobytes()
        ctx.close()
    finally:
        pool.close()


def one_per_tensor(model, shapes, rng, d):
    """One candidate in each tensor: a random entry, increment d."""
    out = []
    flat = 0
    for t, shp in enumerate(shapes):
        size = int(np.prod(shp))
        off = int(rng.integers(0, size))
        if len(shp) == 2:
            j, i = divmod(off, shp[1])
        else:
            j, i = off, 0
        out.append(Candidate(flat + off, t, j, i, np.float32(d)))
        flat += size
    return out


@pytest.mark.parametrize("full", [False, True])
def test_transformer_every_tensor(mca, full):
    cfg = CONFIGS["transformer"] if full else CONFIGS["transformer"].scaled(
        name="tf_small", ctx=32, d_model=64, n_layer=2, n_head=2, d_mlp=128, n_seq=4, K=8)
    banner(f"transformer every tensor full={full}")
    ctx, w = tf_pair(mca, cfg, 38)
    ref = TransformerModel(w["params"], w["tokens"], w["targets"], cfg.vocab, cfg.ctx,
                           cfg.d_model, cfg.n_layer, cfg.n_head, cfg.d_mlp, cfg.ln_eps)
    shapes = [np.shape(p) for p in w["params"]]
    assert len(shapes) == 38
    cands = one_per_tensor(ref, shapes, np.random.Generator(np.random.PCG64(38)), 0.02)
    rec = np.zeros(len(cands), dtype=mca.CAND_DTYPE)
    for n, c in enumerate(cands):
        rec[n]["flat"], rec[n]["layer"], rec[n]["j"], rec[n]["i"] = c.flat, c.layer, c.j, c.i
        rec[n]["d"] = c.d
    _, gdl = ctx.eval_losses(rec)
    ctx.rollback()
    ps = ParityStats(f"transformer every tensor full={full}")
    if full:
        pool = OraclePool("transformer", cfg)
        try:
            res = pool.delta_of(cands)
        finally:
            pool.close()
    else:
        res = [ref.delta(c) for c in cands]
    dls = [r[0] for r in res]
    mags = [r[1] for r in res]
    check_step(ps, gdl, dls, mags, [KAPPA_TF] * len(cands), [0.0] * len(cands), False, -1, -1,
               tag="every tensor")
    # every tensor's candidate moves the loss, except a key bias: it adds the
    # same amount to every score of a query, which the softmax cancels
    for (name, _), d, g in zip(ref.layout, dls, gdl):
        if not name.endswith(".bk"):
            assert d != 0.0 and g != 0.0, name
    ctx.close()
