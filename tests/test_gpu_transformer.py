"""GPU parity of the decoder Transformer path against the fp64 oracle.

Each candidate's loss is the full loss of the net with one parameter changed
(the definition; the oracle recomputes everything in fp64); the device runs
each candidate's forward pass from the first stage its parameter changes.
Workloads: a reduced model (ctx 32, d 64, 2 heads, 2 blocks, 4 sequences)
for explicit steps and a replayed device run, and the full char-level model
(vocab 65, ctx 128, d 128, 4 heads, MLP 512, 2 blocks, 64 sequences) at
K = 16.  Candidate records bit-exact, losses within relative 1e-5, decisions
equal outside the tie band |dL| < 1e-6, committed parameters bit-exact.
"""
import numpy as np
import pytest
import torch

from oracle import mca as omca
from oracle.transformer import TransformerModel
from parity_util import REL_TOL, TIE, ParityStats, assert_cands_equal, check_step

# The device recomputes the reached positions' losses in fp32 and subtracts
# the cached ones; each position's rounding is a few ulp of l_n + max|z| and
# independent of the others, so the floor is 8 ulp of their root-sum-square
# (the oracle's R).
KAPPA_TF = 8.0
from workloads import CONFIGS, transformer_workload

pytestmark = pytest.mark.gpu


def banner(msg):
    print(f"[gpu] {msg}", flush=True)


@pytest.fixture(scope="module")
def mca():
    from paper_2607_08406_amd import mca as m
    m.load_library()
    assert torch.cuda.is_available()
    return m


def make_pair(mca, cfg, k_max):
    w = transformer_workload(cfg)
    desc = mca.transformer_desc(cfg.vocab, cfg.ctx, cfg.d_model, cfg.n_layer, cfg.n_head,
                                cfg.d_mlp, delta=cfg.delta, ln_eps=cfg.ln_eps,
                                accept_ties=cfg.accept_ties, seed=cfg.seed_stream,
                                stream_tag=cfg.stream_tag)
    ctx = mca.TransformerContext(desc, w["params"], w["tokens"], w["targets"], k_max=k_max)
    ref = TransformerModel(w["params"], w["tokens"], w["targets"], cfg.vocab, cfg.ctx,
                           cfg.d_model, cfg.n_layer, cfg.n_head, cfg.d_mlp, cfg.ln_eps)
    return ctx, ref, w


def assert_params_equal(ctx, ref):
    got, _ = ctx.params()
    for t, (a, b) in enumerate(zip(got, ref.params)):
        assert a.tobytes() == b.tobytes(), f"tensor {t} differs"


def explicit_steps(ctx, ref, cfg, t0, n, K, stats):
    accepted = 0
    for t in range(t0, t0 + n):
        cands = ctx.propose(t, K)
        L_t, rc, dls, mags, th, chosen = omca.evaluate_all(ref, t, K, cfg.seed_stream,
                                                           cfg.stream_tag, cfg.delta, "weight",
                                                           cfg.accept_ties)
        assert_cands_equal(cands, rc)
        _, gdl = ctx.eval_losses(cands)
        gch = next((k for k in range(K) if omca.accepts(float(gdl[k]), cfg.accept_ties)), -1)
        take = check_step(stats, gdl, dls, mags, [KAPPA_TF] * K, th, cfg.accept_ties, gch,
                          chosen, tag=f"step {t}")
        if take >= 0:
            ctx.commit(take)
            ref.commit(rc[take], L_t + dls[take])
            accepted += 1
        else:
            ctx.rollback()
    return accepted


def replay(ref, cfg, t0, chosen, dloss, K, stats):
    for n in range(len(chosen)):
        t = t0 + n
        L_t, rc, dls, mags, th, orc = omca.evaluate_all(ref, t, K, cfg.seed_stream,
                                                        cfg.stream_tag, cfg.delta, "weight",
                                                        cfg.accept_ties)
        take = check_step(stats, dloss[n], dls, mags, [KAPPA_TF] * K, th, cfg.accept_ties,
                          int(chosen[n]), orc, tag=f"step {t}")
        if take >= 0:
            ref.commit(rc[take], L_t + dls[take])


def small_cfg(**kw):
    base = dict(name="tf_small", ctx=32, d_model=64, n_layer=2, n_head=2, d_mlp=128, n_seq=4,
                K=8)
    base.update(kw)
    return CONFIGS["transformer"].scaled(**base)


def test_transformer_small_explicit_and_device(mca):
    cfg = small_cfg()
    banner(f"{cfg.name} ctx={cfg.ctx} d={cfg.d_model} heads={cfg.n_head}")
    ctx, ref, _ = make_pair(mca, cfg, k_max=8)
    L, t = ctx.loss()
    assert t == 0 and abs(L - ref.loss()) <= REL_TOL * ref.loss(), (L, ref.loss())
    ps = ParityStats("transformer ctx 32 d 64")
    acc = explicit_steps(ctx, ref, cfg, 0, 25, 8, ps)
    assert acc > 3
    assert_params_equal(ctx, ref)
    ctx.set_step(25)
    st, ch, dl = ctx.run_steps(25, 8, trace=True, trace_dloss=True)
    assert st.steps == 25 and st.evaluated == 25 * 8
    replay(ref, cfg, 25, ch, dl, 8, ps)
    assert_params_equal(ctx, ref)
    L, _ = ctx.loss()
    assert abs(L - ref.loss_of(ref.params)) <= REL_TOL * L
    ctx.close()


@pytest.mark.parametrize("vocab", [100, 128])
def test_transformer_wide_vocabulary(mca, vocab):
    """Vocabularies past 80 symbols take the 128-wide output tile; explicit
    steps and a replayed device run against the oracle."""
    cfg = small_cfg(name=f"tf_vocab{vocab}", vocab=vocab)
    banner(f"{cfg.name} vocab={vocab}")
    ctx, ref, _ = make_pair(mca, cfg, k_max=8)
    L, _ = ctx.loss()
    assert abs(L - ref.loss()) <= REL_TOL * ref.loss(), (L, ref.loss())
    ps = ParityStats(f"transformer vocab {vocab}")
    explicit_steps(ctx, ref, cfg, 0, 8, 8, ps)
    ctx.set_step(8)
    st, ch, dl = ctx.run_steps(8, 8, trace=True, trace_dloss=True)
    replay(ref, cfg, 8, ch, dl, 8, ps)
    assert_params_equal(ctx, ref)
    ctx.close()


@pytest.mark.parametrize("d_model,n_head", [(256, 8), (96, 3), (32, 1)])
def test_transformer_model_widths(mca, d_model, n_head):
    """d_model past 128 (rows held as eight float pairs per lane), an odd head
    count, and a single head: explicit steps and a replayed device run
    against the oracle."""
    cfg = small_cfg(name=f"tf_d{d_model}", ctx=16, d_model=d_model, n_head=n_head, d_mlp=64,
                    n_seq=3)
    banner(f"{cfg.name} d={d_model} heads={n_head}")
    ctx, ref, _ = make_pair(mca, cfg, k_max=8)
    L, _ = ctx.loss()
    assert abs(L - ref.loss()) <= REL_TOL * ref.loss(), (L, ref.loss())
    ps = ParityStats(f"transformer d {d_model} heads {n_head}")
    explicit_steps(ctx, ref, cfg, 0, 8, 8, ps)
    ctx.set_step(8)
    st, ch, dl = ctx.run_steps(8, 8, trace=True, trace_dloss=True)
    replay(ref, cfg, 8, ch, dl, 8, ps)
    assert_params_equal(ctx, ref)
    before = ctx.sample_losses()
    ctx.refresh()
    np.testing.assert_allclose(before, ctx.sample_losses(), rtol=1e-5, atol=1e-6)
    ctx.close()


def test_position_embedding_change_is_causal(mca):
    """A change of pos_emb[p] leaves the loss of every position before p
    bit-identical, and moves the loss by what the oracle says."""
    cfg = small_cfg(name="tf_causal", n_seq=3)
    ctx, ref, _ = make_pair(mca, cfg, k_max=1)
    before = ctx.sample_losses().reshape(cfg.n_seq, cfg.ctx)
    p, c = 11, 5
    cand = np.zeros(1, dtype=mca.CAND_DTYPE)
    cand[0]["layer"], cand[0]["j"], cand[0]["i"] = 1, p, c
    cand[0]["flat"] = cfg.vocab * cfg.d_model + p * cfg.d_model + c
    cand[0]["d"] = np.float32(0.05)
    losses, _ = ctx.eval_losses(cand)
    from oracle.philox import Candidate
    oc = Candidate(int(cand[0]["flat"]), 1, p, c, np.float32(0.05), 0)
    exp = ref.eval(oc)
    assert abs(losses[0] - exp) <= REL_TOL * exp
    ctx.commit(0)
    after = ctx.sample_losses().reshape(cfg.n_seq, cfg.ctx)
    assert after[:, :p].tobytes() == before[:, :p].tobytes()
    assert not np.array_equal(after[:, p:], before[:, p:])
    ctx.close()


def test_transformer_rejects_unsupported(mca):
    cfg = small_cfg()
    w = transformer_workload(cfg)
    for kw, code in [(dict(d_model=48), "MCA_EUNSUPPORTED"), (dict(ctx=256), "MCA_EUNSUPPORTED")]:
        args = dict(vocab=cfg.vocab, ctx=cfg.ctx, d_model=cfg.d_model, n_block=cfg.n_layer,
                    n_head=cfg.n_head, d_mlp=cfg.d_mlp)
        args.update(kw)
        d = mca.transformer_desc(**args, delta=cfg.delta)
        with pytest.raises(mca.MCAError) as e:
            mca.mca_plan(d, cfg.n_seq * args["ctx"], 4)
        assert code in str(e.value)
    bad = w["tokens"].copy()
    bad[0, 0] = cfg.vocab
    desc = mca.transformer_desc(cfg.vocab, cfg.ctx, cfg.d_model, cfg.n_layer, cfg.n_head,
                                cfg.d_mlp, delta=cfg.delta)
    with pytest.raises(mca.MCAError) as e:
        mca.TransformerContext(desc, w["params"], bad, w["targets"], k_max=2)
    assert "MCA_EINVAL" in str(e.value)


def test_full_transformer_workload(mca):
    """vocab 65, ctx 128, d 128, 4 heads, MLP 512, 2 blocks, 64 sequences, K=16:
    init loss, one explicit step against the oracle, one device step replayed."""
    cfg = CONFIGS["transformer"]
    banner("transformer char-LM 64x128 K=16")
    ctx, ref, _ = make_pair(mca, cfg, k_max=16)
    L, _ = ctx.loss()
    assert abs(L - ref.loss()) <= REL_TOL * ref.loss()
    ps = ParityStats("transformer full")
    explicit_steps(ctx, ref, cfg, 0, 2, 16, ps)
    assert_params_equal(ctx, ref)
    ctx.set_step(2)
    st, ch, dl = ctx.run_steps(4, 16, trace=True, trace_dloss=True)
    replay(ref, cfg, 2, ch, dl, 16, ps)
    assert_params_equal(ctx, ref)
    ctx.close()


KIND_TENSORS = ["wout", "bout", "lnf.g", "lnf.b", "h0.wproj", "h0.bproj", "h0.wfc", "h0.bfc",
                "h1.wproj", "h1.wfc", "h1.bfc", "h0.ln2.g", "h1.ln2.b", "h0.wq", "pos_emb",
                "tok_emb", "h0.wfc"]  # the last commit is scored incrementally


def test_commit_of_every_evaluation_kind(mca):
    """One candidate on each kind of tensor -- output layer and its bias,
    final-LayerNorm gain and bias (from the committed logits), MLP
    down-projection and up-projection weights and biases of both blocks
    (from the committed block fields), LN2 gains and biases (from their
    block's MLP half), and dense tensors -- evaluated,
    committed, and followed by a batch from the stream scored against the
    new state: every loss change against the oracle, every committed tensor
    bit-exact, the cached losses (read right after an incrementally scored
    commit) equal to a fresh forward pass's."""
    from workloads import transformer_param_shapes
    cfg = small_cfg(name="tf_kinds", n_seq=3)
    ctx, ref, w = make_pair(mca, cfg, k_max=8)
    names = [n for n, _ in transformer_param_shapes(cfg)]
    shapes = [np.shape(p) for p in w["params"]]
    offs = np.concatenate([[0], np.cumsum([int(np.prod(s)) for s in shapes])])
    rng = np.random.default_rng(7)
    ps = ParityStats("transformer commit of every kind")
    from oracle.philox import Candidate
    for step, name in enumerate(KIND_TENSORS):
        t = names.index(name)
        shp = shapes[t]
        j = int(rng.integers(shp[0]))
        i = int(rng.integers(shp[1])) if len(shp) == 2 else 0
        flat = int(offs[t]) + (j * shp[1] + i if len(shp) == 2 else j)
        cand = np.zeros(1, dtype=mca.CAND_DTYPE)
        cand[0]["flat"], cand[0]["layer"], cand[0]["j"], cand[0]["i"] = flat, t, j, i
        cand[0]["d"] = np.float32(0.03)
        _, gdl = ctx.eval_losses(cand)
        oc = Candidate(flat, t, j, i, np.float32(0.03), 0)
        dl, mag = ref.delta(oc)
        check_step(ps, gdl, [dl], [mag], [KAPPA_TF], [0.0], False, -1, -1, tag=name)
        ctx.commit(0)
        ref.commit(oc, ref.loss() + dl)
        # the stream's next batch against the new state
        cands = ctx.propose(100 + step, 8)
        _, gdl = ctx.eval_losses(cands)
        ctx.rollback()
        L_t, rc, dls, mags, th, _ = omca.evaluate_all(ref, 100 + step, 8, cfg.seed_stream,
                                                      cfg.stream_tag, cfg.delta, "weight",
                                                      cfg.accept_ties)
        assert_cands_equal(cands, rc)
        check_step(ps, gdl, dls, mags, [KAPPA_TF] * 8, th, False, -1, -1, tag=f"after {name}")
    assert_params_equal(ctx, ref)
    L, _ = ctx.loss()
    assert abs(L - ref.loss_of(ref.params)) <= REL_TOL * L
    before = ctx.sample_losses()
    ctx.refresh()
    np.testing.assert_allclose(before, ctx.sample_losses(), rtol=1e-5, atol=1e-6)
    ctx.close()
