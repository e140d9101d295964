"""Helpers shared by the GPU parity tests: build a context and an oracle from
the same seeded workload, compare candidate records bit for bit, and compare
per-candidate losses and accept decisions.

Parity bar (fp32 GPU vs fp64 oracle): every candidate's loss within relative
1e-5; every accept decision equal unless the oracle's |dL| < 1e-6 (the tie
band, where fp32 rounding may legitimately flip it); candidate indices,
increments and discrete codes bit-exact; continuous weights bit-exact (both
sides apply the same fp32 w').
"""
import numpy as np

from oracle import mca as omca
from oracle.mlp import FullMLP, IncrementalMLP, MLPState

REL_TOL = 1e-5
TIE = 1e-6


def make_pair(cfg, w, k_max, oracle="incremental"):
    from paper_2607_08406_amd import mca
    scales = w["scales"]
    desc = mca.mlp_desc(cfg.widths, cfg.act, gamma=cfg.gamma, delta=cfg.delta,
                        ternary_scales=scales, pick=cfg.layer_pick,
                        accept_ties=cfg.accept_ties, seed=cfg.seed_stream,
                        stream_tag=cfg.stream_tag)
    ctx = mca.Context(desc, w["weights"], w["X"], w["y"], k_max=k_max, codes=w["codes"])
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


def check_losses(gpu_losses, L_t, ref_losses, accept_ties=False):
    """Per-candidate losses and decisions.  Returns the number of tie-band
    disagreements."""
    ties = 0
    for k, (g, r) in enumerate(zip(gpu_losses, ref_losses)):
        assert abs(g - r) <= REL_TOL * abs(r), (k, g, r)
        if omca.accepts(g - L_t, accept_ties) != omca.accepts(r - L_t, accept_ties):
            assert abs(r - L_t) < TIE, (k, g - L_t, r - L_t)
            ties += 1
    return ties


def explicit_steps(ctx, ref, cfg, t0, n_steps, K):
    """propose / eval_losses / commit-or-rollback on the GPU beside the oracle.
    Decisions follow the oracle (teacher forcing inside the tie band)."""
    ties = accepted = 0
    for t in range(t0, t0 + n_steps):
        cands = ctx.propose(t, K)
        L_t, rc, rl, chosen = omca.evaluate(ref, t, K, cfg.seed_stream, cfg.stream_tag,
                                            cfg.delta, cfg.layer_pick, cfg.accept_ties)
        assert_cands_equal(cands, rc)
        losses, dl = ctx.eval_losses(cands)
        ties += check_losses(losses, L_t, rl, cfg.accept_ties)
        if chosen >= 0:
            ctx.commit(chosen)
            ref.commit(rc[chosen], rl[chosen])
            accepted += 1
        else:
            ctx.rollback()
    return ties, accepted


def replay_trace(ref, cfg, t0, chosen, dloss, K):
    """Replay a device run's trace on the oracle.  A device decision may
    differ from the oracle's only inside the tie band; the oracle then follows
    the device (both decisions are valid)."""
    ties = accepted = 0
    for n in range(len(chosen)):
        t = t0 + n
        L_t, rc, rl, orc = omca.evaluate(ref, t, K, cfg.seed_stream, cfg.stream_tag,
                                         cfg.delta, cfg.layer_pick, cfg.accept_ties)
        if dloss is not None:
            for k in range(K):
                g = L_t + dloss[n, k]
                assert abs(g - rl[k]) <= REL_TOL * abs(rl[k]), (t, k, g, rl[k])
                if omca.accepts(dloss[n, k], cfg.accept_ties) != omca.accepts(rl[k] - L_t, cfg.accept_ties):
                    assert abs(rl[k] - L_t) < TIE, (t, k, dloss[n, k], rl[k] - L_t)
        g = int(chosen[n])
        if g != orc:
            # the first candidate on which the two sides decide differently
            m = min(x if x >= 0 else K for x in (g, orc))
            assert abs(rl[m] - L_t) < TIE, (t, m, g, orc, rl[m] - L_t)
            ties += 1
        if g >= 0:
            ref.commit(rc[g], rl[g])
            accepted += 1
    return ties, accepted


def assert_state_equal(ctx, ref):
    params, codes = ctx.params()
    for l, (a, b) in enumerate(zip(params, ref.state.weights)):
        assert a.tobytes() == b.tobytes(), f"weights of layer {l} differ"
    if codes is not None:
        for l, (a, b) in enumerate(zip(codes, ref.state.codes)):
            np.testing.assert_array_equal(a, b)
