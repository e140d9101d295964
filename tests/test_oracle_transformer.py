"""Pins of the fp64 Transformer oracle.

* The loss against a PyTorch CPU fp64 model built from ``F.layer_norm``,
  ``F.scaled_dot_product_attention`` (causal), ``F.gelu(approximate='none')``
  and ``F.cross_entropy`` -- independent library routines.
* Closed form: a zero output layer gives L = ln(vocab).
* Causality: changing the token at position p leaves earlier logits unchanged.
* Eq. 8 for every parameter type: finite differences of the oracle's loss
  against PyTorch autograd.
"""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle.philox import Candidate
from oracle.transformer import TransformerModel, param_layout

SMALL = dict(vocab=11, ctx=8, d=16, n_layer=2, n_head=4, d_mlp=32)
LAYOUT_ARGS = dict(vocab=11, ctx=8, d=16, n_layer=2, d_mlp=32)


def small_model(seed=0, n_seq=3, std=0.3):
    rng = np.random.Generator(np.random.PCG64(seed))
    layout = param_layout(**LAYOUT_ARGS)
    params = []
    for name, shape in layout:
        if name.endswith("_g"):
            p = 1.0 + 0.2 * rng.standard_normal(shape)
        else:
            p = std * rng.standard_normal(shape)
        params.append(p.astype(np.float32))
    toks = rng.integers(0, SMALL["vocab"], size=(n_seq, SMALL["ctx"]))
    tgts = rng.integers(0, SMALL["vocab"], size=(n_seq, SMALL["ctx"]))
    return params, toks, tgts


def torch_reference(params, toks, tgts, requires_grad=False):
    layout = param_layout(**LAYOUT_ARGS)
    P = {n: torch.tensor(np.asarray(p, dtype=np.float64), requires_grad=requires_grad)
         for (n, _), p in zip(layout, params)}
    d, H = SMALL["d"], SMALL["n_head"]
    t = torch.tensor(toks)
    S, T = t.shape
    x = P["tok_emb"][t] + P["pos_emb"][:T]
    for b in range(SMALL["n_layer"]):
        g = lambda n: P[f"h{b}.{n}"]
        h = F.layer_norm(x, (d,), g("ln1_g"), g("ln1_b"), 1e-5)
        q, k, v = (F.linear(h, g(w), g(bb)) for w, bb in (("wq", "bq"), ("wk", "bk"), ("wv", "bv")))
        split = lambda u: u.view(S, T, H, d // H).transpose(1, 2)
        o = F.scaled_dot_product_attention(split(q), split(k), split(v), is_causal=True)
        o = o.transpose(1, 2).reshape(S, T, d)
        x = x + F.linear(o, g("wo"), g("bo"))
        h = F.layer_norm(x, (d,), g("ln2_g"), g("ln2_b"), 1e-5)
        x = x + F.linear(F.gelu(F.linear(h, g("wfc"), g("bfc")), approximate="none"),
                         g("wproj"), g("bproj"))
    x = F.layer_norm(x, (d,), P["lnf_g"], P["lnf_b"], 1e-5)
    z = F.linear(x, P["wout"], P["bout"])
    L = F.cross_entropy(z.reshape(-1, SMALL["vocab"]), torch.tensor(tgts).reshape(-1))
    return L, P, z


def make(params, toks, tgts):
    return TransformerModel(params, toks, tgts, **SMALL)


def test_loss_matches_torch():
    for seed in range(3):
        params, toks, tgts = small_model(seed)
        ref, _, _ = torch_reference(params, toks, tgts)
        ours = make(params, toks, tgts).loss()
        assert abs(ours - ref.item()) <= 1e-12 * ref.item()


def test_zero_head_gives_log_vocab():
    params, toks, tgts = small_model(4)
    layout = param_layout(**LAYOUT_ARGS)
    for n, (name, _) in enumerate(layout):
        if name in ("wout", "bout"):
            params[n][:] = 0
    assert abs(make(params, toks, tgts).loss() - math.log(SMALL["vocab"])) < 1e-15


def test_causality():
    params, toks, tgts = small_model(5)
    m = make(params, toks, tgts)
    z0 = m.logits_of(m.params)
    p = 5
    toks2 = toks.copy()
    toks2[:, p] = (toks2[:, p] + 1) % SMALL["vocab"]
    m2 = make(params, toks2, tgts)
    z1 = m2.logits_of(m2.params)
    np.testing.assert_array_equal(z0[:, :p], z1[:, :p])
    assert np.abs(z0[:, p:] - z1[:, p:]).max() > 1e-6


def test_finite_difference_every_parameter_type():
    params, toks, tgts = small_model(6)
    L, P, _ = torch_reference(params, toks, tgts, requires_grad=True)
    L.backward()
    m = make(params, toks, tgts)
    L0 = m.loss()
    layout = param_layout(**LAYOUT_ARGS)
    rng = np.random.Generator(np.random.PCG64(1))
    for n, (name, shape) in enumerate(layout):
        grad = P[name].grad.numpy()
        for _ in range(3):
            idx = tuple(int(rng.integers(0, s)) for s in shape)
            if name == "tok_emb" and idx[0] not in set(toks.reshape(-1).tolist()):
                continue
            g = grad[idx]
            j, i = (idx[0], idx[1]) if len(shape) == 2 else (idx[0], 0)
            d = np.float32(2e-4)
            c = Candidate(0, n, j, i, d)
            dw = float(m.new_value(c)) - float(params[n][idx])
            fd = (m.eval(c) - L0) / dw
            assert abs(fd - g) <= 2e-3 * max(abs(g), 1e-2), (name, idx, fd, g)


def test_commit_changes_only_that_entry():
    params, toks, tgts = small_model(7)
    m = make(params, toks, tgts)
    c = m.candidate(1, 1, 0, 0, 0.02)
    Lk = m.eval(c)
    before = [p.copy() for p in m.params]
    m.commit(c, Lk)
    for n, (a, b) in enumerate(zip(before, m.params)):
        diff = np.argwhere(a != b)
        if n == c.layer:
            assert len(diff) <= 1
        else:
            assert len(diff) == 0
    assert m.loss() == Lk
    assert abs(make(m.params, toks, tgts).loss() - Lk) == 0.0
