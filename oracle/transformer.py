"""fp64 oracle of the small causal decoder Transformer and its loss.

Sec. 2.5 trains a four-head Transformer with MCA, choosing every parameter
with equal probability and mutating it within the range of its initial
values; the character-level model is causal with a 65-symbol vocabulary.  The
paper fixes no further detail, so this oracle follows the reading stated in
the design notes: pre-LN blocks h = x + Wo Attn(LN1 x) and
x' = h + Wproj GELU(Wfc LN2 h); learned position embeddings; LayerNorm with
affine gain/bias and eps 1e-5 (biased variance); causal softmax attention with
scale 1/sqrt(d_head); exact (erf) GELU; final LayerNorm; untied output layer
with bias; loss = average next-symbol cross-entropy over every position of
every sequence (Eq. 2, R = 0).  Linear weights are [out, in]: y = x W^T + b.

The loss after a mutation is computed by full recomputation (the definition).
"""
from __future__ import annotations

import numpy as np
from scipy.special import erf

from .philox import Candidate, decode, draw
from .mlp import ce_change, mean_ce, per_sample_ce, softmax


def param_layout(vocab, ctx, d, n_layer, d_mlp):
    """Canonical parameter order: list of (name, shape)."""
    out = [("tok_emb", (vocab, d)), ("pos_emb", (ctx, d))]
    for b in range(n_layer):
        out += [(f"h{b}.ln1_g", (d,)), (f"h{b}.ln1_b", (d,)),
                (f"h{b}.wq", (d, d)), (f"h{b}.bq", (d,)),
                (f"h{b}.wk", (d, d)), (f"h{b}.bk", (d,)),
                (f"h{b}.wv", (d, d)), (f"h{b}.bv", (d,)),
                (f"h{b}.wo", (d, d)), (f"h{b}.bo", (d,)),
                (f"h{b}.ln2_g", (d,)), (f"h{b}.ln2_b", (d,)),
                (f"h{b}.wfc", (d_mlp, d)), (f"h{b}.bfc", (d_mlp,)),
                (f"h{b}.wproj", (d, d_mlp)), (f"h{b}.bproj", (d,))]
    out += [("lnf_g", (d,)), ("lnf_b", (d,)), ("wout", (vocab, d)), ("bout", (vocab,))]
    return out


def layer_norm(x, g, b, eps):
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps) * g + b


def gelu(x):
    """Exact GELU: x * Phi(x) = 0.5 x (1 + erf(x / sqrt 2))."""
    return 0.5 * x * (1.0 + erf(x / np.sqrt(2.0)))


def causal_attention(q, k, v, n_head):
    """Multi-head causal softmax attention on [S, T, d] arrays."""
    S, T, d = q.shape
    dh = d // n_head
    out = np.empty_like(q)
    mask = np.triu(np.ones((T, T), dtype=bool), 1)
    for h in range(n_head):
        sl = slice(h * dh, (h + 1) * dh)
        s = q[:, :, sl] @ k[:, :, sl].transpose(0, 2, 1) / np.sqrt(dh)
        s = np.where(mask, -np.inf, s)
        s = s - s.max(axis=-1, keepdims=True)
        p = np.exp(s)
        p = p / p.sum(axis=-1, keepdims=True)
        out[:, :, sl] = p @ v[:, :, sl]
    return out


class TransformerModel:
    """Committed fp32 parameters of the decoder, evaluated in fp64."""

    def __init__(self, params, tokens, targets, vocab, ctx, d, n_layer, n_head, d_mlp,
                 eps=1e-5):
        self.layout = param_layout(vocab, ctx, d, n_layer, d_mlp)
        assert len(params) == len(self.layout)
        self.params = []
        for p, (name, shape) in zip(params, self.layout):
            p = np.array(p, dtype=np.float32, copy=True)
            assert p.shape == tuple(shape), (name, p.shape, shape)
            self.params.append(p)
        self.tokens = np.asarray(tokens, dtype=np.int64)
        self.targets = np.asarray(targets, dtype=np.int64)
        self.n_layer, self.n_head, self.eps = n_layer, n_head, eps
        self._L = None

    @property
    def shapes(self):
        return [s for _, s in self.layout]

    def logits_of(self, params32):
        P = {name: p.astype(np.float64) for (name, _), p in zip(self.layout, params32)}
        S, T = self.tokens.shape
        x = P["tok_emb"][self.tokens] + P["pos_emb"][:T][None, :, :]
        for b in range(self.n_layer):
            g = lambda n: P[f"h{b}.{n}"]
            h = layer_norm(x, g("ln1_g"), g("ln1_b"), self.eps)
            q = h @ g("wq").T + g("bq")
            k = h @ g("wk").T + g("bk")
            v = h @ g("wv").T + g("bv")
            x = x + causal_attention(q, k, v, self.n_head) @ g("wo").T + g("bo")
            h = layer_norm(x, g("ln2_g"), g("ln2_b"), self.eps)
            x = x + gelu(h @ g("wfc").T + g("bfc")) @ g("wproj").T + g("bproj")
        x = layer_norm(x, P["lnf_g"], P["lnf_b"], self.eps)
        return x @ P["wout"].T + P["bout"]

    def loss_of(self, params32) -> float:
        z = self.logits_of(params32)
        V = z.shape[-1]
        return mean_ce(z.reshape(-1, V), self.targets.reshape(-1))

    def loss(self) -> float:
        if self._L is None:
            self._L = self.loss_of(self.params)
        return self._L

    def candidate(self, seed, tag, t, k, delta, mode="weight") -> Candidate:
        return decode(draw(seed, tag, t, k), self.shapes, delta, mode)

    def _index(self, c: Candidate):
        return (c.j, c.i) if len(self.layout[c.layer][1]) == 2 else (c.j,)

    def new_value(self, c: Candidate) -> np.float32:
        return np.float32(self.params[c.layer][self._index(c)] + c.d)

    def eval(self, c: Candidate) -> float:
        ps = list(self.params)
        p = ps[c.layer].copy()
        p[self._index(c)] = self.new_value(c)
        ps[c.layer] = p
        return self.loss_of(ps)

    def _base(self):
        """The committed logits and per-position losses (kept until a commit)."""
        if getattr(self, "_z0", None) is None:
            z = self.logits_of(self.params)
            V = z.shape[-1]
            self._z0 = z.reshape(-1, V)
            self._l0 = per_sample_ce(self._z0, self.targets.reshape(-1))
        return self._z0, self._l0

    def delta(self, c: Candidate):
        """(dL, R): the loss change by its definition, L(W') - L(W) (Eq. 2),
        here as the mean of the per-position changes of two full fp64
        recomputations (fp64 keeps ~1e-16 of losses near ln 65, far below
        the 1e-6 changes), and R = sqrt(sum_n (l_n + max_c |z_nc|)^2) / N over
        the positions whose loss the change reaches: the size of the
        rounding of an fp32 evaluation that recomputes those positions'
        losses (independent per position, so it adds in quadrature)."""
        z0, l0 = self._base()
        ps = list(self.params)
        p = ps[c.layer].copy()
        p[self._index(c)] = self.new_value(c)
        ps[c.layer] = p
        z1 = self.logits_of(ps).reshape(z0.shape)
        l1 = per_sample_ce(z1, self.targets.reshape(-1))
        moved = np.any(z1 != z0, axis=1)
        N = z0.shape[0]
        size = (l0 + np.abs(z0).max(axis=1))[moved]
        return float((l1 - l0).sum()) / N, float(np.sqrt((size * size).sum())) / N

    def commit(self, c: Candidate, loss_after: float):
        self.params[c.layer][self._index(c)] = self.new_value(c)
        self._L = float(loss_after)
        self._z0 = None
