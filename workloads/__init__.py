"""Seeded synthetic workloads for the Monte Carlo mutation-selection (MCA) hot path.

This module only draws inputs: data sets, labels, initial parameters and the
hyper-parameters of each workload.  It holds none of the method's arithmetic
(no mutation, no loss, no selection), so both the fp64 oracle and the HIP
path can consume it without sharing any computation.

The paper trains on MNIST and Tiny Shakespeare (Sec. 2, Sec. 2.5), neither of
which is available here.  The generators below stand in for them with the same
shapes: 28x28 inputs in [0, 1] with about 19 % non-zero pixels and 10 classes,
and a 65-symbol character stream.  Every generator is a pure function of its
seed (numpy PCG64).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional, Tuple

import numpy as np

__all__ = [
    "MLPConfig", "TransformerConfig", "CONFIGS", "get_config",
    "mlp_workload", "transformer_workload", "template_images",
    "markov_tokens", "transformer_param_shapes",
]


# ----------------------------------------------------------------------------
# configurations
# ----------------------------------------------------------------------------

@dataclass(frozen=True)
class MLPConfig:
    """A bias-free fully connected net z_l = W_l a_{l-1}, a_l = phi(z_l).

    widths = (n_0, ..., n_L); W_l has shape (n_l, n_{l-1}), row j = output
    unit, column i = input unit (the W a convention of Sec. 3.6).
    """
    name: str
    widths: Tuple[int, ...]
    act: str                    # "tanh", "relu" or "gauss" (exp(-gamma z^2))
    n_samples: int
    delta: float                # mutation amplitude (learning rate of Eq. 1)
    K: int                      # candidates scored per step
    steps: int                  # length of the timing window
    data: str                   # "sparse_uniform" or "templates"
    init: str                   # "uniform_half", "uniform_fanin", "he", "small", "ternary"
    weight_mode: str = "fp32"   # "fp32" or "ternary"
    layer_pick: str = "weight"  # "weight": uniform over all weights; "layer": layer first
    gamma: float = 1.0
    accept_ties: bool = False   # False: accept iff dL < 0; True: dL <= 0 (Eq. 6)
    mutation: str = "single"    # "single", "channel_redraw" or "channel_zero" (Sec. 2.3)
    biases: bool = False        # augmented weights [W_l | b_l] (Sec. 2.1's deep nets)
    layer_norm: bool = False    # hidden fields normalized over their layer (Sec. 2.1)
    ln_eps: float = 1e-5
    sticky_steps: int = 0       # block length of the "sticky" layer pick (Sec. 2.1)
    seed_data: int = 0
    seed_teacher: int = 0
    seed_init: int = 0
    seed_stream: int = 0
    stream_tag: int = 0
    kind: str = "mlp"

    @property
    def n_layers(self) -> int:
        return len(self.widths) - 1

    @property
    def n_classes(self) -> int:
        return self.widths[-1]

    def layer_sizes(self):
        b = 1 if self.biases else 0
        return [self.widths[l + 1] * (self.widths[l] + b) for l in range(self.n_layers)]

    @property
    def n_params(self) -> int:
        return int(sum(self.layer_sizes()))

    def scaled(self, **kw) -> "MLPConfig":
        d = dict(self.__dict__)
        d.update(kw)
        return MLPConfig(**d)


@dataclass(frozen=True)
class TransformerConfig:
    """Pre-LN causal decoder: tok+pos embedding, n_layer blocks, final LN, head."""
    name: str
    vocab: int
    ctx: int
    d_model: int
    n_layer: int
    n_head: int
    d_mlp: int
    n_seq: int
    delta: float
    K: int
    steps: int
    init_std: float = 0.02
    ln_eps: float = 1e-5
    accept_ties: bool = False
    seed_data: int = 0
    seed_init: int = 0
    seed_stream: int = 0
    stream_tag: int = 0
    kind: str = "transformer"

    @property
    def n_samples(self) -> int:
        return self.n_seq * self.ctx

    @property
    def n_params(self) -> int:
        return int(sum(int(np.prod(s)) for _, s in transformer_param_shapes(self)))

    def scaled(self, **kw) -> "TransformerConfig":
        d = dict(self.__dict__)
        d.update(kw)
        return TransformerConfig(**d)


def _seeds(c: int):
    return dict(seed_data=1000 + c, seed_teacher=2000 + c, seed_init=3000 + c,
                seed_stream=4000 + c, stream_tag=c)


CONFIGS = {
    # 64-32-10 tanh, N=1024, inputs U[0,1) with 80 % zeroed, teacher labels,
    # weights U(-0.5, 0.5), delta 0.1, K=1, 20,000 steps.
    "tiny": MLPConfig(name="tiny", widths=(64, 32, 10), act="tanh", n_samples=1024,
                      delta=0.1, K=1, steps=20000, data="sparse_uniform",
                      init="uniform_half", **_seeds(1)),
    # 784-16384-10 tanh, N=10,000 template images, delta 0.05, K=64.
    "wide": MLPConfig(name="wide", widths=(784, 16384, 10), act="tanh", n_samples=10000,
                      delta=0.05, K=64, steps=5000, data="templates",
                      init="uniform_fanin", **_seeds(2)),
    # 784 -> 24 x 256 -> 10 tanh, N=4096, layer drawn uniformly, delta 0.01, K=32.
    "deep": MLPConfig(name="deep", widths=(784,) + (256,) * 24 + (10,), act="tanh",
                      n_samples=4096, delta=0.01, K=32, steps=500, data="templates",
                      init="uniform_fanin", layer_pick="layer", **_seeds(3)),
    # ternary 784-1024-1024-10, Gaussian transfer exp(-z^2), N=8192, K=64.
    "ternary": MLPConfig(name="ternary", widths=(784, 1024, 1024, 10), act="gauss",
                         n_samples=8192, delta=0.0, K=64, steps=2000, data="templates",
                         init="ternary", weight_mode="ternary", gamma=1.0, **_seeds(4)),
    # char-level decoder: vocab 65, ctx 128, d 128, 2 layers, 4 heads, MLP 512,
    # 64 sequences of 129 tokens from an order-3 Markov chain, delta 0.02, K=16.
    # channel mutation (Sec. 2.3): five layers 784-1024-1024-1024-10, ReLU,
    # He-scaled weights U(-sqrt(8/n), sqrt(8/n)), no biases, no LN; every
    # candidate re-draws one input-to-output path of weights; a candidate is
    # accepted when the loss does not increase; N=8192, K=16.
    "channel": MLPConfig(name="channel", widths=(784, 1024, 1024, 1024, 10), act="relu",
                         n_samples=8192, delta=0.0, K=16, steps=200, data="templates",
                         init="he", accept_ties=True, mutation="channel_redraw", **_seeds(6)),
    # deep net of Sec. 2.1: 784-256-256-256-10 ReLU with a bias per unit and
    # normalized hidden fields, small weights U(-sqrt(0.1/n), sqrt(0.1/n))
    # with n the hidden width, biases 0, delta 0.01; the layer-sticky schedule
    # (blocks of 32 steps); N=8192, K=32.
    "deepln": MLPConfig(name="deepln", widths=(784, 256, 256, 256, 10), act="relu",
                        n_samples=8192, delta=0.01, K=32, steps=200, data="templates",
                        init="small", biases=True, layer_norm=True, layer_pick="sticky",
                        sticky_steps=32, **_seeds(7)),
    "transformer": TransformerConfig(name="transformer", vocab=65, ctx=128, d_model=128,
                                     n_layer=2, n_head=4, d_mlp=512, n_seq=64, delta=0.02,
                                     K=16, steps=200, seed_data=1005, seed_init=3005,
                                     seed_stream=4005, stream_tag=5),
}


def get_config(name: str):
    return CONFIGS[name]


# ----------------------------------------------------------------------------
# 28x28 ten-class template images (stand-in for MNIST)
# ----------------------------------------------------------------------------

def template_images(seed_templates: int, n_classes: int = 10, side: int = 28,
                    support: int = 149):
    """Ten class templates on a 28x28 grid.

    Each class is the pointwise maximum of three Gaussian bumps (centre
    U[4,23]^2, width U[1.5,3] px, amplitude U[0.5,1]); its support is the
    top-`support` pixels (149/784 = 19.0 %), where the template is F/max F.
    Returns (templates[C, side*side] float64, support mask[C, side*side] bool).
    """
    rng = np.random.Generator(np.random.PCG64(seed_templates))
    yy, xx = np.meshgrid(np.arange(side), np.arange(side), indexing="ij")
    T = np.zeros((n_classes, side * side))
    S = np.zeros((n_classes, side * side), dtype=bool)
    for c in range(n_classes):
        F = np.zeros((side, side))
        for _ in range(3):
            cy, cx = rng.uniform(4, 23, size=2)
            sig = rng.uniform(1.5, 3.0)
            amp = rng.uniform(0.5, 1.0)
            F = np.maximum(F, amp * np.exp(-((yy - cy) ** 2 + (xx - cx) ** 2) / (2 * sig * sig)))
        f = F.reshape(-1)
        top = np.argsort(-f, kind="stable")[:support]
        S[c, top] = True
        T[c, top] = f[top] / f.max()
    return T, S


def _template_data(cfg: MLPConfig):
    T, S = template_images(cfg.seed_teacher, n_classes=cfg.n_classes)
    rng = np.random.Generator(np.random.PCG64(cfg.seed_data))
    N = cfg.n_samples
    y = rng.permutation(np.arange(N) % cfg.n_classes).astype(np.int32)
    noise = rng.standard_normal((N, T.shape[1]))
    X = np.where(S[y], np.clip(T[y] + 0.1 * noise, 0.0, 1.0), 0.0)
    return X.astype(np.float32), y


def _sparse_uniform_data(cfg: MLPConfig):
    """Inputs U[0,1) with each entry independently zeroed w.p. 0.8; labels are
    the argmax of a fixed random tanh teacher of the same widths, weights
    U(-0.5, 0.5), no biases, lowest index on ties."""
    rng = np.random.Generator(np.random.PCG64(cfg.seed_data))
    N, n0 = cfg.n_samples, cfg.widths[0]
    X = rng.uniform(0.0, 1.0, size=(N, n0)) * (rng.uniform(size=(N, n0)) < 0.2)
    X = X.astype(np.float32)
    trng = np.random.Generator(np.random.PCG64(cfg.seed_teacher))
    h = X.astype(np.float64)
    for l in range(cfg.n_layers):
        Wt = trng.uniform(-0.5, 0.5, size=(cfg.widths[l + 1], cfg.widths[l]))
        h = h @ Wt.T
        if l < cfg.n_layers - 1:
            h = np.tanh(h)
    y = np.argmax(h, axis=1).astype(np.int32)
    return X, y


def _init_weights(cfg: MLPConfig):
    """Initial parameters.  Returns (weights fp32 list, codes int8 list or None,
    scales fp32 list or None)."""
    rng = np.random.Generator(np.random.PCG64(cfg.seed_init))
    Ws, codes, scales = [], None, None
    if cfg.init == "ternary":
        codes, scales = [], []
        for l in range(cfg.n_layers):
            shape = (cfg.widths[l + 1], cfg.widths[l])
            u = rng.uniform(size=shape)
            c = np.where(u < 0.5, 0, np.where(u < 0.75, -1, 1)).astype(np.int8)
            s = np.float32(1.0 / np.sqrt(cfg.widths[l]))
            codes.append(c)
            scales.append(s)
            Ws.append((c.astype(np.float32) * s).astype(np.float32))
        return Ws, codes, scales
    for l in range(cfg.n_layers):
        shape = (cfg.widths[l + 1], cfg.widths[l])
        if cfg.init == "uniform_half":
            a = 0.5
        elif cfg.init == "small":  # Sec. 2.1: sqrt(0.1 / n), n the hidden width
            a = np.sqrt(0.1 / cfg.widths[1])
        elif cfg.init == "he":  # He scale of Sec. 2.2: sqrt(8 / fan_in)
            a = np.sqrt(8.0 / cfg.widths[l])
        else:
            a = 1.0 / np.sqrt(cfg.widths[l])
        w = rng.uniform(-a, a, size=shape).astype(np.float32)
        if cfg.biases:  # the bias column, starting at zero
            w = np.concatenate([w, np.zeros((shape[0], 1), np.float32)], axis=1)
        Ws.append(w)
    return Ws, None, None


def mlp_workload(cfg: MLPConfig):
    """(X[N, n0] fp32, y[N] int32, weights, codes, scales) for an MLP config."""
    if cfg.data == "templates":
        X, y = _template_data(cfg)
    elif cfg.data == "sparse_uniform":
        X, y = _sparse_uniform_data(cfg)
    else:
        raise ValueError(cfg.data)
    Ws, codes, scales = _init_weights(cfg)
    return dict(X=X, y=y, weights=Ws, codes=codes, scales=scales)


# ----------------------------------------------------------------------------
# order-3 Markov character stream (stand-in for Tiny Shakespeare)
# ----------------------------------------------------------------------------

def markov_tokens(seed: int, n_seq: int, length: int, vocab: int = 65,
                  alpha: float = 0.1):
    """n_seq sequences of `length` symbols from an order-3 Markov chain.

    The first three symbols are uniform; each visited context (a, b, c) gets
    its own transition row p(. | a b c) ~ Dirichlet(alpha * 1_vocab), drawn
    lazily from a generator seeded by (seed, a, b, c).
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    rows = {}
    out = np.zeros((n_seq, length), dtype=np.int32)
    for s in range(n_seq):
        out[s, :3] = rng.integers(0, vocab, size=3)
        for t in range(3, length):
            key = (int(out[s, t - 3]), int(out[s, t - 2]), int(out[s, t - 1]))
            p = rows.get(key)
            if p is None:
                crng = np.random.Generator(np.random.PCG64([seed, *key]))
                p = crng.dirichlet(np.full(vocab, alpha))
                rows[key] = p
            out[s, t] = rng.choice(vocab, p=p)
    return out, rows


def transformer_param_shapes(cfg: TransformerConfig):
    """Canonical parameter order (names, shapes); Linear weights are [out, in]."""
    d, m, v = cfg.d_model, cfg.d_mlp, cfg.vocab
    shapes = [("tok_emb", (v, d)), ("pos_emb", (cfg.ctx, d))]
    for b in range(cfg.n_layer):
        p = f"h{b}."
        shapes += [(p + "ln1.g", (d,)), (p + "ln1.b", (d,)),
                   (p + "wq", (d, d)), (p + "bq", (d,)),
                   (p + "wk", (d, d)), (p + "bk", (d,)),
                   (p + "wv", (d, d)), (p + "bv", (d,)),
                   (p + "wo", (d, d)), (p + "bo", (d,)),
                   (p + "ln2.g", (d,)), (p + "ln2.b", (d,)),
                   (p + "wfc", (m, d)), (p + "bfc", (m,)),
                   (p + "wproj", (d, m)), (p + "bproj", (d,))]
    shapes += [("lnf.g", (d,)), ("lnf.b", (d,)), ("wout", (v, d)), ("bout", (v,))]
    return shapes


def transformer_workload(cfg: TransformerConfig):
    """(tokens[n_seq, ctx] int32, targets[n_seq, ctx] int32, params list fp32)."""
    toks, _ = markov_tokens(cfg.seed_data, cfg.n_seq, cfg.ctx + 1, cfg.vocab)
    rng = np.random.Generator(np.random.PCG64(cfg.seed_init))
    params = []
    for name, shape in transformer_param_shapes(cfg):
        leaf = name.split(".")[-1]
        if leaf == "g":
            p = np.ones(shape)
        elif leaf == "b" or leaf.startswith("b"):
            p = np.zeros(shape)
        else:
            p = rng.standard_normal(shape) * cfg.init_std
        params.append(np.ascontiguousarray(p, dtype=np.float32))
    return dict(tokens=np.ascontiguousarray(toks[:, :-1]),
                targets=np.ascontiguousarray(toks[:, 1:]), params=params)
