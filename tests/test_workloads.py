"""Statistics of the seeded synthetic inputs (stand-ins for MNIST and Tiny
Shakespeare): density, class balance, reproducibility, Markov transitions."""
import numpy as np
import pytest

from workloads import (CONFIGS, markov_tokens, mlp_workload, template_images,
                       transformer_param_shapes, transformer_workload)


@pytest.mark.parametrize("name", ["wide", "deep", "ternary"])
def test_template_data_statistics(name):
    cfg = CONFIGS[name]
    w = mlp_workload(cfg)
    X, y = w["X"], w["y"]
    assert X.shape == (cfg.n_samples, 784) and X.dtype == np.float32
    assert 0.17 <= (X != 0).mean() <= 0.21
    assert X.min() >= 0 and X.max() <= 1
    counts = np.bincount(y, minlength=10)
    assert counts.max() - counts.min() <= 1
    T, S = template_images(cfg.seed_teacher)
    assert (S.sum(axis=1) == 149).all()
    # every non-zero pixel lies on the support of the sample's template
    assert not (X != 0)[~S[y]].any()


def test_tiny_data_statistics():
    cfg = CONFIGS["tiny"]
    w = mlp_workload(cfg)
    assert abs((w["X"] != 0).mean() - 0.2) < 0.01
    assert w["X"].shape == (1024, 64)
    assert len(np.unique(w["y"])) >= 5
    assert all(abs(W).max() <= 0.5 for W in w["weights"])


def test_reproducible():
    a = mlp_workload(CONFIGS["tiny"])
    b = mlp_workload(CONFIGS["tiny"])
    np.testing.assert_array_equal(a["X"], b["X"])
    np.testing.assert_array_equal(a["weights"][0], b["weights"][0])


def test_ternary_init():
    cfg = CONFIGS["ternary"]
    w = mlp_workload(cfg)
    for l, (c, s, W) in enumerate(zip(w["codes"], w["scales"], w["weights"])):
        assert abs((c == 0).mean() - 0.5) < 0.01
        assert abs((c == 1).mean() - 0.25) < 0.01
        assert s == np.float32(1.0 / np.sqrt(cfg.widths[l]))
        np.testing.assert_array_equal(W, c.astype(np.float32) * s)


def test_uniform_fanin_init_range():
    cfg = CONFIGS["deep"]
    w = mlp_workload(cfg)
    for l, W in enumerate(w["weights"]):
        a = 1 / np.sqrt(cfg.widths[l])
        assert np.abs(W).max() <= a and np.abs(W).max() > 0.9 * a


def test_markov_chain_transitions():
    toks, rows = markov_tokens(123, 40, 200, vocab=7, alpha=0.5)
    counts = {}
    for s in toks:
        for t in range(3, len(s)):
            key = tuple(int(v) for v in s[t - 3:t])
            counts.setdefault(key, np.zeros(7))[s[t]] += 1
    key = max(counts, key=lambda k: counts[k].sum())
    n = counts[key].sum()
    assert n > 50
    p = rows[key]
    expected = n * p
    mask = expected > 5
    chi2 = (((counts[key] - expected) ** 2 / expected)[mask]).sum()
    assert chi2 < 25


def test_transformer_workload_shapes():
    cfg = CONFIGS["transformer"]
    w = transformer_workload(cfg)
    assert w["tokens"].shape == (64, 128) and w["targets"].shape == (64, 128)
    np.testing.assert_array_equal(w["tokens"][:, 1:], w["targets"][:, :-1])
    assert cfg.n_params == 429889
    assert [p.shape for p in w["params"]] == [s for _, s in transformer_param_shapes(cfg)]
