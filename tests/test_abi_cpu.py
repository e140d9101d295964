"""The C-ABI library loads, exports every symbol include/mca.h declares, and
its struct layouts match the binding's mirrors.  Validation paths of the pure
planning call run without a GPU; nothing here launches device code."""
import ctypes
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def binding():
    from paper_2607_08406_amd import mca
    if not os.path.exists(mca.LIB_PATH):
        pytest.fail("libmca.so is not built: run __graft_entry__.build() first")
    mca.load_library()
    return mca


def declared_functions():
    names = set()
    for fn in os.listdir(os.path.join(ROOT, "include")):
        if fn.endswith(".h"):
            text = open(os.path.join(ROOT, "include", fn)).read()
            text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
            names |= set(re.findall(r"\b(mca_\w+)\s*\(", text))
    return sorted(names)


def test_exports_every_declared_symbol(binding):
    lib = ctypes.CDLL(binding.LIB_PATH)
    names = declared_functions()
    assert len(names) >= 18
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) <= set(binding._SIGNATURES), set(names) - set(binding._SIGNATURES)


def test_struct_mirrors(binding):
    lib = binding.load_library()
    for n, st in enumerate(binding.STRUCTS):
        assert lib.mca_struct_size(n) == ctypes.sizeof(st)
    assert ctypes.sizeof(binding.mca_cand) == 32 == binding.CAND_DTYPE.itemsize
    assert lib.mca_struct_size(99) == 0
    assert binding.mca_abi_version() == 3


def test_plan_sizes(binding):
    d = binding.mlp_desc((784, 16384, 10), "tanh", delta=0.05)
    b = binding.mca_plan(d, 10000, 64)
    # X^T + W1 + W2 + Z1 + Z2 dominate: 4 * (784*10048 + 784*16384 + 163840 + 16384*10048 + 10*10048)
    core = 4 * (784 * 10048 + 784 * 16384 + 16384 * 10 + 16384 * 10048 + 10 * 10048)
    assert core < b < core + 8 * 2 ** 20
    assert binding.mca_plan(d, 10000, 1) < b


@pytest.mark.parametrize("mutate,code", [
    (dict(n_layers=0), "MCA_EINVAL"),
    (dict(act=7), "MCA_EINVAL"),
    (dict(pick=3), "MCA_EINVAL"),
    (dict(kind=1), "MCA_EINVAL"),  # a Transformer kind without Transformer sizes
    (dict(kind=5), "MCA_EINVAL"),
    (dict(delta=float("nan")), "MCA_EINVAL"),
])
def test_plan_rejects_bad_descriptions(binding, mutate, code):
    d = binding.mlp_desc((64, 32, 10), "tanh", delta=0.1)
    for k, v in mutate.items():
        setattr(d, k, v)
    with pytest.raises(binding.MCAError) as e:
        binding.mca_plan(d, 1024, 1)
    assert code in str(e.value)


def test_plan_layer_limits(binding):
    """Three-layer MLPs up to a 1024-unit second hidden layer are planned, and
    deeper nets with every hidden layer 256 (or all 512, all 1024) wide;
    other shapes are reported as unsupported."""
    d3 = binding.mlp_desc((784, 1024, 1024, 10), "gauss", delta=0.0)
    b3 = binding.mca_plan(d3, 8192, 64)
    # X^T, W_0..W_2, W_1 transposed, Z_0..Z_2 dominate
    core = 4 * (784 * 8192 + 784 * 1024 + 2 * 1024 * 1024 + 10240 + (1024 + 1024 + 10) * 8192)
    assert core < b3 < core + 16 * 2 ** 20
    deep = binding.mlp_desc((784,) + (256,) * 24 + (10,), "tanh", delta=0.01)
    assert binding.mca_plan(deep, 4096, 32) > 4 * 4096 * 256 * 24
    for widths in [(784, 1024, 2048, 10), (64, 32, 32, 32, 10), (64, 256, 512, 256, 10)]:
        d = binding.mlp_desc(widths, "tanh", delta=0.1)
        with pytest.raises(binding.MCAError) as e:
            binding.mca_plan(d, 1024, 8)
        assert "MCA_EUNSUPPORTED" in str(e.value)
    # plain deep nets with every hidden layer 512 or 1024 wide take the dense
    # per-layer path (continuous weights only)
    for w in (512, 1024):
        d = binding.mlp_desc((784, w, w, w, 10), "tanh", delta=0.1)
        assert binding.mca_plan(d, 1024, 8) > 4 * 1024 * w * 3
    d = binding.mlp_desc((784, 512, 512, 512, 10), "tanh", ternary_scales=[0.1] * 4)
    with pytest.raises(binding.MCAError) as e:
        binding.mca_plan(d, 1024, 8)
    assert "MCA_EUNSUPPORTED" in str(e.value)


def test_plan_transformer(binding):
    """The char-level decoder plans; shapes its kernels do not take are
    reported as unsupported, inconsistent sizes as invalid."""
    d = binding.transformer_desc(65, 128, 128, 2, 4, 512, delta=0.02)
    b = binding.mca_plan(d, 64 * 128, 16)
    # committed streams x_0..x_2 and 16 slots of activations dominate
    assert b > 16 * 64 * 128 * 4 * (3 * 128 + 128 * 3 + 3 * 128 + 512)
    for kw, code in [(dict(d_model=96), "MCA_EUNSUPPORTED"), (dict(ctx=256), "MCA_EUNSUPPORTED"),
                     (dict(d_mlp=100), "MCA_EUNSUPPORTED"), (dict(vocab=200), "MCA_EUNSUPPORTED"), (dict(vocab=1), "MCA_EINVAL")]:
        args = dict(vocab=65, ctx=128, d_model=128, n_block=2, n_head=4, d_mlp=512)
        args.update(kw)
        dd = binding.transformer_desc(**args, delta=0.02)
        with pytest.raises(binding.MCAError) as e:
            binding.mca_plan(dd, 64 * args["ctx"], 16)
        assert code in str(e.value)
    with pytest.raises(binding.MCAError) as e:
        binding.mca_plan(d, 64 * 128 + 1, 16)  # not a whole number of sequences
    assert "MCA_EINVAL" in str(e.value)


def test_plan_rejects_bad_sizes(binding):
    d = binding.mlp_desc((64, 32, 10), "tanh", delta=0.1)
    for N, K in [(0, 1), (1024, 0), (1024, 1025)]:
        with pytest.raises(binding.MCAError):
            binding.mca_plan(d, N, K)
    d = binding.mlp_desc((64, 32, 17), "tanh", delta=0.1)
    with pytest.raises(binding.MCAError):
        binding.mca_plan(d, 100, 1)
    d = binding.mlp_desc((4, 3, 2), "gauss", ternary_scales=[0.0, 1.0])
    with pytest.raises(binding.MCAError):
        binding.mca_plan(d, 100, 1)


def test_last_error_message(binding):
    d = binding.mlp_desc((64, 32, 10), "tanh", delta=0.1)
    with pytest.raises(binding.MCAError):
        binding.mca_plan(d, 1024, 5000)
    assert "k_max" in binding.mca_last_error(None)


def test_plan_channel_rules(binding):
    """Channel mutation (Sec. 2.3): hidden layers all 256, 512 or 1024 wide,
    fp32 weights, no pruning candidates, every sample; deep nets of 512 or
    1024 units plan in channel mode although single mutations do not."""
    for w in (256, 512, 1024):
        for mode in ("channel_redraw", "channel_zero"):
            d = binding.mlp_desc((784, w, w, w, 10), "relu", mutation=mode)
            assert binding.mca_plan(d, 8192, 16) > 0
    assert binding.mca_plan(binding.mlp_desc((784, 512, 10), "relu", mutation="channel_zero"),
                            1000, 4) > 0
    bad = [
        (binding.mlp_desc((784, 300, 300, 10), "relu", mutation="channel_redraw"), "MCA_EUNSUPPORTED"),
        (binding.mlp_desc((784, 256, 512, 10), "relu", mutation="channel_redraw"), "MCA_EUNSUPPORTED"),
        (binding.mlp_desc((784, 10), "relu", mutation="channel_redraw"), "MCA_EUNSUPPORTED"),
        (binding.mlp_desc((784, 256, 10), "relu", mutation="channel_redraw", n_prune=2), "MCA_EUNSUPPORTED"),
        (binding.mlp_desc((784, 256, 10), "relu", mutation="channel_redraw", subset_size=100), "MCA_EUNSUPPORTED"),
        (binding.mlp_desc((784, 256, 10), "relu", ternary_scales=[0.1, 0.1], mutation="channel_zero"), "MCA_EUNSUPPORTED"),
    ]
    for d, code in bad:
        with pytest.raises(binding.MCAError) as e:
            binding.mca_plan(d, 1000, 4)
        assert code in str(e.value)
    d = binding.mlp_desc((784, 256, 10), "relu")
    d.mutation = 9
    with pytest.raises(binding.MCAError) as e:
        binding.mca_plan(d, 1000, 4)
    assert "MCA_EINVAL" in str(e.value)
    # single mutations on a deep net of mixed widths stay unsupported
    with pytest.raises(binding.MCAError):
        binding.mca_plan(binding.mlp_desc((784, 512, 1024, 512, 10), "relu"), 1000, 4)
