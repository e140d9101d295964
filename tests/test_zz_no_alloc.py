"""The no-allocation evaluation entry point (mca_eval_losses_noalloc)
against mca_eval_losses, through the C ABI: on the two-layer, three-layer and
deep paths, two calls in a row (the second with fewer candidates, so the
static scratch holds the first call's larger contents), results equal bit
for bit to the workspace-buffer evaluation; a request beyond the array's size
fails before anything runs; a pending batch of the ordinary path is left
intact."""
import numpy as np
import pytest
import torch

from parity_util import make_pair
from workloads import CONFIGS, mlp_workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def mca():
    from paper_2607_08406_amd import mca as m
    m.load_library()
    assert torch.cuda.is_available()
    return m


CASES = [
    ("wide 784-512-10", CONFIGS["wide"].scaled(name="na_wide", widths=(784, 512, 10),
                                               n_samples=1000), 64, 17),
    ("ternary 784-96-80-10", CONFIGS["ternary"].scaled(name="na_t3", widths=(784, 96, 80, 10),
                                                       n_samples=333), 48, 5),
    ("deep 784-3x256-10", CONFIGS["deep"].scaled(name="na_deep", widths=(784, 256, 256, 256, 10),
                                                 n_samples=300, delta=0.05), 32, 9),
]


@pytest.mark.parametrize("name,cfg,k1,k2", CASES, ids=[c[0] for c in CASES])
def test_noalloc_matches_eval_losses(mca, name, cfg, k1, k2):
    print(f"[gpu] no-alloc {name} K={k1} then K={k2}", flush=True)
    w = mlp_workload(cfg)
    ctx, _ = make_pair(cfg, w, k_max=k1)
    for t, K in ((3, k1), (4, k2)):
        cands = ctx.propose(t, K)
        loss_a, dl_a = mca.mca_eval_losses_noalloc(ctx.ctx, cands)
        loss_b, dl_b = ctx.eval_losses(cands)
        ctx.rollback()
        assert dl_a.tobytes() == dl_b.tobytes(), (t, K)
        assert loss_a.tobytes() == loss_b.tobytes()
        assert np.isfinite(dl_a).all()
    ctx.close()


def test_noalloc_leaves_pending_batch_and_rejects_oversize(mca):
    cfg = CASES[0][1]
    w = mlp_workload(cfg)
    ctx, _ = make_pair(cfg, w, k_max=16)
    cands = ctx.propose(0, 16)
    _, dl = ctx.eval_losses(cands)
    k = int(np.argmin(dl))
    # a no-allocation evaluation in between does not disturb the pending batch
    _, dl2 = mca.mca_eval_losses_noalloc(ctx.ctx, ctx_propose_free(mca, ctx, cands))
    ctx.commit(k)
    L, _ = ctx.loss()
    ref, _ = make_pair(cfg, w, k_max=16)
    ref.eval_losses(cands)
    ref.commit(k)
    assert ctx.loss() == ref.loss()
    for a, b in zip(ctx.params()[0], ref.params()[0]):
        assert a.tobytes() == b.tobytes()
    ref.close()
    ctx.close()
    # deep net at many samples: K x N lists beyond the 8 MiB array
    big = CONFIGS["deep"].scaled(name="na_big", widths=(784, 256, 256, 256, 10), n_samples=40000)
    wb = mlp_workload(big)
    cb, _ = make_pair(big, wb, k_max=4)
    many = np.concatenate([cb.propose(t, 4) for t in range(40)])
    with pytest.raises(mca.MCAError, match="EINVAL"):
        mca.mca_eval_losses_noalloc(cb.ctx, many)
    cb.close()


def ctx_propose_free(mca, ctx, cands):
    """Candidate records without a proposal call (proposing needs no pending
    batch): the same records with a zero increment on the last one."""
    c = cands.copy()
    c[-1]["d"] = 0.0
    return c
