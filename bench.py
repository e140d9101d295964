"""Throughput of the MCA hot path on one MI355X.

A step is one pass of the whole hot path over the data set: K candidates
proposed from the counter-based stream, each scored incrementally against
the committed state (column update, rank-1 update of the logits, fused
softmax cross-entropy, loss-change reduction), the first improving one
committed.  The default workload is the single-hidden-layer wide net
784-16384-10 (tanh) on 10,000 synthetic 28x28 template images, K = 64.

Prints one JSON line: candidate evaluations per second (value), accepted
mutations per second, the roofline of the dominant kernel from HIP events
recorded on the library's stream during the timed region, and the fp64 CPU
oracle timed on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E
MFMA_FP32_PEAK_TFS = 157.3  # MI355X dense fp32 matrix
VALU_FP32_PEAK_TFS = 157.3  # MI355X fp32 vector (256 CUs x 2.4 GHz x 256 flop/clk, packed FMA)


def algorithmic_bytes_per_step(cfg) -> float:
    """Bytes one evaluation launch must move at least (one step of K candidates).

    Shared by all candidates of the step: the logits (4 N C), the cached
    per-sample losses (4 N) and the labels (N, one byte each).  Per candidate
    in the last hidden layer: the input column and the mutated unit's row of
    local fields (8 N); per candidate in the output layer: the input unit's row
    of local fields (4 N).  Candidates fall in each layer in proportion to its
    size (uniform draw over all weights).
    """
    N, C, K = cfg.n_samples, cfg.n_classes, cfg.K
    sizes = cfg.layer_sizes()
    P = float(sum(sizes))
    shared = 4.0 * N * C + 4.0 * N + N
    per_cand = 0.0
    L = cfg.n_layers
    for l, s in enumerate(sizes):
        per_cand += (s / P) * (8.0 * N if l == L - 2 else 4.0 * N)
    return shared + K * per_cand


def eval_bytes(cfg, cands) -> float:
    """Algorithmic bytes of one batched evaluation launch: the shared logits,
    per-sample losses and labels once, plus each candidate's rows (8 N for a
    last-hidden-layer weight, 4 N for a logit-layer weight)."""
    N, C, L = cfg.n_samples, cfg.n_classes, cfg.n_layers
    rows = sum(8.0 * N if int(c["layer"]) == L - 2 else 4.0 * N for c in cands)
    return 4.0 * N * C + 4.0 * N + N + rows


def incremental_phase(ctx, cfg, step: int, batch: int, reps: int):
    """The incremental phases alone (column update, transfer, rank-1 update of
    the logits, fused cross-entropy and per-tile loss-change sums): the batched
    evaluation kernel scoring `batch` candidates of the stream against one
    committed state, timed with HIP events on the library's stream; every
    batch is rolled back."""
    from paper_2607_08406_amd import mca
    cands = ctx.propose(step, batch)
    ctx.eval_losses(cands)
    ctx.rollback()
    mca.mca_get_timing(ctx.ctx, reset=True)
    mca.mca_set_timing(ctx.ctx, 1 << mca.PHASES.index("eval"))
    for _ in range(reps):
        ctx.eval_losses(cands)
        ctx.rollback()
    ms, launches = mca.mca_get_timing(ctx.ctx, reset=True)
    mca.mca_set_timing(ctx.ctx, 0)
    n = int(launches[mca.PHASES.index("eval")])
    avg_s = ms[mca.PHASES.index("eval")] / 1e3 / max(n, 1)
    b = eval_bytes(cfg, cands)
    achieved = b / avg_s / 1e9
    return {"kernel": "k_eval_tiles", "batch": batch, "launches": n,
            "avg_launch_us": avg_s * 1e6, "candidate_evals_per_s": batch / avg_s,
            "bound": "hbm", "bytes_per_launch": b, "achieved": achieved, "peak": HBM_PEAK_GBS,
            "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
            "traffic": (measured_traffic("k_eval_tiles", f"{cfg.name}_B{batch}", 1)
                        if cfg.name == "wide" else None)}


def candidate_flops(cfg, w, cands, params):
    """Algorithmic flops of scoring one step's candidates on the deep or the
    three-layer net (an FMA counts 2).  A mutation in layers 0..L-4 recomputes,
    for each sample whose activation changes, the rank-1 update of the next
    layer (2 n), the dense layers after it (2 n^2 each) and the logits (2 n C);
    one in layer L-3 moves, per affected sample and per nonzero entry of the
    W_{L-2} column, one unit of the last hidden layer (2) and the C logits
    (2 C).  Affected samples: those with a nonzero input (for layer 0 a pixel
    column of the data; for deeper layers the tanh or Gaussian activation,
    nonzero for every sample)."""
    import numpy as np
    L, C, N = cfg.n_layers, cfg.n_classes, cfg.n_samples
    X = w["X"]
    total = 0.0
    for c in cands:
        l, j, i = int(c["layer"]), int(c["j"]), int(c["i"])
        rows = float(np.count_nonzero(X[:, i])) if l == 0 else float(N)
        if l <= L - 4:
            n = cfg.widths[l + 1]
            total += rows * (2 * n + (L - 3 - l) * 2 * n * n + 2 * n * C)
        elif l == L - 3:
            nnz = float(np.count_nonzero(params[L - 2][:, j]))
            total += rows * nnz * (2 + 2 * C)
    return total


def transformer_flops(cfg, cands):
    """Algorithmic flops of one step's Transformer candidates: each runs the
    forward pass from the stage of its tensor (an embedding change: every
    block; a change in block b: blocks b..; the final LayerNorm or output
    layer: only the output layer).  Per block: Q, K, V and output projections
    (4 x 2 N d^2), causal attention (scores and weighted values over the
    T (T+1) / 2 visible pairs per sequence and head), and the MLP (2 x 2 N d m);
    the output layer 2 N d V."""
    N, D, M, V = cfg.n_samples, cfg.d_model, cfg.d_mlp, cfg.vocab
    T, H, S, NB = cfg.ctx, cfg.n_head, cfg.n_seq, cfg.n_layer
    attn = 2 * 2 * S * H * (T * (T + 1) / 2) * (D // H)
    block = 4 * 2 * N * D * D + attn + 2 * 2 * N * D * M
    out = 2 * N * D * V
    total = 0.0
    for c in cands:
        t = int(c["layer"])
        if t < 2:
            nb = NB
        elif t < 2 + 16 * NB:
            nb = NB - (t - 2) // 16
        else:
            nb = 0
        total += nb * block + out
    return total


# Sources each measured kernel is built from: a traffic record holds only
# while their hash is the one recorded beside the counters.
TRAFFIC_SOURCES = {
    "k_step_loop": ["loop_kernel.hip", "loop_kernel.hpp", "device_common.hpp"],
    "k_eval_tiles": ["mlp_kernels.hip", "mlp_kernels.hpp", "device_common.hpp"],
}


def sources_sha256(kernel: str) -> str:
    import hashlib
    h = hashlib.sha256()
    for f in TRAFFIC_SOURCES[kernel]:
        h.update(open(os.path.join(ROOT, "paper_2607_08406_amd", "csrc", f), "rb").read())
    return h.hexdigest()


def measured_traffic(kernel: str, workload: str, units: float):
    """HBM bytes per launch from the committed rocprofv3 FETCH_SIZE / WRITE_SIZE
    summary (calibrated against a plain copy; per step or per batch, times
    `units`), or None when the kernel source has changed since the counters
    were taken."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_traffic.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    if rec.get("source_sha256") != sources_sha256(kernel):
        return None
    return rec["hbm_bytes_per_unit"] * units


def workload_config(cfg):
    if cfg.kind == "transformer":
        return {"workload": (f"{cfg.name} decoder vocab {cfg.vocab}, ctx {cfg.ctx}, "
                             f"d {cfg.d_model}, {cfg.n_head} heads, MLP {cfg.d_mlp}, "
                             f"{cfg.n_layer} blocks, {cfg.n_seq} sequences, K={cfg.K}, "
                             f"delta={cfg.delta}"),
                "K": cfg.K, "n_samples": cfg.n_samples, "n_params": cfg.n_params}
    return {"workload": (f"{cfg.name} MLP {'-'.join(map(str, cfg.widths))} {cfg.act}, "
                         f"N={cfg.n_samples}, K={cfg.K}, delta={cfg.delta}"),
            "K": cfg.K, "n_samples": cfg.n_samples, "widths": list(cfg.widths),
            "n_params": cfg.n_params}


def cpu_baseline(cfg, w, seconds: float):
    """The fp64 oracle (incremental mode for MLPs, full recomputation for the
    Transformer; all K candidates scored per step, as the device does) on the
    host cores, for about `seconds` of work."""
    import numpy as np
    from threadpoolctl import threadpool_info

    from oracle import mca as omca
    t0 = time.perf_counter()
    if cfg.kind == "transformer":
        from oracle.transformer import TransformerModel
        ref = TransformerModel(w["params"], w["tokens"], w["targets"], cfg.vocab, cfg.ctx,
                               cfg.d_model, cfg.n_layer, cfg.n_head, cfg.d_mlp, cfg.ln_eps)
        ref.loss()
    else:
        from oracle.mlp import IncrementalMLP, MLPState
        ref = IncrementalMLP(MLPState(w["weights"], w["codes"], w["scales"]), w["X"], w["y"],
                             cfg.act, cfg.gamma)
    t_init = time.perf_counter() - t0
    n_steps = 0
    evals = 0
    acc = 0
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < seconds:
        rec = omca.step(ref, n_steps, cfg.K, cfg.seed_stream, cfg.stream_tag, cfg.delta,
                        getattr(cfg, "layer_pick", "weight"), cfg.accept_ties, scan_all=True)
        n_steps += 1
        evals += len(rec.losses)
        acc += rec.chosen >= 0
    el = time.perf_counter() - t0
    blas = [i.get("num_threads") for i in threadpool_info() if i.get("user_api") == "blas"]
    mode = "full-recompute" if cfg.kind == "transformer" else "incremental"
    return {"value": evals / el, "unit": "candidate evals/s", "cores": 1,
            "kind": "oracle",
            "sample": (f"fp64 {mode} oracle, first {n_steps} steps x K={cfg.K} of the "
                       f"same workload from the same seeded init ({el:.1f} s; numpy "
                       f"element-wise work on one thread, BLAS threads {blas} for its "
                       f"matrix products; {t_init:.1f} s setup not timed)"),
            "accepted_per_s": acc / el}


def copy_calibration(nbytes: int):
    """A plain device-to-device copy of nbytes (torch's copy kernel), 5 launches."""
    import torch
    src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": nbytes, "launches": 5}), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5000)
    ap.add_argument("--warmup", type=int, default=200)
    ap.add_argument("--workload", default="wide")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--tile", type=int, default=0, help="samples per workgroup (16..64)")
    ap.add_argument("--per-phase", action="store_true",
                    help="one launch per phase per step instead of the persistent loop")
    ap.add_argument("--eval-batch", type=int, default=1024,
                    help="candidates per launch of the incremental-phase measurement "
                         "(one- and two-layer MLPs; 0 skips it)")
    ap.add_argument("--eval-reps", type=int, default=50)
    ap.add_argument("--copy-bytes", type=int, default=0,
                    help="only run a plain device copy of this many bytes (5 times): the "
                         "reference kernel that calibrates FETCH_SIZE / WRITE_SIZE counters")
    args = ap.parse_args()
    if args.copy_bytes:
        copy_calibration(args.copy_bytes)
        return
    if args.gpus != 1:
        print(f"bench.py runs on exactly one GPU; --gpus {args.gpus} is not supported "
              "(the MCA path here is single-GPU; sharding is a design note only)",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2607_08406_amd import mca
    from workloads import CONFIGS, mlp_workload, transformer_workload

    cfg = CONFIGS[args.workload]
    if cfg.kind == "transformer":
        w = transformer_workload(cfg)
        desc = mca.transformer_desc(cfg.vocab, cfg.ctx, cfg.d_model, cfg.n_layer, cfg.n_head,
                                    cfg.d_mlp, delta=cfg.delta, ln_eps=cfg.ln_eps,
                                    accept_ties=cfg.accept_ties, seed=cfg.seed_stream,
                                    stream_tag=cfg.stream_tag)
        ctx = mca.TransformerContext(desc, w["params"], w["tokens"], w["targets"], k_max=cfg.K)
    else:
        w = mlp_workload(cfg)
        desc = mca.mlp_desc(cfg.widths, cfg.act, gamma=cfg.gamma, delta=cfg.delta,
                            ternary_scales=w["scales"], pick=cfg.layer_pick,
                            accept_ties=cfg.accept_ties, seed=cfg.seed_stream,
                            stream_tag=cfg.stream_tag)
        eval_batch = args.eval_batch if cfg.n_layers <= 2 else 0
        ctx = mca.Context(desc, w["weights"], w["X"], w["y"], k_max=max(cfg.K, eval_batch),
                          codes=w["codes"])
    if args.tile:
        ctx.set_option(mca.MCA_OPT_LOOP_TILE, args.tile)
    if args.per_phase:
        ctx.set_option(mca.MCA_OPT_PERSISTENT_LOOP, 0)
    print(f"[bench] {cfg.name}: context ready, warmup {args.warmup} steps", file=sys.stderr,
          flush=True)
    ctx.run_steps(args.warmup, cfg.K)
    mca.mca_get_timing(ctx.ctx, reset=True)
    # the dominant kernel: the persistent step loop (one launch runs every
    # timed step), or the evaluation kernel when each phase is its own launch
    mca.mca_set_timing(ctx.ctx, (1 << mca.PHASES.index("eval")) | (1 << mca.PHASES.index("step_loop")))
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    st, _, _ = ctx.run_steps(args.steps, cfg.K)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms, launches = mca.mca_get_timing(ctx.ctx, reset=True)
    mca.mca_set_timing(ctx.ctx, 0)
    print(f"[bench] timed {args.steps} steps in {wall:.3f} s", file=sys.stderr, flush=True)

    loop = launches[mca.PHASES.index("step_loop")] > 0
    dominant = mca.PHASES.index("step_loop" if loop else "eval")
    n_launch = max(int(launches[dominant]), 1)
    avg_s = ms[dominant] / 1e3 / n_launch
    if cfg.kind == "transformer":
        t_first = st.next_step - args.steps
        flops = [transformer_flops(cfg, ctx.propose(t_first + n, cfg.K))
                 for n in range(0, args.steps, max(args.steps // 50, 1))]
        per_step = float(np.mean(flops))
        achieved = per_step / avg_s / 1e12
        roof = {"bound": "mfma", "kernel": "eval phase (k_tf_gemm dominant)",
                "achieved": achieved, "peak": MFMA_FP32_PEAK_TFS, "unit": "TFLOP/s",
                "frac": achieved / MFMA_FP32_PEAK_TFS, "traffic": None,
                "flops_per_launch": per_step, "avg_launch_us": avg_s * 1e6,
                "launches": int(launches[dominant])}
    elif cfg.n_layers <= 2:
        kernel = "k_step_loop" if loop else "k_eval_tiles"
        # one loop launch covers all timed steps; one eval launch covers one step
        bytes_launch = algorithmic_bytes_per_step(cfg) * (args.steps / n_launch if loop else 1)
        achieved = bytes_launch / avg_s / 1e9
        roof = {"bound": "hbm", "kernel": kernel, "achieved": achieved, "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                "traffic": (measured_traffic(kernel, "wide", args.steps)
                            if loop and cfg.name == "wide" else None),
                "bytes_per_launch": bytes_launch, "avg_launch_us": avg_s * 1e6,
                "launches": int(launches[dominant]),
                "bytes_per_step": algorithmic_bytes_per_step(cfg)}
    else:
        # the evaluation phase of one step: its candidates' algorithmic flops
        params, _ = ctx.params()
        t_first = st.next_step - args.steps
        flops = [candidate_flops(cfg, w, ctx.propose(t_first + n, cfg.K), params)
                 for n in range(0, args.steps, max(args.steps // 50, 1))]
        per_step = float(np.mean(flops))
        achieved = per_step / avg_s / 1e12
        deep = cfg.n_layers >= 4
        peak = MFMA_FP32_PEAK_TFS if deep else VALU_FP32_PEAK_TFS
        roof = {"bound": "mfma" if deep else "alu",
                "kernel": "eval phase (k_chain dominant)" if deep else "eval phase (k_slab dominant)",
                "achieved": achieved, "peak": peak, "unit": "TFLOP/s", "frac": achieved / peak,
                "traffic": None, "flops_per_launch": per_step, "avg_launch_us": avg_s * 1e6,
                "launches": int(launches[dominant])}
    result = {
        "metric": "candidate loss evals/sec + accepted mutations/sec at 1 GPU; % HBM/MFMA roofline",
        "value": st.evaluated / wall,
        "unit": "candidate evals/s",
        "accepted_per_s": st.accepted / wall,
        "accept_rate_per_step": st.accepted / max(st.steps, 1),
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": wall * 1e3 / args.steps,
        "higher_is_better": True,
        "scaling": "strong",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": workload_config(cfg),
        "roofline": roof,
        "final_loss": st.loss,
    }
    if cfg.kind != "transformer" and eval_batch > 0:
        print(f"[bench] incremental phases: {args.eval_reps} batches of {eval_batch}",
              file=sys.stderr, flush=True)
        result["incremental_phase"] = incremental_phase(ctx, cfg, st.next_step, eval_batch,
                                                        args.eval_reps)
    ctx.close()
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle", file=sys.stderr, flush=True)
        result["cpu_baseline"] = cpu_baseline(cfg, w, args.cpu_seconds)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
