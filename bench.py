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
# MI355X fp32 vector: 157.3 TFLOP/s with packed (two-wide) FMA; the library is
# built with packed fp32 instructions off, so one FMA per lane per clock:
# 256 CUs x 2.4 GHz x 128 flop/clk = 78.6 TFLOP/s is the reachable ALU peak.
VALU_FP32_PEAK_TFS = 78.6


def algorithmic_bytes_per_step(cfg) -> float:
    """Bytes one evaluation launch must move at least (one step of K candidates).

    Shared by all candidates of the step: the softmax of the logits (4 N C),
    from which each sample's loss change is formed, and the labels (N, one
    byte each).  Per candidate
    in the last hidden layer: the input column and the mutated unit's row of
    local fields (8 N); per candidate in the output layer: the input unit's row
    of local fields (4 N).  Candidates fall in each layer in proportion to its
    size (uniform draw over all weights).
    """
    N, C, K = cfg.n_samples, cfg.n_classes, cfg.K
    sizes = cfg.layer_sizes()
    P = float(sum(sizes))
    shared = 4.0 * N * C + N
    per_cand = 0.0
    L = cfg.n_layers
    for l, s in enumerate(sizes):
        per_cand += (s / P) * (8.0 * N if l == L - 2 else 4.0 * N)
    return shared + K * per_cand


def eval_bytes(cfg, cands) -> float:
    """Algorithmic bytes of one batched evaluation launch: the shared softmax
    rows and labels once, plus each candidate's rows (8 N for a
    last-hidden-layer weight, 4 N for a logit-layer weight)."""
    N, C, L = cfg.n_samples, cfg.n_classes, cfg.n_layers
    rows = sum(8.0 * N if int(c["layer"]) == L - 2 else 4.0 * N for c in cands)
    return 4.0 * N * C + N + rows


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


def dense_path_flops(cfg, cands, channel: bool):
    """Algorithmic flops of one step on the channel-mutation net (Sec. 2.3) or
    the deep net with biases and normalization (Sec. 2.1), an FMA counting 2.
    Every sample changes.  A channel: its first-layer column (2 N), the
    rank-1 term into the second layer (2 N W), a dense product per later
    hidden layer (2 N W^2) and the logits (2 N W C).  A single mutation in
    layer l below the logits: a dense product per later hidden layer
    (2 N W^2) and the logits (2 N W C); in the logit layer: 2 N."""
    L, C, N, W = cfg.n_layers, cfg.n_classes, cfg.n_samples, cfg.widths[1]
    total = 0.0
    for c in cands:
        if channel:
            total += 2 * N + (2 * N * W if L >= 3 else 2 * N * C) + \
                max(0, L - 3) * 2 * N * W * W + (2 * N * W * C if L >= 3 else 0)
        else:
            l = int(c["layer"])
            total += 2 * N if l == L - 1 else (L - 2 - l) * 2 * N * W * W + 2 * N * W * C
    return total


def transformer_flops(cfg, cands):
    """Algorithmic flops of one step's Transformer candidates (an FMA counts
    2).  Per block: Q, K, V and output projections (4 x 2 N d^2), causal
    attention (scores and weighted values over the T (T+1) / 2 visible pairs
    per sequence and head) and the MLP (2 x 2 N d m); the final LayerNorm and
    output layer 2 N d V.  By the candidate's tensor: an embedding or a
    block's LayerNorm or attention tensor recomputes from its block on (every
    block for the embeddings); an MLP weight or bias of block b moves one
    column of x_{b+1} (2 N; an up-projection adds its rank-1 term through
    the down-projection, 2 N d) and recomputes the blocks after b and the
    output layer; an LN2 gain or bias recomputes block b's MLP and the rest; an output-layer or final-LayerNorm parameter moves one
    logit column (2 N) or a rank-1 term into every logit (2 N V).  The
    cross-entropy (about 3 N V) is counted for every candidate."""
    N, D, M, V = cfg.n_samples, cfg.d_model, cfg.d_mlp, cfg.vocab
    T, H, S, NB = cfg.ctx, cfg.n_head, cfg.n_seq, cfg.n_layer
    attn = 2 * 2 * S * H * (T * (T + 1) / 2) * (D // H)
    block = 4 * 2 * N * D * D + attn + 2 * 2 * N * D * M
    out = 2 * N * D * V
    ce = 3 * N * V
    n_tensors = 2 + 16 * NB + 4
    total = 0.0
    for c in cands:
        t = int(c["layer"])
        if t >= n_tensors - 2:
            total += 2 * N + ce
        elif t >= n_tensors - 4:
            total += 2 * N * V + ce
        elif t < 2:
            total += NB * block + out + ce
        else:
            b, role = (t - 2) // 16, (t - 2) % 16
            if role in (14, 15):      # down-projection weight, bias
                total += 2 * N + (NB - 1 - b) * block + out + ce
            elif role in (12, 13):    # up-projection weight, bias
                total += 2 * N + 2 * N * D + (NB - 1 - b) * block + out + ce
            elif role in (10, 11):    # LN2 gain, bias: the block's MLP half on
                total += 2 * 2 * N * D * M + (NB - 1 - b) * block + out + ce
            else:
                total += (NB - b) * block + out + ce
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
    extra = ""
    if cfg.mutation != "single":
        extra += f", {cfg.mutation.replace('_', ' ')} mutations"
    if cfg.biases or cfg.layer_norm:
        extra += (f", {'biases' if cfg.biases else 'no biases'}"
                  f"{', layer-normalized hidden fields' if cfg.layer_norm else ''}")
    if cfg.layer_pick == "sticky":
        extra += f", layer-sticky blocks of {cfg.sticky_steps} steps"
    return {"workload": (f"{cfg.name} MLP {'-'.join(map(str, cfg.widths))} {cfg.act}, "
                         f"N={cfg.n_samples}, K={cfg.K}, delta={cfg.delta}{extra}"),
            "K": cfg.K, "n_samples": cfg.n_samples, "widths": list(cfg.widths),
            "n_params": cfg.n_params}


def host_threads():
    """Cores this process may run on, and the BLAS threads numpy uses."""
    from threadpoolctl import threadpool_info
    cores = len(os.sched_getaffinity(0))
    blas = [i.get("num_threads") for i in threadpool_info() if i.get("user_api") == "blas"]
    return cores, (blas[0] if blas else None)


def oracle_model(cfg, w, mode):
    """The fp64 oracle: "incremental" (its own field-change evaluator) or
    "full" (the definition: every candidate recomputes the whole forward
    pass).  The Transformer oracle has only the full mode."""
    if cfg.kind == "transformer":
        from oracle.transformer import TransformerModel
        return TransformerModel(w["params"], w["tokens"], w["targets"], cfg.vocab, cfg.ctx,
                                cfg.d_model, cfg.n_layer, cfg.n_head, cfg.d_mlp, cfg.ln_eps)
    if cfg.biases or cfg.layer_norm:
        from oracle.normmlp import NormMLP
        return NormMLP(w["weights"], w["X"], w["y"], cfg.act, cfg.gamma, bias=cfg.biases,
                       ln=cfg.layer_norm, eps=cfg.ln_eps, sticky=cfg.sticky_steps)
    from oracle.mlp import FullMLP, IncrementalMLP, MLPState
    cls = IncrementalMLP if mode == "incremental" else FullMLP
    return cls(MLPState(w["weights"], w["codes"], w["scales"]), w["X"], w["y"], cfg.act, cfg.gamma)


def cpu_baseline(cfg, w, seconds: float, mode: str, scan_all: bool):
    """The fp64 oracle as it stands, on the host cores, for about `seconds`
    of work (at least one candidate).  scan_all: score all K candidates of
    each step (what the device does); otherwise stop at the first one that
    passes, the paper's sequential method."""
    from oracle import mca as omca
    t0 = time.perf_counter()
    ref = oracle_model(cfg, w, mode)
    ref.loss()
    t_init = time.perf_counter() - t0
    n_steps = evals = acc = 0
    pick = getattr(cfg, "layer_pick", "weight")
    if getattr(cfg, "mutation", "single") != "single":
        pick = cfg.mutation  # channel candidates (Sec. 2.3)
    t0 = time.perf_counter()
    while evals == 0 or time.perf_counter() - t0 < seconds:
        rec = omca.step(ref, n_steps, cfg.K, cfg.seed_stream, cfg.stream_tag, cfg.delta,
                        pick, cfg.accept_ties, scan_all=scan_all)
        n_steps += 1
        evals += len(rec.losses)
        acc += rec.chosen >= 0
    el = time.perf_counter() - t0
    cores, blas = host_threads()
    label = {"incremental": "fp64 incremental oracle", "full": "fp64 full-recompute oracle"}[
        "full" if cfg.kind == "transformer" else mode]
    return {"value": evals / el, "unit": "candidate evals/s", "cores": cores,
            "blas_threads": blas, "kind": "oracle", "mode": mode if cfg.kind != "transformer" else "full",
            "scan": "all K" if scan_all else "stop at first improver",
            "sample": (f"{label}, first {n_steps} step(s) x K={cfg.K} "
                       f"({'all scored' if scan_all else 'until the first improver'}) of the same "
                       f"workload from the same seeded init ({el:.1f} s; {t_init:.1f} s setup "
                       f"not timed)"),
            "accepted_per_s": acc / el}


def make_context(cfg, w, k_max, args):
    from paper_2607_08406_amd import mca
    if cfg.kind == "transformer":
        desc = mca.transformer_desc(cfg.vocab, cfg.ctx, cfg.d_model, cfg.n_layer, cfg.n_head,
                                    cfg.d_mlp, delta=cfg.delta, ln_eps=cfg.ln_eps,
                                    accept_ties=cfg.accept_ties, seed=cfg.seed_stream,
                                    stream_tag=cfg.stream_tag)
        return mca.TransformerContext(desc, w["params"], w["tokens"], w["targets"], k_max=k_max)
    desc = mca.mlp_desc(cfg.widths, cfg.act, gamma=cfg.gamma, delta=cfg.delta,
                        ternary_scales=w["scales"], pick=cfg.layer_pick,
                        accept_ties=cfg.accept_ties, seed=cfg.seed_stream,
                        stream_tag=cfg.stream_tag, mutation=cfg.mutation, biases=cfg.biases,
                        layer_norm=cfg.layer_norm, ln_eps=cfg.ln_eps,
                        sticky_steps=cfg.sticky_steps)
    ctx = mca.Context(desc, w["weights"], w["X"], w["y"], k_max=k_max, codes=w["codes"])
    if args.tile:
        ctx.set_option(mca.MCA_OPT_LOOP_TILE, args.tile)
    if args.per_phase:
        ctx.set_option(mca.MCA_OPT_PERSISTENT_LOOP, 0)
    if args.cooperative:
        ctx.set_option(mca.MCA_OPT_LOOP_LAUNCH, 0)
    return ctx


def load_workload(cfg):
    from workloads import mlp_workload, transformer_workload
    return transformer_workload(cfg) if cfg.kind == "transformer" else mlp_workload(cfg)


def measure(cfg, w, steps, warmup, args, eval_batch=0):
    """Time `steps` device steps after `warmup`; returns the result object
    (throughput, roofline of the dominant kernel) and the context."""
    import numpy as np
    import torch

    from paper_2607_08406_amd import mca
    ctx = make_context(cfg, w, max(cfg.K, eval_batch), args)
    # the dominant kernel: the persistent step loop (one launch runs every
    # timed step), or the evaluation phase when each phase is its own launch
    mask = ((1 << mca.PHASES.index("eval")) | (1 << mca.PHASES.index("step_loop"))
            | (1 << mca.PHASES.index("one_loop")))
    # the timers are on from the warmup, which then runs the timed call's
    # exact path (its events made and recorded once); host work between the
    # warmup and the timed call is kept short, since an idle GPU takes longer
    # over the steps that follow
    mca.mca_set_timing(ctx.ctx, mask)
    if warmup:
        ctx.run_steps(warmup, cfg.K)
    mca.mca_get_timing(ctx.ctx, reset=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    st, _, _ = ctx.run_steps(steps, cfg.K)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms, launches = mca.mca_get_timing(ctx.ctx, reset=True)
    mca.mca_set_timing(ctx.ctx, 0)
    one = launches[mca.PHASES.index("one_loop")] > 0
    loop = one or launches[mca.PHASES.index("step_loop")] > 0
    dominant = mca.PHASES.index("one_loop" if one else "step_loop" if loop else "eval")
    n_launch = max(int(launches[dominant]), 1)
    avg_s = ms[dominant] / 1e3 / n_launch
    t_first = st.next_step - steps
    sample = range(0, steps, max(steps // 40, 1))
    if cfg.kind == "transformer":
        per_step = float(np.mean([transformer_flops(cfg, ctx.propose(t_first + n, cfg.K))
                                  for n in sample]))
        achieved = per_step / avg_s / 1e12
        roof = {"bound": "mfma", "kernel": "eval phase (k_tf_gemm dominant)",
                "achieved": achieved, "peak": MFMA_FP32_PEAK_TFS, "unit": "TFLOP/s",
                "frac": achieved / MFMA_FP32_PEAK_TFS, "traffic": None,
                "flops_per_launch": per_step}
    elif cfg.mutation != "single" or cfg.biases or cfg.layer_norm:
        channel = cfg.mutation != "single"
        per_step = float(np.mean([
            dense_path_flops(cfg, ctx.propose_channels(t_first + n, cfg.K) if channel
                             else ctx.propose(t_first + n, cfg.K), channel) for n in sample]))
        achieved = per_step / avg_s / 1e12
        roof = {"bound": "mfma", "kernel": "eval phase (k_channel)" if channel
                else "eval phase (k_norm)", "achieved": achieved, "peak": MFMA_FP32_PEAK_TFS,
                "unit": "TFLOP/s", "frac": achieved / MFMA_FP32_PEAK_TFS, "traffic": None,
                "flops_per_launch": per_step}
    elif cfg.n_layers <= 2:
        kernel = "k_one_loop" if one else "k_step_loop" if loop else "k_eval_tiles"
        # one loop launch covers all timed steps; one eval launch covers one step
        bytes_launch = algorithmic_bytes_per_step(cfg) * (steps / n_launch if loop else 1)
        achieved = bytes_launch / avg_s / 1e9
        roof = {"bound": "hbm" if cfg.name != "tiny" else "latency", "kernel": kernel,
                "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": achieved / HBM_PEAK_GBS,
                "traffic": (measured_traffic(kernel, cfg.name, steps)
                            if loop and cfg.name == "wide" else None),
                "bytes_per_launch": bytes_launch,
                "bytes_per_step": algorithmic_bytes_per_step(cfg)}
    else:
        params, _ = ctx.params()
        per_step = float(np.mean([candidate_flops(cfg, w, ctx.propose(t_first + n, cfg.K), params)
                                  for n in sample]))
        achieved = per_step / avg_s / 1e12
        deep = cfg.n_layers >= 4
        peak = MFMA_FP32_PEAK_TFS if deep else VALU_FP32_PEAK_TFS
        roof = {"bound": "mfma" if deep else "alu",
                "kernel": "eval phase (k_chain dominant)" if deep else "eval phase (k_slab dominant)",
                "achieved": achieved, "peak": peak, "unit": "TFLOP/s", "frac": achieved / peak,
                "traffic": None, "flops_per_launch": per_step}
    roof["avg_launch_us"] = avg_s * 1e6
    roof["launches"] = int(launches[dominant])
    out = {"workload": workload_config(cfg)["workload"], "steps": steps, "warmup": warmup,
           "ms_per_step": wall * 1e3 / steps, "evals_per_s": st.evaluated / wall,
           "accepted_per_s": st.accepted / wall,
           "accept_rate_per_step": st.accepted / max(st.steps, 1),
           "tie_band": int(st.tie_band),
           "tie_band_per_eval": st.tie_band / max(st.evaluated, 1),
           "final_loss": st.loss, "roofline": roof}
    return out, ctx, st, wall


def copy_calibration(nbytes: int):
    """A plain device-to-device copy of nbytes (torch's copy kernel), 5 launches."""
    import torch
    src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": nbytes, "launches": 5}), flush=True)


# Per-config windows of the multi-config line (the headline config times
# exactly --steps): long enough that launch and copy overheads are small.
# deepln draws its layer once per block of 32 steps (sticky schedule) and the
# layers differ in cost, so its window spans 20 blocks
SUB_STEPS = {"tiny": (20000, 200), "deep": (60, 3), "ternary": (1000, 20),
             "transformer": (100, 5), "channel": (20, 2), "deepln": (640, 32)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=2000)
    ap.add_argument("--warmup", type=int, default=100)
    ap.add_argument("--workload", default="wide", help="the headline workload")
    ap.add_argument("--configs", default="tiny,deep,ternary,transformer,channel,deepln",
                    help="the other workloads measured into the same line ('' for none)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--sub-cpu-seconds", type=float, default=3.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--tile", type=int, default=0, help="samples per workgroup (16..64)")
    ap.add_argument("--per-phase", action="store_true",
                    help="one launch per phase per step instead of the persistent loop")
    ap.add_argument("--cooperative", action="store_true",
                    help="launch the persistent loop cooperatively (default: an ordinary launch)")
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

    from workloads import CONFIGS

    cfg = CONFIGS[args.workload]
    w = load_workload(cfg)
    eval_batch = args.eval_batch if cfg.kind != "transformer" and cfg.n_layers <= 2 else 0
    print(f"[bench] {cfg.name}: {args.steps} timed steps after {args.warmup}", file=sys.stderr,
          flush=True)
    head, ctx, st, wall = measure(cfg, w, args.steps, args.warmup, args, eval_batch)
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
        "roofline": head["roofline"],
        "tie_band": head["tie_band"],
        "tie_band_per_eval": head["tie_band_per_eval"],
        "final_loss": st.loss,
    }
    if eval_batch > 0:
        print(f"[bench] incremental phases: {args.eval_reps} batches of {eval_batch}",
              file=sys.stderr, flush=True)
        result["incremental_phase"] = incremental_phase(ctx, cfg, st.next_step, eval_batch,
                                                        args.eval_reps)
    ctx.close()
    subs = {}
    for name in [c for c in args.configs.split(",") if c and c != cfg.name]:
        sc = CONFIGS[name]
        steps, warm = SUB_STEPS.get(name, (200, 10))
        print(f"[bench] {name}: {steps} timed steps after {warm}", file=sys.stderr, flush=True)
        sw = load_workload(sc)
        sub, sctx, _, _ = measure(sc, sw, steps, warm, args)
        sctx.close()
        if not args.no_cpu_baseline:
            sub["cpu_baseline"] = cpu_baseline(sc, sw, args.sub_cpu_seconds, "incremental", True)
        subs[name] = sub
        del sw
    head_sub = dict(head)
    subs[cfg.name] = head_sub
    result["configs"] = subs
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle", file=sys.stderr, flush=True)
        base = cpu_baseline(cfg, w, args.cpu_seconds, "incremental", True)
        if cfg.kind != "transformer":
            # the definition in the paper's sequential mode (stop at the first
            # improver): one or more full fp64 forward passes per candidate
            base["full_recompute"] = cpu_baseline(cfg, w, args.cpu_seconds, "full", False)
        result["cpu_baseline"] = base
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
