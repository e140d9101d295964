"""Replicas of the fp64 oracle in worker processes, for the long parity
windows of the full-size workloads: the K candidates of a step are scored in
parallel (each replica holds the same committed state; commits are applied on
every replica).  The workers are child processes running this file (fresh
interpreters that import only numpy and the oracle, one BLAS thread each,
talking over their stdin/stdout) and never touch the GPU.

Test infrastructure: the decisions and loss changes are exactly those of
oracle.mca.evaluate_all on one model (same per-candidate arithmetic; only the
order in which candidates are scored differs, which nothing depends on).
"""
from __future__ import annotations

import os
import pickle
import struct
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from oracle import mca as omca  # noqa: E402


def _send(f, obj):
    data = pickle.dumps(obj, protocol=pickle.HIGHEST_PROTOCOL)
    f.write(struct.pack("<Q", len(data)))
    f.write(data)
    f.flush()


def _recv(f):
    head = f.read(8)
    if len(head) < 8:
        raise EOFError("oracle worker closed its pipe")
    (n,) = struct.unpack("<Q", head)
    return pickle.loads(f.read(n))


def _build(kind, cfg):
    if kind == "mlp" and (cfg.biases or cfg.layer_norm):
        from oracle.normmlp import NormMLP
        from workloads import mlp_workload
        w = mlp_workload(cfg)
        return NormMLP(w["weights"], w["X"], w["y"], cfg.act, cfg.gamma, bias=cfg.biases,
                       ln=cfg.layer_norm, eps=cfg.ln_eps, sticky=cfg.sticky_steps)
    if kind == "mlp":
        from oracle.mlp import IncrementalMLP, MLPState
        from workloads import mlp_workload
        w = mlp_workload(cfg)
        return IncrementalMLP(MLPState(w["weights"], w["codes"], w["scales"]), w["X"], w["y"],
                              cfg.act, cfg.gamma)
    from oracle.transformer import TransformerModel
    from workloads import transformer_workload
    w = transformer_workload(cfg)
    return TransformerModel(w["params"], w["tokens"], w["targets"], cfg.vocab, cfg.ctx,
                            cfg.d_model, cfg.n_layer, cfg.n_head, cfg.d_mlp, cfg.ln_eps)


def _worker_main():
    fin, fout = sys.stdin.buffer, sys.stdout.buffer
    kind, cfg = _recv(fin)
    model = _build(kind, cfg)
    _send(fout, ("ready", model.loss()))
    while True:
        msg = _recv(fin)
        if msg[0] == "eval":
            _, t, ks, args = msg
            seed, tag, delta, mode, n_prune = args
            out = []
            for k in ks:
                c = (model.candidate(seed, tag, t, k, delta, mode, prune=True) if k < n_prune
                     else model.candidate(seed, tag, t, k, delta, mode))
                dL, mag = model.delta(c)
                out.append((k, c, dL, mag))
            _send(fout, out)
        elif msg[0] == "delta":
            _send(fout, [(n, model.delta(c)) for n, c in msg[1]])
        elif msg[0] == "commit":
            model.commit(msg[1], msg[2])
        elif msg[0] == "state":
            _send(fout, model.state_weights() if hasattr(model, "state_weights")
                  else (model.state.weights if kind == "mlp" else model.params))
        else:
            break


class OraclePool:
    """n replicas of the oracle of one workload (kind "mlp" or "transformer")."""

    def __init__(self, kind, cfg, n=None):
        n = n or min(16, len(os.sched_getaffinity(0)))
        env = dict(os.environ, OMP_NUM_THREADS="1", OPENBLAS_NUM_THREADS="1",
                   MKL_NUM_THREADS="1")
        self.procs = [subprocess.Popen([sys.executable, os.path.abspath(__file__), "--worker"],
                                       stdin=subprocess.PIPE, stdout=subprocess.PIPE, env=env,
                                       cwd=ROOT) for _ in range(n)]
        for p in self.procs:
            _send(p.stdin, (kind, cfg))
        self.L = [_recv(p.stdout)[1] for p in self.procs][0]
        self.kind = kind

    def loss(self):
        return self.L

    def evaluate_all(self, t, K, seed, tag, delta, mode="weight", accept_ties=False,
                     beta=0.0, n_prune=0):
        """Same returns as oracle.mca.evaluate_all (scan_all=True)."""
        n = len(self.procs)
        for w, p in enumerate(self.procs):
            _send(p.stdin, ("eval", t, list(range(w, K, n)), (seed, tag, delta, mode, n_prune)))
        res = {}
        for p in self.procs:
            for k, c, dL, mag in _recv(p.stdout):
                res[k] = (c, dL, mag)
        th = omca.thresholds(seed, tag, t, K, beta)
        cands = [res[k][0] for k in range(K)]
        dls = [res[k][1] for k in range(K)]
        mags = [res[k][2] for k in range(K)]
        chosen = next((k for k in range(K) if omca.accepts(dls[k], accept_ties, th[k])), -1)
        return self.L, cands, dls, mags, th, chosen

    def delta_of(self, cands):
        """model.delta of given candidates, in parallel; in their order."""
        n = len(self.procs)
        for w, p in enumerate(self.procs):
            _send(p.stdin, ("delta", [(k, cands[k]) for k in range(w, len(cands), n)]))
        res = {}
        for p in self.procs:
            for k, r in _recv(p.stdout):
                res[k] = r
        return [res[k] for k in range(len(cands))]

    def commit(self, c, loss_after):
        for p in self.procs:
            _send(p.stdin, ("commit", c, loss_after))
        self.L = float(loss_after)

    def state_weights(self):
        _send(self.procs[0].stdin, ("state",))
        return _recv(self.procs[0].stdout)

    def close(self):
        for p in self.procs:
            try:
                _send(p.stdin, ("close",))
                p.stdin.close()
            except (BrokenPipeError, OSError):
                pass
        for p in self.procs:
            try:
                p.wait(timeout=10)
            except subprocess.TimeoutExpired:
                p.kill()


if __name__ == "__main__" and sys.argv[1:2] == ["--worker"]:
    _worker_main()
