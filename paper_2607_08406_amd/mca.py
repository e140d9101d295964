"""ctypes binding of libmca (include/mca.h): same names, argument marshalling only.

Every step of the hot path runs in the HIP library; this module converts
Python/numpy/torch arguments to the C structs and pointers, turns non-zero
status codes into ``MCAError``, and supplies device memory and the stream from
PyTorch.  torch is imported before the library is loaded so that both share
one HIP runtime.  There is no fallback: if the library is missing or no GPU
is present, calls fail loudly.
"""
from __future__ import annotations

import ctypes
import os
from typing import List, Optional, Sequence

import numpy as np
import torch  # noqa: F401  (loads the HIP runtime the library binds to)

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libmca.so")

MCA_MAX_LAYERS = 32
MCA_MAX_CLASSES = 16
MCA_OK, MCA_EINVAL, MCA_ESTATE, MCA_ENOSPACE = 0, -1, -2, -3
MCA_EDEVICE, MCA_EPOISONED, MCA_EUNSUPPORTED = -4, -5, -6
MCA_NET_MLP, MCA_NET_TRANSFORMER = 0, 1
MCA_ACT_TANH, MCA_ACT_GAUSS, MCA_ACT_RELU = 0, 1, 2
MCA_MUTATE_SINGLE, MCA_MUTATE_CHANNEL_REDRAW, MCA_MUTATE_CHANNEL_ZERO = 0, 1, 2
MCA_WEIGHTS_FP32, MCA_WEIGHTS_TERNARY = 0, 1
MCA_PICK_WEIGHT, MCA_PICK_LAYER, MCA_PICK_STICKY = 0, 1, 2
MCA_RULE_GREEDY, MCA_RULE_METROPOLIS = 0, 1
MCA_OPT_PERSISTENT_LOOP, MCA_OPT_LOOP_TILE, MCA_OPT_LOOP_LAUNCH = 1, 2, 3

STATUS_NAMES = {0: "MCA_OK", -1: "MCA_EINVAL", -2: "MCA_ESTATE", -3: "MCA_ENOSPACE",
                -4: "MCA_EDEVICE", -5: "MCA_EPOISONED", -6: "MCA_EUNSUPPORTED"}


class MCAError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{STATUS_NAMES.get(code, code)}: {msg}")
        self.code = code


class mca_net_desc(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("n_layers", ctypes.c_int32),
                ("widths", ctypes.c_int32 * (MCA_MAX_LAYERS + 1)), ("act", ctypes.c_int32),
                ("gamma", ctypes.c_float), ("weight_mode", ctypes.c_int32),
                ("scales", ctypes.c_float * MCA_MAX_LAYERS), ("pick", ctypes.c_int32),
                ("delta", ctypes.c_float), ("bound", ctypes.c_float),
                ("accept_ties", ctypes.c_int32), ("seed", ctypes.c_uint64),
                ("stream_tag", ctypes.c_uint64), ("vocab", ctypes.c_int32),
                ("ctx", ctypes.c_int32), ("d_model", ctypes.c_int32), ("n_block", ctypes.c_int32),
                ("n_head", ctypes.c_int32), ("d_mlp", ctypes.c_int32), ("ln_eps", ctypes.c_float),
                ("accept_rule", ctypes.c_int32), ("n_prune", ctypes.c_int32),
                ("beta", ctypes.c_double), ("subset_size", ctypes.c_int64),
                ("subset_period", ctypes.c_int64), ("mutation", ctypes.c_int32),
                ("biases", ctypes.c_int32), ("layer_norm", ctypes.c_int32),
                ("sticky_steps", ctypes.c_int32)]


class mca_cand(ctypes.Structure):
    _fields_ = [("flat", ctypes.c_int64), ("layer", ctypes.c_int32), ("j", ctypes.c_int32),
                ("i", ctypes.c_int32), ("d", ctypes.c_float), ("code", ctypes.c_int32),
                ("flags", ctypes.c_int32)]


CAND_DTYPE = np.dtype([("flat", "<i8"), ("layer", "<i4"), ("j", "<i4"), ("i", "<i4"),
                       ("d", "<f4"), ("code", "<i4"), ("flags", "<i4")])
MCA_CAND_PRUNE = 1


class mca_channel(ctypes.Structure):
    _fields_ = [("units", ctypes.c_int32 * (MCA_MAX_LAYERS + 1)),
                ("w_new", ctypes.c_float * MCA_MAX_LAYERS)]


CHANNEL_DTYPE = np.dtype([("units", "<i4", (MCA_MAX_LAYERS + 1,)),
                          ("w_new", "<f4", (MCA_MAX_LAYERS,))])


class mca_data(ctypes.Structure):
    _fields_ = [("n_samples", ctypes.c_int64), ("x", ctypes.POINTER(ctypes.c_float)),
                ("tokens", ctypes.POINTER(ctypes.c_int32)), ("y", ctypes.POINTER(ctypes.c_int32)),
                ("n_seq", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class mca_stats(ctypes.Structure):
    _fields_ = [("steps", ctypes.c_uint64), ("evaluated", ctypes.c_uint64),
                ("accepted", ctypes.c_uint64), ("wasted", ctypes.c_uint64),
                ("tie_band", ctypes.c_uint64), ("loss", ctypes.c_double),
                ("next_step", ctypes.c_uint64)]


class mca_trace(ctypes.Structure):
    _fields_ = [("chosen", ctypes.POINTER(ctypes.c_int32)), ("dloss", ctypes.POINTER(ctypes.c_double))]


class mca_timing(ctypes.Structure):
    _fields_ = [("ms", ctypes.c_double * 8), ("launches", ctypes.c_uint64 * 8)]


STRUCTS = [mca_net_desc, mca_cand, mca_data, mca_stats, mca_trace, mca_timing, mca_channel]

_P = ctypes.c_void_p
_SIGNATURES = {
    "mca_abi_version": (ctypes.c_int, []),
    "mca_struct_size": (ctypes.c_size_t, [ctypes.c_int32]),
    "mca_plan": (ctypes.c_int, [ctypes.POINTER(mca_net_desc), ctypes.c_int64, ctypes.c_int32,
                                ctypes.POINTER(ctypes.c_size_t)]),
    "mca_init": (ctypes.c_int, [ctypes.POINTER(_P), ctypes.POINTER(mca_net_desc), _P, ctypes.c_int32,
                                _P, ctypes.POINTER(mca_data), ctypes.c_int32, _P, ctypes.c_size_t, _P]),
    "mca_propose": (ctypes.c_int, [_P, ctypes.c_uint64, ctypes.c_int32, _P]),
    "mca_eval_losses": (ctypes.c_int, [_P, _P, ctypes.c_int32, _P, _P]),
    "mca_eval_losses_noalloc": (ctypes.c_int, [_P, _P, ctypes.c_int32, _P, _P]),
    "mca_propose_channels": (ctypes.c_int, [_P, ctypes.c_uint64, ctypes.c_int32, _P]),
    "mca_eval_channels": (ctypes.c_int, [_P, _P, ctypes.c_int32, _P, _P]),
    "mca_commit": (ctypes.c_int, [_P, ctypes.c_int32]),
    "mca_rollback": (ctypes.c_int, [_P]),
    "mca_set_option": (ctypes.c_int, [_P, ctypes.c_int32, ctypes.c_int64]),
    "mca_set_step": (ctypes.c_int, [_P, ctypes.c_uint64]),
    "mca_run_steps": (ctypes.c_int, [_P, ctypes.c_uint64, ctypes.c_int32,
                                     ctypes.POINTER(mca_trace), ctypes.POINTER(mca_stats)]),
    "mca_get_params": (ctypes.c_int, [_P, _P, _P]),
    "mca_get_loss": (ctypes.c_int, [_P, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_uint64)]),
    "mca_set_state": (ctypes.c_int, [_P, _P, _P, ctypes.c_uint64]),
    "mca_refresh": (ctypes.c_int, [_P]),
    "mca_get_sample_losses": (ctypes.c_int, [_P, _P]),
    "mca_set_timing": (ctypes.c_int, [_P, ctypes.c_int32]),
    "mca_get_timing": (ctypes.c_int, [_P, ctypes.POINTER(mca_timing), ctypes.c_int32]),
    "mca_destroy": (None, [_P]),
    "mca_last_error": (ctypes.c_char_p, [_P]),
}

_lib = None


def load_library(path: str = LIB_PATH):
    """Load libmca.so (built by paper_2607_08406_amd.build); no fallback."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise MCAError(MCA_EUNSUPPORTED, f"{path} is not built; run paper_2607_08406_amd.build.build()")
    lib = ctypes.CDLL(path)
    for name, (res, args) in _SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    for n, st in enumerate(STRUCTS):
        if lib.mca_struct_size(n) != ctypes.sizeof(st):
            raise MCAError(MCA_EINVAL, f"{st.__name__} mirror has the wrong size")
    _lib = lib
    return lib


def _check(rc: int, ctx=None):
    if rc != MCA_OK:
        msg = load_library().mca_last_error(ctx)
        raise MCAError(rc, msg.decode() if msg else "")


def _ptr_array(arrays, ctype):
    arr = (ctypes.c_void_p * len(arrays))()
    for n, a in enumerate(arrays):
        arr[n] = a.ctypes.data_as(ctypes.c_void_p).value
    return arr


# ---------------------------------------------------------------------------
# descriptions
# ---------------------------------------------------------------------------

def _selection(d: mca_net_desc, beta: float, n_prune: int, subset_size: int,
               subset_period: int):
    d.accept_rule = MCA_RULE_METROPOLIS if beta else MCA_RULE_GREEDY
    d.beta = float(beta)
    d.n_prune = int(n_prune)
    d.subset_size = int(subset_size)
    d.subset_period = int(subset_period)


def mlp_desc(widths: Sequence[int], act: str = "tanh", gamma: float = 1.0, delta: float = 0.0,
             ternary_scales: Optional[Sequence[float]] = None, pick: str = "weight",
             bound: float = 0.0, accept_ties: bool = False, seed: int = 0,
             stream_tag: int = 0, beta: float = 0.0, n_prune: int = 0, subset_size: int = 0,
             subset_period: int = 1, mutation: str = "single", biases: bool = False,
             layer_norm: bool = False, ln_eps: float = 1e-5,
             sticky_steps: int = 0) -> mca_net_desc:
    d = mca_net_desc()
    d.kind = MCA_NET_MLP
    d.n_layers = len(widths) - 1
    for n, w in enumerate(widths):
        d.widths[n] = int(w)
    d.act = {"tanh": MCA_ACT_TANH, "gauss": MCA_ACT_GAUSS, "relu": MCA_ACT_RELU}[act]
    d.mutation = {"single": MCA_MUTATE_SINGLE, "channel_redraw": MCA_MUTATE_CHANNEL_REDRAW,
                  "channel_zero": MCA_MUTATE_CHANNEL_ZERO}[mutation]
    d.gamma = gamma
    if ternary_scales is not None:
        d.weight_mode = MCA_WEIGHTS_TERNARY
        for n, s in enumerate(ternary_scales):
            d.scales[n] = float(np.float32(s))
    d.pick = {"weight": MCA_PICK_WEIGHT, "layer": MCA_PICK_LAYER, "sticky": MCA_PICK_STICKY}[pick]
    d.biases = int(biases)
    d.layer_norm = int(layer_norm)
    d.ln_eps = float(np.float32(ln_eps))
    d.sticky_steps = int(sticky_steps)
    d.delta = float(np.float32(delta))
    d.bound = bound
    d.accept_ties = int(accept_ties)
    d.seed = seed
    d.stream_tag = stream_tag
    _selection(d, beta, n_prune, subset_size, subset_period)
    return d


def transformer_desc(vocab: int, ctx: int, d_model: int, n_block: int, n_head: int,
                     d_mlp: int, delta: float = 0.0, ln_eps: float = 1e-5, bound: float = 0.0,
                     accept_ties: bool = False, seed: int = 0,
                     stream_tag: int = 0, beta: float = 0.0) -> mca_net_desc:
    d = mca_net_desc()
    d.kind = MCA_NET_TRANSFORMER
    d.vocab, d.ctx, d.d_model = int(vocab), int(ctx), int(d_model)
    d.n_block, d.n_head, d.d_mlp = int(n_block), int(n_head), int(d_mlp)
    d.ln_eps = float(np.float32(ln_eps))
    d.weight_mode = MCA_WEIGHTS_FP32
    d.pick = MCA_PICK_WEIGHT
    d.delta = float(np.float32(delta))
    d.bound = bound
    d.accept_ties = int(accept_ties)
    d.seed = seed
    d.stream_tag = stream_tag
    _selection(d, beta, 0, 0, 1)
    return d


# ---------------------------------------------------------------------------
# the calls, with the C names
# ---------------------------------------------------------------------------

def mca_abi_version() -> int:
    return load_library().mca_abi_version()


def mca_plan(desc: mca_net_desc, n_samples: int, k_max: int) -> int:
    out = ctypes.c_size_t(0)
    _check(load_library().mca_plan(ctypes.byref(desc), n_samples, k_max, ctypes.byref(out)))
    return out.value


def mca_init(desc, params: List[np.ndarray], codes, X: np.ndarray, y: np.ndarray, k_max: int,
             workspace: torch.Tensor, stream_ptr: int):
    lib = load_library()
    params = [np.ascontiguousarray(p, dtype=np.float32) for p in params]
    codes_c = None if codes is None else [np.ascontiguousarray(c, dtype=np.int8) for c in codes]
    X = np.ascontiguousarray(X, dtype=np.float32)
    y = np.ascontiguousarray(y, dtype=np.int32)
    data = mca_data()
    data.n_samples = X.shape[0]
    data.x = X.ctypes.data_as(ctypes.POINTER(ctypes.c_float))
    data.y = y.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
    out = ctypes.c_void_p()
    rc = lib.mca_init(ctypes.byref(out), ctypes.byref(desc), _ptr_array(params, ctypes.c_float),
                      len(params), None if codes_c is None else _ptr_array(codes_c, ctypes.c_int8),
                      ctypes.byref(data), k_max, workspace.data_ptr(), workspace.numel(), stream_ptr)
    _check(rc)
    return out


def mca_init_transformer(desc, params: List[np.ndarray], tokens: np.ndarray, targets: np.ndarray,
                         k_max: int, workspace: torch.Tensor, stream_ptr: int):
    """mca_init for a Transformer: tokens and targets are [n_seq][ctx] int32."""
    lib = load_library()
    params = [np.ascontiguousarray(p, dtype=np.float32) for p in params]
    tokens = np.ascontiguousarray(tokens, dtype=np.int32)
    targets = np.ascontiguousarray(targets, dtype=np.int32)
    data = mca_data()
    data.n_samples = tokens.size
    data.n_seq = tokens.shape[0]
    data.tokens = tokens.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
    data.y = targets.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
    out = ctypes.c_void_p()
    rc = lib.mca_init(ctypes.byref(out), ctypes.byref(desc), _ptr_array(params, ctypes.c_float),
                      len(params), None, ctypes.byref(data), k_max, workspace.data_ptr(),
                      workspace.numel(), stream_ptr)
    _check(rc)
    return out


def mca_propose(ctx, step: int, K: int) -> np.ndarray:
    out = np.zeros(K, dtype=CAND_DTYPE)
    _check(load_library().mca_propose(ctx, step, K, out.ctypes.data), ctx)
    return out


def mca_eval_losses(ctx, cands: np.ndarray):
    cands = np.ascontiguousarray(cands, dtype=CAND_DTYPE)
    K = len(cands)
    loss = np.zeros(K)
    dloss = np.zeros(K)
    _check(load_library().mca_eval_losses(ctx, cands.ctypes.data, K, loss.ctypes.data,
                                          dloss.ctypes.data), ctx)
    return loss, dloss


def mca_eval_losses_noalloc(ctx, cands: np.ndarray):
    cands = np.ascontiguousarray(cands, dtype=CAND_DTYPE)
    K = len(cands)
    loss = np.zeros(K)
    dloss = np.zeros(K)
    _check(load_library().mca_eval_losses_noalloc(ctx, cands.ctypes.data, K, loss.ctypes.data,
                                                  dloss.ctypes.data), ctx)
    return loss, dloss


def mca_propose_channels(ctx, step: int, K: int) -> np.ndarray:
    out = np.zeros(K, dtype=CHANNEL_DTYPE)
    _check(load_library().mca_propose_channels(ctx, step, K, out.ctypes.data), ctx)
    return out


def mca_eval_channels(ctx, chans: np.ndarray):
    chans = np.ascontiguousarray(chans, dtype=CHANNEL_DTYPE)
    K = len(chans)
    loss = np.zeros(K)
    dloss = np.zeros(K)
    _check(load_library().mca_eval_channels(ctx, chans.ctypes.data, K, loss.ctypes.data,
                                            dloss.ctypes.data), ctx)
    return loss, dloss


def mca_commit(ctx, k: int):
    _check(load_library().mca_commit(ctx, k), ctx)


def mca_rollback(ctx):
    _check(load_library().mca_rollback(ctx), ctx)


def mca_set_option(ctx, option: int, value: int):
    _check(load_library().mca_set_option(ctx, option, value), ctx)


def mca_set_step(ctx, next_step: int):
    _check(load_library().mca_set_step(ctx, next_step), ctx)


def mca_run_steps(ctx, n_steps: int, K: int, trace: bool = False, trace_dloss: bool = False):
    st = mca_stats()
    tr = None
    chosen = dloss = None
    if trace:
        chosen = np.zeros(n_steps, dtype=np.int32)
        tr = mca_trace()
        tr.chosen = chosen.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
        if trace_dloss:
            dloss = np.zeros(n_steps * K)
            tr.dloss = dloss.ctypes.data_as(ctypes.POINTER(ctypes.c_double))
    _check(load_library().mca_run_steps(ctx, n_steps, K, None if tr is None else ctypes.byref(tr),
                                        ctypes.byref(st)), ctx)
    if dloss is not None:
        dloss = dloss.reshape(n_steps, K)
    return st, chosen, dloss


def mca_get_params(ctx, shapes, ternary: bool = False):
    params = [np.zeros(s, dtype=np.float32) for s in shapes]
    codes = [np.zeros(s, dtype=np.int8) for s in shapes] if ternary else None
    _check(load_library().mca_get_params(ctx, _ptr_array(params, None),
                                         None if codes is None else _ptr_array(codes, None)), ctx)
    return params, codes


def mca_get_loss(ctx):
    L = ctypes.c_double()
    t = ctypes.c_uint64()
    _check(load_library().mca_get_loss(ctx, ctypes.byref(L), ctypes.byref(t)), ctx)
    return L.value, t.value


def mca_set_state(ctx, params, codes, next_step: int):
    params = [np.ascontiguousarray(p, dtype=np.float32) for p in params]
    codes_c = None if codes is None else [np.ascontiguousarray(c, dtype=np.int8) for c in codes]
    _check(load_library().mca_set_state(ctx, _ptr_array(params, None),
                                        None if codes_c is None else _ptr_array(codes_c, None),
                                        next_step), ctx)


def mca_refresh(ctx):
    _check(load_library().mca_refresh(ctx), ctx)


def mca_get_sample_losses(ctx, n: int) -> np.ndarray:
    out = np.zeros(n, dtype=np.float32)
    _check(load_library().mca_get_sample_losses(ctx, out.ctypes.data), ctx)
    return out


PHASES = ["propose", "eval", "select", "commit", "step_loop", "forward", "one_loop"]


def mca_set_timing(ctx, phase_mask: int):
    _check(load_library().mca_set_timing(ctx, int(phase_mask)), ctx)


def mca_get_timing(ctx, reset: bool = False):
    t = mca_timing()
    _check(load_library().mca_get_timing(ctx, ctypes.byref(t), int(reset)), ctx)
    return list(t.ms), list(t.launches)


def mca_destroy(ctx):
    if ctx:
        load_library().mca_destroy(ctx)


def mca_last_error(ctx=None) -> str:
    msg = load_library().mca_last_error(ctx)
    return msg.decode() if msg else ""


# ---------------------------------------------------------------------------
# a context owning its workspace tensor
# ---------------------------------------------------------------------------

class Context:
    """An MCA context on a CUDA (HIP) device; the workspace is a torch tensor."""

    def __init__(self, desc: mca_net_desc, params, X, y, k_max: int, codes=None,
                 device: str = "cuda:0", stream: Optional[torch.cuda.Stream] = None):
        if not torch.cuda.is_available():
            raise MCAError(MCA_EDEVICE, "no GPU visible: the MCA library runs only on the GPU")
        self.desc = desc
        self.shapes = [np.shape(p) for p in params]
        self.ternary = codes is not None
        self.n_samples = int(np.shape(X)[0])
        self.device = torch.device(device)
        self.stream = stream if stream is not None else torch.cuda.current_stream(self.device)
        nbytes = mca_plan(desc, self.n_samples, k_max)
        self.workspace = torch.empty(nbytes, dtype=torch.uint8, device=self.device)
        self.ctx = mca_init(desc, params, codes, X, y, k_max, self.workspace, self.stream.cuda_stream)

    def propose(self, step, K):
        return mca_propose(self.ctx, step, K)

    def eval_losses(self, cands):
        return mca_eval_losses(self.ctx, cands)

    def propose_channels(self, step, K):
        return mca_propose_channels(self.ctx, step, K)

    def eval_channels(self, chans):
        return mca_eval_channels(self.ctx, chans)

    def commit(self, k):
        mca_commit(self.ctx, k)

    def rollback(self):
        mca_rollback(self.ctx)

    def set_option(self, option, value):
        mca_set_option(self.ctx, option, value)

    def set_step(self, next_step):
        mca_set_step(self.ctx, next_step)

    def run_steps(self, n_steps, K, trace=False, trace_dloss=False):
        return mca_run_steps(self.ctx, n_steps, K, trace, trace_dloss)

    def params(self):
        return mca_get_params(self.ctx, self.shapes, self.ternary)

    def loss(self):
        return mca_get_loss(self.ctx)

    def set_state(self, params, codes, next_step):
        mca_set_state(self.ctx, params, codes, next_step)

    def refresh(self):
        mca_refresh(self.ctx)

    def sample_losses(self):
        return mca_get_sample_losses(self.ctx, self.n_samples)

    def close(self):
        if getattr(self, "ctx", None):
            mca_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class TransformerContext(Context):
    """An MCA context of the decoder Transformer; params in canonical order."""

    def __init__(self, desc: mca_net_desc, params, tokens, targets, k_max: int,
                 device: str = "cuda:0", stream: Optional[torch.cuda.Stream] = None):
        if not torch.cuda.is_available():
            raise MCAError(MCA_EDEVICE, "no GPU visible: the MCA library runs only on the GPU")
        self.desc = desc
        self.shapes = [np.shape(p) for p in params]
        self.ternary = False
        self.n_samples = int(np.size(tokens))
        self.device = torch.device(device)
        self.stream = stream if stream is not None else torch.cuda.current_stream(self.device)
        nbytes = mca_plan(desc, self.n_samples, k_max)
        self.workspace = torch.empty(nbytes, dtype=torch.uint8, device=self.device)
        self.ctx = mca_init_transformer(desc, params, tokens, targets, k_max, self.workspace,
                                        self.stream.cuda_stream)
