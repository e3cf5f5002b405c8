"""ctypes binding of libslim.so (include/slim.h) on torch tensors.

Argument marshalling only: every step of the computation runs in the HIP
library.  torch provides device memory and the current stream.  When the
library is missing this module raises at import time; there is no fallback.
"""

from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libslim.so")

SLIM_OK, SLIM_EINVAL, SLIM_EUNSUPPORTED, SLIM_EWORKSPACE, SLIM_EHIP = 0, -1, -2, -3, -4
FAVOR_PLUS, RELU, SQUARE = 0, 1, 2
F32, BF16 = 0, 1
QUERY, KEY = 0, 1
PHASE_FWD, PHASE_BWD = 0, 1
WITHIN_ITER, WITHIN_QUADRATIC, WITHIN_PS = 0, 1, 2
WITHINS = {"iter": WITHIN_ITER, "quadratic": WITHIN_QUADRATIC, "ps": WITHIN_PS}

KINDS = {"favor+": FAVOR_PLUS, "relu": RELU, "square": SQUARE}
DTYPES = {torch.float32: F32, torch.bfloat16: BF16}


class SlimError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"slim status {status}: {msg}")
        self.status = status


class Problem(ctypes.Structure):
    _fields_ = [
        ("B", ctypes.c_int64),
        ("H", ctypes.c_int64),
        ("L", ctypes.c_int64),
        ("d", ctypes.c_int32),
        ("M", ctypes.c_int32),
        ("C", ctypes.c_int32),
        ("dtype", ctypes.c_int32),
        ("kind", ctypes.c_int32),
        ("relu_eps", ctypes.c_float),
        ("dropout", ctypes.c_float),
        ("seed", ctypes.c_uint64),
        ("within", ctypes.c_int32),
        ("reserved", ctypes.c_int32),
    ]


class ModelDesc(ctypes.Structure):
    """slim_model of include/slim_model.h."""

    _fields_ = [
        ("B", ctypes.c_int64),
        ("L", ctypes.c_int64),
        ("D", ctypes.c_int32),
        ("s", ctypes.c_int32),
        ("vocab", ctypes.c_int32),
        ("F", ctypes.c_int32),
        ("C", ctypes.c_int32),
        ("ln_eps", ctypes.c_float),
    ]


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is missing: build it with `python -c 'import __graft_entry__ as g; g.build()'` "
            "or `python paper_2012_11346_amd/build.py`"
        )
    lib = ctypes.CDLL(LIB_PATH)
    P = ctypes.POINTER(Problem)
    vp, fp, i32, sz = ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t
    lib.slim_workspace_bytes.argtypes = [P, i32]
    lib.slim_workspace_bytes.restype = sz
    lib.slim_num_segments.argtypes = [P]
    lib.slim_num_segments.restype = i32
    lib.slim_featmap.argtypes = [P, vp, fp, i32, fp, fp, vp]
    lib.slim_featmap.restype = i32
    lib.slim_context_bytes.argtypes = [P]
    lib.slim_context_bytes.restype = sz
    lib.slim_fwd.argtypes = [P, vp, vp, vp, fp, fp, fp, vp, fp, fp, fp, fp, vp, sz, vp]
    lib.slim_fwd.restype = i32
    lib.slim_bwd.argtypes = [P, vp, vp, vp, fp, fp, fp, fp, vp, vp, fp, fp, vp, vp, vp, fp, fp, fp, vp, sz, vp]
    lib.slim_bwd.restype = i32
    lib.slim_status_string.argtypes = [i32]
    lib.slim_status_string.restype = ctypes.c_char_p
    lib.slim_last_error.argtypes = []
    lib.slim_last_error.restype = ctypes.c_char_p
    lib.slim_time_walk.argtypes = [i32, vp, vp]
    lib.slim_time_walk.restype = i32
    lib.slim_noalloc_scratch_bytes.argtypes = []
    lib.slim_noalloc_scratch_bytes.restype = sz
    lib.slim_fwd_noalloc.argtypes = [P, vp, vp, vp, fp, fp, fp, vp, fp, fp, fp, fp, vp]
    lib.slim_fwd_noalloc.restype = i32
    MP = ctypes.POINTER(ModelDesc)
    lib.slim_model_num_params.argtypes = [MP]
    lib.slim_model_num_params.restype = i32
    lib.slim_model_workspace_bytes.argtypes = [MP]
    lib.slim_model_workspace_bytes.restype = sz
    lib.slim_model_step.argtypes = [MP, vp, ctypes.POINTER(vp), ctypes.POINTER(vp), vp, vp, sz, vp]
    lib.slim_model_step.restype = i32
    return lib


LIB = _load()

EXPORTED = (
    "slim_workspace_bytes",
    "slim_context_bytes",
    "slim_featmap",
    "slim_fwd",
    "slim_bwd",
    "slim_status_string",
    "slim_last_error",
    "slim_num_segments",
    "slim_time_walk",
    "slim_noalloc_scratch_bytes",
    "slim_fwd_noalloc",
    "slim_model_num_params",
    "slim_model_workspace_bytes",
    "slim_model_step",
)


def _check(status: int):
    if status != SLIM_OK:
        raise SlimError(status, LIB.slim_last_error().decode())


def problem(B, H, L, d, M, C, dtype=BF16, kind=FAVOR_PLUS, relu_eps=1e-3, dropout=0.0, seed=0,
            within=WITHIN_ITER) -> Problem:
    if isinstance(dtype, torch.dtype):
        dtype = DTYPES[dtype]
    if isinstance(kind, str):
        kind = KINDS[kind]
    if isinstance(within, str):
        within = WITHINS[within]
    return Problem(int(B), int(H), int(L), int(d), int(M), int(C), int(dtype), int(kind), float(relu_eps),
                   float(dropout), int(seed) & ((1 << 64) - 1), int(within), 0)


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _problem_of(Q: torch.Tensor, W: torch.Tensor, C: int, kind, relu_eps: float, dropout=0.0, seed=0,
                within=WITHIN_ITER) -> Problem:
    if Q.dim() != 4:
        raise ValueError("Q must be [B, H, L, d]")
    B, H, L, d = Q.shape
    return problem(B, H, L, d, W.shape[0], C, DTYPES[Q.dtype], kind, relu_eps, dropout, seed, within)


def _need(t: torch.Tensor, name: str, dtype: torch.dtype, shape=None):
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")


def workspace_bytes(p: Problem, phase: int) -> int:
    n = LIB.slim_workspace_bytes(ctypes.byref(p), int(phase))
    if n == 0:
        err = LIB.slim_last_error().decode()
        if err:
            raise SlimError(SLIM_EINVAL, err)
    return int(n)


def context_bytes(p: Problem) -> int:
    """Bytes of the forward-to-backward context (0: the problem uses none)."""
    return int(LIB.slim_context_bytes(ctypes.byref(p)))


def new_context(Q: torch.Tensor, W: torch.Tensor, C: int, kind="favor+", relu_eps: float = 1e-3, within="iter"):
    """A context buffer for fwd(..., ctx=) and bwd(..., ctx=), or None when the problem uses none."""
    n = context_bytes(_problem_of(Q, W, C, kind, relu_eps, within=within))
    return None if n == 0 else torch.empty(n // 4, dtype=torch.float32, device=Q.device)


def num_segments(p: Problem) -> int:
    return int(LIB.slim_num_segments(ctypes.byref(p)))


def time_walk(phase: int, before: "torch.cuda.Event", after: "torch.cuda.Event") -> None:
    """Have the next fwd (phase PHASE_FWD) or bwd (PHASE_BWD) call of this
    thread record the two timing events around its walk kernel only.  Events
    not yet created (torch creates them lazily) are recorded once here on the
    current stream so that they exist."""
    for ev in (before, after):
        if ev.cuda_event == 0:
            ev.record()
    _check(LIB.slim_time_walk(int(phase), ctypes.c_void_p(before.cuda_event), ctypes.c_void_p(after.cuda_event)))


def _nbytes(t: torch.Tensor) -> int:
    return t.numel() * t.element_size()


def _workspace(p: Problem, phase: int, device, ws: Optional[torch.Tensor]):
    n = workspace_bytes(p, phase)
    if ws is None:
        ws = torch.empty(max(n, 1), dtype=torch.uint8, device=device)
    else:
        _need(ws, "ws", ws.dtype)
        if _nbytes(ws) < n:
            raise ValueError(f"workspace needs {n} bytes, got {_nbytes(ws)}")
    return ws


def featmap(X: torch.Tensor, W: torch.Tensor, role: int, kind="favor+", relu_eps: float = 1e-3):
    """phi_hat [B, H, L, M] float32 and shift (queries [B, H, L], keys [B, H]; None for ReLU)."""
    p = _problem_of(X, W, 1, kind, relu_eps)
    _need(X, "X", X.dtype)
    _need(W, "W", torch.float32, (p.M, p.d))
    phi = torch.empty((p.B, p.H, p.L, p.M), dtype=torch.float32, device=X.device)
    shift = None
    if p.kind == FAVOR_PLUS:
        shift = torch.empty((p.B, p.H, p.L) if role == QUERY else (p.B, p.H), dtype=torch.float32, device=X.device)
    _check(LIB.slim_featmap(ctypes.byref(p), _ptr(X), _ptr(W), int(role), _ptr(phi), _ptr(shift), _stream()))
    return phi, shift


def _need_ctx(p: Problem, ctx: Optional[torch.Tensor]):
    if ctx is None:
        return
    _need(ctx, "ctx", torch.float32)
    if ctx.numel() * 4 < LIB.slim_context_bytes(ctypes.byref(p)):
        raise ValueError("ctx is smaller than slim_context_bytes")


def fwd(Q, K, V, W, C: int, kind="favor+", state_in=None, kshift_in=None, relu_eps: float = 1e-3, ws=None,
        Y=None, state_out=None, kshift_out=None, ctx=None, dropout: float = 0.0, seed: int = 0, within="iter",
        logD=None):
    """Forward sweep.  Returns (Y, state_out [B,H,M,d+1], kshift_out [B,H] or None).
    ctx (optional, from new_context) receives the segment boundary states for bwd;
    logD (optional float32 [B,H,L], tile-walk mode only) the row normalisers.
    dropout / seed: value dropout with per-slice seeds; within: "iter",
    "quadratic" or "ps" (include/slim.h)."""
    p = _problem_of(Q, W, C, kind, relu_eps, dropout, seed, within)
    shp = (p.B, p.H, p.L, p.d)
    for n, t in (("Q", Q), ("K", K), ("V", V)):
        _need(t, n, Q.dtype, shp)
    _need(W, "W", torch.float32, (p.M, p.d))
    sshape = (p.B, p.H, p.M, p.d + 1)
    if state_in is not None:
        _need(state_in, "state_in", torch.float32, sshape)
    if kshift_in is not None:
        _need(kshift_in, "kshift_in", torch.float32, (p.B, p.H))
    dev = Q.device
    Y = torch.empty_like(Q) if Y is None else Y
    _need(Y, "Y", Q.dtype, shp)
    state_out = torch.empty(sshape, dtype=torch.float32, device=dev) if state_out is None else state_out
    _need(state_out, "state_out", torch.float32, sshape)
    if p.kind == FAVOR_PLUS and kshift_out is None:
        kshift_out = torch.empty((p.B, p.H), dtype=torch.float32, device=dev)
    if kshift_out is not None:
        _need(kshift_out, "kshift_out", torch.float32, (p.B, p.H))
    _need_ctx(p, ctx)
    if logD is not None:
        _need(logD, "logD", torch.float32, (p.B, p.H, p.L))
    ws = _workspace(p, PHASE_FWD, dev, ws)
    _check(LIB.slim_fwd(ctypes.byref(p), _ptr(Q), _ptr(K), _ptr(V), _ptr(W), _ptr(state_in), _ptr(kshift_in),
                        _ptr(Y), _ptr(logD), _ptr(state_out), _ptr(kshift_out), _ptr(ctx), _ptr(ws), _nbytes(ws),
                        _stream()))
    return Y, state_out, kshift_out


def bwd(Q, K, V, W, dY, C: int, kshift=None, kind="favor+", state_in=None, kshift_in=None, dstate_out=None,
        want_dstate_in: bool = False, relu_eps: float = 1e-3, ws=None, dQ=None, dK=None, dV=None, dW=None,
        ctx=None, dropout: float = 0.0, seed: int = 0, within="iter", Y=None, logD=None):
    """Backward sweep; kshift is the forward's kshift_out (FAVOR+); ctx (optional)
    is the context the forward wrote for the same inputs; Y (optional) the
    forward's output, from which the row cotangents of the recomputed slices
    are taken, and logD (optional, with Y) its row normalisers, from which the
    state cotangents of the segments are summed before the walks (the bf16
    tile walk; elsewhere ignored).

    Returns (dQ, dK, dV, dW [M, d] float32, dstate_in or None)."""
    p = _problem_of(Q, W, C, kind, relu_eps, dropout, seed, within)
    shp = (p.B, p.H, p.L, p.d)
    for n, t in (("Q", Q), ("K", K), ("V", V), ("dY", dY)):
        _need(t, n, Q.dtype, shp)
    if Y is not None:
        _need(Y, "Y", Q.dtype, shp)
    if logD is not None:
        _need(logD, "logD", torch.float32, (p.B, p.H, p.L))
    _need(W, "W", torch.float32, (p.M, p.d))
    sshape = (p.B, p.H, p.M, p.d + 1)
    for n, t in (("state_in", state_in), ("dstate_out", dstate_out)):
        if t is not None:
            _need(t, n, torch.float32, sshape)
    for n, t in (("kshift", kshift), ("kshift_in", kshift_in)):
        if t is not None:
            _need(t, n, torch.float32, (p.B, p.H))
    dev = Q.device
    dQ = torch.empty_like(Q) if dQ is None else dQ
    dK = torch.empty_like(K) if dK is None else dK
    dV = torch.empty_like(V) if dV is None else dV
    dW = torch.empty((p.M, p.d), dtype=torch.float32, device=dev) if dW is None else dW
    for n, t in (("dQ", dQ), ("dK", dK), ("dV", dV)):
        _need(t, n, Q.dtype, shp)
    _need(dW, "dW", torch.float32, (p.M, p.d))
    dstate_in = torch.empty(sshape, dtype=torch.float32, device=dev) if want_dstate_in else None
    _need_ctx(p, ctx)
    ws = _workspace(p, PHASE_BWD, dev, ws)
    _check(LIB.slim_bwd(ctypes.byref(p), _ptr(Q), _ptr(K), _ptr(V), _ptr(W), _ptr(state_in), _ptr(kshift_in),
                        _ptr(kshift), _ptr(dY), _ptr(Y), _ptr(logD), _ptr(dstate_out), _ptr(dQ), _ptr(dK), _ptr(dV),
                        _ptr(dW), _ptr(dstate_in), _ptr(ctx), _ptr(ws), _nbytes(ws), _stream()))
    return dQ, dK, dV, dW, dstate_in


class _Attention(torch.autograd.Function):
    """slim_fwd as a torch operation whose backward is slim_bwd: between the
    two only the key shift and the state-sized context are kept (with the
    inputs and the output Y, which autograd holds anyway; slim_bwd reads Y)."""

    @staticmethod
    def forward(fctx, Q, K, V, W, C, kind, relu_eps, dropout, seed, within):
        c = new_context(Q, W, C, kind, relu_eps, within)
        # the row normalisers (tile-walk mode): 4 bytes per row, kept like Y
        lD = torch.empty(Q.shape[:3], dtype=torch.float32, device=Q.device) if within == "iter" else None
        Y, _, ks = fwd(Q, K, V, W, C, kind, relu_eps=relu_eps, ctx=c, dropout=dropout, seed=seed, within=within,
                       logD=lD)
        fctx.save_for_backward(Q, K, V, W, Y)
        fctx.args = (C, kind, relu_eps, dropout, seed, within, ks, c, lD)
        return Y

    @staticmethod
    def backward(fctx, dY):
        Q, K, V, W, Y = fctx.saved_tensors
        C, kind, relu_eps, dropout, seed, within, ks, c, lD = fctx.args
        dQ, dK, dV, dW, _ = bwd(Q, K, V, W, dY.contiguous(), C, ks, kind, relu_eps=relu_eps, ctx=c, dropout=dropout,
                                seed=seed, within=within, Y=Y, logD=lD)
        return dQ, dK, dV, dW, None, None, None, None, None, None


def attention(Q, K, V, W, C: int, kind="favor+", relu_eps: float = 1e-3, dropout: float = 0.0, seed: int = 0,
              within="iter"):
    """Causal linear attention Y (eq. 2) of Q, K, V [B, H, L, d] with the
    features of W [M, d], computed slice by slice (Algorithm 1), as a
    differentiable torch operation: gradients reach Q, K, V and W through
    slim_bwd.  Arguments as in fwd."""
    return _Attention.apply(Q, K, V, W, C, kind, relu_eps, dropout, seed, within)


def fwd_noalloc(Q, K, V, W, C: int, kind="favor+", state_in=None, kshift_in=None, relu_eps: float = 1e-3,
                Y=None, state_out=None, kshift_out=None, ctx=None, dropout: float = 0.0, seed: int = 0, logD=None):
    """fwd through slim_fwd_noalloc: the library's static device scratch
    replaces the workspace (outputs not passed in are allocated here, by
    torch, before the call; the call itself allocates nothing)."""
    p = _problem_of(Q, W, C, kind, relu_eps, dropout, seed)
    shp = (p.B, p.H, p.L, p.d)
    for n, t in (("Q", Q), ("K", K), ("V", V)):
        _need(t, n, Q.dtype, shp)
    _need(W, "W", torch.float32, (p.M, p.d))
    sshape = (p.B, p.H, p.M, p.d + 1)
    if state_in is not None:
        _need(state_in, "state_in", torch.float32, sshape)
    if kshift_in is not None:
        _need(kshift_in, "kshift_in", torch.float32, (p.B, p.H))
    dev = Q.device
    Y = torch.empty_like(Q) if Y is None else Y
    _need(Y, "Y", Q.dtype, shp)
    state_out = torch.empty(sshape, dtype=torch.float32, device=dev) if state_out is None else state_out
    _need(state_out, "state_out", torch.float32, sshape)
    if p.kind == FAVOR_PLUS and kshift_out is None:
        kshift_out = torch.empty((p.B, p.H), dtype=torch.float32, device=dev)
    if kshift_out is not None:
        _need(kshift_out, "kshift_out", torch.float32, (p.B, p.H))
    _need_ctx(p, ctx)
    if logD is not None:
        _need(logD, "logD", torch.float32, (p.B, p.H, p.L))
    _check(LIB.slim_fwd_noalloc(ctypes.byref(p), _ptr(Q), _ptr(K), _ptr(V), _ptr(W), _ptr(state_in),
                                _ptr(kshift_in), _ptr(Y), _ptr(logD), _ptr(state_out), _ptr(kshift_out), _ptr(ctx),
                                _stream()))
    return Y, state_out, kshift_out


# ---------------------------------------------------------------- the s-layer model (include/slim_model.h)


def model_param_names(s: int):
    """Parameter order of slim_model_step."""
    names = ["emb"]
    for r in range(s):
        names += [f"{n}{r}" for n in ("Wq", "Wk", "Wv", "ln1_g", "ln1_b", "W1", "b1", "W2", "b2", "ln2_g", "ln2_b")]
    return names + ["Wout", "bout"]


def model_param_shapes(s: int, vocab: int, D: int, F: int) -> dict:
    """Shapes of slim_model_step's parameter tensors (include/slim_model.h)."""
    shp = {"emb": (vocab, D), "Wout": (D, vocab), "bout": (vocab,)}
    for r in range(s):
        shp.update({f"Wq{r}": (D, D), f"Wk{r}": (D, D), f"Wv{r}": (D, D), f"W1{r}": (D, F), f"b1{r}": (F,),
                    f"W2{r}": (F, D), f"b2{r}": (D,)})
        for n in ("ln1_g", "ln1_b", "ln2_g", "ln2_b"):
            shp[f"{n}{r}"] = (D,)
    return shp


def model_desc(B, L, D, s, vocab, F, C, ln_eps=1e-5) -> ModelDesc:
    return ModelDesc(int(B), int(L), int(D), int(s), int(vocab), int(F), int(C), float(ln_eps))


def model_workspace_bytes(m: ModelDesc) -> int:
    return int(LIB.slim_model_workspace_bytes(ctypes.byref(m)))


def model_step(params: dict, tokens, C: int, ln_eps: float = 1e-5, ws=None, grads=None, loss=None):
    """Loss and gradient of the s-layer Performer language model by
    Algorithm 1 (include/slim_model.h).  params: float32 device tensors keyed
    by model_param_names(s); tokens: int32 [B, L].  Returns (loss [1],
    grads dict)."""
    s = sum(1 for k in params if k.startswith("Wq"))
    names = model_param_names(s)
    emb = params["emb"]
    vocab, D = emb.shape
    F = params["W10"].shape[1]
    if tokens.dim() == 1:
        tokens = tokens[None]
    B, L = tokens.shape
    m = model_desc(B, L, D, s, vocab, F, C, ln_eps)
    dev = emb.device
    if tokens.device != dev:
        raise ValueError(f"tokens must be on {dev}")
    _need(tokens, "tokens", torch.int32, (B, L))
    shapes = model_param_shapes(s, vocab, D, F)
    for n in names:
        t = params[n]
        if t.device != dev:
            raise ValueError(f"{n} must be on {dev}")
        _need(t, n, torch.float32, shapes[n])
    if grads is None:
        grads = {n: torch.empty_like(params[n]) for n in names}
    for n in names:
        if grads[n].device != dev:
            raise ValueError(f"grad {n} must be on {dev}")
        _need(grads[n], f"grad {n}", torch.float32, shapes[n])
    loss = torch.empty(1, dtype=torch.float32, device=dev) if loss is None else loss
    _need(loss, "loss", torch.float32, (1,))
    need = model_workspace_bytes(m)
    if need == 0:
        raise SlimError(SLIM_EINVAL, LIB.slim_last_error().decode())
    if ws is None:
        ws = torch.empty(need, dtype=torch.uint8, device=dev)
    else:
        _need(ws, "ws", ws.dtype)
        if _nbytes(ws) < need:
            raise ValueError(f"workspace needs {need} bytes, got {_nbytes(ws)}")
    P = (ctypes.c_void_p * len(names))(*[params[n].data_ptr() for n in names])
    G = (ctypes.c_void_p * len(names))(*[grads[n].data_ptr() for n in names])
    _check(LIB.slim_model_step(ctypes.byref(m), _ptr(tokens), P, G, _ptr(loss), _ptr(ws), _nbytes(ws), _stream()))
    return loss, grads
