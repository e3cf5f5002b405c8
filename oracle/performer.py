"""fp64 CPU oracle for the s-layer Performer language model (Sec. 2.2, eqs.
5-10) and its low-memory training step (Algorithm 1 with Algorithm 2:
slices in the outer loop, layers in the inner loop).

TEST INFRASTRUCTURE ONLY.  Only tests/, __graft_entry__.smoke() and the
cpu_baseline leg of bench.py may import this module.  The product path never
imports, calls or links it, and this module imports nothing from the product
package.

The model (Sec. 2.2), for a batch of token sequences p in {0..V-1}^L:

    X0_l    = E[p_l] + PE(l)                           (emb: token embedding plus sinusoids)
    for r = 1..s:
      A     = [Att(X Wq_j, X Wk_j, X Wv_j)]_j          (eqs. 7-8: heads side by side)
      H     = LN1(A) + X                               (eq. 5)
      X     = LN2(GeLU(H W1 + b1) W2 + b2) + H         (eqs. 6, 9)
    X_out   = X Wout + bout
    loss    = mean over the batch of (L - 1)^-1 sum_{l < L} CE(X_out_l, p_{l+1})   (eq. 10)

Att is the causal linear attention of eq. 2 with the element-wise square map
g(x) = (x_i^2) and M = d (Sec. 4), i.e. the oracle's "square" kind with
W = I_d.  Readings (the paper is silent): PE(l, 2i) = sin(l / 10000^(2i/D)),
PE(l, 2i + 1) = cos(l / 10000^(2i/D)) with positions counted from 0, the
embedding is the plain sum E[p_l] + PE(l), layer normalisation has
eps = 1e-5, GeLU is the exact x Phi(x), and a batch averages eq. 10 over
its sequences.

Two evaluations: `model_full` runs eqs. 5-10 over the whole sequence with
hand-written backward steps; `model_algorithm1` runs Algorithm 1: the
forward carries the attention states B_r of every layer across slices, the
backward walks the slices in reverse, downdating each B_r by what the slice
added (eq. 17), recomputing the slice through all layers and carrying the
state cotangents G_r (eq. 18).  Both return (loss, grads) with grads keyed
like the parameters.
"""

from __future__ import annotations

import math
from typing import Dict, List, Tuple

import numpy as np

from .slim_oracle import attention_backward, attention_forward, slice_bounds, slim_backward, slim_forward

LN_EPS = 1e-5
HEAD_DIM = 64  # d of every head in the paper's configurations (k = d_model / 64)


def _f64(x) -> np.ndarray:
    if hasattr(x, "detach"):
        x = x.detach().cpu().double().numpy()
    return np.asarray(x, dtype=np.float64)


def param_names(s: int) -> List[str]:
    """Parameter keys, in a fixed order."""
    names = ["emb"]
    for r in range(s):
        names += [f"{n}{r}" for n in ("Wq", "Wk", "Wv", "ln1_g", "ln1_b", "W1", "b1", "W2", "b2", "ln2_g", "ln2_b")]
    return names + ["Wout", "bout"]


# ---------------------------------------------------------------- pieces


def positions(l0: int, n: int, D: int) -> np.ndarray:
    """Sinusoidal positional embedding of positions l0 .. l0 + n - 1 (Sec. 2.2, emb)."""
    pos = np.arange(l0, l0 + n, dtype=np.float64)[:, None]
    i = np.arange(D // 2, dtype=np.float64)[None, :]
    ang = pos / np.power(10000.0, 2.0 * i / D)
    pe = np.empty((n, D))
    pe[:, 0::2] = np.sin(ang)
    pe[:, 1::2] = np.cos(ang)
    return pe


def layer_norm(x, g, b, eps=LN_EPS):
    """Row-wise layer normalisation; returns (y, (xhat, rstd)) for the backward."""
    mu = x.mean(axis=-1, keepdims=True)
    xc = x - mu
    var = (xc * xc).mean(axis=-1, keepdims=True)
    rstd = 1.0 / np.sqrt(var + eps)
    xhat = xc * rstd
    return xhat * g + b, (xhat, rstd)


def layer_norm_vjp(dy, g, cache):
    """(dx, dg, db) of layer_norm for the cotangent dy."""
    xhat, rstd = cache
    D = xhat.shape[-1]
    dxh = dy * g
    dx = rstd / D * (D * dxh - dxh.sum(axis=-1, keepdims=True) - xhat * (dxh * xhat).sum(axis=-1, keepdims=True))
    dg = (dy * xhat).reshape(-1, D).sum(axis=0)
    db = dy.reshape(-1, D).sum(axis=0)
    return dx, dg, db


_SQRT2 = math.sqrt(2.0)
_erf = np.vectorize(math.erf)


def gelu(x):
    """x Phi(x) with Phi the standard normal CDF (exact GeLU)."""
    return 0.5 * x * (1.0 + _erf(x / _SQRT2))


def gelu_grad(x):
    """d/dx (x Phi(x)) = Phi(x) + x phi(x)."""
    return 0.5 * (1.0 + _erf(x / _SQRT2)) + x * np.exp(-0.5 * x * x) / math.sqrt(2.0 * math.pi)


def next_token_loss(logits, tokens, l0: int, L: int):
    """Eq. 10 restricted to rows l0 .. l0 + n - 1 of every sequence: the sum of
    CE(logits_l, p_{l+1}) over rows l < L - 1, times 1 / ((L - 1) B).
    Returns (loss, dlogits)."""
    Bn, n, Vn = logits.shape
    z = logits - logits.max(axis=-1, keepdims=True)
    lse = np.log(np.exp(z).sum(axis=-1, keepdims=True))
    logp = z - lse
    w = np.zeros((Bn, n))
    tgt = np.zeros((Bn, n), dtype=np.int64)
    for j in range(n):
        l = l0 + j
        if l < L - 1:
            w[:, j] = 1.0 / ((L - 1) * Bn)
            tgt[:, j] = tokens[:, l + 1]
    loss = -(w * np.take_along_axis(logp, tgt[..., None], axis=-1)[..., 0]).sum()
    d = np.exp(logp)
    np.put_along_axis(d, tgt[..., None], np.take_along_axis(d, tgt[..., None], axis=-1) - 1.0, axis=-1)
    return loss, d * w[..., None]


def _heads(X, W, k):
    """[B, n, D] @ W [D, D] -> [B, k, n, d] (head j = columns j d .. (j + 1) d)."""
    Bn, n, _ = X.shape
    return (X @ W).reshape(Bn, n, k, -1).transpose(0, 2, 1, 3)


def _merge(Z):
    """[B, k, n, d] -> [B, n, k d]."""
    Bn, k, n, d = Z.shape
    return Z.transpose(0, 2, 1, 3).reshape(Bn, n, k * d)


# ---------------------------------------------------------------- one layer


def _layer_forward(P, r, X, att):
    """Eqs. 5-9 for layer r on rows X [B, n, D]; att(Q, K, V) -> Y per head.
    Returns (X_next, cache)."""
    k = P["_k"]
    Q, K, V = (_heads(X, P[f"{n}{r}"], k) for n in ("Wq", "Wk", "Wv"))
    A = _merge(att(Q, K, V))
    n1, c1 = layer_norm(A, P[f"ln1_g{r}"], P[f"ln1_b{r}"])
    H = n1 + X
    Z1 = H @ P[f"W1{r}"] + P[f"b1{r}"]
    G1 = gelu(Z1)
    F = G1 @ P[f"W2{r}"] + P[f"b2{r}"]
    n2, c2 = layer_norm(F, P[f"ln2_g{r}"], P[f"ln2_b{r}"])
    return n2 + H, dict(X=X, Q=Q, K=K, V=V, c1=c1, H=H, Z1=Z1, G1=G1, c2=c2, k=k)


def _layer_backward(P, r, dXn, c, att_vjp, grads):
    """Backward of _layer_forward: adds parameter gradients to `grads`,
    returns dX.  att_vjp(Q, K, V, dY) -> (dQ, dK, dV) per head."""
    dF, dg2, db2n = layer_norm_vjp(dXn, P[f"ln2_g{r}"], c["c2"])
    dH = dXn.copy()
    grads[f"ln2_g{r}"] += dg2
    grads[f"ln2_b{r}"] += db2n
    D = dF.shape[-1]
    grads[f"W2{r}"] += c["G1"].reshape(-1, c["G1"].shape[-1]).T @ dF.reshape(-1, D)
    grads[f"b2{r}"] += dF.reshape(-1, D).sum(axis=0)
    dZ1 = (dF @ P[f"W2{r}"].T) * gelu_grad(c["Z1"])
    grads[f"W1{r}"] += c["H"].reshape(-1, D).T @ dZ1.reshape(-1, dZ1.shape[-1])
    grads[f"b1{r}"] += dZ1.reshape(-1, dZ1.shape[-1]).sum(axis=0)
    dH += dZ1 @ P[f"W1{r}"].T
    dA, dg1, db1n = layer_norm_vjp(dH, P[f"ln1_g{r}"], c["c1"])
    grads[f"ln1_g{r}"] += dg1
    grads[f"ln1_b{r}"] += db1n
    dX = dH.copy()
    k = c["k"]
    Bn, n, _ = dA.shape
    dAh = dA.reshape(Bn, n, k, -1).transpose(0, 2, 1, 3)
    dQ, dK, dV = att_vjp(c["Q"], c["K"], c["V"], dAh)
    X2 = c["X"].reshape(-1, D)
    for name, dZ in (("Wq", dQ), ("Wk", dK), ("Wv", dV)):
        dZm = _merge(dZ).reshape(-1, D)
        grads[f"{name}{r}"] += X2.T @ dZm
        dX += (dZm @ P[f"{name}{r}"].T).reshape(dX.shape)
    return dX


def _embed(P, tokens, l0, n):
    return P["emb"][tokens[:, l0:l0 + n]] + positions(l0, n, P["emb"].shape[1])[None]


def _embed_backward(grads, tokens, l0, n, dX0):
    idx = tokens[:, l0:l0 + n].reshape(-1)
    np.add.at(grads["emb"], idx, dX0.reshape(-1, dX0.shape[-1]))


def _prepare(params, tokens):
    P = {k: _f64(v) for k, v in params.items()}
    tokens = np.asarray(tokens.cpu() if hasattr(tokens, "cpu") else tokens, dtype=np.int64)
    if tokens.ndim == 1:
        tokens = tokens[None]
    s = sum(1 for k in P if k.startswith("Wq"))
    D = P["emb"].shape[1]
    P["_k"] = max(1, D // HEAD_DIM)
    return P, tokens, s


def _zero_grads(P):
    return {k: np.zeros_like(v) for k, v in P.items() if not k.startswith("_")}


def _identity(d):
    return np.eye(d)


# ---------------------------------------------------------------- the whole sequence (definition)


def model_full(params, tokens, heads: int = None):
    """Loss (eq. 10) and its gradient over the whole sequence (eqs. 5-10).
    `heads` overrides the head count k (default d_model / 64)."""
    P, tokens, s = _prepare(params, tokens)
    if heads is not None:
        P["_k"] = heads
    Bn, L = tokens.shape
    D = P["emb"].shape[1]
    d = D // P["_k"]
    I = _identity(d)
    att = lambda Q, K, V: attention_forward(Q, K, V, I, "square")
    att_vjp = lambda Q, K, V, dY: attention_backward(Q, K, V, I, dY, "square")[:3]
    X = _embed(P, tokens, 0, L)
    caches = []
    for r in range(s):
        X, c = _layer_forward(P, r, X, att)
        caches.append(c)
    logits = X @ P["Wout"] + P["bout"]
    loss, dlog = next_token_loss(logits, tokens, 0, L)
    grads = _zero_grads(P)
    grads["Wout"] += X.reshape(-1, D).T @ dlog.reshape(-1, dlog.shape[-1])
    grads["bout"] += dlog.reshape(-1, dlog.shape[-1]).sum(axis=0)
    dX = dlog @ P["Wout"].T
    for r in reversed(range(s)):
        dX = _layer_backward(P, r, dX, caches[r], att_vjp, grads)
    _embed_backward(grads, tokens, 0, L, dX)
    return loss, grads


def model_loss(params, tokens, heads: int = None) -> float:
    """The forward of model_full only (for finite differences)."""
    P, tokens, s = _prepare(params, tokens)
    if heads is not None:
        P["_k"] = heads
    Bn, L = tokens.shape
    d = P["emb"].shape[1] // P["_k"]
    att = lambda Q, K, V: attention_forward(Q, K, V, _identity(d), "square")
    X = _embed(P, tokens, 0, L)
    for r in range(s):
        X, _ = _layer_forward(P, r, X, att)
    return next_token_loss(X @ P["Wout"] + P["bout"], tokens, 0, L)[0]


# ---------------------------------------------------------------- Algorithm 1


def model_algorithm1(params, tokens, C: int, heads: int = None):
    """Loss and gradient by Algorithm 1 (Sec. 3.2-3.3): slices of C rows in
    the outer loop, layers in the inner loop; only the attention states
    B_r (forward) and B_r, G_r (backward) cross slice boundaries."""
    P, tokens, s = _prepare(params, tokens)
    if heads is not None:
        P["_k"] = heads
    Bn, L = tokens.shape
    D = P["emb"].shape[1]
    k = P["_k"]
    d = D // k
    I = _identity(d)
    slices = slice_bounds(L, C)

    # forward (updateProc with onBackprop = False): B_r carried across slices
    Bst = [np.zeros((Bn, k, d, d + 1)) for _ in range(s)]
    loss = 0.0
    for (a, b) in slices:
        X = _embed(P, tokens, a, b - a)
        for r in range(s):
            def att(Q, K, V, r=r):
                Y, st = slim_forward(Q, K, V, I, b - a, "square", state_in=Bst[r], within="quadratic")
                Bst[r] = st
                return Y
            X, _ = _layer_forward(P, r, X, att)
        loss += next_token_loss(X @ P["Wout"] + P["bout"], tokens, a, L)[0]

    # backward (updateProc with onBackprop = True), slices in reverse
    grads = _zero_grads(P)
    G = [np.zeros_like(x) for x in Bst]
    for (a, b) in reversed(slices):
        n = b - a
        X = _embed(P, tokens, a, n)
        caches, after, before = [], [], []
        for r in range(s):
            def att(Q, K, V, r=r):
                # eq. 17: the state before the slice = the state after it
                # minus the slice's own sum
                delta = slim_forward(Q, K, V, I, n, "square", within="quadratic")[1]
                prev = Bst[r] - delta
                after.append(Bst[r])
                before.append(prev)
                return slim_forward(Q, K, V, I, n, "square", state_in=prev, within="quadratic")[0]
            X, c = _layer_forward(P, r, X, att)
            caches.append(c)
        logits = X @ P["Wout"] + P["bout"]
        _, dlog = next_token_loss(logits, tokens, a, L)
        grads["Wout"] += X.reshape(-1, D).T @ dlog.reshape(-1, dlog.shape[-1])
        grads["bout"] += dlog.reshape(-1, dlog.shape[-1]).sum(axis=0)
        dX = dlog @ P["Wout"].T
        for r in reversed(range(s)):
            def att_vjp(Q, K, V, dY, r=r):
                # eq. 18: the cotangent of the state before the slice
                dQ, dK, dV, _, gin = slim_backward(Q, K, V, I, dY, n, "square", after[r], dstate_out=G[r],
                                                   within="quadratic")
                G[r] = gin
                return dQ, dK, dV
            dX = _layer_backward(P, r, dX, caches[r], att_vjp, grads)
        _embed_backward(grads, tokens, a, n, dX)
        for r in range(s):
            Bst[r] = before[r]
    return loss, grads


def grad_discrepancy(g, ref) -> float:
    """||g - ref||_2 / ||ref||_2 over all parameters (the relative
    discrepancy of Sec. 4.1)."""
    num = sum(float(np.sum((_f64(g[k]) - _f64(ref[k])) ** 2)) for k in ref)
    den = sum(float(np.sum(_f64(ref[k]) ** 2)) for k in ref)
    return math.sqrt(num / den)
