"""fp64 CPU oracle for slice-wise causal linear attention (SLiM with one layer).

TEST INFRASTRUCTURE ONLY.  Only tests/, __graft_entry__.smoke() and the
cpu_baseline leg of bench.py may import this module.  The product path (the
HIP library and its Python binding) never imports, calls or links it, and
this module imports nothing from the product package.

Notation follows the paper (Sec. 2.1 and Sec. 3): per head, queries, keys and
values Q, K, V in R^{L x d}; a positive feature map g: R^d -> R^M_+;
Q~ = g(Q), K~ = g(K).  Linear causal attention (eq. 2):

    Y_l = sum_{l' <= l} V_l' (g(K_l')^T g(Q_l)) / sum_{l' <= l} g(K_l')^T g(Q_l)

and its prefix-sum form (eqs. 3-4): R = PS(V_l g(K_l)^T) in R^{L x d x M},
S = PS(g(K_l)) in R^{L x M}, Y_l = R_l g(Q_l) / S_l^T g(Q_l).

The slice-wise algorithm (Sec. 3.2-3.3, Algorithms 1-2, eqs. 14-18) with one
layer (s = 1): split the sequence into N = ceil(L/C) slices, carry the state
B = (R, S) at slice ends forward, then walk the slices in reverse, downdating
B (eq. 17), recomputing each slice, and carrying the state cotangent G
(eq. 18).

Feature maps.  The paper only cites the randomized map (Sec. 2.1, after eq. 2);
the FAVOR+ map implemented here is phi(x)_m = exp(w_m . x - |x|^2 / 2) / sqrt(M)
with W in R^{M x d}, and the ReLU map is phi(x)_m = max(w_m . x, 0) + eps.
Both are unstabilised: fp64 has the range for the inputs used here.  The
map of the paper's experiments (Sec. 4, setup) is the element-wise square
g(x) = (x_i^2)_i with M = d; "square" here is phi(x)_m = (w_m . x)^2, which
is that map for W = I_d.

Arrays are float64 numpy.  Per-head functions take [L, d] arrays; the
batched wrappers take [B, H, L, d] and loop over (b, h) one head at a time.
"""

from __future__ import annotations

import math
from typing import List, Optional, Tuple

import numpy as np

FAVOR_PLUS = "favor+"
RELU = "relu"
SQUARE = "square"
RELU_EPS = 1e-3


def _f64(x) -> np.ndarray:
    if hasattr(x, "detach"):  # torch tensor
        x = x.detach().to("cpu").float().numpy()
    return np.asarray(x, dtype=np.float64)


# --------------------------------------------------------------------------
# feature maps (Sec. 2.1: g maps R^d into positive vectors of length M)
# --------------------------------------------------------------------------


def feature_logits(X, W) -> np.ndarray:
    """w_m . x for every row x of X: [..., L, d] x [M, d] -> [..., L, M]."""
    return _f64(X) @ _f64(W).T


def feature_map(X, W, kind: str, relu_eps: float = RELU_EPS) -> np.ndarray:
    """g(X) row by row.  FAVOR+: exp(Wx - |x|^2/2)/sqrt(M); ReLU: max(Wx,0)+eps;
    square: (Wx)^2 (the paper's x^2 map when W = I)."""
    X = _f64(X)
    W = _f64(W)
    z = X @ W.T
    if kind == FAVOR_PLUS:
        return np.exp(z - 0.5 * np.sum(X * X, axis=-1, keepdims=True)) / math.sqrt(W.shape[0])
    if kind == RELU:
        return np.maximum(z, 0.0) + relu_eps
    if kind == SQUARE:
        return z * z
    raise ValueError(kind)


def feature_map_vjp(X, W, Phi, dPhi, kind: str, mask_W=None) -> Tuple[np.ndarray, np.ndarray]:
    """Chain rule through g for one head: returns (dX [L, d], dW [M, d]).

    FAVOR+: d phi_m / dx = phi_m (w_m - x), d phi_m / dw_m = phi_m x.
    ReLU:   d phi_m / dx = [w_m . x > 0] w_m, d phi_m / dw_m = [w_m . x > 0] x
            (derivative 0 taken at w_m . x = 0).
    square: d phi_m / dx = 2 (w_m . x) w_m, d phi_m / dw_m = 2 (w_m . x) x.

    The ReLU derivative is a 0/1 decision on the sign of w_m . x.  `mask_W`
    (default W) is the matrix that decision is taken with: a caller
    comparing against an implementation that forms w_m . x from a rounded W
    passes that rounded W here, so that both sides decide in the same
    precision (the gradient itself always uses W).
    """
    X = _f64(X)
    W = _f64(W)
    if kind == FAVOR_PLUS:
        Gm = dPhi * Phi
        dX = Gm @ W - X * Gm.sum(axis=-1, keepdims=True)
    elif kind == RELU:
        Wd = W if mask_W is None else _f64(mask_W)
        Gm = dPhi * ((X @ Wd.T) > 0.0)
        dX = Gm @ W
    elif kind == SQUARE:
        Gm = dPhi * (2.0 * (X @ W.T))
        dX = Gm @ W
    else:
        raise ValueError(kind)
    dW = Gm.T @ X
    return dX, dW


# --------------------------------------------------------------------------
# the definition: masked quadratic form (eq. 2, first line)
# --------------------------------------------------------------------------


def quadratic_forward_features(Qf, Kf, V):
    """Y from features by eq. 2 (first line).  Returns (Y, A, D) per head.

    A_ll' = g(Q_l)^T g(K_l') for l' <= l (diagonal included), else 0.
    """
    A = np.tril(Qf @ Kf.T)
    D = A.sum(axis=1)
    N = A @ V
    return N / D[:, None], A, D


def quadratic_backward_features(Qf, Kf, V, dY):
    """Analytic VJP of eq. 2 (first line) w.r.t. (Qf, Kf, V) for one head.

    With N = A V, D = A 1, Y = N / D:
      dN = dY / D,  dD = -(dY . Y) / D,
      dA = tril(dN V^T + dD 1^T),
      dV = A^T dN,  dQf = dA Kf,  dKf = dA^T Qf.
    """
    Y, A, D = quadratic_forward_features(Qf, Kf, V)
    dN = dY / D[:, None]
    dD = -np.sum(dY * Y, axis=1) / D
    dA = np.tril(dN @ V.T + dD[:, None])
    return dA @ Kf, dA.T @ Qf, A.T @ dN


def attention_forward(Q, K, V, W, kind: str, relu_eps: float = RELU_EPS) -> np.ndarray:
    """Y for [B, H, L, d] inputs by the definition (eq. 2)."""
    Q, K, V = _f64(Q), _f64(K), _f64(V)
    Y = np.empty_like(V)
    for b in range(Q.shape[0]):
        for h in range(Q.shape[1]):
            Qf = feature_map(Q[b, h], W, kind, relu_eps)
            Kf = feature_map(K[b, h], W, kind, relu_eps)
            Y[b, h] = quadratic_forward_features(Qf, Kf, V[b, h])[0]
    return Y


def attention_backward(Q, K, V, W, dY, kind: str, relu_eps: float = RELU_EPS, mask_W=None):
    """(dQ, dK, dV, dW) of sum(dY * Y) for the definition (eq. 2).

    dW sums the query and key branches over every (b, h) and row.
    `mask_W`: see feature_map_vjp.
    """
    Q, K, V, dY, W = _f64(Q), _f64(K), _f64(V), _f64(dY), _f64(W)
    dQ = np.empty_like(Q)
    dK = np.empty_like(K)
    dV = np.empty_like(V)
    dW = np.zeros_like(W)
    for b in range(Q.shape[0]):
        for h in range(Q.shape[1]):
            Qf = feature_map(Q[b, h], W, kind, relu_eps)
            Kf = feature_map(K[b, h], W, kind, relu_eps)
            dQf, dKf, dV[b, h] = quadratic_backward_features(Qf, Kf, V[b, h], dY[b, h])
            dQ[b, h], dWq = feature_map_vjp(Q[b, h], W, Qf, dQf, kind, mask_W)
            dK[b, h], dWk = feature_map_vjp(K[b, h], W, Kf, dKf, kind, mask_W)
            dW += dWq + dWk
    return dQ, dK, dV, dW


# --------------------------------------------------------------------------
# slices (Sec. 3.2): N = ceil(L / C), A_n = (n - 1) C, B_n = C except the last
# --------------------------------------------------------------------------


def slice_bounds(L: int, C: int) -> List[Tuple[int, int]]:
    """[(A_n, A_n + B_n)] for n = 1..N, 0-based row ranges."""
    if C < 1:
        raise ValueError("slice length C must be >= 1")
    C = min(C, L)
    return [(a, min(a + C, L)) for a in range(0, L, C)]


def _suffix_sum(x: np.ndarray) -> np.ndarray:
    """sum_{l' >= l} x_l' along axis 0: backprop through a prefix sum (Sec. 3.3)."""
    return np.flip(np.cumsum(np.flip(x, axis=0), axis=0), axis=0)


# --------------------------------------------------------------------------
# Algorithm 1 (s = 1), forward sweep
# --------------------------------------------------------------------------


def slim_forward_head(Q, K, V, W, C: int, kind: str, R0=None, S0=None, within: str = "ps",
                      relu_eps: float = RELU_EPS):
    """Forward sweep of Algorithm 1 for one head.

    B^(0) = (R0, S0) (zero by default); for each slice n the slice's prefix
    states are U^(n) = 1 B^(n-1)^T + PS(T^(n)) (eq. 15) with
    T_l = (V_l g(K_l)^T, g(K_l)); the outputs follow eq. 4 and
    B^(n) = U^(n)_{B_n}.

    `within` chooses how the in-slice prefix sum is evaluated:
      "ps"        explicit prefix sums over [B_n, d, M] (the paper's "PS");
      "quadratic" the masked quadratic form of eq. 2 (first line) inside the
                  slice plus the carried state (eq. 2 second line for B).
    Both give the same numbers up to rounding.

    Returns (Y [L, d], R [d, M], S [M]).
    """
    Q, K, V = _f64(Q), _f64(K), _f64(V)
    L, d = V.shape
    M = _f64(W).shape[0]
    R = np.zeros((d, M)) if R0 is None else _f64(R0).copy()
    S = np.zeros(M) if S0 is None else _f64(S0).copy()
    Y = np.empty((L, d))
    for a, b in slice_bounds(L, C):
        Qf = feature_map(Q[a:b], W, kind, relu_eps)
        Kf = feature_map(K[a:b], W, kind, relu_eps)
        Vs = V[a:b]
        if within == "ps":
            U_R = R[None] + np.cumsum(np.einsum("ld,lm->ldm", Vs, Kf), axis=0)
            U_S = S[None] + np.cumsum(Kf, axis=0)
            N = np.einsum("ldm,lm->ld", U_R, Qf)
            D = np.einsum("lm,lm->l", U_S, Qf)
            R, S = U_R[-1], U_S[-1]
        elif within == "quadratic":
            A = np.tril(Qf @ Kf.T)
            N = Qf @ R.T + A @ Vs
            D = Qf @ S + A.sum(axis=1)
            R = R + Vs.T @ Kf
            S = S + Kf.sum(axis=0)
        else:
            raise ValueError(within)
        Y[a:b] = N / D[:, None]
    return Y, R, S


# --------------------------------------------------------------------------
# Algorithm 1 (s = 1), backward sweep with updateProc(n, True)
# --------------------------------------------------------------------------


def slim_backward_head(Q, K, V, W, dY, C: int, kind: str, R_N, S_N, gR=None, gS=None,
                       within: str = "ps", relu_eps: float = RELU_EPS, mask_W=None):
    """Backward sweep of Algorithm 1 for one head.

    Starts from B^(N) = (R_N, S_N), the state the forward sweep returned,
    and G^(N) = (gR, gS) (zero by default: nothing after the sequence depends
    on B^(N)).  For n = N..1:
      * downdate B^(n-1) = B^(n) - sum_l T_l^(n)                  (eq. 17)
      * recompute the slice from B^(n-1)
      * differentiate Phi^(n) = sum_l dY_l . Y_l + <G^(n), B^(n)>  (Sec. 3.3)
        w.r.t. the slice inputs and w.r.t. B^(n-1): the latter is G^(n-1)
                                                                  (eq. 18)
      * accumulate the slice's share of dW (grad_theta = sum_n grad_theta^(n)).

    Returns (dQ [L, d], dK [L, d], dV [L, d], dW [M, d], gR [d, M], gS [M]);
    (gR, gS) at the end is G^(0), the gradient w.r.t. the initial state.
    """
    Q, K, V, dY = _f64(Q), _f64(K), _f64(V), _f64(dY)
    W = _f64(W)
    L, d = V.shape
    M = W.shape[0]
    R = _f64(R_N).copy()
    S = _f64(S_N).copy()
    gR = np.zeros((d, M)) if gR is None else _f64(gR).copy()
    gS = np.zeros(M) if gS is None else _f64(gS).copy()
    dQ = np.empty((L, d))
    dK = np.empty((L, d))
    dV = np.empty((L, d))
    dW = np.zeros((M, d))
    for a, b in reversed(slice_bounds(L, C)):
        Qf = feature_map(Q[a:b], W, kind, relu_eps)
        Kf = feature_map(K[a:b], W, kind, relu_eps)
        Vs, dYs = V[a:b], dY[a:b]
        # eq. 17: B^(n-1) = B^(n) - sum of the slice's T rows
        R = R - Vs.T @ Kf
        S = S - Kf.sum(axis=0)
        if within == "ps":
            U_R = R[None] + np.cumsum(np.einsum("ld,lm->ldm", Vs, Kf), axis=0)
            U_S = S[None] + np.cumsum(Kf, axis=0)
            N = np.einsum("ldm,lm->ld", U_R, Qf)
            D = np.einsum("lm,lm->l", U_S, Qf)
            Ys = N / D[:, None]
            dN = dYs / D[:, None]
            dD = -np.sum(dYs * Ys, axis=1) / D
            # cotangents of the slice's prefix states U_l
            gU_R = np.einsum("ld,lm->ldm", dN, Qf)
            gU_S = dD[:, None] * Qf
            gU_R[-1] += gR  # Phi gains <G, U_last>
            gU_S[-1] += gS
            dQf = np.einsum("ldm,ld->lm", U_R, dN) + U_S * dD[:, None]
            # through U = 1 B^T + PS(T): a reversed prefix sum for T, a sum for B
            gT_R = _suffix_sum(gU_R)
            gT_S = _suffix_sum(gU_S)
            gR, gS = gT_R[0], gT_S[0]
            dKf = np.einsum("ldm,ld->lm", gT_R, Vs) + gT_S
            dVs = np.einsum("ldm,lm->ld", gT_R, Kf)
        elif within == "quadratic":
            A = np.tril(Qf @ Kf.T)
            N = Qf @ R.T + A @ Vs
            D = Qf @ S + A.sum(axis=1)
            Ys = N / D[:, None]
            dN = dYs / D[:, None]
            dD = -np.sum(dYs * Ys, axis=1) / D
            dA = np.tril(dN @ Vs.T + dD[:, None])
            dQf = dN @ R + dD[:, None] * S[None, :] + dA @ Kf
            dKf = Vs @ gR + gS[None, :] + dA.T @ Qf
            dVs = Kf @ gR.T + A.T @ dN
            gR = gR + dN.T @ Qf
            gS = gS + Qf.T @ dD
        else:
            raise ValueError(within)
        dQ[a:b], dWq = feature_map_vjp(Q[a:b], W, Qf, dQf, kind, mask_W)
        dK[a:b], dWk = feature_map_vjp(K[a:b], W, Kf, dKf, kind, mask_W)
        dV[a:b] = dVs
        dW += dWq + dWk
    return dQ, dK, dV, dW, gR, gS


# --------------------------------------------------------------------------
# batched wrappers; the state travels in the layout [B, H, M, d + 1]
# (columns 0..d-1 hold R^T = sum g(k) v^T, column d holds S = sum g(k))
# --------------------------------------------------------------------------


def pack_state(R: np.ndarray, S: np.ndarray) -> np.ndarray:
    """(R [..., d, M], S [..., M]) -> [..., M, d + 1]."""
    return np.concatenate([np.swapaxes(R, -1, -2), S[..., None]], axis=-1)


def unpack_state(P) -> Tuple[np.ndarray, np.ndarray]:
    """[..., M, d + 1] -> (R [..., d, M], S [..., M])."""
    P = _f64(P)
    return np.swapaxes(P[..., :-1], -1, -2), P[..., -1]


def slim_forward(Q, K, V, W, C: int, kind: str, state_in=None, within: str = "ps",
                 relu_eps: float = RELU_EPS):
    """Algorithm 1 forward for [B, H, L, d] inputs.

    Returns (Y [B, H, L, d], state_out [B, H, M, d + 1]).
    """
    Q, K, V = _f64(Q), _f64(K), _f64(V)
    Bn, Hn, L, d = V.shape
    M = _f64(W).shape[0]
    Y = np.empty_like(V)
    st = np.empty((Bn, Hn, M, d + 1))
    for b in range(Bn):
        for h in range(Hn):
            R0 = S0 = None
            if state_in is not None:
                R0, S0 = unpack_state(_f64(state_in)[b, h])
            Y[b, h], R, S = slim_forward_head(Q[b, h], K[b, h], V[b, h], W, C, kind, R0, S0, within, relu_eps)
            st[b, h] = pack_state(R, S)
    return Y, st


def slim_backward(Q, K, V, W, dY, C: int, kind: str, state_out, dstate_out=None, within: str = "ps",
                  relu_eps: float = RELU_EPS, mask_W=None):
    """Algorithm 1 backward for [B, H, L, d] inputs.

    `state_out` is B^(N) from slim_forward; `dstate_out` is G^(N) (zero if
    None).  Returns (dQ, dK, dV, dW [M, d], dstate_in [B, H, M, d + 1]).
    """
    Q, K, V, dY = _f64(Q), _f64(K), _f64(V), _f64(dY)
    Bn, Hn, L, d = V.shape
    M = _f64(W).shape[0]
    dQ = np.empty_like(Q)
    dK = np.empty_like(K)
    dV = np.empty_like(V)
    dW = np.zeros((M, d))
    gst = np.empty((Bn, Hn, M, d + 1))
    for b in range(Bn):
        for h in range(Hn):
            R_N, S_N = unpack_state(_f64(state_out)[b, h])
            gR = gS = None
            if dstate_out is not None:
                gR, gS = unpack_state(_f64(dstate_out)[b, h])
            dQ[b, h], dK[b, h], dV[b, h], dWh, gR, gS = slim_backward_head(
                Q[b, h], K[b, h], V[b, h], W, dY[b, h], C, kind, R_N, S_N, gR, gS, within, relu_eps, mask_W)
            dW += dWh
            gst[b, h] = pack_state(gR, gS)
    return dQ, dK, dV, dW, gst


# --------------------------------------------------------------------------
# the per-token iterative scheme (Appendix B, first part), from features.
# Used only as a cross-check of the definition on small inputs.
# --------------------------------------------------------------------------


def iterative_forward_features(Qf, Kf, V):
    """Token-by-token curR/curS recurrence (App. B).  Returns (Y, N, D, curR, curS)."""
    L, d = V.shape
    M = Qf.shape[1]
    curR = np.zeros((d, M))
    curS = np.zeros(M)
    N = np.empty((L, d))
    D = np.empty(L)
    for l in range(L):
        curR += np.outer(V[l], Kf[l])
        curS += Kf[l]
        N[l] = curR @ Qf[l]
        D[l] = curS @ Qf[l]
    return N / D[:, None], N, D, curR, curS


def iterative_backward_features(Qf, Kf, V, dN, dD, curR, curS):
    """Reverse token walk of App. B given dL/dN and dL/dD.

    Differs from the printed listing in one place: the key cotangent also
    receives gradS (gradS is accumulated there but never read; S_l depends
    on g(K_l) for every later row, so its cotangent flows back to K).
    Returns (dQf, dKf, dV).
    """
    L, d = V.shape
    M = Qf.shape[1]
    curR = curR.copy()
    curS = curS.copy()
    gradR = np.zeros((d, M))
    gradS = np.zeros(M)
    dQf = np.empty((L, M))
    dKf = np.empty((L, M))
    dV = np.empty((L, d))
    for l in range(L - 1, -1, -1):
        dQf[l] = dD[l] * curS + curR.T @ dN[l]
        curR -= np.outer(V[l], Kf[l])
        curS -= Kf[l]
        gradR += np.outer(dN[l], Qf[l])
        gradS += dD[l] * Qf[l]
        dV[l] = gradR @ Kf[l]
        dKf[l] = gradR.T @ V[l] + gradS
    return dQf, dKf, dV
