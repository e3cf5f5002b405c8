"""Plant plausible slips in the oracle (on the CPU) and check that a pin fails.

Each mutant replaces one oracle function by a copy with one mistake; the
listed pin from test_oracle_pins.py must then raise (an assertion, or a
non-finite value tripping one).
"""

import math

import numpy as np
import pytest

import oracle.slim_oracle as S
import tests.test_oracle_pins as P


def _favor_no_sqrtM(X, W, kind, relu_eps=S.RELU_EPS):
    X, W = S._f64(X), S._f64(W)
    z = X @ W.T
    if kind == S.FAVOR_PLUS:
        return np.exp(z - 0.5 * np.sum(X * X, axis=-1, keepdims=True))
    return np.maximum(z, 0.0) + relu_eps


def _favor_sign_flip(X, W, kind, relu_eps=S.RELU_EPS):
    X, W = S._f64(X), S._f64(W)
    z = X @ W.T
    if kind == S.FAVOR_PLUS:
        return np.exp(z + 0.5 * np.sum(X * X, axis=-1, keepdims=True)) / math.sqrt(W.shape[0])
    return np.maximum(z, 0.0) + relu_eps


def _relu_no_eps(X, W, kind, relu_eps=S.RELU_EPS):
    X, W = S._f64(X), S._f64(W)
    z = X @ W.T
    if kind == S.RELU:
        return np.maximum(z, 0.0)
    return np.exp(z - 0.5 * np.sum(X * X, axis=-1, keepdims=True)) / math.sqrt(W.shape[0])


def _strict_mask(Qf, Kf, V):
    A = np.tril(Qf @ Kf.T, k=-1)
    D = A.sum(axis=1)
    with np.errstate(divide="ignore", invalid="ignore"):
        return (A @ V) / D[:, None], A, D


def _upper_mask(Qf, Kf, V):
    A = np.triu(Qf @ Kf.T)
    D = A.sum(axis=1)
    return (A @ V) / D[:, None], A, D


def _bwd_no_dD(Qf, Kf, V, dY):
    Y, A, D = S.quadratic_forward_features(Qf, Kf, V)
    dN = dY / D[:, None]
    dA = np.tril(dN @ V.T)
    return dA @ Kf, dA.T @ Qf, A.T @ dN


def _bwd_transposed_dA(Qf, Kf, V, dY):
    Y, A, D = S.quadratic_forward_features(Qf, Kf, V)
    dN = dY / D[:, None]
    dD = -np.sum(dY * Y, axis=1) / D
    dA = np.tril(dN @ V.T + dD[:, None])
    return dA.T @ Kf, dA @ Qf, A.T @ dN


def _vjp_no_norm_term(X, W, Phi, dPhi, kind, mask_W=None):
    X, W = S._f64(X), S._f64(W)
    Gm = dPhi * Phi if kind == S.FAVOR_PLUS else dPhi * ((X @ W.T) > 0.0)
    return Gm @ W, Gm.T @ X


def _iter_bwd_printed(Qf, Kf, V, dN, dD, curR, curS):
    # the recurrence as printed: the key cotangent misses gradS
    L, d = V.shape
    M = Qf.shape[1]
    curR, curS = curR.copy(), curS.copy()
    gradR, gradS = np.zeros((d, M)), np.zeros(M)
    dQf, dKf, dVv = np.empty((L, M)), np.empty((L, M)), np.empty((L, d))
    for l in range(L - 1, -1, -1):
        dQf[l] = dD[l] * curS + curR.T @ dN[l]
        curR -= np.outer(V[l], Kf[l])
        curS -= Kf[l]
        gradR += np.outer(dN[l], Qf[l])
        gradS += dD[l] * Qf[l]
        dVv[l] = gradR @ Kf[l]
        dKf[l] = gradR.T @ V[l]
    return dQf, dKf, dVv


def _slim_bwd_no_downdate(Q, K, V, W, dY, C, kind, R_N, S_N, gR=None, gS=None, within="ps", relu_eps=S.RELU_EPS,
                          mask_W=None):
    # skip eq. 17 by adding back what the real routine subtracts
    Wf = S._f64(W)
    Kf_all = S.feature_map(S._f64(K), Wf, kind, relu_eps)
    V_ = S._f64(V)
    out = list(_REAL_BWD(Q, K, V, W, dY, C, kind, S._f64(R_N) + V_.T @ Kf_all, S._f64(S_N) + Kf_all.sum(0),
                         gR, gS, within, relu_eps, mask_W))
    return tuple(out)


_REAL_BWD = S.slim_backward_head


def _vjp_square_no_two(X, W, Phi, dPhi, kind, mask_W=None):
    # the square map's derivative without its factor 2
    X, W = S._f64(X), S._f64(W)
    if kind == S.SQUARE:
        Gm = dPhi * (X @ W.T)
        return Gm @ W, Gm.T @ X
    return _REAL_VJP(X, W, Phi, dPhi, kind, mask_W)


_REAL_VJP = S.feature_map_vjp


def _pack_no_transpose(R, S_):
    # R [.., d, M] laid out without the swap (only shape-compatible when d = M)
    return np.concatenate([R, S_[..., None]], axis=-1)


def _unpack_ones_first(P_):
    P_ = S._f64(P_)
    return np.swapaxes(P_[..., 1:], -1, -2), P_[..., 0]


def _logits_transposed_w(X, W):
    return S._f64(X) @ S._f64(W)


MUTANTS = [
    ("feature_map", _favor_no_sqrtM, lambda: P.test_favor_plus_is_unbiased_for_the_exponential_kernel()),
    ("feature_map", _favor_sign_flip, lambda: P.test_favor_plus_is_unbiased_for_the_exponential_kernel()),
    ("feature_map", _relu_no_eps, lambda: P.test_relu_map_with_identity_features()),
    ("quadratic_forward_features", _strict_mask, lambda: P.test_first_output_is_first_value(S.FAVOR_PLUS)),
    ("quadratic_forward_features", _upper_mask, lambda: P.test_first_output_is_first_value(S.RELU)),
    ("quadratic_backward_features", _bwd_no_dD, lambda: P.test_gradients_match_finite_differences(S.FAVOR_PLUS)),
    ("quadratic_backward_features", _bwd_transposed_dA, lambda: P.test_gradients_match_finite_differences(S.RELU)),
    ("feature_map_vjp", _vjp_no_norm_term, lambda: P.test_gradients_match_finite_differences(S.FAVOR_PLUS)),
    ("iterative_backward_features", _iter_bwd_printed, lambda: P.test_token_recurrence_equals_definition()),
    ("slim_backward_head", _slim_bwd_no_downdate,
     lambda: P.test_slicewise_equals_definition_for_every_slice_length(S.FAVOR_PLUS, "quadratic", 3)),
    ("feature_map_vjp", _vjp_square_no_two, lambda: P.test_gradients_match_finite_differences(S.SQUARE)),
    ("pack_state", _pack_no_transpose, lambda: P.test_state_layout_written_out_by_loops()),
    ("unpack_state", _unpack_ones_first, lambda: P.test_state_layout_written_out_by_loops()),
    ("feature_logits", _logits_transposed_w, lambda: P.test_feature_logits_written_out_by_loops()),
]


@pytest.mark.parametrize("idx", range(len(MUTANTS)))
def test_planted_mistake_is_caught(idx, monkeypatch):
    name, fn, pin = MUTANTS[idx]
    monkeypatch.setattr(S, name, fn)
    # the test module imported `oracle` as O, whose attributes are the originals
    import oracle as O

    monkeypatch.setattr(O, name, fn, raising=False)
    with np.errstate(all="ignore"):
        with pytest.raises((AssertionError, FloatingPointError, ValueError)):
            pin()
