"""Pins of the fp64 oracle against facts that do not come from the oracle itself.

Every check here is chosen so that a plausible slip in the oracle (a dropped
term, a wrong sign, a transposed operand, an off-by-one in the causal mask or
the slicing) fails at least one of them; test_oracle_mutations.py plants such
slips and confirms it.

* finite differences of the forward definition pin every analytic gradient;
* the causal mask and the normaliser are pinned by closed forms: Y_1 = v_1,
  constant keys give a running mean, constant values give a constant output;
* the FAVOR+ map is pinned by its defining property, E_w[g(q)^T g(k)] =
  exp(q^T k) for w ~ N(0, I_d), and by the limit M -> inf, where causal
  linear attention approaches causal softmax attention (eq. 1; scipy's
  softmax is the reference);
* the slice-wise algorithm (Algorithms 1-2) is pinned by its exactness claim:
  the result does not depend on C (Sec. 1, Sec. 4), so it must equal the
  definition for C in {1, 2, 3, 7, L};
* the token-by-token recurrence of Appendix B (with the gradS term restored)
  must equal the definition as well.
"""

import math

import numpy as np
import pytest
import scipy.special

import oracle as O
from synth import orthogonal_gaussian_features


def _rand(shape, seed, scale=1.0):
    return np.random.default_rng(seed).standard_normal(shape) * scale


def _problem(B=1, H=2, L=9, d=3, M=5, seed=0, kind=O.FAVOR_PLUS):
    rng = np.random.default_rng(seed)
    s = d ** -0.25
    Q = rng.standard_normal((B, H, L, d)) * s
    K = rng.standard_normal((B, H, L, d)) * s
    V = rng.standard_normal((B, H, L, d))
    dY = rng.standard_normal((B, H, L, d))
    W = orthogonal_gaussian_features(M, d, rng)
    return Q, K, V, W, dY


def _loss(Q, K, V, W, dY, kind):
    return float(np.sum(dY * O.attention_forward(Q, K, V, W, kind)))


def _fd_grad(f, X, h=1e-6):
    g = np.zeros_like(X)
    it = np.nditer(X, flags=["multi_index"])
    for _ in it:
        i = it.multi_index
        x0 = X[i]
        X[i] = x0 + h
        fp = f()
        X[i] = x0 - h
        fm = f()
        X[i] = x0
        g[i] = (fp - fm) / (2 * h)
    return g


def _rel(a, b):
    return float(np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300))


# ---------------------------------------------------------------- P1: finite differences


@pytest.mark.parametrize("kind", [O.FAVOR_PLUS, O.RELU, O.SQUARE])
def test_gradients_match_finite_differences(kind):
    Q, K, V, W, dY = _problem(B=1, H=2, L=6, d=3, M=5, seed=1)
    dQ, dK, dV, dW = O.attention_backward(Q, K, V, W, dY, kind)
    for name, X, g in (("Q", Q, dQ), ("K", K, dK), ("V", V, dV), ("W", W, dW)):
        fd = _fd_grad(lambda: _loss(Q, K, V, W, dY, kind), X)
        assert _rel(g, fd) < 1e-7, name


# ---------------------------------------------------------------- closed forms


@pytest.mark.parametrize("kind", [O.FAVOR_PLUS, O.RELU, O.SQUARE])
def test_first_output_is_first_value(kind):
    """Only l' = 1 contributes to Y_1, whatever the features (eq. 2)."""
    Q, K, V, W, _ = _problem(L=8, seed=2)
    Y = O.attention_forward(Q, K, V, W, kind)
    assert np.max(np.abs(Y[:, :, 0] - V[:, :, 0])) < 1e-14


@pytest.mark.parametrize("kind", [O.FAVOR_PLUS, O.RELU, O.SQUARE])
def test_constant_keys_give_running_mean(kind):
    """Equal keys make every weight in row l equal: Y_l is the mean of V_1..V_l,
    Y does not depend on Q, and dV_j = sum_{l >= j} dY_l / l."""
    Q, K, V, W, dY = _problem(L=10, seed=3)
    K[:] = K[:, :, :1]
    Y = O.attention_forward(Q, K, V, W, kind)
    counts = np.arange(1, 11)[None, None, :, None]
    assert np.max(np.abs(Y - np.cumsum(V, axis=2) / counts)) < 1e-13
    dQ, dK, dV, dW = O.attention_backward(Q, K, V, W, dY, kind)
    assert np.max(np.abs(dQ)) < 1e-12
    ref_dV = np.flip(np.cumsum(np.flip(dY / counts, axis=2), axis=2), axis=2)
    assert np.max(np.abs(dV - ref_dV)) < 1e-13


@pytest.mark.parametrize("kind", [O.FAVOR_PLUS, O.RELU, O.SQUARE])
def test_constant_values_give_constant_output(kind):
    Q, K, V, W, dY = _problem(L=9, seed=4)
    V[:] = V[:, :, :1]
    Y = O.attention_forward(Q, K, V, W, kind)
    assert np.max(np.abs(Y - V)) < 1e-13
    dQ, dK, dV, dW = O.attention_backward(Q, K, V, W, dY, kind)
    for g in (dQ, dK, dW):
        assert np.max(np.abs(g)) < 1e-12


@pytest.mark.parametrize("kind", [O.FAVOR_PLUS, O.RELU, O.SQUARE])
def test_value_gradient_sums_to_output_gradient(kind):
    """Rows of the attention matrix sum to one, so sum_j dV_j = sum_l dY_l."""
    Q, K, V, W, dY = _problem(L=11, seed=5)
    _, _, dV, _ = O.attention_backward(Q, K, V, W, dY, kind)
    assert np.max(np.abs(dV.sum(axis=2) - dY.sum(axis=2))) < 1e-12


def test_euler_identities_of_feature_gradients():
    """Y is homogeneous of degree 0 in each g(Q_l) and jointly in all g(K_l')."""
    rng = np.random.default_rng(6)
    Qf, Kf = rng.random((12, 7)) + 0.1, rng.random((12, 7)) + 0.1
    V, dY = rng.standard_normal((12, 4)), rng.standard_normal((12, 4))
    dQf, dKf, _ = O.quadratic_backward_features(Qf, Kf, V, dY)
    assert np.max(np.abs(np.sum(Qf * dQf, axis=1))) < 1e-12
    assert abs(np.sum(Kf * dKf)) < 1e-12


def test_scale_invariances_and_linearity():
    rng = np.random.default_rng(7)
    Qf, Kf = rng.random((10, 6)) + 0.1, rng.random((10, 6)) + 0.1
    V = rng.standard_normal((10, 3))
    Y = O.quadratic_forward_features(Qf, Kf, V)[0]
    c = rng.random((10, 1)) + 0.5
    assert _rel(O.quadratic_forward_features(c * Qf, Kf, V)[0], Y) < 1e-14
    assert _rel(O.quadratic_forward_features(Qf, 3.7 * Kf, V)[0], Y) < 1e-14
    # a per-row key scale is not a symmetry
    assert _rel(O.quadratic_forward_features(Qf, c * Kf, V)[0], Y) > 1e-3
    V2 = rng.standard_normal((10, 3))
    Y2 = O.quadratic_forward_features(Qf, Kf, V2)[0]
    Y12 = O.quadratic_forward_features(Qf, Kf, 2.0 * V - 0.5 * V2)[0]
    assert _rel(Y12, 2.0 * Y - 0.5 * Y2) < 1e-13


# ---------------------------------------------------------------- feature maps


def test_favor_plus_is_unbiased_for_the_exponential_kernel():
    """E_w[g(q)^T g(k)] = exp(q^T k) for iid w ~ N(0, I) (Gaussian MGF)."""
    rng = np.random.default_rng(8)
    d, M = 4, 1 << 17
    q = rng.standard_normal((6, d)) * 0.5
    k = rng.standard_normal((6, d)) * 0.5
    W = rng.standard_normal((M, d))
    ratio = (O.feature_map(q, W, O.FAVOR_PLUS) @ O.feature_map(k, W, O.FAVOR_PLUS).T) / np.exp(q @ k.T)
    assert abs(np.mean(ratio) - 1.0) < 0.02
    assert np.max(np.abs(ratio - 1.0)) < 0.25


def test_favor_plus_attention_approaches_softmax_attention():
    """With many features the map recovers causal softmax attention (eq. 1)."""
    rng = np.random.default_rng(9)
    d, L, M = 4, 8, 1 << 18
    q = rng.standard_normal((L, d)) * d ** -0.25
    k = rng.standard_normal((L, d)) * d ** -0.25
    v = rng.standard_normal((L, d))
    W = orthogonal_gaussian_features(M, d, rng)
    Y = O.attention_forward(q[None, None], k[None, None], v[None, None], W, O.FAVOR_PLUS)[0, 0]
    logits = np.where(np.tril(np.ones((L, L))) > 0, q @ k.T, -np.inf)
    Ys = scipy.special.softmax(logits, axis=1) @ v
    assert np.max(np.abs(Y - Ys)) < 0.05


def test_relu_map_with_identity_features():
    """W = I reduces the ReLU map to max(x, 0) + eps, coordinate by coordinate."""
    X = np.array([[0.5, -2.0, 0.0], [1.25, 3.0, -0.1]])
    out = O.feature_map(X, np.eye(3), O.RELU)
    assert np.array_equal(out, np.array([[0.501, 0.001, 0.001], [1.251, 3.001, 0.001]]))


def test_relu_map_gradient_mask():
    X = np.array([[0.5, -2.0]])
    W = np.eye(2)
    Phi = O.feature_map(X, W, O.RELU)
    dX, dW = O.feature_map_vjp(X, W, Phi, np.array([[1.0, 1.0]]), O.RELU)
    assert np.array_equal(dX, np.array([[1.0, 0.0]]))
    assert np.array_equal(dW, np.array([[0.5, -2.0], [0.0, 0.0]]))


# ---------------------------------------------------------------- Algorithm 1: C-invariance


@pytest.mark.parametrize("kind", [O.FAVOR_PLUS, O.RELU, O.SQUARE])
@pytest.mark.parametrize("within", ["ps", "quadratic"])
@pytest.mark.parametrize("C", [1, 2, 3, 7, 20])
def test_slicewise_equals_definition_for_every_slice_length(kind, within, C):
    Q, K, V, W, dY = _problem(B=2, H=1, L=20, d=3, M=6, seed=10)
    Y0 = O.attention_forward(Q, K, V, W, kind)
    g0 = O.attention_backward(Q, K, V, W, dY, kind)
    Y, st = O.slim_forward(Q, K, V, W, C, kind, within=within)
    assert _rel(Y, Y0) < 1e-12
    # the final state is the full prefix sum of T_l = (V_l g(K_l)^T, g(K_l))
    Kf = O.feature_map(K, W, kind)
    R = np.einsum("bhld,bhlm->bhdm", V, Kf)
    assert _rel(st, O.pack_state(R, Kf.sum(axis=2))) < 1e-12
    dQ, dK, dV, dW, gst = O.slim_backward(Q, K, V, W, dY, C, kind, st, within=within)
    for g, r in zip((dQ, dK, dV, dW), g0):
        assert _rel(g, r) < 1e-11


def test_slice_bounds_ragged_tail():
    assert O.slice_bounds(10, 4) == [(0, 4), (4, 8), (8, 10)]
    assert O.slice_bounds(10, 10) == [(0, 10)]
    assert O.slice_bounds(10, 64) == [(0, 10)]
    assert O.slice_bounds(4096, 1366)[-1] == (2732, 4096)
    with pytest.raises(ValueError):
        O.slice_bounds(10, 0)


@pytest.mark.parametrize("kind", [O.FAVOR_PLUS, O.RELU, O.SQUARE])
def test_state_gradient_matches_finite_differences(kind):
    """G^(0) = dL/dB^(0), with L = sum dY.Y + <G^(N), B^(N)> (eqs. 17-18)."""
    Q, K, V, W, dY = _problem(B=1, H=1, L=7, d=3, M=4, seed=11)
    rng = np.random.default_rng(12)
    st0 = np.abs(rng.standard_normal((1, 1, 4, 4))) + 0.2
    gN = rng.standard_normal((1, 1, 4, 4))

    def loss():
        Y, st = O.slim_forward(Q, K, V, W, 3, kind, state_in=st0)
        return float(np.sum(dY * Y) + np.sum(gN * st))

    Y, st = O.slim_forward(Q, K, V, W, 3, kind, state_in=st0)
    dQ, dK, dV, dW, g0 = O.slim_backward(Q, K, V, W, dY, 3, kind, st, dstate_out=gN)
    assert _rel(g0, _fd_grad(loss, st0)) < 1e-7
    assert _rel(dQ, _fd_grad(loss, Q)) < 1e-7
    assert _rel(dK, _fd_grad(loss, K)) < 1e-7
    assert _rel(dW, _fd_grad(loss, W)) < 1e-7


@pytest.mark.parametrize("within", ["ps", "quadratic"])
def test_streaming_in_two_calls_equals_one_call(within):
    """B^(n) is an exact checkpoint of the scan: split the sequence, hand the
    state forward and the state cotangent backward."""
    Q, K, V, W, dY = _problem(B=1, H=2, L=13, d=3, M=5, seed=13)
    kind, C, cut = O.FAVOR_PLUS, 4, 6
    Y, st = O.slim_forward(Q, K, V, W, C, kind, within=within)
    g = O.slim_backward(Q, K, V, W, dY, C, kind, st, within=within)
    p1 = [x[:, :, :cut] for x in (Q, K, V, dY)]
    p2 = [x[:, :, cut:] for x in (Q, K, V, dY)]
    Y1, st1 = O.slim_forward(*p1[:3], W, C, kind, within=within)
    Y2, st2 = O.slim_forward(*p2[:3], W, C, kind, state_in=st1, within=within)
    assert _rel(np.concatenate([Y1, Y2], axis=2), Y) < 1e-13
    assert _rel(st2, st) < 1e-13
    dQ2, dK2, dV2, dW2, g1 = O.slim_backward(*p2[:3], W, p2[3], C, kind, st2, within=within)
    dQ1, dK1, dV1, dW1, g0 = O.slim_backward(*p1[:3], W, p1[3], C, kind, st1, dstate_out=g1, within=within)
    assert _rel(np.concatenate([dQ1, dQ2], axis=2), g[0]) < 1e-12
    assert _rel(np.concatenate([dK1, dK2], axis=2), g[1]) < 1e-12
    assert _rel(np.concatenate([dV1, dV2], axis=2), g[2]) < 1e-12
    assert _rel(dW1 + dW2, g[3]) < 1e-12
    assert _rel(g0, g[4]) < 1e-12


# ---------------------------------------------------------------- Appendix B recurrence


def test_token_recurrence_equals_definition():
    rng = np.random.default_rng(14)
    L, M, d = 15, 6, 4
    Qf, Kf = rng.random((L, M)) + 0.05, rng.random((L, M)) + 0.05
    V, dY = rng.standard_normal((L, d)), rng.standard_normal((L, d))
    Y0, A, D0 = O.quadratic_forward_features(Qf, Kf, V)
    Y, N, D, curR, curS = O.iterative_forward_features(Qf, Kf, V)
    assert _rel(Y, Y0) < 1e-13
    dN = dY / D[:, None]
    dD = -np.sum(dY * Y, axis=1) / D
    dQf, dKf, dV = O.iterative_backward_features(Qf, Kf, V, dN, dD, curR, curS)
    r = O.quadratic_backward_features(Qf, Kf, V, dY)
    for g, ref in zip((dQf, dKf, dV), r):
        assert _rel(g, ref) < 1e-12


# ---------------------------------------------------------------- state layout and logits, element by element


def test_state_layout_written_out_by_loops():
    """pack_state / unpack_state against the [B, H, M, d + 1] layout written
    out entry by entry: row m of a head holds sum_l g(K_l)_m V_l[e] in column
    e < d and sum_l g(K_l)_m in column d (the layout the library's state
    tensors use, eqs. 14-16)."""
    rng = np.random.default_rng(21)
    Bn, Hn, L, d, M = 2, 3, 5, 3, 4
    Kf = rng.random((Bn, Hn, L, M)) + 0.1
    V = rng.standard_normal((Bn, Hn, L, d))
    expect = np.zeros((Bn, Hn, M, d + 1))
    for b in range(Bn):
        for h in range(Hn):
            for m in range(M):
                for e in range(d):
                    for l in range(L):
                        expect[b, h, m, e] += Kf[b, h, l, m] * V[b, h, l, e]
                for l in range(L):
                    expect[b, h, m, d] += Kf[b, h, l, m]
    # R [.., d, M] = sum_l V_l g(K_l)^T and S [.., M] = sum_l g(K_l), formed by loops as well
    R = np.zeros((Bn, Hn, d, M))
    S = np.zeros((Bn, Hn, M))
    for b in range(Bn):
        for h in range(Hn):
            for l in range(L):
                for e in range(d):
                    for m in range(M):
                        R[b, h, e, m] += V[b, h, l, e] * Kf[b, h, l, m]
                S[b, h] += Kf[b, h, l]
    packed = O.pack_state(R, S)
    assert packed.shape == (Bn, Hn, M, d + 1)
    assert _rel(packed, expect) < 1e-14
    R2, S2 = O.unpack_state(expect)
    assert _rel(R2, R) < 1e-14 and _rel(S2, S) < 1e-14
    # the forward sweep's final state is that sum
    W = orthogonal_gaussian_features(M, d, rng)
    Q = rng.standard_normal((Bn, Hn, L, d)) * 0.5
    Kx = rng.standard_normal((Bn, Hn, L, d)) * 0.5
    _, st = O.slim_forward(Q, Kx, V, W, 2, O.RELU)
    phi = np.zeros((Bn, Hn, L, M))
    for b in range(Bn):
        for h in range(Hn):
            for l in range(L):
                for m in range(M):
                    phi[b, h, l, m] = max(sum(W[m, e] * Kx[b, h, l, e] for e in range(d)), 0.0) + O.RELU_EPS
    for b in range(Bn):
        for h in range(Hn):
            for m in range(M):
                assert abs(st[b, h, m, d] - phi[b, h, :, m].sum()) < 1e-12
                for e in range(d):
                    ref = sum(phi[b, h, l, m] * V[b, h, l, e] for l in range(L))
                    assert abs(st[b, h, m, e] - ref) < 1e-12


def test_feature_logits_written_out_by_loops():
    """feature_logits(X, W)[.., l, m] = sum_e W[m, e] X[.., l, e], and the
    FAVOR+ map is exp of it minus |x|^2 / 2, over sqrt(M) (Sec. 2.1)."""
    rng = np.random.default_rng(22)
    X = rng.standard_normal((2, 3, 4))
    W = rng.standard_normal((5, 4))
    Z = O.feature_logits(X, W)
    assert Z.shape == (2, 3, 5)
    Phi = O.feature_map(X, W, O.FAVOR_PLUS)
    for i in range(2):
        for l in range(3):
            n2 = sum(X[i, l, e] ** 2 for e in range(4))
            for m in range(5):
                z = sum(W[m, e] * X[i, l, e] for e in range(4))
                assert abs(Z[i, l, m] - z) < 1e-13
                assert abs(Phi[i, l, m] - math.exp(z - n2 / 2) / math.sqrt(5)) < 1e-13 * Phi[i, l, m] + 1e-300
    # a hand-checked value: x = (1, 2), w = (3, -1): w.x = 1, |x|^2/2 = 2.5
    assert O.feature_logits(np.array([[1.0, 2.0]]), np.array([[3.0, -1.0]]))[0, 0] == 1.0
    assert abs(O.feature_map(np.array([[1.0, 2.0]]), np.array([[3.0, -1.0]]), O.FAVOR_PLUS)[0, 0]
               - math.exp(-1.5)) < 1e-15


def test_relu_decision_matrix_only_moves_the_mask():
    """mask_W changes only the 0/1 decisions of the ReLU derivative: the same
    signs give the same gradients, and the opposite matrix gives the
    complementary mask, so the two gradients add up to the all-ones mask's
    (dPhi W, dPhi^T X)."""
    rng = np.random.default_rng(23)
    X = rng.standard_normal((7, 4))
    W = rng.standard_normal((5, 4))
    Phi = O.feature_map(X, W, O.RELU)
    dPhi = rng.standard_normal((7, 5))
    dX, dW = O.feature_map_vjp(X, W, Phi, dPhi, O.RELU)
    dX1, dW1 = O.feature_map_vjp(X, W, Phi, dPhi, O.RELU, mask_W=W * (1 + 1e-9))
    assert np.array_equal(dX, dX1) and np.array_equal(dW, dW1)
    dXn, dWn = O.feature_map_vjp(X, W, Phi, dPhi, O.RELU, mask_W=-W)
    assert _rel(dX + dXn, dPhi @ W) < 1e-14
    assert _rel(dW + dWn, dPhi.T @ X) < 1e-14


def test_square_map_is_the_papers_elementwise_square():
    """With W = I_d (M = d) the square map is g(x) = (x_i^2)_i, the map of
    the paper's experiments (Sec. 4, setup); its VJP is 2 x_i dPhi_i."""
    rng = np.random.default_rng(24)
    X = rng.standard_normal((6, 5))
    I = np.eye(5)
    assert np.array_equal(O.feature_map(X, I, O.SQUARE), X * X)
    dPhi = rng.standard_normal((6, 5))
    dX, dW = O.feature_map_vjp(X, I, X * X, dPhi, O.SQUARE)
    assert _rel(dX, 2.0 * X * dPhi) < 1e-15
    # dW[m, e] = sum_l 2 x_lm dPhi_lm x_le
    ref = np.zeros((5, 5))
    for l in range(6):
        for m in range(5):
            for e in range(5):
                ref[m, e] += 2.0 * X[l, m] * dPhi[l, m] * X[l, e]
    assert _rel(dW, ref) < 1e-14
