"""Pins of the fp64 oracle of the s-layer Performer (Sec. 2.2, eqs. 5-10) and of
its Algorithm 1 evaluation (Sec. 3.2-3.3), on the CPU.

* the hand-written gradient against central finite differences of the loss,
  for every parameter tensor (random directions);
* Algorithm 1 (slices outer, layers inner, eq. 17 downdates, eq. 18
  cotangents) against the whole-sequence evaluation for several C, as the
  paper states the result does not depend on C (Sec. 3.3);
* closed forms: zero output weights give loss ln |Sigma| (eq. 10's mean over
  L - 1 rows), cross-entropy gradients sum to zero per row and vanish on the
  last row, layer normalisation's moments, GeLU's odd part, the sinusoids;
* planted mistakes, each caught by one of the pins above.
"""

import math

import numpy as np
import pytest

import oracle.performer as OP
from synth import ModelConfig, make_model, make_tokens

TINY = ModelConfig("tiny", L=7, D=8, s=2, vocab=11, B=2, heads=2)


def _tiny(seed=0):
    return make_model(TINY, seed=seed, perturb_ln=True), make_tokens(TINY, seed=seed)


def _fd_check(P, tok, heads, names=None, eps=1e-6, tol=1e-6):
    loss, g = OP.model_full(P, tok, heads=heads)
    Pd = {k: v.double().numpy() for k, v in P.items()}
    rng = np.random.default_rng(5)
    for name in names or list(Pd):
        d = rng.standard_normal(Pd[name].shape)
        pp, pm = dict(Pd), dict(Pd)
        pp[name] = Pd[name] + eps * d
        pm[name] = Pd[name] - eps * d
        fd = (OP.model_loss(pp, tok, heads=heads) - OP.model_loss(pm, tok, heads=heads)) / (2 * eps)
        an = float(np.sum(g[name] * d))
        assert abs(fd - an) <= tol * max(1.0, abs(an)), f"{name}: fd {fd} analytic {an}"


def test_gradients_match_finite_differences():
    P, tok = _tiny()
    _fd_check(P, tok, heads=2)


@pytest.mark.parametrize("C", [1, 2, 3, 7, 100])
def test_algorithm1_equals_the_whole_sequence(C):
    P, tok = _tiny(seed=1)
    loss, g = OP.model_full(P, tok, heads=2)
    l1, g1 = OP.model_algorithm1(P, tok, C, heads=2)
    assert abs(l1 - loss) <= 1e-12 * abs(loss)
    assert OP.grad_discrepancy(g1, g) <= 1e-12


def test_zero_output_weights_give_log_alphabet():
    P, tok = _tiny(seed=2)
    P["Wout"] = P["Wout"] * 0
    P["bout"] = P["bout"] * 0
    loss, g = OP.model_full(P, tok, heads=2)
    assert abs(loss - math.log(TINY.vocab)) < 1e-12
    # bout's gradient: mean over the L - 1 predicted rows of (1/V - onehot)
    tgt = np.asarray(tok)[:, 1:].reshape(-1)
    expect = np.full(TINY.vocab, 1.0 / TINY.vocab) - np.bincount(tgt, minlength=TINY.vocab) / tgt.size
    np.testing.assert_allclose(g["bout"], expect, atol=1e-14)


def test_cross_entropy_rows():
    rng = np.random.default_rng(3)
    logits = rng.standard_normal((2, 5, 7))
    tok = rng.integers(0, 7, size=(2, 9))
    loss, d = OP.next_token_loss(logits, tok, 4, 9)  # rows 4..8 of L = 9: row 8 predicts nothing
    np.testing.assert_allclose(d.sum(axis=-1), 0.0, atol=1e-15)
    assert np.all(d[:, -1] == 0.0)
    z = logits[:, :4] - np.log(np.exp(logits[:, :4]).sum(-1, keepdims=True))
    ref = -sum(z[b, j, tok[b, 5 + j]] for b in range(2) for j in range(4)) / (8 * 2)
    assert abs(loss - ref) < 1e-14


def test_layer_norm_moments_and_gelu_identities():
    rng = np.random.default_rng(4)
    x = 3.0 + 2.0 * rng.standard_normal((6, 10))
    y, _ = OP.layer_norm(x, np.ones(10), np.zeros(10))
    np.testing.assert_allclose(y.mean(-1), 0.0, atol=1e-14)
    var = x.var(-1)
    np.testing.assert_allclose((y * y).mean(-1), var / (var + OP.LN_EPS), rtol=1e-12)
    t = rng.standard_normal(50) * 3
    np.testing.assert_allclose(OP.gelu(t) - OP.gelu(-t), t, atol=1e-14)
    assert OP.gelu(np.array([0.0]))[0] == 0.0
    np.testing.assert_allclose(OP.gelu_grad(np.array([0.0])), 0.5, atol=1e-15)


def test_sinusoids():
    pe = OP.positions(0, 5, 6)
    np.testing.assert_allclose(pe[0], [0, 1, 0, 1, 0, 1], atol=1e-15)
    np.testing.assert_allclose(pe[:, 0], np.sin(np.arange(5)), atol=1e-15)
    np.testing.assert_allclose(pe[:, 3], np.cos(np.arange(5) / 10000 ** (2 / 6)), atol=1e-15)
    np.testing.assert_allclose(OP.positions(3, 2, 6), pe[3:5], atol=1e-15)


# ---------------------------------------------------------------- planted mistakes


def _ln_vjp_no_mean(dy, g, cache):
    xhat, rstd = cache
    D = xhat.shape[-1]
    dxh = dy * g
    dx = rstd / D * (D * dxh - xhat * (dxh * xhat).sum(axis=-1, keepdims=True))
    return dx, (dy * xhat).reshape(-1, D).sum(0), dy.reshape(-1, D).sum(0)


def _gelu_grad_tanh(x):
    return 0.5 * (1.0 + np.tanh(0.7978845608 * (x + 0.044715 * x ** 3)))


def _loss_over_L(logits, tokens, l0, L):
    loss, d = REAL_LOSS(logits, tokens, l0, L)
    return loss * (L - 1) / L, d * (L - 1) / L


REAL_LOSS = OP.next_token_loss


def _positions_from_one(l0, n, D):
    return REAL_POS(l0 + 1, n, D)


REAL_POS = OP.positions


@pytest.mark.parametrize(
    "attr, fake, pin",
    [
        ("layer_norm_vjp", _ln_vjp_no_mean, lambda: test_gradients_match_finite_differences()),
        ("gelu_grad", _gelu_grad_tanh, lambda: test_gradients_match_finite_differences()),
        ("next_token_loss", _loss_over_L, lambda: test_zero_output_weights_give_log_alphabet()),
        ("positions", _positions_from_one, lambda: test_sinusoids()),
    ],
)
def test_planted_mistakes_are_caught(attr, fake, pin, monkeypatch):
    monkeypatch.setattr(OP, attr, fake)
    with pytest.raises(AssertionError):
        pin()


def test_algorithm1_without_downdate_is_caught(monkeypatch):
    """Algorithm 1 recomputing each slice from the state after it (no eq. 17)
    fails the comparison with the whole sequence."""
    real = OP.slim_forward

    def no_downdate(Q, K, V, W, C, kind, state_in=None, within="ps", relu_eps=1e-3):
        if state_in is None:
            Y, st = real(Q, K, V, W, C, kind, None, within, relu_eps)
            return Y, st * 0  # the slice's own sum is never subtracted
        return real(Q, K, V, W, C, kind, state_in, within, relu_eps)

    monkeypatch.setattr(OP, "slim_forward", no_downdate)
    with pytest.raises(AssertionError):
        test_algorithm1_equals_the_whole_sequence(3)
