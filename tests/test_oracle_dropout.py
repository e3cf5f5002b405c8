"""Pins of the oracle's value dropout (Sec. 5: per-slice seeds reused in the
forward and backward passes) against facts outside it: numpy's Philox
generator, the binomial keep rate, the unbiased scaling, the layout rules of
the definition in oracle/dropout.py, and finite differences."""

import numpy as np
import pytest

import oracle as O
from tests.test_oracle_pins import _fd_grad, _problem, _rel


@pytest.mark.parametrize("key, ctr", [((0x1234567890ABCDEF, 0x0FEDCBA987654321), (6, 0, 0, 0)),
                                      ((0, 0), (1, 2, 3, 4)),
                                      ((2 ** 64 - 1, 17), (2 ** 63 + 5, 2 ** 64 - 1, 7, 2 ** 40))])
def test_philox_matches_numpy(key, ctr):
    """numpy.random.Philox is Philox4x64-10 and increments its 256-bit
    counter before each block: started at ctr - 1 it returns the block of ctr."""
    g = np.random.Philox(key=np.array(key, dtype=np.uint64),
                         counter=np.array([ctr[0] - 1] + list(ctr[1:]), dtype=np.uint64))
    ref = [int(v) for v in g.random_raw(4)]
    out = O.philox4x64_10(tuple(np.uint64(c) for c in ctr), tuple(np.uint64(k) for k in key))
    assert [int(v) for v in out] == ref


def test_keep_rate_and_unbiased_scale():
    p = 0.2
    m = O.value_mask(2, 3, 700, 64, 64, p, seed=7)
    n = m.size
    assert abs(m.mean() - (1 - p)) < 5 * np.sqrt(p * (1 - p) / n)
    assert O.keep_threshold(0.0) == 0 and np.all(O.value_mask(1, 1, 50, 32, 8, 0.0, 3) == 1.0)
    # E[s m] = 1: the output scale undoes the expected loss of mass
    s = O.output_scale(p)
    assert abs(s * (1 - p) - 1) < 1e-7


def test_masks_follow_slices_and_heads():
    """Slice n has its own seed: the same row position in two slices draws
    different masks; rows of slice 0 do not depend on C beyond it; the head
    enters only as b H + h."""
    m8 = O.value_mask(1, 1, 64, 64, 8, 0.5, seed=11)
    same = np.mean(m8[0, 0, 0:8] == m8[0, 0, 8:16])
    assert 0.35 < same < 0.65
    a = O.value_mask(1, 2, 32, 64, 16, 0.3, seed=5)
    b = O.value_mask(1, 2, 32, 64, 32, 0.3, seed=5)
    assert np.array_equal(a[..., :16, :], b[..., :16, :])
    assert not np.array_equal(a[..., 16:, :], b[..., 16:, :])
    x = O.value_mask(2, 3, 20, 32, 8, 0.3, seed=9)
    y = O.value_mask(1, 6, 20, 32, 8, 0.3, seed=9)
    assert np.array_equal(x[1, 0], y[0, 3])
    assert not np.array_equal(O.value_mask(1, 1, 20, 32, 8, 0.3, seed=9), O.value_mask(1, 1, 20, 32, 8, 0.3, seed=10))


@pytest.mark.parametrize("kind", [O.FAVOR_PLUS, O.RELU, O.SQUARE])
def test_dropout_gradients_match_finite_differences(kind):
    Q, K, V, W, dY = _problem(B=1, H=2, L=7, d=3, M=4, seed=31)
    C, p, seed = 3, 0.3, 99

    def loss():
        return float(np.sum(dY * O.dropout_forward(O.attention_forward, Q, K, V, W, kind, C, p, seed)))

    g = O.dropout_backward(O.attention_backward, Q, K, V, W, dY, kind, C, p, seed)
    for X, gx in zip((Q, K, V, W), g):
        assert _rel(gx, _fd_grad(loss, X)) < 1e-7


def test_dropout_without_drops_is_the_attention():
    Q, K, V, W, dY = _problem(B=1, H=2, L=9, d=3, M=5, seed=32)
    Y = O.dropout_forward(O.attention_forward, Q, K, V, W, O.FAVOR_PLUS, 4, 0.0, 1)
    assert _rel(Y, O.attention_forward(Q, K, V, W, O.FAVOR_PLUS)) < 1e-15


def test_planted_mistakes_are_caught(monkeypatch):
    """A generator with its multipliers swapped, and masks without the slice
    in the key, each fail a pin above."""
    import oracle.dropout as D

    real = D.philox4x64_10

    def swapped(ctr, key):
        m0, m1 = D._M0, D._M1
        monkeypatch.setattr(D, "_M0", m1)
        monkeypatch.setattr(D, "_M1", m0)
        try:
            return real(ctr, key)
        finally:
            monkeypatch.setattr(D, "_M0", m0)
            monkeypatch.setattr(D, "_M1", m1)

    monkeypatch.setattr(O, "philox4x64_10", swapped)
    with pytest.raises(AssertionError):
        test_philox_matches_numpy((0, 0), (1, 2, 3, 4))
    monkeypatch.setattr(O, "philox4x64_10", real)

    def no_slice_key(ctr, key):
        return real(ctr, (key[0], np.zeros_like(np.asarray(key[1]))))

    monkeypatch.setattr(D, "philox4x64_10", no_slice_key)
    with pytest.raises(AssertionError):
        test_masks_follow_slices_and_heads()
