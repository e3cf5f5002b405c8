"""GPU parity of the quadratic within-slice mode (each slice evaluated as the
masked quadratic form of eq. 2 from the state before it, slices one after
another) against the fp64 oracle, and against the tile-walk mode on the
same inputs.  Bars as everywhere: max-relative error <= 2e-2 (bf16)."""

import os

import numpy as np
import pytest
import torch

import oracle as O
from synth import Workload, make_inputs
from tests.gpu_common import TOL, dev, host64, mask_w, need_gpu, report

pytestmark = pytest.mark.gpu

# name, B, H, L, d, M, C, kind, forced workgroups per head (None: planned)
CASES = [
    ("ragged_c64", 2, 3, 300, 64, 256, 64, "favor+", None),
    ("c100", 1, 2, 250, 64, 256, 100, "favor+", None),
    ("relu_c_above_L", 2, 2, 200, 64, 128, 256, "relu", None),
    ("d32_m256_c40", 1, 2, 333, 32, 256, 40, "favor+", None),
    ("d32_m128_relu_c16", 2, 1, 170, 32, 128, 16, "relu", None),
    ("c1", 1, 1, 40, 64, 128, 1, "favor+", None),
    ("c512_strided", 1, 2, 1100, 64, 256, 512, "favor+", 3),
    ("relu_c300_strided", 1, 1, 1000, 32, 256, 300, "relu", 2),
]


class _env:
    """Set debugging variables of the library for one block."""

    def __init__(self, **kv):
        self.kv = {k: v for k, v in kv.items() if v is not None}

    def __enter__(self):
        self.old = {k: os.environ.get(k) for k in self.kv}
        for k, v in self.kv.items():
            os.environ[k] = str(v)

    def __exit__(self, *exc):
        for k, v in self.old.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v


def _inputs(i, B, H, L, d, M, C, kind):
    return make_inputs(Workload(f"quad{i}", 700 + i, B, H, L, d, M, (C,), "bf16", kind))


@pytest.mark.parametrize("i", range(len(CASES)))
def test_quadratic_forward(i):
    need_gpu()
    from paper_2012_11346_amd import slim

    name, B, H, L, d, M, C, kind, nwg = CASES[i]
    print(f"[quadratic fwd] case={name} B={B} H={H} L={L} d={d} M={M} C={C} {kind} workgroups={nwg}", flush=True)
    x = _inputs(i, B, H, L, d, M, C, kind)
    Q, K, V, W = (dev(x[k]) for k in ("Q", "K", "V", "W"))
    with _env(SLIM_QUAD_WORKGROUPS=nwg):
        Y, st, ks = slim.fwd(Q, K, V, W, C, kind, within="quadratic")
    Yi, sti, ksi = slim.fwd(Q, K, V, W, C, kind)
    torch.cuda.synchronize()
    tol = TOL["bf16"]
    Yref = O.attention_forward(x["Q"], x["K"], x["V"], x["W"], kind)
    report("Y", host64(Y), Yref, tol)
    report("Y vs tile walk", host64(Y), host64(Yi), tol)
    _, stref = O.slim_forward(x["Q"], x["K"], x["V"], x["W"], C, kind, within="quadratic")
    s = host64(st)
    if kind == "favor+":
        s = s * np.exp(host64(ks))[:, :, None, None]
        assert torch.equal(ks.cpu(), ksi.cpu()), "both modes take the same key shift"
    report("state_out", s, stref, tol)


def test_quadratic_forward_resumes():
    """state_out and kshift_out of a first call resume the scan: two calls
    on the halves equal one call on the whole sequence."""
    need_gpu()
    from paper_2012_11346_amd import slim

    B, H, L, d, M, C = 1, 2, 290, 64, 256, 64
    x = _inputs(20, B, H, L, d, M, C, "favor+")
    Q, K, V, W = (dev(x[k]) for k in ("Q", "K", "V", "W"))
    cut = 128 + 5
    part = lambda t, a, b: t[:, :, a:b].contiguous()
    Y1, st1, ks1 = slim.fwd(part(Q, 0, cut), part(K, 0, cut), part(V, 0, cut), W, C, within="quadratic")
    Y2, st2, ks2 = slim.fwd(part(Q, cut, L), part(K, cut, L), part(V, cut, L), W, C, state_in=st1, kshift_in=ks1,
                            within="quadratic")
    torch.cuda.synchronize()
    Yref = O.attention_forward(x["Q"], x["K"], x["V"], x["W"], "favor+")
    report("Y (two calls)", np.concatenate([host64(Y1), host64(Y2)], axis=2), Yref, TOL["bf16"])


def test_quadratic_forward_dropout():
    """Value dropout draws the same masks in both modes (slice n's key is
    (seed, n))."""
    need_gpu()
    from paper_2012_11346_amd import slim

    B, H, L, d, M, C, p, seed = 1, 2, 300, 64, 256, 64, 0.2, 41
    x = _inputs(21, B, H, L, d, M, C, "favor+")
    Q, K, V, W = (dev(x[k]) for k in ("Q", "K", "V", "W"))
    Y, st, ks = slim.fwd(Q, K, V, W, C, dropout=p, seed=seed, within="quadratic")
    torch.cuda.synchronize()
    Yr = O.dropout_forward(O.attention_forward, x["Q"], x["K"], x["V"], x["W"], "favor+", C, p, seed)
    report("Y (dropout)", host64(Y), Yr, TOL["bf16"])


def test_quadratic_rejects_unbuilt_problems():
    need_gpu()
    from paper_2012_11346_amd import slim

    x = _inputs(22, 1, 1, 64, 32, 64, 32, "favor+")
    with pytest.raises(RuntimeError, match="quadratic"):
        slim.fwd(dev(x["Q"]), dev(x["K"]), dev(x["V"]), dev(x["W"]), 32, within="quadratic")


# name, B, H, L, d, M, C, kind, forced workgroups per head, forced runs of the downdates
BWD_CASES = [
    ("ragged_c64", 2, 3, 300, 64, 256, 64, "favor+", None, None),
    ("c100_one_run", 1, 2, 250, 64, 256, 100, "favor+", None, 1),
    ("relu_c_above_L", 2, 2, 200, 64, 128, 256, "relu", None, None),
    ("d32_m256_c40", 1, 2, 333, 32, 256, 40, "favor+", None, None),
    ("d32_m128_relu_c16_runs3", 2, 1, 170, 32, 128, 16, "relu", None, 3),
    ("c1", 1, 1, 40, 64, 128, 1, "favor+", None, None),
    ("c512_strided", 1, 2, 1100, 64, 256, 512, "favor+", 3, None),
    ("relu_c300_strided", 1, 1, 1000, 32, 256, 300, "relu", 2, 2),
    ("many_slices_c32", 1, 2, 2048, 64, 256, 32, "favor+", None, None),
]


@pytest.mark.parametrize("i", range(len(BWD_CASES)))
def test_quadratic_backward(i):
    need_gpu()
    from paper_2012_11346_amd import slim

    name, B, H, L, d, M, C, kind, nwg, runs = BWD_CASES[i]
    print(f"[quadratic bwd] case={name} B={B} H={H} L={L} d={d} M={M} C={C} {kind} workgroups={nwg} runs={runs}",
          flush=True)
    x = _inputs(40 + i, B, H, L, d, M, C, kind)
    Q, K, V, W, dY = (dev(x[k]) for k in ("Q", "K", "V", "W", "dY"))
    with _env(SLIM_QUAD_WORKGROUPS=nwg, SLIM_QUAD_RUNS=runs):
        Y, st, ks = slim.fwd(Q, K, V, W, C, kind, within="quadratic")
        g = slim.bwd(Q, K, V, W, dY, C, ks, kind, within="quadratic")
    gi = slim.bwd(Q, K, V, W, dY, C, ks, kind)
    torch.cuda.synchronize()
    tol = TOL["bf16"]
    ref = O.attention_backward(x["Q"], x["K"], x["V"], x["W"], x["dY"], kind, mask_W=mask_w(x))
    for n, a, r, b in zip(("dQ", "dK", "dV", "dW"), g[:4], ref, gi[:4]):
        report(n, host64(a), r, tol)
        report(n + " vs tile walk", host64(a), host64(b), tol)


def test_quadratic_state_cotangent_and_chaining():
    """The backward of the second half, its G^(0) fed to the backward of the
    first half, equals the backward of the whole sequence (both halves in the
    quadratic mode); G^(0) matches Algorithm 1."""
    need_gpu()
    from paper_2012_11346_amd import slim

    B, H, L, d, M, C, kind = 1, 2, 400, 64, 256, 64, "favor+"
    x = _inputs(60, B, H, L, d, M, C, kind)
    cut = 200 + 3
    tol = TOL["bf16"]
    Q, K, V, W, dY = (dev(x[k]) for k in ("Q", "K", "V", "W", "dY"))
    half = lambda t, a, b: t[:, :, a:b].contiguous()
    q = "quadratic"
    Y1, st1, ks1 = slim.fwd(half(Q, 0, cut), half(K, 0, cut), half(V, 0, cut), W, C, kind, within=q)
    Y2, st2, ks2 = slim.fwd(half(Q, cut, L), half(K, cut, L), half(V, cut, L), W, C, kind, state_in=st1,
                            kshift_in=ks1, within=q)
    g2 = slim.bwd(half(Q, cut, L), half(K, cut, L), half(V, cut, L), W, half(dY, cut, L), C, ks2, kind,
                  state_in=st1, kshift_in=ks1, want_dstate_in=True, within=q)
    g1 = slim.bwd(half(Q, 0, cut), half(K, 0, cut), half(V, 0, cut), W, half(dY, 0, cut), C, ks1, kind,
                  dstate_out=g2[4], within=q)
    torch.cuda.synchronize()
    ref = O.attention_backward(x["Q"], x["K"], x["V"], x["W"], x["dY"], kind, mask_W=mask_w(x))
    report("dQ (chained)", np.concatenate([host64(g1[0]), host64(g2[0])], axis=2), ref[0], tol)
    report("dK (chained)", np.concatenate([host64(g1[1]), host64(g2[1])], axis=2), ref[1], tol)
    report("dV (chained)", np.concatenate([host64(g1[2]), host64(g2[2])], axis=2), ref[2], tol)
    report("dW (chained)", host64(g1[3]) + host64(g2[3]), ref[3], tol)
    st_full = O.slim_forward(x["Q"], x["K"], x["V"], x["W"], C, kind)[1]
    go = O.slim_backward(x["Q"][:, :, cut:], x["K"][:, :, cut:], x["V"][:, :, cut:], x["W"], x["dY"][:, :, cut:], C,
                         kind, st_full, mask_W=mask_w(x))[4]
    g0 = host64(g2[4]) * np.exp(-host64(ks1))[:, :, None, None]
    report("dstate_in", g0, go, tol)


@pytest.mark.parametrize("kind", ["favor+", "relu"])
def test_quadratic_backward_dropout(kind):
    """Value dropout in the backward: the masks regenerated per slice, dropped
    value elements with exactly zero gradient."""
    need_gpu()
    from paper_2012_11346_amd import slim

    B, H, L, d, M, C, p, seed = 1, 2, 300, 64, 128, 64, 0.3, 2 ** 62 + 11
    x = _inputs(61 if kind == "favor+" else 62, B, H, L, d, M, C, kind)
    Q, K, V, W, dY = (dev(x[k]) for k in ("Q", "K", "V", "W", "dY"))
    Y, st, ks = slim.fwd(Q, K, V, W, C, kind, dropout=p, seed=seed, within="quadratic")
    g = slim.bwd(Q, K, V, W, dY, C, ks, kind, dropout=p, seed=seed, within="quadratic")
    torch.cuda.synchronize()
    ref = O.dropout_backward(O.attention_backward, x["Q"], x["K"], x["V"], x["W"], x["dY"], kind, C, p, seed,
                             mask_W=mask_w(x))
    for n, a, r in zip(("dQ", "dK", "dV", "dW"), g[:4], ref):
        report(n, host64(a), r, TOL["bf16"])
    m = O.value_mask(B, H, L, d, C, p, seed)
    assert torch.count_nonzero(g[2].cpu()[torch.from_numpy(m == 0)]).item() == 0
