"""GPU parity of the explicit prefix-sum within-slice mode ("PS": the state
after every row of a slice written out, then used) against the fp64
oracle's definition (eq. 2) and against the tile-walk mode, on seeded
synthetic inputs.  Bars as everywhere: max-relative error <= 1e-5 (float32)
and <= 2e-2 (bf16 inputs and outputs).

The mode forms the logits in float32 from the float32 W, so the ReLU
derivative's 0/1 decisions are taken with W itself on both sides."""

import numpy as np
import pytest
import torch

import oracle as O
from synth import Workload, make_inputs
from tests.gpu_common import TOL, dev, host64, need_gpu, report

pytestmark = pytest.mark.gpu

# name, B, H, L, d, M, C, dtype, kind
CASES = [
    ("f32_headline_shape", 1, 2, 150, 64, 256, 64, "f32", "favor+"),
    ("f32_ragged_c7", 2, 1, 61, 32, 64, 7, "f32", "favor+"),
    ("f32_c1", 1, 1, 20, 32, 128, 1, "f32", "favor+"),
    ("f32_relu_c_above_L", 1, 2, 90, 64, 128, 200, "f32", "relu"),
    ("f32_square_identity", 1, 2, 130, 64, 64, 32, "f32", "square"),
    ("bf16_c64", 2, 2, 300, 64, 256, 64, "bf16", "favor+"),
    ("bf16_relu_d32", 1, 3, 170, 32, 128, 48, "bf16", "relu"),
    ("bf16_square_identity", 1, 2, 260, 64, 64, 100, "bf16", "square"),
]


def _inputs(i, B, H, L, d, M, C, dtype, kind):
    x = make_inputs(Workload(f"ps{i}", 900 + i, B, H, L, d, M, (C,), dtype, kind))
    if kind == "square":
        x["W"] = torch.eye(64, dtype=torch.float32)  # the paper's map g(x) = (x_i^2)
    return x


@pytest.mark.parametrize("i", range(len(CASES)))
def test_ps_forward_and_backward(i):
    need_gpu()
    from paper_2012_11346_amd import slim

    name, B, H, L, d, M, C, dtype, kind = CASES[i]
    print(f"[ps] case={name} B={B} H={H} L={L} d={d} M={M} C={C} {dtype} {kind}", flush=True)
    x = _inputs(i, B, H, L, d, M, C, dtype, kind)
    Q, K, V, W, dY = (dev(x[k]) for k in ("Q", "K", "V", "W", "dY"))
    Y, st, ks = slim.fwd(Q, K, V, W, C, kind, within="ps")
    g = slim.bwd(Q, K, V, W, dY, C, ks, kind, within="ps")
    torch.cuda.synchronize()
    tol = TOL[dtype]
    report("Y", host64(Y), O.attention_forward(x["Q"], x["K"], x["V"], x["W"], kind), tol)
    _, stref = O.slim_forward(x["Q"], x["K"], x["V"], x["W"], C, kind, within="quadratic")
    s = host64(st)
    if kind == "favor+":
        s = s * np.exp(host64(ks))[:, :, None, None]
    report("state_out", s, stref, tol)
    ref = O.attention_backward(x["Q"], x["K"], x["V"], x["W"], x["dY"], kind)
    for n, a, r in zip(("dQ", "dK", "dV", "dW"), g[:4], ref):
        report(n, host64(a), r, tol)


def test_ps_agrees_with_the_tile_walk():
    """Both modes evaluate the same sums: at bf16 the outputs agree within
    the bar."""
    need_gpu()
    from paper_2012_11346_amd import slim

    B, H, L, d, M, C, kind = 1, 2, 400, 64, 256, 64, "favor+"
    x = _inputs(30, B, H, L, d, M, C, "bf16", kind)
    Q, K, V, W, dY = (dev(x[k]) for k in ("Q", "K", "V", "W", "dY"))
    Yp, _, ksp = slim.fwd(Q, K, V, W, C, kind, within="ps")
    gp = slim.bwd(Q, K, V, W, dY, C, ksp, kind, within="ps")
    Yi, _, ksi = slim.fwd(Q, K, V, W, C, kind)
    gi = slim.bwd(Q, K, V, W, dY, C, ksi, kind)
    torch.cuda.synchronize()
    tol = TOL["bf16"]
    report("Y ps vs walk", host64(Yp), host64(Yi), tol)
    for n, a, b in zip(("dQ", "dK", "dV", "dW"), gp[:4], gi[:4]):
        report(n + " ps vs walk", host64(a), host64(b), tol)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_ps_state_cotangent_and_chaining(dtype):
    """Two calls on the halves: the second's forward resumes from the first's
    state_out / kshift_out, its backward hands G^(0) to the first's; the
    result equals the whole sequence's gradient."""
    need_gpu()
    from paper_2012_11346_amd import slim

    B, H, L, d, M, C, kind = 1, 2, 260, 64, 128, 32, "favor+"
    x = _inputs(31 if dtype == "f32" else 32, B, H, L, d, M, C, dtype, kind)
    cut = 130 + 7
    tol = TOL[dtype]
    Q, K, V, W, dY = (dev(x[k]) for k in ("Q", "K", "V", "W", "dY"))
    half = lambda t, a, b: t[:, :, a:b].contiguous()
    Y1, st1, ks1 = slim.fwd(half(Q, 0, cut), half(K, 0, cut), half(V, 0, cut), W, C, kind, within="ps")
    Y2, st2, ks2 = slim.fwd(half(Q, cut, L), half(K, cut, L), half(V, cut, L), W, C, kind, state_in=st1,
                            kshift_in=ks1, within="ps")
    g2 = slim.bwd(half(Q, cut, L), half(K, cut, L), half(V, cut, L), W, half(dY, cut, L), C, ks2, kind,
                  state_in=st1, kshift_in=ks1, want_dstate_in=True, within="ps")
    g1 = slim.bwd(half(Q, 0, cut), half(K, 0, cut), half(V, 0, cut), W, half(dY, 0, cut), C, ks1, kind,
                  dstate_out=g2[4], within="ps")
    torch.cuda.synchronize()
    report("Y (two calls)", np.concatenate([host64(Y1), host64(Y2)], axis=2),
           O.attention_forward(x["Q"], x["K"], x["V"], x["W"], kind), tol)
    ref = O.attention_backward(x["Q"], x["K"], x["V"], x["W"], x["dY"], kind)
    report("dQ (chained)", np.concatenate([host64(g1[0]), host64(g2[0])], axis=2), ref[0], tol)
    report("dK (chained)", np.concatenate([host64(g1[1]), host64(g2[1])], axis=2), ref[1], tol)
    report("dV (chained)", np.concatenate([host64(g1[2]), host64(g2[2])], axis=2), ref[2], tol)
    report("dW (chained)", host64(g1[3]) + host64(g2[3]), ref[3], tol)


def test_ps_rejects_dropout():
    need_gpu()
    from paper_2012_11346_amd import slim

    x = _inputs(33, 1, 1, 64, 32, 64, 32, "bf16", "favor+")
    with pytest.raises(RuntimeError, match="dropout"):
        slim.fwd(dev(x["Q"]), dev(x["K"]), dev(x["V"]), dev(x["W"]), 32, dropout=0.1, seed=1, within="ps")
