"""GPU parity of the square feature map g(x)_m = (w_m . x)^2: with W = I and
M = d it is the element-wise square of the paper's experiments (Sec. 4,
setup), run here at the paper's per-layer shapes (B = 1, d = 64, heads =
d_model / 64, L from 512 to 16384); with a random W it is the same map after
a projection.  Bars as everywhere: max-relative error <= 1e-5 (fp32),
<= 2e-2 (bf16)."""

import numpy as np
import pytest
import torch

import oracle as O
from synth import Workload, make_inputs
from tests.gpu_common import TOL, dev, host64, need_gpu, report

pytestmark = pytest.mark.gpu

# name, B, H, L, d, C, dtype, identity W
CASES = [
    ("f32_d32_random_w", 1, 2, 200, 32, 16, "f32", False),
    ("f32_d64_identity", 1, 1, 130, 64, 7, "f32", True),
    ("bf16_identity_c64", 1, 4, 512, 64, 64, "bf16", True),
    ("bf16_random_w_ragged", 2, 3, 300, 64, 100, "bf16", False),
    ("bf16_d32_identity_cL", 2, 2, 200, 32, 256, "bf16", True),
    ("bf16_identity_segments", 1, 2, 4096, 64, 64, "bf16", True),
]


def _inputs(i, B, H, L, d, dtype, identity):
    x = make_inputs(Workload(f"square{i}", 500 + i, B, H, L, d, 64, (64,), dtype, "square"))
    if identity:
        x["W"] = torch.eye(64, d, dtype=torch.float32)
    return x


@pytest.mark.parametrize("i", range(len(CASES)))
def test_square_map_forward_backward(i):
    need_gpu()
    from paper_2012_11346_amd import slim

    name, B, H, L, d, C, dtype, identity = CASES[i]
    print(f"[square] case={name} B={B} H={H} L={L} d={d} M=64 C={C} {dtype}", flush=True)
    x = _inputs(i, B, H, L, d, dtype, identity)
    Q, K, V, W, dY = (dev(x[k]) for k in ("Q", "K", "V", "W", "dY"))
    lD = torch.empty((B, H, L), dtype=torch.float32, device=Q.device)
    Y, st, ks = slim.fwd(Q, K, V, W, C, "square", logD=lD)
    dQ, dK, dV, dW, _ = slim.bwd(Q, K, V, W, dY, C, ks, "square", Y=Y, logD=lD)
    torch.cuda.synchronize()
    assert ks is None
    tol = TOL[dtype]
    report("Y", host64(Y), O.attention_forward(x["Q"], x["K"], x["V"], x["W"], O.SQUARE), tol)
    # logD = log2 of D_t = g(q_t) . sum_{j <= t} g(k_j) (eq. 2; no shifts for this map)
    Pq, Pk = (O.feature_map(x[n], x["W"], O.SQUARE) for n in ("Q", "K"))
    Dt = np.einsum("bhlm,bhlm->bhl", Pq, np.cumsum(Pk, axis=2))
    err = float(np.max(np.abs(np.exp2(host64(lD) - np.log2(Dt)) - 1.0)))
    print(f"  logD: max |D / D_ref - 1| = {err:.3e} (tol {tol})", flush=True)
    assert err <= tol
    _, stref = O.slim_forward(x["Q"], x["K"], x["V"], x["W"], C, O.SQUARE, within="quadratic")
    report("state_out", host64(st), stref, tol)
    ref = O.attention_backward(x["Q"], x["K"], x["V"], x["W"], x["dY"], O.SQUARE)
    for n, a, r in zip(("dQ", "dK", "dV", "dW"), (dQ, dK, dV, dW), ref):
        report(n, host64(a), r, tol)


# the per-layer attention shapes of the paper's configurations I-IV
# (L, d_model) = (512, 256), (1024, 512), (4096, 1024), (16384, 1024): heads = d_model / 64
PAPER_SHAPES = [(512, 4), (1024, 8), (4096, 16), (16384, 16)]


@pytest.mark.parametrize("L, H", PAPER_SHAPES)
def test_square_map_at_the_papers_shapes(L, H):
    """B = 1, d = M = 64, W = I, bf16, C = 64; the oracle on one sampled head."""
    need_gpu()
    from paper_2012_11346_amd import slim

    print(f"[square paper shape] L={L} H={H}", flush=True)
    x = make_inputs(Workload(f"sq_paper_{L}", 520 + H, 1, H, L, 64, 64, (64,), "bf16", "square"))
    x["W"] = torch.eye(64, dtype=torch.float32)
    Q, K, V, W, dY = (dev(x[k]) for k in ("Q", "K", "V", "W", "dY"))
    Y, st, _ = slim.fwd(Q, K, V, W, 64, "square")
    dQ, dK, dV, dW, _ = slim.bwd(Q, K, V, W, dY, 64, None, "square")
    torch.cuda.synchronize()
    h = H - 1
    sl = lambda t: t[:, h:h + 1]
    Yr, sto = O.slim_forward(sl(x["Q"]), sl(x["K"]), sl(x["V"]), x["W"], 256, O.SQUARE, within="quadratic")
    gr = O.slim_backward(sl(x["Q"]), sl(x["K"]), sl(x["V"]), x["W"], sl(x["dY"]), 256, O.SQUARE, sto,
                         within="quadratic")
    report("Y (one head)", host64(sl(Y)), Yr, TOL["bf16"])
    for n, a, r in zip(("dQ", "dK", "dV"), (dQ, dK, dV), gr[:3]):
        report(f"{n} (one head)", host64(sl(a)), r, TOL["bf16"])
    # dW sums every head: check it against the oracle over all heads only for
    # the shorter shapes (the oracle runs in seconds there)
    if L * H <= 1024 * 8:
        gall = O.attention_backward(x["Q"], x["K"], x["V"], x["W"], x["dY"], O.SQUARE)
        report("dW (all heads)", host64(dW), gall[3], TOL["bf16"])
