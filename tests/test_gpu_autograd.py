"""slim.attention as a torch operation: autograd's gradients are those of
slim_bwd given the forward's Y and (tile-walk mode) logD, bitwise, and match
the fp64 oracle within the bars, in every within-slice mode; dropout draws
the same masks in the backward."""

import pytest
import torch

import oracle as O
from synth import Workload, make_inputs
from tests.gpu_common import TOL, dev, host64, mask_w, need_gpu, report

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("within", ["iter", "quadratic", "ps"])
def test_autograd_equals_the_backward_call(within):
    need_gpu()
    from paper_2012_11346_amd import slim

    B, H, L, d, M, C = 2, 2, 300, 64, 256, 64
    print(f"[autograd] within={within} B={B} H={H} L={L} d={d} M={M} C={C}", flush=True)
    x = make_inputs(Workload(f"ag_{within}", 980, B, H, L, d, M, (C,), "bf16", "favor+"))
    Q, K, V, W, dY = (dev(x[k]) for k in ("Q", "K", "V", "W", "dY"))
    leaves = [t.clone().requires_grad_(True) for t in (Q, K, V, W)]
    Y = slim.attention(*leaves, C, within=within)
    (Y.float() * dY.float()).sum().backward()
    lD = torch.empty(Q.shape[:3], dtype=torch.float32, device=Q.device) if within == "iter" else None
    Y2, _, ks = slim.fwd(Q, K, V, W, C, within=within, logD=lD)
    g = slim.bwd(Q, K, V, W, dY, C, ks, within=within, Y=Y2, logD=lD)
    torch.cuda.synchronize()
    assert torch.equal(Y.detach(), Y2)
    for n, leaf, ref in zip(("dQ", "dK", "dV", "dW"), leaves, g[:4]):
        assert torch.equal(leaf.grad, ref), n
    oref = O.attention_backward(x["Q"], x["K"], x["V"], x["W"], x["dY"], "favor+",
                                mask_W=None if within == "ps" else mask_w(x))
    for n, leaf, r in zip(("dQ", "dK", "dV", "dW"), leaves, oref):
        report(n, host64(leaf.grad), r, TOL["bf16"])


def test_autograd_with_dropout():
    need_gpu()
    from paper_2012_11346_amd import slim

    B, H, L, d, M, C, p, seed = 1, 2, 200, 64, 128, 64, 0.25, 7
    x = make_inputs(Workload("ag_drop", 981, B, H, L, d, M, (C,), "bf16", "favor+"))
    Q, K, V, W, dY = (dev(x[k]) for k in ("Q", "K", "V", "W", "dY"))
    leaves = [t.clone().requires_grad_(True) for t in (Q, K, V, W)]
    Y = slim.attention(*leaves, C, dropout=p, seed=seed)
    (Y.float() * dY.float()).sum().backward()
    lD = torch.empty(Q.shape[:3], dtype=torch.float32, device=Q.device)
    Y2, _, ks = slim.fwd(Q, K, V, W, C, dropout=p, seed=seed, logD=lD)
    g = slim.bwd(Q, K, V, W, dY, C, ks, dropout=p, seed=seed, Y=Y2, logD=lD)
    torch.cuda.synchronize()
    for n, leaf, ref in zip(("dQ", "dK", "dV", "dW"), leaves, g[:4]):
        assert torch.equal(leaf.grad, ref), n
