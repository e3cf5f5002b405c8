"""GPU parity at the workloads' full sizes, in the launch configuration the
benchmark times (whole batch, the library's own segment plan).

The kernels run on the whole batch; the fp64 oracle (Algorithm 1 slice by
slice, whose exact result does not depend on C) computes a sample of whole
heads, row by row.  dW sums over every head, so a second backward with dY
zero outside the sampled heads isolates their share: its dW must match the
oracle's dW of the sample, every other head's dQ, dK, dV must be exactly zero
(dY = 0 makes every cotangent zero), and the sampled heads' dQ, dK, dV must
be bitwise those of the first backward (heads do not interact).

As in the benchmark, the backward gets the forward's Y and (tile-walk mode)
logD, unless `given` is off (then it recomputes them and carries the
segments' cotangents, D6).
"""

import numpy as np
import pytest
import torch

import oracle as O
from synth import make_inputs, workload
from tests.gpu_common import TOL, dev, host64, mask_w, need_gpu, report

pytestmark = pytest.mark.gpu

ORACLE_C = 64  # slice length of the oracle run (the exact result is the same for every C)


def _sample(t, heads):
    """[B, H, L, d] tensor -> [1, n, L, d] float64 array of the sampled heads."""
    return np.stack([host64(t[b, h]) for b, h in heads])[None]


def _oracle(x, heads, kind):
    Q, K, V, dY = (_sample(x[k], heads) for k in ("Q", "K", "V", "dY"))
    W = host64(x["W"])
    Y, st = O.slim_forward(Q, K, V, W, ORACLE_C, kind, within="quadratic")
    dQ, dK, dV, dW, _ = O.slim_backward(Q, K, V, W, dY, ORACLE_C, kind, st, within="quadratic",
                                        mask_W=mask_w(x))
    return Y, dQ, dK, dV, dW


def _check(tag, x, heads, C, kind, ref, within="iter", given=True):
    from paper_2012_11346_amd import slim

    tol = TOL[{torch.bfloat16: "bf16", torch.float32: "f32"}[x["Q"].dtype]]
    print(f"[full size] {tag} C={C} {within} given={given}: forward + backward on the whole batch", flush=True)
    Q, K, V, W, dY = (dev(x[k]) for k in ("Q", "K", "V", "W", "dY"))
    lD = torch.empty(Q.shape[:3], dtype=torch.float32, device=Q.device) if given and within == "iter" else None
    Y, st, ks = slim.fwd(Q, K, V, W, C, kind, within=within, logD=lD)
    Yg = Y if given else None
    g = slim.bwd(Q, K, V, W, dY, C, ks, kind, within=within, Y=Yg, logD=lD)
    torch.cuda.synchronize()
    Yr, dQr, dKr, dVr, dWr = ref
    report(f"{tag} C={C} Y (sampled heads)", _sample(Y, heads), Yr, tol)
    for n, a, r in zip(("dQ", "dK", "dV"), g[:3], (dQr, dKr, dVr)):
        report(f"{tag} C={C} {n} (sampled heads)", _sample(a, heads), r, tol)

    print(f"[full size] {tag} C={C}: backward with dY zero outside the sampled heads", flush=True)
    mask = torch.zeros(dY.shape[:2], dtype=torch.bool, device=dY.device)
    for b, h in heads:
        mask[b, h] = True
    dYm = torch.where(mask[:, :, None, None], dY, torch.zeros_like(dY))
    gm = slim.bwd(Q, K, V, W, dYm, C, ks, kind, within=within, Y=Yg, logD=lD)
    torch.cuda.synchronize()
    report(f"{tag} C={C} dW (sampled heads' share)", host64(gm[3]), dWr, tol)
    for n, a, full in zip(("dQ", "dK", "dV"), gm[:3], g[:3]):
        assert torch.count_nonzero(a[~mask]).item() == 0, f"{n}: heads with dY = 0 must get exact zeros"
        assert torch.equal(a[mask], full[mask]), f"{n}: sampled heads differ between the two backward calls"
    del Q, K, V, W, dY, dYm, Y, Yg, lD, st, ks, g, gm
    torch.cuda.empty_cache()


def test_mid_batch_full_size():
    """B=8, H=8, L=4096, d=64, M=256, FAVOR+, C=128, bf16."""
    need_gpu()
    wl = workload("mid_bf16")
    heads = [(0, 0), (3, 5), (7, 7)]
    x = make_inputs(wl)
    ref = _oracle(x, heads, wl.kind)
    for C in wl.C:
        _check(wl.name, x, heads, C, wl.kind, ref)


def test_slice_sweep_full_size():
    """B=4, H=8, L=32768, d=64, M=256, FAVOR+, bf16, every C of the sweep."""
    need_gpu()
    wl = workload("sweep_32k")
    heads = [(0, 0), (3, 7)]
    x = make_inputs(wl)
    print("[full size] oracle on the sampled heads", flush=True)
    ref = _oracle(x, heads, wl.kind)
    for C in wl.C:
        _check(wl.name, x, heads, C, wl.kind, ref)


def test_slice_sweep_full_size_without_forward_outputs():
    """The headline problem at C=64 with the backward recomputing N and D
    and carrying the segments' cotangents (no Y, no logD)."""
    need_gpu()
    wl = workload("sweep_32k")
    heads = [(2, 1)]
    x = make_inputs(wl)
    print("[full size] oracle on the sampled head", flush=True)
    ref = _oracle(x, heads, wl.kind)
    _check(wl.name, x, heads, 64, wl.kind, ref, given=False)


def test_slice_sweep_full_size_rounded_w():
    """The headline problem at C=64 with a bf16-representable W (the other
    tests pass the unrounded float32 W the interface takes)."""
    need_gpu()
    wl = workload("sweep_32k")
    heads = [(1, 2)]
    x = make_inputs(wl, round_w=True)
    print("[full size] oracle on the sampled head (rounded W)", flush=True)
    ref = _oracle(x, heads, wl.kind)
    _check(wl.name + " rounded W", x, heads, 64, wl.kind, ref)


def test_headline_shape_float32_ps_mode():
    """The headline problem in float32 (B=4, H=8, L=32768, d=64, M=256,
    C=64): the explicit prefix-sum mode, the one that takes float32 at
    d M > 4096, at the float32 bar."""
    need_gpu()
    wl = workload("sweep_32k").with_(name="sweep_32k_f32", dtype="f32")
    heads = [(2, 5)]
    x = make_inputs(wl)
    print("[full size] oracle on the sampled head (float32 inputs)", flush=True)
    ref = _oracle(x, heads, wl.kind)
    _check(wl.name, x, heads, 64, wl.kind, ref, within="ps")


def test_long_context_full_size():
    """B=1, H=8, L=262144, d=64, M=256, FAVOR+, C=512, bf16."""
    need_gpu()
    wl = workload("long_256k")
    heads = [(0, 5)]
    x = make_inputs(wl)
    print("[full size] oracle on the sampled head", flush=True)
    ref = _oracle(x, heads, wl.kind)
    for C in wl.C:
        _check(wl.name, x, heads, C, wl.kind, ref)


@pytest.mark.parametrize("layer", range(6))
def test_relu_layer_stack_full_size(layer):
    """One layer of the six-layer ReLU stack: B=2, H=16, L=16384, d=64,
    M=128, C=256, bf16 (the layers are independent operations)."""
    need_gpu()
    wl = workload("relu_stack")
    assert wl.layers == 6
    heads = [(layer % 2, (5 * layer + 3) % 16)]
    x = make_inputs(wl, layer=layer)
    ref = _oracle(x, heads, wl.kind)
    for C in wl.C:
        _check(f"{wl.name} layer {layer}", x, heads, C, wl.kind, ref)
