"""GPU parity of value dropout with per-slice seeds (Sec. 5): the forward and
the backward regenerate the masks of each slice from its seed (the key
(seed, n) of slice n), so the downdates of the reverse walk subtract exactly
the masked contributions that were added; the oracle draws the same masks
from its own Philox4x64-10 (pinned against numpy's).  Bars as everywhere."""

import os

import numpy as np
import pytest
import torch

import oracle as O
from synth import Workload, make_inputs
from tests.gpu_common import TOL, dev, host64, mask_w, need_gpu, report

pytestmark = pytest.mark.gpu

# name, B, H, L, d, M, C, dtype, kind, p, seed, forced segments
CASES = [
    ("f32_d32_c16", 1, 2, 200, 32, 64, 16, "f32", "favor+", 0.2, 5, None),
    ("bf16_c64", 1, 2, 300, 64, 256, 64, "bf16", "favor+", 0.1, 123456789012345, None),
    ("bf16_relu_segments", 1, 2, 4096, 64, 128, 100, "bf16", "relu", 0.3, 2 ** 63 + 7, None),
    ("bf16_d32_segments_c40", 2, 1, 900, 32, 256, 40, "bf16", "favor+", 0.5, 77, 5),
    ("bf16_square_segments", 1, 3, 700, 64, 64, 64, "bf16", "square", 0.1, 9, 4),
]


@pytest.mark.parametrize("i, given_y", [(i, False) for i in range(len(CASES))] + [(1, True), (3, True), (4, True)] +
                         [(1, "logD"), (2, "logD"), (3, "logD")])
def test_dropout_forward_backward(i, given_y):
    """given_y: the backward also gets the forward's Y (with its dropout);
    "logD": and its logD (the carry-free backward)."""
    need_gpu()
    from paper_2012_11346_amd import slim

    name, B, H, L, d, M, C, dtype, kind, p, seed, segs = CASES[i]
    print(f"[dropout] case={name} B={B} H={H} L={L} d={d} M={M} C={C} {dtype} {kind} p={p} segments={segs} "
          f"given_y={given_y}", flush=True)
    x = make_inputs(Workload(name, 600 + i, B, H, L, d, M, (C,), dtype, kind))
    old = os.environ.get("SLIM_SEGMENTS")
    if segs is not None:
        os.environ["SLIM_SEGMENTS"] = str(segs)
    try:
        Q, K, V, W, dY = (dev(x[k]) for k in ("Q", "K", "V", "W", "dY"))
        lD = torch.empty((B, H, L), dtype=torch.float32, device=Q.device) if given_y == "logD" else None
        Y, st, ks = slim.fwd(Q, K, V, W, C, kind, dropout=p, seed=seed, logD=lD)
        dQ, dK, dV, dW, _ = slim.bwd(Q, K, V, W, dY, C, ks, kind, dropout=p, seed=seed, Y=Y if given_y else None,
                                     logD=lD)
        torch.cuda.synchronize()
    finally:
        if old is None:
            os.environ.pop("SLIM_SEGMENTS", None)
        else:
            os.environ["SLIM_SEGMENTS"] = old
    tol = TOL[dtype]
    Yr = O.dropout_forward(O.attention_forward, x["Q"], x["K"], x["V"], x["W"], kind, C, p, seed)
    report("Y", host64(Y), Yr, tol)
    # the state holds sum g(k) (m v)^T, unscaled
    m = O.value_mask(B, H, L, d, C, p, seed)
    _, stref = O.slim_forward(x["Q"], x["K"], m * host64(x["V"]), x["W"], C, kind, within="quadratic")
    s = host64(st)
    if kind == "favor+":
        s = s * np.exp(host64(ks))[:, :, None, None]
    report("state_out", s, stref, tol)
    ref = O.dropout_backward(O.attention_backward, x["Q"], x["K"], x["V"], x["W"], x["dY"], kind, C, p, seed,
                             mask_W=mask_w(x))
    for n, a, r in zip(("dQ", "dK", "dV", "dW"), (dQ, dK, dV, dW), ref):
        report(n, host64(a), r, tol)
    # dropped value elements get exactly zero gradient
    assert torch.count_nonzero(dV.cpu()[torch.from_numpy(m == 0)]).item() == 0


def test_dropout_masks_follow_the_slices():
    """The same inputs with another slice length draw other masks (slice n's
    seed is (seed, n)), and p = 0 is exactly the attention without dropout."""
    need_gpu()
    from paper_2012_11346_amd import slim

    x = make_inputs(Workload("drop_c", 650, 1, 2, 256, 64, 256, (64,), "bf16", "favor+"))
    Q, K, V, W = (dev(x[k]) for k in ("Q", "K", "V", "W"))
    Y64 = slim.fwd(Q, K, V, W, 64, "favor+", dropout=0.2, seed=3)[0]
    Y32 = slim.fwd(Q, K, V, W, 32, "favor+", dropout=0.2, seed=3)[0]
    Y0 = slim.fwd(Q, K, V, W, 64, "favor+", dropout=0.0, seed=3)[0]
    Yn = slim.fwd(Q, K, V, W, 64, "favor+")[0]
    torch.cuda.synchronize()
    assert torch.equal(Y0, Yn)
    # rows of the first slice of 32 agree (same seed, same rows), later ones differ
    assert torch.equal(Y64[:, :, :1], Y32[:, :, :1])
    assert not torch.equal(Y64[:, :, 64:], Y32[:, :, 64:])
    for C, Yc in ((64, Y64), (32, Y32)):
        Yr = O.dropout_forward(O.attention_forward, x["Q"], x["K"], x["V"], x["W"], "favor+", C, 0.2, 3)
        report(f"Y C={C}", host64(Yc), Yr, TOL["bf16"])
