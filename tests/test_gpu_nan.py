"""NaN inputs: the calls finish, NaN reaches the outputs the definition
(eq. 2) makes depend on it, and heads without NaN inputs stay finite.

One NaN in a query row touches only that row's output (queries never enter
the state); one NaN in a key row reaches every later row of its head
through the state (and the rows before it only where they share its tile,
depending on how a mode masks the causal scores).  The key shift is a
maximum that skips NaN, so it stays finite and the other heads are
untouched.  In the backward every head's dW share is summed, so dW is NaN.
"""

import numpy as np
import pytest
import torch

from synth import Workload, make_inputs
from tests.gpu_common import dev, need_gpu

pytestmark = pytest.mark.gpu

# name, d, M, dtype, within
CASES = [
    ("iter_bf16", 64, 256, "bf16", "iter"),
    ("iter_f32", 64, 64, "f32", "iter"),
    ("quadratic_bf16", 64, 256, "bf16", "quadratic"),
    ("ps_bf16", 64, 256, "bf16", "ps"),
]
QROW, KROW = 37, 100  # NaN in Q[0, 1, QROW, 5] and in K[1, 0, KROW, 3]


@pytest.mark.parametrize("i", range(len(CASES)))
def test_nan_inputs(i):
    need_gpu()
    from paper_2012_11346_amd import slim

    name, d, M, dtype, within = CASES[i]
    B, H, L, C = 2, 2, 300, 64
    print(f"[nan] case={name} B={B} H={H} L={L} d={d} M={M} C={C} {dtype} {within}", flush=True)
    x = make_inputs(Workload(f"nan{i}", 950 + i, B, H, L, d, M, (C,), dtype, "favor+"))
    x["Q"][0, 1, QROW, 5] = float("nan")
    x["K"][1, 0, KROW, 3] = float("nan")
    Q, K, V, W, dY = (dev(x[k]) for k in ("Q", "K", "V", "W", "dY"))
    Y, st, ks = slim.fwd(Q, K, V, W, C, within=within)
    g = slim.bwd(Q, K, V, W, dY, C, ks, within=within)
    torch.cuda.synchronize()
    Y = Y.float().cpu()
    assert torch.isfinite(ks).all(), "the key shift skips NaN"
    # the query's row only
    assert torch.isnan(Y[0, 1, QROW]).all()
    rows = torch.arange(L) != QROW
    assert torch.isfinite(Y[0, 1, rows]).all()
    # the key's row and every later one of its head; rows of earlier tiles untouched
    assert torch.isnan(Y[1, 0, KROW:]).all()
    assert torch.isfinite(Y[1, 0, : KROW // 32 * 32]).all()
    # heads without NaN inputs
    for b, h in ((0, 0), (1, 1)):
        assert torch.isfinite(Y[b, h]).all(), (b, h)
        for n, t in zip(("dQ", "dK", "dV"), g[:3]):
            assert torch.isfinite(t[b, h].float()).all(), (n, b, h)
    for b, h in ((0, 1), (1, 0)):
        assert any(torch.isnan(t[b, h].float()).any() for t in g[:3]), (b, h)
    assert torch.isnan(g[3]).any()
    assert np.isfinite(st[0, 0].cpu().numpy()).all() and np.isnan(st[1, 0].cpu().numpy()).any()
