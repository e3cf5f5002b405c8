"""GPU checks of the forward-to-backward context (slim_context_bytes).

With a context the forward stores its segment boundary states and the
backward reads them instead of rebuilding them from the keys and values.
Both ways run the same kernels on the same parts with the same key shift, so
every output must be bitwise identical with and without the context; the
parity of those outputs with the fp64 oracle is covered by the other GPU
tests (and checked here once more for one case).
"""

import pytest
import torch

import oracle as O
from synth import Workload, make_inputs
from tests.gpu_common import TOL, dev, host64, mask_w, need_gpu, report

pytestmark = pytest.mark.gpu

CASES = [
    # name, B, H, L, d, M, C, kind, with initial state
    ("favor_m256", 2, 2, 2048, 64, 256, 64, "favor+", False),
    ("favor_m256_state", 1, 3, 1500, 64, 256, 100, "favor+", True),
    ("relu_m128", 2, 2, 1024, 64, 128, 32, "relu", False),
    ("favor_d32_m128", 1, 4, 1200, 32, 128, 48, "favor+", True),
]


@pytest.mark.parametrize("i", range(len(CASES)))
def test_context_changes_nothing(i):
    need_gpu()
    from paper_2012_11346_amd import slim

    name, B, H, L, d, M, C, kind, with_state = CASES[i]
    print(f"\n[context] {name}: B={B} H={H} L={L} d={d} M={M} C={C} {kind} state={with_state}", flush=True)
    wl = Workload(name, 700 + i, B, H, L, d, M, (C,), "bf16", kind)
    x = make_inputs(wl)
    Q, K, V, W, dY = (dev(x[k]) for k in ("Q", "K", "V", "W", "dY"))
    p = slim.problem(B, H, L, d, M, C, torch.bfloat16, kind)
    assert slim.num_segments(p) > 1
    ctx = slim.new_context(Q, W, C, kind)
    assert ctx is not None and ctx.numel() * 4 == slim.context_bytes(p)
    st_in = ks_in = g_out = None
    if with_state:
        gen = torch.Generator(device="cpu").manual_seed(11 + i)
        st_in = dev(torch.rand((B, H, M, d + 1), generator=gen) * 3.0)
        ks_in = dev(torch.randn((B, H), generator=gen))
        g_out = dev(torch.randn((B, H, M, d + 1), generator=gen) * 1e-2)

    Y0, s0, k0 = slim.fwd(Q, K, V, W, C, kind, state_in=st_in, kshift_in=ks_in)
    g0 = slim.bwd(Q, K, V, W, dY, C, k0, kind, state_in=st_in, kshift_in=ks_in, dstate_out=g_out,
                  want_dstate_in=with_state)
    ctx.fill_(float("nan"))  # every entry the backward reads must come from the forward
    Y1, s1, k1 = slim.fwd(Q, K, V, W, C, kind, state_in=st_in, kshift_in=ks_in, ctx=ctx)
    g1 = slim.bwd(Q, K, V, W, dY, C, k1, kind, state_in=st_in, kshift_in=ks_in, dstate_out=g_out,
                  want_dstate_in=with_state, ctx=ctx)
    torch.cuda.synchronize()
    assert torch.equal(Y0, Y1) and torch.equal(s0, s1)
    if kind == "favor+":
        assert torch.equal(k0, k1)
    for n, a, b in zip(("dQ", "dK", "dV", "dW", "dstate_in"), g0, g1):
        if a is None:
            assert b is None
            continue
        assert torch.equal(a, b), n
    assert torch.isfinite(ctx).all()

    if i == 0:
        Yr = O.attention_forward(x["Q"], x["K"], x["V"], x["W"], kind)
        gr = O.attention_backward(x["Q"], x["K"], x["V"], x["W"], x["dY"], kind, mask_W=mask_w(x))
        tol = TOL["bf16"]
        report("Y", host64(Y1), Yr, tol)
        for n, a, r in zip(("dQ", "dK", "dV", "dW"), g1[:4], gr):
            report(n, host64(a), r, tol)
