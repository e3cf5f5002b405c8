"""slim_fwd_noalloc: the forward on the library's static device scratch.

Called through the C ABI (ctypes on libslim.so) and compared with slim_fwd on
a caller-provided workspace: two calls in a row on one device, the second
with a smaller problem (the scratch keeps the first call's contents), and
the outputs must equal slim_fwd's bit for bit (same kernels, same launch
plan); the first is also checked against the fp64 oracle on a sampled head.
"""

import ctypes

import numpy as np
import pytest
import torch

import oracle as O
from synth import Workload, make_inputs
from tests.gpu_common import TOL, dev, host64, need_gpu, report


def _abi_fwd(S, p, Q, K, V, W, Y, st, ks, ctx, ws):
    args = [ctypes.byref(p), S._ptr(Q), S._ptr(K), S._ptr(V), S._ptr(W), None, None, S._ptr(Y), None, S._ptr(st),
            S._ptr(ks), S._ptr(ctx)]
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if ws is None:
        return S.LIB.slim_fwd_noalloc(*args, stream)
    return S.LIB.slim_fwd(*args, S._ptr(ws), ctypes.c_size_t(ws.numel()), stream)


def test_noalloc_rejects_problems_beyond_the_scratch():
    """Checked on the host before any HIP call (no GPU needed)."""
    from paper_2012_11346_amd import slim as S

    cap = S.LIB.slim_noalloc_scratch_bytes()
    assert cap == 72 << 20
    big = S.problem(64, 8, 4096, 64, 256, 64, S.BF16, S.FAVOR_PLUS)
    assert S.workspace_bytes(big, S.PHASE_FWD) > cap
    st = S.LIB.slim_fwd_noalloc(ctypes.byref(big), *([ctypes.c_void_p(16)] * 4), None, None,
                                ctypes.c_void_p(16), None, ctypes.c_void_p(16), ctypes.c_void_p(16), None, None)
    assert st == S.SLIM_EUNSUPPORTED
    assert "static scratch" in S.LIB.slim_last_error().decode()


@pytest.mark.gpu
def test_noalloc_forward_equals_workspace_forward():
    need_gpu()
    from paper_2012_11346_amd import slim as S

    cases = [("first", Workload("noalloc_a", 910, 4, 8, 4096, 64, 256, (64,), "bf16", "favor+"), 64),
             ("second, smaller", Workload("noalloc_b", 911, 1, 2, 300, 64, 256, (100,), "bf16", "favor+"), 100)]
    for tag, wl, C in cases:
        print(f"[noalloc] {tag}: B={wl.B} H={wl.H} L={wl.L} d={wl.d} M={wl.M} C={C}", flush=True)
        x = make_inputs(wl)
        Q, K, V, W = (dev(x[k]) for k in ("Q", "K", "V", "W"))
        p = S.problem(wl.B, wl.H, wl.L, wl.d, wl.M, C, S.BF16, S.FAVOR_PLUS)
        need = S.workspace_bytes(p, S.PHASE_FWD)
        assert 0 < need <= S.LIB.slim_noalloc_scratch_bytes()
        ctxb = S.context_bytes(p)
        outs = []
        for use_ws in (True, False):
            Y = torch.empty_like(Q)
            st = torch.empty((wl.B, wl.H, wl.M, wl.d + 1), dtype=torch.float32, device=Q.device)
            ks = torch.empty((wl.B, wl.H), dtype=torch.float32, device=Q.device)
            ctx = torch.empty(max(1, ctxb // 4), dtype=torch.float32, device=Q.device) if ctxb else None
            ws = torch.empty(need, dtype=torch.uint8, device=Q.device) if use_ws else None
            rc = _abi_fwd(S, p, Q, K, V, W, Y, st, ks, ctx, ws)
            assert rc == S.SLIM_OK, S.LIB.slim_last_error().decode()
            torch.cuda.synchronize()
            outs.append((Y, st, ks, ctx))
        (Y0, st0, ks0, c0), (Y1, st1, ks1, c1) = outs
        assert torch.equal(Y0, Y1) and torch.equal(st0, st1) and torch.equal(ks0, ks1)
        if c0 is not None:
            assert torch.equal(c0, c1)
        # and both match the definition on one head
        b, h = wl.B - 1, wl.H - 1
        Yr = O.attention_forward(x["Q"][b:b + 1, h:h + 1], x["K"][b:b + 1, h:h + 1], x["V"][b:b + 1, h:h + 1],
                                 x["W"], "favor+")
        report(f"{tag}: Y (noalloc, one head)", host64(Y1[b:b + 1, h:h + 1]), Yr, TOL["bf16"])
