"""The C ABI library loads, exports what include/*.h declare, and rejects
bad arguments on the host with the documented status codes (no GPU needed:
validation happens before any HIP call)."""

import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = [os.path.join(ROOT, "include", h) for h in sorted(os.listdir(os.path.join(ROOT, "include"))) if h.endswith(".h")]


def _declared():
    names = set()
    for h in HEADERS:
        text = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        names |= set(re.findall(r"\b(slim_[a-z_]+)\s*\(", text))
    return sorted(names)


@pytest.fixture(scope="module")
def S():
    from paper_2012_11346_amd import slim

    return slim


def test_every_declared_symbol_is_exported(S):
    names = _declared()
    assert "slim_fwd" in names and "slim_bwd" in names and "slim_featmap" in names
    for n in names:
        assert hasattr(S.LIB, n), n
    assert set(names) == set(S.EXPORTED)


def test_status_strings(S):
    for code in (S.SLIM_OK, S.SLIM_EINVAL, S.SLIM_EUNSUPPORTED, S.SLIM_EWORKSPACE, S.SLIM_EHIP):
        assert S.LIB.slim_status_string(code).decode()
    assert S.LIB.slim_status_string(123).decode() == "unknown status"


def _p(S, **kw):
    base = dict(B=2, H=3, L=1000, d=64, M=256, C=64, dtype=S.BF16, kind=S.FAVOR_PLUS)
    base.update(kw)
    return S.problem(**base)


def test_workspace_is_flat_in_L(S):
    sizes = [S.workspace_bytes(_p(S, L=L), ph) for L in (32768, 262144, 1 << 21) for ph in (S.PHASE_BWD,)]
    assert len(set(sizes)) == 1
    fw = [S.workspace_bytes(_p(S, L=L), S.PHASE_FWD) for L in (32768, 262144, 1 << 21)]
    assert len(set(fw)) == 1
    # the segment count depends on B*H (device fill), not on L
    assert S.num_segments(_p(S, L=32768)) == S.num_segments(_p(S, L=1 << 21)) > 1


def test_context_is_state_sized_and_flat_in_L(S):
    """The forward-to-backward context holds P2 + 1 boundary states per head:
    its size depends on B H, M, d and the device, not on L."""
    sizes = [S.context_bytes(_p(S, L=L)) for L in (32768, 262144, 1 << 21)]
    assert len(set(sizes)) == 1 and sizes[0] > 0
    per_state = 256 * 65 * 4
    assert sizes[0] % (2 * 3 * per_state) == 0
    # bf16 problems on the key-sum kernel only; fp32 problems and sequences
    # of one tile (one part, nothing to hand over) use none
    assert S.context_bytes(_p(S, dtype=S.F32, d=32, M=64)) == 0
    assert S.context_bytes(_p(S, L=32)) == 0
    # short sequences: one part (one exact boundary state) per tile
    assert S.context_bytes(_p(S, L=64 * 5)) == 2 * 3 * (10 + 1) * per_state
    assert S.context_bytes(_p(S, C=0)) == 0


@pytest.mark.parametrize(
    "kw, code",
    [
        (dict(C=0), -1),
        (dict(L=0), -1),
        (dict(B=0), -1),
        (dict(dtype=7), -1),
        (dict(kind=5), -1),
        (dict(d=48), -2),
        (dict(M=96), -2),
        (dict(M=512), -2),
        (dict(L=(1 << 23) + 1), -2),  # one bf16 head of d=64 rows above 1 GiB
        (dict(B=300, H=300), -2),
    ],
)
def test_invalid_problems_are_rejected(S, kw, code):
    p = _p(S, **kw)
    assert S.LIB.slim_workspace_bytes(ctypes.byref(p), 0) == 0
    assert S.LIB.slim_num_segments(ctypes.byref(p)) == 0
    st = S.LIB.slim_fwd(ctypes.byref(p), 1, 1, 1, 1, None, None, 1, None, 1, 1, None, 1, 1 << 30, None)
    assert st == code
    assert S.LIB.slim_last_error().decode()


# a fake, suitably aligned device address: validation rejects before any use
A = 1 << 12


def test_null_pointers_are_rejected_before_any_launch(S):
    p = _p(S)
    # arguments: p, Q, K, V, W, state_in, kshift_in, Y, logD, state_out, kshift_out, ctx, ws, ws_bytes, stream
    st = S.LIB.slim_fwd(ctypes.byref(p), None, A, A, A, None, None, A, None, A, A, None, A, 1 << 30, None)
    assert st == S.SLIM_EINVAL
    # FAVOR+ needs a key-shift output
    st = S.LIB.slim_fwd(ctypes.byref(p), A, A, A, A, None, None, A, None, A, None, None, A, 1 << 30, None)
    assert st == S.SLIM_EINVAL
    # a state without its shift
    st = S.LIB.slim_fwd(ctypes.byref(p), A, A, A, A, A, None, A, None, A, A, None, A, 1 << 30, None)
    assert st == S.SLIM_EINVAL
    # arguments: p, Q, K, V, W, state_in, kshift_in, kshift, dY, Y, logD, dstate_out, dQ, dK, dV, dW,
    # dstate_in, ctx, ws, ws_bytes, stream
    st = S.LIB.slim_bwd(ctypes.byref(p), A, A, A, A, None, None, A, A, None, None, None, None, A, A,
                        A, None, None, A, 1 << 30, None)
    assert st == S.SLIM_EINVAL  # dQ missing
    st = S.LIB.slim_bwd(ctypes.byref(p), A, A, A, A, None, None, None, A, None, None, None, A, A, A,
                        A, None, None, A, 1 << 30, None)
    assert st == S.SLIM_EINVAL  # kshift missing (FAVOR+)
    st = S.LIB.slim_bwd(ctypes.byref(p), A, A, A, A, A, None, A, A, None, None, None, A, A, A,
                        A, None, None, A, 1 << 30, None)
    assert st == S.SLIM_EINVAL  # state_in without kshift_in
    st = S.LIB.slim_bwd(ctypes.byref(p), A, A, A, A, None, None, A, A, None, None, None, A, A, A,
                        A, None, None, A, 0, None)
    assert st == S.SLIM_EWORKSPACE
    st = S.LIB.slim_featmap(ctypes.byref(p), None, A, 0, A, A, None)
    assert st == S.SLIM_EINVAL
    st = S.LIB.slim_featmap(ctypes.byref(p), A, A, 5, A, A, None)
    assert st == S.SLIM_EINVAL


def test_misaligned_tensors_are_rejected_before_any_launch(S):
    p = _p(S)
    # a row tensor (dY) 8 bytes off a 16-byte boundary
    st = S.LIB.slim_bwd(ctypes.byref(p), A, A, A, A, None, None, A, A + 8, None, None, None, A, A, A,
                        A, None, None, A, 1 << 30, None)
    assert st == S.SLIM_EINVAL and "aligned" in S.LIB.slim_last_error().decode()
    # the optional Y, likewise
    st = S.LIB.slim_bwd(ctypes.byref(p), A, A, A, A, None, None, A, A, A + 8, None, None, A, A, A,
                        A, None, None, A, 1 << 30, None)
    assert st == S.SLIM_EINVAL and "aligned" in S.LIB.slim_last_error().decode()
    # logD: 4-byte aligned; only with Y in the backward; only in the tile-walk mode
    st = S.LIB.slim_fwd(ctypes.byref(p), A, A, A, A, None, None, A, A + 2, A, A, None, A, 1 << 30, None)
    assert st == S.SLIM_EINVAL and "aligned" in S.LIB.slim_last_error().decode()
    st = S.LIB.slim_bwd(ctypes.byref(p), A, A, A, A, None, None, A, A, None, A, None, A, A, A,
                        A, None, None, A, 1 << 30, None)
    assert st == S.SLIM_EINVAL and "with Y" in S.LIB.slim_last_error().decode()
    q = _p(S, within=S.WITHIN_QUADRATIC)
    st = S.LIB.slim_fwd(ctypes.byref(q), A, A, A, A, None, None, A, A, A, A, None, A, 1 << 30, None)
    assert st == S.SLIM_EUNSUPPORTED and "logD" in S.LIB.slim_last_error().decode()
    # the workspace
    st = S.LIB.slim_fwd(ctypes.byref(p), A, A, A, A, None, None, A, None, A, A, None, A + 4, 1 << 30, None)
    assert st == S.SLIM_EINVAL
    # a float tensor (W) off a 4-byte boundary
    st = S.LIB.slim_fwd(ctypes.byref(p), A, A, A, A + 2, None, None, A, None, A, A, None, A, 1 << 30, None)
    assert st == S.SLIM_EINVAL
    st = S.LIB.slim_featmap(ctypes.byref(p), A + 8, A, 0, A, A, None)
    assert st == S.SLIM_EINVAL


def test_square_map_needs_64_features(S):
    import ctypes

    for M in (128, 256):
        p = _p(S, M=M, kind=S.SQUARE)
        assert S.LIB.slim_workspace_bytes(ctypes.byref(p), S.PHASE_FWD) == 0
        assert "square" in S.LIB.slim_last_error().decode()
    assert S.LIB.slim_workspace_bytes(ctypes.byref(_p(S, M=64, kind=S.SQUARE)), S.PHASE_BWD) > 0


def test_dropout_probability_is_checked(S):
    import ctypes

    for p in (-0.1, 1.0, float("nan")):
        assert S.LIB.slim_workspace_bytes(ctypes.byref(_p(S, dropout=p)), S.PHASE_FWD) == 0
        assert "dropout" in S.LIB.slim_last_error().decode()
    assert S.LIB.slim_workspace_bytes(ctypes.byref(_p(S, dropout=0.5, seed=2 ** 64 - 1)), S.PHASE_FWD) > 0


def test_relu_needs_positive_eps(S):
    p = _p(S, kind=S.RELU)
    p.relu_eps = 0.0
    assert S.LIB.slim_num_segments(ctypes.byref(p)) == 0


def test_walk_timer_arguments(S):
    """slim_time_walk validates its arguments on the host (no HIP call)."""
    ev = ctypes.c_void_p(0x1000)
    assert S.LIB.slim_time_walk(7, ev, ev) == S.SLIM_EINVAL
    assert S.LIB.slim_time_walk(S.PHASE_BWD, ev, None) == S.SLIM_EINVAL
    assert S.LIB.slim_time_walk(S.PHASE_FWD, None, None) == S.SLIM_OK
    assert S.LIB.slim_time_walk(S.PHASE_BWD, None, None) == S.SLIM_OK


# ---------------------------------------------------------------- the model step (include/slim_model.h)


def _m(S, **kw):
    base = dict(B=1, L=16384, D=1024, s=3, vocab=256, F=4096, C=512)
    base.update(kw)
    return S.model_desc(**base)


def test_model_workspace_grows_with_C_not_L(S):
    ws = [S.model_workspace_bytes(_m(S, L=L)) for L in (16384, 65536, 1 << 20)]
    assert ws[0] > 0 and len(set(ws)) == 1
    # the activations of one slice scale with C
    w1, w2 = S.model_workspace_bytes(_m(S, C=512)), S.model_workspace_bytes(_m(S, C=1024))
    assert 1.8 * w1 < w2 < 2.2 * w1
    assert S.LIB.slim_model_num_params(ctypes.byref(_m(S))) == 11 * 3 + 3
    assert S.LIB.slim_model_num_params(None) == 0


@pytest.mark.parametrize(
    "kw",
    [dict(D=96), dict(D=0), dict(D=8192), dict(vocab=1), dict(vocab=70000), dict(F=6), dict(C=0), dict(L=1),
     dict(s=0), dict(B=0), dict(ln_eps=0.0), dict(L=1 << 22, C=1 << 22)],
)
def test_invalid_models_are_rejected(S, kw):
    m = _m(S, **kw)
    assert S.model_workspace_bytes(m) == 0
    n = S.LIB.slim_model_num_params(ctypes.byref(m))
    arr = (ctypes.c_void_p * max(n, 1))(*([A] * max(n, 1)))
    st = S.LIB.slim_model_step(ctypes.byref(m), A, arr, arr, A, A, 1 << 40, None)
    assert st in (S.SLIM_EINVAL, S.SLIM_EUNSUPPORTED)


def test_model_step_checks_pointers_and_workspace(S):
    m = _m(S, L=64, C=16)
    n = S.LIB.slim_model_num_params(ctypes.byref(m))
    arr = (ctypes.c_void_p * n)(*([A] * n))
    need = S.model_workspace_bytes(m)
    st = S.LIB.slim_model_step(ctypes.byref(m), None, arr, arr, A, A, need, None)
    assert st == S.SLIM_EINVAL
    holed = (ctypes.c_void_p * n)(*([A] * (n - 1) + [None]))
    st = S.LIB.slim_model_step(ctypes.byref(m), A, arr, holed, A, A, need, None)
    assert st == S.SLIM_EINVAL
    st = S.LIB.slim_model_step(ctypes.byref(m), A, arr, arr, A, A, need - 1, None)
    assert st == S.SLIM_EWORKSPACE
    st = S.LIB.slim_model_step(ctypes.byref(m), A, arr, arr, A, A + 16, need, None)
    assert st == S.SLIM_EINVAL  # not 256-byte aligned


def test_model_param_shapes_match_the_synthetic_model(S):
    from synth import ModelConfig, make_model

    cfg = ModelConfig("shapes", L=8, D=128, s=2, vocab=37, B=1)
    P = make_model(cfg)
    shp = S.model_param_shapes(cfg.s, cfg.vocab, cfg.D, cfg.F)
    assert list(P) == S.model_param_names(cfg.s) and set(shp) == set(P)
    for k, v in P.items():
        assert tuple(v.shape) == shp[k], k


def test_ps_mode_sizing_and_checks(S):
    """The explicit prefix-sum mode: any dtype and shape (float32 at d = 64,
    M = 256 included), its states written out for C rows (the workspace grows
    with C, and is flat in L once the sequence has at least 64 slices); no
    dropout."""
    p = lambda **kw: _p(S, within=S.WITHIN_PS, **kw)
    f32 = p(dtype=S.F32, L=4096)
    assert S.workspace_bytes(f32, S.PHASE_FWD) > 0 and S.workspace_bytes(f32, S.PHASE_BWD) > 0
    ws0 = lambda q, ph: S.LIB.slim_workspace_bytes(ctypes.byref(q), ph)  # 0 for a rejected problem
    assert ws0(_p(S, dtype=S.F32, L=4096), S.PHASE_FWD) == 0  # the other modes reject it
    a, b = (S.workspace_bytes(p(C=c, L=1 << 16), S.PHASE_FWD) for c in (64, 128))
    assert 1.8 * a < b < 2.2 * a
    # the backward's grows linearly in C (twice the rows' states, plus parts of fixed size)
    w = [S.workspace_bytes(p(C=c, L=1 << 16), S.PHASE_BWD) for c in (64, 128, 192)]
    assert abs((w[2] - w[1]) - (w[1] - w[0])) <= 1024 and w[1] - w[0] > 1.9 * (b - a)
    assert len({S.workspace_bytes(p(C=64, L=L), S.PHASE_BWD) for L in (1 << 13, 1 << 16, 1 << 19)}) == 1
    assert ws0(p(dropout=0.1), S.PHASE_FWD) == 0
    assert S.context_bytes(p(L=1 << 16)) == 0
