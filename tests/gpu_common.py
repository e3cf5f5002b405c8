"""Helpers shared by the GPU parity tests: device placement, error metrics."""

import numpy as np
import pytest
import torch

# max-relative-error bars (error = max|x - ref| / max|ref|, per tensor)
TOL = {"f32": 1e-5, "bf16": 2e-2}


def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def dev(t):
    return t.to("cuda")


def host64(t):
    return t.detach().to("cpu").double().numpy()


def max_rel(x, ref) -> float:
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = float(np.max(np.abs(ref)))
    return float(np.max(np.abs(x - ref)) / (den if den > 0 else 1.0))


def l2_rel(x, ref) -> float:
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    return float(np.linalg.norm(x - ref) / max(np.linalg.norm(ref), 1e-300))


def report(name, x, ref, tol):
    e = max_rel(x, ref)
    print(f"  {name}: max_rel={e:.3e} l2_rel={l2_rel(x, ref):.3e} (tol {tol:g})", flush=True)
    assert np.all(np.isfinite(np.asarray(x))), f"{name} has non-finite values"
    assert e <= tol, f"{name}: max_rel {e:.3e} > {tol:g}"
    return e


def mask_w(x):
    """The W the oracle takes the ReLU derivative's 0/1 decisions with, for
    the inputs x: the library forms the logits w_m . x of bf16 problems from
    the bf16 split hi + lo of the float32 W (hi = RNE(w), lo = RNE(w - hi)),
    so for those the decision is taken with hi + lo (the same precision on
    both sides); fp32 problems use W itself (None)."""
    if x["Q"].dtype != torch.bfloat16:
        return None
    W = x["W"].float()
    hi = W.to(torch.bfloat16).float()
    lo = (W - hi).to(torch.bfloat16).float()
    return hi.double().numpy() + lo.double().numpy()
