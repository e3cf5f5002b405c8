"""Synthetic inputs for slice-wise causal linear attention.

Recipe (one seeded stream per tensor, so that any tensor can be regenerated
on its own):

* Q, K, V ~ N(0, 1) * d**(-1/4), drawn in float32 from PCG64, then rounded
  to the workload dtype with round-to-nearest-even (bf16) or kept (fp32).
  The d**(-1/4) pre-scale plays the role of the usual 1/sqrt(d) temperature
  split between queries and keys; the attention itself has no temperature
  (Sec. 2.1, eq. 1).
* dY ~ N(0, 1), same rounding.
* W [M, d]: random features for the FAVOR+ map, built in float64 as
  ceil(M/d) independent blocks; each block is the orthogonal factor of a
  d x d Gaussian matrix (sign-fixed by diag(R)) whose rows are rescaled to
  the norms of independent N(0, I_d) draws; blocks are stacked and cut to M
  rows, then stored as float32 and handed to the library as such (the
  library's interface takes W in float32).  `round_w=True` rounds it to
  bf16 (RNE) first, so that W is also bf16-representable; the oracle
  always consumes exactly the W the library gets.  W is an input of the
  method, so the results do not depend on how it was drawn.

The paper benchmarks random byte strings pushed through a randomly
initialised model (Sec. 4.1); the per-head Q, K, V of such a model are close
to Gaussian, which is what these draws stand in for.  No dataset is used.
"""

from __future__ import annotations

import dataclasses
import math
from typing import Dict, Optional, Tuple

import numpy as np

SEED = 201211346

# tensor ids inside one (workload, layer) stream family
_TENSOR_IDS = {"Q": 0, "K": 1, "V": 2, "dY": 3, "W": 4}


@dataclasses.dataclass(frozen=True)
class Workload:
    """One benchmark / parity shape.  Sizes per attention op."""

    name: str
    wid: int
    B: int
    H: int
    L: int
    d: int
    M: int
    C: Tuple[int, ...]
    dtype: str  # "f32" or "bf16"
    kind: str  # "favor+" or "relu"
    layers: int = 1

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


WORKLOADS: Dict[str, Workload] = {
    w.name: w
    for w in [
        # tiny exact check, fp32
        Workload("tiny_exact", 0, 1, 1, 256, 32, 64, (32,), "f32", "favor+"),
        # medium bf16 case the quadratic definition still handles on the CPU
        Workload("mid_bf16", 1, 8, 8, 4096, 64, 256, (128,), "bf16", "favor+"),
        # headline: L = 32k, slice-length sweep
        Workload("sweep_32k", 2, 4, 8, 32768, 64, 256, (64, 256, 1024, 4096, 32768), "bf16", "favor+"),
        # long context, state-only memory
        Workload("long_256k", 3, 1, 8, 262144, 64, 256, (512,), "bf16", "favor+"),
        # ReLU map, six independent layers
        Workload("relu_stack", 4, 2, 16, 16384, 64, 128, (256,), "bf16", "relu", layers=6),
    ]
}


def workload(name: str) -> Workload:
    return WORKLOADS[name]


def _stream(wid: int, layer: int, tensor: str, seed: int = SEED) -> np.random.Generator:
    ss = np.random.SeedSequence(seed, spawn_key=(int(wid), int(layer), _TENSOR_IDS[tensor]))
    return np.random.Generator(np.random.PCG64(ss))


def draw_gaussian(shape, wid: int, layer: int, tensor: str, scale: float = 1.0, seed: int = SEED) -> np.ndarray:
    """float32 N(0, scale^2) draws from the (wid, layer, tensor) stream."""
    g = _stream(wid, layer, tensor, seed)
    x = g.standard_normal(size=shape, dtype=np.float32)
    if scale != 1.0:
        x *= np.float32(scale)
    return x


def orthogonal_gaussian_features(M: int, d: int, rng: np.random.Generator) -> np.ndarray:
    """[M, d] float64 block-orthogonal Gaussian random features."""
    blocks = []
    for _ in range(int(math.ceil(M / d))):
        G = rng.standard_normal((d, d))
        Qm, Rm = np.linalg.qr(G)
        Qm = Qm * np.sign(np.diag(Rm))[None, :]
        norms = np.linalg.norm(rng.standard_normal((d, d)), axis=1)
        blocks.append(Qm.T * norms[:, None])
    return np.concatenate(blocks, axis=0)[:M]


def round_to_dtype(x: np.ndarray, dtype: str):
    """Round a float array to the storage dtype.  Returns a torch CPU tensor.

    bf16 rounding is round-to-nearest-even from float32 (torch's conversion).
    """
    import torch

    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    if dtype == "bf16":
        return t.to(torch.bfloat16)
    if dtype == "f32":
        return t
    raise ValueError(dtype)


def make_inputs(
    wl: Workload,
    layer: int = 0,
    seed: int = SEED,
    tensors=("Q", "K", "V", "dY", "W"),
    scale_qk: Optional[float] = None,
    round_w: bool = False,
):
    """Seeded inputs of one attention op of a workload.

    Returns a dict of torch CPU tensors: Q, K, V, dY in the workload dtype
    with shape [B, H, L, d]; W float32 [M, d].  `scale_qk` multiplies Q and K
    on top of the d**(-1/4) pre-scale (used by stress tests); `round_w`
    makes W bf16-representable.
    """
    shp = (wl.B, wl.H, wl.L, wl.d)
    s = wl.d ** -0.25
    out = {}
    for name in tensors:
        if name == "W":
            import torch

            W = orthogonal_gaussian_features(wl.M, wl.d, _stream(wl.wid, layer, "W", seed))
            Wt = torch.from_numpy(np.ascontiguousarray(W, dtype=np.float32))
            if round_w:
                Wt = Wt.to(torch.bfloat16).to(torch.float32)
            out["W"] = Wt
            continue
        scale = 1.0 if name == "dY" else s
        if name in ("Q", "K") and scale_qk is not None:
            scale *= scale_qk
        out[name] = round_to_dtype(draw_gaussian(shp, wl.wid, layer, name, scale, seed), wl.dtype)
    return out
