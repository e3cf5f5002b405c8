"""Random-init parameters and random byte strings for the s-layer Performer
language model (Sec. 2.2, eqs. 5-10; Sec. 4: configurations I-IV with
d_ff = 4 d_model, k = d_model / 64 heads, s = 3 layers, alphabet
{0, ..., 255}, batch 1).

Recipe (one seeded PCG64 stream per tensor): linear weights and biases
uniform in +-1/sqrt(fan_in) (the common default of linear layers), the
token embedding N(0, 1), layer-normalisation gains 1 and shifts 0 (tests
that must exercise them draw them instead: `perturb_ln=True`), tokens
uniform over the alphabet, as the paper's benchmarks use random strings.
No arithmetic of the model itself lives here.
"""

from __future__ import annotations

import dataclasses
from typing import Dict

import numpy as np
import torch

from .inputs import SEED

VOCAB = 256


@dataclasses.dataclass(frozen=True)
class ModelConfig:
    name: str
    L: int
    D: int  # d_model
    s: int = 3
    vocab: int = VOCAB
    B: int = 1
    heads: int = 0  # 0: D / 64

    @property
    def k(self) -> int:
        return self.heads or self.D // 64

    @property
    def F(self) -> int:
        return 4 * self.D


# the paper's configurations (Sec. 4): (L, d_model)
MODEL_CONFIGS = {
    "I": ModelConfig("I", 512, 256),
    "II": ModelConfig("II", 1024, 512),
    "III": ModelConfig("III", 4096, 1024),
    "IV": ModelConfig("IV", 16384, 1024),
}


def _rng(cfg_id: int, tensor: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(SEED, spawn_key=(7, cfg_id, tensor))))


def param_names(s: int):
    names = ["emb"]
    for r in range(s):
        names += [f"{n}{r}" for n in ("Wq", "Wk", "Wv", "ln1_g", "ln1_b", "W1", "b1", "W2", "b2", "ln2_g", "ln2_b")]
    return names + ["Wout", "bout"]


def make_model(cfg: ModelConfig, seed: int = 0, perturb_ln: bool = False) -> Dict[str, torch.Tensor]:
    """float32 parameters of the model, keyed as param_names(cfg.s)."""
    D, F, V = cfg.D, cfg.F, cfg.vocab
    shapes = {"emb": (V, D), "Wout": (D, V), "bout": (V,)}
    fan = {"Wout": D, "bout": D}
    for r in range(cfg.s):
        for n in ("Wq", "Wk", "Wv"):
            shapes[f"{n}{r}"] = (D, D)
            fan[f"{n}{r}"] = D
        shapes[f"W1{r}"], fan[f"W1{r}"] = (D, F), D
        shapes[f"b1{r}"], fan[f"b1{r}"] = (F,), D
        shapes[f"W2{r}"], fan[f"W2{r}"] = (F, D), F
        shapes[f"b2{r}"], fan[f"b2{r}"] = (D,), F
        for n in ("ln1_g", "ln1_b", "ln2_g", "ln2_b"):
            shapes[f"{n}{r}"] = (D,)
    out = {}
    for i, name in enumerate(param_names(cfg.s)):
        g = _rng(seed * 1000 + 17, i)
        shp = shapes[name]
        if name == "emb":
            x = g.standard_normal(shp, dtype=np.float32)
        elif name.startswith("ln"):
            if perturb_ln:
                x = (1.0 if "_g" in name else 0.0) + 0.3 * g.standard_normal(shp).astype(np.float32)
            else:
                x = np.full(shp, 1.0 if "_g" in name else 0.0, dtype=np.float32)
        else:
            b = 1.0 / np.sqrt(fan[name])
            x = g.uniform(-b, b, shp).astype(np.float32)
        out[name] = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return out


def make_tokens(cfg: ModelConfig, seed: int = 0) -> torch.Tensor:
    """int32 [B, L] tokens uniform over the alphabet."""
    g = _rng(seed * 1000 + 23, 0)
    return torch.from_numpy(g.integers(0, cfg.vocab, size=(cfg.B, cfg.L), dtype=np.int32))
