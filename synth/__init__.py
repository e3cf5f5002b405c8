"""Seeded synthetic inputs shared by the oracle tests, the GPU tests and the bench.

This package holds no arithmetic of the attention method itself: it draws
random numbers, builds the random-feature matrix from its recipe, and rounds
values to the storage dtype.  Neither the oracle nor the HIP path is imported.
"""

from .inputs import (  # noqa: F401
    SEED,
    WORKLOADS,
    Workload,
    draw_gaussian,
    orthogonal_gaussian_features,
    make_inputs,
    round_to_dtype,
    workload,
)
from .model import MODEL_CONFIGS, ModelConfig, make_model, make_tokens  # noqa: F401
