"""Slice-wise exact causal linear attention (SLiM, one layer) for MI355X.

The computation lives in the HIP library libslim.so (C ABI: include/slim.h);
`paper_2012_11346_amd.slim` is its ctypes binding on torch tensors.
"""

from . import slim  # noqa: F401
from .slim import bwd, featmap, fwd, num_segments, problem, workspace_bytes  # noqa: F401
