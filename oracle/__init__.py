"""fp64 CPU oracle for slice-wise causal linear attention.

TEST INFRASTRUCTURE ONLY: imported by tests/, by __graft_entry__.smoke() and by
the cpu_baseline leg of bench.py, never by the product package.  It shares no
code with the HIP path.
"""

from .slim_oracle import (  # noqa: F401
    FAVOR_PLUS,
    RELU,
    RELU_EPS,
    SQUARE,
    attention_backward,
    attention_forward,
    feature_logits,
    feature_map,
    feature_map_vjp,
    iterative_backward_features,
    iterative_forward_features,
    pack_state,
    quadratic_backward_features,
    quadratic_forward_features,
    slice_bounds,
    slim_backward,
    slim_backward_head,
    slim_forward,
    slim_forward_head,
    unpack_state,
)
from .dropout import (  # noqa: F401
    dropout_backward,
    dropout_forward,
    keep_threshold,
    output_scale,
    philox4x64_10,
    value_mask,
)
from .performer import (  # noqa: F401
    grad_discrepancy,
    model_algorithm1,
    model_full,
    model_loss,
)
