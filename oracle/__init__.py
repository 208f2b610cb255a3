"""Float64 CPU oracle of the two-axis tabular transformer layer.

TEST INFRASTRUCTURE ONLY: imported by the test-suite, the smoke check and the CPU-baseline leg
of the benchmark, never by the GPU package.  See layer.py for what it computes and the readings
it takes where the paper is silent.
"""

from .layer import (LN_EPS, PARAM_ORDER, attention, attention_backward, attention_probs,
                    dataset_backward, dataset_forward, gelu, gelu_grad, layer_backward,
                    layer_forward, layernorm, layernorm_backward, pack_params, param_count,
                    param_shapes, stack_backward, stack_forward, unpack_params)

__all__ = [
    "LN_EPS", "PARAM_ORDER", "attention", "attention_backward", "attention_probs",
    "dataset_backward", "dataset_forward", "gelu", "gelu_grad", "layer_backward",
    "layer_forward", "layernorm", "layernorm_backward", "pack_params", "param_count",
    "param_shapes", "stack_backward", "stack_forward", "unpack_params",
]
