"""Float64 CPU oracle of the two-axis tabular transformer layer.

TEST INFRASTRUCTURE ONLY: imported by the test-suite, the smoke check and the CPU-baseline leg
of the benchmark, never by the GPU package.  See layer.py (the post-norm baseline block) and
prenorm.py (the pre-norm RMSNorm block of the current best record), ends.py (the encoders,
decoder and loss around the stack) and optim.py (gradient clipping, Muon, schedule-free AdamW)
for what they compute and the readings they take where the paper is silent.
"""

from .layer import (LN_EPS, PARAM_ORDER, attention, attention_backward, attention_probs,
                    dataset_backward, dataset_forward, gelu, gelu_grad, layer_backward,
                    layer_forward, layernorm, layernorm_backward, pack_params, param_count,
                    param_shapes, stack_backward, stack_forward, unpack_params)
from .prenorm import (PRENORM_PARAM_ORDER, RMS_EPS, pack_prenorm_params, prenorm_dataset_backward,
                      prenorm_dataset_forward, prenorm_layer_backward, prenorm_layer_forward,
                      prenorm_param_count, prenorm_param_shapes, prenorm_stack_backward,
                      prenorm_stack_forward, rmsnorm, rmsnorm_backward, thinking_rows_backward,
                      thinking_rows_forward, unpack_prenorm_params)

__all__ = [
    "LN_EPS", "PARAM_ORDER", "attention", "attention_backward", "attention_probs",
    "dataset_backward", "dataset_forward", "gelu", "gelu_grad", "layer_backward",
    "layer_forward", "layernorm", "layernorm_backward", "pack_params", "param_count",
    "param_shapes", "stack_backward", "stack_forward", "unpack_params",
    "PRENORM_PARAM_ORDER", "RMS_EPS", "pack_prenorm_params", "prenorm_dataset_backward",
    "prenorm_dataset_forward", "prenorm_layer_backward", "prenorm_layer_forward",
    "prenorm_param_count", "prenorm_param_shapes", "prenorm_stack_backward",
    "prenorm_stack_forward", "rmsnorm", "rmsnorm_backward", "thinking_rows_backward",
    "thinking_rows_forward", "unpack_prenorm_params",
]
