"""CPU oracle for the DeepPCR hot path (numpy float64).

TEST INFRASTRUCTURE: imported only by the test suite, the smoke check and the
benchmark's CPU-baseline leg, never by the GPU library or its binding.
"""
from .deeppcr_oracle import (  # noqa: F401
    TANH_MLP, TANH_RESIDUAL, SIGMOID_MLP, SIGMOID_RESIDUAL, RELU_MLP, RELU_RESIDUAL,
    is_residual, activation, step, step_jacobian, preactivation, seq_forward,
    layer_inputs, all_jacobians, all_steps, seq_solve, pcr_solve,
    reversed_transposed_system, num_levels, initial_guess, newton_forward,
    residual_norm, newton_forward_residual,
    seq_backward, loss,
)
from . import resnet_oracle  # noqa: F401
from . import diffusion_oracle  # noqa: F401
from . import sharded_oracle  # noqa: F401
