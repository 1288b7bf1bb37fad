"""fp64 CPU oracle of the PI-GAN training step.

TEST INFRASTRUCTURE: imported only by the tests, the package smoke check and
the benchmark's CPU-baseline leg.  It shares no code with the HIP path.
"""
from .pigan_oracle import (  # noqa: F401
    unpack, pack, gen_forward, gen_backward, mlp_forward, mlp_backward,
    darcy_residual, sensor_rows, colloc_rows, gen_jets, snapshots,
    train_step_group, train_step, real_snapshots,
    critic_input_grad, tangent_output_grad, gradient_penalty,
)
