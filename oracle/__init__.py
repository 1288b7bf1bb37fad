"""fp64 CPU oracle of the PI-GAN training step.

TEST INFRASTRUCTURE: imported only by the tests, the package smoke check and
the benchmark's CPU-baseline leg.  It shares no code with the HIP path.
"""
from .pigan_oracle import (  # noqa: F401
    unpack, pack, gen_forward, gen_backward, mlp_forward, mlp_backward,
    darcy_residual, sensor_rows, colloc_rows, gen_jets, snapshots,
    train_step_group, train_step, real_snapshots,
    critic_input_grad, tangent_output_grad, gradient_penalty,
    trunk_unpack, trunk_pack, trunk_skip, trunk_forward, trunk_backward, trunk_snapshots,
    train_step_group_trunk, train_step_trunk, real_snapshots_trunk,
    train_step_hier, real_snapshots_hier,
)
