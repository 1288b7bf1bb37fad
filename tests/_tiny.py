"""Small workload shapes shared by the oracle and parity tests."""
from paper_1910_13444_amd.configs import Workload

TINY2 = Workload("tiny2d", "fp32", G=1, d=2, n_z=2, L=2, W=3, S=2, P=3, n_sY=2, n_sU=2,
                 L_D=2, W_D=3, B_r=2, f_const=0.5, seed=7)
TINY1 = Workload("tiny1d", "fp32", G=1, d=1, n_z=2, L=2, W=4, S=3, P=2, n_sY=2, n_sU=3,
                 L_D=1, W_D=4, B_r=2, f_const=1.0, seed=8)
TINY3 = Workload("tiny3d", "fp32", G=2, d=3, n_z=1, L=3, W=3, S=2, P=2, n_sY=1, n_sU=2,
                 L_D=2, W_D=2, B_r=3, f_const=-0.25, seed=9)
