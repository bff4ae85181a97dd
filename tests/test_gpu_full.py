"""GPU parity at the full workload sizes, in the launch configuration that
bench.py times (one occ_step_batched call per step over all matrices of the
workload, error buffer and Q carried from step to step).

Every matrix of a step is checked against the invariants that hold at any
size (M_hat + err == A, orthonormal P_hat, residual orthogonal to P_hat);
the float64 oracle follows every matrix of the single-matrix workloads and a
sample of the batched ones (one matrix of each shape), along its own
trajectory.  Tolerances as in test_gpu_parity.py.  The 1024 x 1024 workload
runs at full size there.
"""

import pytest

from gpu_util import assert_parity, run_workload
from workloads import WORKLOADS

pytestmark = pytest.mark.gpu


def _run(key, oracle_mats=None):
    w = WORKLOADS[key]
    print(f"[full] {w.name}: {len(w.shapes)} matrices, rank {w.rank}, iters {w.iters}, "
          f"{w.steps} steps", flush=True)
    res, _, _ = run_workload(w, w.steps, batched=True, oracle_mats=oracle_mats,
                             invariants_all=True)
    assert_parity(res, w.m_dtype, w.name)


def test_full_act_grad_8192x4096_bf16_r16_8_steps():
    _run(2)


def test_full_stage_weights_36_matrices_f32_r32_t2():
    # layer 0 and layer 8 of each of the four shapes
    _run(3, oracle_mats=[0, 1, 2, 3, 32, 33, 34, 35])


def test_full_embedding_51200x3072_zipf_f32_r64():
    _run(4)


def test_full_act_grad_4x16384x8192_bf16_r128_t2():
    _run(5, oracle_mats=[0, 3])
