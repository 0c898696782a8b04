"""GPU parity at the edges of what the library accepts: the most registers (32), the
widest one-row head count (64, the LDS-partials path), the smallest head dimension on the
MFMA path (d = 8, half of one k-step), 64 query heads on the MFMA path, anchor rows that
end one past a row block, and candidates far below the launch bound of a ragged batch."""
import numpy as np
import pytest

import oracle
from paper_2605_29657_amd import occam

from parity import custom_stage
from test_gpu_parity import run_and_check

pytestmark = pytest.mark.gpu


def test_32_registers_and_64_heads_on_the_one_row_path():
    sb = custom_stage(B=2, R=32, H=64, Hkv=64, d=64, T=[1, 1], N=[300, 7], seed=21)
    run_and_check(sb, 1.0)


def test_smallest_head_dim_on_the_mfma_path_with_32_registers():
    sb = custom_stage(B=2, R=32, H=8, Hkv=2, d=8, T=[3, 129], N=[40, 257], seed=22)
    run_and_check(sb, 1.0)


def test_64_query_heads_on_the_mfma_path():
    sb = custom_stage(B=1, R=1, H=64, Hkv=8, d=128, T=[256], N=[1000], seed=23)
    run_and_check(sb, 2.0)


def test_mean_threshold_and_register_max_at_32_registers():
    sb = custom_stage(B=3, R=32, H=4, Hkv=4, d=64, T=[7, 1, 64], N=[5, 0, 600], seed=24)
    run_and_check(sb, 1.5, reduce=oracle.REG_MAX)
    run_and_check(sb, 0.9, reduce=oracle.CAND_MEAN)


def test_candidates_far_below_the_launch_bound():
    # Ragged batch whose launch bound (max_cands) is set far above every sample.
    sb = custom_stage(B=3, R=2, H=4, Hkv=4, d=32, T=[16, 16, 16], N=[3, 50, 1], seed=25)
    run_and_check(sb, 1.0, max_cands=4096)
