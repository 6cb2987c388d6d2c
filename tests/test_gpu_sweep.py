"""A fixed-seed slice of the random parity sweep (tests/sweep_parity.py) in
the GPU suite: 60 fp32, 25 bf16-input, 30 exponential-weight, 25
bf16-output and 20 forward-only cases, each with its own operator, shape,
grid policy and deterministic switch, against the oracle at the parity
tests' bars (a slice cancelled below the rounding bound of its inputs is
held to that floor, as in test_near_one_hot_slices_at_the_fp32_floor)."""
import random

import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

import sweep_parity as S  # noqa: E402

LEGS = [("fp32", 60), ("bf16", 25), ("exp", 30), ("bf16o", 25), ("forward-only", 20)]


def test_random_parity_sweep(oracle_mod):
    rng = random.Random(7)
    n = 0
    for leg, count in LEGS:
        for _ in range(count):
            S.run_case(rng, leg, n, 7)
            n += 1
