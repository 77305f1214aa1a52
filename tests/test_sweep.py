"""CPU side of the parity sweep: every seeded random configuration is a valid
model and resume (the host planner accepts it), and the address replays of
both kernels (restore and checkpoint write) stay in bounds and cover exactly
the rows they must."""
import pytest

from sweep import LIMIT_CASES, SWEEP_SIZE, describe, limit_case, sweep_case
from test_gather_indexing import emulate as emulate_checkpoint_write
from test_kernel_indexing import emulate as emulate_restore


@pytest.mark.parametrize("i", range(SWEEP_SIZE))
def test_sweep_addresses(i):
    case = sweep_case(i)
    print(describe(case))
    emulate_restore(case)
    emulate_checkpoint_write(case)


@pytest.mark.parametrize("name", sorted(LIMIT_CASES))
def test_limit_addresses(name):
    case = limit_case(name)
    print(describe(case))
    emulate_restore(case)
    emulate_checkpoint_write(case)
