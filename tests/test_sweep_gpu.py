"""GPU side of the parity sweep: for every seeded random configuration, the
restore against a full oracle restore (every cache byte) and the checkpoint
write against the oracle quantizer (bit for bit)."""
import pytest

from paper_2609_26219_amd import binding as pb
from parity import check_both_orders, check_checkpoint_write, log
from sweep import LIMIT_CASES, SWEEP_SIZE, describe, limit_case, sweep_case

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch as _t
    if not _t.cuda.is_available():
        pytest.skip("no GPU")
    pb.load()
    return _t


@pytest.mark.parametrize("i", range(SWEEP_SIZE))
def test_sweep_parity(i, torch):
    case = sweep_case(i)
    log(f"[gpu] sweep {i}: {describe(case)}")
    check_both_orders(case)
    check_checkpoint_write(case, torch)


@pytest.mark.parametrize("name", sorted(LIMIT_CASES))
def test_limit_parity(name, torch):
    case = limit_case(name)
    log(f"[gpu] limits {name}: {describe(case)}")
    check_both_orders(case)
    check_checkpoint_write(case, torch)
