"""The resume planner (Eq. 9, 11, 12): pins of the oracle and parity of
libpkv's pkv_plan_repair with it.  All on the CPU."""
import ctypes

import numpy as np
import pytest

from oracle import planner as op
from paper_2609_26219_amd import binding as pb


def test_hand_worked_plan():
    # N = 10, B = 4: blocks {0..3}, {4..7}, {8, 9}.  d_hat = 2: D = {0, 1}.
    imp = [0.9, 0.9, 0.1, 0.7, 0.2, 0.05, 0.3, 0.3, 0.7, 0.0]
    # candidates 2..9 (8 tokens); kappa 1/8 -> k = floor(1 + 1/2) = 1: the tie
    # between tokens 3 and 8 (0.7) goes to token 3 (block 0), so block 2 stays in F
    assert op.repair_mask(10, 4, 2, imp, 1 / 8) == ([1, 0, 0], 1)
    # kappa 2/8 -> k = 2: tokens 3 and 8 -> blocks 0 and 2
    assert op.repair_mask(10, 4, 2, imp, 2 / 8) == ([1, 0, 1], 2)
    # kappa 4/8 -> k = 4: tokens 3, 8, then the 0.3 tie 6, 7 -> all blocks
    assert op.repair_mask(10, 4, 2, imp, 4 / 8) == ([1, 1, 1], 4)
    # kappa 0: only the dirty window
    assert op.repair_mask(10, 4, 2, imp, 0.0) == ([1, 0, 0], 0)
    # d_hat past the suffix: everything is dirty, nothing left to rank
    assert op.repair_mask(10, 4, 50, imp, 0.5) == ([1, 1, 1], 0)
    # the count rounds half up: 3 candidates * 0.5 = 1.5 -> 2
    assert op.nonlocal_count(3, 0.5) == 2 and op.nonlocal_count(1000, 0.015) == 15


@pytest.mark.parametrize("seed", range(6))
def test_oracle_properties(seed):
    rng = np.random.default_rng(seed)
    N = int(rng.integers(1, 700))
    B = int(rng.choice([1, 4, 16, 32, 64]))
    d = int(rng.integers(0, N + 20))
    kappa = float(rng.choice([0.0, 0.015, 0.1, 0.5, 1.0]))
    imp = rng.choice(np.linspace(0, 1, 17), size=N).astype(np.float32)  # many ties
    mask, h = op.repair_mask(N, B, d, imp, kappa)
    D = op.dirty_set(N, d)
    H = op.nonlocal_set(imp, D, kappa)
    cand = [i for i in range(N) if i >= min(d, N)]
    assert len(H) == h == op.nonlocal_count(len(cand), kappa) and len(set(H)) == len(H)
    assert not set(H) & set(D)
    rest = [i for i in cand if i not in set(H)]
    if H and rest:
        assert min(imp[H]) >= max(imp[rest])  # H holds the best scores
    for b in range(len(mask)):
        covers = range(b * B, min(N, (b + 1) * B))
        assert mask[b] == int(any(i in set(D) or i in set(H) for i in covers))
    if kappa == 1.0:
        assert all(mask)


@pytest.mark.parametrize("seed", range(8))
def test_library_matches_oracle(seed):
    rng = np.random.default_rng(100 + seed)
    N = int(rng.integers(0, 5000))
    B = int(rng.choice([1, 8, 16, 32, 64, 1024]))
    d = int(rng.integers(0, N + 100))
    kappa = float(rng.choice([0.0, 0.015, 1 / 64, 0.2, 0.999, 1.0]))
    if seed % 2:
        imp = rng.lognormal(size=N).astype(np.float32)
    else:
        imp = rng.integers(0, 5, size=N).astype(np.float32)  # heavy ties
    mask, h = pb.pkv_plan_repair(N, B, d, imp, kappa)
    want, want_h = op.repair_mask(N, B, d, imp, kappa)
    assert mask.tolist() == want and h == want_h


def test_plan_repair_argument_errors():
    imp = np.ones(10, np.float32)
    m = np.zeros(4, np.uint8)
    ip, mp = imp.ctypes.data, m.ctypes.data
    for args in [(-1, 4, 0, ip, 0.1, mp), (10, 0, 0, ip, 0.1, mp), (10, 2000, 0, ip, 0.1, mp),
                 (10, 4, -1, ip, 0.1, mp), (10, 4, 0, ip, -0.1, mp), (10, 4, 0, ip, 1.5, mp),
                 (10, 4, 0, ip, float("nan"), mp), (10, 4, 0, None, 0.1, mp), (10, 4, 0, ip, 0.1, None)]:
        assert pb.pkv_plan_repair_status(*args) == pb.PKV_ERR_INVALID_ARGUMENT, args
    bad = imp.copy()
    bad[3] = np.nan
    assert pb.pkv_plan_repair_status(10, 4, 0, bad.ctypes.data, 0.1, mp) == pb.PKV_ERR_INVALID_ARGUMENT
    assert pb.pkv_plan_repair_status(0, 4, 0, None, 0.1, None) == pb.PKV_OK
