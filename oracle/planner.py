"""CPU oracle of PatchKV's resume planner.  TEST INFRASTRUCTURE ONLY.

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
import this module.  It states in plain Python what the planner computes at
resume time (PatchKV Section IV-B, Eq. 9, 11 and 12), for one request whose
aligned suffix ``S`` has ``N`` tokens (token ``i`` of ``S`` lies ``i`` tokens
past the edit) split into blocks of ``B`` tokens:

1. the online dirty set (Eq. 9): ``D = {i in S : i < min(d_hat, N)}``, with
   ``d_hat`` the length model's prediction (an input here);
2. the nonlocal set (Eq. 11): ``H`` = the ``k`` tokens of ``S \\ D`` with the
   highest stored importance ``I_i(0)``, ``k = floor(kappa * |S \\ D| + 1/2)``
   (in double precision), ties going to the smaller index;
3. block rounding (Eq. 12): ``R`` = the blocks that contain a token of
   ``D u H``; ``F`` = every other block.

The count ``k`` and the tie rule are readings: the paper names a top-kappa
fraction without fixing its rounding or ties.
"""
from __future__ import annotations

import math
from typing import List, Sequence, Tuple


def dirty_set(N: int, d_hat: int) -> List[int]:
    """Eq. 9."""
    return list(range(min(d_hat, N)))


def nonlocal_count(candidates: int, kappa: float) -> int:
    return min(max(int(math.floor(kappa * candidates + 0.5)), 0), candidates)


def nonlocal_set(importance: Sequence[float], dirty: Sequence[int], kappa: float) -> List[int]:
    """Eq. 11: top fraction kappa of the candidates outside D by importance."""
    in_d = set(dirty)
    cand = [i for i in range(len(importance)) if i not in in_d]
    k = nonlocal_count(len(cand), kappa)
    ranked = sorted(cand, key=lambda i: (-float(importance[i]), i))
    return ranked[:k]


def block_round(tokens: Sequence[int], N: int, B: int) -> List[int]:
    """BlockRound_S(A): the blocks of S meeting the token set A."""
    nb = -(-N // B)
    return sorted({i // B for i in tokens if 0 <= i < N and i // B < nb})


def repair_mask(N: int, B: int, d_hat: int, importance: Sequence[float], kappa: float) -> Tuple[List[int], int]:
    """Eq. 12: (mask over the blocks of S, 1 = in R), and |H|."""
    D = dirty_set(N, d_hat)
    H = nonlocal_set(importance, D, kappa)
    R = set(block_round(list(D) + list(H), N, B))
    return [1 if b in R else 0 for b in range(-(-N // B))], len(H)
