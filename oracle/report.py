"""Reporting formulas of Sec. 3.2 and Sec. 5.1.

Eq. L-and-speedup: L = E_i[l_i + 1] lies in [1, K+1].  Sec. 5.1 evaluates the
theoretical speedup as S = L / (1 + c) with c = C_D / C_T the per-iteration
draft-to-target cost ratio, and the throughput column of the main table as the
34 tok/s target-only rate times S.
"""
from typing import Sequence


def mean_accepted_length(accept_lengths: Sequence[int]) -> float:
    """L = mean of (l_i + 1) over iterations."""
    return sum(int(l) + 1 for l in accept_lengths) / len(accept_lengths)


def theoretical_speedup(L: float, c: float) -> float:
    """S = L / (1 + c)."""
    return L / (1.0 + c)


def iid_expected_L(p: float, K: int) -> float:
    """E[l+1] when each draft token independently matches with probability p:
    sum_{j=0..K} p^j, the closed form (1 - p^(K+1)) / (1 - p) for p < 1."""
    return sum(p ** j for j in range(K + 1))
