"""Per-layer cache budgets that decrease with depth at a fixed total (section 3.1: the runs use the
PyramidKV allocation, whose budgets fall with depth while the total stays that of a uniform
budget B per layer).

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper does not print the schedule.  Reading (R26), after PyramidKV's arithmetic sequence:
  B_min = max(1, floor(B / beta)),  B_max = 2 B - B_min,
  b(l)  = B_max - l (B_max - B_min) / (n_layers - 1)       (exact rational; b = B for one layer)
and the integer budget rounds b(l) away from B (up above B, down below it).  b(l) + b(n-1-l) = 2 B,
so the rounded pair still sums to 2 B and the total is exactly n_layers * B.

Parity unpinned: the schedule is a reading (R26); the tests pin this function to its own
arithmetic (a hand-worked case, the exact total, monotone decrease, symmetry), not to the paper.
"""
from __future__ import annotations

import math
from fractions import Fraction
from typing import List


def pyramid_budgets(budget: int, n_layers: int, beta: float) -> List[int]:
    if budget < 1 or n_layers < 1 or not beta >= 1.0:
        raise ValueError("budget >= 1, n_layers >= 1 and beta >= 1 are required")
    if n_layers == 1:
        return [budget]
    b_min = max(1, math.floor(budget / beta))
    b_max = 2 * budget - b_min
    out = []
    for layer in range(n_layers):
        b = Fraction(b_max) - Fraction(layer * (b_max - b_min), n_layers - 1)
        out.append(math.ceil(b) if b >= budget else math.floor(b))
    return out
