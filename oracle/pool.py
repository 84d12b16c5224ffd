"""Budget manager rotation: reference for the tests.

TEST INFRASTRUCTURE ONLY. Nothing in the library's product path may import,
call or execute this module; only the tests use it. It shares no code with
the HIP library.

What is computed (paper: paragraphs "Budget Manager" and "Pool rotation";
hyperparameter table: B = 20, R = 10, phi = 0.5, least-trained priority):
B of the N cartridges sit on the GPU at a time. After every R optimizer
steps, phi B of them go back to host memory and as many offloaded ones come
in, the ones trained least so far first. A cartridge off the GPU gets no
gradient while it is away.

Readings where the paper is silent: n = min(floor(phi B), N - B) cartridges
swap per rotation; the evicted ones are the active cartridges with the most
steps, the admitted ones the offloaded cartridges with the fewest (ties: the
lower id in both); the first active set is the B least-trained cartridges.
"""
from __future__ import annotations

import math
from typing import List, Sequence, Tuple


def swap_count(budget: int, phi: float, offloaded: int) -> int:
    return min(int(math.floor(phi * budget + 1e-9)), offloaded)


def plan_rotation(steps: Sequence[int], active: Sequence[bool], budget: int,
                  phi: float) -> Tuple[List[int], List[int]]:
    """(evict, admit) cartridge ids of one rotation."""
    act = [c for c in range(len(steps)) if active[c]]
    off = [c for c in range(len(steps)) if not active[c]]
    n = min(swap_count(budget, phi, len(off)), len(act))
    evict = sorted(act, key=lambda c: (-steps[c], c))[:n]
    admit = sorted(off, key=lambda c: (steps[c], c))[:n]
    return evict, admit


def first_active(steps: Sequence[int], budget: int) -> List[int]:
    return sorted(range(len(steps)), key=lambda c: (steps[c], c))[:budget]
