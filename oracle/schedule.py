"""One-forward-one-backward pipeline order (test infrastructure only).

Section 3.1 of the paper: each GPU issues forward and backward tasks in a
round-robin way, several mini-batches are in flight, and every backward task
produces one weight update (so a time unit is one F/B pair and W_t is the
version after t updates).

The oracle places tasks on a grid of half time units with every hop between
neighbouring stages taking one half unit: mini-batch m enters stage 0 at 2m,
so its forward at stage k runs at 2m + k, its loss is reached after stage
N-1 at 2m + N, and its backward at stage k runs at 2m + N + (N - 1 - k).
A stage therefore starts with N - k forwards, then alternates backward and
forward, then drains its remaining backwards.
"""
from typing import List, Tuple


def forward_time(k: int, N: int, m: int) -> int:
    return 2 * m + k


def backward_time(k: int, N: int, m: int) -> int:
    return 2 * m + N + (N - 1 - k)


def stage_tasks(k: int, N: int, M: int) -> List[Tuple[str, int]]:
    """Task order ('F'|'B', mini-batch) of stage k for M mini-batches."""
    ev = [(forward_time(k, N, m), "F", m) for m in range(M)]
    ev += [(backward_time(k, N, m), "B", m) for m in range(M)]
    ev.sort()
    return [(kind, m) for _, kind, m in ev]


def pipeline_tasks(N: int, M: int) -> List[Tuple[int, str, int]]:
    """All stages' tasks (stage, 'F'|'B', mini-batch) in half-unit time order;
    tasks of different stages in the same half unit are independent and are
    listed by stage index."""
    ev = []
    for k in range(N):
        ev += [(forward_time(k, N, m), k, "F", m) for m in range(M)]
        ev += [(backward_time(k, N, m), k, "B", m) for m in range(M)]
    ev.sort()
    return [(k, kind, m) for _, k, kind, m in ev]
