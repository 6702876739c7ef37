"""Startup cost table C(B, rho) and its lookup (App. C, cost-table profiling protocol).

Before serving, one verify step per captured batch size B_c and ratio bucket
rho runs on dummy inputs at the budget K_rho(B_c) of Eq. dcut-budget (the
budget forced alone), and the median step time over a few repetitions becomes
C(B_c, rho).  At decode time the selector reads the row of the captured batch
size nearest to the live batch (ties to the larger one) and passes
(K_rho(B), C(B_c, rho)) as the candidate budgets and costs of the selection
call.  The budgets and the nearest-batch rule are the library's host helpers;
the steps and the timer are supplied by the caller.
"""
from __future__ import annotations

import dataclasses
import json
import statistics
from typing import Callable, Dict, List, Sequence, Tuple

from . import lib as L

PAPER_RATIOS = ((1, 4), (1, 2), (3, 4), (1, 1))      # 25 %, 50 %, 75 %, 100 %


@dataclasses.dataclass
class CostTable:
    D: int
    ratios: List[Tuple[int, int]]       # ratio buckets as exact fractions num/den
    batch: List[int]                    # captured batch sizes, ascending
    ms: List[List[float]]               # ms[b][r]: median step time of K_{ratio r}(batch[b])

    def budgets(self, B: int) -> List[int]:
        """K_rho(B) for every bucket, in exact integer arithmetic."""
        return L.budgets_from_ratios(B, self.D, self.ratios)

    def row(self, B: int) -> Tuple[int, List[float]]:
        """The captured batch size nearest to B and its costs."""
        b = L.nearest_batch(B, self.batch)
        if b < 0:
            raise ValueError("empty cost table")
        return self.batch[b], list(self.ms[b])

    def candidates(self, B: int) -> Tuple[List[int], List[float]]:
        """Candidate budgets at the live batch B and the costs read at the nearest
        captured batch size, ready for the selection call."""
        return self.budgets(B), self.row(B)[1]

    def to_json(self) -> str:
        return json.dumps(dataclasses.asdict(self))

    @staticmethod
    def from_json(text: str) -> "CostTable":
        d = json.loads(text)
        return CostTable(d["D"], [tuple(r) for r in d["ratios"]], list(d["batch"]), d["ms"])


def profile(steps: Dict[int, Callable[[List[int]], None]], D: int,
            ratios: Sequence[Tuple[int, int]] = PAPER_RATIOS,
            time_ms: Callable[[Callable[[], None], int], List[float]] = None,
            reps: int = 10, warmup: int = 2) -> CostTable:
    """Profile C(B_c, rho) for every captured batch size (the keys of `steps`).

    steps[B_c](budgets) runs one whole verify step of batch B_c with the given
    candidate budgets (one budget forces it); time_ms(fn, n) runs fn n times
    and returns each run's time in ms."""
    if time_ms is None:
        raise ValueError("a timer is required")
    batch = sorted(steps)
    ms = []
    for Bc in batch:
        row = []
        for K in L.budgets_from_ratios(Bc, D, ratios):
            fn = lambda K=K: steps[Bc]([K])
            time_ms(fn, warmup)
            row.append(float(statistics.median(time_ms(fn, reps))))
        ms.append(row)
    return CostTable(D, [tuple(r) for r in ratios], batch, ms)


def event_timer(stream=None):
    """A time_ms for `profile`: device time of each run from HIP events on the stream."""
    import torch

    def time_ms(fn, n):
        s = torch.cuda.current_stream() if stream is None else stream
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n)]
        for a, b in evs:
            a.record(s)
            fn()
            b.record(s)
        torch.cuda.synchronize()
        return [a.elapsed_time(b) for a, b in evs]
    return time_ms
