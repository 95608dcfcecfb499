"""Speedup reporting of the MEP loop (Sec. 4.1.4).

The paper scores a kernel by Speedup = t_baseline / t_optimized, with t the
average (here: the Eq. 3 trimmed mean) execution time, and counts only
optimizations that pass the functional-equivalence check in its averages.
These helpers apply that rule to the library's own candidate selection; they
only combine timings that the kernels produced.
"""
from __future__ import annotations

import math
from typing import Iterable, Optional, Sequence


def speedup(t_baseline: float, t_optimized: float) -> float:
    """Speedup = t_baseline / t_optimized (Sec. 4.1.4)."""
    if not (t_baseline > 0 and t_optimized > 0):
        raise ValueError("times must be positive")
    return t_baseline / t_optimized


def average_speedup(values: Iterable[Optional[float]]) -> float:
    """Arithmetic mean over the entries that passed FE.

    An entry that failed functional equivalence is None (the paper's 'Err');
    it is left out of the mean rather than counted as zero or one.  NaN when
    no entry passed."""
    kept = [float(v) for v in values if v is not None]
    return sum(kept) / len(kept) if kept else math.nan


def selection_speedup(results: Sequence, best: int) -> Optional[float]:
    """Standalone speedup of one round of candidate selection.

    ``results`` is the per-candidate list of (trimmed mean ms, FE error, FE
    passed) that ``mep_select_variant`` returns; candidate 0 is the baseline
    K^(d).  None when the chosen candidate or the baseline was not timed."""
    if best < 0 or best >= len(results):
        return None
    t0, t1 = results[0][0], results[best][0]
    if not results[best][2] or not (t0 > 0 and t1 > 0):
        return None
    return speedup(t0, t1)
