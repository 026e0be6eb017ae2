"""Search-quality metrics as the paper defines them.

- speedup = time of the untransformed program / time of the tuned one
  (Sec. 4.2);
- sample efficiency = speedup / number of samples (Sec. 4.2);
- sample reduction = samples of the baseline search / samples of the new
  one, and efficiency gain = ratio of the two sample efficiencies (the
  derived columns of Table 1);
- averages over platform/operator pairs are geometric means (Table 1).
Best-so-far curves are formed per run (monotone by construction) before any
averaging across runs.
"""
from __future__ import annotations

import math
from typing import Iterable, List, Optional, Sequence


def speedup(t_untuned: float, t_tuned: float) -> float:
    return t_untuned / t_tuned


def sample_efficiency(speedup_value: float, samples: float) -> float:
    return speedup_value / samples


def sample_reduction(samples_baseline: float, samples_new: float) -> float:
    return samples_baseline / samples_new


def efficiency_gain(speedup_new: float, samples_new: float, speedup_base: float,
                    samples_base: float) -> float:
    return sample_efficiency(speedup_new, samples_new) / sample_efficiency(speedup_base, samples_base)


def geomean(xs: Iterable[float]) -> float:
    xs = list(xs)
    return math.exp(sum(math.log(x) for x in xs) / len(xs))


def best_so_far(values: Sequence[float]) -> List[float]:
    out, best = [], -math.inf
    for v in values:
        best = max(best, v)
        out.append(best)
    return out


def samples_to_reach(curve: Sequence[float], target: float) -> Optional[int]:
    """1-based number of samples after which the best-so-far reaches target."""
    for i, v in enumerate(curve):
        if v >= target:
            return i + 1
    return None


def mean_curve(curves: Sequence[Sequence[float]]) -> List[float]:
    """Average of per-run best-so-far curves, truncated to the shortest run."""
    n = min(len(c) for c in curves)
    return [sum(c[i] for c in curves) / len(curves) for i in range(n)]
