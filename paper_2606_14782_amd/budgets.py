"""Budget schedules of the backbone compression method.

BACON ranks the candidates of every (layer, KV head) under a budget K_{l,h}
that the backbone method allocates (Sec. 4, Preliminaries); BACON itself keeps
that allocation.  A uniform budget gives SnapKV's setting; `pyramid` gives a
per-layer schedule that shrinks with depth, the allocation PyramidKV uses.
The per-layer budgets are passed with each layer's call (the sequences stay
fixed for the prompt).
"""
from __future__ import annotations

import math


def uniform(budget: int, num_layers: int) -> list[int]:
    """The same budget at every layer."""
    if budget < 1 or num_layers < 1:
        raise ValueError("budget and num_layers must be >= 1")
    return [budget] * num_layers


def pyramid(mean_budget: int, num_layers: int, ratio: float = 0.25) -> list[int]:
    """Per-layer budgets decreasing linearly with depth.

    The first layer gets k0, the last ratio * k0, linear in between, and the
    budgets sum to num_layers * mean_budget exactly (largest-remainder
    rounding); each is at least 1.  ratio = 1 is the uniform schedule.
    """
    if mean_budget < 1 or num_layers < 1:
        raise ValueError("mean_budget and num_layers must be >= 1")
    if not 0.0 < ratio <= 1.0:
        raise ValueError("ratio must be in (0, 1]")
    total = mean_budget * num_layers
    if num_layers == 1:
        return [mean_budget]
    k0 = 2.0 * mean_budget / (1.0 + ratio)
    k1 = ratio * k0
    raw = [k0 + (k1 - k0) * l / (num_layers - 1) for l in range(num_layers)]
    raw = [max(1.0, x) for x in raw]
    scale = total / sum(raw)
    raw = [x * scale for x in raw]
    base = [max(1, math.floor(x)) for x in raw]
    rest = total - sum(base)
    # hand the remainder to the largest shortfalls raw - base (earlier layers
    # first on ties); layers raised to the floor of 1 have none
    order = sorted(range(num_layers), key=lambda l: (-(raw[l] - base[l]), l))
    i = 0
    while rest > 0:
        base[order[i % num_layers]] += 1
        rest -= 1
        i += 1
    while rest < 0:                       # only when flooring at 1 overshot
        l = max(range(num_layers), key=lambda j: (base[j], j))   # last of the largest
        base[l] -= 1
        rest += 1
    return base
