"""Plain oracle of the run-time DN selection (Eq. 11).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import or run anything in this package.

Section 4.4 (system monitoring and network selection): every DN is profiled
once for its cost (FLOPs), latency, memory footprint and accuracy, and the
values are kept as a look-up table.  At run time the device state gives an
allowed latency L_d, available memory M_d, a minimum accuracy A_min and a
power budget P_d (power read from a FLOPs-to-power table), and the DN chosen
is the one of least FLOPs that satisfies every constraint (Eq. 11).

Readings where the paper is silent: ties in FLOPs go to the lower mode index;
when no DN satisfies the constraints there is no answer (None); a missing
column (no accuracy or no power data) places no constraint.
"""
from __future__ import annotations

import math
from typing import Optional, Sequence


def select_dn(flops: Sequence[float], latency: Sequence[float], memory: Sequence[float],
              accuracy: Optional[Sequence[float]] = None,
              power: Optional[Sequence[float]] = None,
              L_d: float = math.inf, M_d: float = math.inf, A_min: float = -math.inf,
              P_d: float = math.inf) -> Optional[int]:
    """min over DNs of FLOPs(DN) s.t. Latency <= L_d, Memory <= M_d,
    Accuracy >= A_min (and Power <= P_d), as in Eq. 11."""
    feasible = []
    for k in range(len(flops)):
        ok = latency[k] <= L_d and memory[k] <= M_d
        if accuracy is not None:
            ok = ok and accuracy[k] >= A_min
        if power is not None:
            ok = ok and power[k] <= P_d
        if ok:
            feasible.append(k)
    if not feasible:
        return None
    best = feasible[0]
    for k in feasible[1:]:
        if flops[k] < flops[best]:
            best = k
    return best
