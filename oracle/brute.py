"""Scalar brute-force attention over Python floats -- TEST INFRASTRUCTURE ONLY.

Eq. (1) written out element by element with ``math.exp``: no NumPy, no vectorisation, so it shares
no arithmetic routine with the other two oracle routes. Meant for Sq, Sk <= 4.
"""

from __future__ import annotations

import math
from typing import List, Sequence, Tuple


def brute_attention(q: Sequence[Sequence[float]], k: Sequence[Sequence[float]],
                    v: Sequence[Sequence[float]], scale: float, causal: bool
                    ) -> Tuple[List[List[float]], List[float]]:
    """One head; returns (O as a list of rows, LSE list). Causal alignment is bottom-right."""
    sq, sk = len(q), len(k)
    dv = len(v[0]) if sk else 0
    out, lses = [], []
    for i in range(sq):
        scores = []
        for j in range(sk):
            if causal and j > i + (sk - sq):
                continue
            dot = 0.0
            for a, b in zip(q[i], k[j]):
                dot += float(a) * float(b)
            scores.append((j, scale * dot))
        if not scores:
            out.append([0.0] * dv)
            lses.append(-math.inf)
            continue
        mx = max(sc for _, sc in scores)
        weights = [(j, math.exp(sc - mx)) for j, sc in scores]
        total = sum(w for _, w in weights)
        row = []
        for c in range(dv):
            acc = 0.0
            for j, w in weights:
                acc += w * float(v[j][c])
            row.append(acc / total)
        out.append(row)
        lses.append(mx + math.log(total))
    return out, lses
