"""Oracle: candidate ranking and Spearman correlation.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Alg. 1 picks i* = argmax_i r_i over the verifier scores.  Ranking fidelity
is measured per prompt as the Spearman correlation between the cached
scores S^_i and the full-compute scores S_i over matched seeds, together
with top-1 agreement and regret max_i S_i - S_{argmax S^} (Sec.
Experiments, definitions and protocol).

Readings: ties in the ordering go to the lower candidate index; Spearman
uses average ranks for ties and is the Pearson correlation of the two rank
vectors; it is undefined (NaN) for fewer than two candidates or a constant
score vector.
"""
from __future__ import annotations

import math
from typing import List, Sequence, Tuple


def order_desc(s: Sequence[float]) -> List[int]:
    """Candidate indices by decreasing score; equal scores keep index order."""
    return sorted(range(len(s)), key=lambda i: (-float(s[i]), i))


def average_ranks(s: Sequence[float]) -> List[float]:
    """1-based ranks in increasing score; tied values share the mean rank."""
    n = len(s)
    idx = sorted(range(n), key=lambda i: float(s[i]))
    ranks = [0.0] * n
    pos = 0
    while pos < n:
        end = pos
        while end + 1 < n and float(s[idx[end + 1]]) == float(s[idx[pos]]):
            end += 1
        mean_rank = (pos + end) / 2.0 + 1.0
        for q in range(pos, end + 1):
            ranks[idx[q]] = mean_rank
        pos = end + 1
    return ranks


def pearson(x: Sequence[float], y: Sequence[float]) -> float:
    n = len(x)
    if n < 2:
        return float("nan")
    mx = sum(x) / n
    my = sum(y) / n
    sxy = sum((a - mx) * (b - my) for a, b in zip(x, y))
    sxx = sum((a - mx) ** 2 for a in x)
    syy = sum((b - my) ** 2 for b in y)
    if sxx == 0.0 or syy == 0.0:
        return float("nan")
    return sxy / math.sqrt(sxx * syy)


def spearman(a: Sequence[float], b: Sequence[float]) -> float:
    return pearson(average_ranks(a), average_ranks(b))


def argmax_first(s: Sequence[float]) -> int:
    return order_desc(s)[0]


def rank_report(s_cached: Sequence[float], s_full: Sequence[float]) -> Tuple[List[int], List[int], float, int, float]:
    """(order_cached, order_full, rho, top1_agree, regret)."""
    oc, of = order_desc(s_cached), order_desc(s_full)
    rho = spearman(s_cached, s_full)
    top1 = int(oc[0] == of[0])
    regret = max(float(v) for v in s_full) - float(s_full[oc[0]])
    return oc, of, rho, top1, regret
