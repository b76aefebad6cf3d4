"""Comparison helpers for the GPU-vs-oracle parity tests.

Bars (from the method's tolerance statement): schedules and rankings match
exactly, except a decision whose oracle indicator lies within 1e-3 relative
of tau (an excused flip; that stream is then compared in replay mode);
final latents within relative L2 2e-2 for the bf16 path and 1e-4 for the
fp32 path."""
import math

import numpy as np

TOL = {0: 2e-2, 1: 1e-4}       # dtype -> relative L2 bound on latents
EXCUSE = 1e-3


def rel_l2(a, b):
    a = np.asarray(a, np.float64).ravel()
    b = np.asarray(b, np.float64).ravel()
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def oracle_masks(res, n_cand, n_branch, T):
    m = np.zeros((T, n_cand * n_branch), np.uint8)
    a = np.full((T, n_cand * n_branch), np.nan)
    for r in res.log:
        m[r.k - 1, r.i * n_branch + r.b] = 1 if r.compute else 0
        if r.a is not None:
            a[r.k - 1, r.i * n_branch + r.b] = r.a
    return m, a


def compare_schedules(gpu_masks, ora_masks, ora_a, tau):
    """Returns (excused_streams, report); raises AssertionError on an
    unexcused decision mismatch."""
    T, S = ora_masks.shape
    excused = {}
    for s in range(S):
        for k in range(T):
            if gpu_masks[k, s] != ora_masks[k, s]:
                a = ora_a[k, s]
                gap = abs(a - tau) / tau if (tau > 0 and math.isfinite(tau) and not math.isnan(a)) else math.inf
                assert gap <= EXCUSE, (
                    f"schedule mismatch stream {s} step {k + 1}: gpu {gpu_masks[k, s]} oracle "
                    f"{ora_masks[k, s]}, oracle a={a!r}, |a-tau|/tau={gap:.3e} > {EXCUSE}")
                excused[s] = (k + 1, gap)
                break
    return excused
