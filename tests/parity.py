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


def token_errors(a, b, pt=1, ph=2, pw=2):
    """Per-token error of latent ``a`` against ``b`` ([C][F][H][W]; a token
    is one pt x ph x pw patch over all channels): ||a_t - b_t|| divided by
    the RMS token norm of b.  The RMS of these values is the relative L2
    error of the whole latent, so an error confined to a few tokens shows
    here at full size instead of diluted by the token count."""
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    C, F, H, W = b.shape
    def tok(x):
        x = x.reshape(C, F // pt, pt, H // ph, ph, W // pw, pw)
        return x.transpose(1, 3, 5, 0, 2, 4, 6).reshape((F // pt) * (H // ph) * (W // pw), -1)
    ta, tb = tok(a), tok(b)
    rms = math.sqrt(float(np.mean(np.sum(tb * tb, axis=1))))
    return np.linalg.norm(ta - tb, axis=1) / max(rms, 1e-300)


def row_errors(a, b):
    """Per-row version of :func:`token_errors` for [rows][features] arrays
    (sampled tokens of a patchified latent)."""
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    rms = math.sqrt(float(np.mean(np.sum(b * b, axis=1))))
    return np.linalg.norm(a - b, axis=1) / max(rms, 1e-300)


def order_desc(s):
    """Candidates by decreasing score, equal scores lower index first."""
    return sorted(range(len(s)), key=lambda i: (-float(s[i]), i))


def discordant_pairs(order_ref, order_gpu):
    """Pairs (x, y) that the reference ranks x above y and the GPU ranks y
    above x."""
    pos = {c: i for i, c in enumerate(order_gpu)}
    out = []
    for i in range(len(order_ref)):
        for j in range(i + 1, len(order_ref)):
            x, y = order_ref[i], order_ref[j]
            if pos[x] > pos[y]:
                out.append((x, y))
    return out


def check_ranking(s_gpu, s_ref, gap_tol, excused_cands=()):
    """Rankings must match exactly.  A swapped pair is excused only if one
    of its two candidates had an excused schedule flip, or the oracle's
    score gap between the two is within ``gap_tol`` (4x the score error
    measured on the replayed schedule).  Returns the discordant pairs."""
    s_gpu = np.asarray(s_gpu, np.float64)
    s_ref = np.asarray(s_ref, np.float64)
    pairs = discordant_pairs(order_desc(s_ref), order_desc(s_gpu))
    bad = [(x, y, float(abs(s_ref[x] - s_ref[y]))) for x, y in pairs
           if x not in excused_cands and y not in excused_cands and abs(s_ref[x] - s_ref[y]) > gap_tol]
    assert not bad, (f"unexcused ranking swaps (x, y, oracle gap) {bad}; gap tolerance {gap_tol:.3e}; "
                     f"oracle order {order_desc(s_ref)}, gpu order {order_desc(s_gpu)}")
    return pairs
