"""Oracle: cached rollout G_tau(c, s), scorer and CachedSearch exploration.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Follows the paper step by step, in float64:

* Euler step of the probability-flow ODE on the decreasing grid
  t_1 = 1 > ... > t_{T+1} = 0 (Sec. Preliminaries, Eq. euler);
* classifier-free guidance v_u + w (v_c - v_u) (Eq. cfg), one transformer
  call per guidance branch;
* the transformation-vector cache (Sec. Adaptive transformation-vector
  caching): a computed call stores Delta = v(x_ref) - x_ref (Eq. delta) and
  x_ref; a skipped call returns x + Delta (Eq. skip);
* the accumulated drift indicator a += ||x - x_ref|| / ||x_ref|| (Eq.
  indicator): skip while a <= tau, otherwise compute, refresh Delta and
  x_ref and reset a to 0; the first K_w and last K_c steps, and any call
  before the first Delta exists, always compute;
* independent (Delta, x_ref, a) per guidance branch (Sec. per-branch cache
  state), reset at the start of every generation (Alg. 1);
* the static variant that computes every k-th step between warmup and
  cooldown (Sec. properties);
* the scorer, a fixed random projection s = <w, x_{T+1}> / sqrt(D), which
  stands in for the verifier V of Alg. 1.

Readings where the paper is silent:
  - steps are 1-based; steps 1..K_w and T-K_c+1..T are forced computes;
  - every computed call (forced or not) refreshes Delta, x_ref and resets a;
    a forced step does not add to a;
  - a call whose ||x_ref|| is 0 computes;
  - both branches receive the latent x_{t_k} of the current step;
  - static mode with period k computes a step s (K_w < s <= T-K_c) iff
    (s - K_w) is a multiple of k; other steps in that range reuse Delta;
  - attention-output broadcasting (PAB, one of the published engines of
    Sec. Ranking preservation across published caching methods and Table
    tab:baselines; self range 2, cross range 6):
    the cached quantity is each attention branch's output after its output
    projection and before the self-attention gate, per block, stream and
    branch; steps 1..K_w and T-K_c+1..T compute every attention; a step s
    in between recomputes a branch with range r iff (s - K_w) is a multiple
    of r (the phase of the static variant) or no output is stored yet, and
    otherwise reuses the stored output (multiplied by the current step's
    gate); every call of every step runs the rest of the transformer;
  - the sampler's internal x0 estimate after step k (used for the preview
    score of the pruned search, Sec. Composition with pruned search) is the
    rectified-flow extrapolation x0_hat = x_{t_{k+1}} - t_{k+1} * v~_k, which
    equals x_{t_k} - t_k * v~_k.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Callable, Dict, List, Optional, Sequence

import numpy as np

from . import dit

CACHE_OFF, CACHE_ADAPTIVE, CACHE_STATIC, CACHE_PAB = 0, 1, 2, 3


@dataclasses.dataclass
class StepRecord:
    """One cache decision: step k (1-based), candidate i, branch b,
    ``a`` = the indicator compared with tau (None on a forced step), and
    ``compute`` = whether the transformer was evaluated."""
    k: int
    i: int
    b: int
    a: Optional[float]
    compute: bool


@dataclasses.dataclass
class RolloutResult:
    latents: np.ndarray          # [N][C][F][H][W] float64, x_{T+1}
    log: List[StepRecord]
    n_compute: int
    n_calls: int
    x0_hat: Optional[np.ndarray] = None   # [N][...] x0 estimate after step `preview_step`

    def schedule(self, i: int, b: int) -> List[bool]:
        return [r.compute for r in self.log if r.i == i and r.b == b]

    def a_values(self, i: int, b: int) -> List[Optional[float]]:
        return [r.a for r in self.log if r.i == i and r.b == b]


def is_forced(k: int, T: int, k_warm: int, k_cool: int, has_ref: bool, mode: int) -> bool:
    return (mode == CACHE_OFF) or (k <= k_warm) or (k > T - k_cool) or (not has_ref)


def cached_rollout_one(x1: np.ndarray, velocity_fns: Sequence[Callable[[np.ndarray, float], np.ndarray]],
                       timesteps: Sequence[float], *, tau: float, k_warm: int, k_cool: int,
                       guidance: float, mode: int = CACHE_ADAPTIVE, static_k: int = 2,
                       cand: int = 0, log: Optional[List[StepRecord]] = None,
                       preview_step: Optional[int] = None, preview_out: Optional[list] = None) -> np.ndarray:
    """One candidate's rollout.  ``velocity_fns[b](x, t)`` is the transformer
    call of guidance branch b (b = 0 conditional, b = 1 unconditional).  With
    ``preview_step`` = k, the x0 estimate after step k is appended to
    ``preview_out``."""
    B = len(velocity_fns)
    T = len(timesteps) - 1
    x = dit.as64(x1).copy()
    # cache state per branch, reset at the start of the generation (Alg. 1)
    has_ref = [False] * B
    a = [0.0] * B
    xref: List[Optional[np.ndarray]] = [None] * B
    delta: List[Optional[np.ndarray]] = [None] * B
    for k in range(1, T + 1):
        t_k, t_next = float(timesteps[k - 1]), float(timesteps[k])
        v = [None] * B
        for b in range(B):
            forced = is_forced(k, T, k_warm, k_cool, has_ref[b], mode)
            compute = True
            a_seen: Optional[float] = None
            if not forced:
                if mode == CACHE_STATIC:
                    compute = ((k - k_warm) % static_k) == 0
                else:
                    num = math.sqrt(float(np.sum((x - xref[b]) ** 2)))
                    den = math.sqrt(float(np.sum(xref[b] ** 2)))
                    if den == 0.0:
                        compute = True
                    else:
                        a[b] += num / den
                        a_seen = a[b]
                        compute = not (a[b] <= tau)
            if compute:
                v[b] = dit.as64(velocity_fns[b](x, t_k))
                delta[b] = v[b] - x
                xref[b] = x.copy()
                a[b] = 0.0
                has_ref[b] = True
            else:
                v[b] = x + delta[b]
            if log is not None:
                log.append(StepRecord(k, cand, b, a_seen, compute))
        vt = v[0] if B == 1 else v[1] + guidance * (v[0] - v[1])
        x = x + (t_next - t_k) * vt
        if preview_step is not None and k == preview_step and preview_out is not None:
            preview_out.append(x - t_next * vt)
    return x


def pab_computes(k: int, T: int, k_warm: int, k_cool: int, r: int, have: bool) -> bool:
    """Whether step k recomputes an attention branch of broadcast range r."""
    if k <= k_warm or k > T - k_cool or not have:
        return True
    return (k - k_warm) % r == 0


def pab_rollout_one(x1: np.ndarray, W: Dict[str, np.ndarray], cfg, embs: Sequence[np.ndarray],
                    timesteps: Sequence[float], *, r_self: int, r_cross: int, k_warm: int,
                    k_cool: int, guidance: float, sched: Optional[list] = None) -> np.ndarray:
    """One candidate's rollout with attention-output broadcasting: every
    step evaluates the transformer for every guidance branch (Eq. cfg, Eq.
    euler), reusing each block's stored attention outputs on the steps the
    schedule marks.  ``sched`` collects (k, self computed, cross computed)."""
    B = len(embs)
    T = len(timesteps) - 1
    x = dit.as64(x1).copy()
    stored = [[{"self": None, "cross": None} for _ in range(cfg.n_blocks)] for _ in range(B)]
    for k in range(1, T + 1):
        t_k, t_next = float(timesteps[k - 1]), float(timesteps[k])
        cs = pab_computes(k, T, k_warm, k_cool, r_self, stored[0][0]["self"] is not None)
        cc = pab_computes(k, T, k_warm, k_cool, r_cross, stored[0][0]["cross"] is not None)
        if sched is not None:
            sched.append((k, cs, cc))
        v = []
        for b in range(B):
            io = [{"self": None if cs else stored[b][j]["self"],
                   "cross": None if cc else stored[b][j]["cross"]} for j in range(cfg.n_blocks)]
            v.append(dit.as64(dit.velocity(x, t_k, embs[b], W, cfg, attn_io=io)))
            for j in range(cfg.n_blocks):
                stored[b][j]["self"] = io[j]["self_out"]
                stored[b][j]["cross"] = io[j]["cross_out"]
        vt = v[0] if B == 1 else v[1] + guidance * (v[0] - v[1])
        x = x + (t_next - t_k) * vt
    return x


def pab_rollout(wl, *, n_cand: Optional[int] = None, r_self: Optional[int] = None,
                r_cross: Optional[int] = None, W: Optional[Dict[str, np.ndarray]] = None):
    """Oracle PAB rollouts of a synthetic workload's first ``n_cand`` seeds.
    Returns (latents [N][...], schedule [(k, self computed, cross computed)])."""
    r = wl.roll
    if W is None:
        W = {k: v.astype(np.float64) for k, v in wl.named_weights().items()}
    embs = [dit.text_embedding(c, W) for c in wl.ctx[:r.n_branch]]
    x1 = wl.noise if n_cand is None else wl.noise[:n_cand]
    outs, sched = [], []
    for i in range(x1.shape[0]):
        outs.append(pab_rollout_one(x1[i], W, wl.model, embs, [float(t) for t in wl.timesteps],
                                    r_self=r.pab_self if r_self is None else r_self,
                                    r_cross=r.pab_cross if r_cross is None else r_cross,
                                    k_warm=r.k_warm, k_cool=r.k_cool, guidance=r.guidance,
                                    sched=sched if i == 0 else None))
    return np.stack(outs), sched


def dit_velocity_fns(W: Dict[str, np.ndarray], cfg, ctx: Sequence[np.ndarray]):
    """Transformer calls per guidance branch; the text embedding of each
    branch's context is computed once per rollout (it depends on c only)."""
    embs = [dit.text_embedding(c, W) for c in ctx]
    return [(lambda x, t, e=e: dit.velocity(x, t, e, W, cfg)) for e in embs]


def cached_rollout(x1: np.ndarray, velocity_fns, timesteps, *, tau: float, k_warm: int,
                   k_cool: int, guidance: float = 5.0, mode: int = CACHE_ADAPTIVE,
                   static_k: int = 2, preview_step: Optional[int] = None) -> RolloutResult:
    """N independent candidate rollouts, x1 [N][...]."""
    log: List[StepRecord] = []
    outs = []
    prev: list = []
    for i in range(x1.shape[0]):
        outs.append(cached_rollout_one(x1[i], velocity_fns, timesteps, tau=tau, k_warm=k_warm,
                                       k_cool=k_cool, guidance=guidance, mode=mode,
                                       static_k=static_k, cand=i, log=log,
                                       preview_step=preview_step, preview_out=prev))
    n_comp = sum(1 for r in log if r.compute)
    return RolloutResult(np.stack(outs), log, n_comp, len(log),
                         np.stack(prev) if prev else None)


def score(latents: np.ndarray, w: np.ndarray) -> np.ndarray:
    """s_i = <w, x_i> / sqrt(D) for every candidate (float64)."""
    X = dit.as64(latents).reshape(latents.shape[0], -1)
    D = X.shape[1]
    return (X @ dit.as64(w)) / math.sqrt(D)


def run_workload(wl, *, tau: Optional[float] = None, mode: Optional[int] = None,
                 n_cand: Optional[int] = None, preview_step: Optional[int] = None) -> RolloutResult:
    """Oracle rollout of a synthetic workload (see ``synth.make_workload``)."""
    from_cfg = wl.roll
    W = {k: v.astype(np.float64) for k, v in wl.named_weights().items()}
    fns = dit_velocity_fns(W, wl.model, wl.ctx[:from_cfg.n_branch])
    x1 = wl.noise if n_cand is None else wl.noise[:n_cand]
    return cached_rollout(x1, fns, [float(t) for t in wl.timesteps],
                          tau=from_cfg.tau if tau is None else tau,
                          k_warm=from_cfg.k_warm, k_cool=from_cfg.k_cool,
                          guidance=from_cfg.guidance,
                          mode=from_cfg.mode if mode is None else mode,
                          static_k=from_cfg.static_k, preview_step=preview_step)


def pruned_search(wl, *, prune_step: int, keep: int, tau: Optional[float] = None):
    """Pruned composition (Sec. Composition with pruned search): all
    candidates run cached to ``prune_step``, are scored on their x0 estimate,
    the ``keep`` best continue to the end.  Candidates are independent, so the
    survivors' trajectories are those of the unpruned cached rollout.
    Returns (kept indices in candidate order, preview scores, final scores of
    the kept candidates, winner index)."""
    res = run_workload(wl, tau=tau, preview_step=prune_step)
    prev = score(res.x0_hat, wl.scorer)
    order = sorted(range(len(prev)), key=lambda i: (-prev[i], i))
    kept = sorted(order[:keep])
    final = score(res.latents[kept], wl.scorer)
    winner = kept[sorted(range(len(kept)), key=lambda j: (-final[j], j))[0]]
    return kept, prev, final, winner, res

