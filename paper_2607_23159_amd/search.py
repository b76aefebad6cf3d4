"""CachedSearch driver over the C ABI (Alg. 1 of the paper).

Exploration runs N cached rollouts G_tau(c, s_i) as one batched rollout,
scores the final latents and ranks them; the full-compute reference is the
same call with the cache off.  Commit regenerates the winning seed at full
compute.  This module only sequences library calls and moves buffers; all
arithmetic runs in the library's kernels.
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional

import numpy as np
import torch

from . import binding as B
from .synth import CACHE_OFF, Workload


def _dev(a: np.ndarray, device: str = "cuda") -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(device)


class GpuModel:
    """A model handle whose weights were uploaded from a flat float32 array."""

    def __init__(self, cfg, weights: np.ndarray, dtype: Optional[int] = None, stream=None):
        self.cfg = cfg
        self.desc = B.model_desc(cfg, dtype)
        n = B.cs_model_weight_count(self.desc)
        if n != weights.size:
            raise ValueError(f"weight array has {weights.size} values, model needs {n}")
        w = _dev(weights)
        self.stream = stream
        self.h = B.cs_model_init(self.desc, w, n, stream)
        del w
        torch.cuda.synchronize()

    def velocity(self, x: torch.Tensor, t: float, ctx: torch.Tensor) -> torch.Tensor:
        v = torch.empty_like(x)
        B.cs_velocity(self.h, x, x.shape[0], t, ctx, v)
        torch.cuda.synchronize()
        return v

    def close(self):
        if self.h:
            B.cs_model_free(self.h)
            self.h = 0

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


@dataclasses.dataclass
class GpuRollout:
    latents: np.ndarray            # [N][C][F][H][W] float32
    masks: np.ndarray              # [T][S] uint8 (1 = computed)
    a: np.ndarray                  # [T][S] float64 (NaN = forced)
    scores: Optional[np.ndarray]   # [N] float64
    computed: int
    calls: int
    self_reused: int = 0           # PAB: calls that reused stored attention outputs
    cross_reused: int = 0

    def schedule(self, i: int, b: int, n_branch: int) -> List[bool]:
        return [bool(m) for m in self.masks[:, i * n_branch + b]]


def decision_records(masks: np.ndarray, a: np.ndarray, n_branch: int, computed_by: str = "rule"):
    """Per-call decision records of a rollout from its [T][S] masks and
    indicator values (S = N * n_branch, stream s = candidate s // n_branch,
    branch s % n_branch): step k (1-based), candidate i, branch b, the
    indicator a compared with tau at that call (None where the call was
    forced), and the decision ("compute" or "skip")."""
    T, S = masks.shape
    out = []
    for k in range(T):
        for st in range(S):
            av = float(a[k, st])
            out.append({"k": k + 1, "i": st // n_branch, "b": st % n_branch,
                        "a": None if np.isnan(av) else av,
                        "decision": "compute" if masks[k, st] else "skip"})
    return out


def write_decision_log(path: str, masks: np.ndarray, a: np.ndarray, n_branch: int) -> int:
    """Write the decision records as JSON lines; returns the record count."""
    import json
    recs = decision_records(masks, a, n_branch)
    with open(path, "w") as f:
        for r in recs:
            f.write(json.dumps(r) + "\n")
    return len(recs)


class Inputs:
    """Device copies of a workload's per-rollout inputs."""

    def __init__(self, wl: Workload):
        self.x1 = _dev(wl.noise.reshape(wl.noise.shape[0], -1))
        self.ctx = [_dev(c) for c in wl.ctx]
        self.w = _dev(wl.scorer)


def run_rollout(model: GpuModel, wl: Workload, inputs: Optional[Inputs] = None, *,
                tau: Optional[float] = None, mode: Optional[int] = None,
                n_cand: Optional[int] = None, override: Optional[np.ndarray] = None,
                record: bool = True, score: bool = True, pab_self: Optional[int] = None,
                pab_cross: Optional[int] = None) -> GpuRollout:
    """One batched rollout of the first ``n_cand`` seeds of the workload.

    ``override`` [T][S] replays a given schedule (1 = compute)."""
    inp = inputs or Inputs(wl)
    r = wl.roll
    n = r.n_cand if n_cand is None else n_cand
    kw = {"n_cand": n}
    if tau is not None:
        kw["tau"] = tau
    if mode is not None:
        kw["mode"] = mode
    if pab_self is not None:
        kw["pab_self"] = pab_self
    if pab_cross is not None:
        kw["pab_cross"] = pab_cross
    desc = B.RolloutDesc(r, wl.timesteps, **kw)
    S = n * r.n_branch
    x1 = inp.x1[:n]
    h = B.cs_rollout_init(model.h, desc, x1, inp.ctx[0], inp.ctx[1] if r.n_branch == 2 else None)
    try:
        T = r.n_steps
        masks = np.zeros((T, S), np.uint8)
        avals = np.full((T, S), np.nan)
        for k in range(1, T + 1):
            if record or override is not None:
                ovr = None if override is None else override[k - 1]
                m, a = B.cs_cache_decide(h, k, S, ovr)
                masks[k - 1], avals[k - 1] = m, a
            B.cs_denoise_step(h, k)
        lat = torch.empty_like(x1)
        B.cs_rollout_latents(h, lat)
        scores = B.cs_score(h, inp.w, n) if score else None
        st = B.cs_rollout_stats(h)
        torch.cuda.synchronize()
        return GpuRollout(lat.cpu().numpy().reshape((n,) + wl.noise.shape[1:]), masks, avals, scores,
                          int(st.computed), int(st.calls), int(st.self_reused), int(st.cross_reused))
    finally:
        B.cs_rollout_free(h)


@dataclasses.dataclass
class SearchResult:
    winner: int
    order_cached: List[int]
    order_full: Optional[List[int]]
    rho: Optional[float]
    top1: Optional[int]
    cached: GpuRollout
    full: Optional[GpuRollout]
    delivered: np.ndarray


def cached_search(model: GpuModel, wl: Workload, *, tau: Optional[float] = None,
                  mode: str = "keep", with_reference: bool = True) -> SearchResult:
    """Alg. 1: explore N cached rollouts, rank, keep the cached winner or
    commit (regenerate the winning seed with the cache off).  With
    ``with_reference`` the full rollouts of the same seeds are also run and
    the cached ranking is compared with theirs."""
    inp = Inputs(wl)
    cached = run_rollout(model, wl, inp, tau=tau)
    full = run_rollout(model, wl, inp, mode=CACHE_OFF) if with_reference else None
    if full is not None:
        oc, of, rho, top1 = B.cs_rank(cached.scores, full.scores)
    else:
        oc, of, rho, top1 = B.cs_rank(cached.scores, None)
    win = oc[0]
    if mode == "commit":
        one = Workload(wl.name, wl.model, dataclasses.replace(wl.roll, n_cand=1), wl.weights, wl.ctx,
                       wl.noise[win:win + 1], wl.scorer, wl.timesteps)
        delivered = run_rollout(model, one, mode=CACHE_OFF).latents[0]
    else:
        delivered = cached.latents[win]
    return SearchResult(win, oc, of, rho, top1, cached, full, delivered)


@dataclasses.dataclass
class PrunedResult:
    kept: List[int]                # surviving candidates (original indices)
    preview_scores: np.ndarray     # [N] scores of the x0 estimates at prune_step
    final_scores: np.ndarray       # [len(kept)]
    winner: int                    # original index
    latents: np.ndarray            # [len(kept)][...] cached latents of the survivors
    delivered: np.ndarray          # committed (full-compute) or kept latent of the winner
    computed: int
    calls: int


def pruned_search(model: GpuModel, wl: Workload, *, prune_step: int, keep: int,
                  tau: Optional[float] = None, mode: str = "commit") -> PrunedResult:
    """Pruned composition (Sec. Composition with pruned search): run all N
    candidates cached to ``prune_step``, score the x0 estimate, continue only
    the ``keep`` best (cache state intact), rank them on their final latents,
    then commit (regenerate the winner at full compute) or keep the draft."""
    inp = Inputs(wl)
    r = wl.roll
    N, T = r.n_cand, r.n_steps
    if not (1 <= prune_step < T and 1 <= keep <= N):
        raise ValueError("need 1 <= prune_step < n_steps and 1 <= keep <= n_cand")
    desc = B.RolloutDesc(r, wl.timesteps, **({} if tau is None else {"tau": tau}))
    h = B.cs_rollout_init(model.h, desc, inp.x1, inp.ctx[0], inp.ctx[1] if r.n_branch == 2 else None)
    try:
        B.cs_rollout_enable_preview(h, True)
        for k in range(1, prune_step + 1):
            B.cs_denoise_step(h, k)
        prev = B.cs_preview_score(h, inp.w, N)
        order, _, _, _ = B.cs_rank(prev, None)
        kept = sorted(order[:keep])       # retain takes increasing indices
        B.cs_rollout_retain(h, kept)
        B.cs_rollout_enable_preview(h, False)
        for k in range(prune_step + 1, T + 1):
            B.cs_denoise_step(h, k)
        final = B.cs_score(h, inp.w, keep)
        lat = torch.empty_like(inp.x1[:keep])
        B.cs_rollout_latents(h, lat)
        st = B.cs_rollout_stats(h)
        torch.cuda.synchronize()
        lat_np = lat.cpu().numpy().reshape((keep,) + wl.noise.shape[1:])
    finally:
        B.cs_rollout_free(h)
    j = B.cs_rank(final, None)[0][0]
    win = kept[j]
    if mode == "commit":
        one = Workload(wl.name, wl.model, dataclasses.replace(r, n_cand=1), wl.weights, wl.ctx,
                       wl.noise[win:win + 1], wl.scorer, wl.timesteps)
        delivered = run_rollout(model, one, mode=CACHE_OFF).latents[0]
    else:
        delivered = lat_np[j]
    return PrunedResult(kept, prev, final, win, lat_np, delivered, int(st.computed), int(st.calls))
