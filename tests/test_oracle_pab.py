"""Pins of the oracle's attention-output broadcasting (PAB) rollout.

The schedule is checked against a hand-derived table; the rollout against
properties fixed by its definition: range 1 never reuses, so it equals the
uncached rollout; and a branch whose output projection is zero outputs its
bias at every step, so reusing it must reproduce the uncached rollout
exactly, which fails if the reused value carries a stale gate, comes from
another block, or skips the projection bias.
"""
import json
import os

import numpy as np
import pytest

from oracle import rollout as R
from paper_2607_23159_amd import synth

GOLD = os.path.join(os.path.dirname(__file__), "golden", "pab_schedule.json")


def _schedule(T, kw, kc, r):
    have, out = False, []
    for k in range(1, T + 1):
        if R.pab_computes(k, T, kw, kc, r, have):
            out.append(k)
            have = True
    return out


def test_schedule_matches_hand_derived_table():
    cases = json.load(open(GOLD))["cases"]
    for c in cases:
        assert _schedule(c["T"], c["k_warm"], c["k_cool"], c["r"]) == c["computes"], c


def _wl(n_branch=1, init="stress"):
    return synth.make_workload("tiny", n_branch=n_branch, n_cand=1, init=init)


def _full(wl, W):
    fns = R.dit_velocity_fns(W, wl.model, wl.ctx[:wl.roll.n_branch])
    res = R.cached_rollout(wl.noise[:1], fns, [float(t) for t in wl.timesteps], tau=0.0,
                           k_warm=wl.roll.k_warm, k_cool=wl.roll.k_cool,
                           guidance=wl.roll.guidance, mode=R.CACHE_OFF)
    return res.latents


def _W(wl):
    return {k: v.astype(np.float64) for k, v in wl.named_weights().items()}


@pytest.mark.parametrize("nb", [1, 2])
def test_range_one_is_uncached_rollout(nb):
    wl = _wl(nb)
    W = _W(wl)
    lat, sched = R.pab_rollout(wl, r_self=1, r_cross=1, W=W)
    assert all(cs and cc for _, cs, cc in sched)
    np.testing.assert_array_equal(lat, _full(wl, W))


@pytest.mark.parametrize("branch", ["self", "cross"])
def test_zero_projection_reuse_is_exact(branch):
    wl = _wl(2)
    W = _W(wl)
    m = wl.model
    for j in range(m.n_blocks):
        key = f"blk{j}.o_w" if branch == "self" else f"blk{j}.cao_w"
        W[key] = np.zeros_like(W[key])
    # the gate must actually change over the steps for this pin to bite
    rs, rc = (2, 1) if branch == "self" else (1, 3)
    lat, sched = R.pab_rollout(wl, r_self=rs, r_cross=rc, W=W)
    reused = [k for k, cs, cc in sched if not (cs if branch == "self" else cc)]
    assert reused, "schedule never reused"
    np.testing.assert_allclose(lat, _full(wl, W), rtol=0, atol=1e-12)


def test_gate_varies_between_steps():
    """The zero-projection pin detects a stale gate only if the
    time-dependent self-attention gate differs between steps."""
    from oracle import dit
    wl = _wl(1)
    W = _W(wl)
    d = wl.model.hidden
    _, m1 = dit.time_embedding(float(wl.timesteps[2]), W, wl.model.freq_dim)
    _, m2 = dit.time_embedding(float(wl.timesteps[3]), W, wl.model.freq_dim)
    assert np.max(np.abs(m1.reshape(6, d)[2] - m2.reshape(6, d)[2])) > 1e-6


def test_planted_block_mixup_breaks_the_pin(monkeypatch):
    """Plant a mistake in the oracle (block j reuses block j+1's stored
    self-attention output) and check that the zero-projection pin fails."""
    from oracle import dit
    orig = dit.velocity

    def wrong(x, t, emb, W, cfg, last_block_rows=None, attn_io=None):
        if attn_io is not None:
            selfs = [io["self"] for io in attn_io]
            for j, io in enumerate(attn_io):
                io["self"] = selfs[(j + 1) % len(selfs)]
        return orig(x, t, emb, W, cfg, last_block_rows, attn_io)

    wl = _wl(1)
    W = _W(wl)
    for j in range(wl.model.n_blocks):
        W[f"blk{j}.o_w"] = np.zeros_like(W[f"blk{j}.o_w"])
    full = _full(wl, W)
    monkeypatch.setattr(dit, "velocity", wrong)
    lat, _ = R.pab_rollout(wl, r_self=2, r_cross=1, W=W)
    assert np.max(np.abs(lat - full)) > 1e-6


def test_reuse_changes_the_result():
    wl = _wl(1)
    W = _W(wl)
    lat, sched = R.pab_rollout(wl, r_self=2, r_cross=6, W=W)
    full = _full(wl, W)
    assert np.linalg.norm(lat - full) / np.linalg.norm(full) > 1e-6
    n_self = sum(cs for _, cs, _ in sched)
    n_cross = sum(cc for _, _, cc in sched)
    assert (n_self, n_cross) == (6, 3)  # T = 10, K_w = K_c = 1
