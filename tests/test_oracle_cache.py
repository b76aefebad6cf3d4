"""Pins of the oracle's cache rule, Euler/CFG update and scorer.

They check the oracle against things other than itself: a closed form
worked out by hand from the paper's equations (tests/golden), the
invariants the paper states for the method (tau = 0 reproduces the uncached
rollout exactly; forced warmup/cooldown windows), and algebraic identities.
"""
import json
import math
import os

import numpy as np
import pytest

from oracle import rollout as R
from paper_2607_23159_amd import synth

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _neg(x, t):
    return -x


def _grid(T):
    return [1.0 - k / T for k in range(T + 1)]


@pytest.mark.parametrize("case", json.load(open(os.path.join(GOLD, "cache_rule_closed_form.json")))["cases"])
def test_closed_form_cache_schedule(case):
    tau = math.inf if case["tau"] == "inf" else float(case["tau"])
    x1 = synth.make_latent_batch((3, 2, 4, 4), seed=7)
    res = R.cached_rollout(x1, [_neg], _grid(10), tau=tau, k_warm=1, k_cool=1, guidance=1.0)
    for i in range(3):
        sched = res.schedule(i, 0)
        got = [k + 1 for k, c in enumerate(sched) if c]
        assert got == case["computes"]
        for k, a in case.get("a_seen", {}).items():
            assert res.a_values(i, 0)[int(k) - 1] == pytest.approx(a, rel=1e-12)
    np.testing.assert_allclose(res.latents, case["scale"] * x1.astype(np.float64), rtol=1e-9)


def test_closed_form_off_mode_equals_tau0():
    x1 = synth.make_latent_batch((2, 2, 4, 4), seed=3)
    a = R.cached_rollout(x1, [_neg], _grid(10), tau=0.0, k_warm=1, k_cool=1, guidance=1.0)
    b = R.cached_rollout(x1, [_neg], _grid(10), tau=0.3, k_warm=1, k_cool=1, guidance=1.0,
                         mode=R.CACHE_OFF)
    assert a.n_compute == b.n_compute == 20
    assert np.array_equal(a.latents, b.latents)


def test_no_skip_before_first_delta():
    """K_w = 0: the first call still computes (no Delta exists yet)."""
    x1 = synth.make_latent_batch((1, 2, 4, 4), seed=5)
    res = R.cached_rollout(x1, [_neg], _grid(10), tau=math.inf, k_warm=0, k_cool=0, guidance=1.0)
    assert res.schedule(0, 0) == [True] + [False] * 9


def test_static_schedule():
    x1 = synth.make_latent_batch((1, 2, 4, 4), seed=5)
    res = R.cached_rollout(x1, [_neg], _grid(10), tau=0.0, k_warm=2, k_cool=2, guidance=1.0,
                           mode=R.CACHE_STATIC, static_k=3)
    # forced 1,2 and 9,10; in 3..8 computes where (k - 2) % 3 == 0 -> 5, 8
    got = [k + 1 for k, c in enumerate(res.schedule(0, 0)) if c]
    assert got == [1, 2, 5, 8, 9, 10]


def test_cfg_weight_one_is_conditional_only():
    """w = 1 turns Eq. cfg into the conditional velocity."""
    x1 = synth.make_latent_batch((2, 2, 4, 4), seed=11)
    cond = lambda x, t: -x + 0.3 * t
    unc = lambda x, t: 0.5 * x
    two = R.cached_rollout(x1, [cond, unc], _grid(10), tau=0.1, k_warm=1, k_cool=1, guidance=1.0)
    one = R.cached_rollout(x1, [cond], _grid(10), tau=0.1, k_warm=1, k_cool=1, guidance=1.0)
    np.testing.assert_allclose(two.latents, one.latents, rtol=1e-12, atol=1e-12)


def test_cfg_combination_closed_form():
    """Constant branch velocities: x_{T+1} = x_1 - (u + w (c - u)) (t_1 - t_{T+1} = 1)."""
    x1 = synth.make_latent_batch((1, 2, 4, 4), seed=12)
    c0, u0 = 0.7, -0.2
    res = R.cached_rollout(x1, [lambda x, t: np.full_like(x, c0), lambda x, t: np.full_like(x, u0)],
                           _grid(5), tau=0.0, k_warm=1, k_cool=1, guidance=5.0, mode=R.CACHE_OFF)
    np.testing.assert_allclose(res.latents[0], x1[0].astype(np.float64) - (u0 + 5.0 * (c0 - u0)), rtol=1e-12)


def test_euler_linear_velocity():
    """v(x) = lambda x, uniform grid: x_{T+1} = (1 - lambda/T)^T x_1 (uncached)."""
    x1 = synth.make_latent_batch((1, 2, 4, 4), seed=13)
    lam = 0.7
    res = R.cached_rollout(x1, [lambda x, t: lam * x], _grid(8), tau=0.0, k_warm=1, k_cool=1,
                           guidance=1.0, mode=R.CACHE_OFF)
    np.testing.assert_allclose(res.latents[0], (1 - lam / 8) ** 8 * x1[0].astype(np.float64), rtol=1e-12)


def test_score_is_normalised_projection():
    D = 2 * 4 * 4 * 2
    w = synth.make_latent_batch((D,), seed=1)
    e = np.zeros((D, 2, 2, 4, 4))
    e.reshape(D, -1)[np.arange(D), np.arange(D)] = 1.0
    s = R.score(e, w)
    np.testing.assert_allclose(s, w.astype(np.float64) / math.sqrt(D), rtol=1e-12)


# ------------------------------------------------------------- full DiT, tiny
@pytest.fixture(scope="module")
def tiny_b2():
    return synth.make_workload("tiny", n_branch=2, init="stress")


def test_tau0_reproduces_uncached_bitwise(tiny_b2):
    """Off mode recovers G(c, s); tau = 0 computes every call, bit for bit."""
    a = R.run_workload(tiny_b2, tau=0.0, n_cand=2)
    b = R.run_workload(tiny_b2, mode=R.CACHE_OFF, n_cand=2)
    assert a.n_compute == a.n_calls == b.n_calls
    assert np.array_equal(a.latents, b.latents)


def test_tau_inf_computes_only_forced(tiny_b2):
    res = R.run_workload(tiny_b2, tau=math.inf, n_cand=2)
    r = tiny_b2.roll
    for i in range(2):
        for b in range(2):
            assert sum(res.schedule(i, b)) == r.k_warm + r.k_cool


def test_branch_schedules_coincide(tiny_b2):
    """Both branches see the same latent, so their schedules coincide."""
    res = R.run_workload(tiny_b2, n_cand=2)
    for i in range(2):
        assert res.schedule(i, 0) == res.schedule(i, 1)
    assert 0 < res.n_compute < res.n_calls


def test_rollout_deterministic(tiny_b2):
    a = R.run_workload(tiny_b2, n_cand=1)
    b = R.run_workload(tiny_b2, n_cand=1)
    assert np.array_equal(a.latents, b.latents)


def test_x0_estimate_closed_form():
    """Constant velocity c: x_{k+1} = x_1 - (1 - t_{k+1}) c and the x0 estimate
    x_{k+1} - t_{k+1} c equals x_1 - c at every step (the exact endpoint)."""
    x1 = synth.make_latent_batch((2, 2, 4, 4), seed=21)
    c = 0.37
    for k in (1, 4, 7):
        res = R.cached_rollout(x1, [lambda x, t: np.full_like(x, c)], _grid(8), tau=0.0, k_warm=1, k_cool=1,
                               guidance=1.0, mode=R.CACHE_OFF, preview_step=k)
        np.testing.assert_allclose(res.x0_hat, x1.astype(np.float64) - c, rtol=1e-12, atol=1e-12)


def test_pruned_search_keeps_top_preview_and_matches_unpruned(tiny_b2):
    kept, prev, final, winner, res = R.pruned_search(tiny_b2, prune_step=4, keep=2)
    order = sorted(range(len(prev)), key=lambda i: (-prev[i], i))
    assert kept == sorted(order[:2])
    full = R.run_workload(tiny_b2)
    np.testing.assert_array_equal(res.latents, full.latents)   # preview does not perturb
    np.testing.assert_allclose(final, R.score(full.latents[kept], tiny_b2.scorer))
    assert winner in kept


# ------------------------------------------------------------- exact tie
def _exact_tie_run(fn=None):
    """v(x) = -x on the grid 1, 3/4, 1/2, 1/4, 0 with x_1 = 1: every value
    is a short dyadic fraction, so the indicator reaches tau = 1/4 exactly
    at step 2 (x_2 = 5/4 x_1; ||x_2 - x_1|| / ||x_1|| = 1/4)."""
    x1 = np.ones((1, 2, 4, 4))
    run = fn or R.cached_rollout
    return run(x1, [_neg], _grid(4), tau=0.25, k_warm=1, k_cool=1, guidance=1.0), x1


def test_indicator_equal_to_tau_skips():
    """Skip while a <= tau (Sec. Method, adaptive skip rule): at a = tau
    exactly the call reuses Delta.  Hand-derived: computes at 1, 3, 4;
    a = 1/4 at step 2 and 1/4 + 7/16 at step 3; x_5 = 2.24609375 x_1."""
    res, x1 = _exact_tie_run()
    assert res.schedule(0, 0) == [True, False, True, True]
    assert res.a_values(0, 0) == [None, 0.25, 0.6875, None]
    assert np.array_equal(res.latents, 2.24609375 * x1)


# -------------------------------------------- planted mistakes are caught
import inspect


def _planted(old, new):
    """A copy of the oracle's per-candidate rollout with one line changed."""
    src = inspect.getsource(R.cached_rollout_one)
    assert old in src, old
    ns = dict(R.__dict__)
    exec(compile(src.replace(old, new), "<planted>", "exec"), ns)
    return ns["cached_rollout_one"]


def _closed_form_holds():
    try:
        for case in json.load(open(os.path.join(GOLD, "cache_rule_closed_form.json")))["cases"]:
            test_closed_form_cache_schedule(case)
        test_indicator_equal_to_tau_skips()
    except AssertionError:
        return False
    return True


@pytest.mark.parametrize("old,new", [
    ("compute = not (a[b] <= tau)", "compute = not (a[b] < tau)"),          # strictness
    ("                a[b] = 0.0\n", ""),                                      # no reset after a compute
    ("den = math.sqrt(float(np.sum(xref[b] ** 2)))",
     "den = math.sqrt(float(np.sum(x ** 2)))"),                               # wrong normaliser
    ("v[b] = x + delta[b]", "v[b] = x - delta[b]"),                          # sign of the reuse
    ("x = x + (t_next - t_k) * vt", "x = x + (t_k - t_next) * vt"),          # Euler direction
])
def test_planted_rule_mistake_breaks_a_pin(monkeypatch, old, new):
    """Each plausible slip in the cache rule or the update fails one of the
    hand-derived pins above (the pins are not restatements of the code)."""
    assert _closed_form_holds()
    monkeypatch.setattr(R, "cached_rollout_one", _planted(old, new))
    assert not _closed_form_holds()
