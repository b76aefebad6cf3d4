"""GPU parity of attention-output broadcasting (PAB) against the oracle.

Rollouts with stored attention outputs reused on the schedule's steps are
compared with the float64 oracle (latents, scores, reuse counts) at tiny
shapes for fp32 and bf16, one and two guidance branches, and at Wan widths;
range 1 must reproduce the uncached rollout bit for bit; a zero output
projection makes reuse exact; calls PAB does not support fail with
CS_E_UNSUPPORTED or CS_E_INVAL."""
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

from oracle import rollout as orl
from paper_2607_23159_amd import binding as B
from paper_2607_23159_amd import synth
from paper_2607_23159_amd.search import GpuModel, Inputs, run_rollout
from parity import TOL, rel_l2


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.lib()


def pab_workload(name, n_branch, dtype, init="stress", n_cand=None, **kw):
    kw.setdefault("pab_self", 2)
    kw.setdefault("pab_cross", 3)
    return synth.make_workload(name, n_branch=n_branch, dtype=dtype, init=init, n_cand=n_cand,
                               mode=synth.CACHE_PAB, **kw)


def check_pab(gm, wl, dtype, W=None):
    r = wl.roll
    lat, sched = orl.pab_rollout(wl, W=W)
    g = run_rollout(gm, wl)
    S = r.n_cand * r.n_branch
    n_self = sum(1 for _, cs, _ in sched if not cs)
    n_cross = sum(1 for _, _, cc in sched if not cc)
    say(f"  reused steps self {n_self} cross {n_cross}; gpu counters {g.self_reused} {g.cross_reused}")
    assert (g.self_reused, g.cross_reused) == (n_self * S, n_cross * S)
    assert g.computed == g.calls == S * r.n_steps
    assert (g.masks == 1).all()
    for i in range(r.n_cand):
        err = rel_l2(g.latents[i], lat[i])
        say(f"  cand {i} rel_l2 {err:.3e}")
        assert err < TOL[dtype], (i, err)
    s_ref = orl.score(lat, wl.scorer)
    np.testing.assert_allclose(g.scores, s_ref, rtol=0, atol=TOL[dtype] * np.abs(s_ref).max() + 1e-9)
    return g, lat


@pytest.mark.parametrize("n_branch", [1, 2])
@pytest.mark.parametrize("dtype", [synth.DTYPE_FP32, synth.DTYPE_BF16])
def test_pab_rollout_tiny(dtype, n_branch):
    say(f"PAB rollout tiny dtype={dtype} B={n_branch}")
    wl = pab_workload("tiny", n_branch, dtype)
    gm = GpuModel(wl.model, wl.weights)
    g, lat = check_pab(gm, wl, dtype)
    # reuse really happened and changed the result against the uncached rollout
    off = run_rollout(gm, wl, mode=synth.CACHE_OFF)
    assert g.self_reused > 0 and g.cross_reused > 0
    assert rel_l2(g.latents, off.latents) > 1e-5


@pytest.mark.parametrize("n_branch", [1, 2])
def test_pab_rollout_wan_mid_bf16(n_branch):
    say(f"PAB rollout wan_mid bf16 B={n_branch} N=2, ranges 2 / 6")
    wl = pab_workload("wan_mid", n_branch, synth.DTYPE_BF16, init="paper", n_cand=2, pab_self=2,
                      pab_cross=6)
    gm = GpuModel(wl.model, wl.weights)
    check_pab(gm, wl, synth.DTYPE_BF16)


@pytest.mark.parametrize("dtype", [synth.DTYPE_FP32, synth.DTYPE_BF16])
def test_pab_range_one_bitwise_equals_off(dtype):
    wl = pab_workload("tiny", 2, dtype, pab_self=1, pab_cross=1)
    gm = GpuModel(wl.model, wl.weights)
    a = run_rollout(gm, wl)
    b = run_rollout(gm, wl, mode=synth.CACHE_OFF)
    assert a.self_reused == a.cross_reused == 0
    assert np.array_equal(a.latents, b.latents)
    assert np.array_equal(a.scores, b.scores)


def test_pab_zero_projection_reuse_matches_off():
    """fp32: with zero output projections the stored outputs are the biases,
    so reusing them must give the uncached result up to rounding."""
    wl = pab_workload("tiny", 2, synth.DTYPE_FP32, pab_self=2, pab_cross=3)
    m = wl.model
    named = synth.unflatten(m, wl.weights)
    for j in range(m.n_blocks):
        for key in (f"blk{j}.o_w", f"blk{j}.cao_w"):
            named[key] = np.zeros_like(named[key])
    flat = np.concatenate([named[n].ravel() for n, _, _ in synth.weight_spec(m)]).astype(np.float32)
    gm = GpuModel(m, flat)
    a = run_rollout(gm, wl)
    b = run_rollout(gm, wl, mode=synth.CACHE_OFF)
    assert a.self_reused > 0 and a.cross_reused > 0
    assert rel_l2(a.latents, b.latents) < 1e-6


def test_pab_unsupported_calls():
    wl = pab_workload("tiny", 1, synth.DTYPE_FP32)
    gm = GpuModel(wl.model, wl.weights)
    inp = Inputs(wl)
    r = wl.roll
    with pytest.raises(B.CsError) as e:
        B.cs_rollout_init(gm.h, B.RolloutDesc(r, wl.timesteps, pab_self=0), inp.x1, inp.ctx[0])
    assert e.value.status == B.CS_E_INVAL
    h = B.cs_rollout_init(gm.h, B.RolloutDesc(r, wl.timesteps), inp.x1, inp.ctx[0])
    try:
        with pytest.raises(B.CsError) as e:
            B.cs_cache_decide(h, 1, r.n_cand, np.ones(r.n_cand, np.uint8))
        assert e.value.status == B.CS_E_UNSUPPORTED
        with pytest.raises(B.CsError) as e:
            B.cs_rollout_export(h)
        assert e.value.status == B.CS_E_UNSUPPORTED
        with pytest.raises(B.CsError) as e:
            B.cs_rollout_retain(h, [0])
        assert e.value.status == B.CS_E_UNSUPPORTED
        # the rollout is still usable after the refused calls
        for k in range(1, r.n_steps + 1):
            B.cs_denoise_step(h, k)
        st = B.cs_rollout_stats(h)
        assert st.steps_done == r.n_steps
    finally:
        B.cs_rollout_free(h)
