"""GPU parity: the HIP path (through the C ABI) against the float64 oracle.

Velocity parity per model shape (tiny, Wan2.1-1.3B, Wan2.2-5B and
Wan2.1-14B widths at 384 tokens, one Wan2.1-1.3B block at the full 32,760
tokens on sampled tokens), rollout
parity (schedules, latents, scores, rankings) on the tiny workload for
fp32 and bf16, one and two guidance branches and tau in
{0, 0.05, 0.1, 0.2, inf}, and a Wan-width rollout."""
import math
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

from oracle import dit as odit
from oracle import rank as orank
from oracle import rollout as orl
from paper_2607_23159_amd import synth
from paper_2607_23159_amd import binding as B
from paper_2607_23159_amd.search import GpuModel, Inputs, run_rollout
from parity import TOL, check_ranking, compare_schedules, oracle_masks, rel_l2, row_errors, token_errors


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.lib()


_models = {}


def gpu_model(name, dtype, init):
    key = (name, dtype, init)
    if key not in _models:
        m = synth.MODELS[name].with_dtype(dtype)
        _models[key] = (GpuModel(m, synth.make_weights(m, init=init)), m)
    return _models[key]


def oracle_weights(m, init):
    return {k: v.astype(np.float64) for k, v in synth.unflatten(m, synth.make_weights(m, init=init)).items()}


# ----------------------------------------------------------------- velocity
@pytest.mark.parametrize("dtype", [synth.DTYPE_FP32, synth.DTYPE_BF16])
@pytest.mark.parametrize("init", ["paper", "stress"])
def test_velocity_tiny(dtype, init):
    say(f"velocity tiny dtype={dtype} init={init}")
    gm, m = gpu_model("tiny", dtype, init)
    W = oracle_weights(m, init)
    x = synth.make_noise(m, 3, seed0=500)
    ctx = synth.make_context(m, 1)
    for t in (1.0, 0.55, 0.05):
        v = gm.velocity(torch.from_numpy(x.reshape(3, -1)).cuda(), t, torch.from_numpy(ctx).cuda())
        v = v.cpu().numpy().reshape(x.shape)
        emb = odit.text_embedding(ctx, W)
        for i in range(3):
            ref = odit.velocity(x[i], t, emb, W, m)
            err = rel_l2(v[i], ref)
            tok = token_errors(v[i], ref).max()
            say(f"  t={t} i={i} rel_l2={err:.3e} max per-token {tok:.3e}")
            assert err < TOL[dtype] / 4
            assert tok < TOL[dtype]


@pytest.mark.parametrize("dtype", [synth.DTYPE_FP32, synth.DTYPE_BF16])
@pytest.mark.parametrize("init", ["paper", "stress"])
def test_velocity_wan_mid(init, dtype):
    """Wan2.1-1.3B widths (d = 1536, 12 x 128 heads, FFN 8960, 2 blocks, 384
    tokens) in both arithmetic paths."""
    say(f"velocity wan_mid dtype={dtype} init={init}")
    gm, m = gpu_model("wan_mid", dtype, init)
    W = oracle_weights(m, init)
    x = synth.make_noise(m, 2, seed0=600)
    ctx = synth.make_context(m, 1)
    v = gm.velocity(torch.from_numpy(x.reshape(2, -1)).cuda(), 0.7, torch.from_numpy(ctx).cuda())
    v = v.cpu().numpy().reshape(x.shape)
    emb = odit.text_embedding(ctx, W)
    for i in range(2):
        ref = odit.velocity(x[i], 0.7, emb, W, m)
        err = rel_l2(v[i], ref)
        tok = token_errors(v[i], ref).max()
        say(f"  i={i} rel_l2={err:.3e} max per-token {tok:.3e}")
        assert err < TOL[dtype] / 2
        assert tok < TOL[dtype]


@pytest.mark.parametrize("name", ["wan5b_mid", "wan14b_mid"])
def test_velocity_wide_models_bf16(name):
    """Wan2.2-5B and Wan2.1-14B widths (d = 3072 / 5120, 24 / 40 heads, FFN
    14336 / 13824, 2 blocks, 384 tokens): the widest projections and head
    counts the workloads use, against the oracle."""
    say(f"velocity {name} bf16 stress init")
    m = synth.MODELS[name].with_dtype(synth.DTYPE_BF16)
    flat = synth.make_weights(m, init="stress")
    W = {k: v.astype(np.float64) for k, v in synth.unflatten(m, flat).items()}
    gm = GpuModel(m, flat)
    try:
        x = synth.make_noise(m, 1, seed0=650)
        ctx = synth.make_context(m, 1)
        v = gm.velocity(torch.from_numpy(x.reshape(1, -1)).cuda(), 0.6, torch.from_numpy(ctx).cuda())
        v = v.cpu().numpy().reshape(x.shape)
        ref = odit.velocity(x[0], 0.6, odit.text_embedding(ctx, W), W, m)
        err = rel_l2(v[0], ref)
        tok = token_errors(v[0], ref).max()
        say(f"  rel_l2={err:.3e} max per-token {tok:.3e}")
        assert err < TOL[0] / 2
        assert tok < TOL[0]
    finally:
        gm.close()


def test_velocity_full_length_block_sampled():
    """One Wan2.1-1.3B block at 32,760 tokens (ragged last key tile, 256-row
    GEMM tail), checked on sampled tokens."""
    say("velocity wan13b_block1 bf16 full length, sampled tokens")
    gm, m = gpu_model("wan13b_block1", synth.DTYPE_BF16, "stress")
    W = oracle_weights(m, "stress")
    x = synth.make_noise(m, 1, seed0=700)
    ctx = synth.make_context(m, 1)
    v = gm.velocity(torch.from_numpy(x.reshape(1, -1)).cuda(), 0.8, torch.from_numpy(ctx).cuda())
    vp = odit.patchify(v.cpu().numpy().reshape(x.shape[1:]), 1, 2, 2)
    rows = np.array([0, 1, 63, 255, 256, 4097, 16383, 32511, 32512, 32700, 32759])
    ref = odit.velocity(x[0], 0.8, odit.text_embedding(ctx, W), W, m, last_block_rows=rows)
    err = rel_l2(vp[rows], ref)
    tok = row_errors(vp[rows], ref)
    say(f"  sampled rel_l2={err:.3e} per-token {np.round(tok, 5).tolist()}")
    assert err < TOL[0] / 2
    assert tok.max() < TOL[0] / 2      # every sampled token on its own, same bar


def test_batch_invariance_velocity():
    """A latent's velocity is bitwise the same alone or inside a batch."""
    gm, m = gpu_model("tiny", synth.DTYPE_BF16, "stress")
    x = torch.from_numpy(synth.make_noise(m, 5, seed0=800).reshape(5, -1)).cuda()
    ctx = torch.from_numpy(synth.make_context(m, 1)).cuda()
    full = gm.velocity(x, 0.4, ctx)
    for i in (0, 2, 4):
        one = gm.velocity(x[i:i + 1].contiguous(), 0.4, ctx)
        assert torch.equal(one[0], full[i])
    two = gm.velocity(x[1:3].contiguous(), 0.4, ctx)
    assert torch.equal(two, full[1:3])


# ------------------------------------------------------------------ rollouts
_oracle_cache = {}


def oracle_rollout(wl, tau, mode=None, key=None):
    k = (key, tau, mode)
    if k not in _oracle_cache:
        _oracle_cache[k] = orl.run_workload(wl, tau=tau, mode=mode)
    return _oracle_cache[k]


_wls = {}


def workload(name, n_branch, init, dtype):
    k = (name, n_branch, init, dtype)
    if k not in _wls:
        _wls[k] = synth.make_workload(name, n_branch=n_branch, init=init, dtype=dtype)
    return _wls[k]


def check_rollout(gm, wl, tau, dtype, okey):
    """The cached rollout against the oracle's: schedules exact (a flip is
    excused only within 1e-3 relative of tau, and that rollout is then
    compared in replay mode), latents within the relative L2 bar and every
    token within twice it, scores within the bar, and rankings exact except
    swapped pairs that involve an excused flip or lie within the score
    error (parity.check_ranking)."""
    r = wl.roll
    res = oracle_rollout(wl, tau, key=okey)
    om, oa = oracle_masks(res, r.n_cand, r.n_branch, r.n_steps)
    g0 = run_rollout(gm, wl, tau=tau)
    excused = compare_schedules(g0.masks, om, oa, tau)
    say(f"  tau={tau} computed gpu {g0.computed}/{g0.calls} oracle {res.n_compute}/{res.n_calls} excused={excused}")
    g = g0
    if excused:
        g = run_rollout(gm, wl, tau=tau, override=om)
        assert np.array_equal(g.masks, om)
    for i in range(r.n_cand):
        err = rel_l2(g.latents[i], res.latents[i])
        tok = token_errors(g.latents[i], res.latents[i]).max()
        assert err < TOL[dtype], (i, err)
        assert tok < 2 * TOL[dtype], (i, tok)
    s_ref = orl.score(res.latents, wl.scorer)
    np.testing.assert_allclose(g.scores, s_ref, rtol=0, atol=TOL[dtype] * np.abs(s_ref).max() + 1e-9)
    # ranking of the rollout as run (not replayed) against the oracle's
    gap_tol = 4 * np.abs(g.scores - s_ref).max()
    check_ranking(g0.scores, s_ref, gap_tol, {s // r.n_branch for s in excused})
    return g, res


@pytest.mark.parametrize("n_branch", [1, 2])
@pytest.mark.parametrize("dtype", [synth.DTYPE_FP32, synth.DTYPE_BF16])
def test_rollout_tiny(dtype, n_branch):
    say(f"rollout tiny dtype={dtype} B={n_branch}")
    gm, m = gpu_model("tiny", dtype, "stress")
    wl = workload("tiny", n_branch, "stress", dtype)
    for tau in (0.0, 0.05, 0.1, 0.2, math.inf):
        check_rollout(gm, wl, tau, dtype, okey=("tiny", n_branch))


@pytest.mark.parametrize("n_branch", [1, 2])
@pytest.mark.parametrize("dtype", [synth.DTYPE_FP32, synth.DTYPE_BF16])
def test_rollout_tiny_paper_init(dtype, n_branch):
    """The tiny workload exactly as its configuration states it: random
    init N(0, 0.02), N = 4 candidates, T = 10 Euler steps, tau = 0.1 (plus
    the rest of the tau set), scored by the fixed projection and ranked."""
    say(f"rollout tiny paper init dtype={dtype} B={n_branch}")
    gm, m = gpu_model("tiny", dtype, "paper")
    wl = workload("tiny", n_branch, "paper", dtype)
    assert (wl.roll.n_cand, wl.roll.n_steps, wl.roll.tau) == (4, 10, 0.1)
    for tau in (0.1, 0.0, 0.05, 0.2, math.inf):
        check_rollout(gm, wl, tau, dtype, okey=("tiny_paper", n_branch))


@pytest.mark.parametrize("n_branch", [1, 2])
def test_no_warmup_window_computes_until_first_delta(n_branch):
    """K_w = 0 (and K_c = 0): no step is forced by a window, yet the first
    step of every branch computes because no Delta exists yet (Alg. 1 resets
    the cache; the indicator rule can only skip once a reference is stored).
    With tau = inf that is the only computed step; with tau = 0.1 the
    schedule follows the oracle's."""
    gm, m = gpu_model("tiny", synth.DTYPE_FP32, "stress")
    wl = synth.make_workload("tiny", n_branch=n_branch, init="stress", dtype=synth.DTYPE_FP32,
                             k_warm=0, k_cool=0)
    r = wl.roll
    g = run_rollout(gm, wl, tau=math.inf)
    want = np.zeros((r.n_steps, r.n_cand * n_branch), np.uint8)
    want[0] = 1
    assert np.array_equal(g.masks, want)
    assert np.isnan(g.a[0]).all() and not np.isnan(g.a[1:]).any()
    res = orl.run_workload(wl, tau=math.inf)
    om, _ = oracle_masks(res, r.n_cand, n_branch, r.n_steps)
    assert np.array_equal(om, want)
    for i in range(r.n_cand):
        assert rel_l2(g.latents[i], res.latents[i]) < TOL[1]
    check_rollout(gm, wl, 0.1, synth.DTYPE_FP32, okey=("tiny_kw0", n_branch))


A_RTOL = {synth.DTYPE_FP32: 1e-6, synth.DTYPE_BF16: 5e-3}   # measured: 6e-8 / 7.5e-4


@pytest.mark.parametrize("n_branch", [1, 2])
@pytest.mark.parametrize("dtype", [synth.DTYPE_FP32, synth.DTYPE_BF16])
def test_indicator_values_match_oracle(dtype, n_branch):
    """The accumulated drift statistic a (Eq. indicator) the decision kernel
    reports at every step, on the oracle's schedule (replay, so both sides
    follow the same trajectory): present on exactly the steps where the
    oracle evaluates the rule, and equal to the oracle's value within the
    latents' agreement (fp32 path: 1e-6 relative; bf16: 5e-3)."""
    gm, m = gpu_model("tiny", dtype, "stress")
    wl = workload("tiny", n_branch, "stress", dtype)
    r = wl.roll
    res = oracle_rollout(wl, 0.1, key=("tiny", n_branch))
    om, oa = oracle_masks(res, r.n_cand, r.n_branch, r.n_steps)
    g = run_rollout(gm, wl, tau=0.1, override=om)
    assert np.array_equal(g.masks, om)
    assert np.array_equal(np.isnan(g.a), np.isnan(oa))
    both = ~np.isnan(oa)
    assert both.sum() > 0
    rel = np.abs(g.a[both] - oa[both]) / np.abs(oa[both])
    say(f"indicator dtype={dtype} B={n_branch}: {both.sum()} values, max rel diff {rel.max():.3e}")
    assert rel.max() < A_RTOL[dtype]


@pytest.mark.parametrize("n_branch", [1, 2])
def test_rollout_wan_mid_bf16(n_branch):
    """Wan2.1-1.3B widths (head dim 128, K = 1536 and 8960 projections):
    conditional only, and with classifier-free guidance (two branches)."""
    say(f"rollout wan_mid bf16 B={n_branch} N=2")
    gm, m = gpu_model("wan_mid", synth.DTYPE_BF16, "paper")
    wl = synth.make_workload("wan_mid", n_branch=n_branch, init="paper", n_cand=2)
    g, res = check_rollout(gm, wl, 0.1, synth.DTYPE_BF16, okey=("wan_mid", n_branch))
    assert 0 < res.n_compute < res.n_calls


# ---------------------------------------------------------------- invariants
@pytest.mark.parametrize("dtype", [synth.DTYPE_FP32, synth.DTYPE_BF16])
def test_tau0_bitwise_equals_off(dtype):
    gm, m = gpu_model("tiny", dtype, "stress")
    wl = workload("tiny", 2, "stress", dtype)
    a = run_rollout(gm, wl, tau=0.0)
    b = run_rollout(gm, wl, mode=synth.CACHE_OFF)
    assert a.computed == a.calls == b.computed
    assert np.array_equal(a.latents, b.latents)
    assert np.array_equal(a.scores, b.scores)


def test_tau_inf_forced_only_and_branches_coincide():
    gm, m = gpu_model("tiny", synth.DTYPE_BF16, "stress")
    wl = workload("tiny", 2, "stress", synth.DTYPE_BF16)
    g = run_rollout(gm, wl, tau=math.inf)
    r = wl.roll
    assert (g.masks.sum(axis=0) == r.k_warm + r.k_cool).all()
    g = run_rollout(gm, wl, tau=0.1)
    for i in range(r.n_cand):
        assert np.array_equal(g.masks[:, 2 * i], g.masks[:, 2 * i + 1])


def test_static_mode_schedule():
    gm, m = gpu_model("tiny", synth.DTYPE_FP32, "stress")
    wl = synth.make_workload("tiny", dtype=synth.DTYPE_FP32, init="stress", mode=synth.CACHE_STATIC,
                             static_k=3, k_warm=2, k_cool=2)
    g = run_rollout(gm, wl)
    want = [1 if k in (1, 2, 5, 8, 9, 10) else 0 for k in range(1, 11)]
    assert (g.masks == np.array(want, np.uint8)[:, None]).all()
    res = orl.run_workload(wl)
    for i in range(wl.roll.n_cand):
        assert rel_l2(g.latents[i], res.latents[i]) < TOL[1]


def test_degenerate_schedules():
    """Degenerate settings of the skip rule (Sec. Method, adaptive skip rule
    and its static variant): the static period 1 computes every call and the
    literal warmup and cooldown windows K_w = K_c = 5 at T = 10 force every
    call even at tau = inf, both bitwise equal to the uncached rollout; a
    one-step rollout (T = 1, its only call forced) matches the oracle."""
    gm, m = gpu_model("tiny", synth.DTYPE_BF16, "stress")
    wl = workload("tiny", 2, "stress", synth.DTYPE_BF16)
    off = run_rollout(gm, wl, mode=synth.CACHE_OFF)
    st1 = synth.make_workload("tiny", n_branch=2, dtype=synth.DTYPE_BF16, init="stress",
                              mode=synth.CACHE_STATIC, static_k=1)
    for w, kw in ((st1, {}), (synth.make_workload("tiny", n_branch=2, dtype=synth.DTYPE_BF16, init="stress",
                                                  k_warm=5, k_cool=5), {"tau": math.inf})):
        g = run_rollout(gm, w, **kw)
        assert g.computed == g.calls == off.calls
        assert np.array_equal(g.latents, off.latents) and np.array_equal(g.scores, off.scores)
    for dtype in (synth.DTYPE_FP32, synth.DTYPE_BF16):
        gm1, _ = gpu_model("tiny", dtype, "stress")
        one = synth.make_workload("tiny", n_branch=2, dtype=dtype, init="stress", n_steps=1)
        assert list(one.timesteps) == [1.0, 0.0]
        g = run_rollout(gm1, one)
        assert g.masks.shape == (1, 2 * one.roll.n_cand) and g.masks.all()
        res = orl.run_workload(one)
        for i in range(one.roll.n_cand):
            err = rel_l2(g.latents[i], res.latents[i])
            say(f"  T=1 dtype={dtype} i={i} rel_l2={err:.3e}")
            assert err < TOL[dtype]


def test_replay_override_follows_given_schedule():
    gm, m = gpu_model("tiny", synth.DTYPE_FP32, "stress")
    wl = workload("tiny", 1, "stress", synth.DTYPE_FP32)
    T, S = wl.roll.n_steps, wl.roll.n_cand
    ovr = np.zeros((T, S), np.uint8)
    ovr[0] = 1
    ovr[4] = 1
    ovr[8] = 1
    ovr[-1] = 1
    g = run_rollout(gm, wl, override=ovr)
    assert np.array_equal(g.masks, ovr)
    # the same schedule in the oracle (velocity calls replayed via STATIC-like mask)
    W = {k: v.astype(np.float64) for k, v in wl.named_weights().items()}
    fns = orl.dit_velocity_fns(W, wl.model, wl.ctx[:1])
    # k_warm=1, k_cool=1, static period 4 computes steps 1, 5, 9, 10
    res = orl.cached_rollout(wl.noise, fns, [float(t) for t in wl.timesteps], tau=0.0, k_warm=1, k_cool=1,
                             guidance=5.0, mode=orl.CACHE_STATIC, static_k=4)
    om, _ = oracle_masks(res, S, 1, T)
    assert np.array_equal(om, ovr)
    for i in range(S):
        assert rel_l2(g.latents[i], res.latents[i]) < TOL[1]


def test_checkpoint_resume_bitwise():
    gm, m = gpu_model("tiny", synth.DTYPE_BF16, "stress")
    wl = workload("tiny", 2, "stress", synth.DTYPE_BF16)
    ref = run_rollout(gm, wl, tau=0.1, record=False)
    inp = Inputs(wl)
    r = wl.roll
    desc = B.RolloutDesc(r, wl.timesteps, tau=0.1)
    h = B.cs_rollout_init(gm.h, desc, inp.x1, inp.ctx[0], inp.ctx[1])
    for k in range(1, 5):
        B.cs_denoise_step(h, k)
    blob = B.cs_rollout_export(h)
    B.cs_rollout_free(h)
    h2 = B.cs_rollout_init(gm.h, desc, inp.x1, inp.ctx[0], inp.ctx[1])
    B.cs_rollout_import(h2, blob)
    with pytest.raises(B.CsError) as e:
        B.cs_denoise_step(h2, 4)
    assert e.value.status == B.CS_E_STATE
    for k in range(5, r.n_steps + 1):
        B.cs_denoise_step(h2, k)
    out = torch.empty_like(inp.x1)
    B.cs_rollout_latents(h2, out)
    torch.cuda.synchronize()
    B.cs_rollout_free(h2)
    assert np.array_equal(out.cpu().numpy().reshape(ref.latents.shape), ref.latents)


@pytest.mark.parametrize("dtype", [synth.DTYPE_FP32, synth.DTYPE_BF16])
def test_static_schedule_at_the_adaptive_skip_fraction(dtype):
    """The uniform baseline at a matched budget: the static period whose
    skip fraction is closest to the adaptive rule's (tau = 0.1) is run on the
    GPU and in the oracle; schedules equal, latents within the bar, and both
    rankings are compared with the full rollouts' on each side (the GPU's
    rho / top-1 must equal the oracle's unless a near tie)."""
    import bench
    gm, m = gpu_model("tiny", dtype, "stress")
    wl = workload("tiny", 1, "stress", dtype)
    r = wl.roll
    res_a = oracle_rollout(wl, 0.1, key=("tiny", 1))
    skip = 1.0 - res_a.n_compute / res_a.n_calls
    k = bench.matched_static_period(r.n_steps, r.k_warm, r.k_cool, skip)
    say(f"static at matched skip: adaptive skip {skip:.2f}, period {k}")
    import dataclasses
    wl_s = synth.Workload(wl.name, wl.model, dataclasses.replace(r, mode=synth.CACHE_STATIC, static_k=k),
                          wl.weights, wl.ctx, wl.noise, wl.scorer, wl.timesteps)
    g = run_rollout(gm, wl_s)
    res_s = orl.run_workload(wl_s)
    om, _ = oracle_masks(res_s, r.n_cand, 1, r.n_steps)
    assert np.array_equal(g.masks, om)
    assert g.computed == res_s.n_compute == r.n_cand * bench.static_computes(r.n_steps, r.k_warm, r.k_cool, k)
    for i in range(r.n_cand):
        assert rel_l2(g.latents[i], res_s.latents[i]) < TOL[dtype]
    s_ref = orl.score(res_s.latents, wl.scorer)
    check_ranking(g.scores, s_ref, 4 * np.abs(g.scores - s_ref).max())
    full = oracle_rollout(wl, 0.0, mode=orl.CACHE_OFF, key=("tiny", 1))
    f_ref = orl.score(full.latents, wl.scorer)
    _, _, rho_o, top1_o, _ = orank.rank_report(list(s_ref), list(f_ref))
    g_full = run_rollout(gm, wl, mode=synth.CACHE_OFF)
    _, _, rho_g, top1_g = B.cs_rank(g.scores, g_full.scores)
    say(f"  static: rho gpu {rho_g} oracle {rho_o}, top-1 gpu {top1_g} oracle {top1_o}")
    if np.min(np.diff(np.sort(s_ref))) > 4 * np.abs(g.scores - s_ref).max() and \
            np.min(np.diff(np.sort(f_ref))) > 4 * np.abs(g_full.scores - f_ref).max():
        assert rho_g == pytest.approx(rho_o, abs=1e-12) and top1_g == top1_o


def test_decision_log_matches_oracle_log():
    """The per-call decision log written from a GPU rollout (fp32 path,
    tau = 0.1) equals the oracle's own decision log call by call: same
    decisions, forced calls without an indicator, indicators within 1e-6."""
    from paper_2607_23159_amd.search import decision_records
    gm, m = gpu_model("tiny", synth.DTYPE_FP32, "stress")
    wl = workload("tiny", 2, "stress", synth.DTYPE_FP32)
    res = oracle_rollout(wl, 0.1, key=("tiny", 2))
    g = run_rollout(gm, wl, tau=0.1)
    recs = {(d["k"], d["i"], d["b"]): d for d in decision_records(g.masks, g.a, 2)}
    assert len(recs) == len(res.log) == wl.roll.n_cand * 2 * wl.roll.n_steps
    for o in res.log:
        d = recs[(o.k, o.i, o.b)]
        assert d["decision"] == ("compute" if o.compute else "skip"), (o, d)
        if o.a is None:
            assert d["a"] is None
        else:
            assert d["a"] == pytest.approx(o.a, rel=1e-6)
